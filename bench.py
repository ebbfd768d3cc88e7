"""PACE hot-path benchmark on one MI355X.

A step is one pass of every hot-path kernel over the 4K-frame workload
(3836x2156 RGB image, Qwen2.5-VL-7B shapes): APC density and 2x downsample of the
image, vision-encoder window attention (700 windows of <= 64 patches, 16 heads,
d = 80) and full attention over 42,196 patches with the per-key mass, causal GQA
prefill over 10,549 visual + 128 text tokens (28/4 heads, d = 128) with the
text-query mass of every visual key, and DDAE fusion + top-K (10%) + gather of the
kept rows of a 10,549 x 3584 bf16 hidden-state matrix.  Inputs are synthetic and
seeded, already resident in HBM when the timed region starts.

Prints one JSON line.  `value` is the step's algorithmic attention FLOP rate
(all three attention passes' 4*d*(visible pairs)*heads, over the whole step time).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "attn_fwd_rot_vit_full_frame4k_traffic.md")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2608_27206_amd", "csrc", "attention.hip")


def measured_traffic():
    """HBM bytes per launch of the dominant kernel from the committed rocprofv3 counter summary,
    or None when there is none or the kernel source changed since the counters were taken."""
    import hashlib
    try:
        txt = open(TRAFFIC_SUMMARY).read()
        src = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()
    except OSError:
        return None
    vals = {}
    for line in txt.splitlines():
        if ":" in line and line.strip().startswith("- "):
            k, v = line.strip()[2:].split(":", 1)
            vals[k.strip()] = v.strip().strip("`")
    if vals.get("kernel_source_sha256") != src:
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3, help="workload id (3 = 4K frame)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="wall-clock budget of the oracle CPU baseline sample (0 = skip)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="before warm-up, copy this many MiB device to device once (a plain copy "
                         "of known size that calibrates the HBM byte counters of a profile run)")
    ap.add_argument("--no-graph", dest="graph", action="store_false",
                    help="skip timing the step captured in a HIP graph and replayed")
    return ap.parse_args()


def time_graph_replays(torch, step, stream, steps):
    """The same step captured once in a HIP graph and replayed `steps` times (after the timed eager
    steps, outside their region): the per-step time without host launch overhead."""
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        step(None)
    stream.wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(None)
    g.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def main():
    a = parse()
    if a.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only; --gpus must be 1 "
                          "(multi-GPU sharding is described in the design notes, not built)"}))
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2608_27206_amd import pace
    from paper_2608_27206_amd import workloads as wl

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    w = wl.make_workload(a.config)
    L = w.layouts[0]
    img_np = w.images[0]
    H, W, _ = img_np.shape
    vit, pre = w.vit, w.prefill

    def bf(x):
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)

    def i32(x):
        return torch.from_numpy(np.asarray(x, np.int32)).to(dev)

    img = torch.from_numpy(img_np).to(dev)
    vq, vk, vv = bf(vit.q), bf(vit.k), bf(vit.v)
    cu_win, cu_full = i32(vit.cu_windows), i32(vit.cu_full)
    max_win = int(np.diff(vit.cu_windows).max())
    Np, Hv, dv = vit.q.shape
    pq, pk, pv = bf(pre.q), bf(pre.k), bf(pre.v)
    p_cu, p_vis, p_cuv = i32(pre.cu_seqlens), i32(pre.vis_len), i32(pre.cu_vis)
    p_mqs, p_mql = i32(pre.mq_start), i32(pre.mq_len)
    S = int(pre.cu_seqlens[-1])
    Nv = int(pre.vis_len[0])
    T = int(pre.text_len[0])
    Hq, Hkv, dq = pre.q.shape[1], pre.k.shape[1], pre.q.shape[2]
    hidden = bf(w.hidden)
    perm = i32(vit.vis_perm)
    K = pace.keep_count(w.keep_ratio, Nv)
    oH, oW = (int(round(H * w.downsample_scale)), int(round(W * w.downsample_scale))) \
        if w.downsample_scale else pace.apc_target_size(0.5, H, W, 0, 1e18, 28)

    # outputs and workspaces, allocated once
    f32 = dict(dtype=torch.float32, device=dev)
    rho = torch.empty(4, **f32)
    dpatch = torch.empty(L.n_patches, **f32)
    ws_apc = torch.empty(pace.lib().pace_apc_density_workspace_size(H, W, 14), dtype=torch.uint8, device=dev)
    small = torch.empty((oH, oW, 3), dtype=torch.uint8, device=dev)
    o_win = torch.empty_like(vq)
    lse_win = torch.empty((Hv, Np), **f32)
    mass_win = torch.empty((Hv, Np), **f32)
    o_full = torch.empty_like(vq)
    lse_full = torch.empty((Hv, Np), **f32)
    mass_vis = torch.empty((Hv, Np), **f32)
    o_pre = torch.empty_like(pq)
    lse_pre = torch.empty((Hq, S), **f32)
    mass_llm = torch.empty((Hq, Nv), **f32)
    idx = torch.empty(K, dtype=torch.int32, device=dev)
    scores = torch.empty(Nv, **f32)
    fuse = torch.empty((1, 4), **f32)
    kept = torch.empty((K, hidden.shape[1]), dtype=hidden.dtype, device=dev)
    ws_sel = torch.empty(pace.lib().pace_ddae_select_workspace_size(Nv, 1), dtype=torch.uint8, device=dev)
    ws_vit = torch.empty(pace.lib().pace_vit_attention_workspace_size(Np, Hv, dv, 1, Np), dtype=torch.uint8,
                         device=dev)

    stream = torch.cuda.current_stream()
    names = ("apc", "resize", "vit_win", "vit_fwd", "vit_mass", "prefill", "select")

    def new_events():
        return {n: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                for n in names}

    # The vision mass pass needs only the forward's LSE, and the LLM prefill needs neither it nor
    # its result (it takes the vision encoder's output, which the forward has produced): the two
    # run side by side, the mass on a second stream (default priority), and the selection waits
    # for both.  The mass kernel's last round of workgroups leaves CUs idle that the prefill fills.
    side = torch.cuda.Stream()

    def run(name, fn, ev):
        cur = torch.cuda.current_stream()
        if ev is not None:
            ev[name][0].record(cur)
        fn()
        if ev is not None:
            ev[name][1].record(cur)

    def step(ev, overlap=True):
        run("apc", lambda: pace.apc_density(img, 14, 0.10, 0.6, 1.5, d_out=dpatch, rho_out=rho,
                                            workspace=ws_apc), ev)
        run("resize", lambda: pace.apc_downsample(img, oH, oW, dst=small), ev)
        run("vit_win", lambda: pace.vit_attention(vq, vk, vv, cu_win, max_win, o=o_win, lse=lse_win,
                                                  mass=mass_win), ev)
        run("vit_fwd", lambda: pace.vit_attention(vq, vk, vv, cu_full, Np, o=o_full, lse=lse_full,
                                                  want_mass=False, workspace=ws_vit), ev)
        def vis_mass():
            pace.vit_attention_mass(vq, vk, cu_full, Np, lse_full, mass=mass_vis)

        def prefill():
            pace.prefill_attention_with_mass(pq, pk, pv, p_cu, S, p_vis, p_cuv, Nv, Nv, p_mqs, p_mql, T,
                                             o=o_pre, lse=lse_pre, mass=mass_llm)
        if overlap:
            cur = torch.cuda.current_stream()
            side.wait_stream(cur)
            with torch.cuda.stream(side):
                vis_mass()
            prefill()
            cur.wait_stream(side)
        else:
            run("vit_mass", vis_mass, ev)
            run("prefill", prefill, ev)
        run("select", lambda: pace.ddae_select(mass_vis, 4, perm, mass_llm, [Nv], [K], mode=w.fusion_mode,
                                               tau=w.tau, hidden=hidden, idx_out=idx, score_out=scores,
                                               fuse_out=fuse, out=kept, workspace=ws_sel), ev)

    if a.copy_calibration_mib > 0:
        nbytes = a.copy_calibration_mib << 20
        c_src = torch.empty(nbytes, dtype=torch.uint8, device=dev).fill_(1)
        c_dst = torch.empty_like(c_src)
        torch.cuda.synchronize()
        c_dst.copy_(c_src)
        torch.cuda.synchronize()
        del c_src, c_dst
    for _ in range(a.warmup):
        step(None)
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record(stream)
    for i in range(a.steps):
        step(None)
    t_end.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t_start.elapsed_time(t_end) / a.steps
    # per-part times from the same number of steps run serially on one stream (after the timed
    # region: the side-by-side parts would otherwise time each other's share of the GPU)
    step_events = [new_events() for _ in range(a.steps)]
    s_start = torch.cuda.Event(enable_timing=True)
    s_end = torch.cuda.Event(enable_timing=True)
    s_start.record(stream)
    for i in range(a.steps):
        step(step_events[i], overlap=False)
    s_end.record(stream)
    torch.cuda.synchronize()
    serial_ms = s_start.elapsed_time(s_end) / a.steps
    per = {n: 0.0 for n in names}
    for ev in step_events:
        for n in names:
            per[n] += ev[n][0].elapsed_time(ev[n][1])
    per = {n: v / a.steps for n, v in per.items()}
    graph_ms = time_graph_replays(torch, step, stream, a.steps) if a.graph else None
    nxt = measure_next(pace, pq, pk, pv, p_cu, S, p_vis, p_cuv, Nv, T, idx, K, stream)
    nxt["preview_block"] = measure_preview(pace, wl, img, L, stream)

    # algorithmic work
    win_sizes = np.diff(vit.cu_windows).astype(np.float64)
    flop_win = 4.0 * dv * Hv * float(np.sum(win_sizes ** 2))
    flop_full = 4.0 * dv * Hv * float(Np) ** 2
    flop_pre = 4.0 * dq * Hq * (S * (S + 1) / 2.0)
    flop_attn = flop_win + flop_full + flop_pre
    bytes_win = 4.0 * Np * Hv * dv * 2 + 2.0 * Hv * Np * 4
    bytes_sel = Hv * Np * 4 + Hq * Nv * 4 + 4 * K + 2.0 * K * hidden.shape[1] * 2
    bytes_apc = H * W * 3 + 4.0 * L.n_patches
    bytes_resize = H * W * 3 + oH * oW * 3
    t_fwd = per["vit_fwd"] * 1e-3
    achieved = flop_full / t_fwd / 1e12 if t_fwd > 0 else 0.0
    value = flop_attn / (ms_per_step * 1e-3) / 1e12

    result = {
        "metric": "attn TFLOP/s (% bf16 MFMA peak) + DDAE select tokens/s (% HBM BW), 1 GPU",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Qwen2.5-VL-7B-shaped inputs)",
        "config": {"workload": wl.CONFIG_NAMES[a.config], "image": f"{W}x{H}",
                   "vit_patches": int(Np), "vit_heads": int(Hv), "vit_head_dim": int(dv),
                   "windows": int(len(win_sizes)), "prefill_tokens": S, "visual_tokens": Nv,
                   "text_tokens": T, "llm_heads": f"{Hq}/{Hkv}", "llm_head_dim": int(dq),
                   "keep": K, "hidden": int(hidden.shape[1]), "resize_to": f"{oW}x{oH}"},
        "roofline": {"kernel": "attn_fwd_rot<80> (vision full attention, 42,196 patches x 16 heads)",
                     "bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic()},
        "schedule": "vision mass on a second stream beside the prefill; breakdown_ms and step_roofline "
                    "from the same steps run serially on one stream",
        "serial_ms_per_step": round(serial_ms, 4),
        "breakdown_ms": {n: round(v, 4) for n, v in per.items()},
        "graph_ms_per_step": None if graph_ms is None else round(graph_ms, 4),
        "attention": {
            "vit_full_fwd_tflops": round(achieved, 2),
            "vit_full_fwd_plus_mass_tflops": round(flop_full / ((per["vit_fwd"] + per["vit_mass"]) * 1e-3) / 1e12, 2)
            if per["vit_fwd"] + per["vit_mass"] > 0 else None,
            "prefill_fwd_plus_mass_tflops": round(flop_pre / (per["prefill"] * 1e-3) / 1e12, 2)
            if per["prefill"] > 0 else None,
            "vit_window_gbs": round(bytes_win / (per["vit_win"] * 1e-3) / 1e9, 1) if per["vit_win"] > 0 else None,
        },
        "select": {
            "tokens_per_s": round(Nv / (per["select"] * 1e-3), 1) if per["select"] > 0 else None,
            "gbs": round(bytes_sel / (per["select"] * 1e-3) / 1e9, 1) if per["select"] > 0 else None,
            "hbm_frac": round(bytes_sel / (per["select"] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4) if per["select"] > 0 else None,
        },
        "apc": {
            "density_gbs": round(bytes_apc / (per["apc"] * 1e-3) / 1e9, 1) if per["apc"] > 0 else None,
            "resize_gbs": round(bytes_resize / (per["resize"] * 1e-3) / 1e9, 1) if per["resize"] > 0 else None,
        },
        # every step of the path against the roofline that bounds it (algorithmic work per step)
        "step_roofline": {
            "apc_density": _hbm_row(bytes_apc, per["apc"]),
            "apc_downsample": _hbm_row(bytes_resize, per["resize"]),
            "vit_window_attention": _hbm_row(bytes_win, per["vit_win"]),
            "vit_full_attention_fwd": _mfma_row(flop_full, per["vit_fwd"]),
            "vit_full_attention_fwd_plus_mass": _mfma_row(flop_full, per["vit_fwd"] + per["vit_mass"]),
            "prefill_attention_with_mass": _mfma_row(flop_pre, per["prefill"]),
            "ddae_select_gather": _hbm_row(bytes_sel, per["select"]),
        },
        "next": nxt,
    }
    if a.cpu_seconds > 0:
        result["cpu_baseline"] = cpu_baseline(vit, a.cpu_seconds)
    print(json.dumps(result), flush=True)


def _hbm_row(nbytes, ms):
    if ms <= 0:
        return None
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "ms": round(ms, 4), "algorithmic_bytes": int(nbytes), "achieved": round(gbs, 1),
            "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4)}


def _mfma_row(flop, ms):
    if ms <= 0:
        return None
    tf = flop / (ms * 1e-3) / 1e12
    return {"bound": "mfma", "ms": round(ms, 4), "algorithmic_flop": float(flop), "achieved": round(tf, 1),
            "unit": "TFLOP/s", "frac": round(tf / PEAK_BF16_TFLOPS, 4)}


def measure_next(pace, pq, pk, pv, p_cu, S, p_vis, p_cuv, Nv, T, idx, K, stream, reps=5):
    """Outside the timed step: (1) the all-query ("Vision + Text") S_llm, i.e. the prefill's
    mass pass with every row of the sequence querying; (2) the context after pruning: gather
    Q/K/V of the K kept visual tokens and the T text tokens, then the same prefill kernel on
    those T + K tokens (what the decoder layers after the extraction layer run)."""
    import torch

    dev = pq.device
    Hq, dq = pq.shape[1], pq.shape[2]

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    zero = torch.zeros(1, dtype=torch.int32, device=dev)
    all_rows = torch.tensor([S], dtype=torch.int32, device=dev)
    o = torch.empty_like(pq)
    lse = torch.empty((Hq, S), dtype=torch.float32, device=dev)
    mass = torch.empty((Hq, Nv), dtype=torch.float32, device=dev)
    t_all = timed(lambda: pace.prefill_attention_with_mass(pq, pk, pv, p_cu, S, p_vis, p_cuv, Nv, Nv, zero,
                                                            all_rows, S, o=o, lse=lse, mass=mass))
    keep = torch.cat([idx.long(), torch.arange(Nv, S, device=dev)]).to(torch.int32)
    Sp = K + T
    qc, kc, vc = (torch.empty((Sp,) + tuple(x.shape[1:]), dtype=x.dtype, device=dev) for x in (pq, pk, pv))
    t_gather = timed(lambda: [pace.gather_rows(x, keep, out=y) for x, y in ((pq, qc), (pk, kc), (pv, vc))])
    cu = torch.tensor([0, Sp], dtype=torch.int32, device=dev)
    oc = torch.empty_like(qc)
    lc = torch.empty((Hq, Sp), dtype=torch.float32, device=dev)
    t_post = timed(lambda: pace.prefill_attention_with_mass(qc, kc, vc, cu, Sp, None, None, 0, 0, None, None, 0,
                                                             want_mass=False, o=oc, lse=lc))
    t_full = timed(lambda: pace.prefill_attention_with_mass(pq, pk, pv, p_cu, S, None, None, 0, 0, None, None,
                                                             0, want_mass=False, o=o, lse=lse))
    flop_full = 4.0 * dq * Hq * (S * (S + 1) / 2.0)
    flop_post = 4.0 * dq * Hq * (Sp * (Sp + 1) / 2.0)
    return {
        "vision_text_mass": {"ms": round(t_all, 4), "query_rows": int(S),
                             "note": "prefill forward + all-query mass (the paper's Vision+Text source)"},
        "post_prune_prefill": {"tokens": int(Sp), "full_tokens": int(S), "gather_qkv_ms": round(t_gather, 4),
                               "prefill_ms": round(t_post, 4), "full_prefill_ms": round(t_full, 4),
                               "speedup": round(t_full / t_post, 2) if t_post > 0 else None,
                               "tflops_post": round(flop_post / (t_post * 1e-3) / 1e12, 1) if t_post > 0 else None,
                               "tflops_full": round(flop_full / (t_full * 1e-3) / 1e12, 1) if t_full > 0 else None},
    }


def measure_preview(pace, wl, img, L, stream, reps=3):
    """Outside the timed step: APC's shallow preview (the vision encoder's first block with seeded
    weights, at the original resolution) on the same image, then the density of its embeddings."""
    import numpy as np
    import torch

    dev = img.device
    w = wl.preview_weights(3)
    wdev = pace.preview_weights_to_device(w, dev)
    f_alg = int(w["wg"].shape[0])   # hidden units of the block (the device copy pads to a multiple of 8)
    order = torch.from_numpy(L.order.astype(np.int32)).to(dev)
    cu = torch.from_numpy(L.cu_windows.astype(np.int32)).to(dev)
    maxw = int(np.max(L.window_sizes))
    N = int(L.order.shape[0])
    D, F = wdev["dim"], wdev["ffn"]
    out = torch.empty((N, D), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(pace.lib().pace_apc_preview_workspace_size(N, D, F, 14), dtype=torch.uint8, device=dev)
    rho = torch.empty(4, dtype=torch.float32, device=dev)
    dd = torch.empty(N, dtype=torch.float32, device=dev)
    wsd = torch.empty(pace.lib().pace_apc_density_features_workspace_size(N, D), dtype=torch.uint8, device=dev)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    t_block = timed(lambda: pace.apc_preview(img, 14, order, cu, maxw, wdev, out=out, workspace=ws))
    t_dens = timed(lambda: pace.apc_density_features(out, d_out=dd, rho_out=rho, workspace=wsd))
    win = np.diff(L.cu_windows).astype(np.float64)
    flop = 2.0 * N * D * (3 * 14 * 14 + 4 * D + 3 * f_alg) + 4.0 * 80 * (D // 80) * float(np.sum(win ** 2))
    H, W = int(img.shape[0]), int(img.shape[1])
    pixel_ms = {}
    for name, kind in pace.PIXEL_STATISTICS.items():
        wsp = torch.empty(pace.lib().pace_apc_pixel_density_workspace_size(H, W, 14, kind), dtype=torch.uint8,
                          device=dev)
        pixel_ms[name] = round(timed(lambda: pace.apc_pixel_density(img, kind, 14, d_out=dd, rho_out=rho,
                                                                    workspace=wsp)), 4)
    return {"ms": round(t_block, 4), "tflops": round(flop / (t_block * 1e-3) / 1e12, 1), "patches": N,
            "dim": D, "ffn": F, "density_features_ms": round(t_dens, 4), "pixel_statistic_density_ms": pixel_ms,
            "note": "seeded-weight first vision block at the original resolution (patch embedding, "
                    "window attention, SwiGLU MLP) + APC density of its embeddings; the four "
                    "training-free pixel-statistic previews with their densities"}


def cpu_baseline(vit, budget_s: float):
    """The float64 oracle (unchanged) on the host cores: O and LSE of query rows of the 4K
    full attention, all 16 heads, over all 42,196 keys, in chunks of 256 rows until the time
    budget is spent.  Reported in the metric's unit (algorithmic attention TFLOP/s)."""
    import numpy as np

    from oracle import attention as oatt
    from paper_2608_27206_amd import workloads as wl

    cores = None
    try:
        from threadpoolctl import threadpool_info
        blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        if blas:
            cores = int(max(p["num_threads"] for p in blas))
    except Exception:  # pragma: no cover
        pass
    if cores is None:
        cores = len(os.sched_getaffinity(0))
    q = wl.bf16_bits_to_f64(vit.q)
    k = wl.bf16_bits_to_f64(vit.k)
    v = wl.bf16_bits_to_f64(vit.v)
    N, H, d = q.shape
    rows_done = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < budget_s and rows_done < N:
        rows = np.arange(rows_done, min(N, rows_done + 256))
        oatt.attention_rows(q, k, v, 0, N, rows, False, 1 / math.sqrt(d))
        rows_done += rows.size
    dt = time.perf_counter() - t0
    flops = 4.0 * d * H * rows_done * N
    return {"value": round(flops / dt / 1e12, 5), "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": f"float64 oracle attention (O, LSE) for the first {rows_done} of {N} query rows "
                      f"x {H} heads of the 4K full attention over all {N} keys, {dt:.1f} s wall"}


if __name__ == "__main__":
    main()
