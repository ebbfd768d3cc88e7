"""PACE hot-path benchmark on one MI355X.

A step is one pass of every hot-path kernel over one seeded workload (Qwen2.5-VL-7B shapes),
inputs already resident in HBM when the timed region starts.  The default (--config 3) is
the 4K frame (3836x2156 RGB): APC density and 2x downsample of the image, vision-encoder
window attention (700 windows of <= 64 patches, 16 heads, d = 80) and full attention over
42,196 patches with the per-key mass, causal GQA prefill over 10,549 visual + 128 text
tokens (28/4 heads, d = 128) with the text-query mass of every visual key, and DDAE fusion +
top-K (10%) + gather of the kept rows of a 10,549 x 3584 bf16 hidden-state matrix.
--config 1 and 2 run the same step on a 448x448 and a 1344x1344 image (the resize takes APC's
own rho within the 256..2048 x 28^2 pixel budget), --config 4 on the packed batch of eight
images (per-image density, resize and keep count; the attention passes over cu_seqlens; one
segmented selection), and --config 0 on the tiny prefill (prefill with mass, then fusion with
a given vision mass, top-K and gather).  Sizes that follow rho are read back once before the
timed steps.

Prints one JSON line.  `value` is the step's algorithmic attention FLOP rate
(every attention pass's 4*d*(visible pairs)*heads, over the whole step time).
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
    ap.add_argument("--config", type=int, default=3, choices=range(5),
                    help="workload id: 0 tiny prefill, 1 448x448, 2 1344x1344, 3 4K frame (default), 4 varlen batch")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="wall-clock budget of the oracle CPU baseline sample (0 = skip)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="before warm-up, copy this many MiB device to device once (a plain copy "
                         "of known size that calibrates the HBM byte counters of a profile run)")
    ap.add_argument("--no-graph", dest="graph", action="store_false",
                    help="time the steps launched kernel by kernel instead of replaying the step captured "
                         "in a HIP graph")
    ap.add_argument("--select-sweep", action="store_true",
                    help="instead of the step: DDAE selection + gather over batches of 1, 4, 16 and 64 "
                         "images of 4K-frame shapes (one JSON line per batch)")
    return ap.parse_args()


def select_sweep(a):
    """DDAE fuse + top-K + gather (pace_ddae_select_varlen, one call) over B images of the 4K frame's
    shapes (16 x 42,196 vision masses, 28 x 10,549 text masses, the window-order permutation, a
    10,549 x 3584 bf16 hidden matrix per image, K = 1,055 each), B = 1, 4, 16, 64: how the rate
    approaches the HBM roofline once the fixed latency of the two launches is amortised.  Masses are
    seeded Gamma draws (the selection's cost does not depend on their values)."""
    import numpy as np
    import torch

    from paper_2608_27206_amd import pace
    from paper_2608_27206_amd import workloads as wl

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    L = wl.vit_layout(2156 // 14, 3836 // 14)
    nv, npatch = L.n_vis, L.n_patches
    K = pace.keep_count(0.10, nv)
    stream = torch.cuda.current_stream()
    for B in (1, 4, 16, 64):
        g = torch.Generator(device=dev)
        g.manual_seed(1000 + B)
        vis = torch.empty((16, B * npatch), device=dev).exponential_(generator=g)
        llm = torch.empty((28, B * nv), device=dev).exponential_(generator=g)
        perm = torch.from_numpy(np.tile(L.vis_perm.astype(np.int32), B)).to(dev)
        hidden = torch.empty((B * nv, wl.HIDDEN), dtype=torch.bfloat16, device=dev).normal_(generator=g)
        nvs, keeps = [nv] * B, [K] * B
        idx = torch.empty(B * K, dtype=torch.int32, device=dev)
        sc = torch.empty(B * nv, dtype=torch.float32, device=dev)
        fz = torch.empty((B, 4), dtype=torch.float32, device=dev)
        out = torch.empty((B * K, wl.HIDDEN), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(pace.lib().pace_ddae_select_workspace_size(B * nv, B), dtype=torch.uint8, device=dev)

        def call():
            pace.ddae_select(vis, 4, perm, llm, nvs, keeps, mode=0, tau=0.5, hidden=hidden, idx_out=idx,
                             score_out=sc, fuse_out=fz, out=out, workspace=ws)
        for _ in range(3):
            call()
        torch.cuda.synchronize()
        ts = []
        for _ in range(max(5, a.steps)):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            call()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        ms = sorted(ts)[len(ts) // 2]
        nbytes = float(B) * (16 * npatch * 4 + 28 * nv * 4 + 4 * K + 2.0 * K * wl.HIDDEN * 2)
        gbs = nbytes / (ms * 1e-3) / 1e9
        print(json.dumps({"select_sweep": {"images": B, "tokens": B * nv, "kept": B * K, "ms": round(ms, 4),
                                           "tokens_per_s": round(B * nv / (ms * 1e-3), 1),
                                           "algorithmic_bytes": int(nbytes), "gbs": round(gbs, 1),
                                           "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)}}), flush=True)
        del vis, llm, perm, hidden, out, ws
        torch.cuda.empty_cache()


def capture_step_graph(torch, step, stream):
    """The step captured once in a HIP graph (the vision mass forks onto a second stream inside
    the capture and joins before the selection), after one pass on a side stream and followed
    by one replay, both outside any timed region."""
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
    return g


MIN_PIXELS = 256 * 28 * 28    # APC's dynamic budget (reading R4): the resize keeps at least this area
MAX_PIXELS = 2048 * 28 * 28   # ... and at most this one (the paper's fixed setting of 2048 * 28 * 28)


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:  # pragma: no cover
        pass
    return "unknown"


def build_workload_step(a, torch, np, pace, wl, dev):
    """Device inputs, outputs and the ordered parts of one step of the hot path for workload
    a.config.  Returns a dict: parts [(name, fn, side, join)], work {name: (bound, amount)},
    config (the JSON config object), roof (name and label of the dominant kernel's part),
    flop_attn (algorithmic attention FLOPs of the step), cpu (oracle sample closure), extra."""
    w = wl.make_workload(a.config)

    def bf(x):
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)

    def i32(x):
        return torch.from_numpy(np.asarray(x, np.int32)).to(dev)

    f32 = dict(dtype=torch.float32, device=dev)
    pre = w.prefill
    pq, pk, pv = bf(pre.q), bf(pre.k), bf(pre.v)
    p_cu, p_vis, p_cuv = i32(pre.cu_seqlens), i32(pre.vis_len), i32(pre.cu_vis)
    p_mqs, p_mql = i32(pre.mq_start), i32(pre.mq_len)
    S_tot = int(pre.cu_seqlens[-1])
    seqlens = np.diff(pre.cu_seqlens)
    max_s = int(seqlens.max())
    nvs = [int(x) for x in pre.vis_len]
    Nv = int(sum(nvs))
    Hq, Hkv, dq = pre.q.shape[1], pre.k.shape[1], pre.q.shape[2]
    hidden = bf(w.hidden)
    o_pre = torch.empty_like(pq)
    lse_pre = torch.empty((Hq, S_tot), **f32)
    mass_llm = torch.empty((Hq, max(1, Nv)), **f32)
    parts, work = [], {}
    flop_pre = 4.0 * dq * Hq * float(np.sum(seqlens.astype(np.float64) * (seqlens + 1) / 2.0))

    def prefill():
        pace.prefill_attention_with_mass(pq, pk, pv, p_cu, max_s, p_vis, p_cuv, Nv, int(pre.vis_len.max()), p_mqs,
                                         p_mql, int(pre.mq_len.max()), o=o_pre, lse=lse_pre, mass=mass_llm)

    cfg = {"workload": wl.CONFIG_NAMES[a.config], "prefill_tokens": S_tot, "visual_tokens": Nv,
           "text_tokens": int(pre.text_len.sum()), "llm_heads": f"{Hq}/{Hkv}", "llm_head_dim": int(dq),
           "hidden": int(w.hidden.shape[1])}
    extra = {}
    if w.vit is None:
        # tiny DDAE prefill: the vision mass is given (Dirichlet), fixed 50/50 fusion
        K = pace.keep_count(w.keep_ratio, Nv)
        keeps = [K]
        vis_mass = torch.from_numpy(w.vit_mass).to(dev)
        merge, perm = 1, None
        parts.append(("prefill", prefill, False, False))
        work["prefill"] = ("mfma", flop_pre)
        roof = ("prefill", "attn_fwd<128, true> + attn_mass<128, true> (causal GQA prefill with text-query mass)")
        flop_attn = flop_pre
        cfg.update({"keep": K, "fusion": "fixed 0.5/0.5"})
    else:
        vit = w.vit
        vq, vk, vv = bf(vit.q), bf(vit.k), bf(vit.v)
        cu_win, cu_full = i32(vit.cu_windows), i32(vit.cu_full)
        max_win = int(np.diff(vit.cu_windows).max())
        full_lens = np.diff(vit.cu_full).astype(np.float64)
        max_full = int(full_lens.max())
        Np, Hv, dv = vit.q.shape
        nseg = len(full_lens)
        perm, merge = i32(vit.vis_perm), 4
        imgs = [torch.from_numpy(im).to(dev) for im in w.images]
        ws_apc = [torch.empty(pace.lib().pace_apc_density_workspace_size(im.shape[0], im.shape[1], 14),
                              dtype=torch.uint8, device=dev) for im in w.images]
        rhos = [torch.empty(3, **f32) for _ in w.images]
        dps = [torch.empty((im.shape[0] // 14) * (im.shape[1] // 14), **f32) for im in w.images]
        # the resize size and the per-image K follow the density: read once from the GPU here (a caller
        # reads rho back before sizing the resize); the timed steps reuse these sizes
        for im, ws, r, d in zip(imgs, ws_apc, rhos, dps):
            pace.apc_density(im, 14, 0.10, 0.6, 1.5, d_out=d, rho_out=r, workspace=ws)
        torch.cuda.synchronize()
        rho_h = [float(r.cpu()[2]) for r in rhos]
        sizes = []
        for im, rh in zip(w.images, rho_h):
            H, W = im.shape[0], im.shape[1]
            if w.downsample_scale:
                sizes.append((int(round(H * w.downsample_scale)), int(round(W * w.downsample_scale))))
            else:
                sizes.append(pace.apc_target_size(rh, H, W, MIN_PIXELS, MAX_PIXELS, 28))
        smalls = [torch.empty((oh, ow, 3), dtype=torch.uint8, device=dev) for oh, ow in sizes]
        if a.config == 4:
            keeps = [pace.keep_from_density(rh, nv) for rh, nv in zip(rho_h, nvs)]
        else:
            keeps = [pace.keep_count(w.keep_ratio, Nv)]
        o_win = torch.empty_like(vq)
        lse_win = torch.empty((Hv, Np), **f32)
        mass_win = torch.empty((Hv, Np), **f32)
        o_full = torch.empty_like(vq)
        lse_full = torch.empty((Hv, Np), **f32)
        vis_mass = torch.empty((Hv, Np), **f32)
        ws_vit = torch.empty(pace.lib().pace_vit_attention_workspace_size(Np, Hv, dv, nseg, max_full),
                             dtype=torch.uint8, device=dev)

        def apc():
            for im, ws, r, d in zip(imgs, ws_apc, rhos, dps):
                pace.apc_density(im, 14, 0.10, 0.6, 1.5, d_out=d, rho_out=r, workspace=ws)

        def resize():
            for im, sm in zip(imgs, smalls):
                pace.apc_downsample(im, sm.shape[0], sm.shape[1], dst=sm)

        # one image's density then its resize: the images are independent, so with several of them
        # the overlapped step runs these chains side by side on a few streams
        def image_chain(i):
            def run():
                pace.apc_density(imgs[i], 14, 0.10, 0.6, 1.5, d_out=dps[i], rho_out=rhos[i], workspace=ws_apc[i])
                pace.apc_downsample(imgs[i], smalls[i].shape[0], smalls[i].shape[1], dst=smalls[i])
            return run

        if len(imgs) > 1:
            extra["image_chains"] = [image_chain(i) for i in range(len(imgs))]

        parts += [
            ("apc", apc, False, False),
            ("resize", resize, False, False),
            ("vit_win", lambda: pace.vit_attention(vq, vk, vv, cu_win, max_win, o=o_win, lse=lse_win,
                                                   mass=mass_win), False, False),
            ("vit_fwd", lambda: pace.vit_attention(vq, vk, vv, cu_full, max_full, o=o_full, lse=lse_full,
                                                   want_mass=False, workspace=ws_vit), False, False),
            # the vision mass needs only the forward's LSE and the prefill neither (it takes the encoder's
            # output): the mass runs on a second stream beside the prefill, the selection joins both
            ("vit_mass", lambda: pace.vit_attention_mass(vq, vk, cu_full, max_full, lse_full, mass=vis_mass),
             True, False),
            ("prefill", prefill, False, False),
        ]
        win_sizes = np.diff(vit.cu_windows).astype(np.float64)
        flop_full = 4.0 * dv * Hv * float(np.sum(full_lens ** 2))
        work.update({
            "apc": ("hbm", float(sum(im.shape[0] * im.shape[1] * 3 + 4.0 * (im.shape[0] // 14) * (im.shape[1] // 14)
                                    for im in w.images))),
            "resize": ("hbm", float(sum(im.shape[0] * im.shape[1] * 3 + oh * ow * 3
                                       for im, (oh, ow) in zip(w.images, sizes)))),
            "vit_win": ("hbm", 4.0 * Np * Hv * dv * 2 + 2.0 * Hv * Np * 4),
            "vit_fwd": ("mfma", flop_full),
            "vit_mass": ("mfma", 0.0),
            "prefill": ("mfma", flop_pre),
        })
        flop_attn = 4.0 * dv * Hv * float(np.sum(win_sizes ** 2)) + flop_full + flop_pre
        roof = ("vit_fwd", "pace_vit_attention call on the full-attention segments: attn_vt_clear + attn_v_amax + "
                           f"attn_vt_prep + attn_fwd_rot<80> ({Np:,} patches in {nseg} segment(s) x {Hv} heads); "
                           "attn_fwd_rot is 99% of it")
        cfg.update({"images": [f"{im.shape[1]}x{im.shape[0]}" for im in w.images], "vit_patches": int(Np),
                    "vit_heads": int(Hv), "vit_head_dim": int(dv), "vit_segments": nseg,
                    "windows": int(len(win_sizes)), "keep": keeps if len(keeps) > 1 else keeps[0],
                    "resize_to": [f"{ow}x{oh}" for oh, ow in sizes] if len(sizes) > 1 else f"{sizes[0][1]}x{sizes[0][0]}"})
        extra["flop_full"] = flop_full
        extra.update({"vq": vq, "vk": vk, "vv": vv, "img": imgs[0], "layout": w.layouts[0]})
    ktot = int(sum(keeps))
    idx = torch.empty(max(1, ktot), dtype=torch.int32, device=dev)
    scores = torch.empty(max(1, Nv), **f32)
    fuse = torch.empty((len(keeps), 4), **f32)
    kept = torch.empty((max(1, ktot), hidden.shape[1]), dtype=hidden.dtype, device=dev)
    ws_sel = torch.empty(pace.lib().pace_ddae_select_workspace_size(Nv, len(keeps)), dtype=torch.uint8, device=dev)
    parts.append(("select", lambda: pace.ddae_select(vis_mass, merge, perm, mass_llm, nvs, keeps, mode=w.fusion_mode,
                                                     tau=w.tau, w_llm_fixed=w.w_llm_fixed, hidden=hidden,
                                                     idx_out=idx, score_out=scores, fuse_out=fuse, out=kept,
                                                     workspace=ws_sel), False, True))
    Hv_sel = vis_mass.shape[0]
    work["select"] = ("hbm", float(Hv_sel * vis_mass.shape[1] * 4 + Hq * Nv * 4 + 4 * ktot
                                   + 2.0 * ktot * hidden.shape[1] * 2))
    extra.update({"pq": pq, "pk": pk, "pv": pv, "p_cu": p_cu, "p_vis": p_vis, "p_cuv": p_cuv, "S": S_tot, "Nv": Nv,
                  "T": int(pre.text_len.sum()), "idx": idx, "K": ktot, "w": w})
    return {"parts": parts, "work": work, "config": cfg, "roof": roof, "flop_attn": flop_attn, "extra": extra}


def main():
    a = parse()
    if a.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only; --gpus must be 1 "
                          "(multi-GPU sharding is described in the design notes, not built)"}))
        sys.exit(2)
    if a.select_sweep:
        select_sweep(a)
        return
    import numpy as np
    import torch

    from paper_2608_27206_amd import pace
    from paper_2608_27206_amd import workloads as wl

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    B = build_workload_step(a, torch, np, pace, wl, dev)
    parts, work, ex = B["parts"], B["work"], B["extra"]
    names = [p[0] for p in parts]
    stream = torch.cuda.current_stream()
    side = torch.cuda.Stream()   # default priority
    # several images: their density + resize chains fork onto up to four streams (default
    # priority) in the overlapped step and join before the window attention
    chains = ex.get("image_chains")
    img_streams = [torch.cuda.Stream() for _ in range(min(4, len(chains)))] if chains else []

    def new_events():
        return {n: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for n in names}

    def step(ev, overlap=True):
        cur = torch.cuda.current_stream()
        pending = False
        for name, fn, on_side, join in parts:
            if overlap and chains and name in ("apc", "resize"):
                if name == "apc":
                    for sm in img_streams:
                        sm.wait_stream(cur)
                    for i, chain in enumerate(chains):
                        with torch.cuda.stream(img_streams[i % len(img_streams)]):
                            chain()
                    for sm in img_streams:
                        cur.wait_stream(sm)
                continue
            if overlap and join and pending:
                cur.wait_stream(side)
                pending = False
            if overlap and on_side:
                side.wait_stream(cur)
                with torch.cuda.stream(side):
                    fn()
                pending = True
                continue
            if ev is not None:
                ev[name][0].record(cur)
            fn()
            if ev is not None:
                ev[name][1].record(cur)
        if pending:
            cur.wait_stream(side)

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
    graph = capture_step_graph(torch, step, stream) if a.graph else None

    def timed_steps(run):
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record(stream)
        for _ in range(a.steps):
            run()
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / a.steps

    # the timed region: K steps, each a replay of the captured step (or, with --no-graph, the
    # step launched kernel by kernel); then the same K steps launched kernel by kernel
    ms_per_step = timed_steps(graph.replay if graph is not None else lambda: step(None))
    eager_ms = timed_steps(lambda: step(None))
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
    nxt = None
    if a.config == 3:
        nxt = measure_next(pace, ex["pq"], ex["pk"], ex["pv"], ex["p_cu"], ex["S"], ex["p_vis"], ex["p_cuv"],
                           ex["Nv"], ex["T"], ex["idx"], ex["K"], stream)
        nxt["preview_block"] = measure_preview(pace, wl, ex["img"], ex["layout"], stream)

    roof_name, roof_label = B["roof"]
    t_roof = per[roof_name] * 1e-3
    achieved = work[roof_name][1] / t_roof / 1e12 if t_roof > 0 else 0.0
    value = B["flop_attn"] / (ms_per_step * 1e-3) / 1e12
    sel_ms = per["select"]

    step_roofline = {}
    labels = {"apc": "apc_density", "resize": "apc_downsample", "vit_win": "vit_window_attention",
              "vit_fwd": "vit_full_attention_fwd", "prefill": "prefill_attention_with_mass",
              "select": "ddae_select_gather"}
    for n in names:
        if n == "vit_mass":
            continue
        bound, amount = work[n]
        step_roofline[labels[n]] = _hbm_row(amount, per[n]) if bound == "hbm" else _mfma_row(amount, per[n])
    if "vit_mass" in per:
        step_roofline["vit_full_attention_fwd_plus_mass"] = _mfma_row(work["vit_fwd"][1], per["vit_fwd"] + per["vit_mass"])

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
        "config": B["config"],
        "roofline": {"kernel": roof_label, "bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic() if a.config == 3 else None},
        "schedule": ("each timed step replays the step captured once in a HIP graph" if graph is not None
                     else "each timed step launched kernel by kernel") +
                    " (vision mass on a second stream beside the prefill" +
                    ("; the images' density and resize chains on %d streams side by side" % len(img_streams)
                     if chains else "") + "); eager_ms_per_step: the same "
                    "steps launched kernel by kernel; breakdown_ms and step_roofline from the same steps "
                    "run serially on one stream",
        "eager_ms_per_step": round(eager_ms, 4),
        "serial_ms_per_step": round(serial_ms, 4),
        "breakdown_ms": {n: round(v, 4) for n, v in per.items()},
        "select": {
            "tokens_per_s": round(ex["Nv"] / (sel_ms * 1e-3), 1) if sel_ms > 0 else None,
            "gbs": round(work["select"][1] / (sel_ms * 1e-3) / 1e9, 1) if sel_ms > 0 else None,
            "hbm_frac": round(work["select"][1] / (sel_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4) if sel_ms > 0 else None,
        },
        # every step of the path against the roofline that bounds it (algorithmic work per step)
        "step_roofline": step_roofline,
        "next": nxt,
    }
    if a.cpu_seconds > 0:
        result["cpu_baseline"] = cpu_baseline(ex["w"], a.cpu_seconds)
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
    rho = torch.empty(3, dtype=torch.float32, device=dev)
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


def cpu_baseline(w, budget_s: float):
    """The float64 oracle (unchanged) on the host cores, in the metric's unit (algorithmic attention
    TFLOP/s): O and LSE of query rows of the first image's full attention, all 16 heads, over all of
    its keys, in chunks of 256 rows until the time budget is spent; for the tiny workload (no vision
    encoder), the whole causal prefill, repeated until the budget is spent."""
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
    t0 = time.perf_counter()
    if w.vit is None:
        p = w.prefill
        q, k, v = (wl.bf16_bits_to_f64(x) for x in (p.q, p.k, p.v))
        S = int(p.cu_seqlens[-1])
        reps = 0
        while time.perf_counter() - t0 < budget_s:
            oatt.prefill_attention(q, k, v, p.cu_seqlens, p.vis_len, p.mq_start, p.mq_len, 1 / math.sqrt(q.shape[2]))
            reps += 1
        dt = time.perf_counter() - t0
        flops = reps * 4.0 * q.shape[2] * q.shape[1] * S * (S + 1) / 2.0
        sample = f"float64 oracle causal prefill with text-query mass ({S} tokens, {q.shape[1]} heads), {reps} runs, {dt:.1f} s wall"
    else:
        vit = w.vit
        n0 = int(vit.cu_full[1])
        q = wl.bf16_bits_to_f64(vit.q[:n0])
        k = wl.bf16_bits_to_f64(vit.k[:n0])
        v = wl.bf16_bits_to_f64(vit.v[:n0])
        N, H, d = q.shape
        rows_done = 0
        while time.perf_counter() - t0 < budget_s and rows_done < N:
            rows = np.arange(rows_done, min(N, rows_done + 256))
            oatt.attention_rows(q, k, v, 0, N, rows, False, 1 / math.sqrt(d))
            rows_done += rows.size
        dt = time.perf_counter() - t0
        flops = 4.0 * d * H * rows_done * N
        sample = (f"float64 oracle attention (O, LSE) for the first {rows_done} of {N} query rows x {H} heads of "
                  f"the first image's full attention over all {N} keys, {dt:.1f} s wall")
    return {"value": round(flops / dt / 1e12, 5), "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "cpu_model": cpu_model(), "sample": sample}


if __name__ == "__main__":
    main()
