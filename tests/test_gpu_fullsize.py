"""GPU parity at the full workload sizes, in the launch configuration bench.py times.

Where the float64 oracle cannot redo the whole problem in seconds, it checks sampled
outputs one by one (query rows of the full attention, sampled prefill rows) and the
properties that hold at any size (each head's mass sums to the number of query rows).
Everything else is compared element by element: every window, the text-query mass of
every visual key, every patch distance, every fused score and kept index.
APC's Eq. 1 at 4K comes from tests/golden/apc_fullsize.json (oracle-only script)."""
import hashlib
import json
import math
import os

import numpy as np
import pytest

from oracle import apc as oapc
from oracle import attention as oatt
from oracle import ddae as oddae
from paper_2608_27206_amd import workloads as wl
from tests.gpu_util import (dev_bf16, dev_f32, dev_i32, dev_u8, host, host_bf16_to_f64, rho4,
                            kept_sets_agree, load_e2e_golden, mass_ok, oracle_mass_parallel, say)

pytestmark = pytest.mark.gpu

GOLD = os.path.join(os.path.dirname(__file__), "golden", "apc_fullsize.json")
O_TOL, LSE_TOL = 2e-2, 1e-3


@pytest.fixture(scope="module")
def w4k():
    say("building the 4K workload")
    return wl.make_workload(3)


@pytest.fixture(scope="module")
def wvar():
    say("building the varlen workload")
    return wl.make_workload(4)


def _f64(bits):
    return wl.bf16_bits_to_f64(bits)


def _check_rows(q, k, v, o_gpu, lse_gpu, a, b, rows, causal, heads):
    """Oracle O and LSE for selected rows of segment [a, b), head by head."""
    scale = 1 / math.sqrt(q.shape[2])
    hq, hkv = q.shape[1], k.shape[1]
    for h in heads:
        kv = h // (hq // hkv)
        O, L, _ = oatt.attention_segment(_f64(q[a:b, h:h + 1]), _f64(k[a:b, kv:kv + 1]),
                                         _f64(v[a:b, kv:kv + 1]), causal, scale, rows=rows)
        got_o = o_gpu[a + np.asarray(rows), h]
        assert np.max(np.abs(got_o - O[:, 0])) <= O_TOL, (h, np.max(np.abs(got_o - O[:, 0])))
        assert np.max(np.abs(lse_gpu[h, a + np.asarray(rows)] - L[0])) <= LSE_TOL


def _vit_bench_sequence(vit, cu, maxlen):
    """The calls bench.py times: forward with LSE, then the mass pass."""
    from paper_2608_27206_amd import pace
    import torch
    Q, K, V, CU = dev_bf16(vit.q), dev_bf16(vit.k), dev_bf16(vit.v), dev_i32(cu)
    o, lse, _ = pace.vit_attention(Q, K, V, CU, maxlen, want_mass=False)
    mass = pace.vit_attention_mass(Q, K, CU, maxlen, lse)
    torch.cuda.synchronize()
    return host_bf16_to_f64(o), host(lse), host(mass)


ROT_ROWS = 384   # query rows per workgroup of the long-segment forward


def test_frame4k_vit_full_attention(w4k):
    """O and LSE of all 16 heads on 1,000+ rows: the first and last row of every 384-row
    workgroup of the forward plus random ones; the per-key mass of two heads element by element
    over all 42,196 keys; and each head's mass totals N."""
    vit = w4k.vit
    N = vit.q.shape[0]
    say(f"4K full attention N={N}")
    o, lse, mass = _vit_bench_sequence(vit, vit.cu_full, N)
    rs = np.random.default_rng(0)
    starts = np.arange(0, N, ROT_ROWS)
    rows = np.unique(np.concatenate([starts, np.minimum(starts + ROT_ROWS - 1, N - 1), [1, N // 2, N - 2],
                                     rs.integers(0, N, 800)]))
    assert rows.size >= 1000
    _check_rows(vit.q, vit.k, vit.v, o, lse, 0, N, rows, False, range(vit.q.shape[1]))
    for h in (0, 9):
        say(f"4K full attention: oracle mass of head {h} over all {N} rows")
        ref = oracle_mass_parallel(_f64(vit.q[:, h]), _f64(vit.k[:, h]), False, 1 / math.sqrt(80), np.arange(N))
        err, rel = mass_ok(mass[h], ref, N)
        assert err <= 0, (h, rel)
    # every row's probabilities sum to one, so each head's mass totals N
    np.testing.assert_allclose(mass.sum(axis=1), N, rtol=1e-4)
    assert np.all(mass >= 0)


def _e2e_gpu_selection(w, keeps):
    """The chain bench.py times, on the GPU alone: full attention of every image (forward, then
    the mass pass), the causal prefill with the text-query mass, and the DDAE selection of the
    images' K_b tokens from those masses.  Returns (kept global indices, fused scores)."""
    from paper_2608_27206_amd import pace
    import torch
    vit, p = w.vit, w.prefill
    cu = vit.cu_full
    Q, K, CU = dev_bf16(vit.q), dev_bf16(vit.k), dev_i32(cu)
    maxlen = int(np.diff(cu).max())
    _, lse, _ = pace.vit_attention(Q, K, dev_bf16(vit.v), CU, maxlen, want_mass=False)
    vis_mass = pace.vit_attention_mass(Q, K, CU, maxlen, lse)
    pc = p.cu_seqlens
    _, _, llm_mass = pace.prefill_attention_with_mass(
        dev_bf16(p.q), dev_bf16(p.k), dev_bf16(p.v), dev_i32(pc), int(np.diff(pc).max()),
        dev_i32(p.vis_len), dev_i32(p.cu_vis), int(p.cu_vis[-1]), int(p.vis_len.max()),
        dev_i32(p.mq_start), dev_i32(p.mq_len), int(p.mq_len.max()))
    nvs = [L.n_vis for L in w.layouts]
    idx, sc, _, _ = pace.ddae_select(vis_mass, 4, dev_i32(vit.vis_perm), llm_mass, nvs, list(keeps),
                                     mode=w.fusion_mode, tau=w.tau)
    torch.cuda.synchronize()
    return host(idx).astype(np.int64), host(sc).astype(np.float64)


def _check_e2e(idx, sc, nvs, keeps, S_g, idx_g):
    """Per image, the GPU's kept set against the oracle-only one: equal up to swaps whose oracle
    scores lie within 1e-3, and the fused scores within 1e-3 of the oracle's."""
    assert np.max(np.abs(sc - S_g)) <= 1e-3, np.max(np.abs(sc - S_g))
    off = koff = 0
    for b, (n, K) in enumerate(zip(nvs, keeps)):
        ok, msg = kept_sets_agree(idx[koff:koff + K], idx_g[koff:koff + K], S_g)
        assert ok, (b, msg)
        say(f"image {b}: {n} tokens, keep {K}: {msg}")
        off += n
        koff += K


def test_frame4k_e2e_selection(w4k):
    """Section 3.3 end to end at 4K: the tokens the GPU keeps from its own attention masses against
    the tokens the oracle keeps from its own (tests/golden/e2e_select.npz)."""
    nv_g, keep_g, S_g, idx_g = load_e2e_golden(3, w4k)
    say(f"4K end to end: keep {list(keep_g)} of {list(nv_g)}")
    idx, sc = _e2e_gpu_selection(w4k, keep_g)
    _check_e2e(idx, sc, nv_g, keep_g, S_g, idx_g)


def test_frame4k_windows(w4k):
    vit = w4k.vit
    cu = vit.cu_windows
    say(f"4K windows: {len(cu) - 1} segments")
    o, lse, mass = _vit_bench_sequence(vit, cu, int(np.diff(cu).max()))
    Or, Lr, Mr = oatt.vit_attention(_f64(vit.q), _f64(vit.k), _f64(vit.v), cu, 1 / math.sqrt(80))
    assert np.max(np.abs(o - Or)) <= O_TOL
    assert np.max(np.abs(lse - Lr)) <= LSE_TOL
    err, rel = mass_ok(mass, Mr, 64)
    assert err <= 0, rel


def _prefill_gpu(p):
    from paper_2608_27206_amd import pace
    import torch
    cu = p.cu_seqlens
    o, lse, mass = pace.prefill_attention_with_mass(
        dev_bf16(p.q), dev_bf16(p.k), dev_bf16(p.v), dev_i32(cu), int(np.diff(cu).max()),
        dev_i32(p.vis_len), dev_i32(p.cu_vis), int(p.cu_vis[-1]), int(p.vis_len.max()),
        dev_i32(p.mq_start), dev_i32(p.mq_len), int(p.mq_len.max()))
    torch.cuda.synchronize()
    return host_bf16_to_f64(o), host(lse), host(mass)


def _check_prefill_sequence(p, o, lse, mass, b, nrows):
    a, e = int(p.cu_seqlens[b]), int(p.cu_seqlens[b + 1])
    nv, nt = int(p.vis_len[b]), int(p.text_len[b])
    rs = np.random.default_rng(b)
    rows = np.unique(np.concatenate([[0, nv - 1, nv, e - a - 1], rs.integers(0, e - a, nrows)]))
    scale = 1 / math.sqrt(p.q.shape[2])
    hq, hkv = p.q.shape[1], p.k.shape[1]
    off = int(p.cu_vis[b])
    for h in range(hq):
        kv = h // (hq // hkv)
        O, L, M = oatt.attention_segment(_f64(p.q[a:e, h:h + 1]), _f64(p.k[a:e, kv:kv + 1]),
                                         _f64(p.v[a:e, kv:kv + 1]), True, scale, rows=rows,
                                         mass_rows=np.arange(nv, nv + nt))
        assert np.max(np.abs(o[a + rows, h] - O[:, 0])) <= O_TOL
        assert np.max(np.abs(lse[h, a + rows] - L[0])) <= LSE_TOL
        err, rel = mass_ok(mass[h, off:off + nv], M[0, :nv], nt)
        assert err <= 0, (b, h, rel)


def test_frame4k_prefill(w4k):
    p = w4k.prefill
    say(f"4K prefill S={p.q.shape[0]}")
    o, lse, mass = _prefill_gpu(p)
    _check_prefill_sequence(p, o, lse, mass, 0, 28)


def test_frame4k_apc(w4k):
    from paper_2608_27206_amd import pace
    import torch
    img = w4k.images[0]
    gold = json.load(open(GOLD))["frame4k"]
    assert hashlib.sha256(img.tobytes()).hexdigest() == gold["sha256"], "image generator changed"
    rho, d = pace.apc_density(dev_u8(img), 14, 0.10, 0.6, 1.5)
    torch.cuda.synchronize()
    T = oapc.l2_normalise(oapc.patch_features(img))
    d_ref = oapc.detail_distances(T, oapc.background_direction(T))
    np.testing.assert_allclose(host(d), d_ref, atol=1e-4)
    np.testing.assert_allclose(rho4(host(rho)), [gold["rho_g"], gold["rho_d"], gold["rho"], gold["phi"]], atol=1e-4)
    # at gamma = 1.5 rho_d is clamped at 1 (the tail mean is 1.92); above the tail mean it is
    # d_top / gamma, which pins the frame's tail mean itself (the 4,220 largest of 42,196 d_i)
    gamma = 2.5
    assert gold["d_top"] < gamma
    rho2, _ = pace.apc_density(dev_u8(img), 14, 0.10, 0.6, gamma)
    torch.cuda.synchronize()
    r2 = host(rho2)
    rho_d = gold["d_top"] / gamma
    np.testing.assert_allclose(r2[:3], [gold["rho_g"], rho_d, 0.6 * gold["rho_g"] + 0.4 * rho_d], atol=1e-4)


def test_frame4k_select(w4k):
    """4K-shaped masses (16 x 42,196 vision, 28 x 10,549 text) with the real window-order
    permutation; the fused scores, kept set and gathered rows against the oracle."""
    from paper_2608_27206_amd import pace
    import torch
    L = w4k.layouts[0]
    nv = L.n_vis
    rs = np.random.default_rng(3)
    vis = rs.gamma(0.5, size=(16, L.n_patches)).astype(np.float32)
    llm = rs.gamma(0.3, size=(28, nv)).astype(np.float32)
    K = oddae.keep_count(0.10, nv)
    assert K == pace.keep_count(0.10, nv) == 1055
    idx, sc, fz, out = pace.ddae_select(dev_f32(vis), 4, dev_i32(L.vis_perm), dev_f32(llm), [nv], [K],
                                        mode=0, tau=0.5, hidden=dev_bf16(w4k.hidden))
    torch.cuda.synchronize()
    S_ref, st = oddae.fuse(vis.astype(np.float64), llm.astype(np.float64), 4, L.vis_perm, 0, 0.5)
    np.testing.assert_allclose(host(sc), S_ref, atol=1e-5)
    np.testing.assert_allclose(host(fz)[0], st, atol=1e-5)
    ok, msg = kept_sets_agree(host(idx), oddae.topk_indices(S_ref, K), S_ref)
    assert ok, msg
    import torch as t
    np.testing.assert_array_equal(out.view(t.int16).cpu().numpy().view(np.uint16), w4k.hidden[host(idx)])
    # fed the oracle's scores (fp32), the ranking and gather are bit-exact
    S32 = S_ref.astype(np.float32)
    idx2, out2 = pace.topk_gather(dev_f32(S32), K, dev_bf16(w4k.hidden))
    torch.cuda.synchronize()
    ref2 = oddae.topk_indices(S32, K)
    np.testing.assert_array_equal(host(idx2), ref2)
    np.testing.assert_array_equal(out2.view(t.int16).cpu().numpy().view(np.uint16), w4k.hidden[ref2])


def test_varlen_vit(wvar):
    """Per image of the packed batch: O and LSE of all 16 heads on the first and last row of every
    384-row workgroup plus 64 random rows, and the per-key mass of one head (a different one per
    image) element by element."""
    vit = wvar.vit
    cu = vit.cu_full
    say(f"varlen full attention: segments {np.diff(cu).tolist()}")
    o, lse, mass = _vit_bench_sequence(vit, cu, int(np.diff(cu).max()))
    for b in range(len(cu) - 1):
        a, e = int(cu[b]), int(cu[b + 1])
        n = e - a
        rs = np.random.default_rng(b)
        starts = np.arange(0, n, ROT_ROWS)
        rows = np.unique(np.concatenate([starts, np.minimum(starts + ROT_ROWS - 1, n - 1), [n - 1],
                                         rs.integers(0, n, 64)]))
        _check_rows(vit.q, vit.k, vit.v, o, lse, a, e, rows, False, range(16))
        h = (5 * b) % 16
        ref = oracle_mass_parallel(_f64(vit.q[a:e, h]), _f64(vit.k[a:e, h]), False, 1 / math.sqrt(80),
                                   np.arange(n))
        err, rel = mass_ok(mass[h, a:e], ref, n)
        assert err <= 0, (b, h, rel)
        np.testing.assert_allclose(mass[:, a:e].sum(axis=1), n, rtol=1e-4)
    # windows of the first and last image, element by element
    cw = vit.cu_windows
    ow, lw, mw = _vit_bench_sequence(vit, cw, int(np.diff(cw).max()))
    for b in (0, len(cu) - 2):
        a, e = int(cu[b]), int(cu[b + 1])
        segs = cw[(cw >= a) & (cw <= e)] - a
        Or, Lr, Mr = oatt.vit_attention(_f64(vit.q[a:e]), _f64(vit.k[a:e]), _f64(vit.v[a:e]), segs,
                                        1 / math.sqrt(80))
        assert np.max(np.abs(ow[a:e] - Or)) <= O_TOL
        assert np.max(np.abs(lw[:, a:e] - Lr)) <= LSE_TOL
        err, rel = mass_ok(mw[:, a:e], Mr, 64)
        assert err <= 0, rel


def test_varlen_prefill(wvar):
    p = wvar.prefill
    say(f"varlen prefill: seqs {np.diff(p.cu_seqlens).tolist()}")
    o, lse, mass = _prefill_gpu(p)
    for b in range(len(p.vis_len)):
        _check_prefill_sequence(p, o, lse, mass, b, 6)


def test_varlen_apc_keep_and_select(wvar):
    """Per-image density (against the stored oracle values), the per-image K it sets, and the
    segmented selection into one compacted buffer."""
    from paper_2608_27206_amd import pace
    import torch
    gold = json.load(open(GOLD))["varlen8"]
    nvs = [L.n_vis for L in wvar.layouts]
    keeps_gpu, keeps_ref = [], []
    for img, g, nv in zip(wvar.images, gold, nvs):
        assert hashlib.sha256(img.tobytes()).hexdigest() == g["sha256"]
        rho, _ = pace.apc_density(dev_u8(img), 14, 0.10, 0.6, 1.5)
        torch.cuda.synchronize()
        r = host(rho)
        np.testing.assert_allclose(rho4(r), [g["rho_g"], g["rho_d"], g["rho"], g["phi"]], atol=1e-4)
        keeps_gpu.append(pace.keep_from_density(float(r[2]), nv))
        keeps_ref.append(oddae.keep_from_density(g["rho"], nv))
    assert keeps_gpu == keeps_ref
    assert len(set(keeps_ref)) > 1
    rs = np.random.default_rng(5)
    nt = sum(nvs)
    vis = rs.gamma(0.5, size=(16, 4 * nt)).astype(np.float32)
    llm = rs.gamma(0.3, size=(28, nt)).astype(np.float32)
    perm = wvar.vit.vis_perm
    idx, sc, fz, out = pace.ddae_select(dev_f32(vis), 4, dev_i32(perm), dev_f32(llm), nvs, keeps_ref,
                                        mode=0, hidden=dev_bf16(wvar.hidden))
    torch.cuda.synchronize()
    idx = host(idx)
    off = koff = 0
    for b, (n, K) in enumerate(zip(nvs, keeps_ref)):
        S_ref, st = oddae.fuse(vis[:, 4 * off:4 * (off + n)].astype(np.float64),
                               llm[:, off:off + n].astype(np.float64), 4, perm[off:off + n], 0)
        np.testing.assert_allclose(host(sc)[off:off + n], S_ref, atol=1e-5)
        ok, msg = kept_sets_agree(idx[koff:koff + K] - off, oddae.topk_indices(S_ref, K), S_ref)
        assert ok, (b, msg)
        off += n
        koff += K
    import torch as t
    np.testing.assert_array_equal(out.view(t.int16).cpu().numpy().view(np.uint16), wvar.hidden[idx])


def test_varlen_e2e_selection(wvar):
    """The packed batch end to end: each image's K from its APC density on the GPU (equal to the
    oracle's), the GPU's full-attention and prefill masses, the segmented selection; every
    image's kept set against the oracle-only selection (tests/golden/e2e_select.npz)."""
    from paper_2608_27206_amd import pace
    import torch
    nv_g, keep_g, S_g, idx_g = load_e2e_golden(4, wvar)
    keeps = []
    for img, nv in zip(wvar.images, nv_g):
        rho, _ = pace.apc_density(dev_u8(img), 14, 0.10, 0.6, 1.5)
        torch.cuda.synchronize()
        keeps.append(pace.keep_from_density(float(host(rho)[2]), int(nv)))
    assert keeps == list(keep_g)
    idx, sc = _e2e_gpu_selection(wvar, keeps)
    _check_e2e(idx, sc, nv_g, keep_g, S_g, idx_g)
