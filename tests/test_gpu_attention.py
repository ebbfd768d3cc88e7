"""GPU parity of the attention kernels against the float64 oracle.

Bars: O max-abs error <= 2e-2, LSE abs error <= 1e-3, per-key mass relative error <= 1e-3
(|m_gpu - m_ref| <= 1e-3 m_ref + 1e-12 |Q_set|); keys no querying row can see get exactly 0."""
import math

import numpy as np
import pytest

from oracle import attention as oatt
from paper_2608_27206_amd import workloads as wl
from tests.gpu_util import (dev_bf16, dev_i32, host, host_bf16_to_f64, mass_ok, say)

pytestmark = pytest.mark.gpu

O_TOL = 2e-2
LSE_TOL = 1e-3


def _vit_case(seed, cu, H, d):
    N = cu[-1]
    q = wl.random_bf16(seed, (N, H, d))
    k = wl.random_bf16(seed + 1, (N, H, d))
    v = wl.random_bf16(seed + 2, (N, H, d))
    return q, k, v


def _run_vit(q, k, v, cu, maxlen):
    from paper_2608_27206_amd import pace
    import torch
    o, lse, mass = pace.vit_attention(dev_bf16(q), dev_bf16(k), dev_bf16(v), dev_i32(cu), maxlen)
    torch.cuda.synchronize()
    return host_bf16_to_f64(o), host(lse), host(mass)


def _check_vit(q, k, v, cu, d):
    N = cu[-1]
    maxlen = int(np.max(np.diff(cu)))
    say(f"vit case N={N} H={q.shape[1]} d={d} nseg={len(cu) - 1} maxlen={maxlen}")
    o, lse, mass = _run_vit(q, k, v, cu, maxlen)
    Or, Lr, Mr = oatt.vit_attention(wl.bf16_bits_to_f64(q), wl.bf16_bits_to_f64(k),
                                    wl.bf16_bits_to_f64(v), cu, 1 / math.sqrt(d))
    assert np.max(np.abs(o - Or)) <= O_TOL
    assert np.max(np.abs(lse - Lr)) <= LSE_TOL
    err, rel = mass_ok(mass, Mr, maxlen)
    assert err <= 0, f"mass rel err {rel}"
    for a, b in zip(cu[:-1], cu[1:]):   # rows of a segment sum to 1
        np.testing.assert_allclose(mass[:, a:b].sum(1), b - a, rtol=1e-4)


@pytest.mark.parametrize("d", [80, 128])
def test_vit_full_ragged(d):
    cu = [0, 1000]
    q, k, v = _vit_case(1, cu, 4, d)
    _check_vit(q, k, v, cu, d)


@pytest.mark.parametrize("d", [80, 128])
def test_vit_windows_and_ragged_segments(d):
    sizes = [64, 64, 16, 4, 64, 1, 33, 130, 64, 257]
    cu = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    q, k, v = _vit_case(5, cu, 3, d)
    _check_vit(q, k, v, cu, d)


@pytest.mark.parametrize("d", [80, 128])
def test_vit_short_windows_single_pass(d):
    """Segments of at most 64 tokens with mass requested take the single-pass window kernel
    (O, LSE and mass together)."""
    sizes = [64, 16, 4, 1, 33, 64, 50, 63, 64]
    cu = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    q, k, v = _vit_case(7, cu, 3, d)
    _check_vit(q, k, v, cu, d)


def test_vit_short_windows_large_logits():
    sizes = [64, 7, 64, 40]
    cu = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    N = int(cu[-1])
    q = wl.random_bf16(41, (N, 2, 80), 2.5)
    k = wl.random_bf16(42, (N, 2, 80), 2.5)
    v = wl.random_bf16(43, (N, 2, 80))
    _check_vit(q, k, v, cu, 80)


def test_vit_large_logits():
    """Logits with std ~ 6 stress the online max and the rescaling."""
    cu = [0, 700]
    N, H, d = 700, 2, 80
    q = wl.random_bf16(11, (N, H, d), 2.5)
    k = wl.random_bf16(12, (N, H, d), 2.5)
    v = wl.random_bf16(13, (N, H, d))
    _check_vit(q, k, v, cu, d)


def test_vit_long_segments_d80():
    """Segments of 1024 rows or more take the rotation forward kernel at head dim 80 (fp16
    PV product on V^T tiles in the workspace); shorter segments of the same call, at offsets
    that are not multiples of 8, go through it too."""
    sizes = [1100, 37, 1536, 300, 1]
    cu = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    q, k, v = _vit_case(21, cu, 2, 80)
    _check_vit(q, k, v, cu, 80)


def test_vit_long_segment_large_logits_d80():
    cu = [0, 1290]
    N, H, d = 1290, 2, 80
    q = wl.random_bf16(31, (N, H, d), 2.5)
    k = wl.random_bf16(32, (N, H, d), 2.5)
    v = wl.random_bf16(33, (N, H, d))
    _check_vit(q, k, v, cu, d)


@pytest.mark.parametrize("vscale", [300.0, 1e-5])
def test_vit_long_segment_value_range_d80(vscale):
    """The rotation kernel converts V to fp16: large values (well inside fp16's range) and
    tiny ones (fp16 subnormals) keep O within 2e-2 of its largest magnitude."""
    sizes = [1030, 70]
    cu = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    N, H, d = int(cu[-1]), 2, 80
    q = wl.random_bf16(41, (N, H, d))
    k = wl.random_bf16(42, (N, H, d))
    v = wl.random_bf16(43, (N, H, d), vscale)
    say(f"vit long segment, V scale {vscale}")
    o, lse, _ = _run_vit(q, k, v, cu, int(max(sizes)))
    Or, Lr, _ = oatt.vit_attention(wl.bf16_bits_to_f64(q), wl.bf16_bits_to_f64(k), wl.bf16_bits_to_f64(v),
                                   cu, 1 / math.sqrt(d), with_mass=False)
    assert np.max(np.abs(o - Or)) <= O_TOL * np.max(np.abs(Or))
    assert np.max(np.abs(lse - Lr)) <= LSE_TOL


def _scale_bits(v, k):
    """bf16 bits of v * 2^k, exactly (the exponent field moves by k; zeros stay zero)."""
    v = v.astype(np.int32)
    e = (v >> 7) & 0xFF
    assert np.all((e == 0) | ((e + k > 0) & (e + k < 255)))
    return np.where(e == 0, v, v + (k << 7)).astype(np.uint16)


@pytest.mark.parametrize("k", [17, -20, 100, -100])
def test_vit_long_segment_any_finite_v_d80(k):
    """V at 2^k times N(0,1) (up to ~6e5 at k = 17, ~1e-6 at k = -20, and 2^+-100): fp16 holds
    none of these directly, but the long-segment kernel scales each (segment, head) by a power
    of two before the fp16 PV product and undoes it on the output, so O(2^k V) is exactly
    2^k O(V), bit for bit, and the LSE is unchanged; O also matches the oracle within 2e-2 of
    its largest magnitude."""
    sizes = [1100, 70]
    cu = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    N, H, d = int(cu[-1]), 2, 80
    q, kk, v = _vit_case(44, cu, H, d)
    vs = _scale_bits(v, k)
    say(f"vit long segment, V scaled by 2^{k}")
    o0, l0, m0 = _run_vit(q, kk, v, cu, int(max(sizes)))
    o1, l1, m1 = _run_vit(q, kk, vs, cu, int(max(sizes)))
    np.testing.assert_array_equal(o1, np.ldexp(o0, k))
    np.testing.assert_array_equal(l1, l0)
    np.testing.assert_array_equal(m1, m0)
    Or, Lr, _ = oatt.vit_attention(wl.bf16_bits_to_f64(q), wl.bf16_bits_to_f64(kk), wl.bf16_bits_to_f64(vs),
                                   cu, 1 / math.sqrt(d), with_mass=False)
    assert np.max(np.abs(o1 - Or)) <= O_TOL * np.max(np.abs(Or))
    assert np.max(np.abs(l1 - Lr)) <= LSE_TOL


def test_vit_long_segment_neighbour_out_of_fp16_range_d80():
    """Two long segments packed in one call, the second with V at ~2^20 (beyond fp16): the first
    segment's O and LSE equal, bit for bit, those of a call whose second segment is unscaled
    (no tile of one segment reads the other's V^T columns, and each has its own scale), and the
    second segment's O is exactly 2^20 times its unscaled output."""
    sizes = [1100, 1030]
    cu = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    N, H, d = int(cu[-1]), 2, 80
    q, kk, v = _vit_case(45, cu, H, d)
    v2 = v.copy()
    v2[1100:] = _scale_bits(v[1100:], 20)
    o0, l0, _ = _run_vit(q, kk, v, cu, 1100)
    o1, l1, _ = _run_vit(q, kk, v2, cu, 1100)
    np.testing.assert_array_equal(o1[:1100], o0[:1100])
    np.testing.assert_array_equal(o1[1100:], np.ldexp(o0[1100:], 20))
    np.testing.assert_array_equal(l1, l0)
    assert np.all(np.isfinite(o1))


@pytest.mark.parametrize("sizes,d", [([0, 64, 0, 17, 0], 80),              # windows, fused mass
                                     ([1100, 0, 0, 37, 1030, 0], 80),     # long-segment kernel
                                     ([0, 300, 0, 129], 128)])            # general kernel
def test_vit_empty_segments(sizes, d):
    """Empty segments (equal neighbouring offsets) are skipped: the other segments' outputs,
    LSE and mass match the oracle and every row's mass still sums over its own segment."""
    cu = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    q, k, v = _vit_case(51, cu, 2, d)
    _check_vit(q, k, v, cu, d)


@pytest.mark.parametrize("sizes", [[1023], [1024], [1025, 63], [1087, 64, 1], [1152, 1151, 5]])
def test_vit_long_segment_tile_boundaries_d80(sizes):
    """Lengths around the long-segment kernel's threshold (1024 rows) and last tiles holding
    1, 63 or 64 keys, with short segments in the same call."""
    cu = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    q, k, v = _vit_case(61 + len(sizes), cu, 2, 80)
    _check_vit(q, k, v, cu, 80)


def _run_prefill(p, d_override=None):
    from paper_2608_27206_amd import pace
    import torch
    cu = p.cu_seqlens
    seqlens = np.diff(cu)
    o, lse, mass = pace.prefill_attention_with_mass(
        dev_bf16(p.q), dev_bf16(p.k), dev_bf16(p.v), dev_i32(cu), int(seqlens.max()),
        dev_i32(p.vis_len), dev_i32(p.cu_vis), int(p.cu_vis[-1]), int(p.vis_len.max()),
        dev_i32(p.mq_start), dev_i32(p.mq_len), int(p.mq_len.max()))
    torch.cuda.synchronize()
    return host_bf16_to_f64(o), host(lse), host(mass)


def _check_prefill(p):
    d = p.q.shape[2]
    say(f"prefill case Ntot={p.q.shape[0]} Hq={p.q.shape[1]} Hkv={p.k.shape[1]} d={d} "
        f"B={len(p.vis_len)}")
    o, lse, mass = _run_prefill(p)
    Or, Lr, Mr = oatt.prefill_attention(wl.bf16_bits_to_f64(p.q), wl.bf16_bits_to_f64(p.k),
                                        wl.bf16_bits_to_f64(p.v), p.cu_seqlens, p.vis_len,
                                        p.mq_start, p.mq_len, 1 / math.sqrt(d))
    assert np.max(np.abs(o - Or)) <= O_TOL
    assert np.max(np.abs(lse - Lr)) <= LSE_TOL
    err, rel = mass_ok(mass[:, :Mr.shape[1]], Mr, int(p.mq_len.max()))
    assert err <= 0, f"mass rel err {rel}"
    return mass, Mr


def test_prefill_tiny_config():
    w = wl.make_workload(0)
    mass, Mr = _check_prefill(w.prefill)
    # every visual key is seen by every text row: per head the mass sums to the text length
    np.testing.assert_allclose(mass.sum(1), Mr.sum(1), rtol=1e-4)


def _packed(seed, vis, text, hq, hkv, d):
    seqlens = [a + b for a, b in zip(vis, text)]
    n = sum(seqlens)
    cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32)
    cuv = np.concatenate([[0], np.cumsum(vis)]).astype(np.int32)
    return wl.PrefillInputs(q=wl.random_bf16(seed, (n, hq, d)), k=wl.random_bf16(seed + 1, (n, hkv, d)),
                            v=wl.random_bf16(seed + 2, (n, hkv, d)), cu_seqlens=cu,
                            vis_len=np.asarray(vis, np.int32), text_len=np.asarray(text, np.int32),
                            cu_vis=cuv, salient=[])


def test_prefill_varlen_gqa_d128():
    _check_prefill(_packed(21, [100, 300, 7], [40, 64, 5], 28, 4, 128))


@pytest.mark.parametrize("d", [128, 80])
def test_prefill_visual_tokens_after_a_text_prefix(d):
    """Sequences laid out [text prefix][visual][text query] (a system prompt before the image):
    the mass of the visual keys from the query text against the oracle, one sequence with an
    empty prefix."""
    from paper_2608_27206_amd import pace
    import torch
    prefix, vis, text = [13, 0, 70], [100, 300, 7], [40, 64, 5]
    seqlens = [a + b + c for a, b, c in zip(prefix, vis, text)]
    n = sum(seqlens)
    cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32)
    cuv = np.concatenate([[0], np.cumsum(vis)]).astype(np.int32)
    hq, hkv = (28, 4) if d == 128 else (8, 2)
    q, k, v = (wl.random_bf16(71 + i, (n, h, d)) for i, h in enumerate((hq, hkv, hkv)))
    mq_start = np.asarray([a + b for a, b in zip(prefix, vis)], np.int32)
    mq_len = np.asarray(text, np.int32)
    say(f"prefill with text prefixes {prefix}, d={d}")
    o, lse, mass = pace.prefill_attention_with_mass(
        dev_bf16(q), dev_bf16(k), dev_bf16(v), dev_i32(cu), int(max(seqlens)), dev_i32(np.asarray(vis, np.int32)),
        dev_i32(cuv), int(cuv[-1]), int(max(vis)), dev_i32(mq_start), dev_i32(mq_len), int(mq_len.max()),
        vis_start=dev_i32(np.asarray(prefix, np.int32)))
    torch.cuda.synchronize()
    Or, Lr, Mr = oatt.prefill_attention(wl.bf16_bits_to_f64(q), wl.bf16_bits_to_f64(k), wl.bf16_bits_to_f64(v),
                                        cu, vis, mq_start, mq_len, 1 / math.sqrt(d), vis_start=prefix)
    assert np.max(np.abs(host_bf16_to_f64(o) - Or)) <= O_TOL
    assert np.max(np.abs(host(lse) - Lr)) <= LSE_TOL
    err, rel = mass_ok(host(mass)[:, :Mr.shape[1]], Mr, int(mq_len.max()))
    assert err <= 0, f"mass rel err {rel}"


def test_prefill_varlen_d80():
    _check_prefill(_packed(31, [130, 9], [70, 200], 8, 2, 80))


def test_prefill_all_rows_mass():
    """'Vision + Text' source: every row of the sequence queries; causal keys see fewer rows."""
    p = _packed(41, [150, 40], [50, 9], 14, 2, 128)
    p.text_len = p.text_len.copy()
    seqlens = np.diff(p.cu_seqlens)
    p2 = wl.PrefillInputs(q=p.q, k=p.k, v=p.v, cu_seqlens=p.cu_seqlens, vis_len=p.vis_len,
                          text_len=p.text_len, cu_vis=p.cu_vis, salient=[])
    from paper_2608_27206_amd import pace
    import torch
    o, lse, mass = pace.prefill_attention_with_mass(
        dev_bf16(p2.q), dev_bf16(p2.k), dev_bf16(p2.v), dev_i32(p2.cu_seqlens), int(seqlens.max()),
        dev_i32(p2.vis_len), dev_i32(p2.cu_vis), int(p2.cu_vis[-1]), int(p2.vis_len.max()),
        dev_i32([0, 0]), dev_i32(seqlens), int(seqlens.max()))
    torch.cuda.synchronize()
    _, _, Mr = oatt.prefill_attention(wl.bf16_bits_to_f64(p2.q), wl.bf16_bits_to_f64(p2.k),
                                      wl.bf16_bits_to_f64(p2.v), p2.cu_seqlens, p2.vis_len,
                                      [0, 0], seqlens, 1 / math.sqrt(128))
    err, rel = mass_ok(host(mass), Mr, int(seqlens.max()))
    assert err <= 0, f"mass rel err {rel}"


def test_prefill_no_querying_rows_gives_zero_mass():
    p = _packed(51, [64], [16], 4, 1, 128)
    from paper_2608_27206_amd import pace
    import torch
    o, lse, mass = pace.prefill_attention_with_mass(
        dev_bf16(p.q), dev_bf16(p.k), dev_bf16(p.v), dev_i32(p.cu_seqlens), 80, dev_i32(p.vis_len),
        dev_i32(p.cu_vis), 64, 64, dev_i32([64]), dev_i32([0]), 0)
    torch.cuda.synchronize()
    assert np.all(host(mass) == 0)


def test_mass_only_entry_matches_fused_call():
    from paper_2608_27206_amd import pace
    import torch
    cu = np.array([0, 64, 128, 500], np.int32)
    q, k, v = _vit_case(61, cu, 2, 80)
    Q, K, V, CU = dev_bf16(q), dev_bf16(k), dev_bf16(v), dev_i32(cu)
    o, lse, mass = pace.vit_attention(Q, K, V, CU, 372)
    o2, lse2, _ = pace.vit_attention(Q, K, V, CU, 372, want_mass=False)
    m2 = pace.vit_attention_mass(Q, K, CU, 372, lse2)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(mass), host(m2))
    np.testing.assert_array_equal(host(lse), host(lse2))


@pytest.mark.parametrize("case", range(8))
def test_vit_random_shapes(case):
    """Seeded random shapes: head count, head dim, and segment mixes that cross the kernels'
    selection rules (all segments of at most 64 tokens -> the fused window kernel; a segment of
    1,024+ tokens at head dim 80 -> the rotation kernel; otherwise the general forward)."""
    rng = np.random.default_rng(900 + case)
    kind = case % 4
    d = 80 if kind == 2 else int(rng.choice([80, 128]))   # the rotation kernel is head dim 80 only
    H = int(rng.choice([1, 3, 5]))
    if kind == 0:     # windows only
        sizes = rng.integers(1, 65, size=int(rng.integers(1, 12)))
    elif kind == 1:   # short and mid segments
        sizes = rng.integers(1, 700, size=int(rng.integers(1, 5)))
    elif kind == 2:   # one long segment among short ones
        sizes = np.concatenate([rng.integers(1, 200, size=2), [int(rng.integers(1024, 1600))]])
    else:             # empty segments mixed in
        sizes = rng.integers(0, 300, size=int(rng.integers(2, 7)))
        sizes[rng.integers(0, sizes.size)] = 0
    sizes = [int(x) for x in sizes]
    if sum(sizes) == 0:
        sizes[0] = 1
    cu = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    q, k, v = _vit_case(1000 + case, cu, H, d)
    _check_vit(q, k, v, cu, d)


@pytest.mark.parametrize("case", range(6))
def test_prefill_random_shapes(case):
    """Seeded random GQA prefills: groups of 1-7 query heads per KV head, head dim 80 or 128,
    images of 1-3 sequences with random visual and text lengths (text may be as short as 1)."""
    rng = np.random.default_rng(950 + case)
    d = int(rng.choice([80, 128]))
    hkv = int(rng.choice([1, 2, 4]))
    group = int(rng.integers(1, 8))
    nb = int(rng.integers(1, 4))
    vis = [int(x) for x in rng.integers(1, 400, size=nb)]
    text = [int(x) for x in rng.integers(1, 150, size=nb)]
    _check_prefill(_packed(2000 + case, vis, text, hkv * group, hkv, d))
