"""Pins for the attention oracle: pure-Python brute force on tiny inputs, closed forms,
invariants of the softmax and torch's float64 scaled_dot_product_attention as an
independent library routine."""
import math

import numpy as np
import pytest

from oracle import attention as oatt


def _brute(q, k, v, segs, causal, scale, mass_rows_fn):
    """Loops over (segment, head, query, key) with math.exp; returns O, LSE, mass."""
    N, hq, d = q.shape
    hkv = k.shape[1]
    g = hq // hkv
    O = np.zeros((N, hq, v.shape[2]))
    L = np.zeros((hq, N))
    M = np.zeros((hq, N))
    for (a, b) in segs:
        mrows = set(mass_rows_fn(a, b))
        for h in range(hq):
            kv = h // g
            for i in range(a, b):
                keys = [j for j in range(a, b) if (not causal or j <= i)]
                s = [scale * sum(q[i, h, t] * k[j, kv, t] for t in range(d)) for j in keys]
                mx = max(s)
                e = [math.exp(x - mx) for x in s]
                z = sum(e)
                for jj, j in enumerate(keys):
                    p = e[jj] / z
                    O[i, h, :] += p * v[j, kv, :]
                    if i in mrows:
                        M[h, j] += p
                L[h, i] = mx + math.log(z)
    return O, L, M


def test_vit_attention_brute_force():
    rs = np.random.default_rng(0)
    cu = [0, 5, 6, 13]                       # segments of 5, 1 and 7 tokens
    q = rs.standard_normal((13, 3, 4))
    k = rs.standard_normal((13, 3, 4))
    v = rs.standard_normal((13, 3, 5))
    scale = 0.7
    O, L, M = oatt.vit_attention(q, k, v, cu, scale)
    segs = [(cu[i], cu[i + 1]) for i in range(3)]
    Ob, Lb, Mb = _brute(q, k, v, segs, False, scale, lambda a, b: range(a, b))
    np.testing.assert_allclose(O, Ob, atol=1e-12)
    np.testing.assert_allclose(L, Lb, atol=1e-12)
    np.testing.assert_allclose(M, Mb, atol=1e-12)


def test_prefill_gqa_causal_brute_force():
    rs = np.random.default_rng(1)
    cu = [0, 7, 16]
    vis = [4, 6]
    q = rs.standard_normal((16, 6, 3))
    k = rs.standard_normal((16, 2, 3))
    v = rs.standard_normal((16, 2, 3))
    mq_start, mq_len = [4, 6], [3, 3]
    O, L, M = oatt.prefill_attention(q, k, v, cu, vis, mq_start, mq_len, 0.5)
    segs = [(0, 7), (7, 16)]
    Ob, Lb, Mb = _brute(q, k, v, segs, True, 0.5,
                        lambda a, b: range(a + (4 if a == 0 else 6), b))
    np.testing.assert_allclose(O, Ob, atol=1e-12)
    np.testing.assert_allclose(L, Lb, atol=1e-12)
    expect_mass = np.concatenate([Mb[:, 0:4], Mb[:, 7:13]], axis=1)
    np.testing.assert_allclose(M, expect_mass, atol=1e-12)


def test_prefill_visual_tokens_after_a_text_prefix_brute_force():
    """Visual tokens at an offset (a system prompt before the image): the mass of visual key j
    of sequence b is column vis_start[b] + j of the brute-force mass."""
    rs = np.random.default_rng(5)
    cu = [0, 9, 20]
    vis_start, vis = [2, 3], [4, 5]
    q = rs.standard_normal((20, 4, 3))
    k = rs.standard_normal((20, 2, 3))
    v = rs.standard_normal((20, 2, 3))
    mq_start, mq_len = [6, 8], [3, 3]
    O, L, M = oatt.prefill_attention(q, k, v, cu, vis, mq_start, mq_len, 0.5, vis_start=vis_start)
    segs = [(0, 9), (9, 20)]
    Ob, Lb, Mb = _brute(q, k, v, segs, True, 0.5, lambda a, b: range(a + (6 if a == 0 else 8), b))
    np.testing.assert_allclose(O, Ob, atol=1e-12)
    np.testing.assert_allclose(L, Lb, atol=1e-12)
    expect_mass = np.concatenate([Mb[:, 2:6], Mb[:, 12:17]], axis=1)
    np.testing.assert_allclose(M, expect_mass, atol=1e-12)


def test_against_torch_sdpa_float64():
    torch = pytest.importorskip("torch")
    import torch.nn.functional as F
    rs = np.random.default_rng(2)
    n, hq, hkv, d = 40, 8, 2, 16
    q = rs.standard_normal((n, hq, d))
    k = rs.standard_normal((n, hkv, d))
    v = rs.standard_normal((n, hkv, d))
    O, L, _ = oatt.attention_segment(q, k, v, True, 1 / math.sqrt(d))
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(k).permute(1, 0, 2)[None].repeat_interleave(hq // hkv, dim=1)
    tv = torch.from_numpy(v).permute(1, 0, 2)[None].repeat_interleave(hq // hkv, dim=1)
    ref = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True)[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(O, ref, atol=1e-12)
    # LSE from torch's logsumexp of the masked logits
    s = torch.einsum("hqd,hkd->hqk", tq[0], tk[0]) / math.sqrt(d)
    s = s.masked_fill(torch.triu(torch.ones(n, n, dtype=torch.bool), 1), float("-inf"))
    np.testing.assert_allclose(L, torch.logsumexp(s, -1).numpy(), atol=1e-12)


def test_zero_query_closed_forms_causal():
    """Q = 0: every visible key gets P = 1 / (#visible).  Causal row i sees i + 1 keys, so
    O[i] = mean(V[0..i]), LSE[i] = ln(i + 1) and mass[k] = sum_{i>=k, i in rows} 1 / (i + 1)."""
    rs = np.random.default_rng(3)
    n = 12
    q = np.zeros((n, 2, 4))
    k = rs.standard_normal((n, 1, 4))
    v = rs.standard_normal((n, 1, 4))
    O, L, M = oatt.attention_segment(q, k, v, True, 1.0, mass_rows=range(5, 12))
    for i in range(n):
        np.testing.assert_allclose(O[i, 0], v[: i + 1, 0].mean(0), atol=1e-14)
        assert L[1, i] == pytest.approx(math.log(i + 1), abs=1e-14)
    for kk in range(n):
        expect = sum(1.0 / (i + 1) for i in range(max(kk, 5), 12))
        assert M[0, kk] == pytest.approx(expect, abs=1e-14)


def test_zero_query_closed_forms_full():
    rs = np.random.default_rng(4)
    q = np.zeros((9, 2, 3))
    k = rs.standard_normal((9, 2, 3))
    v = rs.standard_normal((9, 2, 3))
    O, L, M = oatt.vit_attention(q, k, v, [0, 9], 1.3)
    np.testing.assert_allclose(O, np.broadcast_to(v.mean(0), O.shape), atol=1e-14)
    np.testing.assert_allclose(L, math.log(9), atol=1e-14)
    np.testing.assert_allclose(M, 1.0, atol=1e-14)          # 9 rows x 1/9 each


def test_gqa_head_mapping():
    """V of KV head j is the constant j + 1 and Q = 0, so query head h must output
    h // (Hq/Hkv) + 1.  Catches h % Hkv."""
    n, hq, hkv = 6, 8, 4
    q = np.zeros((n, hq, 2))
    k = np.random.default_rng(5).standard_normal((n, hkv, 2))
    v = np.zeros((n, hkv, 2))
    for j in range(hkv):
        v[:, j, :] = j + 1
    O, _, _ = oatt.attention_segment(q, k, v, True, 1.0)
    for h in range(hq):
        np.testing.assert_allclose(O[:, h, :], h // (hq // hkv) + 1, atol=1e-14)


def test_length_one_segments():
    rs = np.random.default_rng(6)
    q = rs.standard_normal((4, 2, 3))
    k = rs.standard_normal((4, 2, 3))
    v = rs.standard_normal((4, 2, 3))
    O, L, M = oatt.vit_attention(q, k, v, [0, 1, 2, 3, 4], 0.9)
    np.testing.assert_allclose(O, v, atol=1e-15)
    np.testing.assert_allclose(L, 0.9 * np.einsum("nhd,nhd->hn", q, k), atol=1e-14)
    np.testing.assert_allclose(M, 1.0, atol=1e-15)


def test_mass_invariants_windows_and_causal():
    rs = np.random.default_rng(7)
    cu = [0, 16, 32, 36, 37]
    q = rs.standard_normal((37, 2, 5)) * 2
    k = rs.standard_normal((37, 2, 5))
    v = rs.standard_normal((37, 2, 5))
    _, _, M = oatt.vit_attention(q, k, v, cu, 0.5)
    for a, b in zip(cu[:-1], cu[1:]):
        np.testing.assert_allclose(M[:, a:b].sum(1), b - a, atol=1e-12)   # rows sum to 1
    assert np.all(M > 0)
    # causal: keys after the last querying row receive nothing; totals equal the row count
    _, _, Mc = oatt.attention_segment(q[:20], k[:20], v[:20], True, 0.5, mass_rows=range(3, 9))
    assert np.all(Mc[:, 9:] == 0)
    np.testing.assert_allclose(Mc.sum(1), 6, atol=1e-12)


def test_rows_subset_matches_full():
    rs = np.random.default_rng(8)
    q = rs.standard_normal((30, 4, 8))
    k = rs.standard_normal((30, 2, 8))
    v = rs.standard_normal((30, 2, 8))
    O, L, _ = oatt.attention_segment(q, k, v, True, 0.3)
    rows = [0, 7, 29]
    o2, l2 = oatt.attention_rows(q, k, v, 0, 30, rows, True, 0.3)
    np.testing.assert_allclose(o2, O[rows], atol=1e-14)
    np.testing.assert_allclose(l2, L[:, rows], atol=1e-14)


def test_chunked_rows_match_brute_force():
    """The oracle walks query rows in chunks and adds each chunk's column sums into the mass;
    with a chunk of 4 rows over segments of 11 and 13 tokens (three and four chunks, ragged last
    ones) O, LSE and the mass must still equal the pure-Python brute force, so a chunk that
    overwrote instead of adding, or an offset slip between chunks, fails here."""
    rs = np.random.default_rng(11)
    q = rs.standard_normal((24, 2, 3))
    k = rs.standard_normal((24, 2, 3))
    v = rs.standard_normal((24, 2, 4))
    segs = [(0, 11), (11, 24)]
    for causal in (False, True):
        for a, b in segs:
            O, L, M = oatt.attention_segment(q[a:b], k[a:b], v[a:b], causal, 0.6,
                                             mass_rows=np.arange(b - a), chunk=4)
            Ob, Lb, Mb = _brute(q[a:b], k[a:b], v[a:b], [(0, b - a)], causal, 0.6, lambda x, y: range(x, y))
            np.testing.assert_allclose(O, Ob, atol=1e-12)
            np.testing.assert_allclose(L, Lb, atol=1e-12)
            np.testing.assert_allclose(M, Mb, atol=1e-12)
    # a subset of rows, and mass rows that start inside a chunk and span three of them
    rows = [1, 2, 7, 10]
    O, L, M = oatt.attention_segment(q[:11], k[:11], v[:11], True, 0.6, rows=rows,
                                     mass_rows=np.arange(2, 11), chunk=4)
    Ob, Lb, Mb = _brute(q[:11], k[:11], v[:11], [(0, 11)], True, 0.6, lambda x, y: range(2, 11))
    np.testing.assert_allclose(O, Ob[rows], atol=1e-12)
    np.testing.assert_allclose(L, Lb[:, rows], atol=1e-12)
    np.testing.assert_allclose(M, Mb, atol=1e-12)


def test_default_chunk_past_one_chunk():
    """More rows than the default chunk (600 > 512): O and LSE against torch's float64 SDPA, and
    each head's mass against the closed total (every row's probabilities sum to one) and a
    direct float64 column sum of the full probability matrix."""
    torch = pytest.importorskip("torch")
    import torch.nn.functional as F
    rs = np.random.default_rng(12)
    n, h, d = 600, 2, 8
    q = rs.standard_normal((n, h, d))
    k = rs.standard_normal((n, h, d))
    v = rs.standard_normal((n, h, d))
    O, L, M = oatt.attention_segment(q, k, v, False, 1 / math.sqrt(d), mass_rows=np.arange(n))
    qt, kt, vt = (torch.from_numpy(x).permute(1, 0, 2).contiguous() for x in (q, k, v))
    ref = F.scaled_dot_product_attention(qt, kt, vt).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(O, ref, atol=1e-12)
    S = torch.einsum("qhd,khd->hqk", torch.from_numpy(q), torch.from_numpy(k)) / math.sqrt(d)
    np.testing.assert_allclose(L, torch.logsumexp(S, dim=2).numpy(), atol=1e-12)
    np.testing.assert_allclose(M, torch.softmax(S, dim=2).sum(dim=1).numpy(), atol=1e-10)
    np.testing.assert_allclose(M.sum(axis=1), n, rtol=1e-12)
