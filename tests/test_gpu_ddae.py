"""GPU parity of DDAE selection (fusion, top-K, gather) against the float64 oracle.

Top-K and gather fed the oracle's scores (as fp32) must be bit-exact; fused scores agree to
1e-5; end to end, kept sets may differ only on pairs whose oracle scores lie within 1e-3."""
import numpy as np
import pytest

from oracle import ddae as oddae
from paper_2608_27206_amd import workloads as wl
from tests.gpu_util import dev_bf16, dev_f32, dev_i32, host, kept_sets_agree, say

pytestmark = pytest.mark.gpu


def _topk_case(S32, K, hidden_bits):
    from paper_2608_27206_amd import pace
    import torch
    idx, out = pace.topk_gather(dev_f32(S32), K, dev_bf16(hidden_bits))
    torch.cuda.synchronize()
    ref = oddae.topk_indices(S32.astype(np.float32), K)
    got = host(idx).astype(np.int64)
    np.testing.assert_array_equal(got, ref)
    import torch as t
    out_bits = out.view(t.int16).cpu().numpy().view(np.uint16)
    np.testing.assert_array_equal(out_bits, hidden_bits[ref])


@pytest.mark.parametrize("n,K,levels", [(196, 20, None), (10549, 1055, None), (5000, 500, 3),
                                        (1000, 1, None), (1000, 999, None), (777, 77, 1),
                                        # ~41 and ~82 equal scores per level: ties ranked by
                                        # the one-wave path and by the LDS loop
                                        (4096, 1000, 100), (4096, 1024, 50),
                                        # largest image held in registers, and past it (the
                                        # scores are then re-read from memory)
                                        (16384, 1639, None), (16385, 1700, 4), (40000, 4000, None)])
def test_topk_gather_bit_exact_on_oracle_scores(n, K, levels):
    say(f"topk n={n} K={K} levels={levels}")
    rs = np.random.default_rng(n * 7 + K)
    if levels is None:
        S = rs.random(n).astype(np.float32)
    else:
        S = (rs.integers(0, levels, n) / max(1, levels)).astype(np.float32)
    S[::97] = 0.0
    hidden = wl.random_bf16(n, (n, 256))
    _topk_case(S, K, hidden)


@pytest.mark.parametrize("case", range(8))
def test_topk_gather_random_shapes(case):
    """Seeded random sizes on both sides of the register path's limit (16,384 scores), random
    K in [1, n - 1], scores continuous or on a few levels (ties), hidden rows of 64-512 values."""
    rs = np.random.default_rng(700 + case)
    n = int(rs.choice([int(rs.integers(2, 3000)), int(rs.integers(3000, 16385)), int(rs.integers(16385, 40000))]))
    K = int(rs.integers(1, n))
    levels = None if case % 2 == 0 else int(rs.integers(1, 200))
    say(f"topk random n={n} K={K} levels={levels}")
    if levels is None:
        S = rs.random(n).astype(np.float32)
    else:
        S = (rs.integers(0, levels, n) / levels).astype(np.float32)
    hidden = wl.random_bf16(case, (n, 64 * int(rs.integers(1, 9))))
    _topk_case(S, K, hidden)


def test_topk_negative_and_signed_zero():
    S = np.array([-1.0, -0.0, 0.0, 2.0, -3.5, 1e-30, -1e-30, 0.5] * 30, np.float32)
    hidden = wl.random_bf16(99, (S.size, 64))
    _topk_case(S, 37, hidden)


def test_topk_edge_counts():
    from paper_2608_27206_amd import pace
    import torch
    S = np.random.default_rng(3).random(300).astype(np.float32)
    for K in (0, 300):
        idx, _ = pace.topk_gather(dev_f32(S), K, None)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(idx), np.arange(K))


def _fuse_case(vis, llm, merge, perm, mode, K, hidden=None):
    from paper_2608_27206_amd import pace
    import torch
    nv = llm.shape[1]
    idx, sc, fz, out = pace.ddae_select(dev_f32(vis), merge, None if perm is None else dev_i32(perm),
                                        dev_f32(llm), [nv], [K], mode=mode, tau=0.5,
                                        w_llm_fixed=0.5,
                                        hidden=None if hidden is None else dev_bf16(hidden))
    torch.cuda.synchronize()
    S_ref, st = oddae.fuse(vis.astype(np.float64), llm.astype(np.float64), merge, perm, mode, 0.5, 0.5)
    np.testing.assert_allclose(host(sc), S_ref, atol=1e-5)
    np.testing.assert_allclose(host(fz)[0], st, atol=1e-5)
    idx_ref = oddae.topk_indices(S_ref, K)
    ok, msg = kept_sets_agree(host(idx), idx_ref, S_ref)
    assert ok, msg
    # given the GPU's own fp32 scores, the selection is exactly the oracle's rule
    np.testing.assert_array_equal(host(idx), oddae.topk_indices(host(sc), K))
    if hidden is not None:
        import torch as t
        got = out.view(t.int16).cpu().numpy().view(np.uint16)
        np.testing.assert_array_equal(got, hidden[host(idx)])
    return host(idx)


def test_fuse_dynamic_with_merge_and_perm():
    rs = np.random.default_rng(7)
    nv = 2304
    vis = rs.gamma(0.5, size=(16, 4 * nv)).astype(np.float32)
    llm = rs.gamma(0.3, size=(28, nv)).astype(np.float32)
    perm = rs.permutation(nv).astype(np.int32)
    _fuse_case(vis, llm, 4, perm, 0, 231, wl.random_bf16(7, (nv, 3584)))


def test_fuse_dynamic_large_image_from_memory():
    """An image too large for the register-resident path (more than 16,384 tokens)."""
    rs = np.random.default_rng(12)
    nv = 20000
    vis = rs.gamma(0.5, size=(4, nv)).astype(np.float32)
    llm = rs.gamma(0.3, size=(6, nv)).astype(np.float32)
    _fuse_case(vis, llm, 1, None, 0, 2000)


def test_fuse_fixed_tiny_config_end_to_end_inputs():
    w = wl.make_workload(0)
    rs = np.random.default_rng(8)
    llm = rs.gamma(0.5, size=(8, 196)).astype(np.float32)
    _fuse_case(w.vit_mass.astype(np.float32), llm, 1, None, 1, 20, w.hidden)


def test_fuse_constant_map():
    rs = np.random.default_rng(9)
    vis = np.ones((2, 400), np.float32)
    llm = rs.random((3, 400)).astype(np.float32)
    _fuse_case(vis, llm, 1, None, 0, 40)


def test_varlen_segments():
    from paper_2608_27206_amd import pace
    import torch
    rs = np.random.default_rng(10)
    nvs = [256, 1000, 37, 2304]
    keeps = [oddae.keep_count(r, n) for r, n in zip([0.05, 0.25, 0.1, 0.17], nvs)]
    nt = sum(nvs)
    vis = rs.gamma(0.5, size=(16, 4 * nt)).astype(np.float32)
    llm = rs.gamma(0.3, size=(28, nt)).astype(np.float32)
    perm = np.concatenate([rs.permutation(n) for n in nvs]).astype(np.int32)
    hidden = wl.random_bf16(10, (nt, 512))
    idx, sc, fz, out = pace.ddae_select(dev_f32(vis), 4, dev_i32(perm), dev_f32(llm), nvs, keeps,
                                        mode=0, hidden=dev_bf16(hidden))
    torch.cuda.synchronize()
    idx = host(idx)
    off = 0
    koff = 0
    for b, (n, K) in enumerate(zip(nvs, keeps)):
        S_ref, st = oddae.fuse(vis[:, 4 * off:4 * (off + n)].astype(np.float64),
                               llm[:, off:off + n].astype(np.float64), 4, perm[off:off + n], 0)
        np.testing.assert_allclose(host(sc)[off:off + n], S_ref, atol=1e-5)
        np.testing.assert_allclose(host(fz)[b], st, atol=1e-5)
        got = idx[koff:koff + K] - off
        ok, msg = kept_sets_agree(got, oddae.topk_indices(S_ref, K), S_ref)
        assert ok, msg
        np.testing.assert_array_equal(got, oddae.topk_indices(host(sc)[off:off + n], K))
        off += n
        koff += K
    import torch as t
    np.testing.assert_array_equal(out.view(t.int16).cpu().numpy().view(np.uint16), hidden[idx])


def test_determinism():
    from paper_2608_27206_amd import pace
    import torch
    rs = np.random.default_rng(11)
    vis = rs.gamma(0.5, size=(16, 4 * 3000)).astype(np.float32)
    llm = rs.gamma(0.3, size=(28, 3000)).astype(np.float32)
    r1 = pace.ddae_select(dev_f32(vis), 4, None, dev_f32(llm), [3000], [300])
    r2 = pace.ddae_select(dev_f32(vis), 4, None, dev_f32(llm), [3000], [300])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(r1[0]), host(r2[0]))
    np.testing.assert_array_equal(host(r1[1]), host(r2[1]))


@pytest.mark.parametrize("big", [False, True])
def test_varlen_more_images_than_one_launch(big):
    """150 images in one call (three launches of at most 64 images; one image past the
    register-resident size when `big`, so its launch takes the general path), against the
    oracle per image: scores, fusion weights, kept sets and the gathered rows."""
    from paper_2608_27206_amd import pace
    import torch
    import torch as t
    rs = np.random.default_rng(150 + big)
    nvs = [int(x) for x in rs.integers(1, 400, size=150)]
    if big:
        nvs[100] = 17000
    keeps = [oddae.keep_count(float(r), n) for r, n in zip(rs.uniform(0.0, 1.0, size=150), nvs)]
    nt = sum(nvs)
    say(f"varlen 150 images, {nt} tokens, keep {sum(keeps)}")
    vis = rs.gamma(0.5, size=(2, nt)).astype(np.float32)
    llm = rs.gamma(0.3, size=(3, nt)).astype(np.float32)
    hidden = wl.random_bf16(nt, (nt, 64))
    idx, sc, fz, out = pace.ddae_select(dev_f32(vis), 1, None, dev_f32(llm), nvs, keeps,
                                        mode=0, hidden=dev_bf16(hidden))
    torch.cuda.synchronize()
    idx, sc, fz = host(idx), host(sc), host(fz)
    assert idx.size == sum(keeps)
    off = koff = 0
    for b, (n, K) in enumerate(zip(nvs, keeps)):
        S_ref, st = oddae.fuse(vis[:, off:off + n].astype(np.float64),
                               llm[:, off:off + n].astype(np.float64), 1, None, 0)
        np.testing.assert_allclose(sc[off:off + n], S_ref, atol=1e-5)
        np.testing.assert_allclose(fz[b], st, atol=1e-5)
        got = idx[koff:koff + K] - off
        ok, msg = kept_sets_agree(got, oddae.topk_indices(S_ref, K), S_ref)
        assert ok, (b, msg)
        np.testing.assert_array_equal(got, oddae.topk_indices(sc[off:off + n], K))
        off += n
        koff += K
    np.testing.assert_array_equal(out.view(t.int16).cpu().numpy().view(np.uint16), hidden[idx])


def test_varlen_keep_none_all_and_many_rows():
    """Images whose K is 0, all of the image, or spread over many gather workgroups, in one
    batch; and a batch with an image past the register-resident size (every image then takes
    the general path)."""
    from paper_2608_27206_amd import pace
    import torch
    import torch as t
    for nvs, ratios in (([300, 64, 16384, 5000, 1], [0.0, 1.0, 0.5, 0.1, 1.0]),
                        ([17000, 300, 2], [0.1, 0.3, 0.5])):
        say(f"varlen nvs={nvs}")
        rs = np.random.default_rng(sum(nvs))
        keeps = [oddae.keep_count(r, n) for r, n in zip(ratios, nvs)]
        nt = sum(nvs)
        vis = rs.gamma(0.5, size=(2, nt)).astype(np.float32)
        llm = rs.gamma(0.3, size=(3, nt)).astype(np.float32)
        hidden = wl.random_bf16(nt, (nt, 64))
        idx, sc, fz, out = pace.ddae_select(dev_f32(vis), 1, None, dev_f32(llm), nvs, keeps,
                                            mode=0, hidden=dev_bf16(hidden))
        torch.cuda.synchronize()
        idx = host(idx)
        assert idx.size == sum(keeps)
        off = koff = 0
        for b, (n, K) in enumerate(zip(nvs, keeps)):
            S_ref, st = oddae.fuse(vis[:, off:off + n].astype(np.float64),
                                   llm[:, off:off + n].astype(np.float64), 1, None, 0)
            np.testing.assert_allclose(host(sc)[off:off + n], S_ref, atol=1e-5)
            np.testing.assert_allclose(host(fz)[b], st, atol=1e-5)
            got = idx[koff:koff + K] - off
            ok, msg = kept_sets_agree(got, oddae.topk_indices(S_ref, K), S_ref)
            assert ok, msg
            np.testing.assert_array_equal(got, oddae.topk_indices(host(sc)[off:off + n], K))
            off += n
            koff += K
        np.testing.assert_array_equal(out.view(t.int16).cpu().numpy().view(np.uint16), hidden[idx])


def test_topk_many_rows_per_workgroup():
    """K large enough that each gather workgroup copies more than the minimum four rows."""
    rs = np.random.default_rng(21)
    S = rs.random(16000).astype(np.float32)
    S[5000:9000] = 0.5   # a long run of ties at the threshold
    _topk_case(S, 8000, wl.random_bf16(21, (16000, 48)))


def test_per_tile_and_global_selection():
    """InternVL-style tiles (the cross-model study): "-T" keeps ceil(ratio * n) tokens inside
    each tile (one segment per tile), "-G" keeps the same total over all tiles' tokens at once
    (one segment).  Both against the oracle rule."""
    from paper_2608_27206_amd import pace
    import torch
    rs = np.random.default_rng(31)
    tiles = [256] * 6 + [256]          # six 448x448 tiles and the thumbnail, 256 tokens each
    nt = sum(tiles)
    vis = rs.gamma(0.5, size=(16, nt)).astype(np.float32)
    llm = rs.gamma(0.3, size=(28, nt)).astype(np.float32)
    hidden = wl.random_bf16(31, (nt, 128))
    per = [oddae.keep_count(0.1, n) for n in tiles]
    idx_t, sc_t, _, out_t = pace.ddae_select(dev_f32(vis), 1, None, dev_f32(llm), tiles, per,
                                             hidden=dev_bf16(hidden))
    idx_g, sc_g, _, out_g = pace.ddae_select(dev_f32(vis), 1, None, dev_f32(llm), [nt], [sum(per)],
                                             hidden=dev_bf16(hidden))
    torch.cuda.synchronize()
    # -T: every tile keeps exactly its own share, chosen by its own normalised scores
    got_t = host(idx_t)
    off = koff = 0
    for n, K in zip(tiles, per):
        S_ref, _ = oddae.fuse(vis[:, off:off + n].astype(np.float64), llm[:, off:off + n].astype(np.float64), 1,
                              None, 0)
        part = got_t[koff:koff + K] - off
        assert np.all((part >= 0) & (part < n))
        ok, msg = kept_sets_agree(part, oddae.topk_indices(S_ref, K), S_ref)
        assert ok, msg
        off += n
        koff += K
    # -G: one ranking over all tiles; the per-tile counts follow the scores
    S_g, _ = oddae.fuse(vis.astype(np.float64), llm.astype(np.float64), 1, None, 0)
    ok, msg = kept_sets_agree(host(idx_g), oddae.topk_indices(S_g, sum(per)), S_g)
    assert ok, msg
    import torch as t
    np.testing.assert_array_equal(out_t.view(t.int16).cpu().numpy().view(np.uint16), hidden[got_t])
    np.testing.assert_array_equal(out_g.view(t.int16).cpu().numpy().view(np.uint16), hidden[host(idx_g)])
