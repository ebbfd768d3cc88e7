"""GPU parity of APC density and resize against the float64 oracle.

Density: d_i within 1e-4, rho_g / rho_d / rho / phi within 1e-4 (fp32 accumulation).
Resize: the rounded output equals the oracle's wherever the oracle's exact value is more
than 1e-3 from a rounding boundary, and is within one level everywhere."""
import numpy as np
import pytest

from oracle import apc as oapc
from paper_2608_27206_amd import workloads as wl
from tests.gpu_util import dev_u8, host, rho4, say

pytestmark = pytest.mark.gpu


def _density(img, tail=0.1):
    from paper_2608_27206_amd import pace
    import torch
    rho, d = pace.apc_density(dev_u8(img), 14, tail, 0.6, 1.5)
    torch.cuda.synchronize()
    return host(rho), host(d)


def _check_density(img, tail=0.1):
    say(f"apc density {img.shape}")
    rho, d = _density(img, tail)
    ref = oapc.apc_density(img, 14, tail)
    np.testing.assert_allclose(d, ref["d"], atol=1e-4)
    np.testing.assert_allclose(rho4(rho), [ref["rho_g"], ref["rho_d"], ref["rho"], ref["phi"]], atol=1e-4)
    return rho


def test_density_img448():
    _check_density(wl.make_image(1, 448, 448))


def test_density_ragged_tiles_and_tails():
    img = wl.make_image(5, 14 * 7, 14 * 37)        # 37 patches per row: 2 full tiles + 5
    _check_density(img, 0.05)
    _check_density(img, 0.2)


def test_density_odd_byte_count():
    """7-pixel patches on a 21 x 35 image: H*W*3 is odd, so the last pixels sit in a
    partial dword at the end of the buffer."""
    from paper_2608_27206_amd import pace
    import torch
    img = np.random.default_rng(6).integers(0, 256, size=(21, 35, 3), dtype=np.uint8)
    assert (img.size % 4) != 0
    rho, d = pace.apc_density(dev_u8(img), 7, 0.1, 0.6, 1.5)
    torch.cuda.synchronize()
    ref = oapc.apc_density(img, 7, 0.1)
    np.testing.assert_allclose(host(d), ref["d"], atol=1e-4)
    np.testing.assert_allclose(rho4(host(rho)), [ref["rho_g"], ref["rho_d"], ref["rho"], ref["phi"]], atol=1e-4)


def test_density_more_patches_than_the_register_tail():
    """51,072 patches: more than the tail kernel holds in registers (49,152), so the
    distances are re-read from memory for the top-10% selection.  phi is checked through
    the identity mean pairwise cosine = ||mean T||^2, which the CPU tests pin against the
    double sum (the double sum itself would take minutes here)."""
    img = wl.make_image(7, 14 * 228, 14 * 224)
    say(f"apc density {img.shape} (tail from memory)")
    rho, d = _density(img)
    T = oapc.l2_normalise(oapc.patch_features(img, 14))
    phi = float(np.sum(T.mean(axis=0) ** 2))
    d_ref = oapc.detail_distances(T, oapc.background_direction(T))
    rho_d = min(oapc.tail_mean(d_ref, 0.1) / oapc.GAMMA, 1.0)
    np.testing.assert_allclose(d, d_ref, atol=1e-4)
    np.testing.assert_allclose(rho4(rho), [1 - phi, rho_d, oapc.ALPHA * (1 - phi) + (1 - oapc.ALPHA) * rho_d, phi],
                               atol=1e-4)


def test_density_uniform_and_mirrored():
    u = np.full((56, 84, 3), 77, np.uint8)
    rho = _check_density(u)
    assert abs(rho[2]) < 1e-5
    left = np.random.default_rng(5).integers(0, 256, size=(42, 56, 3), dtype=np.uint8)
    rho = _check_density(np.concatenate([left, 255 - left], axis=1))
    assert abs(rho[2] - 13 / 15) < 1e-4


@pytest.mark.parametrize("n_b", [60, 200, 270])
def test_density_tail_ties_in_each_ranking_path(n_b):
    """Exact ties at the tail threshold.  576 patches of two kinds (n_b of kind B, the rest A,
    at seeded positions): the minority kind lies farther from the mean direction, and all its
    patches have bitwise equal distances, so the n_tail = 58 largest are 58 of its n_b equal
    values and the threshold bin holds all n_b of them.  60 candidates are ranked by one wave,
    200 by the LDS loop and 270 by the radix select; 576 is not a multiple of 1024, so the
    tail's zero padding slots are present too.  gamma = 100 keeps rho_d = d_top / 100 unclamped."""
    from paper_2608_27206_amd import pace
    import torch
    rng = np.random.default_rng(40 + n_b)
    a = rng.integers(0, 256, size=(14, 14, 3), dtype=np.uint8)
    b = rng.integers(0, 256, size=(14, 14, 3), dtype=np.uint8)
    kinds = np.zeros(24 * 24, bool)
    kinds[rng.choice(24 * 24, n_b, replace=False)] = True
    img = np.empty((24 * 14, 24 * 14, 3), np.uint8)
    for i, is_b in enumerate(kinds):
        r, c = divmod(i, 24)
        img[14 * r:14 * r + 14, 14 * c:14 * c + 14] = b if is_b else a
    say(f"apc density tail ties: {n_b} of 576 patches at the threshold")
    rho, d = pace.apc_density(dev_u8(img), 14, 0.1, 0.6, 100.0)
    torch.cuda.synchronize()
    rho, d = host(rho), host(d)
    ref = oapc.apc_density(img, 14, 0.1, gamma=100.0)
    assert len(np.unique(d[kinds])) == 1 and d[kinds][0] > d[~kinds][0]
    np.testing.assert_allclose(d, ref["d"], atol=1e-4)
    np.testing.assert_allclose(rho[1] * 100.0, ref["d_top"], atol=1e-5)
    np.testing.assert_allclose(rho4(rho), [ref["rho_g"], ref["rho_d"], ref["rho"], ref["phi"]], atol=1e-4)


@pytest.mark.parametrize("case", range(6))
def test_density_random_shapes(case):
    """Seeded random images: patch size 7, 14 or 16, 1-40 patches per side, tail fractions in
    (0, 1]; d_i and rho against the oracle."""
    from paper_2608_27206_amd import pace
    import torch
    rng = np.random.default_rng(300 + case)
    P = int(rng.choice([7, 14, 16]))
    gh, gw = int(rng.integers(1, 41)), int(rng.integers(1, 41))
    tail = float(rng.choice([0.01, 0.1, 0.37, 1.0]))
    img = rng.integers(0, 256, size=(gh * P, gw * P, 3), dtype=np.uint8)
    img[: (gh * P) // 2] //= 3                      # some structure: a darker half
    say(f"apc density random {img.shape} patch={P} tail={tail}")
    rho, d = pace.apc_density(dev_u8(img), P, tail, 0.6, 1.5)
    torch.cuda.synchronize()
    ref = oapc.apc_density(img, P, tail)
    np.testing.assert_allclose(host(d), ref["d"], atol=1e-4)
    np.testing.assert_allclose(rho4(host(rho)), [ref["rho_g"], ref["rho_d"], ref["rho"], ref["phi"]], atol=1e-4)


@pytest.mark.parametrize("patch,gh,gw", [(1, 40, 37), (2, 23, 31), (5, 17, 29), (3, 64, 70), (11, 9, 67)])
def test_density_small_and_odd_patches(patch, gh, gw):
    """Patch sizes whose rows split unevenly over a patch's four threads (3P bytes: 3, 6, 15, 9
    and 33), with a tile row of more than 64 patches (a second tile per patch row); d_i and rho
    against the oracle."""
    from paper_2608_27206_amd import pace
    import torch
    rng = np.random.default_rng(400 + patch)
    img = rng.integers(0, 256, size=(gh * patch, gw * patch, 3), dtype=np.uint8)
    img[:, : (gw * patch) // 3] //= 2
    say(f"apc density {img.shape} patch={patch}")
    rho, d = pace.apc_density(dev_u8(img), patch, 0.1, 0.6, 1.5)
    torch.cuda.synchronize()
    ref = oapc.apc_density(img, patch, 0.1)
    np.testing.assert_allclose(host(d), ref["d"], atol=1e-4)
    np.testing.assert_allclose(rho4(host(rho)), [ref["rho_g"], ref["rho_d"], ref["rho"], ref["phi"]], atol=1e-4)


def _check_resize(img, oh, ow):
    from paper_2608_27206_amd import pace
    import torch
    say(f"resize {img.shape} -> {oh}x{ow}")
    out = pace.apc_downsample(dev_u8(img), oh, ow)
    torch.cuda.synchronize()
    got = host(out).astype(np.int64)
    exact = oapc.resize_bicubic_exact(img, oh, ow)
    ref = oapc.round_u8(exact).astype(np.int64)
    frac = exact - np.floor(exact)
    near = np.abs(frac - 0.5) < 1e-3
    assert np.max(np.abs(got - ref)) <= 1
    assert np.all(got[~near] == ref[~near])
    return got


@pytest.mark.parametrize("shape,out", [((448, 448), (224, 224)), ((448, 448), (308, 308)),
                                       ((150, 333), (149, 100)), ((96, 128), (96, 128)),
                                       ((300, 200), (37, 23)), ((64, 64), (2, 2)),
                                       ((2156, 3836), (1078, 1918)), ((250, 200), (100, 80)),
                                       ((300, 128), (150, 128)), ((210, 330), (90, 150))])
def test_resize_parity(shape, out):
    img = wl.make_image(3, *shape)
    _check_resize(img, *out)


@pytest.mark.parametrize("case", range(6))
def test_resize_random_shapes(case):
    """Seeded random sizes: input sides 1-700; in even cases outputs from 1/32 of each side up to
    the side (the staged kernels), in odd cases shrink factors drawn log-uniformly in [1, 300]
    per side (beyond 32x the per-pixel kernel runs)."""
    rng = np.random.default_rng(400 + case)
    H, W = int(rng.integers(1, 701)), int(rng.integers(1, 701))
    if case % 2:
        oh = min(H, max(1, round(H / 10 ** rng.uniform(0, np.log10(300)))))
        ow = min(W, max(1, round(W / 10 ** rng.uniform(0, np.log10(300)))))
    else:
        oh = int(rng.integers(max(1, -(-H // 32)), H + 1))
        ow = int(rng.integers(max(1, -(-W // 32)), W + 1))
    img = rng.integers(0, 256, size=(H, W, 3), dtype=np.uint8)
    _check_resize(img, oh, ow)


@pytest.mark.parametrize("shape,out", [((64, 64), (1, 1)), ((700, 500), (10, 7)), ((300, 2000), (5, 40)),
                                       ((1000, 40), (1, 1)), ((90, 4000), (80, 30)), ((2156, 3836), (20, 30)),
                                       ((1, 3000), (1, 20)), ((3000, 1), (2, 1)), ((33, 33), (1, 33))])
def test_resize_beyond_32x(shape, out):
    """Shrinks beyond 32x per side (one side or both; down to a single pixel), per output pixel
    from memory, against the oracle."""
    rng = np.random.default_rng(shape[0] * 7 + shape[1])
    img = rng.integers(0, 256, size=(*shape, 3), dtype=np.uint8)
    img[: shape[0] // 2] //= 2
    _check_resize(img, *out)


# ---------------------------------------------------------------- caller-supplied embeddings
def _check_features(bits, tail=0.1, atol=1e-4):
    from paper_2608_27206_amd import pace
    import torch
    from tests.gpu_util import dev_bf16
    say(f"apc density features {bits.shape}")
    rho, d = pace.apc_density_features(dev_bf16(bits), tail, 0.6, 1.5)
    torch.cuda.synchronize()
    ref = oapc.embedding_density(wl.bf16_bits_to_f64(bits), tail)
    np.testing.assert_allclose(host(d), ref["d"], atol=atol)
    np.testing.assert_allclose(rho4(host(rho)), [ref["rho_g"], ref["rho_d"], ref["rho"], ref["phi"]], atol=atol)
    return host(rho), host(d)


# 20,000 and 46,000 rows reach the tail's 32- and 48-distance forms
@pytest.mark.parametrize("n,dim", [(3000, 1280), (777, 8), (130, 592), (64, 3584), (500, 3), (257, 100),
                                   (20000, 16), (46000, 8)])
def test_density_features_random(n, dim):
    rs = np.random.default_rng(n + dim)
    x = rs.normal(size=(n, dim)).astype(np.float32) + rs.normal(size=(1, dim)).astype(np.float32)
    _check_features(wl.f32_to_bf16_bits(x))


def test_density_features_of_patch_pixels_match_image_path():
    """The pixel stand-in features, rounded to bf16 and fed as embeddings."""
    img = wl.make_image(1, 448, 448)
    f = oapc.patch_features(img, 14).astype(np.float32)
    _check_features(wl.f32_to_bf16_bits(f))


def test_density_features_opposite_identical_and_zero_rows():
    rs = np.random.default_rng(6)
    x = rs.normal(size=(50, 64)).astype(np.float32)
    x = np.concatenate([x, -x, np.zeros((1, 64), np.float32)])
    rho, d = _check_features(wl.f32_to_bf16_bits(x))
    assert abs(rho[0] - 1.0) < 1e-5 and d[100] == 0.0
    rho, d = _check_features(wl.f32_to_bf16_bits(np.tile(x[:1], (33, 1))))
    assert abs(rho[0]) < 1e-5 and np.max(d) < 1e-3   # phi = 1 - rho_g = 1


def test_density_features_beyond_the_register_tail():
    """More rows than the tail kernel holds in registers (49,152): the tail re-reads d."""
    rs = np.random.default_rng(8)
    x = rs.normal(size=(50000, 16)).astype(np.float32)
    _check_features(wl.f32_to_bf16_bits(x))


# ---------------------------------------------------------------- pixel-statistic previews
# Preview vectors: within rtol 1e-5 + atol 1e-6 of the float64 oracle (fp32 sums of at most 256
# terms; the octant of each gradient is exact integer arithmetic on both sides).  Densities of
# those vectors: the 1e-4 bar of the image path.
@pytest.mark.parametrize("kind", [0, 1, 2, 3])
@pytest.mark.parametrize("shape,patch", [((448, 448), 14), ((196, 308), 14), ((48, 80), 16), ((9, 12), 3)])
def test_pixel_features_parity(kind, shape, patch):
    from paper_2608_27206_amd import pace
    import torch
    img = wl.make_image(1, shape[0], shape[1])
    say(f"pixel features kind={kind} {shape} patch={patch}")
    got = pace.apc_pixel_features(dev_u8(img), kind, patch)
    torch.cuda.synchronize()
    ref = oapc.pixel_statistic_features(img, patch, kind)
    assert got.shape == ref.shape
    np.testing.assert_allclose(host(got), ref, rtol=1e-5, atol=1e-6)


@pytest.mark.parametrize("kind", [0, 1, 2, 3])
@pytest.mark.parametrize("shape", [(448, 448), (196, 308)])
def test_pixel_density_parity(kind, shape):
    from paper_2608_27206_amd import pace
    import torch
    img = wl.make_image(2, shape[0], shape[1])
    say(f"pixel density kind={kind} {shape}")
    rho, d = pace.apc_pixel_density(dev_u8(img), kind, 14)
    torch.cuda.synchronize()
    ref = oapc.pixel_density(img, 14, kind)
    np.testing.assert_allclose(host(d), ref["d"], atol=1e-4)
    np.testing.assert_allclose(rho4(host(rho)), [ref["rho_g"], ref["rho_d"], ref["rho"], ref["phi"]], atol=1e-4)


def test_pixel_features_full_frame():
    """All four previews of a 2156 x 3836 frame (42,196 patches) against the oracle, element by
    element."""
    from paper_2608_27206_amd import pace
    import torch
    img = wl.make_image(1, 2156, 3836)
    dimg = dev_u8(img)
    for kind in range(4):
        say(f"pixel features full frame kind={kind}")
        got = pace.apc_pixel_features(dimg, kind, 14)
        torch.cuda.synchronize()
        np.testing.assert_allclose(host(got), oapc.pixel_statistic_features(img, 14, kind), rtol=1e-5, atol=1e-6)


def test_pixel_density_flat_and_tiled():
    """A flat image: zero edge and Laplacian vectors, so phi = 0 and rho_g = 1; a tiling of one
    patch: equal RGB-statistic vectors, phi = 1 and every d_i = 0 (up to rounding)."""
    from paper_2608_27206_amd import pace
    import torch
    flat = np.full((56, 84, 3), 77, np.uint8)
    for kind in (2, 3):
        rho, d = pace.apc_pixel_density(dev_u8(flat), kind, 14)
        torch.cuda.synchronize()
        assert host(rho)[0] == 1.0 and np.all(host(d) == 0)   # phi = 0
    tile = np.random.default_rng(3).integers(0, 256, size=(14, 14, 3), dtype=np.uint8)
    rho, d = pace.apc_pixel_density(dev_u8(np.tile(tile, (4, 5, 1))), 0, 14)
    torch.cuda.synchronize()
    assert abs(host(rho)[0]) < 1e-5 and np.max(host(d)) < 1e-3


def test_pixel_rejects_bad_kind_and_patch():
    from paper_2608_27206_amd import pace
    img = dev_u8(wl.make_image(1, 28, 28))
    with pytest.raises(pace.PaceError, match="kind"):
        pace.apc_pixel_features(img, 4, 14)
    with pytest.raises(pace.PaceError, match="patch"):
        pace.apc_pixel_features(img, 0, 28 * 0 + 17)


def test_images_on_parallel_streams_match_serial():
    """Independent images' density and resize chains run side by side on four streams (as the
    benchmark's multi-image step does) give bit-identical d, rho and resized pixels to the same
    calls in series: the calls share no state beyond their own arguments and workspaces."""
    from paper_2608_27206_amd import pace
    import torch
    w = wl.make_workload(4)
    imgs = [dev_u8(im) for im in w.images]
    say(f"{len(imgs)} images on 4 streams: " + ", ".join(f"{im.shape[1]}x{im.shape[0]}" for im in w.images))
    lib = pace.lib()

    def buffers():
        out = []
        for im in w.images:
            H, W = im.shape[:2]
            out.append({"ws": torch.empty(lib.pace_apc_density_workspace_size(H, W, 14), dtype=torch.uint8, device="cuda"),
                        "d": torch.empty((H // 14) * (W // 14), dtype=torch.float32, device="cuda"),
                        "rho": torch.empty(3, dtype=torch.float32, device="cuda"),
                        "small": torch.empty((H // 2, W // 2, 3), dtype=torch.uint8, device="cuda")})
        return out

    def chain(img, b):
        pace.apc_density(img, 14, 0.10, 0.6, 1.5, d_out=b["d"], rho_out=b["rho"], workspace=b["ws"])
        pace.apc_downsample(img, b["small"].shape[0], b["small"].shape[1], dst=b["small"])

    serial = buffers()
    for img, b in zip(imgs, serial):
        chain(img, b)
    torch.cuda.synchronize()
    par = buffers()
    cur = torch.cuda.current_stream()
    streams = [torch.cuda.Stream() for _ in range(4)]
    for rep in range(2):
        for b in par:
            for t in b.values():
                t.fill_(3)
        for s in streams:
            s.wait_stream(cur)
        for i, (img, b) in enumerate(zip(imgs, par)):
            with torch.cuda.stream(streams[i % 4]):
                chain(img, b)
        for s in streams:
            cur.wait_stream(s)
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(serial, par)):
            for k in ("d", "rho", "small"):
                assert torch.equal(a[k], b[k]), f"pass {rep}, image {i}: {k} differs from the serial calls"
