"""Pins for the APC oracle (Section 3.2): closed forms, brute force and bounds.

None of these recompute the oracle's own formulas: expected values come from hand
derivations (tests/golden), colour-level closed forms in 3 dimensions, pure-Python
brute force over small inputs, or library routines."""
import json
import math
import os

import numpy as np
import pytest

from oracle import apc

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def test_defaults_match_paper_constants():
    hp = _gold("paper_hyperparameters.json")
    assert apc.ALPHA == hp["alpha"]["value"]
    assert apc.GAMMA == hp["gamma"]["value"]
    assert apc.TAIL_FRAC == hp["tail_frac"]["value"]


def _uniform(H, W, rgb):
    img = np.empty((H, W, 3), np.uint8)
    img[:] = np.asarray(rgb, np.uint8)
    return img


def test_uniform_image_closed_form():
    g = _gold("apc_closed_forms.json")["uniform_image"]
    r = apc.apc_density(_uniform(56, 84, (200, 31, 77)))
    assert r["phi"] == pytest.approx(g["phi"], abs=1e-12)
    assert r["rho_g"] == pytest.approx(g["rho_g"], abs=1e-12)
    assert np.max(np.abs(r["d"])) < 1e-7
    assert r["rho_d"] == pytest.approx(g["rho_d"], abs=1e-7)
    assert r["rho"] == pytest.approx(g["rho"], abs=1e-7)


def test_mirrored_image_closed_form():
    g = _gold("apc_closed_forms.json")["mirrored_image"]
    rs = np.random.default_rng(5)
    left = rs.integers(0, 256, size=(42, 56, 3), dtype=np.uint8)   # 3 x 4 patches
    img = np.concatenate([left, 255 - left], axis=1)               # 3 x 8 patches
    r = apc.apc_density(img)
    assert r["phi"] == pytest.approx(g["phi"], abs=1e-12)
    assert r["rho_g"] == pytest.approx(g["rho_g"], abs=1e-12)
    np.testing.assert_allclose(r["d"], 1.0, atol=1e-12)
    assert r["rho_d"] == pytest.approx(g["rho_d"], abs=1e-12)
    assert r["rho"] == pytest.approx(g["rho"], abs=1e-12)


def _unit3(rgb):
    f = np.asarray(rgb, np.float64) / 127.5 - 1.0
    return f / np.linalg.norm(f)


@pytest.mark.parametrize("n_a,n_b", [(1, 15), (3, 13), (5, 11), (8, 8)])
def test_two_colour_closed_form(n_a, n_b):
    """Patches of two flat colours a, b.  A flat patch's feature repeats its colour's 3-vector,
    so T = u_colour (repeated, /sqrt(196)) and cos(T_a, T_b) = u_a . u_b in 3-D.  With
    p = n_a / N: phi = p^2 + q^2 + 2 p q cos; c = p T_a + q T_b;
    d_a^2 = 2 - 2 (p + q cos) / |c|, d_b^2 = 2 - 2 (q + p cos) / |c|, |c|^2 = phi."""
    ca, cb = (250, 10, 40), (20, 60, 230)
    N = n_a + n_b
    patches = [ca] * n_a + [cb] * n_b
    img = np.empty((14, 14 * N, 3), np.uint8)
    for i, c in enumerate(patches):
        img[:, 14 * i:14 * (i + 1), :] = c
    cos = float(_unit3(ca) @ _unit3(cb))
    p, q = n_a / N, n_b / N
    phi = p * p + q * q + 2 * p * q * cos
    nc = math.sqrt(phi)
    da = math.sqrt(max(0.0, 2 - 2 * (p + q * cos) / nc))
    db = math.sqrt(max(0.0, 2 - 2 * (q + p * cos) / nc))
    n_tail = math.ceil(0.1 * N - 1e-9)
    ds = sorted([da] * n_a + [db] * n_b, reverse=True)[:n_tail]
    d_top = sum(ds) / n_tail
    rho_d = min(d_top / 1.5, 1.0)
    rho = 0.6 * (1 - phi) + 0.4 * rho_d
    r = apc.apc_density(img)
    assert r["phi"] == pytest.approx(phi, abs=1e-12)
    assert r["rho_g"] == pytest.approx(1 - phi, abs=1e-12)
    np.testing.assert_allclose(np.sort(r["d"]), np.sort([da] * n_a + [db] * n_b), atol=1e-7)
    assert r["d_top"] == pytest.approx(d_top, abs=1e-7)
    assert r["rho"] == pytest.approx(rho, abs=1e-7)


def test_patch_order_is_raster_over_patch_grid():
    """Feature row py*gw + px holds patch (py, px); its first entries are that patch's pixel
    (0, 0) channels.  Catches a transposed patch grid."""
    gh, gw = 3, 5
    img = np.zeros((14 * gh, 14 * gw, 3), np.uint8)
    for py in range(gh):
        for px in range(gw):
            img[14 * py:14 * (py + 1), 14 * px:14 * (px + 1), 0] = 10 * py + px
    f = apc.patch_features(img)
    assert f.shape == (gh * gw, 588)
    for py in range(gh):
        for px in range(gw):
            assert f[py * gw + px, 0] == pytest.approx((10 * py + px) / 127.5 - 1.0)


def test_phi_pairwise_brute_force():
    """Eq. 1 by explicit Python double loop over pairs on a tiny image."""
    rs = np.random.default_rng(1)
    img = rs.integers(0, 256, size=(28, 42, 3), dtype=np.uint8)      # 6 patches
    f = apc.patch_features(img)
    T = f / np.linalg.norm(f, axis=1, keepdims=True)
    N = T.shape[0]
    tot = 0.0
    for i in range(N):
        for j in range(N):
            a, b = T[i], T[j]
            tot += sum(x * y for x, y in zip(a, b)) / (math.sqrt(sum(x * x for x in a)) *
                                                       math.sqrt(sum(y * y for y in b)))
    assert apc.global_density(T) == pytest.approx(tot / (N * N), abs=1e-12)
    # identity: sum_ij T_i.T_j = |sum_i T_i|^2 (check of the chunked evaluation)
    assert apc.global_density(T, chunk=2) == pytest.approx(float(np.sum(T, 0) @ np.sum(T, 0)) / N ** 2,
                                                           abs=1e-12)


@pytest.mark.parametrize("n,frac", [(10, 0.1), (11, 0.1), (1024, 0.1), (196, 0.05), (30, 0.2), (1, 0.1)])
def test_tail_mean_brute_force(n, frac):
    rs = np.random.default_rng(n)
    d = rs.random(n)
    k = max(1, math.ceil(frac * n - 1e-9))
    # exact ceil for decimal fractions
    from fractions import Fraction
    kk = max(1, -(-Fraction(str(frac)) * n // 1))
    assert k == kk
    expect = sum(sorted(d.tolist(), reverse=True)[:k]) / k
    assert apc.tail_mean(d, frac) == pytest.approx(expect, abs=1e-12)


def test_bounds_random_images():
    rs = np.random.default_rng(7)
    for _ in range(3):
        img = rs.integers(0, 256, size=(56, 70, 3), dtype=np.uint8)
        r = apc.apc_density(img)
        assert 0 <= r["rho_g"] <= 1 + 1e-12
        assert np.all(r["d"] >= 0) and np.all(r["d"] <= 2 + 1e-12)
        assert 0 <= r["rho_d"] <= 1 and 0 <= r["rho"] <= 1 + 1e-12


def test_target_size_rules():
    # rho inside the budget: area ratio rho, sides * sqrt(rho), snapped to 28
    assert apc.target_size(0.25, 1120, 1680, 0, 1e12, 28) == (560, 840)
    # hard cap binds: max_pixels / area
    oh, ow = apc.target_size(0.9, 2000, 2000, 0, 1000 * 1000, 1)
    assert (oh, ow) == (1000, 1000)
    # floor binds for rho = 0
    oh, ow = apc.target_size(0.0, 1000, 1000, 250000, 1e12, 1)
    assert (oh, ow) == (500, 500)
    # never larger than the input, never below one snap
    assert apc.target_size(1.0, 50, 50, 0, 1e12, 28) == (28, 28)
    assert apc.target_size(0.0, 3000, 3000, 0, 1e12, 28) == (28, 28)


# ---------------------------------------------------------------- caller-supplied embeddings
def test_embedding_density_equals_image_path_on_patch_features():
    """Feeding the pixel stand-in features as embeddings reproduces the image path."""
    img = np.random.default_rng(5).integers(0, 256, size=(112, 140, 3), dtype=np.uint8)
    ref = apc.apc_density(img, 14)
    got = apc.embedding_density(apc.patch_features(img, 14))
    for key in ("phi", "rho_g", "rho_d", "rho"):
        assert abs(got[key] - ref[key]) < 1e-12
    np.testing.assert_allclose(got["d"], ref["d"], atol=1e-12)


def test_embedding_density_is_scale_invariant_per_row():
    rs = np.random.default_rng(3)
    x = rs.normal(size=(300, 40))
    scale = rs.uniform(0.01, 100.0, size=(300, 1))
    a = apc.embedding_density(x)
    b = apc.embedding_density(x * scale)
    for key in ("phi", "rho_g", "rho_d", "rho"):
        assert abs(a[key] - b[key]) < 1e-12


def test_embedding_density_dot_form_matches_cosines_for_nonzero_rows():
    rs = np.random.default_rng(4)
    x = rs.normal(size=(257, 33)) + 0.3
    T = apc.normalise_embeddings(x)
    assert abs(apc.global_density_dot(T) - apc.global_density(T)) < 1e-12
    # explicit double loop on a small case
    y = rs.normal(size=(7, 5))
    Ty = apc.normalise_embeddings(y)
    brute = sum(float(Ty[i] @ Ty[j]) for i in range(7) for j in range(7)) / 49
    assert abs(apc.global_density_dot(Ty) - brute) < 1e-14


def test_embedding_density_opposite_rows_and_zero_row():
    """Rows and their negatives: c = 0, so phi = 0, rho_g = 1 and every unit row has d = 1; a zero
    row is a zero direction, so its distance is ||c_hat|| (here 0)."""
    rs = np.random.default_rng(5)
    x = rs.normal(size=(50, 16))
    x = np.concatenate([x, -x, np.zeros((1, 16))])
    r = apc.embedding_density(x)
    assert abs(r["phi"]) < 1e-15 and abs(r["rho_g"] - 1.0) < 1e-15
    np.testing.assert_allclose(r["d"][:100], 1.0, atol=1e-12)
    assert r["d"][100] == 0.0
    # identical rows: phi = 1 and every distance is 0
    s = apc.embedding_density(np.tile(rs.normal(size=(1, 16)), (20, 1)))
    assert abs(s["phi"] - 1.0) < 1e-12 and np.max(s["d"]) < 1e-7


# ---------------------------------------------------------------- pixel-statistic previews
def test_pixel_statistics_shapes_and_closed_forms():
    rs = np.random.default_rng(9)
    img = rs.integers(0, 256, size=(28, 42, 3), dtype=np.uint8)
    for kind, dim in ((0, 6), (1, 64), (2, 8), (3, 196)):
        f = apc.pixel_statistic_features(img, 14, kind)
        assert f.shape == (6, dim)
    # RGB statistics: a patch of one colour has that colour's mean and zero spread
    flat = np.zeros((14, 14, 3), np.uint8)
    flat[...] = (10, 200, 255)
    f = apc.pixel_statistic_features(flat, 14, 0)
    np.testing.assert_allclose(f[0], [10 / 255, 200 / 255, 1.0, 0, 0, 0], atol=1e-14)
    # population std (ddof 0): half the pixels 0 and half 255 give mean 0.5 and std 0.5 in every
    # channel; a quarter at 255 gives mean 1/4 and std sqrt(1/4 * 3/4) (ddof 1 would scale the
    # spread by sqrt(196/195))
    split = np.zeros((14, 14, 3), np.uint8)
    split[:, :7] = 255
    np.testing.assert_allclose(apc.pixel_statistic_features(split, 14, 0)[0], [0.5] * 6, atol=1e-14)
    quarter = np.zeros((14, 14, 3), np.uint8)
    quarter[:7, :7] = 255
    np.testing.assert_allclose(apc.pixel_statistic_features(quarter, 14, 0)[0],
                               [0.25] * 3 + [math.sqrt(3) / 4] * 3, atol=1e-14)
    # colour entropy: the terms of a patch sum to its entropy; half black half white -> ln 2
    half = np.zeros((14, 14, 3), np.uint8)
    half[:7] = 255
    e = apc.pixel_statistic_features(half, 14, 1)[0]
    assert abs(e.sum() - math.log(2)) < 1e-15 and np.count_nonzero(e) == 2
    # one colour: zero entropy; Laplacian and edges vanish on a constant image
    assert np.all(apc.pixel_statistic_features(flat, 14, 1) == 0)
    assert np.all(apc.pixel_statistic_features(flat, 14, 3) == 0)
    assert np.all(apc.pixel_statistic_features(flat, 14, 2) == 0)


def test_pixel_statistics_edges_and_laplacian_by_hand():
    """A vertical step edge: Sobel gx = 4 * step at the two columns beside it (grey scaled by
    1000), gy = 0, so all magnitude lands in octant 0 (gradient pointing +x) and the octant-0
    total is 2 columns * 14 rows * 4 * step / (255 * 196).  The Laplacian is +-step/255 beside
    the edge."""
    img = np.zeros((14, 14, 3), np.uint8)
    img[:, 7:] = 100                       # grey 100 on the right
    e = apc.pixel_statistic_features(img, 14, 2)[0]
    assert abs(e[0] - 2 * 14 * 4 * 100 / (255 * 196)) < 1e-12 and np.all(e[1:] == 0)
    lap = apc.pixel_statistic_features(img, 14, 3)[0].reshape(14, 14)
    np.testing.assert_allclose(lap[:, 6], -100 / 255, atol=1e-12)
    np.testing.assert_allclose(lap[:, 7], 100 / 255, atol=1e-12)
    assert np.all(lap[:, :6] == 0) and np.all(lap[:, 8:] == 0)
    # the mirrored edge points the other way: octant 4
    e2 = apc.pixel_statistic_features(img[:, ::-1].copy(), 14, 2)[0]
    assert e2[4] > 0 and np.count_nonzero(e2) == 1


def test_pixel_statistics_octants_against_atan2():
    rs = np.random.default_rng(10)
    gx = rs.integers(-50, 51, size=5000)
    gy = rs.integers(-50, 51, size=5000)
    o = apc._octant(gx, gy)
    ang = np.degrees(np.arctan2(gy, gx)) % 360.0
    away = np.abs(ang / 45.0 - np.round(ang / 45.0)) > 1e-9     # not on a boundary
    np.testing.assert_array_equal(o[away], np.floor(ang[away] / 45.0).astype(np.int64))
    assert apc._octant(np.array([0]), np.array([0]))[0] == 0


def test_pixel_density_special_cases():
    """A tiling of one patch makes every preview vector equal: phi = 1, rho_g = 0 and every
    d_i = 0 (for kinds whose vector is not zero).  A flat image has zero edge and Laplacian
    vectors: every direction is zero, so phi = 0 and rho_g = 1."""
    rs = np.random.default_rng(11)
    tile = rs.integers(0, 256, size=(14, 14, 3), dtype=np.uint8)
    img = np.tile(tile, (3, 4, 1))
    for kind in (0, 1):
        r = apc.pixel_density(img, 14, kind)
        assert abs(r["phi"] - 1.0) < 1e-12 and np.max(r["d"]) < 1e-7
    flat = np.full((28, 28, 3), 77, np.uint8)
    for kind in (2, 3):
        r = apc.pixel_density(flat, 14, kind)
        assert r["phi"] == 0.0 and r["rho_g"] == 1.0
