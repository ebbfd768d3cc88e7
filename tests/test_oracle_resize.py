"""Pins for the oracle's bicubic resize (Appendix, Detailed Implementation Specifics: sides
scaled by sqrt(r) with bicubic interpolation)."""
import numpy as np
import pytest

from oracle import apc


def _keys(x, a=-0.5):
    """Keys' cubic written out per piece, for hand-checking single weights."""
    x = abs(x)
    if x <= 1:
        return (a + 2) * x ** 3 - (a + 3) * x ** 2 + 1
    if x < 2:
        return a * x ** 3 - 5 * a * x ** 2 + 8 * a * x - 4 * a
    return 0.0


def test_keys_kernel_values():
    # interpolating kernel: 1 at 0, 0 at the integers, Keys' a = -0.5 value at 1.5 is -0.0625
    k = apc.keys_cubic(np.array([0.0, 1.0, 2.0, 0.5, 1.5, -1.5]))
    np.testing.assert_allclose(k, [1.0, 0.0, 0.0, 0.5625, -0.0625, -0.0625], atol=1e-15)


def test_identity_at_scale_one():
    rs = np.random.default_rng(0)
    img = rs.integers(0, 256, size=(37, 53, 3), dtype=np.uint8)
    np.testing.assert_array_equal(apc.resize_bicubic(img, 37, 53), img)


def test_constant_image_stays_constant():
    img = np.full((90, 70, 3), 123, np.uint8)
    out = apc.resize_bicubic_exact(img, 41, 33)
    np.testing.assert_allclose(out, 123.0, atol=1e-9)


def test_linear_ramp_interior_exact():
    """A symmetric normalised filter reproduces a linear function at the output centre.
    Input value 2x + 10 at column x; 2x downsample: output o has centre at input index 2o + 0.5,
    so the value is 4o + 11 wherever no tap is dropped at the border."""
    W = 64
    img = np.zeros((8, W, 3), np.uint8)
    img[:, :, :] = (2 * np.arange(W) + 10)[None, :, None]
    out = apc.resize_bicubic_exact(img, 8, W // 2)
    o = np.arange(W // 2)
    interior = slice(2, W // 2 - 2)
    np.testing.assert_allclose(out[0, interior, 0], (4 * o + 11)[interior], atol=1e-9)


def test_2x_weights_by_hand():
    """Output pixel 5 of a 2x shrink of 20 pixels: centre 11.0, stretched support 4, taps at
    input centres 7.5 ... 14.5, weight Keys((x_i - 11) / 2) normalised."""
    Wm = apc.resize_weights(20, 10)
    xs = np.arange(20) + 0.5
    w = np.array([_keys((x - 11.0) / 2.0) for x in xs])
    w[np.abs((xs - 11.0) / 2.0) >= 2.0] = 0.0
    np.testing.assert_allclose(Wm[5], w / w.sum(), atol=1e-15)
    assert np.count_nonzero(Wm[5]) == 8


def test_border_taps_dropped_and_renormalised():
    Wm = apc.resize_weights(20, 10)
    np.testing.assert_allclose(Wm.sum(axis=1), 1.0, atol=1e-14)
    assert np.all(Wm[0, 6:] == 0)          # left border: only taps inside the image remain


def test_upsample_uses_unstretched_kernel():
    Wm = apc.resize_weights(10, 20)
    # output 9: centre (9.5) * 0.5 = 4.75; taps with |x_i - 4.75| < 2 -> input centres 3.5..6.5
    xs = np.arange(10) + 0.5
    w = np.array([_keys(x - 4.75) for x in xs])
    np.testing.assert_allclose(Wm[9], w / w.sum(), atol=1e-15)


def test_against_pil_bicubic_informational():
    """PIL's BICUBIC (named by the paper) rounds and clips between its two passes and uses
    fixed-point weights; the filter is otherwise the same.  On a smooth image the two agree
    to one level; on noise, PIL's clipped overshoot moves a few pixels further."""
    PIL = pytest.importorskip("PIL.Image")
    from paper_2608_27206_amd import workloads as wl
    smooth = wl.make_image(1, 448, 448, textured_frac=0.0)
    for (oh, ow) in [(224, 224), (300, 300)]:
        ours = apc.resize_bicubic(smooth, oh, ow).astype(int)
        ref = np.asarray(PIL.fromarray(smooth).resize((ow, oh), PIL.Resampling.BICUBIC)).astype(int)
        assert np.max(np.abs(ours - ref)) <= 1
    rs = np.random.default_rng(3)
    img = rs.integers(0, 256, size=(96, 128, 3), dtype=np.uint8)
    for (oh, ow) in [(48, 64), (67, 91), (96, 128)]:
        ours = apc.resize_bicubic(img, oh, ow).astype(int)
        ref = np.asarray(PIL.fromarray(img).resize((ow, oh), PIL.Resampling.BICUBIC)).astype(int)
        assert np.mean(np.abs(ours - ref) <= 1) > 0.99
