"""Pins of the preview-block oracle (oracle/preview.py) against closed forms, the other oracle
modules and structural invariants of the block."""
import math

import numpy as np

from oracle import apc, attention as oatt, preview as opv
from paper_2608_27206_amd import workloads as wl


def _weights(seed=1, dim=160, ffn=96, patch=4):
    w = wl.preview_weights(seed, dim, ffn, patch)
    return {k: (wl.bf16_bits_to_f64(v) if v.dtype == np.uint16 else v.astype(np.float64)) for k, v in w.items()}


def test_patch_rows_match_the_image_feature_in_raster_order():
    img = np.random.default_rng(0).integers(0, 256, size=(56, 84, 3), dtype=np.uint8)
    order = np.arange((56 // 14) * (84 // 14))
    np.testing.assert_array_equal(opv.patch_rows(img, 14, order), apc.patch_features(img, 14))
    lay = wl.vit_layout(4, 6)
    np.testing.assert_array_equal(opv.patch_rows(img, 14, lay.order), apc.patch_features(img, 14)[lay.order])


def test_rmsnorm_and_silu_closed_forms():
    g = np.array([2.0, -1.0, 0.5])
    x = np.full((1, 3), 3.0)
    np.testing.assert_allclose(opv.rmsnorm(x, g), 3.0 / math.sqrt(9.0 + 1e-6) * g[None, :], rtol=1e-15)
    y = np.array([[3.0, 4.0, 0.0]])
    np.testing.assert_allclose(opv.rmsnorm(y, np.ones(3)), y / math.sqrt(25.0 / 3 + 1e-6), rtol=1e-15)
    assert opv.silu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(opv.silu(np.array([1.0, -2.0])), [1 / (1 + math.exp(-1)), -2 / (1 + math.exp(2))],
                               rtol=1e-15)


def test_block_without_residual_branches_is_the_patch_embedding():
    w = _weights()
    for k in ("wo", "wd"):
        w[k] = np.zeros_like(w[k])
    for k in ("bo", "bd"):
        w[k] = np.zeros_like(w[k])
    X = np.random.default_rng(2).uniform(-1, 1, size=(40, 48))
    out = opv.preview_block(X, w, np.array([0, 16, 32, 40]))
    np.testing.assert_allclose(out, X @ w["pe"].T, rtol=1e-13, atol=1e-13)


def test_single_token_windows_attend_to_themselves():
    """With one token per window the attention output is v itself, so the block is a closed
    chain of linear maps and norms."""
    w = _weights(3)
    X = np.random.default_rng(4).uniform(-1, 1, size=(12, 48))
    out = opv.preview_block(X, w, np.arange(13))
    h0 = X @ w["pe"].T
    v = opv.rmsnorm(h0, w["g1"]) @ w["wv"].T + w["bv"]
    h1 = h0 + v @ w["wo"].T + w["bo"]
    u = opv.rmsnorm(h1, w["g2"])
    ref = h1 + (opv.silu(u @ w["wg"].T + w["bg"]) * (u @ w["wu"].T + w["bu"])) @ w["wd"].T + w["bd"]
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)


def test_windows_do_not_see_each_other():
    w = _weights(5)
    rs = np.random.default_rng(6)
    X = rs.uniform(-1, 1, size=(48, 48))
    cu = np.array([0, 16, 32, 48])
    a = opv.preview_block(X, w, cu)
    X2 = X.copy()
    X2[16:32] = rs.uniform(-1, 1, size=(16, 48))
    b = opv.preview_block(X2, w, cu)
    np.testing.assert_array_equal(a[:16], b[:16])
    np.testing.assert_array_equal(a[32:], b[32:])
    assert np.abs(a[16:32] - b[16:32]).max() > 1e-3


def test_attention_step_is_the_attention_oracle():
    """The block's attention is the (separately pinned) window attention oracle on q, k, v."""
    w = _weights(7)
    X = np.random.default_rng(8).uniform(-1, 1, size=(20, 48))
    cu = np.array([0, 8, 20])
    N, D = 20, 160
    u = opv.rmsnorm(X @ w["pe"].T, w["g1"])
    q = (u @ w["wq"].T + w["bq"]).reshape(N, 2, 80)
    k = (u @ w["wk"].T + w["bk"]).reshape(N, 2, 80)
    v = (u @ w["wv"].T + w["bv"]).reshape(N, 2, 80)
    o = np.zeros((N, 2, 80))
    for a, b in ((0, 8), (8, 20)):
        for h in range(2):
            S = q[a:b, h] @ k[a:b, h].T / math.sqrt(80)
            P = np.exp(S - S.max(axis=1, keepdims=True))
            o[a:b, h] = (P / P.sum(axis=1, keepdims=True)) @ v[a:b, h]
    o2, _, _ = oatt.vit_attention(q, k, v, cu, 1 / math.sqrt(80), with_mass=False)
    np.testing.assert_allclose(o2, o, rtol=1e-12, atol=1e-13)
