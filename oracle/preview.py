"""Oracle for the shallow feature preview of APC (Section 3.2, "Shallow Feature Preview": the
vision encoder's initial block, K = 1, run at the original resolution; the appendix's
implementation details fix K = 1).

TEST INFRASTRUCTURE ONLY: imported by tests and the benchmark's CPU-baseline leg, never by the
product path.

The paper runs the first block of Qwen2.5-VL's vision encoder with its trained weights, which are
not available.  This is a block of the same structure with seeded weights, so its values (and the
rho they lead to) are unpinned with respect to the paper:
  patch embedding   each patch's 3*P*P pixels, mapped to x/127.5 - 1, times W_pe -> D values
  attention         h1 = h0 + W_o A(RMSNorm_1(h0)) + b_o, where A is multi-head softmax attention
                    inside each window of 8 x 8 patches (heads of 80 values, scale 1/sqrt(80)),
                    q/k/v = W_{q,k,v} RMSNorm_1(h0) + b_{q,k,v}
  MLP               out = h1 + W_d (silu(W_g u + b_g) * (W_u u + b_u)) + b_d, u = RMSNorm_2(h1)
RMSNorm(x) = x / sqrt(mean(x^2) + 1e-6) * gamma.  Readings (listed in the design notes): the pixel
normalisation is the stand-in feature's x/127.5 - 1; rotary position encoding is left out.
Tokens are in the encoder's window-major order (rows of the patch matrix are given in that
order; the windows are consecutive row ranges).  Every step is float64.
"""
from __future__ import annotations

import math

import numpy as np

from . import attention as oatt

EPS = 1e-6
HEAD_DIM = 80


def patch_rows(img: np.ndarray, patch: int, order: np.ndarray) -> np.ndarray:
    """Patch pixels mapped to x/127.5 - 1, one row per token: token t is raster patch order[t];
    within a patch the components run over patch row, pixel column, channel."""
    H, W, C = img.shape
    gh, gw = H // patch, W // patch
    x = img[: gh * patch, : gw * patch, :].astype(np.float64) / 127.5 - 1.0
    x = x.reshape(gh, patch, gw, patch, C).transpose(0, 2, 1, 3, 4).reshape(gh * gw, patch * patch * C)
    return x[np.asarray(order, dtype=np.int64)]


def rmsnorm(x: np.ndarray, gamma: np.ndarray) -> np.ndarray:
    return x / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + EPS) * gamma[None, :]


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def linear(x: np.ndarray, w: np.ndarray, b=None) -> np.ndarray:
    """x [M, K] times w [N, K] transposed, plus b [N]."""
    y = x @ w.T
    return y if b is None else y + b[None, :]


def preview_block(X: np.ndarray, w: dict, cu_windows: np.ndarray) -> np.ndarray:
    """The block on patch rows X [N, 3*P*P] (float64); w holds float64 weights
    pe [D, 3PP], g1, wq, bq, wk, bk, wv, bv, wo, bo, g2, wg, bg, wu, bu, wd, bd.
    Returns the token embeddings [N, D]."""
    N = X.shape[0]
    D = w["pe"].shape[0]
    H = D // HEAD_DIM
    h0 = linear(X, w["pe"])
    u = rmsnorm(h0, w["g1"])
    q = linear(u, w["wq"], w["bq"]).reshape(N, H, HEAD_DIM)
    k = linear(u, w["wk"], w["bk"]).reshape(N, H, HEAD_DIM)
    v = linear(u, w["wv"], w["bv"]).reshape(N, H, HEAD_DIM)
    o, _, _ = oatt.vit_attention(q, k, v, cu_windows, 1.0 / math.sqrt(HEAD_DIM), with_mass=False)
    h1 = h0 + linear(o.reshape(N, D), w["wo"], w["bo"])
    u2 = rmsnorm(h1, w["g2"])
    m = silu(linear(u2, w["wg"], w["bg"])) * linear(u2, w["wu"], w["bu"])
    return h1 + linear(m, w["wd"], w["bd"])
