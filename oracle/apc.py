"""Oracle for the Adaptive Pixel Compressor (Section 3.2, "Condense").

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the benchmark's
CPU-baseline leg, never by the product path.

Steps, in the paper's order:
  feature preview  T_i, l2-normalised per patch             (Section 3.2, "Shallow Feature Preview")
  global density   phi = mean over all N^2 pairs of cos(T_i, T_j)   (Eq. 1); rho_g = 1 - phi (Eq. 2)
  background       c = mean_i T_i, c_hat = c / ||c||          (Section 3.2, "Local Detail Contrast")
  detail distance  d_i = ||T_i - c_hat||
  tail mean        mean of the top 10% of d_i; rho_d = min(d_top / gamma, 1)
  retention        rho = alpha * rho_g + (1 - alpha) * rho_d   ("Adaptive Condensation")
  resize           width and height each scaled by sqrt(r), r = rho under the budget, bicubic
                   (Appendix, "Detailed Implementation Specifics")

Readings where the paper is silent (listed in the design notes):
  * The preview network's weights are not available, so the per-patch feature is
    the patch's pixels mapped to x/127.5 - 1 (a 3*P*P vector), one of the
    pixel-statistic previews of the preview ablation.  Values of rho therefore
    differ from the paper's: parity with the paper's own rho is unpinned.
  * "top 10%" keeps ceil(0.10 * N) distances, at least one.
  * When ||c|| = 0 the baseline direction is the zero vector, so every d_i = ||T_i||.
    A norm at or below C_ZERO = 1e-5 (phi <= 1e-10) counts as zero: an exactly cancelling
    mean leaves only rounding noise, whose direction is meaningless.
  * The hard budget is a clamp of the area ratio r between a floor and a cap, and
    output sides are snapped to a multiple of ``snap``.
  * Bicubic: Keys' cubic convolution with a = -0.5, filter stretched by the
    shrink factor (antialiasing), pixel-centre alignment, taps outside the image
    dropped and the remaining weights renormalised, one rounding (half up) at
    the end.
"""
from __future__ import annotations

import math

import numpy as np

# Hyperparameters from Section 4.1 (Implementation Details) and the tail-percentile study.
ALPHA = 0.6
GAMMA = 1.5
TAIL_FRAC = 0.10
C_ZERO = 1e-5


def count_for_fraction(frac: float, n: int, at_least_one: bool = False) -> int:
    """ceil(frac * n) with a 1e-9 guard against float products such as 0.1*30 = 3.0000000000000004."""
    k = int(math.ceil(frac * n - 1e-9))
    k = max(0, min(n, k))
    if at_least_one and n > 0:
        k = max(1, k)
    return k


def patch_features(img: np.ndarray, patch: int = 14) -> np.ndarray:
    """Per-patch feature vectors, patches in raster order (row-major over the patch grid).

    Each patch's pixels (patch x patch x 3) are mapped to x/127.5 - 1 and flattened."""
    H, W, C = img.shape
    gh, gw = H // patch, W // patch
    x = img[: gh * patch, : gw * patch, :].astype(np.float64) / 127.5 - 1.0
    x = x.reshape(gh, patch, gw, patch, C).transpose(0, 2, 1, 3, 4)
    return x.reshape(gh * gw, patch * patch * C)


def l2_normalise(f: np.ndarray) -> np.ndarray:
    """T_i = f_i / ||f_i||  (Section 3.2: preview embeddings are l2-normalised)."""
    n = np.linalg.norm(f, axis=1, keepdims=True)
    return f / n


def global_density(T: np.ndarray, chunk: int = 1024) -> float:
    """Eq. 1: phi = (1/N^2) sum_i sum_j T_i.T_j / (||T_i|| ||T_j||), as a double sum over
    all ordered pairs (rows taken in chunks so the N x N matrix is never held)."""
    N = T.shape[0]
    norms = np.linalg.norm(T, axis=1)
    total = 0.0
    for a in range(0, N, chunk):
        b = min(N, a + chunk)
        cos = (T[a:b] @ T.T) / (norms[a:b, None] * norms[None, :])
        total += float(cos.sum())
    return total / (N * N)


def background_direction(T: np.ndarray) -> np.ndarray:
    """c = (1/N) sum_i T_i, c_hat = c / ||c|| (zero vector when ||c|| <= C_ZERO)."""
    c = T.mean(axis=0)
    nc = float(np.linalg.norm(c))
    if nc <= C_ZERO:
        return np.zeros_like(c)
    return c / nc


def detail_distances(T: np.ndarray, c_hat: np.ndarray) -> np.ndarray:
    """d_i = ||T_i - c_hat||_2."""
    return np.linalg.norm(T - c_hat[None, :], axis=1)


def tail_mean(d: np.ndarray, tail_frac: float = TAIL_FRAC) -> float:
    """Mean of the ceil(tail_frac * N) largest distances (at least one)."""
    n_tail = count_for_fraction(tail_frac, d.shape[0], at_least_one=True)
    top = np.sort(d)[::-1][:n_tail]
    return float(top.mean())


def density_from_features(T: np.ndarray, tail_frac: float = TAIL_FRAC, alpha: float = ALPHA,
                          gamma: float = GAMMA) -> dict:
    """The APC scores for l2-normalised preview embeddings T [N, D]."""
    phi = global_density(T)
    rho_g = 1.0 - phi                                   # Eq. 2
    c_hat = background_direction(T)
    d = detail_distances(T, c_hat)
    d_top = tail_mean(d, tail_frac)
    rho_d = min(d_top / gamma, 1.0)
    rho = alpha * rho_g + (1.0 - alpha) * rho_d
    return {"phi": phi, "rho_g": rho_g, "rho_d": rho_d, "rho": rho, "d": d,
            "d_top": d_top, "c_hat": c_hat}


def normalise_embeddings(x: np.ndarray, eps: float = 1e-12) -> np.ndarray:
    """T_i = x_i / max(||x_i||, eps) for caller-supplied preview embeddings (Section 3.2: the
    embeddings are l2-normalised).  Reading: a zero embedding is a zero direction (T_i = 0)."""
    x = np.asarray(x, dtype=np.float64)
    n = np.linalg.norm(x, axis=1, keepdims=True)
    return x / np.maximum(n, eps)


def global_density_dot(T: np.ndarray, chunk: int = 1024) -> float:
    """Eq. 1 for normalised rows written as dot products, (1/N^2) sum_i sum_j T_i . T_j over all
    ordered pairs; equal to global_density for unit rows and defined when a row is zero."""
    N = T.shape[0]
    total = 0.0
    for a in range(0, N, chunk):
        b = min(N, a + chunk)
        total += float((T[a:b] @ T.T).sum())
    return total / (N * N)


def embedding_density(x: np.ndarray, tail_frac: float = TAIL_FRAC, alpha: float = ALPHA,
                      gamma: float = GAMMA) -> dict:
    """The APC scores of caller-supplied preview embeddings x [N, D] (the paper's preview is the
    first vision-encoder block): the steps of density_from_features after normalisation."""
    T = normalise_embeddings(x)
    phi = global_density_dot(T)
    rho_g = 1.0 - phi                                   # Eq. 2
    c_hat = background_direction(T)
    d = detail_distances(T, c_hat)
    d_top = tail_mean(d, tail_frac)
    rho_d = min(d_top / gamma, 1.0)
    rho = alpha * rho_g + (1.0 - alpha) * rho_d
    return {"phi": phi, "rho_g": rho_g, "rho_d": rho_d, "rho": rho, "d": d,
            "d_top": d_top, "c_hat": c_hat}


# ---------------------------------------------------------------- pixel-statistic previews
# Pixel-statistic previews of the preview-signal study (Appendix, shallow feature preview
# ablation): RGB statistics, colour entropy, edge density and a Laplacian, named there as
# weight-free stand-ins for the first encoder block but not given as formulas.  Readings
# (listed in the design notes): each is a vector per patch, so that the cosine-based density
# steps apply unchanged (a scalar per patch would make every cosine +-1):
#   0 RGB statistics  mean and population std of each channel of x/255      (6 values)
#   1 colour entropy  -p_k ln p_k for the 64 colours of 4 levels per channel (64 values; their
#                     sum is the patch's colour entropy)
#   2 edge density    Sobel gradient magnitude of the grey image summed per orientation octant,
#                     divided by 255 * patch^2                             (8 values)
#   3 Laplacian       the 4-neighbour Laplacian of the grey image / 255     (patch^2 values)
# Grey = (299 R + 587 G + 114 B) / 1000; gradients and the Laplacian take neighbours across patch
# borders, with the image edge clamped.  The octant of a gradient (gx, gy) is decided exactly
# from integers: 0 for angles in [0, 45) degrees, 1 for [45, 90), ..., counter-clockwise with
# y pointing down the image rows; the zero gradient falls in octant 0 with magnitude 0.
PIXEL_FEATURE_DIMS = {0: lambda P: 6, 1: lambda P: 64, 2: lambda P: 8, 3: lambda P: P * P}


def _grey1000(img: np.ndarray) -> np.ndarray:
    """1000 x the grey value: the exact integer 299 R + 587 G + 114 B."""
    x = img.astype(np.int64)
    return 299 * x[..., 0] + 587 * x[..., 1] + 114 * x[..., 2]


def _octant(gx: np.ndarray, gy: np.ndarray) -> np.ndarray:
    """Octant index 0..7 of the angle atan2(gy, gx) in [0, 360) degrees, from exact comparisons."""
    ax, ay = np.abs(gx), np.abs(gy)
    oct_ = np.zeros(gx.shape, dtype=np.int64)
    up = gy >= 0
    # quadrant I (gx > 0, gy >= 0): 0 if ay < ax else 1; II (gx <= 0, gy > 0): 2 if ax <= ay else 3;
    # III (gx < 0, gy <= 0): 4 if ay < ax else 5; IV (gx >= 0, gy < 0): 6 if ax <= ay else 7
    q1 = (gx > 0) & up
    q2 = (gx <= 0) & (gy > 0)
    q3 = (gx < 0) & (gy <= 0)
    q4 = (gx >= 0) & (gy < 0)
    oct_[q1] = np.where(ay[q1] < ax[q1], 0, 1)
    oct_[q2] = np.where(ax[q2] <= ay[q2], 2, 3)
    oct_[q3] = np.where(ay[q3] < ax[q3], 4, 5)
    oct_[q4] = np.where(ax[q4] <= ay[q4], 6, 7)
    return oct_


def pixel_statistic_features(img: np.ndarray, patch: int, kind: int) -> np.ndarray:
    """Per-patch pixel-statistic feature vectors [N, dim], patches in raster order."""
    H, W, _ = img.shape
    gh, gw = H // patch, W // patch
    img = img[: gh * patch, : gw * patch]
    N = gh * gw

    def per_patch(a):   # [H, W, ...] -> [N, patch*patch, ...]
        a = a.reshape((gh, patch, gw, patch) + a.shape[2:])
        a = np.moveaxis(a, 2, 1)
        return a.reshape((N, patch * patch) + a.shape[4:])

    if kind == 0:
        x = per_patch(img.astype(np.float64) / 255.0)          # [N, P*P, 3]
        return np.concatenate([x.mean(axis=1), x.std(axis=1)], axis=1)
    if kind == 1:
        q = img.astype(np.int64) // 64                          # 4 levels per channel
        colour = per_patch(q[..., 0] * 16 + q[..., 1] * 4 + q[..., 2])
        feats = np.zeros((N, 64))
        for i in range(N):
            p = np.bincount(colour[i], minlength=64) / float(patch * patch)
            nz = p > 0
            feats[i, nz] = -p[nz] * np.log(p[nz])
        return feats
    # gradients and the Laplacian on 1000 x grey: exact integers, so the octants are exact
    pi = np.pad(_grey1000(img), 1, mode="edge")
    if kind == 3:
        lap = 4 * pi[1:-1, 1:-1] - pi[:-2, 1:-1] - pi[2:, 1:-1] - pi[1:-1, :-2] - pi[1:-1, 2:]
        return per_patch(lap / 255000.0)
    if kind == 2:
        gx = (pi[:-2, 2:] + 2 * pi[1:-1, 2:] + pi[2:, 2:]) - (pi[:-2, :-2] + 2 * pi[1:-1, :-2] + pi[2:, :-2])
        gy = (pi[2:, :-2] + 2 * pi[2:, 1:-1] + pi[2:, 2:]) - (pi[:-2, :-2] + 2 * pi[:-2, 1:-1] + pi[:-2, 2:])
        mag = np.sqrt(gx.astype(np.float64) ** 2 + gy.astype(np.float64) ** 2) / 1000.0
        o = per_patch(_octant(gx, gy))
        m = per_patch(mag)
        feats = np.zeros((N, 8))
        for k in range(8):
            feats[:, k] = np.where(o == k, m, 0.0).sum(axis=1)
        return feats / (255.0 * patch * patch)
    raise ValueError(f"unknown pixel statistic {kind}")


def pixel_density(img: np.ndarray, patch: int, kind: int, tail_frac: float = TAIL_FRAC,
                  alpha: float = ALPHA, gamma: float = GAMMA) -> dict:
    """APC scores with a pixel-statistic preview: the density steps of embedding_density over
    pixel_statistic_features (a zero feature vector is a zero direction)."""
    return embedding_density(pixel_statistic_features(img, patch, kind), tail_frac, alpha, gamma)


def apc_density(img: np.ndarray, patch: int = 14, tail_frac: float = TAIL_FRAC,
                alpha: float = ALPHA, gamma: float = GAMMA) -> dict:
    """APC density of a uint8 HWC image, with the pixel stand-in feature."""
    T = l2_normalise(patch_features(img, patch))
    return density_from_features(T, tail_frac, alpha, gamma)


# ---------------------------------------------------------------- resize
def target_size(rho: float, H: int, W: int, min_pixels: float, max_pixels: float,
                snap: int) -> tuple:
    """Output size after APC's resize: area ratio r = rho clamped to [r_floor, r_cap], with
    r_cap = min(1, max_pixels/(H W)) and r_floor = min(r_cap, min_pixels/(H W)); each side is
    scaled by sqrt(r), rounded half up to a multiple of ``snap`` and kept within
    [min(snap, X), floor(X/snap)*snap]."""
    area = float(H) * float(W)
    r_cap = min(1.0, max_pixels / area)
    r_floor = min(r_cap, min_pixels / area)
    r = min(max(float(rho), r_floor), r_cap)
    s = math.sqrt(r)

    def side(X):
        o = int(math.floor(X * s / snap + 0.5)) * snap
        o = min(o, (X // snap) * snap)
        return max(o, min(snap, X))
    return side(H), side(W)


def keys_cubic(x: np.ndarray, a: float = -0.5) -> np.ndarray:
    """Keys' cubic convolution kernel."""
    x = np.abs(np.asarray(x, dtype=np.float64))
    w = np.zeros_like(x)
    m1 = x <= 1.0
    m2 = (x > 1.0) & (x < 2.0)
    w[m1] = (a + 2.0) * x[m1] ** 3 - (a + 3.0) * x[m1] ** 2 + 1.0
    w[m2] = a * x[m2] ** 3 - 5.0 * a * x[m2] ** 2 + 8.0 * a * x[m2] - 4.0 * a
    return w


def resize_weights(n_in: int, n_out: int) -> np.ndarray:
    """Dense [n_out, n_in] matrix of 1-D bicubic weights (rows sum to 1).

    Output pixel o has centre (o + 0.5) * n_in / n_out in input coordinates; input pixel i
    has centre i + 0.5.  The kernel is stretched by f = max(1, n_in / n_out)."""
    scale = n_in / n_out
    f = max(1.0, scale)
    Wm = np.zeros((n_out, n_in), dtype=np.float64)
    centres_in = np.arange(n_in, dtype=np.float64) + 0.5
    for o in range(n_out):
        c = (o + 0.5) * scale
        dist = (centres_in - c) / f
        w = keys_cubic(dist)
        w[np.abs(dist) >= 2.0] = 0.0
        Wm[o] = w / w.sum()
    return Wm


def resize_bicubic_exact(img: np.ndarray, oH: int, oW: int) -> np.ndarray:
    """Separable resize in float64 with no intermediate rounding -> float64 [oH, oW, 3]."""
    Wy = resize_weights(img.shape[0], oH)
    Wx = resize_weights(img.shape[1], oW)
    x = img.astype(np.float64)
    out = np.empty((oH, oW, img.shape[2]), dtype=np.float64)
    for c in range(img.shape[2]):
        out[:, :, c] = Wy @ x[:, :, c] @ Wx.T
    return out


def round_u8(v: np.ndarray) -> np.ndarray:
    return np.clip(np.floor(v + 0.5), 0, 255).astype(np.uint8)


def resize_bicubic(img: np.ndarray, oH: int, oW: int) -> np.ndarray:
    return round_u8(resize_bicubic_exact(img, oH, oW))
