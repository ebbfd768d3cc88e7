"""Oracle for the Dynamic Dual-Attention Extractor (Section 3.3, "Extract").

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the benchmark's
CPU-baseline leg, never by the product path.

Steps, in the paper's order:
  S_llm, S_vis  attention read-outs, each min-max normalised to [0, 1]
  sigma         standard deviation of each normalised map (confidence proxy)
  weights       (alpha_w, beta_w) = softmax([sigma_llm, sigma_vis] / tau)   (fusion equation)
                or fixed weights (the Fixed Fusion / Only-ViT / Only-LLM variants of the
                fusion ablation)
  S_final       alpha_w * S_llm + beta_w * S_vis
  top-K         rank by S_final, keep the K best                            (end of Section 3.3)
  prune         the kept tokens form the shortened LLM context (Figure 4 caption)

Readings where the paper is silent (listed in the design notes):
  * S_vis per LLM token: the final-block mass summed over heads, then over each 2x2
    merge group (4 consecutive tokens in window-major order), then taken to LLM
    raster order through ``vis_perm`` (vis_perm[i] = merged ViT index of LLM token i).
  * S_llm: the mass summed over query heads.
  * min-max of a constant map is the zero map; sigma is the population std.
  * K = ceil(ratio * N) (with a 1e-9 guard), ties broken toward the lower index, and the
    kept indices are returned in ascending order (original token order).
"""
from __future__ import annotations

import math
from typing import Optional

import numpy as np

TAU = 0.5   # Section 4.1, Implementation Details


def keep_count(ratio: float, n: int) -> int:
    """K = ceil(ratio * n) clamped to [0, n]; the 1e-9 guard absorbs float products such as
    0.1 * 30 = 3.0000000000000004."""
    k = int(math.ceil(ratio * n - 1e-9))
    return max(0, min(n, k))


def keep_from_density(rho: float, n: int, ratio_lo: float = 0.05, ratio_hi: float = 0.25) -> int:
    """Per-image K in a batch whose keep ratios APC's density sets (reading: linear map of rho
    onto [ratio_lo, ratio_hi])."""
    r = min(max(ratio_lo + (ratio_hi - ratio_lo) * rho, ratio_lo), ratio_hi)
    return keep_count(r, n)


def minmax(x: np.ndarray) -> np.ndarray:
    lo, hi = float(x.min()), float(x.max())
    if hi == lo:
        return np.zeros_like(x, dtype=np.float64)
    return (x - lo) / (hi - lo)


def vis_token_map(vis_mass: np.ndarray, merge: int, vis_perm: Optional[np.ndarray]) -> np.ndarray:
    """Head-summed vision mass per LLM visual token (before normalisation)."""
    v = np.asarray(vis_mass, dtype=np.float64).sum(axis=0)
    v = v.reshape(-1, merge).sum(axis=1)
    if vis_perm is not None:
        v = v[np.asarray(vis_perm, dtype=np.int64)]
    return v


def llm_token_map(llm_mass: np.ndarray) -> np.ndarray:
    return np.asarray(llm_mass, dtype=np.float64).sum(axis=0)


def fuse(vis_mass, llm_mass, merge: int = 4, vis_perm=None, mode: int = 0, tau: float = TAU,
         w_llm_fixed: float = 0.5):
    """S_final and (sigma_llm, sigma_vis, w_llm, w_vis).  mode 0: confidence softmax; mode 1:
    fixed weights (w_llm_fixed, 1 - w_llm_fixed)."""
    S_vis = minmax(vis_token_map(vis_mass, merge, vis_perm))
    S_llm = minmax(llm_token_map(llm_mass))
    sig_l = float(S_llm.std())           # population std (ddof = 0)
    sig_v = float(S_vis.std())
    if mode == 0:
        z = np.array([sig_l, sig_v]) / tau
        e = np.exp(z - z.max())
        w_l, w_v = e / e.sum()
    else:
        w_l, w_v = w_llm_fixed, 1.0 - w_llm_fixed
    S = w_l * S_llm + w_v * S_vis
    return S, (sig_l, sig_v, float(w_l), float(w_v))


def topk_indices(S: np.ndarray, K: int) -> np.ndarray:
    """The K highest scores, ties broken toward the lower index, returned ascending."""
    S = np.asarray(S)
    order = np.lexsort((np.arange(S.shape[0]), -S))
    return np.sort(order[:K]).astype(np.int64)


def gather(hidden: np.ndarray, idx: np.ndarray) -> np.ndarray:
    return hidden[np.asarray(idx, dtype=np.int64)]


def select(vis_mass, llm_mass, K: int, merge: int = 4, vis_perm=None, mode: int = 0,
           tau: float = TAU, w_llm_fixed: float = 0.5):
    S, stats = fuse(vis_mass, llm_mass, merge, vis_perm, mode, tau, w_llm_fixed)
    return topk_indices(S, K), S, stats
