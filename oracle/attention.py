"""Oracle for softmax attention with log-sum-exp and per-key attention mass.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the benchmark's
CPU-baseline leg, never by the product path.

This is textbook scaled dot-product attention, evaluated head by head in float64:
    S = Q K^T * scale,  masked entries -inf,  P = exp(S - max) / sum,  O = P V,
    LSE = max + ln(sum).
The attention mass is what Section 3.3 reads out of the two attention passes: for
each key, the sum of the normalised probabilities P[q, k] over a set of query rows.
  * S_vis comes from the final vision block's self-attention (Appendix, "Detailed
    Implementation Specifics"); the mass sums over every query of the image's
    full-attention segment.
  * S_llm comes from the cross-modal attention of an early LLM layer; the graded
    path sums over the text query rows (the "Text" source of the attention-token
    study); other sources are other query ranges of the same sum.

Layouts follow the device API: tokens are rows, [N, heads, d]; segments
(windows, images, packed sequences) are given by cumulative offsets and never
attend to each other.  Grouped-query attention maps query head h to KV head
h // (Hq / Hkv).  The sequence of a prefill is [visual tokens][text tokens],
causal (key index <= query index).
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np


def _softmax_rows(S: np.ndarray):
    """Row softmax of S (rows may contain -inf, never a whole row)."""
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    l = E.sum(axis=1, keepdims=True)
    return E / l, (m + np.log(l))[:, 0]


def attention_segment(q: np.ndarray, k: np.ndarray, v: np.ndarray, causal: bool, scale: float,
                      rows: Optional[Sequence[int]] = None,
                      mass_rows: Optional[Sequence[int]] = None, chunk: int = 512):
    """Attention inside one segment.

    q [n, Hq, d], k/v [n, Hkv, d] float64.  Returns (O [len(rows), Hq, d],
    LSE [Hq, len(rows)], mass [Hq, n]) where ``rows`` selects the query rows
    evaluated (default: all) and mass sums P over ``mass_rows`` (default: none ->
    zeros)."""
    n, hq, d = q.shape
    hkv = k.shape[1]
    group = hq // hkv
    rows = np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)
    mrows = np.zeros(0, dtype=np.int64) if mass_rows is None else np.asarray(mass_rows, np.int64)
    O = np.zeros((rows.shape[0], hq, v.shape[2]), dtype=np.float64)
    LSE = np.zeros((hq, rows.shape[0]), dtype=np.float64)
    mass = np.zeros((hq, n), dtype=np.float64)
    keys = np.arange(n)
    for h in range(hq):
        kv = h // group
        K = k[:, kv, :]
        V = v[:, kv, :]
        # outputs for the requested rows
        for a in range(0, rows.shape[0], chunk):
            r = rows[a:a + chunk]
            S = (q[r, h, :] @ K.T) * scale
            if causal:
                S = np.where(keys[None, :] > r[:, None], -np.inf, S)
            P, lse = _softmax_rows(S)
            O[a:a + chunk, h, :] = P @ V
            LSE[h, a:a + chunk] = lse
        # mass: column sums of the normalised probabilities over the querying rows
        for a in range(0, mrows.shape[0], chunk):
            r = mrows[a:a + chunk]
            S = (q[r, h, :] @ K.T) * scale
            if causal:
                S = np.where(keys[None, :] > r[:, None], -np.inf, S)
            P, _ = _softmax_rows(S)
            mass[h] += P.sum(axis=0)
    return O, LSE, mass


def vit_attention(q, k, v, cu_seqlens, scale: float, with_mass: bool = True):
    """Non-causal attention inside each segment of ``cu_seqlens`` (windows or whole images).

    Returns O [N, H, d], LSE [H, N] and mass [H, N], where mass[h, k] sums P over every
    query row of the segment that holds key k."""
    N, H, d = q.shape
    O = np.zeros((N, H, v.shape[2]))
    LSE = np.zeros((H, N))
    mass = np.zeros((H, N))
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    for s in range(cu.shape[0] - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        if b <= a:
            continue
        o, lse, m = attention_segment(q[a:b], k[a:b], v[a:b], False, scale,
                                      mass_rows=(np.arange(b - a) if with_mass else None))
        O[a:b] = o
        LSE[:, a:b] = lse
        mass[:, a:b] = m
    return O, LSE, mass


def prefill_attention(q, k, v, cu_seqlens, vis_len, mq_start, mq_len, scale: float, vis_start=None):
    """Causal grouped-query attention over packed sequences, with visual-key mass.

    Sequence b spans rows [cu[b], cu[b+1]); its tokens [vis_start[b], vis_start[b] + vis_len[b])
    are visual (vis_start None: the first vis_len[b]).  The mass of visual key j of sequence b
    sums P over the query rows [mq_start[b], mq_start[b]+mq_len[b]) of that sequence (positions
    relative to the sequence start).

    Returns O [Ntot, Hq, d], LSE [Hq, Ntot], mass [Hq, sum vis_len] (sequences concatenated)."""
    Ntot, hq, d = q.shape
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    O = np.zeros((Ntot, hq, v.shape[2]))
    LSE = np.zeros((hq, Ntot))
    masses = []
    for s in range(cu.shape[0] - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        st, ln = int(mq_start[s]), int(mq_len[s])
        o, lse, m = attention_segment(q[a:b], k[a:b], v[a:b], True, scale,
                                      mass_rows=np.arange(st, st + ln))
        O[a:b] = o
        LSE[:, a:b] = lse
        vs = 0 if vis_start is None else int(vis_start[s])
        masses.append(m[:, vs: vs + int(vis_len[s])])
    mass = np.concatenate(masses, axis=1) if masses else np.zeros((hq, 0))
    return O, LSE, mass


def attention_rows(q, k, v, seg_start: int, seg_len: int, rows, causal: bool, scale: float):
    """O and LSE for selected query rows (positions relative to the segment) of one segment;
    for checking a few rows of a large problem one by one."""
    a, b = seg_start, seg_start + seg_len
    o, lse, _ = attention_segment(q[a:b], k[a:b], v[a:b], causal, scale, rows=rows)
    return o, lse
