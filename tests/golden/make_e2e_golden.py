"""Writes tests/golden/e2e_select.npz: the end-to-end DDAE selection of the seeded 448 x 448,
1344 x 1344, 4K-frame and varlen workloads, computed by the float64 oracle alone.

Section 3.3 ("Extract") in the paper's order: S_vis is the attention mass every patch receives
in the image's full-attention block (all query rows, summed over the 16 heads, then over each
2 x 2 merge group, then taken to LLM order), S_llm the mass every visual key receives from the
text query rows of the causal prefill (summed over the 28 query heads); both are min-max
normalised, fused with softmax(sigma / tau) weights, and the top-K tokens are kept.  K is
ceil(0.10 N) for one image; in the varlen batch it follows each image's APC density (the keep
ratio 0.05 + 0.20 rho, with rho from tests/golden/apc_fullsize.json).  The attention over 42,196
patches takes minutes of float64 work, too slow for a test, hence this file.

Stored per workload c in {1, 2, 3, 4}:
  c{c}_nv     int32 [B]   visual tokens per image
  c{c}_keep   int32 [B]   K per image
  c{c}_S      float32 [sum nv]  S_final per token (images concatenated)
  c{c}_idx    int32 [sum K]     kept global token indices, ascending within each image
  c{c}_sha    str             sha256 of the workload's q/k bits (vision and prefill)

Run from the repository root:  python tests/golden/make_e2e_golden.py [--procs 8]
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time
from concurrent.futures import ProcessPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import attention as oatt  # noqa: E402
from oracle import ddae as oddae  # noqa: E402
from paper_2608_27206_amd import workloads as wl  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))


def workload_sha(w) -> str:
    h = hashlib.sha256()
    for a in (w.vit.q, w.vit.k, w.prefill.q, w.prefill.k):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def _one_head_mass(args):
    """Mass of every key of one segment for one head, summed over the given query rows."""
    q_bits, k_bits, mass_rows, causal, scale = args
    q = wl.bf16_bits_to_f64(q_bits)[:, None, :]
    k = wl.bf16_bits_to_f64(k_bits)[:, None, :]
    _, _, m = oatt.attention_segment(q, k, k, causal, scale, rows=np.arange(0), mass_rows=mass_rows)
    return m[0]


def _init_worker():
    for var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[var] = "1"
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:  # pragma: no cover
        pass


def oracle_selection(w, pool, keeps):
    vit, pre = w.vit, w.prefill
    H = vit.q.shape[1]
    hq, hkv = pre.q.shape[1], pre.k.shape[1]
    scores, kept = [], []
    nvs = [L.n_vis for L in w.layouts]
    for b, L in enumerate(w.layouts):
        a, e = int(vit.cu_full[b]), int(vit.cu_full[b + 1])
        n = e - a
        tasks = [(vit.q[a:e, h], vit.k[a:e, h], np.arange(n), False, 1 / math.sqrt(vit.q.shape[2]))
                 for h in range(H)]
        vis_mass = np.stack(list(pool.map(_one_head_mass, tasks)))           # [16, n]
        pa, pe = int(pre.cu_seqlens[b]), int(pre.cu_seqlens[b + 1])
        nv, nt = int(pre.vis_len[b]), int(pre.text_len[b])
        assert nv == L.n_vis
        tasks = [(pre.q[pa:pe, h], pre.k[pa:pe, h // (hq // hkv)], np.arange(nv, nv + nt), True,
                  1 / math.sqrt(pre.q.shape[2])) for h in range(hq)]
        llm_mass = np.stack(list(pool.map(_one_head_mass, tasks)))[:, :nv]    # [28, nv]
        S, _ = oddae.fuse(vis_mass, llm_mass, wl.MERGE * wl.MERGE, L.vis_perm, w.fusion_mode, w.tau)
        idx = oddae.topk_indices(S, keeps[b])
        scores.append(S)
        kept.append(idx + sum(nvs[:b]))
    return np.concatenate(scores), np.concatenate(kept)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--procs", type=int, default=8)
    a = ap.parse_args()
    apc_gold = json.load(open(os.path.join(HERE, "apc_fullsize.json")))
    out = {}
    with ProcessPoolExecutor(max_workers=a.procs, initializer=_init_worker) as pool:
        for c in (1, 2, 3, 4):
            t0 = time.time()
            w = wl.make_workload(c)
            nvs = [L.n_vis for L in w.layouts]
            if c == 4:
                keeps = [oddae.keep_from_density(g["rho"], nv) for g, nv in zip(apc_gold["varlen8"], nvs)]
            else:
                keeps = [oddae.keep_count(w.keep_ratio, nv) for nv in nvs]
            S, idx = oracle_selection(w, pool, keeps)
            out[f"c{c}_nv"] = np.asarray(nvs, np.int32)
            out[f"c{c}_keep"] = np.asarray(keeps, np.int32)
            out[f"c{c}_S"] = S.astype(np.float32)
            out[f"c{c}_idx"] = idx.astype(np.int32)
            out[f"c{c}_sha"] = np.asarray(workload_sha(w))
            print(f"config {c}: {len(nvs)} image(s), nv {nvs}, keep {keeps}, {time.time() - t0:.0f} s", flush=True)
    path = os.path.join(HERE, "e2e_select.npz")
    np.savez_compressed(path, **out)
    print("wrote", path)


if __name__ == "__main__":
    main()
