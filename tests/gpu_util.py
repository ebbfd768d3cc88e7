"""Helpers for the GPU parity tests: moving seeded inputs to the device and back."""
import sys

import numpy as np

from paper_2608_27206_amd import workloads as wl


def torch():
    import torch as _t
    return _t


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def dev_bf16(bits: np.ndarray):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(bits).view(np.int16).copy()).view(t.bfloat16).cuda()


def dev_i32(a):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).cuda()


def dev_f32(a):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.float32))).cuda()


def dev_u8(a):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).cuda()


def host_bf16_to_f64(x) -> np.ndarray:
    t = torch()
    return wl.bf16_bits_to_f64(x.detach().view(t.int16).cpu().numpy().view(np.uint16))


def host(x) -> np.ndarray:
    return x.detach().cpu().numpy()


def mass_ok(gpu, ref, nq, rel=1e-3):
    """Per-key mass parity: |m_gpu - m_ref| <= rel * m_ref + 1e-12 * |Q_set|."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(gpu - ref) - (rel * np.abs(ref) + 1e-12 * nq)
    return float(err.max()), float((np.abs(gpu - ref) / np.maximum(np.abs(ref), 1e-30)).max())


def kept_sets_agree(idx_gpu, idx_ref, S_ref, band=1e-3):
    """Kept sets may differ only by swapping tokens whose oracle scores lie within `band`."""
    a = set(int(i) for i in idx_gpu)
    b = set(int(i) for i in idx_ref)
    only_gpu = sorted(a - b)
    only_ref = sorted(b - a)
    if len(only_gpu) != len(only_ref):
        return False, f"sizes differ {len(a)} vs {len(b)}"
    if not only_gpu:
        return True, "identical"
    lo = min(S_ref[i] for i in only_gpu)
    hi = max(S_ref[i] for i in only_ref)
    return (hi - lo) <= band, f"{len(only_gpu)} swaps, spread {hi - lo:.3g}"


def oracle_mass_parallel(q, k, causal, scale, mass_rows, workers=8):
    """The oracle's per-key mass of one head (q, k float64 [n, d]) over `mass_rows`, the rows split
    into `workers` groups run on threads (numpy releases the GIL inside its loops) and the
    groups' column sums added.  Test-side parallelism only: every group is a plain oracle call."""
    from concurrent.futures import ThreadPoolExecutor

    from oracle import attention as oatt
    rows = np.asarray(mass_rows, dtype=np.int64)
    parts = [r for r in np.array_split(rows, workers) if r.size]

    def one(r):
        _, _, m = oatt.attention_segment(q[:, None, :], k[:, None, :], k[:, None, :], causal, scale,
                                         rows=np.arange(0), mass_rows=r)
        return m[0]
    with ThreadPoolExecutor(max_workers=workers) as ex:
        return np.sum(list(ex.map(one, parts)), axis=0)


def load_e2e_golden(config_id, workload):
    """Oracle-only end-to-end selection (tests/golden/make_e2e_golden.py) for one workload:
    (nv, keep, S_final, kept idx), after checking the workload's inputs are the ones it used."""
    import hashlib
    import os
    z = np.load(os.path.join(os.path.dirname(__file__), "golden", "e2e_select.npz"))
    c = f"c{config_id}_"
    h = hashlib.sha256()
    for a in (workload.vit.q, workload.vit.k, workload.prefill.q, workload.prefill.k):
        h.update(np.ascontiguousarray(a).tobytes())
    assert str(z[c + "sha"]) == h.hexdigest(), "workload generator changed since the golden file"
    return z[c + "nv"], z[c + "keep"], z[c + "S"].astype(np.float64), z[c + "idx"].astype(np.int64)


def rho4(rho) -> np.ndarray:
    """The density call's (rho_g, rho_d, rho) with phi = 1 - rho_g (Eq. 2) appended, for
    comparison with the oracle's (rho_g, rho_d, rho, phi)."""
    r = np.asarray(host(rho) if not isinstance(rho, np.ndarray) else rho, dtype=np.float64)
    return np.array([r[0], r[1], r[2], 1.0 - r[0]])
