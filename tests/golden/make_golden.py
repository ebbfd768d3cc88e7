"""Writes tests/golden/apc_fullsize.json: APC scores of the seeded full-size images,
computed by the float64 oracle alone (Eq. 1 as the literal pairwise double sum takes
minutes at 4K, too slow to redo inside a test).

Run from the repository root:  python tests/golden/make_golden.py
"""
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import apc  # noqa: E402
from paper_2608_27206_amd import workloads as wl  # noqa: E402


def entry(img):
    t0 = time.time()
    r = apc.apc_density(img)
    return {
        "shape": list(img.shape),
        "sha256": hashlib.sha256(img.tobytes()).hexdigest(),
        "phi": r["phi"], "rho_g": r["rho_g"], "rho_d": r["rho_d"], "rho": r["rho"],
        "d_top": r["d_top"], "oracle_seconds": round(time.time() - t0, 1),
    }


def main():
    out = {"_about": "APC density of the seeded workload images, float64 oracle (tests/golden/make_golden.py)"}
    out["frame4k"] = entry(wl.make_workload(3).images[0])
    w4 = wl.make_workload(4)
    out["varlen8"] = [entry(im) for im in w4.images]
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "apc_fullsize.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main()
