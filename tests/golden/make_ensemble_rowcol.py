"""Writes ensemble_rowcol_strassen2_128.json: App. B.1's synthetic ensemble
evaluated by the CPU oracle alone.

Every one of the 512 sign variants of two-level Strassen on 128 x 128
operands, one scale per row of A's and per column of B's block sums, E4M3,
products of the decoded codes summed exactly and rounded once to fp32; 200
pairs with entries uniform on [-1, 1] and 200 on [0, 1] (synthetic
.ensemble_pair), every pair evaluated under every variant.  Per variant:
the average relative Frobenius error over all pairs, over the even-numbered
and over the odd-numbered pairs; per distribution: spread (largest /
smallest average) and the correlation of the two halves across variants.

Run from the repository root:  python tests/golden/make_ensemble_rowcol.py
"""
import json
import os
import sys
from multiprocessing import Pool

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)
os.environ.setdefault("OMP_NUM_THREADS", "1")

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from oracle import scheme_ops as so  # noqa: E402
from oracle import schemes  # noqa: E402
import synthetic as sy  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "ensemble_rowcol_strassen2_128.json")


def variant_tables():
    s2 = so.power(schemes.strassen(), 2)
    return [oracle.flatten_f32(so.gauge(s2, np.diag(d), np.diag(e), np.diag(f)))
            for d, e, f in sy.sign_orbit(4, 4, 4)]


_TABS = None


def pair_errors(job):
    global _TABS
    if _TABS is None:
        _TABS = variant_tables()
    lo, p = job
    A, B = sy.ensemble_pair(lo, p)
    Cref = oracle.reference_f64(A, B)
    return [oracle.rel_fro(oracle.lowp_matmul(A, B, t, d, scale_mode=oracle.SCALE_ROWCOL), Cref)
            for t, d in _TABS]


def main():
    out = {"_about": __doc__.strip().splitlines()[0],
           "design": "every pair under every variant; pairs from synthetic.ensemble_pair",
           "pairs": sy.ENSEMBLE_PAIRS, "n": sy.ENSEMBLE_N, "seed": sy.ENSEMBLE_SEED}
    procs = int(os.environ.get("ENSEMBLE_PROCS", os.cpu_count() or 1))
    with Pool(procs) as pool:
        for lo, key in ((-1.0, "uniform_pm1"), (0.0, "uniform_01")):
            err = np.array(pool.map(pair_errors, [(lo, p) for p in range(sy.ENSEMBLE_PAIRS)])).T
            avg, ev, od = err.mean(1), err[:, 0::2].mean(1), err[:, 1::2].mean(1)
            out[key] = dict(spread=float(avg.max() / avg.min()),
                            split_half_corr=float(np.corrcoef(ev, od)[0, 1]),
                            avg=[float(v) for v in avg], even=[float(v) for v in ev],
                            odd=[float(v) for v in od])
            print(key, out[key]["spread"], out[key]["split_half_corr"], flush=True)
    json.dump(out, open(OUT, "w"))


if __name__ == "__main__":
    main()
