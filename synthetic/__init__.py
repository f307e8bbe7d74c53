"""Seeded synthetic inputs shared by the oracle-side tests and the GPU path.

This module holds no arithmetic of the method: it only draws operands and
gauge elements (the random inputs the method is evaluated on) and names the
workloads.  Both the oracle and the HIP path receive exactly these arrays.

Workloads stand in for the paper's model activations and weights, which are
not available: Gaussian, Student-t and outlier-channel activations and
Gaussian weights at LLM projection shapes, and the gauge orbits of the paper's
sign variants (Sec. 2.1) or of random invertible block-space transforms.
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass, field, replace

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    M: int
    K: int
    N: int
    scheme: str            # base scheme: strassen | laderman | classical
    levels: int            # recursion levels of the base scheme
    gauge_kind: str        # "gl" (random invertible, base grid) | "sign" (flattened grid)
    G: int                 # orbit size evaluated
    fmts: tuple = ("e4m3",)
    a_dist: str = "normal"  # normal | t3
    a_sigma: float = 1.0
    a_outliers: int = 0
    a_outlier_scale: float = 1.0
    b_sigma: float = 1.0
    sign_sampled: bool = False  # sample the sign orbit instead of enumerating it
    seed: int = 20260902
    notes: str = ""

    def grid(self):
        base = {"strassen": (2, 2, 2), "laderman": (3, 3, 3), "classical": (1, 1, 1)}[self.scheme]
        return tuple(b ** self.levels for b in base)


WORKLOADS = {
    # Strassen rank 7, one level, 256^2 Gaussian, 64 random GL(2) gauges.
    "strassen1_256_gl64": Workload(
        "strassen1_256_gl64", 256, 256, 256, "strassen", 1, "gl", 64),
    # Two-level Strassen (4x4x4, rank 49), full 512-element sign orbit,
    # 2048x4096 activations with 8 outlier channels x100 times 4096x4096 weights.
    "strassen2_2048x4096x4096_sign512": Workload(
        "strassen2_2048x4096x4096_sign512", 2048, 4096, 4096, "strassen", 2, "sign", 512,
        a_outliers=8, a_outlier_scale=100.0, b_sigma=0.02),
    # Laderman 3x3x3 rank 23, 512 random GL(3) gauges, E4M3 and E5M2.
    "laderman1_3072x4608x12288_gl512": Workload(
        "laderman1_3072x4608x12288_gl512", 3072, 4608, 12288, "laderman", 1, "gl", 512,
        fmts=("e4m3", "e5m2"), a_outliers=16, a_outlier_scale=300.0, b_sigma=0.02),
    # MLP up-projection, Student-t(3) activations, full sign orbit.
    "strassen2_4096x4096x14336_sign512": Workload(
        "strassen2_4096x4096x14336_sign512", 4096, 4096, 14336, "strassen", 2, "sign", 512,
        a_dist="t3", b_sigma=0.02),
    # MLP down-projection, three levels (8x8x8, rank 343), 512 sampled sign variants.
    "strassen3_8192x27648x5120_sign512": Workload(
        "strassen3_8192x27648x5120_sign512", 8192, 27648, 5120, "strassen", 3, "sign", 512,
        a_dist="t3", a_outliers=32, a_outlier_scale=1000.0, b_sigma=0.015, sign_sampled=True),
}

# Stand-ins for the layer slices on which App. E counts the overflow
# correction's multiplications (512 token rows, 1024 output channels, the
# layer's full inner dimension; groups of 128, blocks of inner length 32):
# two down projections (heavy-tailed inputs with a few large channels) and a
# gate projection (Gaussian inputs with outlier channels).
CORRECTION_SLICES = {
    "down_512x13824x1024": Workload(
        "down_512x13824x1024", 512, 13824, 1024, "strassen", 2, "sign", 1,
        a_dist="t3", a_outliers=8, a_outlier_scale=50.0, b_sigma=0.02, seed=20261203),
    "gate_512x4096x1024": Workload(
        "gate_512x4096x1024", 512, 4096, 1024, "strassen", 2, "sign", 1,
        a_outliers=16, a_outlier_scale=20.0, b_sigma=0.02, seed=20261204),
    "down_512x11008x1024": Workload(
        "down_512x11008x1024", 512, 11008, 1024, "strassen", 2, "sign", 1,
        a_dist="t3", a_outliers=4, a_outlier_scale=100.0, b_sigma=0.02, seed=20261205),
}

# Order of the workloads as listed for the method's evaluation: the first is
# the small case the oracle finishes in seconds, the second the headline one.
WORKLOAD_ORDER = list(WORKLOADS)


def scaled(w: Workload, M: int, K: int, N: int, G: int | None = None, name: str | None = None):
    """The same recipe at another shape (for tests at sizes the oracle runs fast)."""
    return replace(w, M=M, K=K, N=N, G=w.G if G is None else G,
                   name=name or f"{w.name}@{M}x{K}x{N}")


def _streams(seed: int, n: int):
    return [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(n)]


def operands(w: Workload, seed: int | None = None):
    """A (M x K) and B (K x N) as float32, row-major.

    A: N(0, a_sigma^2) or Student-t with 3 degrees of freedom (unscaled); then
    `a_outliers` distinct columns (inner-dimension channels), drawn without
    replacement, are multiplied by `a_outlier_scale`.
    B: N(0, b_sigma^2), b_sigma read as a standard deviation.
    """
    rs_a, rs_b, rs_o = _streams(w.seed if seed is None else seed, 3)
    if w.a_dist == "normal":
        A = rs_a.standard_normal((w.M, w.K), dtype=np.float32)
        if w.a_sigma != 1.0:
            A *= np.float32(w.a_sigma)
    elif w.a_dist == "t3":
        A = rs_a.standard_t(3, size=(w.M, w.K)).astype(np.float32)
    elif w.a_dist == "uniform01":
        A = rs_a.random((w.M, w.K), dtype=np.float32)
    elif w.a_dist == "uniform11":
        A = (rs_a.random((w.M, w.K), dtype=np.float32) * 2 - 1).astype(np.float32)
    else:
        raise ValueError(w.a_dist)
    if w.a_outliers:
        cols = rs_o.choice(w.K, size=w.a_outliers, replace=False)
        A[:, cols] *= np.float32(w.a_outlier_scale)
    B = rs_b.standard_normal((w.K, w.N), dtype=np.float32)
    if w.b_sigma != 1.0:
        B *= np.float32(w.b_sigma)
    return np.ascontiguousarray(A), np.ascontiguousarray(B)


def gl_matrix(rng, n: int, lo=-2.0, hi=2.0, max_cond=50.0):
    """An n x n matrix with iid U[lo, hi] entries, redrawn until its 2-norm
    condition number is below max_cond."""
    while True:
        P = rng.uniform(lo, hi, size=(n, n))
        if np.linalg.cond(P, 2) < max_cond:
            return P


def gl_gauges(m: int, k: int, n: int, count: int, seed: int):
    """`count` gauge triples (P, Q, S) in GL(m) x GL(k) x GL(n)."""
    rng = np.random.default_rng(seed)
    return [(gl_matrix(rng, m), gl_matrix(rng, k), gl_matrix(rng, n)) for _ in range(count)]


def _sign_vectors(dim: int):
    """All +-1 vectors of length dim with first entry +1, lexicographic with
    +1 before -1 (so the all-ones vector comes first)."""
    return [(1.0,) + t for t in itertools.product((1.0, -1.0), repeat=dim - 1)]


def sign_orbit(m: int, k: int, n: int):
    """The paper's sign variants (Sec. 2.1): all (d, e, f) with d_1 = e_1 =
    f_1 = 1; identity first.  For the 4x4x4 grid there are 512."""
    return [(d, e, f) for d in _sign_vectors(m) for e in _sign_vectors(k) for f in _sign_vectors(n)]


def sample_sign_orbit(m: int, k: int, n: int, count: int, seed: int):
    """`count` distinct sign variants drawn without replacement, identity first."""
    rng = np.random.default_rng(seed)
    total_bits = (m - 1) + (k - 1) + (n - 1)
    seen = {0}
    codes = [0]
    while len(codes) < count:
        c = int(rng.integers(0, 2 ** total_bits))
        if c not in seen:
            seen.add(c)
            codes.append(c)
    out = []
    for c in codes:
        bits = [(c >> b) & 1 for b in range(total_bits)][::-1]
        sg = [1.0 - 2.0 * b for b in bits]
        d = (1.0,) + tuple(sg[: m - 1])
        e = (1.0,) + tuple(sg[m - 1: m - 1 + k - 1])
        f = (1.0,) + tuple(sg[m - 1 + k - 1:])
        out.append((d, e, f))
    return out


def gauges(w: Workload, count: int | None = None, seed: int | None = None):
    """The workload's gauge elements as (P, Q, S) float64 matrices.

    'gl': random invertible transforms of the base grid (the identity is not
    included; callers evaluate it separately).  'sign': diagonal sign
    matrices on the flattened grid, the full orbit in lexicographic order or
    a seeded sample, identity first in both cases.
    """
    count = w.G if count is None else count
    s = (w.seed if seed is None else seed) + 7
    if w.gauge_kind == "gl":
        base = {"strassen": (2, 2, 2), "laderman": (3, 3, 3), "classical": (1, 1, 1)}[w.scheme]
        return gl_gauges(*base, count, s)
    gm, gk, gn = w.grid()
    if w.sign_sampled:
        sv = sample_sign_orbit(gm, gk, gn, count, s)
    else:
        sv = sign_orbit(gm, gk, gn)[:count]
    return [(np.diag(d), np.diag(e), np.diag(f)) for d, e, f in sv]


def identity_gauge(w: Workload):
    if w.gauge_kind == "gl":
        base = {"strassen": (2, 2, 2), "laderman": (3, 3, 3), "classical": (1, 1, 1)}[w.scheme]
    else:
        base = w.grid()
    return tuple(np.eye(b) for b in base)


def ratio_sample_positions(rows: int, cols: int, count: int, seed: int):
    """Seeded sample of (row, col) positions, for checks at full size."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, rows, size=count), rng.integers(0, cols, size=count)


# The synthetic ensemble of App. B.1: pairs of n x n operands with iid
# entries uniform on [lo, 1] (lo = -1 or 0), 200 pairs per distribution,
# every pair evaluated under each of the 512 sign variants of two-level
# Strassen.  Pair p of a distribution is drawn from its own stream, so any
# subset of pairs can be regenerated.
ENSEMBLE_SEED = 20260903
ENSEMBLE_PAIRS = 200
ENSEMBLE_N = 128


def ensemble_pair(lo: float, p: int, n: int = ENSEMBLE_N, seed: int = ENSEMBLE_SEED):
    rng = np.random.default_rng([seed, 0 if lo < 0 else 1, p])
    A = rng.uniform(lo, 1.0, (n, n)).astype(np.float32)
    B = rng.uniform(lo, 1.0, (n, n)).astype(np.float32)
    return A, B


__all__ = ["Workload", "WORKLOADS", "WORKLOAD_ORDER", "scaled", "operands", "gauges",
           "gl_gauges", "sign_orbit", "sample_sign_orbit", "identity_gauge",
           "ratio_sample_positions", "field", "ensemble_pair", "ENSEMBLE_PAIRS", "ENSEMBLE_N",
           "ENSEMBLE_SEED"]
