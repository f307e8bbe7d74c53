"""Coefficient tables of the bilinear schemes the oracle evaluates.

TEST INFRASTRUCTURE ONLY: see oracle/__init__.py.

A scheme is (U, V, W, m, k, n, R) in the notation of eq. (1) (Sec. 2.1):
A is split into an m x k grid of blocks A_il, B into a k x n grid B_lj, and

    M_r = (sum_il u[r, il] A_il) (sum_lj v[r, lj] B_lj),   C_ij = sum_r w[r, ij] M_r.

Grid positions are flattened row-major: (i, l) -> i*k + l, (l, j) -> l*n + j,
(i, j) -> i*n + j.  Tables are float64 arrays of shape (R, m*k), (R, k*n),
(R, m*n).

The tables are written here as the linear forms of each product, parsed by a
small reader, so that they can be compared by eye with the printed source.
"""
from __future__ import annotations

import re
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Scheme:
    U: np.ndarray
    V: np.ndarray
    W: np.ndarray
    m: int
    k: int
    n: int
    R: int


def _linear_form(text: str, letter: str, rows: int, cols: int) -> np.ndarray:
    """Parse a signed sum such as 'a11+a12-a21' into a rows*cols vector."""
    out = np.zeros(rows * cols)
    text = text.replace(" ", "")
    for sign, idx in re.findall(r"([+-]?)" + letter + r"(\d\d)", text):
        i, j = int(idx[0]) - 1, int(idx[1]) - 1
        out[i * cols + j] += -1.0 if sign == "-" else 1.0
    return out


def _from_forms(products, outputs, m, k, n) -> Scheme:
    R = len(products)
    U = np.stack([_linear_form(a, "a", m, k) for a, _ in products])
    V = np.stack([_linear_form(b, "b", k, n) for _, b in products])
    W = np.zeros((R, m * n))
    for (i, j), form in outputs.items():
        for sign, r in re.findall(r"([+-]?)m(\d+)", form.replace(" ", "")):
            W[int(r) - 1, (i - 1) * n + (j - 1)] += -1.0 if sign == "-" else 1.0
    return Scheme(U, V, W, m, k, n, R)


def strassen() -> Scheme:
    """Strassen's 2x2x2 rank-7 algorithm as printed in App. A.1 (the table of
    the seven products with the rows each reads and feeds, in the proof of
    Theorem 1)."""
    products = [
        ("a11 + a22", "b11 + b22"),   # M1
        ("a21 + a22", "b11"),         # M2
        ("a11", "b12 - b22"),         # M3
        ("a22", "b21 - b11"),         # M4
        ("a11 + a12", "b22"),         # M5
        ("a21 - a11", "b11 + b12"),   # M6
        ("a12 - a22", "b21 + b22"),   # M7
    ]
    outputs = {
        (1, 1): "m1 + m4 - m5 + m7",
        (1, 2): "m3 + m5",
        (2, 1): "m2 + m4",
        (2, 2): "m1 - m2 + m3 + m6",
    }
    return _from_forms(products, outputs, 2, 2, 2)


def laderman() -> Scheme:
    """Laderman's 3x3x3 rank-23 algorithm (J. D. Laderman, Bull. AMS 82(1),
    1976).  The paper does not print it; it is the second base scheme of the
    evaluated workloads.  Its correctness is pinned by the Brent equations."""
    products = [
        ("a11 + a12 + a13 - a21 - a22 - a32 - a33", "b22"),                   # m1
        ("a11 - a21", "-b12 + b22"),                                         # m2
        ("a22", "-b11 + b12 + b21 - b22 - b23 - b31 + b33"),                 # m3
        ("-a11 + a21 + a22", "b11 - b12 + b22"),                             # m4
        ("a21 + a22", "-b11 + b12"),                                         # m5
        ("a11", "b11"),                                                      # m6
        ("-a11 + a31 + a32", "b11 - b13 + b23"),                             # m7
        ("-a11 + a31", "b13 - b23"),                                         # m8
        ("a31 + a32", "-b11 + b13"),                                         # m9
        ("a11 + a12 + a13 - a22 - a23 - a31 - a32", "b23"),                   # m10
        ("a32", "-b11 + b13 + b21 - b22 - b23 - b31 + b32"),                 # m11
        ("-a13 + a32 + a33", "b22 + b31 - b32"),                             # m12
        ("a13 - a33", "b22 - b32"),                                          # m13
        ("a13", "b31"),                                                      # m14
        ("a32 + a33", "-b31 + b32"),                                         # m15
        ("-a13 + a22 + a23", "b23 + b31 - b33"),                             # m16
        ("a13 - a23", "b23 - b33"),                                          # m17
        ("a22 + a23", "-b31 + b33"),                                         # m18
        ("a12", "b21"),                                                      # m19
        ("a23", "b32"),                                                      # m20
        ("a21", "b13"),                                                      # m21
        ("a31", "b12"),                                                      # m22
        ("a33", "b33"),                                                      # m23
    ]
    outputs = {
        (1, 1): "m6 + m14 + m19",
        (1, 2): "m1 + m4 + m5 + m6 + m12 + m14 + m15",
        (1, 3): "m6 + m7 + m9 + m10 + m14 + m16 + m18",
        (2, 1): "m2 + m3 + m4 + m6 + m14 + m16 + m17",
        (2, 2): "m2 + m4 + m5 + m6 + m20",
        (2, 3): "m14 + m16 + m17 + m18 + m21",
        (3, 1): "m6 + m7 + m8 + m11 + m12 + m13 + m14",
        (3, 2): "m12 + m13 + m14 + m15 + m22",
        (3, 3): "m6 + m7 + m8 + m9 + m23",
    }
    return _from_forms(products, outputs, 3, 3, 3)


def classical(m: int = 1, k: int = 1, n: int = 1) -> Scheme:
    """The classical algorithm, R = m*k*n, one product A_il B_lj per (i,l,j)
    (Sec. 2.1).  With m = k = n = 1 it is the plain product, the classical
    FP8 baseline."""
    R = m * k * n
    U = np.zeros((R, m * k))
    V = np.zeros((R, k * n))
    W = np.zeros((R, m * n))
    r = 0
    for i in range(m):
        for l in range(k):
            for j in range(n):
                U[r, i * k + l] = 1.0
                V[r, l * n + j] = 1.0
                W[r, i * n + j] = 1.0
                r += 1
    return Scheme(U, V, W, m, k, n, R)


BASE_SCHEMES = {"strassen": strassen, "laderman": laderman, "classical": classical}
