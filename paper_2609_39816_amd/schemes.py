"""Coefficient tables of the base schemes the library ships with.

Layout (the library's fm_scheme_load convention, eq. (1) of Sec. 2.1):
U is R x (m*k) over A's blocks (i, l) row-major, V is R x (k*n) over B's
blocks (l, j), W is R x (m*n) over C's blocks (i, j); float64.

  * strassen  -- Strassen's 2x2x2 rank-7 algorithm as the paper prints it
    (App. A.1, the table of the seven products and the four output blocks).
  * laderman  -- Laderman's 3x3x3 rank-23 algorithm (Bull. AMS 82(1), 1976);
    not in the paper, used for the 3x3x3 workload.
  * classical -- the plain product, R = m*k*n.
"""
from __future__ import annotations

import numpy as np


def strassen():
    # columns:        A11 A12 A21 A22
    U = np.array([[1, 0, 0, 1],    # M1 = (A11 + A22)(B11 + B22)
                  [0, 0, 1, 1],    # M2 = (A21 + A22) B11
                  [1, 0, 0, 0],    # M3 = A11 (B12 - B22)
                  [0, 0, 0, 1],    # M4 = A22 (B21 - B11)
                  [1, 1, 0, 0],    # M5 = (A11 + A12) B22
                  [-1, 0, 1, 0],   # M6 = (A21 - A11)(B11 + B12)
                  [0, 1, 0, -1]],  # M7 = (A12 - A22)(B21 + B22)
                 dtype=np.float64)
    # columns:        B11 B12 B21 B22
    V = np.array([[1, 0, 0, 1],
                  [1, 0, 0, 0],
                  [0, 1, 0, -1],
                  [-1, 0, 1, 0],
                  [0, 0, 0, 1],
                  [1, 1, 0, 0],
                  [0, 0, 1, 1]], dtype=np.float64)
    # columns:        C11 C12 C21 C22
    W = np.array([[1, 0, 0, 1],    # C11 = M1 + M4 - M5 + M7, C22 = M1 - M2 + M3 + M6
                  [0, 0, 1, -1],   # C21 = M2 + M4
                  [0, 1, 0, 1],    # C12 = M3 + M5
                  [1, 0, 1, 0],
                  [-1, 1, 0, 0],
                  [0, 0, 0, 1],
                  [1, 0, 0, 0]], dtype=np.float64)
    return U, V, W, 2, 2, 2


# Laderman's products as (A-coefficients, B-coefficients) over the 3x3 grids
# in row-major order, and the nine outputs as lists of product numbers
# (1-based); every nonzero coefficient is +1 or -1.
_LADERMAN_A = [
    [1, 1, 1, -1, -1, 0, 0, -1, -1],
    [1, 0, 0, -1, 0, 0, 0, 0, 0],
    [0, 0, 0, 0, 1, 0, 0, 0, 0],
    [-1, 0, 0, 1, 1, 0, 0, 0, 0],
    [0, 0, 0, 1, 1, 0, 0, 0, 0],
    [1, 0, 0, 0, 0, 0, 0, 0, 0],
    [-1, 0, 0, 0, 0, 0, 1, 1, 0],
    [-1, 0, 0, 0, 0, 0, 1, 0, 0],
    [0, 0, 0, 0, 0, 0, 1, 1, 0],
    [1, 1, 1, 0, -1, -1, -1, -1, 0],
    [0, 0, 0, 0, 0, 0, 0, 1, 0],
    [0, 0, -1, 0, 0, 0, 0, 1, 1],
    [0, 0, 1, 0, 0, 0, 0, 0, -1],
    [0, 0, 1, 0, 0, 0, 0, 0, 0],
    [0, 0, 0, 0, 0, 0, 0, 1, 1],
    [0, 0, -1, 0, 1, 1, 0, 0, 0],
    [0, 0, 1, 0, 0, -1, 0, 0, 0],
    [0, 0, 0, 0, 1, 1, 0, 0, 0],
    [0, 1, 0, 0, 0, 0, 0, 0, 0],
    [0, 0, 0, 0, 0, 1, 0, 0, 0],
    [0, 0, 0, 1, 0, 0, 0, 0, 0],
    [0, 0, 0, 0, 0, 0, 1, 0, 0],
    [0, 0, 0, 0, 0, 0, 0, 0, 1],
]
_LADERMAN_B = [
    [0, 0, 0, 0, 1, 0, 0, 0, 0],
    [0, -1, 0, 0, 1, 0, 0, 0, 0],
    [-1, 1, 0, 1, -1, -1, -1, 0, 1],
    [1, -1, 0, 0, 1, 0, 0, 0, 0],
    [-1, 1, 0, 0, 0, 0, 0, 0, 0],
    [1, 0, 0, 0, 0, 0, 0, 0, 0],
    [1, 0, -1, 0, 0, 1, 0, 0, 0],
    [0, 0, 1, 0, 0, -1, 0, 0, 0],
    [-1, 0, 1, 0, 0, 0, 0, 0, 0],
    [0, 0, 0, 0, 0, 1, 0, 0, 0],
    [-1, 0, 1, 1, -1, -1, -1, 1, 0],
    [0, 0, 0, 0, 1, 0, 1, -1, 0],
    [0, 0, 0, 0, 1, 0, 0, -1, 0],
    [0, 0, 0, 0, 0, 0, 1, 0, 0],
    [0, 0, 0, 0, 0, 0, -1, 1, 0],
    [0, 0, 0, 0, 0, 1, 1, 0, -1],
    [0, 0, 0, 0, 0, 1, 0, 0, -1],
    [0, 0, 0, 0, 0, 0, -1, 0, 1],
    [0, 0, 0, 1, 0, 0, 0, 0, 0],
    [0, 0, 0, 0, 0, 0, 0, 1, 0],
    [0, 0, 1, 0, 0, 0, 0, 0, 0],
    [0, 1, 0, 0, 0, 0, 0, 0, 0],
    [0, 0, 0, 0, 0, 0, 0, 0, 1],
]
_LADERMAN_C = [
    [6, 14, 19],
    [1, 4, 5, 6, 12, 14, 15],
    [6, 7, 9, 10, 14, 16, 18],
    [2, 3, 4, 6, 14, 16, 17],
    [2, 4, 5, 6, 20],
    [14, 16, 17, 18, 21],
    [6, 7, 8, 11, 12, 13, 14],
    [12, 13, 14, 15, 22],
    [6, 7, 8, 9, 23],
]


def laderman():
    U = np.array(_LADERMAN_A, dtype=np.float64)
    V = np.array(_LADERMAN_B, dtype=np.float64)
    W = np.zeros((23, 9))
    for ij, prods in enumerate(_LADERMAN_C):
        for p in prods:
            W[p - 1, ij] = 1.0
    return U, V, W, 3, 3, 3


def classical(m: int = 1, k: int = 1, n: int = 1):
    R = m * k * n
    U = np.zeros((R, m * k))
    V = np.zeros((R, k * n))
    W = np.zeros((R, m * n))
    for r, (i, l, j) in enumerate((i, l, j) for i in range(m) for l in range(k) for j in range(n)):
        U[r, i * k + l] = V[r, l * n + j] = W[r, i * n + j] = 1.0
    return U, V, W, m, k, n


BASE = {"strassen": strassen, "laderman": laderman, "classical": classical}
