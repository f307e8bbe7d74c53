"""Scheme transforms and coefficient quantities, in float64.

TEST INFRASTRUCTURE ONLY: see oracle/__init__.py.

Every arithmetic step here is a plain Python float (IEEE float64) operation
in the order written, so the results are reproducible bit for bit:

  * Kronecker power (two-level Strassen is Strassen applied to its own
    blocks, Sec. 1 and Sec. 2.1): product index r = r1*R + r2 (outer level
    first), block index i = i1*m + i2, and coefficients multiplied left to
    right from the outer level.
  * Gauge action.  Sec. 2.1 runs the algorithm on DAE and EBF with sign
    matrices D, E, F and flips the result back.  The general form used here
    runs it on P A Q and Q^-1 B S (P, Q, S invertible, acting on block rows and
    columns) and undoes it with P^-1 . S^-1, which gives
        U'_r = P^T U_r Q^T,  V'_r = Q^-T V_r S^T,  W'_r = P^-1 W_r S^-1,
    and for sign matrices reduces to the paper's d_i e_l u, e_l f_j v,
    d_i f_j w.
  * Criteria of App. B.1 (Phi, nonzeros, largest magnitude, Q, E) and the
    headroom quantities of Sec. 4.2 (L_A, L_B, L_W, code bound, inner length).
"""
from __future__ import annotations

import numpy as np

from .schemes import Scheme


def as_matrices(vec: np.ndarray, rows: int, cols: int):
    return [[float(vec[a * cols + b]) for b in range(cols)] for a in range(rows)]


def kron(s1: Scheme, s2: Scheme) -> Scheme:
    """Scheme s2 applied inside every block of s1 (outer level s1)."""
    m, k, n = s1.m * s2.m, s1.k * s2.k, s1.n * s2.n
    R = s1.R * s2.R
    U = np.zeros((R, m * k))
    V = np.zeros((R, k * n))
    W = np.zeros((R, m * n))
    for r1 in range(s1.R):
        for r2 in range(s2.R):
            r = r1 * s2.R + r2
            for i1 in range(s1.m):
                for i2 in range(s2.m):
                    for l1 in range(s1.k):
                        for l2 in range(s2.k):
                            U[r, (i1 * s2.m + i2) * k + (l1 * s2.k + l2)] = (
                                float(s1.U[r1, i1 * s1.k + l1]) * float(s2.U[r2, i2 * s2.k + l2]))
            for l1 in range(s1.k):
                for l2 in range(s2.k):
                    for j1 in range(s1.n):
                        for j2 in range(s2.n):
                            V[r, (l1 * s2.k + l2) * n + (j1 * s2.n + j2)] = (
                                float(s1.V[r1, l1 * s1.n + j1]) * float(s2.V[r2, l2 * s2.n + j2]))
            for i1 in range(s1.m):
                for i2 in range(s2.m):
                    for j1 in range(s1.n):
                        for j2 in range(s2.n):
                            W[r, (i1 * s2.m + i2) * n + (j1 * s2.n + j2)] = (
                                float(s1.W[r1, i1 * s1.n + j1]) * float(s2.W[r2, i2 * s2.n + j2]))
    return Scheme(U, V, W, m, k, n, R)


def power(s: Scheme, levels: int) -> Scheme:
    """s applied recursively `levels` times, flattened to one level."""
    if levels < 1:
        raise ValueError("levels must be >= 1")
    out = s
    for _ in range(levels - 1):
        out = kron(out, s)
    return out


def inverse(P):
    """Inverse of a small float64 matrix given as nested lists.

    n <= 3: adjugate divided by the determinant (cofactor expansion along the
    first row).  n > 3: Gauss-Jordan elimination with partial pivoting.
    """
    n = len(P)
    if n == 1:
        return [[1.0 / P[0][0]]]
    if n == 2:
        a, b = P[0]
        c, d = P[1]
        det = a * d - b * c
        if det == 0.0:
            raise ZeroDivisionError("singular")
        return [[d / det, -b / det], [-c / det, a / det]]
    if n == 3:
        a, b, c = P[0]
        d, e, f = P[1]
        g, h, i = P[2]
        c00 = e * i - f * h
        c01 = -(d * i - f * g)
        c02 = d * h - e * g
        c10 = -(b * i - c * h)
        c11 = a * i - c * g
        c12 = -(a * h - b * g)
        c20 = b * f - c * e
        c21 = -(a * f - c * d)
        c22 = a * e - b * d
        det = a * c00 + b * c01 + c * c02
        if det == 0.0:
            raise ZeroDivisionError("singular")
        return [[c00 / det, c10 / det, c20 / det],
                [c01 / det, c11 / det, c21 / det],
                [c02 / det, c12 / det, c22 / det]]
    M = [list(map(float, row)) + [1.0 if a == b else 0.0 for b in range(n)]
         for a, row in enumerate(P)]
    for col in range(n):
        piv = max(range(col, n), key=lambda rr: abs(M[rr][col]))
        if M[piv][col] == 0.0:
            raise ZeroDivisionError("singular")
        M[col], M[piv] = M[piv], M[col]
        p = M[col][col]
        M[col] = [x / p for x in M[col]]
        for rr in range(n):
            if rr != col and M[rr][col] != 0.0:
                f = M[rr][col]
                M[rr] = [x - f * y for x, y in zip(M[rr], M[col])]
    return [row[n:] for row in M]


def _left_t(P, X):
    """P^T X: out[a][b] = sum_c P[c][a] X[c][b], c ascending from 0.0."""
    rows, cols = len(P[0]), len(X[0])
    out = []
    for a in range(rows):
        row = []
        for b in range(cols):
            s = 0.0
            for c in range(len(P)):
                s = s + P[c][a] * X[c][b]
            row.append(s)
        out.append(row)
    return out


def _left(P, X):
    """P X: out[a][b] = sum_c P[a][c] X[c][b], c ascending from 0.0."""
    out = []
    for a in range(len(P)):
        row = []
        for b in range(len(X[0])):
            s = 0.0
            for c in range(len(X)):
                s = s + P[a][c] * X[c][b]
            row.append(s)
        out.append(row)
    return out


def _right_t(X, Q):
    """X Q^T: out[a][b] = sum_c X[a][c] Q[b][c], c ascending from 0.0."""
    out = []
    for a in range(len(X)):
        row = []
        for b in range(len(Q)):
            s = 0.0
            for c in range(len(X[0])):
                s = s + X[a][c] * Q[b][c]
            row.append(s)
        out.append(row)
    return out


def _right(X, Q):
    """X Q: out[a][b] = sum_c X[a][c] Q[c][b], c ascending from 0.0."""
    out = []
    for a in range(len(X)):
        row = []
        for b in range(len(Q[0])):
            s = 0.0
            for c in range(len(Q)):
                s = s + X[a][c] * Q[c][b]
            row.append(s)
        out.append(row)
    return out


def gauge(s: Scheme, P, Q, S) -> Scheme:
    """Gauge-transformed scheme (P: m x m, Q: k x k, S: n x n).

    U'_r = (P^T U_r) Q^T, V'_r = (Q^-T V_r) S^T, W'_r = (P^-1 W_r) S^-1,
    each matrix product summed over its inner index in ascending order.
    """
    P = [list(map(float, row)) for row in np.asarray(P, dtype=np.float64)]
    Q = [list(map(float, row)) for row in np.asarray(Q, dtype=np.float64)]
    S = [list(map(float, row)) for row in np.asarray(S, dtype=np.float64)]
    assert len(P) == s.m and len(Q) == s.k and len(S) == s.n
    Pinv, Qinv, Sinv = inverse(P), inverse(Q), inverse(S)
    U = np.zeros_like(s.U)
    V = np.zeros_like(s.V)
    W = np.zeros_like(s.W)
    for r in range(s.R):
        u = _right_t(_left_t(P, as_matrices(s.U[r], s.m, s.k)), Q)
        v = _right_t(_left_t(Qinv, as_matrices(s.V[r], s.k, s.n)), S)
        w = _right(_left(Pinv, as_matrices(s.W[r], s.m, s.n)), Sinv)
        U[r] = np.array(u).reshape(-1)
        V[r] = np.array(v).reshape(-1)
        W[r] = np.array(w).reshape(-1)
    return Scheme(U, V, W, s.m, s.k, s.n, s.R)


def sign_gauge(s: Scheme, d, e, f) -> Scheme:
    """Sign variant with D = diag(d), E = diag(e), F = diag(f) (Sec. 2.1)."""
    return gauge(s, np.diag(np.asarray(d, float)), np.diag(np.asarray(e, float)),
                 np.diag(np.asarray(f, float)))


def to_f32(s: Scheme):
    """Coefficients rounded once to fp32 (round to nearest even)."""
    return (s.U.astype(np.float32), s.V.astype(np.float32), s.W.astype(np.float32))


def brent_residual(s: Scheme) -> float:
    """Largest violation of the Brent equations
    sum_r u[r,il] v[r,l'j] w[r,i'j'] = [i=i'][l=l'][j=j'], the condition for
    eq. (1) to compute AB for every A and B."""
    T = np.einsum("ra,rb,rc->abc", s.U, s.V, s.W)
    E = np.zeros_like(T)
    for i in range(s.m):
        for l in range(s.k):
            for j in range(s.n):
                E[i * s.k + l, l * s.n + j, i * s.n + j] = 1.0
    return float(np.abs(T - E).max())


def evaluate_f64(s: Scheme, A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """Eq. (1) in float64: block sums, R block products (library matmul),
    reconstruction.  Used to check that a scheme computes AB."""
    M, K = A.shape
    N = B.shape[1]
    br, bk, bc = M // s.m, K // s.k, N // s.n
    Ab = [[A[i * br:(i + 1) * br, l * bk:(l + 1) * bk] for l in range(s.k)] for i in range(s.m)]
    Bb = [[B[l * bk:(l + 1) * bk, j * bc:(j + 1) * bc] for j in range(s.n)] for l in range(s.k)]
    C = np.zeros((M, N))
    for r in range(s.R):
        T = sum(s.U[r, i * s.k + l] * Ab[i][l] for i in range(s.m) for l in range(s.k))
        S = sum(s.V[r, l * s.n + j] * Bb[l][j] for l in range(s.k) for j in range(s.n))
        Mr = T @ S
        for i in range(s.m):
            for j in range(s.n):
                w = s.W[r, i * s.n + j]
                if w != 0.0:
                    C[i * br:(i + 1) * br, j * bc:(j + 1) * bc] += w * Mr
    return C


def criteria(s: Scheme) -> dict:
    """Coefficient criteria of App. B.1 and the headroom quantities of
    Sec. 4.2, all read from the coefficients alone."""
    U, V, W = np.abs(s.U), np.abs(s.V), np.abs(s.W)
    phi = float(np.sum((U ** 2).sum(1) * (V ** 2).sum(1) * (W ** 2).sum(1)))
    nnz = int((s.U != 0).sum() + (s.V != 0).sum() + (s.W != 0).sum())
    maxabs = float(max(U.max(), V.max(), W.max()))
    alpha = (s.U != 0).sum(1)
    beta = (s.V != 0).sum(1)
    a1 = U.sum(1)
    b1 = V.sum(1)
    Qp = 0
    Ep = 0.0
    for ij in range(s.m * s.n):
        used = np.nonzero(s.W[:, ij])[0]
        gamma = len(used)
        Qp = max(Qp, gamma + int(max(alpha[used] + beta[used])))
        Ep = max(Ep, float(np.sum(a1 * b1 * W[:, ij])))
    LA = float(a1.max())
    LB = float(b1.max())
    LW = float(W.sum(0).max())
    bA = int(127 // LA)
    bB = int(127 // LB)
    # largest inner block length h with L_W * h * (L_A b_A)(L_B b_B) < 2^31
    denom = LW * (LA * bA) * (LB * bB)
    h = int((2 ** 31 - 1) // denom)
    while LW * (h + 1) * (LA * bA) * (LB * bB) < 2 ** 31:
        h += 1
    while LW * h * (LA * bA) * (LB * bB) >= 2 ** 31:
        h -= 1
    return dict(phi=phi, nnz=nnz, maxabs=maxabs, Q=Qp, E=Ep, L_A=LA, L_B=LB,
                L_W=LW, b_A=bA, b_B=bB, h_max_int32=h, R=s.R)
