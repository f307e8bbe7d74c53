"""CPU oracle for low-precision evaluation of bilinear fast-matmul schemes.

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
CPU-baseline leg of bench.py may import, call or link anything under oracle/.
The product path (paper_2609_39816_amd and its HIP library) never uses it,
and the two share no code: no kernels, headers, helpers, coefficient tables
or constant generators.  Only the seeded input generators of `synthetic`
feed both.

The oracle follows the paper step by step (plain loops, float64 where the
paper leaves the precision free):
  * eq. (1), Sec. 2.1: block sums, R block products, reconstruction;
  * the FP8 schedule of App. B.1: block sums rounded to e4m3 before
    multiplying, products and their combination in fp32;
  * App. F: FP8 simulated by rounding to the format and decoding, against a
    float64 reference; error = relative Frobenius norm (App. B.1);
  * orbit statistics with the conventions of App. B.2 (upper median,
    spread = largest / smallest, count above 2).
Readings where the paper is silent (one scale per block-sum tensor by
default, fmaf combination order, exact block products rounded once) are
stated at each function in fm_oracle.c; the finer granularity of App. B.1's
synthetic matrices (one scale per row of A's block sums and per column of
B's) is the SCALE_ROWCOL mode; the models' group scales (1 x 128 groups on
A's block sums, 128 x 128 blocks on B's bf16-rounded block sums, products
returned in bf16) are SCALE_GROUP.

Every function is parity-pinned by tests/test_oracle_*.py.
"""
from __future__ import annotations

import ctypes as ct
import os

import numpy as np

from . import build as _build
from . import scheme_ops, schemes  # noqa: F401  (re-exported)
from .schemes import Scheme

E4M3, E5M2 = 0, 1
FMT = {"e4m3": E4M3, "e5m2": E5M2}
# scale granularity: one scale per block-sum tensor, or (App. B.1's
# synthetic form) one per row of each A-side and per column of each B-side
# block sum
SCALE_TENSOR, SCALE_ROWCOL, SCALE_GROUP = 0, 1, 2
GROUP = 128  # inner-dimension group (and B-side block width) of SCALE_GROUP

_lib = None


def lib():
    global _lib
    if _lib is None:
        if _build.needs_build():
            _build.build()
        L = ct.CDLL(_build.LIB)
        f, d, i, i64, p = ct.c_float, ct.c_double, ct.c_int, ct.c_int64, ct.c_void_p
        sig = {
            "orc_fp8_encode": (ct.c_uint8, [f, i]),
            "orc_fp8_decode": (d, [ct.c_uint8, i]),
            "orc_fp8_max": (d, [i]),
            "orc_fp8_encode_array": (None, [p, i64, i, p]),
            "orc_fp8_decode_array": (None, [p, i64, i, p]),
            "orc_block_sum": (None, [p, i, i, i, i, p, p]),
            "orc_tensor_scale": (f, [p, i64, i, p]),
            "orc_quantize_tensor": (f, [p, i64, i, p]),
            "orc_block_product": (None, [p, p, f, f, i, i, i, i, p]),
            "orc_block_product_at": (None, [p, p, f, f, i, i, i, i, p, p, i, p]),
            "orc_reconstruct": (None, [p, p, i, i, i, i, i, p]),
            "orc_reference_f64": (None, [p, p, i, i, i, p]),
            "orc_reference_f64_at": (d, [p, p, i, i, i, i]),
            "orc_error_sums": (None, [p, p, i64, p, p]),
            "orc_lowp_matmul": (i, [p, p, i, i, i, i, i, i, i, p, p, p, i, p, p, p, p, p, p]),
            "orc_form_operands": (None, [p, i, i, i, i, i, p, i, p, p]),
            "orc_quantize_rows": (None, [p, i, i, i, p, p]),
            "orc_quantize_cols": (None, [p, i, i, i, p, p]),
            "orc_block_product_rc": (None, [p, p, p, p, i, i, i, i, p]),
            "orc_lowp_matmul_sm": (i, [p, p, i, i, i, i, i, i, i, p, p, p, i, i, p, p, p, p, p, p]),
            "orc_form_operands_sm": (None, [p, i, i, i, i, i, p, i, i, i, p, p]),
            "orc_int8_quantize_a": (None, [p, i, i, i, i, p, p]),
            "orc_int8_quantize_b": (None, [p, i, i, i, i, p, p]),
            "orc_int8_group_product": (None, [p, p, i, i, i, i, i, p]),
            "orc_int8_classical": (None, [p, p, p, p, i, i, i, i, p]),
            "orc_int8_group_product_fast": (None, [p, p, i, i, i, i, i, i, i, i, i, i, p, p, p, i,
                                                   p, p]),
            "orc_int8_fast": (i, [p, p, p, p, i, i, i, i, i, i, i, i, i, p, p, p, p, p]),
            "orc_int8_split": (None, [i64, p, p]),
            "orc_block_product_groups": (None, [p, p, p, p, i, i, i, i, p]),
            "orc_block_product_groups_acc": (None, [p, p, p, p, i, i, i, i, i, p]),
            "orc_bf16_round": (f, [f]),
            "orc_row_exponent": (i, [p, i]),
            "orc_joint_round_position": (i, [p, p, p, p, i, i, i, p]),
            "orc_repair_gram": (None, [p, p, i, i, i, p]),
            "orc_lowp_matmul_repaired": (i, [p, p, i, i, i, i, i, i, i, p, p, p, i, i, p, p, p, p,
                                             p, p, p]),
            "orc_int8_group_product_corrected": (None, [p, p, i, i, i, i, i, i, i, i, i, i, p, p,
                                                        p, p, p, p]),
            "orc_int8_fast_corrected": (i, [p, p, p, p, i, i, i, i, i, i, i, i, i, p, p, p, p,
                                            p, p]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ct.c_void_p)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


# --------------------------------------------------------------------------
# FP8 codec
# --------------------------------------------------------------------------
def fp8_encode(x, fmt: int = E4M3) -> np.ndarray:
    x = _f32(np.atleast_1d(x))
    out = np.empty(x.shape, np.uint8)
    lib().orc_fp8_encode_array(_ptr(x), x.size, fmt, _ptr(out))
    return out


def fp8_decode(c, fmt: int = E4M3) -> np.ndarray:
    c = np.ascontiguousarray(np.atleast_1d(c), dtype=np.uint8)
    out = np.empty(c.shape, np.float64)
    lib().orc_fp8_decode_array(_ptr(c), c.size, fmt, _ptr(out))
    return out


def fp8_max(fmt: int = E4M3) -> float:
    return lib().orc_fp8_max(fmt)


# --------------------------------------------------------------------------
# Steps of the schedule
# --------------------------------------------------------------------------
def block_sum(X, gr: int, gc: int, coef) -> np.ndarray:
    X = _f32(X)
    rows, cols = X.shape
    c = _f32(coef).reshape(-1)
    assert c.size == gr * gc and rows % gr == 0 and cols % gc == 0
    T = np.empty((rows // gr, cols // gc), np.float32)
    lib().orc_block_sum(_ptr(X), rows, cols, gr, gc, _ptr(c), _ptr(T))
    return T


def quantize_tensor(T, fmt: int = E4M3):
    """(codes, d, r): one scale for the whole tensor."""
    T = _f32(T)
    codes = np.empty(T.shape, np.uint8)
    d = lib().orc_quantize_tensor(_ptr(T), T.size, fmt, _ptr(codes))
    r = ct.c_float()
    lib().orc_tensor_scale(_ptr(T), T.size, fmt, ct.byref(r))
    return codes, np.float32(d), np.float32(r.value)


def quantize_rows(T, fmt: int = E4M3):
    """(codes, d): one scale per row of T (App. B.1, block sums of A)."""
    T = _f32(T)
    rows, cols = T.shape
    codes = np.empty(T.shape, np.uint8)
    d = np.empty(rows, np.float32)
    lib().orc_quantize_rows(_ptr(T), rows, cols, fmt, _ptr(codes), _ptr(d))
    return codes, d


def quantize_cols(T, fmt: int = E4M3):
    """(codes, d): one scale per column of T (App. B.1, block sums of B)."""
    T = _f32(T)
    rows, cols = T.shape
    codes = np.empty(T.shape, np.uint8)
    d = np.empty(cols, np.float32)
    lib().orc_quantize_cols(_ptr(T), rows, cols, fmt, _ptr(codes), _ptr(d))
    return codes, d


def form_operands(X, gr: int, gc: int, coef, fmt: int = E4M3, scale_mode: int = SCALE_TENSOR,
                  side: int = 0):
    """Block sums of one operand for every product r, quantized.
    Returns codes (R, rows/gr, cols/gc) in X's orientation and scales d: (R,)
    per tensor, or with SCALE_ROWCOL (R, rows/gr) for side 0 (A, per row)
    and (R, cols/gc) for side 1 (B, per column), or with SCALE_GROUP
    (R, Kb/128, Mb) for side 0 and (R, Kb/128, Nb/128) for side 1."""
    X = _f32(X)
    coef = _f32(coef)
    R = coef.shape[0]
    rows, cols = X.shape
    codes = np.empty((R, rows // gr, cols // gc), np.uint8)
    br, bc = rows // gr, cols // gc
    if scale_mode == SCALE_TENSOR:
        d = np.empty(R, np.float32)
    elif scale_mode == SCALE_ROWCOL:
        d = np.empty((R, br if side == 0 else bc), np.float32)
    else:
        assert bc % GROUP == 0 and (side == 0 or br % GROUP == 0)
        d = np.empty((R, bc // GROUP, br) if side == 0 else (R, br // GROUP, bc // GROUP),
                     np.float32)
    lib().orc_form_operands_sm(_ptr(X), rows, cols, gr, gc, R, _ptr(coef), fmt, scale_mode, side,
                               _ptr(codes), _ptr(d))
    return codes, d


def block_product(Tq, Sq, dT, dS, fmt: int = E4M3) -> np.ndarray:
    Tq = np.ascontiguousarray(Tq, np.uint8)
    Sq = np.ascontiguousarray(Sq, np.uint8)
    br, bk = Tq.shape
    bk2, bc = Sq.shape
    assert bk == bk2
    out = np.empty((br, bc), np.float32)
    lib().orc_block_product(_ptr(Tq), _ptr(Sq), float(dT), float(dS), br, bc, bk, fmt, _ptr(out))
    return out


def block_product_rc(Tq, Sq, dT, dS, fmt: int = E4M3) -> np.ndarray:
    """Block product with a scale per row of Tq (dT, br values) and per
    column of Sq (dS, bc values)."""
    Tq = np.ascontiguousarray(Tq, np.uint8)
    Sq = np.ascontiguousarray(Sq, np.uint8)
    br, bk = Tq.shape
    bk2, bc = Sq.shape
    assert bk == bk2
    dT, dS = _f32(dT), _f32(dS)
    assert dT.size == br and dS.size == bc
    out = np.empty((br, bc), np.float32)
    lib().orc_block_product_rc(_ptr(Tq), _ptr(Sq), _ptr(dT), _ptr(dS), br, bc, bk, fmt, _ptr(out))
    return out


def block_product_groups(Tq, Sq, dT, dS, fmt: int = E4M3, bf16: bool = True) -> np.ndarray:
    """Block product with group scales: dT (Kb/128, br), dS (Kb/128, bc/128);
    per group the exact sum rounded once is added by fmaf with dT * dS, and
    the product is returned rounded to bf16 (bf16=False: the fp32
    accumulator itself)."""
    Tq = np.ascontiguousarray(Tq, np.uint8)
    Sq = np.ascontiguousarray(Sq, np.uint8)
    br, bk = Tq.shape
    bk2, bc = Sq.shape
    assert bk == bk2 and bk % GROUP == 0 and bc % GROUP == 0
    dT, dS = _f32(dT), _f32(dS)
    assert dT.shape == (bk // GROUP, br) and dS.shape == (bk // GROUP, bc // GROUP)
    out = np.empty((br, bc), np.float32)
    lib().orc_block_product_groups_acc(_ptr(Tq), _ptr(Sq), _ptr(dT), _ptr(dS), br, bc, bk, fmt,
                                       int(bf16), _ptr(out))
    return out


def bf16_round(x) -> np.ndarray:
    """fp32 values rounded to the nearest bf16 (ties to even), as fp32."""
    x = _f32(x)
    f = lib().orc_bf16_round
    return np.array([f(float(v)) for v in x.reshape(-1)], np.float32).reshape(x.shape)


def block_product_at(Tq, Sq, dT, dS, xs, zs, fmt: int = E4M3) -> np.ndarray:
    Tq = np.ascontiguousarray(Tq, np.uint8)
    Sq = np.ascontiguousarray(Sq, np.uint8)
    br, bk = Tq.shape
    bc = Sq.shape[1]
    xs = np.ascontiguousarray(xs, np.int32)
    zs = np.ascontiguousarray(zs, np.int32)
    out = np.empty(xs.size, np.float32)
    lib().orc_block_product_at(_ptr(Tq), _ptr(Sq), float(dT), float(dS), br, bc, bk, fmt,
                               _ptr(xs), _ptr(zs), xs.size, _ptr(out))
    return out


def lowp_matmul_at(Tq, dT, Sq, dS, W, gm: int, gn: int, xs, zs, fmt: int = E4M3) -> np.ndarray:
    """The FP8 schedule's output at sampled positions, for shapes where the
    whole output is too slow to compute here.  From the quantized operands
    of every product (Tq (R, Mb, Kb), Sq (R, Kb, Nb), per-tensor scales dT,
    dS (R,)), the block products M_r at the in-block positions (xs[t], zs[t])
    and, from them, eq. (1)'s reconstruction of every output block at those
    positions, with the same arithmetic as the whole-output schedule.
    Returns C (gm, gn, S): C[i, j, t] is output entry
    (i Mb + xs[t], j Nb + zs[t])."""
    W = _f32(W)
    R = W.shape[0]
    xs = np.ascontiguousarray(xs, np.int32)
    zs = np.ascontiguousarray(zs, np.int32)
    S = xs.size
    Mr = np.empty((R, 1, S), np.float32)
    for r in range(R):
        Mr[r, 0] = block_product_at(Tq[r], Sq[r], dT[r], dS[r], xs, zs, fmt)
    return reconstruct(Mr, W, gm, gn).reshape(gm, gn, S)


def reconstruct(Mr, W, gm: int, gn: int) -> np.ndarray:
    Mr = _f32(Mr)
    R, br, bc = Mr.shape
    W = _f32(W)
    C = np.empty((gm * br, gn * bc), np.float32)
    lib().orc_reconstruct(_ptr(Mr), _ptr(W), R, gm, gn, br, bc, _ptr(C))
    return C


def reference_f64(A, B) -> np.ndarray:
    A, B = _f32(A), _f32(B)
    M, K = A.shape
    N = B.shape[1]
    C = np.empty((M, N), np.float64)
    lib().orc_reference_f64(_ptr(A), _ptr(B), M, N, K, _ptr(C))
    return C


def reference_f64_at(A, B, i: int, j: int) -> float:
    A, B = _f32(A), _f32(B)
    return lib().orc_reference_f64_at(_ptr(A), _ptr(B), B.shape[1], A.shape[1], i, j)


def error_sums(C, Cref):
    C = _f32(C)
    Cref = np.ascontiguousarray(Cref, np.float64)
    e, r = ct.c_double(), ct.c_double()
    lib().orc_error_sums(_ptr(C), _ptr(Cref), C.size, ct.byref(e), ct.byref(r))
    return e.value, r.value


def rel_fro(C, Cref) -> float:
    e, r = error_sums(C, Cref)
    return float(np.sqrt(e) / np.sqrt(r))


# --------------------------------------------------------------------------
# Whole schedule for one scheme
# --------------------------------------------------------------------------
def lowp_matmul(A, B, scheme_f32, dims, fmt: int = E4M3, keep: bool = False,
                scale_mode: int = SCALE_TENSOR):
    """FP8 evaluation of one scheme (fp32 coefficient tables U, V, W of the
    flattened scheme, dims = (m, k, n, R)).  Returns C, or with keep=True a
    dict with C, Tq (R, Mb, Kb), dT, Sq (R, Kb, Nb), dS and Mr (R, Mb, Nb);
    dT and dS are (R,) per tensor, (R, Mb) and (R, Nb) with SCALE_ROWCOL, or
    (R, Kb/128, Mb) and (R, Kb/128, Nb/128) with SCALE_GROUP."""
    U, V, W = (_f32(t) for t in scheme_f32)
    gm, gk, gn, R = dims
    A, B = _f32(A), _f32(B)
    M, K = A.shape
    N = B.shape[1]
    if M % gm or K % gk or N % gn:
        raise ValueError("shape not divisible by the block grid")
    br, bk, bc = M // gm, K // gk, N // gn
    C = np.empty((M, N), np.float32)
    if keep:
        Tq = np.empty((R, br, bk), np.uint8)
        Sq = np.empty((R, bk, bc), np.uint8)
        if scale_mode == SCALE_ROWCOL:
            dT, dS = np.empty((R, br), np.float32), np.empty((R, bc), np.float32)
        elif scale_mode == SCALE_GROUP:
            dT = np.empty((R, bk // GROUP, br), np.float32)
            dS = np.empty((R, bk // GROUP, bc // GROUP), np.float32)
        else:
            dT, dS = np.empty(R, np.float32), np.empty(R, np.float32)
        Mr = np.empty((R, br, bc), np.float32)
        args = [_ptr(Tq), _ptr(dT), _ptr(Sq), _ptr(dS), _ptr(Mr)]
    else:
        args = [None] * 5
    rc = lib().orc_lowp_matmul_sm(_ptr(A), _ptr(B), M, N, K, gm, gk, gn, R, _ptr(U), _ptr(V),
                                  _ptr(W), fmt, scale_mode, _ptr(C), *args)
    if rc != 0:
        raise ValueError("orc_lowp_matmul failed")
    if keep:
        return dict(C=C, Tq=Tq, dT=dT, Sq=Sq, dS=dS, Mr=Mr)
    return C


# --------------------------------------------------------------------------
# Repairs (App. C, the repair rules) on the group-scale schedule
# --------------------------------------------------------------------------
REPAIR_ROWS, REPAIR_WEIGHTS = 1, 2
REPAIR_SWEEPS = 12


def row_exponents(A) -> np.ndarray:
    """k_t with d_t = 2^k_t = 2^ceil(log2(max(RMS(row t), 1e-3)))."""
    A = _f32(A)
    return np.array([lib().orc_row_exponent(_ptr(A[t]), A.shape[1]) for t in range(A.shape[0])],
                    np.int32)


def repair_gram(U, W) -> np.ndarray:
    """H_rs = <w_r, w_s> <u_r, u_s> (float64 inner products, one fp32 rounding)."""
    U, W = _f32(U), _f32(W)
    R = U.shape[0]
    H = np.empty((R, R), np.float32)
    lib().orc_repair_gram(_ptr(U), _ptr(W), R, U.shape[1], W.shape[1], _ptr(H))
    return H


def joint_round_position(s, q, d, H, fmt: int = E4M3, max_sweeps: int = REPAIR_SWEEPS):
    """Joint rounding of one position: (codes (R,), sweeps made)."""
    s, q, d, H = _f32(s), _f32(q), _f32(d), _f32(H)
    R = s.size
    codes = np.empty(R, np.uint8)
    n = lib().orc_joint_round_position(_ptr(s), _ptr(q), _ptr(d), _ptr(H), R, fmt, max_sweeps,
                                       _ptr(codes))
    return codes, int(n)


def lowp_matmul_repaired(A, B, scheme_f32, dims, fmt: int = E4M3, flags: int = 3,
                         keep: bool = False):
    """The group-scale schedule with repairs (flags: REPAIR_ROWS,
    REPAIR_WEIGHTS).  Returns C, or with keep=True a dict with C, Tq, dT,
    Sq, dS, Mr and the row exponents."""
    U, V, W = (_f32(t) for t in scheme_f32)
    gm, gk, gn, R = dims
    A, B = _f32(A), _f32(B)
    M, K = A.shape
    N = B.shape[1]
    br, bk, bc = M // gm, K // gk, N // gn
    C = np.empty((M, N), np.float32)
    Tq = np.empty((R, br, bk), np.uint8)
    Sq = np.empty((R, bk, bc), np.uint8)
    dT = np.empty((R, bk // GROUP, br), np.float32)
    dS = np.empty((R, bk // GROUP, bc // GROUP), np.float32)
    Mr = np.empty((R, br, bc), np.float32)
    kx = np.empty(M, np.int32)
    rc = lib().orc_lowp_matmul_repaired(_ptr(A), _ptr(B), M, N, K, gm, gk, gn, R, _ptr(U), _ptr(V),
                                        _ptr(W), fmt, flags, _ptr(C), _ptr(Tq), _ptr(dT), _ptr(Sq),
                                        _ptr(dS), _ptr(Mr), _ptr(kx))
    if rc != 0:
        raise ValueError("shape not supported by the group-scale schedule")
    if keep:
        return dict(C=C, Tq=Tq, dT=dT, Sq=Sq, dS=dS, Mr=Mr, rowexp=kx)
    return C


def flatten_f32(s: Scheme):
    """(U, V, W) rounded to fp32 and the dims (m, k, n, R)."""
    return scheme_ops.to_f32(s), (s.m, s.k, s.n, s.R)


def classical_fp8(A, B, fmt: int = E4M3, scale_mode: int = SCALE_TENSOR):
    """Classical FP8 baseline: the plain product (R = 1) with one scale per
    operand (or per row of A and column of B), same rule as the block sums."""
    s = schemes.classical(1, 1, 1)
    tabs, dims = flatten_f32(s)
    return lowp_matmul(A, B, tabs, dims, fmt, scale_mode=scale_mode)


def orbit_stats(ratios, identity_value=None) -> dict:
    """Orbit statistics with the conventions of App. B.2: count, smallest,
    median (the upper of the two middle values for an even count), largest,
    spread = largest / smallest, and the number above 2."""
    x = np.sort(np.asarray(ratios, dtype=np.float64))
    n = x.size
    out = dict(count=int(n), min=float(x[0]), median=float(x[n // 2]), max=float(x[-1]),
               spread=float(x[-1] / x[0]), n_above_2=int((x > 2).sum()))
    if identity_value is not None:
        out["identity"] = float(identity_value)
    return out


def default_threads() -> int:
    return int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))


# --------------------------------------------------------------------------
# Integer codes and the classical int8 operator (Sec. 2.2, App. D), and the
# fast realization of Sec. 4.2 (Prop. 1)
# --------------------------------------------------------------------------
def int8_quantize_a(A, g: int, b: int):
    """Codes (M, K) int8 and scales d (M, K/g): one scale per row and group."""
    A = _f32(A)
    M, K = A.shape
    assert K % g == 0
    codes = np.empty((M, K), np.int8)
    d = np.empty((M, K // g), np.float32)
    lib().orc_int8_quantize_a(_ptr(A), M, K, g, b, _ptr(codes), _ptr(d))
    return codes, d


def int8_quantize_b(B, g: int, b: int):
    """Codes (K, N) int8 and scales d (K/g, N): one scale per column and group."""
    B = _f32(B)
    K, N = B.shape
    assert K % g == 0
    codes = np.empty((K, N), np.int8)
    d = np.empty((K // g, N), np.float32)
    lib().orc_int8_quantize_b(_ptr(B), K, N, g, b, _ptr(codes), _ptr(d))
    return codes, d


def int8_group_product(Ac, Bc, g: int, gi: int):
    Ac = np.ascontiguousarray(Ac, np.int8)
    Bc = np.ascontiguousarray(Bc, np.int8)
    M, K = Ac.shape
    N = Bc.shape[1]
    P = np.empty((M, N), np.int64)
    lib().orc_int8_group_product(_ptr(Ac), _ptr(Bc), M, N, K, g, gi, _ptr(P))
    return P


def int8_classical(Ac, dA, Bc, dB, g: int):
    """The classical int8 operator: fp32 output (M, N)."""
    Ac = np.ascontiguousarray(Ac, np.int8)
    Bc = np.ascontiguousarray(Bc, np.int8)
    dA, dB = _f32(dA), _f32(dB)
    M, K = Ac.shape
    N = Bc.shape[1]
    out = np.empty((M, N), np.float32)
    lib().orc_int8_classical(_ptr(Ac), _ptr(dA), _ptr(Bc), _ptr(dB), M, N, K, g, _ptr(out))
    return out


def int8_group_product_fast(Ac, Bc, scheme_f32, dims, g: int, gi: int, h: int,
                            round_fp8: bool = False):
    """One group's product computed call by call with the scheme; returns
    (P as float64 (M, N), violations of (i), violations of (ii))."""
    U, V, W = (_f32(t) for t in scheme_f32)
    gm, gk, gn, R = dims
    Ac = np.ascontiguousarray(Ac, np.int8)
    Bc = np.ascontiguousarray(Bc, np.int8)
    M, K = Ac.shape
    N = Bc.shape[1]
    P = np.empty((M, N), np.float64)
    viol = np.zeros(2, np.int64)
    lib().orc_int8_group_product_fast(_ptr(Ac), _ptr(Bc), M, N, K, g, gi, h, gm, gk, gn, R,
                                      _ptr(U), _ptr(V), _ptr(W), int(round_fp8), _ptr(P),
                                      _ptr(viol))
    return P, int(viol[0]), int(viol[1])


def int8_fast(Ac, dA, Bc, dB, scheme_f32, dims, g: int, h: int):
    """The fast realization's output (M, N) fp32 and the violation counts of
    conditions (i) and (ii) seen while computing it."""
    U, V, W = (_f32(t) for t in scheme_f32)
    gm, gk, gn, R = dims
    Ac = np.ascontiguousarray(Ac, np.int8)
    Bc = np.ascontiguousarray(Bc, np.int8)
    dA, dB = _f32(dA), _f32(dB)
    M, K = Ac.shape
    N = Bc.shape[1]
    out = np.empty((M, N), np.float32)
    viol = np.zeros(2, np.int64)
    rc = lib().orc_int8_fast(_ptr(Ac), _ptr(dA), _ptr(Bc), _ptr(dB), M, N, K, g, h, gm, gk, gn, R,
                             _ptr(U), _ptr(V), _ptr(W), _ptr(out), _ptr(viol))
    if rc != 0:
        raise ValueError("tiling does not fit the shape")
    return out, int(viol[0]), int(viol[1])


def int8_split(s: int):
    """Eq. (2)'s split of an exact block sum: (s0, q) with s = s0 + 256 q,
    q = floor((s + 128) / 256)."""
    s0, q = ct.c_int64(), ct.c_int64()
    lib().orc_int8_split(int(s), ct.byref(s0), ct.byref(q))
    return s0.value, q.value


def int8_fast_corrected(Ac, dA, Bc, dB, scheme_f32, dims, g: int, h: int):
    """The corrected realization (Sec. 4.3, eq. (2)): output (M, N) fp32 and a
    dict with the largest sum of absolute weighted terms per output entry
    (term_bound), split-range violations, the number of overflowing block
    sums, and the multiplication counts: main (A0 B0 products), sparse and
    gathered correction counts, and classical int8's M N K."""
    U, V, W = (_f32(t) for t in scheme_f32)
    gm, gk, gn, R = dims
    Ac = np.ascontiguousarray(Ac, np.int8)
    Bc = np.ascontiguousarray(Bc, np.int8)
    dA, dB = _f32(dA), _f32(dB)
    M, K = Ac.shape
    N = Bc.shape[1]
    out = np.empty((M, N), np.float32)
    stats = np.zeros(3, np.float64)
    counts = np.zeros(3, np.float64)
    rc = lib().orc_int8_fast_corrected(_ptr(Ac), _ptr(dA), _ptr(Bc), _ptr(dB), M, N, K, g, h, gm,
                                       gk, gn, R, _ptr(U), _ptr(V), _ptr(W), _ptr(out),
                                       _ptr(stats), _ptr(counts))
    if rc != 0:
        raise ValueError("tiling does not fit the shape")
    return out, dict(term_bound=stats[0], split_violations=int(stats[1]), overflows=int(stats[2]),
                     main=counts[0], sparse=counts[1], gathered=counts[2],
                     classical=float(M) * N * K)


def certificate(s: Scheme, b_A: int, b_B: int, h: int, g: int, gk: int):
    """Conditions (i)-(iii) of Prop. 1 for a scheme with integer coefficients
    (int32 accumulation): (i) L_A b_A <= 127 and L_B b_B <= 127; (ii)
    max(L_W h (L_A b_A)(L_B b_B), g b_A b_B) < 2^31; (iii) a call (gk blocks
    of inner length h) lies within one group (g a multiple of gk h)."""
    c = scheme_ops.criteria(s)
    LA, LB, LW = c["L_A"], c["L_B"], c["L_W"]
    i_ok = LA * b_A <= 127 and LB * b_B <= 127
    ii_ok = max(LW * h * (LA * b_A) * (LB * b_B), g * b_A * b_B) < 2 ** 31
    iii_ok = g % (gk * h) == 0
    return dict(L_A=LA, L_B=LB, L_W=LW, i=bool(i_ok), ii=bool(ii_ok), iii=bool(iii_ok),
                certified=bool(i_ok and ii_ok and iii_ok))
