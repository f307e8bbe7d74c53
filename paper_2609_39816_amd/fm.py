"""Python binding of libfm (include/fm.h): argument marshalling only.

Every step of the FP8 schedule runs in the library's HIP kernels; PyTorch
only provides device memory and the current stream.  Importing this module
fails loudly if the compiled library is missing: there is no CPU fallback.
"""
from __future__ import annotations

import ctypes as ct
import os
import re

import numpy as np

try:  # torch first: libfm then binds to the HIP runtime torch has loaded
    import torch
except ImportError:  # pragma: no cover - torch is part of the environment
    torch = None

from . import schemes as _schemes

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfm.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "fm.h")

E4M3, E5M2 = 0, 1
ACC_BF16, ACC_FP8 = 0, 1
SCALE_TENSOR, SCALE_ROWCOL, SCALE_GROUP = 0, 1, 2  # fm_scale_mode
REPAIR_ROWS, REPAIR_WEIGHTS = 0x100, 0x200  # OR-ed into SCALE_GROUP
FMTS = {"e4m3": E4M3, "e5m2": E5M2}
ERRORS = {0: "FM_OK", -1: "FM_E_ARG", -2: "FM_E_SHAPE", -3: "FM_E_BRENT", -4: "FM_E_SINGULAR",
          -5: "FM_E_NONFINITE", -6: "FM_E_WORKSPACE", -7: "FM_E_HIP", -8: "FM_E_MISMATCH",
          -9: "FM_E_NOMEM", -10: "FM_E_UNSUPPORTED", -11: "FM_E_RANGE", -12: "FM_E_UNCERTIFIED"}


class FmError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code
        self.name = ERRORS.get(code, str(code))


class _Stats(ct.Structure):
    _fields_ = [("rel_fro", ct.c_double), ("err_sq", ct.c_double), ("ref_sq", ct.c_double),
                ("max_abs", ct.c_double)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libfm is not built ({LIB_PATH} missing); run __graft_entry__.build() "
                          "or python paper_2609_39816_amd/build.py")
    L = ct.CDLL(LIB_PATH)
    p, i, d, sz, i64 = ct.c_void_p, ct.c_int, ct.c_double, ct.c_size_t, ct.c_int64
    pp = ct.POINTER(ct.c_void_p)
    sig = {
        "fm_strerror": (ct.c_char_p, [i]),
        "fm_last_error": (ct.c_char_p, []),
        "fm_version": (ct.c_char_p, []),
        "fm_scheme_load": (i, [p, p, p, i, i, i, i, pp]),
        "fm_gauge_apply": (i, [p, p, p, p, pp]),
        "fm_gauge_apply_batch": (i, [p, i, p, p, p, pp]),
        "fm_scheme_kron": (i, [p, i, pp]),
        "fm_scheme_dims": (i, [p, p, p, p, p]),
        "fm_scheme_coeffs": (i, [p, p, p, p]),
        "fm_scheme_coeffs_f32": (i, [p, i, p, p, p]),
        "fm_scheme_free": (None, [p]),
        "fm_workspace_size": (sz, [p, i, i, i, i, i, i]),
        "fm_error_workspace_size": (sz, [i, i]),
        "fm_form_operands": (i, [p, i, p, p, i, i, i, i, p, p, p, p, p, sz, p]),
        "fm_block_products": (i, [p, p, p, p, i, i, i, i, i, p, p]),
        "fm_reconstruct": (i, [p, i, p, i, i, p, p, sz, p]),
        "fm_matmul_lowp": (i, [p, p, p, p, i, i, i, i, i, p, sz, p]),
        "fm_reference_f64": (i, [p, p, p, i, i, i, p]),
        "fm_error_stats": (i, [p, p, i, i, ct.POINTER(_Stats), p, sz, p]),
        "fm_error_stats_noalloc": (i, [p, p, i, i, ct.POINTER(_Stats), p]),
        "fm_orbit_eval": (i, [p, i, p, p, p, i, i, i, i, i, p, p, sz, p]),
        "fm_workspace_size_scaled": (sz, [p, i, i, i, i, i, i, i]),
        "fm_form_operands_scaled": (i, [p, i, p, p, i, i, i, i, i, p, p, p, p, p, sz, p]),
        "fm_block_products_scaled": (i, [p, p, p, p, i, i, i, i, i, i, p, p]),
        "fm_matmul_lowp_scaled": (i, [p, p, p, p, i, i, i, i, i, i, p, sz, p]),
        "fm_orbit_eval_scaled": (i, [p, i, p, p, p, i, i, i, i, i, i, p, p, sz, p]),
        "fm_int8_quantize": (i, [p, i, i, i, i, p, p, p, p]),
        "fm_int8_matmul_classical": (i, [p, p, p, p, i, i, i, i, p, p]),
        "fm_int8_certify": (i, [p, i, i, i, i, i, p, p]),
        "fm_int8_workspace_size": (sz, [p, i, i, i, i, i, i]),
        "fm_int8_matmul_fast": (i, [p, i, p, p, p, p, i, i, i, i, i, i, i, p, p, sz, p]),
        "fm_int8_certify_corrected": (i, [p, i, i, i, i, i, p, p]),
        "fm_int8_workspace_size_corrected": (sz, [p, i, i, i, i, i, i]),
        "fm_int8_matmul_corrected": (i, [p, i, p, p, p, p, i, i, i, i, i, i, i, p, p, sz, p]),
        "fm_int8_plan_create": (i, [p, i, i, i, i, i, i, i, i, i, p, sz, p, pp]),
        "fm_int8_plan_run": (i, [p, p, p, p, p, p, p]),
        "fm_int8_plan_free": (None, [p]),
        "fm_fp8_encode": (i, [p, i64, i, i, p, p]),
        "fm_bf16_round": (i, [p, i64, i, p, p]),
        "fm_scheme_kernel_family": (ct.c_char_p, [p, i]),
        "fm_scheme_sign_variant": (i, [p, i, i, ct.POINTER(ct.c_int), ct.POINTER(ct.c_uint64)]),
        "fm_status": (i, [p, sz, p]),
        "fm_set_block_product_arithmetic": (i, [i]),
        "fm_timing_enable": (i, [i]),
        "fm_timing_reset": (i, []),
        "fm_timing_read": (i, [ct.c_char_p, ct.POINTER(ct.c_int), ct.POINTER(ct.c_double)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    return L


lib = _load()


def header_functions():
    """Names of the functions include/fm.h declares."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(fm_\w+)\s*\(", text, re.M)))


def _check(rc: int):
    if rc != 0:
        raise FmError(rc, lib.fm_last_error().decode())


def _dptr(t):
    return ct.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ct.c_void_p(stream.cuda_stream)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _np_ptr(a):
    return a.ctypes.data_as(ct.c_void_p)


def _cuda(t, dtype):
    if not (t.is_cuda and t.dtype == dtype and t.is_contiguous()):
        raise ValueError(f"expected a contiguous {dtype} tensor on the GPU")
    return t


# The library sees only pointers and sizes: the shapes of the tensors behind
# them are checked here, before any call.
def _matmul_shapes(A, B):
    """(M, K, N) of A (M, K) times B (K, N), both contiguous fp32 on one GPU."""
    _cuda(A, torch.float32), _cuda(B, torch.float32)
    if A.dim() != 2 or B.dim() != 2 or A.shape[1] != B.shape[0] or A.device != B.device:
        raise ValueError(f"A {tuple(A.shape)} and B {tuple(B.shape)} are not M x K and K x N "
                         "on one device")
    return A.shape[0], A.shape[1], B.shape[1]


def _out(out, shape, dtype, device):
    """A new output tensor, or the caller's after checking it."""
    if out is None:
        return torch.empty(shape, dtype=dtype, device=device)
    _cuda(out, dtype)
    if tuple(out.shape) != tuple(shape) or out.device != torch.device(device):
        raise ValueError(f"out must be {tuple(shape)} on {device}, got {tuple(out.shape)}")
    return out


def _ws(ws, device):
    """Pointer and byte size of a caller's workspace (a contiguous GPU tensor)."""
    if not (ws.is_cuda and ws.is_contiguous()) or ws.device != torch.device(device):
        raise ValueError(f"the workspace must be a contiguous tensor on {device}")
    return _dptr(ws), ws.numel() * ws.element_size()


class Scheme:
    """A bilinear scheme held by the library (fm_scheme*)."""

    def __init__(self, handle: int):
        self._h = ct.c_void_p(handle)

    def __del__(self):
        h = getattr(self, "_h", None)
        free = getattr(lib, "fm_scheme_free", None) if lib is not None else None
        if h is not None and h.value and free is not None:
            free(h)
            self._h = None

    @property
    def handle(self):
        return self._h

    @classmethod
    def load(cls, U, V, W, m: int, k: int, n: int) -> "Scheme":
        U, V, W = _f64(U), _f64(V), _f64(W)
        R = U.shape[0]
        out = ct.c_void_p()
        _check(lib.fm_scheme_load(_np_ptr(U), _np_ptr(V), _np_ptr(W), m, n, k, R, ct.byref(out)))
        return cls(out.value)

    @classmethod
    def base(cls, name: str) -> "Scheme":
        U, V, W, m, k, n = _schemes.BASE[name]()
        return cls.load(U, V, W, m, k, n)

    def gauge(self, P, Q, S) -> "Scheme":
        P, Q, S = _f64(P), _f64(Q), _f64(S)
        out = ct.c_void_p()
        _check(lib.fm_gauge_apply(self._h, _np_ptr(P), _np_ptr(Q), _np_ptr(S), ct.byref(out)))
        return Scheme(out.value)

    def gauge_orbit(self, gauges) -> list:
        """Gauged copies for a list of (P, Q, S), in one library call."""
        G = len(gauges)
        if G == 0:
            return []
        P = _f64(np.stack([g[0] for g in gauges]))
        Q = _f64(np.stack([g[1] for g in gauges]))
        S = _f64(np.stack([g[2] for g in gauges]))
        out = (ct.c_void_p * G)()
        _check(lib.fm_gauge_apply_batch(self._h, G, _np_ptr(P), _np_ptr(Q), _np_ptr(S), out))
        return [Scheme(h) for h in out]

    def kron(self, levels: int) -> "Scheme":
        out = ct.c_void_p()
        _check(lib.fm_scheme_kron(self._h, levels, ct.byref(out)))
        return Scheme(out.value)

    @property
    def dims(self):
        m, n, k, R = ct.c_int(), ct.c_int(), ct.c_int(), ct.c_int()
        _check(lib.fm_scheme_dims(self._h, ct.byref(m), ct.byref(n), ct.byref(k), ct.byref(R)))
        return m.value, k.value, n.value, R.value  # (m, k, n, R)

    def coeffs(self):
        m, k, n, R = self.dims
        U, V, W = np.empty((R, m * k)), np.empty((R, k * n)), np.empty((R, m * n))
        _check(lib.fm_scheme_coeffs(self._h, _np_ptr(U), _np_ptr(V), _np_ptr(W)))
        return U, V, W

    def coeffs_f32(self, levels: int = 1):
        m, k, n, R = self.dims
        m, k, n, R = m ** levels, k ** levels, n ** levels, R ** levels
        U = np.empty((R, m * k), np.float32)
        V = np.empty((R, k * n), np.float32)
        W = np.empty((R, m * n), np.float32)
        _check(lib.fm_scheme_coeffs_f32(self._h, levels, _np_ptr(U), _np_ptr(V), _np_ptr(W)))
        return U, V, W

    def kernel_family(self, levels: int = 1) -> str:
        return lib.fm_scheme_kernel_family(self._h, levels).decode()

    def sign_variant(self, levels: int = 1, side: int = 0):
        """(is_sign, neg_mask): whether the flattened scheme's side (0: A,
        1: B) is a sign variant of its family's base scheme, and the mask of
        negated blocks."""
        flag, mask = ct.c_int(), ct.c_uint64()
        _check(lib.fm_scheme_sign_variant(self._h, levels, side, ct.byref(flag), ct.byref(mask)))
        return bool(flag.value), int(mask.value)

    def flat_dims(self, levels: int = 1):
        m, k, n, R = self.dims
        return m ** levels, k ** levels, n ** levels, R ** levels


def workspace_size(s: Scheme, M: int, N: int, K: int, levels: int = 1, G: int = 1,
                   chunk: int = 0, scale_mode: int = SCALE_TENSOR) -> int:
    return int(lib.fm_workspace_size_scaled(s.handle, M, N, K, levels, G, chunk, scale_mode))


def workspace(nbytes: int, device=None):
    """Zero-filled device workspace (torch allocations are 256-byte aligned)."""
    return torch.zeros(max(int(nbytes), 256), dtype=torch.uint8, device=device or "cuda")


def form_operands(s: Scheme, A, B, levels: int = 1, fmt: int = E4M3, ws=None, stream=None,
                  scale_mode: int = SCALE_TENSOR):
    """Quantized block sums: Tq (R, Mb, Kb) u8, Sq (R, Nb, Kb) u8 (transposed),
    dT (R,) and dS (R,) fp32, or (R, Mb) and (R, Nb) with SCALE_ROWCOL, or
    (R, Kb/128, Mb) and (R, Kb/128, Nb/128) with SCALE_GROUP."""
    M, K, N = _matmul_shapes(A, B)
    gm, gk, gn, R = s.flat_dims(levels)
    Mb, Nb = M // gm, N // gn
    Tq = torch.empty((R, Mb, K // gk), dtype=torch.uint8, device=A.device)
    Sq = torch.empty((R, Nb, K // gk), dtype=torch.uint8, device=A.device)
    Kb = K // gk
    shp = {SCALE_ROWCOL: ((R, Mb), (R, Nb)),
           SCALE_GROUP: ((R, Kb // 128, Mb), (R, Kb // 128, Nb // 128))}.get(scale_mode & 0xff,
                                                                           ((R,), (R,)))
    dT = torch.empty(shp[0], dtype=torch.float32, device=A.device)
    dS = torch.empty(shp[1], dtype=torch.float32, device=A.device)
    if ws is None:
        ws = workspace(workspace_size(s, M, N, K, levels, 1, 1, scale_mode), A.device)
    _check(lib.fm_form_operands_scaled(s.handle, levels, _dptr(A), _dptr(B), M, N, K, fmt,
                                       scale_mode, _dptr(Tq), _dptr(Sq), _dptr(dT), _dptr(dS),
                                       *_ws(ws, A.device), _stream(stream)))
    return Tq, Sq, dT, dS


def block_products(Tq, Sq, dT, dS, fmt: int = E4M3, out=None, stream=None,
                   scale_mode: int = SCALE_TENSOR):
    """Mout[b] = ((Tq[b] Sq[b]^T) * dT) * dS; dT, dS per product (batch,) or,
    with SCALE_ROWCOL, per row (batch, Mb) and per column (batch, Nb); with
    SCALE_GROUP per group (batch, Kb/128, Mb) and (batch, Kb/128, Nb/128),
    products returned in bf16 (as fp32 values)."""
    _cuda(Tq, torch.uint8), _cuda(Sq, torch.uint8)
    if Tq.dim() != 3 or Sq.dim() != 3 or Sq.shape[0] != Tq.shape[0] or Sq.shape[2] != Tq.shape[2] \
            or Sq.device != Tq.device:
        raise ValueError(f"Tq {tuple(Tq.shape)} and Sq {tuple(Sq.shape)} are not "
                         "(batch, Mb, Kb) and (batch, Nb, Kb) on one device")
    batch, Mb, Kb = Tq.shape
    Nb = Sq.shape[1]
    want = {SCALE_ROWCOL: (batch * Mb, batch * Nb),
            SCALE_GROUP: (batch * (Kb // 128) * Mb, batch * (Kb // 128) * (Nb // 128))
            }.get(scale_mode, (batch, batch))
    if (dT.numel(), dS.numel()) != want:
        raise ValueError(f"scale arrays hold {dT.numel()} and {dS.numel()} values, need {want}")
    _cuda(dT, torch.float32), _cuda(dS, torch.float32)
    if scale_mode in (SCALE_ROWCOL, SCALE_GROUP):
        # the kernels read scales in aligned 16-byte chunks: give them a
        # fresh, padded copy whenever the caller's arrays are not such
        def padded(t):
            if t.data_ptr() % 16 == 0 and t.numel() % 4 == 0:
                return t
            p = torch.zeros((t.numel() + 3) // 4 * 4, dtype=torch.float32, device=t.device)
            p[:t.numel()] = t.reshape(-1)
            return p
        dT, dS = padded(dT), padded(dS)
    out = _out(out, (batch, Mb, Nb), torch.float32, Tq.device)
    _check(lib.fm_block_products_scaled(_dptr(Tq), _dptr(Sq), _dptr(dT), _dptr(dS), batch, Mb, Nb,
                                        Kb, fmt, scale_mode, _dptr(out), _stream(stream)))
    return out


def reconstruct(s: Scheme, Mprod, M: int, N: int, levels: int = 1, ws=None, stream=None):
    _cuda(Mprod, torch.float32)
    gm, gk, gn, R = s.flat_dims(levels)
    if M % gm or N % gn or Mprod.numel() != R * (M // gm) * (N // gn):
        raise ValueError(f"Mprod holds {Mprod.numel()} values, not R x (M/{gm}) x (N/{gn})")
    C = torch.empty((M, N), dtype=torch.float32, device=Mprod.device)
    if ws is None:
        ws = workspace(workspace_size(s, M, N, gk * 16, levels, 1, 1), Mprod.device)
    _check(lib.fm_reconstruct(s.handle, levels, _dptr(Mprod), M, N, _dptr(C),
                              *_ws(ws, Mprod.device), _stream(stream)))
    return C


def matmul_lowp(s: Scheme, A, B, levels: int = 1, fmt: int = E4M3, ws=None, out=None,
                stream=None, scale_mode: int = SCALE_TENSOR):
    M, K, N = _matmul_shapes(A, B)
    out = _out(out, (M, N), torch.float32, A.device)
    if ws is None:
        ws = workspace(workspace_size(s, M, N, K, levels, 1, 1, scale_mode), A.device)
    _check(lib.fm_matmul_lowp_scaled(s.handle, _dptr(A), _dptr(B), _dptr(out), M, N, K, levels,
                                     fmt, scale_mode, *_ws(ws, A.device), _stream(stream)))
    return out


def reference_f64(A, B, out=None, stream=None):
    M, K, N = _matmul_shapes(A, B)
    out = _out(out, (M, N), torch.float64, A.device)
    _check(lib.fm_reference_f64(_dptr(A), _dptr(B), _dptr(out), M, N, K, _stream(stream)))
    return out


def _error_shapes(C, Cref):
    _cuda(C, torch.float32), _cuda(Cref, torch.float64)
    if C.dim() != 2 or tuple(C.shape) != tuple(Cref.shape) or C.device != Cref.device:
        raise ValueError(f"C {tuple(C.shape)} and C_ref {tuple(Cref.shape)} differ")
    return C.shape


def error_stats(C, Cref, ws=None, stream=None) -> dict:
    M, N = _error_shapes(C, Cref)
    if ws is None:
        ws = workspace(lib.fm_error_workspace_size(M, N), C.device)
    st = _Stats()
    _check(lib.fm_error_stats(_dptr(C), _dptr(Cref), M, N, ct.byref(st), *_ws(ws, C.device),
                              _stream(stream)))
    return dict(rel_fro=st.rel_fro, err_sq=st.err_sq, ref_sq=st.ref_sq, max_abs=st.max_abs)


def error_stats_noalloc(C, Cref, stream=None) -> dict:
    """error_stats without a workspace: the library's static device scratch
    holds the partial sums (calls overlapping on one device race)."""
    M, N = _error_shapes(C, Cref)
    st = _Stats()
    _check(lib.fm_error_stats_noalloc(_dptr(C), _dptr(Cref), M, N, ct.byref(st), _stream(stream)))
    return dict(rel_fro=st.rel_fro, err_sq=st.err_sq, ref_sq=st.ref_sq, max_abs=st.max_abs)


def orbit_eval(gauged, A, B, Cref, levels: int = 1, fmt: int = E4M3, ws=None, chunk: int = 0,
               stream=None, scale_mode: int = SCALE_TENSOR) -> np.ndarray:
    """Relative Frobenius errors of the FP8 schedule for every gauged scheme."""
    M, K, N = _matmul_shapes(A, B)
    _cuda(Cref, torch.float64)
    if tuple(Cref.shape) != (M, N) or Cref.device != A.device:
        raise ValueError(f"C_ref must be ({M}, {N}) on {A.device}, got {tuple(Cref.shape)}")
    G = len(gauged)
    if G < 1:
        raise ValueError("the orbit needs at least one scheme")
    handles = (ct.c_void_p * G)(*[g.handle.value for g in gauged])
    if ws is None:
        ws = workspace(workspace_size(gauged[0], M, N, K, levels, G, chunk, scale_mode), A.device)
    out = np.empty(G, np.float64)
    _check(lib.fm_orbit_eval_scaled(ct.cast(handles, ct.c_void_p), G, _dptr(A), _dptr(B),
                                    _dptr(Cref), M, N, K, levels, fmt, scale_mode, _np_ptr(out),
                                    *_ws(ws, A.device), _stream(stream)))
    return out


def fp8_encode(x, fmt: int = E4M3, impl: int = 0, stream=None):
    _cuda(x, torch.float32)
    out = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    _check(lib.fm_fp8_encode(_dptr(x), x.numel(), fmt, impl, _dptr(out), _stream(stream)))
    return out


def bf16_round(x, impl: int = 0, stream=None):
    _cuda(x, torch.float32)
    out = torch.empty_like(x)
    _check(lib.fm_bf16_round(_dptr(x), x.numel(), impl, _dptr(out), _stream(stream)))
    return out


def status(ws, stream=None):
    _check(lib.fm_status(*_ws(ws, ws.device), _stream(stream)))


_arith = ACC_BF16


def set_block_product_arithmetic(acc: int):
    """ACC_BF16 (exact products, fp32 sums; default) or ACC_FP8 (FP8 matrix
    instructions)."""
    global _arith
    _check(lib.fm_set_block_product_arithmetic(acc))
    _arith = acc


def get_block_product_arithmetic() -> int:
    """The arithmetic last selected through set_block_product_arithmetic."""
    return _arith


def timing_enable(on: bool = True):
    _check(lib.fm_timing_enable(1 if on else 0))


def timing_reset():
    _check(lib.fm_timing_reset())


def timing_read(kernel_class: str):
    """(launches, total milliseconds) of one kernel class since the last reset."""
    n, ms = ct.c_int(), ct.c_double()
    _check(lib.fm_timing_read(kernel_class.encode(), ct.byref(n), ct.byref(ms)))
    return n.value, ms.value


TIMED_CLASSES = ("form_amax", "form_quant", "block_gemm", "recon", "reference")


def version() -> str:
    return lib.fm_version().decode()


# ------------------------------------------------------------ integer path
def int8_quantize(X, g: int = 128, b: int = 31, flag=None, stream=None):
    """Codes (rows, K) int8 and group-major scales (K/g, rows) fp32 of X:
    one scale per row and group of g along K (App. D).  Quantize B through
    its transpose."""
    _cuda(X, torch.float32)
    rows, K = X.shape
    codes = torch.empty((rows, K), dtype=torch.int8, device=X.device)
    d = torch.empty((K // g, rows), dtype=torch.float32, device=X.device)
    _check(lib.fm_int8_quantize(_dptr(X), rows, K, g, b, _dptr(codes), _dptr(d),
                                _dptr(flag) if flag is not None else None, _stream(stream)))
    return codes, d


def _int8_operands(Ac, dA, BTc, dB, g, out):
    """Shapes of the integer operators' arguments, checked against each other
    (the library sees only pointers): Ac (M, K), BTc (N, K) int8; dA (K/g, M),
    dB (K/g, N) fp32; out (M, N) fp32."""
    _cuda(Ac, torch.int8), _cuda(BTc, torch.int8), _cuda(dA, torch.float32), _cuda(dB, torch.float32)
    M, K = Ac.shape
    N = BTc.shape[0]
    if BTc.shape[1] != K or g <= 0 or K % g:
        raise ValueError("Ac and BTc must share K, a multiple of g")
    if tuple(dA.shape) != (K // g, M) or tuple(dB.shape) != (K // g, N):
        raise ValueError("scales must be (K/g, M) and (K/g, N)")
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=Ac.device)
    _cuda(out, torch.float32)
    if tuple(out.shape) != (M, N):
        raise ValueError("out must be (M, N)")
    return M, N, K, out


def int8_matmul_classical(Ac, dA, BTc, dB, g: int = 128, out=None, stream=None):
    """The classical int8 operator: Ac (M, K), BTc (N, K) codes; dA (K/g, M),
    dB (K/g, N); fp32 output (M, N)."""
    M, N, K, out = _int8_operands(Ac, dA, BTc, dB, g, out)
    _check(lib.fm_int8_matmul_classical(_dptr(Ac), _dptr(dA), _dptr(BTc), _dptr(dB), M, N, K, g,
                                        _dptr(out), _stream(stream)))
    return out


def int8_certify(s: Scheme, levels: int = 1, b_A: int = 31, b_B: int = 31, h: int = 32,
                 g: int = 128) -> dict:
    """Prop. 1's conditions (i)-(iii) and L_A, L_B, L_W for the flattened scheme."""
    cond = (ct.c_int * 3)()
    L = (ct.c_double * 3)()
    _check(lib.fm_int8_certify(s.handle, levels, b_A, b_B, h, g, cond, L))
    return dict(i=bool(cond[0]), ii=bool(cond[1]), iii=bool(cond[2]),
                certified=bool(cond[0] and cond[1] and cond[2]), L_A=L[0], L_B=L[1], L_W=L[2])


def int8_workspace_size(s: Scheme, M: int, N: int, K: int, levels: int = 1, g: int = 128,
                        h: int = 32, correct: bool = False) -> int:
    fn = lib.fm_int8_workspace_size_corrected if correct else lib.fm_int8_workspace_size
    return int(fn(s.handle, levels, M, N, K, g, h))


def int8_certify_corrected(s: Scheme, levels: int = 1, b_A: int = 127, b_B: int = 127,
                           h: int = 32, g: int = 128) -> dict:
    """The corrected computation's certificate (App. D): conditions and bounds."""
    cond = (ct.c_int * 3)()
    bnd = (ct.c_double * 3)()
    _check(lib.fm_int8_certify_corrected(s.handle, levels, b_A, b_B, h, g, cond, bnd))
    return dict(split=bool(cond[0]), int32=bool(cond[1]), one_group=bool(cond[2]),
                certified=bool(cond[0] and cond[1] and cond[2]), term_bound=bnd[0],
                qmax_A=int(bnd[1]), qmax_B=int(bnd[2]))


def int8_matmul_fast(s: Scheme, Ac, dA, BTc, dB, levels: int = 1, g: int = 128, h: int = 32,
                     b_A: int = 31, b_B: int = 31, ws=None, out=None, stream=None):
    """The certified fast realization (Sec. 4.2): same output bits as
    int8_matmul_classical for codes within the bounds."""
    M, N, K, out = _int8_operands(Ac, dA, BTc, dB, g, out)
    if ws is None:
        need = int8_workspace_size(s, M, N, K, levels, g, h)
        if need == 0:
            raise FmError(-1, "fm_int8_workspace_size: arguments not supported")
        ws = workspace(need, Ac.device)
    _check(lib.fm_int8_matmul_fast(s.handle, levels, _dptr(Ac), _dptr(dA), _dptr(BTc), _dptr(dB),
                                   M, N, K, g, h, b_A, b_B, _dptr(out), *_ws(ws, Ac.device),
                                   _stream(stream)))
    return out


def int8_matmul_corrected(s: Scheme, Ac, dA, BTc, dB, levels: int = 1, g: int = 128,
                          h: int = 32, b_A: int = 127, b_B: int = 127, ws=None, out=None,
                          stream=None):
    """The fast realization with the overflow correction (Sec. 4.3, eq. (2)):
    same output bits as int8_matmul_classical up to code bound 127."""
    M, N, K, out = _int8_operands(Ac, dA, BTc, dB, g, out)
    if ws is None:
        need = int8_workspace_size(s, M, N, K, levels, g, h, correct=True)
        if need == 0:
            raise FmError(-1, "fm_int8_workspace_size_corrected: arguments not supported")
        ws = workspace(need, Ac.device)
    _check(lib.fm_int8_matmul_corrected(s.handle, levels, _dptr(Ac), _dptr(dA), _dptr(BTc),
                                        _dptr(dB), M, N, K, g, h, b_A, b_B, _dptr(out),
                                        *_ws(ws, Ac.device), _stream(stream)))
    return out


class Int8Plan:
    """A prepared fast call (fm_int8_plan_*): the scheme's tables and tile
    schedule are written to the workspace once; run() then launches only the
    block-sum and product kernels.  Holds its workspace."""

    def __init__(self, s: Scheme, M: int, N: int, K: int, levels: int = 1, g: int = 128,
                 h: int = 32, b_A: int = 31, b_B: int = 31, correct: bool = False, ws=None,
                 device=None, stream=None):
        self._h = None
        need = int8_workspace_size(s, M, N, K, levels, g, h, correct)
        if need == 0:
            raise FmError(-1, "fm_int8_workspace_size: arguments not supported")
        self.ws = ws if ws is not None else workspace(need, device)
        self.M, self.N, self.K, self.g = M, N, K, g
        out = ct.c_void_p()
        _check(lib.fm_int8_plan_create(s.handle, levels, M, N, K, g, h, b_A, b_B, int(correct),
                                       *_ws(self.ws, self.ws.device), _stream(stream),
                                       ct.byref(out)))
        self._h = out.value

    def __del__(self):
        if getattr(self, "_h", None) and lib is not None:
            lib.fm_int8_plan_free(ct.c_void_p(self._h))
            self._h = None

    def run(self, Ac, dA, BTc, dB, out=None, stream=None):
        M, N, K, out = _int8_operands(Ac, dA, BTc, dB, self.g, out)
        if (M, N, K) != (self.M, self.N, self.K):
            raise ValueError("operands do not have the planned shapes")
        _check(lib.fm_int8_plan_run(ct.c_void_p(self._h), _dptr(Ac), _dptr(dA), _dptr(BTc),
                                    _dptr(dB), _dptr(out), _stream(stream)))
        return out
