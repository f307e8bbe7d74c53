"""Pins of the oracle's arithmetic: the FP8 codec, block sums, scales, block
products, reconstruction, and the whole schedule on tiny inputs.

References used here are independent of the oracle's code: nearest-code
search over every FP8 value, torch's own FP8 casts, exact rational
arithmetic (fractions.Fraction) for products and fused multiply-adds,
numpy's float64 matmul where the sum it forms is exact, and closed forms.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import scheme_ops as so
from oracle import schemes
import synthetic as sy

E4M3, E5M2 = oracle.E4M3, oracle.E5M2


# ---------------------------------------------------------------------------
# Independent FP8 reference: nearest representable value by search.
# ---------------------------------------------------------------------------
def _fp8_value_table(fmt):
    """Positive finite FP8 values indexed by code, from the format's layout
    (OCP E4M3FN: bias 7, no infinities, S.1111.111 is NaN; E5M2: bias 15,
    exponent 31 is inf/NaN)."""
    eb, mb, bias = (4, 3, 7) if fmt == E4M3 else (5, 2, 15)
    vals = {}
    for code in range(128):
        e, m = code >> mb, code & ((1 << mb) - 1)
        if fmt == E4M3 and e == 15 and m == 7:
            continue
        if fmt == E5M2 and e == 31:
            continue
        if e == 0:
            v = Fraction(m, 1 << mb) * Fraction(2) ** (1 - bias)
        else:
            v = (1 + Fraction(m, 1 << mb)) * Fraction(2) ** (e - bias)
        vals[code] = v
    return vals


def nearest_code(x: float, fmt) -> int:
    """Nearest finite code to fp32 x; ties to the even code; beyond the
    largest finite value, the largest finite value."""
    table = _nearest_cache(fmt)
    codes, values = table
    a = abs(Fraction(float(x)))
    sign = 0x80 if np.signbit(x) else 0
    idx = np.searchsorted(values, float(a))  # values exact in float64
    if idx >= len(values):
        return sign | codes[-1]
    if idx == 0:
        return sign | codes[0]
    lo, hi = Fraction(values[idx - 1]), Fraction(values[idx])
    if a == hi:
        return sign | codes[idx]
    dlo, dhi = a - lo, hi - a
    if dlo < dhi:
        c = codes[idx - 1]
    elif dhi < dlo:
        c = codes[idx]
    else:
        c = codes[idx - 1] if codes[idx - 1] % 2 == 0 else codes[idx]
    return sign | c


_NC = {}


def _nearest_cache(fmt):
    if fmt not in _NC:
        vals = _fp8_value_table(fmt)
        codes = sorted(vals, key=lambda c: vals[c])
        _NC[fmt] = (codes, np.array([float(vals[c]) for c in codes]))
    return _NC[fmt]


def structured_f32_values():
    """Every fp32 high half (sign, exponent, top 7 mantissa bits) with low
    halves that sit on, just above and just below every FP8 rounding tie."""
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], dtype=np.uint32)
    bits = (hi[:, None] | lows[None, :]).reshape(-1)
    x = bits.view(np.float32)
    return x[np.isfinite(x)]


@pytest.mark.parametrize("fmt", [E4M3, E5M2])
def test_encoder_matches_nearest_code_search(fmt):
    x = structured_f32_values()
    got = oracle.fp8_encode(x, fmt)
    # vectorized nearest search over the sorted positive values
    codes, values = _nearest_cache(fmt)
    codes = np.array(codes)
    a = np.abs(x.astype(np.float64))
    idx = np.clip(np.searchsorted(values, a), 1, len(values) - 1)
    lo, hi = values[idx - 1], values[idx]
    twice = 2.0 * a  # exact; lo + hi exact too
    mid = lo + hi
    pick_hi = (twice > mid) | ((twice == mid) & (codes[idx - 1] % 2 == 1))
    c = np.where(pick_hi, codes[idx], codes[idx - 1])
    c = np.where(a >= values[-1], codes[-1], c)
    c = np.where(a <= values[0], codes[0], c)
    want = (c | np.where(np.signbit(x), 0x80, 0)).astype(np.uint8)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, (x[bad[:5]], got[bad[:5]], want[bad[:5]])
    # spot-check the vectorized reference against the scalar search
    for v in x[:: 9973]:
        assert nearest_code(v, fmt) == oracle.fp8_encode(v, fmt)[0]


@pytest.mark.parametrize("fmt,dtype,limit", [(E4M3, "float8_e4m3fn", 448.0),
                                              (E5M2, "float8_e5m2", 57344.0)])
def test_encoder_matches_torch_cast_in_range(fmt, dtype, limit):
    torch = pytest.importorskip("torch")
    x = structured_f32_values()
    x = x[np.abs(x) <= limit]
    got = oracle.fp8_encode(x, fmt)
    t = torch.from_numpy(x.copy()).to(getattr(torch, dtype)).view(torch.uint8).numpy()
    assert np.array_equal(got, t)


def test_format_constants():
    assert oracle.fp8_max(E4M3) == 448.0
    assert oracle.fp8_max(E5M2) == 57344.0
    assert oracle.fp8_decode([0x01], E4M3)[0] == 2.0 ** -9
    assert oracle.fp8_decode([0x01], E5M2)[0] == 2.0 ** -16
    assert np.isnan(oracle.fp8_decode([0x7F], E4M3)[0])
    assert oracle.fp8_decode([0x7C], E5M2)[0] == np.inf
    # round trip of every finite code
    for fmt in (E4M3, E5M2):
        codes = np.arange(256, dtype=np.uint8)
        v = oracle.fp8_decode(codes, fmt)
        ok = np.isfinite(v)
        back = oracle.fp8_encode(v[ok].astype(np.float32), fmt)
        assert np.array_equal(back, codes[ok])


def test_e4m3_uniform_codebook_bound(golden):
    """App. D: a dense uniform codebook on e4m3 whose sums of L = 4 codes stay
    representable has J <= floor(2^4 / 4) = 4: every integer up to 16 is an
    e4m3 value, 17 is not."""
    J = golden["e4m3_uniform_codebook_J"]["value"]
    assert J == 2 ** 4 // 4
    ints = np.arange(-4 * J, 4 * J + 1).astype(np.float32)
    assert np.array_equal(oracle.fp8_decode(oracle.fp8_encode(ints)), ints)
    assert oracle.fp8_decode(oracle.fp8_encode(np.float32(4 * J + 1)))[0] != 4 * J + 1


# ---------------------------------------------------------------------------
# Exact rational helpers: correctly rounded fp32 and fused multiply-add.
# ---------------------------------------------------------------------------
def round_to_f32(q: Fraction, neg_zero=False) -> np.float32:
    """Round a rational to the nearest fp32 (ties to even), subnormals kept."""
    if q == 0:
        return np.float32(-0.0) if neg_zero else np.float32(0.0)
    sign = -1 if q < 0 else 1
    a = abs(q)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)
    quantum = Fraction(2) ** (e - 23)
    n = a / quantum
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    v = float(fl * quantum)
    return np.float32(sign * v)


def fmaf_exact(a, b, c) -> np.float32:
    a, b, c = np.float32(a), np.float32(b), np.float32(c)
    q = Fraction(float(a)) * Fraction(float(b)) + Fraction(float(c))
    prod_neg = (np.signbit(a) != np.signbit(b))
    both_neg_zero = q == 0 and prod_neg and np.signbit(c)
    return round_to_f32(q, neg_zero=both_neg_zero)


def test_round_to_f32_helper_matches_numpy():
    rng = np.random.default_rng(0)
    for v in rng.standard_normal(200) * 10.0 ** rng.integers(-40, 30, 200):
        assert round_to_f32(Fraction(float(v))) == np.float32(v)


# ---------------------------------------------------------------------------
# Block products and the whole schedule against exact arithmetic.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("fmt", [E4M3, E5M2])
def test_block_product_is_exact_sum_rounded_once(fmt):
    rng = np.random.default_rng(3)
    finite = [c for c in range(256) if np.isfinite(oracle.fp8_decode([c], fmt)[0])]
    Tq = rng.choice(finite, size=(3, 37)).astype(np.uint8)
    Sq = rng.choice(finite, size=(37, 5)).astype(np.uint8)
    dT, dS = np.float32(0.37), np.float32(1.9e-3)
    got = oracle.block_product(Tq, Sq, dT, dS, fmt)
    vt = oracle.fp8_decode(Tq, fmt)
    vs = oracle.fp8_decode(Sq, fmt)
    for x in range(3):
        for z in range(5):
            q = sum(Fraction(float(vt[x, y])) * Fraction(float(vs[y, z])) for y in range(37))
            m = round_to_f32(q)
            m = np.float32(m * dT)
            m = np.float32(m * dS)
            assert got[x, z].view(np.uint32) == m.view(np.uint32)
    at = oracle.block_product_at(Tq, Sq, dT, dS, [0, 2, 1], [4, 0, 3], fmt)
    assert np.array_equal(at, got[[0, 2, 1], [4, 0, 3]])


def test_block_product_equals_library_matmul_of_decoded_codes():
    """For E4M3 every partial sum is a multiple of 2^-18 below 2^36, so a
    float64 matmul (any summation order) forms the same exact sum."""
    rng = np.random.default_rng(4)
    A = rng.standard_normal((64, 256)).astype(np.float32)
    B = rng.standard_normal((256, 48)).astype(np.float32)
    qa, da, _ = oracle.quantize_tensor(A)
    qb, db, _ = oracle.quantize_tensor(B)
    exact = oracle.fp8_decode(qa) @ oracle.fp8_decode(qb)
    want = ((exact.astype(np.float32) * da).astype(np.float32) * db).astype(np.float32)
    got = oracle.block_product(qa, qb, da, db)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def brute_force_schedule(A, B, U, V, W, dims, fmt, rowcol=False):
    """The whole FP8 schedule in exact rationals, written independently:
    ascending row-major fmaf block sums from +0, tensor amax (or, with
    rowcol, the amax of each row of A's block sums and of each column of
    B's, App. B.1), correctly rounded scales, nearest-code rounding, exact
    block products rounded once and scaled by two fp32 multiplications,
    fmaf reconstruction."""
    gm, gk, gn, R = dims
    M, K = A.shape
    N = B.shape[1]
    br, bk, bc = M // gm, K // gk, N // gn
    fmax = Fraction(448 if fmt == E4M3 else 57344)
    codes_val = {c: Fraction(float(v)) for c, v in enumerate(oracle.fp8_decode(np.arange(256, dtype=np.uint8), fmt)) if np.isfinite(v)}

    def scale(values):
        amax = max(abs(Fraction(float(t))) for t in values)
        if amax == 0:
            return np.float32(1), np.float32(1)
        return round_to_f32(fmax / amax), round_to_f32(amax / fmax)

    def form(X, gr, gc, coef, rows, cols, per=None):
        # per: None (one scale), "row" or "col"
        T = np.zeros((rows, cols), np.float32)
        for x in range(rows):
            for y in range(cols):
                acc = np.float32(0.0)
                for p in range(gr):
                    for q in range(gc):
                        u = np.float32(coef[p * gc + q])
                        if u == 0:
                            continue
                        acc = fmaf_exact(u, X[p * rows + x, q * cols + y], acc)
                T[x, y] = acc
        if per is None:
            r, d = scale(T.reshape(-1))
            R_ = np.full((rows, cols), r, np.float32)
        elif per == "row":
            rd = [scale(T[x]) for x in range(rows)]
            R_ = np.array([[rd[x][0]] * cols for x in range(rows)], np.float32)
            d = np.array([rd[x][1] for x in range(rows)], np.float32)
        else:
            rd = [scale(T[:, y]) for y in range(cols)]
            R_ = np.array([[rd[y][0] for y in range(cols)] for _ in range(rows)], np.float32)
            d = np.array([rd[y][1] for y in range(cols)], np.float32)
        Q = np.zeros((rows, cols), np.uint8)
        for x in range(rows):
            for y in range(cols):
                Q[x, y] = nearest_code(np.float32(T[x, y] * R_[x, y]), fmt)
        return Q, d

    Mr = []
    Tqs, Sqs, dTs, dSs = [], [], [], []
    for r in range(R):
        Tq, dT = form(A, gm, gk, U[r], br, bk, "row" if rowcol else None)
        Sq, dS = form(B, gk, gn, V[r], bk, bc, "col" if rowcol else None)
        P = np.zeros((br, bc), np.float32)
        for x in range(br):
            for z in range(bc):
                q = sum(codes_val[int(Tq[x, y])] * codes_val[int(Sq[y, z])] for y in range(bk))
                m = round_to_f32(q)
                st = dT[x] if rowcol else dT
                ss = dS[z] if rowcol else dS
                P[x, z] = np.float32(np.float32(m * st) * ss)
        Mr.append(P)
        Tqs.append(Tq), Sqs.append(Sq), dTs.append(dT), dSs.append(dS)
    C = np.zeros((M, N), np.float32)
    for i in range(gm):
        for j in range(gn):
            for x in range(br):
                for z in range(bc):
                    acc = np.float32(0.0)
                    for r in range(R):
                        w = np.float32(W[r, i * gn + j])
                        if w == 0:
                            continue
                        acc = fmaf_exact(w, Mr[r][x, z], acc)
                    C[i * br + x, j * bc + z] = acc
    return dict(C=C, Tq=np.array(Tqs), Sq=np.array(Sqs), dT=np.array(dTs), dS=np.array(dSs),
                Mr=np.array(Mr))


@pytest.mark.parametrize("fmt", [E4M3, E5M2])
@pytest.mark.parametrize("which", ["identity", "gl"])
def test_whole_schedule_matches_exact_brute_force(fmt, which):
    rng = np.random.default_rng(11)
    A = rng.standard_normal((4, 6)).astype(np.float32)
    B = rng.standard_normal((6, 4)).astype(np.float32)
    s = schemes.strassen()
    if which == "gl":
        P, Q, S = sy.gl_gauges(2, 2, 2, 1, seed=5)[0]
        s = so.gauge(s, P, Q, S)
    tabs, dims = oracle.flatten_f32(s)
    got = oracle.lowp_matmul(A, B, tabs, dims, fmt, keep=True)
    want = brute_force_schedule(A, B, *tabs, dims, fmt)
    for key in ("Tq", "Sq"):
        assert np.array_equal(got[key], want[key]), key
    for key in ("dT", "dS", "Mr", "C"):
        assert np.array_equal(np.asarray(got[key]).view(np.uint32),
                              np.asarray(want[key], np.float32).view(np.uint32)), key


@pytest.mark.parametrize("fmt", [E4M3, E5M2])
@pytest.mark.parametrize("which", ["identity", "gl"])
def test_row_column_scales_match_exact_brute_force(fmt, which):
    """App. B.1's finer granularity (a scale per row of A's block sums and
    per column of B's) against the exact-rational schedule."""
    rng = np.random.default_rng(12)
    A = rng.standard_normal((4, 6)).astype(np.float32)
    B = rng.standard_normal((6, 8)).astype(np.float32)
    A[1] *= 300.0  # rows of very different magnitude
    s = schemes.strassen()
    if which == "gl":
        P, Q, S = sy.gl_gauges(2, 2, 2, 1, seed=6)[0]
        s = so.gauge(s, P, Q, S)
    tabs, dims = oracle.flatten_f32(s)
    got = oracle.lowp_matmul(A, B, tabs, dims, fmt, keep=True, scale_mode=oracle.SCALE_ROWCOL)
    want = brute_force_schedule(A, B, *tabs, dims, fmt, rowcol=True)
    assert got["dT"].shape == (7, 2) and got["dS"].shape == (7, 4)
    for key in ("Tq", "Sq"):
        assert np.array_equal(got[key], want[key]), key
    for key in ("dT", "dS", "Mr", "C"):
        assert np.array_equal(np.asarray(got[key]).view(np.uint32),
                              np.asarray(want[key], np.float32).view(np.uint32)), key


def test_one_by_one_blocks_reduce_to_fp32_strassen():
    """With 1x1 blocks every block sum is a single number, which quantizes to
    +-FMAX exactly, so the FP8 schedule equals Strassen evaluated in fp32 up
    to a few roundings: C = AB to ~1e-6 relative to |A||B|."""
    rng = np.random.default_rng(2)
    for _ in range(20):
        A = rng.standard_normal((2, 2)).astype(np.float32)
        B = rng.standard_normal((2, 2)).astype(np.float32)
        for s in (schemes.strassen(), so.gauge(schemes.strassen(), *sy.gl_gauges(2, 2, 2, 1, int(rng.integers(1 << 30)))[0])):
            tabs, dims = oracle.flatten_f32(s)
            out = oracle.lowp_matmul(A, B, tabs, dims, keep=True)
            assert set(np.unique(out["Tq"] & 0x7F)) <= {0x00, 0x7E}
            exact = A.astype(np.float64) @ B.astype(np.float64)
            scale = np.abs(A).astype(np.float64) @ np.abs(B).astype(np.float64)
            cond = float(np.abs(s.U).sum() * np.abs(s.V).sum() * np.abs(s.W).sum())
            assert np.all(np.abs(out["C"] - exact) <= 1e-6 * cond * scale.max())


def test_negating_a_negates_codes_and_keeps_scales():
    rng = np.random.default_rng(8)
    A = rng.standard_normal((16, 32)).astype(np.float32)
    s2 = so.power(schemes.strassen(), 2)
    q1, d1 = oracle.form_operands(A, 4, 4, s2.U.astype(np.float32))
    q2, d2 = oracle.form_operands(-A, 4, 4, s2.U.astype(np.float32))
    assert np.array_equal(d1, d2)
    nz = q1 != 0
    assert np.array_equal(q2[nz], q1[nz] ^ 0x80)
    assert np.all(q2[~nz] == 0)


def test_power_of_two_scaling_leaves_codes_unchanged():
    rng = np.random.default_rng(9)
    A = rng.standard_normal((16, 32)).astype(np.float32)
    s = schemes.strassen()
    q1, d1 = oracle.form_operands(A, 2, 2, s.U.astype(np.float32))
    q2, d2 = oracle.form_operands(A * np.float32(2.0 ** -7), 2, 2, s.U.astype(np.float32))
    assert np.array_equal(q1, q2)
    assert np.array_equal(d2, d1 * np.float32(2.0 ** -7))


def test_all_zero_tensor_has_unit_scale():
    codes, d, r = oracle.quantize_tensor(np.zeros((4, 4), np.float32))
    assert d == 1.0 and r == 1.0 and not codes.any()


def test_block_sum_visits_blocks_in_row_major_order():
    """Order matters for fp32 fmaf chains: with values chosen so that each
    partial sum rounds, the row-major order gives a result the reversed
    order does not."""
    X = np.zeros((2, 2), np.float32)
    X[0, 0], X[0, 1], X[1, 0] = 1.0, np.float32(2.0 ** -24), np.float32(2.0 ** -24)
    c = np.array([1, 1, 1, 0], np.float32)
    t = oracle.block_sum(X, 2, 2, c)[0, 0]
    ordered = fmaf_exact(1, X[1, 0], fmaf_exact(1, X[0, 1], fmaf_exact(1, X[0, 0], 0)))
    reverse = fmaf_exact(1, X[0, 0], fmaf_exact(1, X[0, 1], fmaf_exact(1, X[1, 0], 0)))
    assert t == ordered and ordered != reverse


def test_classical_error_matches_operand_rounding_errors():
    """Classical FP8: C - AB ~ E_A B + A E_B with independent rounding errors,
    so rel_fro ~ sqrt(dA^2 + dB^2), where dA = ||deq(A) - A|| / ||A||.  The
    operand errors come from the independent nearest-code search."""
    rng = np.random.default_rng(12)
    A = rng.standard_normal((128, 256)).astype(np.float32)
    B = rng.standard_normal((256, 96)).astype(np.float32)
    Cref = oracle.reference_f64(A, B)
    err = oracle.rel_fro(oracle.classical_fp8(A, B), Cref)
    codes, values = _nearest_cache(E4M3)

    def rel_round_err(X):
        s = 448.0 / np.abs(X).max()
        y = (X * np.float32(s)).astype(np.float32).reshape(-1)
        vals = np.array([float(oracle.fp8_decode([nearest_code(v, E4M3)])[0]) for v in y])
        return np.linalg.norm(vals / s - X.reshape(-1)) / np.linalg.norm(X)

    dA, dB = rel_round_err(A), rel_round_err(B)
    assert abs(err / np.hypot(dA, dB) - 1.0) < 0.05
    assert 0.03 < err < 0.045


def test_reference_is_float64_product():
    rng = np.random.default_rng(13)
    A = rng.integers(-50, 50, size=(7, 9)).astype(np.float32)
    B = rng.integers(-50, 50, size=(9, 5)).astype(np.float32)
    assert np.array_equal(oracle.reference_f64(A, B), A.astype(np.int64) @ B.astype(np.int64))
    assert oracle.reference_f64_at(A, B, 3, 2) == float(A.astype(np.int64)[3] @ B.astype(np.int64)[:, 2])


def test_error_sums_and_stats_conventions():
    C = np.array([[1.0, 2.0]], np.float32)
    Cref = np.array([[1.5, 2.0]])
    e, r = oracle.error_sums(C, Cref)
    assert e == 0.25 and r == 1.5 ** 2 + 4.0
    st = oracle.orbit_stats([4.0, 1.0, 3.0, 2.0], identity_value=3.0)
    assert st["median"] == 3.0  # upper of the two middle values
    assert st["spread"] == 4.0 and st["n_above_2"] == 2 and st["count"] == 4


def test_levels_equal_kron_power_bit_for_bit():
    """Evaluating two-level Strassen is evaluating the flattened 4x4x4 scheme:
    the oracle sees only flattened tables, and the flattening is exact."""
    s2 = so.power(schemes.strassen(), 2)
    s2b = so.kron(schemes.strassen(), schemes.strassen())
    for a, b in ((s2.U, s2b.U), (s2.V, s2b.V), (s2.W, s2b.W)):
        assert np.array_equal(a, b)


def test_sampled_outputs_equal_whole_schedule():
    """The sampled form used at full size gives the whole-output schedule's
    bits at every sampled position, for a GL-gauged two-level Strassen with
    ragged in-block positions."""
    w = sy.scaled(sy.WORKLOADS["strassen1_256_gl64"], 48, 80, 64, G=2)
    A, B = sy.operands(w)
    P, Q, S = sy.gauges(w)[1]
    tabs, dims = oracle.flatten_f32(so.power(so.gauge(schemes.strassen(), P, Q, S), 2))
    U, V, W = tabs
    gm, gk, gn, R = dims
    for fmt in (E4M3, E5M2):
        full = oracle.lowp_matmul(A, B, tabs, dims, fmt, keep=True)
        tq, dt = oracle.form_operands(A, gm, gk, U, fmt)
        sq, ds = oracle.form_operands(B, gk, gn, V, fmt)
        assert np.array_equal(tq, full["Tq"]) and np.array_equal(sq, full["Sq"])
        Mb, Nb = A.shape[0] // gm, B.shape[1] // gn
        xs, zs = np.meshgrid(np.arange(Mb), np.arange(Nb), indexing="ij")
        got = oracle.lowp_matmul_at(tq, dt, sq, ds, W, gm, gn, xs.ravel(), zs.ravel(), fmt)
        want = full["C"].reshape(gm, Mb, gn, Nb).transpose(0, 2, 1, 3).reshape(gm, gn, -1)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
