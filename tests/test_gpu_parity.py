"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on
the same seeded inputs.

Bars (written into each check):
  * FP8 operand codes and scales: bit-exact.
  * Block products: relative Frobenius <= 1e-5 per product (the oracle's are
    the exact sums rounded once; the matrix cores accumulate in fp32).
  * Output C: relative Frobenius <= 1e-5 against the oracle's C.
  * Orbit errors: within 1% relative of the oracle's.
  * float64 reference: relative <= 1e-12.
Shapes cover several tiles and ragged tails (block sizes not multiples of
the 128 x 128 x 128 GEMM tile), every kernel family and the generic kernels.
"""
import sys

import numpy as np
import pytest

import oracle
from oracle import scheme_ops as so
from oracle import schemes as osch
import synthetic as sy
from bench import default_chunk

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU-only machines, never run
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2609_39816_amd import fm  # noqa: E402

DEV = torch.device("cuda:0")
FMT = {"e4m3": fm.E4M3, "e5m2": fm.E5M2}
OFMT = {"e4m3": oracle.E4M3, "e5m2": oracle.E5M2}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def gpu(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def bits(x):
    return np.ascontiguousarray(x, np.float32).view(np.uint32)


class OracleSchemes:
    """Oracle-side gauged schemes, built on first use (pure-Python float64)."""

    def __init__(self, w, gauges):
        self.w, self.gauges, self.cache = w, gauges, {}
        self.base = osch.BASE_SCHEMES[w.scheme]()
        self.flat = so.power(self.base, w.levels) if w.gauge_kind == "sign" else None

    def __getitem__(self, i):
        if i not in self.cache:
            P, Q, S = self.gauges[i]
            if self.w.gauge_kind == "sign":
                self.cache[i] = so.gauge(self.flat, P, Q, S)
            else:
                self.cache[i] = so.power(so.gauge(self.base, P, Q, S), self.w.levels)
        return self.cache[i]


def schemes_for(w, gauges):
    """(hip schemes, oracle schemes, levels passed to the library)."""
    base_h = fm.Scheme.base(w.scheme)
    if w.gauge_kind == "sign":
        flat_h = base_h.kron(w.levels) if w.levels > 1 else base_h
        hips = [flat_h.gauge(P, Q, S) for P, Q, S in gauges]
        return hips, OracleSchemes(w, gauges), 1
    hips = [base_h.gauge(P, Q, S) for P, Q, S in gauges]
    return hips, OracleSchemes(w, gauges), w.levels


def check_operands(h, o, levels, A, B, At, Bt, fmt):
    Tq, Sq, dT, dS = fm.form_operands(h, At, Bt, levels, FMT[fmt])
    tabs, dims = oracle.flatten_f32(o)
    U, V, W = tabs
    gm, gk, gn, R = dims
    tq, dt = oracle.form_operands(A, gm, gk, U, OFMT[fmt])
    sq, ds = oracle.form_operands(B, gk, gn, V, OFMT[fmt])
    assert np.array_equal(Tq.cpu().numpy(), tq), "Tq not bit-exact"
    assert np.array_equal(Sq.cpu().numpy(), sq.transpose(0, 2, 1)), "Sq not bit-exact"
    assert np.array_equal(dT.cpu().numpy().view(np.uint32), dt.view(np.uint32)), "dT not bit-exact"
    assert np.array_equal(dS.cpu().numpy().view(np.uint32), ds.view(np.uint32)), "dS not bit-exact"
    return Tq, Sq, dT, dS, tq, sq, dt, ds


def run_workload(w, n_oracle, fmt="e4m3", check_products=2):
    say(f"[parity] {w.name} fmt={fmt} G={w.G}")
    A, B = sy.operands(w)
    At, Bt = gpu(A), gpu(B)
    gauges = [sy.identity_gauge(w)] + sy.gauges(w)
    hips, orcs, levels = schemes_for(w, gauges)
    Cref_o = oracle.reference_f64(A, B)
    Cref = fm.reference_f64(At, Bt)
    assert rel(Cref.cpu().numpy(), Cref_o) <= 1e-12
    # classical baseline
    cl_h = fm.Scheme.base("classical")
    C_cl = fm.matmul_lowp(cl_h, At, Bt, 1, FMT[fmt])
    C_cl_o = oracle.lowp_matmul(A, B, *oracle.flatten_f32(osch.classical()), OFMT[fmt])
    assert rel(C_cl.cpu().numpy(), C_cl_o) <= 1e-5
    st = fm.error_stats(C_cl, Cref)
    e_o, r_o = oracle.error_sums(C_cl_o, Cref_o)
    err_cl_o = np.sqrt(e_o) / np.sqrt(r_o)
    assert abs(st["rel_fro"] / err_cl_o - 1) <= 1e-2
    assert abs(st["ref_sq"] / r_o - 1) <= 1e-12
    # orbit on the GPU, all gauges
    errs = fm.orbit_eval(hips, At, Bt, Cref, levels, FMT[fmt])
    assert np.all(np.isfinite(errs))
    picks = sorted(set([0, 1, len(hips) - 1] + list(range(0, len(hips), max(1, len(hips) // n_oracle)))))[:n_oracle]
    for gi in picks:
        h, o = hips[gi], orcs[gi]
        Tq, Sq, dT, dS, tq, sq, dt, ds = check_operands(h, o, levels, A, B, At, Bt, fmt)
        Mg = fm.block_products(Tq, Sq, dT, dS, FMT[fmt])
        # every block product of the first and the last picked gauge, the
        # first few of the others
        nprod = tq.shape[0] if gi in (picks[0], picks[-1]) else min(check_products, tq.shape[0])
        Mg_h = Mg.cpu().numpy()
        for r in range(nprod):
            Mo = oracle.block_product(tq[r], sq[r], dt[r], ds[r], OFMT[fmt])
            assert rel(Mg_h[r], Mo) <= 1e-5, f"gauge {gi}: block product {r}"
        tabs, dims = oracle.flatten_f32(o)
        Co = oracle.lowp_matmul(A, B, tabs, dims, OFMT[fmt])
        Cg = fm.matmul_lowp(h, At, Bt, levels, FMT[fmt]).cpu().numpy()
        assert rel(Cg, Co) <= 1e-5, f"gauge {gi}: C rel {rel(Cg, Co):.3e}"
        Cr = fm.reconstruct(h, Mg, w.M, w.N, levels).cpu().numpy()
        assert rel(Cr, Co) <= 1e-5
        e_want = oracle.rel_fro(Co, Cref_o)
        assert abs(errs[gi] / e_want - 1) <= 1e-2, f"gauge {gi}: {errs[gi]} vs {e_want}"
    return errs / st["rel_fro"]


# ----------------------------------------------------------------- codec
def structured_values(limit):
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], dtype=np.uint32)
    x = (hi[:, None] | lows[None, :]).reshape(-1).view(np.float32)
    return x[np.isfinite(x) & (np.abs(x) <= limit)]


@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
def test_fp8_encoder_bit_exact(fmt):
    """The kernels' encoder equals the oracle's on every fp32 high half with
    low halves on, above and below each rounding tie, up to the largest value
    the schedule can produce, FMAX (1 + 2^-23)^2."""
    fmax = 448.0 if fmt == "e4m3" else 57344.0
    x = structured_values(fmax * (1 + 2.0 ** -21))
    want = oracle.fp8_encode(x, OFMT[fmt])
    xg = gpu(x)
    for impl in (0, 2):
        got = fm.fp8_encode(xg, FMT[fmt], impl).cpu().numpy()
        bad = np.nonzero(got != want)[0]
        assert bad.size == 0, (impl, x[bad[:8]], got[bad[:8]], want[bad[:8]])


@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
def test_fp8_hardware_conversion_report(fmt):
    """Reports whether the gfx950 conversion instructions round like the
    oracle over the reachable range (they are used only if they do)."""
    fmax = 448.0 if fmt == "e4m3" else 57344.0
    x = structured_values(fmax * (1 + 2.0 ** -21))
    want = oracle.fp8_encode(x, OFMT[fmt])
    got = fm.fp8_encode(gpu(x), FMT[fmt], 1).cpu().numpy()
    bad = np.nonzero(got != want)[0]
    say(f"[codec] hardware {fmt}: {bad.size} of {x.size} differ; first: "
        f"{[(float(x[i]), int(got[i]), int(want[i])) for i in bad[:6]]}")


def test_bf16_rounding_bit_exact():
    """The group schedule's bf16 rounding on the device (the gfx950
    conversion the formation kernels use, and the integer rounding) equals
    the oracle's on every finite fp32 high half with low halves on, above and
    below each tie, subnormals included."""
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], dtype=np.uint32)
    x = (hi[:, None] | lows[None, :]).reshape(-1).view(np.float32)
    x = x[np.isfinite(oracle.bf16_round(x))]
    want = bits(oracle.bf16_round(x))
    xg = gpu(x)
    for impl in (0, 1, 2):
        got = bits(fm.bf16_round(xg, impl).cpu().numpy())
        bad = np.nonzero(got != want)[0]
        assert bad.size == 0, (impl, x[bad[:8]], got[bad[:8]], want[bad[:8]])


# ------------------------------------------------------------ workloads
def test_strassen1_gl64_full_workload():
    w = sy.WORKLOADS["strassen1_256_gl64"]
    ratios = run_workload(w, n_oracle=65)
    st = oracle.orbit_stats(ratios[1:], identity_value=ratios[0])
    say(f"[parity] {w.name} ratio stats {st}")
    assert st["max"] > st["min"] > 0


def test_strassen2_sign_orbit_scaled():
    w = sy.scaled(sy.WORKLOADS["strassen2_2048x4096x4096_sign512"], 256, 512, 512, G=512)
    ratios = run_workload(w, n_oracle=6)
    assert ratios.shape == (513,)


def test_laderman_gl_scaled_ragged_both_formats():
    # block sizes 48 x 64 x 80: every GEMM tile is ragged, K is shorter than one step
    w = sy.scaled(sy.WORKLOADS["laderman1_3072x4608x12288_gl512"], 144, 192, 240, G=8)
    for fmt in ("e4m3", "e5m2"):
        run_workload(w, n_oracle=3, fmt=fmt)


def test_strassen2_student_t_scaled():
    w = sy.scaled(sy.WORKLOADS["strassen2_4096x4096x14336_sign512"], 512, 256, 896, G=16)
    run_workload(w, n_oracle=3)


def test_strassen3_sampled_signs_scaled():
    w = sy.scaled(sy.WORKLOADS["strassen3_8192x27648x5120_sign512"], 256, 512, 384, G=8)
    run_workload(w, n_oracle=3, check_products=3)


def test_generic_kernels():
    """Schemes whose nonzero structure has no compiled kernel run on the
    generic formation and reconstruction kernels: a block permutation of
    two-level Strassen's 4 x 4 grid (exact coefficients), the plain 2 x 2 x 2
    product (E5M2), and a dense GL(4) gauge (operands and orbit errors only:
    its coefficients amplify fp32 rounding of the products by cond(P)cond(S))."""
    say("[parity] generic kernels")
    w = sy.scaled(sy.WORKLOADS["strassen2_2048x4096x4096_sign512"], 128, 256, 192, G=1)
    A, B = sy.operands(w)
    At, Bt = gpu(A), gpu(B)
    perm = np.eye(4)[[1, 0, 3, 2]]
    P, Q, S = perm, np.eye(4)[[2, 3, 0, 1]], np.eye(4)
    h = fm.Scheme.base("strassen").kron(2).gauge(P, Q, S)
    assert h.kernel_family(1) == "generic"
    o = so.gauge(so.power(osch.strassen(), 2), P, Q, S)
    check_operands(h, o, 1, A, B, At, Bt, "e4m3")
    Co = oracle.lowp_matmul(A, B, *oracle.flatten_f32(o))
    Cg = fm.matmul_lowp(h, At, Bt).cpu().numpy()
    assert rel(Cg, Co) <= 1e-5
    U, V, W, m, k, n = fm._schemes.classical(2, 2, 2)
    hc = fm.Scheme.load(U, V, W, m, k, n)
    assert hc.kernel_family(1) == "generic"
    oc = osch.classical(2, 2, 2)
    check_operands(hc, oc, 1, A, B, At, Bt, "e5m2")
    Co = oracle.lowp_matmul(A, B, *oracle.flatten_f32(oc), oracle.E5M2)
    assert rel(fm.matmul_lowp(hc, At, Bt, 1, fm.E5M2).cpu().numpy(), Co) <= 1e-5
    P, Q, S = sy.gl_gauges(4, 4, 4, 1, seed=77)[0]
    hg = fm.Scheme.base("strassen").kron(2).gauge(P, Q, S)
    og = so.gauge(so.power(osch.strassen(), 2), P, Q, S)
    assert hg.kernel_family(1) == "generic"
    check_operands(hg, og, 1, A, B, At, Bt, "e4m3")
    Cref = fm.reference_f64(At, Bt)
    e = fm.orbit_eval([hg, h], At, Bt, Cref)
    Cref_o = oracle.reference_f64(A, B)
    want = [oracle.rel_fro(oracle.lowp_matmul(A, B, *oracle.flatten_f32(x)), Cref_o) for x in (og, o)]
    assert np.all(np.abs(e / np.array(want) - 1) <= 1e-2)


def test_family_structure_with_unshared_coefficients():
    """Two-level Strassen with each product's A coefficients scaled by its
    own power of two (W scaled back): the family's nonzero structure, so the
    family kernels take it, but chains that share blocks no longer share
    coefficients, so the prefix-shared formation must not be used; codes and
    scales stay bit-exact and the output within 1e-5 of the oracle's."""
    say("[parity] family structure, unshared coefficients")
    w = sy.scaled(sy.WORKLOADS["strassen2_2048x4096x4096_sign512"], 256, 256, 256, G=1)
    A, B = sy.operands(w)
    At, Bt = gpu(A), gpu(B)
    U, V, W, m, k, n = fm._schemes.strassen()
    alpha = np.array([2.0, 0.5, 4.0, 1.0, 0.25, 8.0, 2.0])
    h = fm.Scheme.load(U * alpha[:, None], V, W / alpha[:, None], m, k, n).kron(2)
    assert h.kernel_family(1) == "Strassen2"
    base = osch.strassen()
    scaled = osch.Scheme(base.U * alpha[:, None], base.V, base.W / alpha[:, None], base.m, base.k,
                         base.n, base.R)
    o = so.power(scaled, 2)
    check_operands(h, o, 1, A, B, At, Bt, "e4m3")
    Co = oracle.lowp_matmul(A, B, *oracle.flatten_f32(o))
    assert rel(fm.matmul_lowp(h, At, Bt).cpu().numpy(), Co) <= 1e-5


def test_block_products_over_every_code():
    """Codes drawn uniformly from every finite FP8 value (subnormals, both
    signs, the largest values): the default arithmetic stays within 1e-6 of
    the exact sums rounded once; the FP8 matrix instructions are reported and
    bounded."""
    rng = np.random.default_rng(5)
    for fmt in ("e4m3", "e5m2"):
        vals = oracle.fp8_decode(np.arange(256, dtype=np.uint8), OFMT[fmt])
        finite = np.nonzero(np.isfinite(vals))[0].astype(np.uint8)
        Tq = rng.choice(finite, size=(3, 80, 256)).astype(np.uint8)
        Sq = rng.choice(finite, size=(3, 72, 256)).astype(np.uint8)
        dT = np.array([1.0, 0.5, 3.0], np.float32)
        dS = np.array([0.25, 1.0, 1.0 / 3.0], np.float32)
        want = np.stack([oracle.block_product(Tq[b], Sq[b].T, dT[b], dS[b], OFMT[fmt]) for b in range(3)])
        args = (gpu(Tq), gpu(Sq), gpu(dT), gpu(dS), FMT[fmt])
        got = fm.block_products(*args).cpu().numpy()
        r = rel(got, want)
        say(f"[parity] every-code products {fmt}: default rel {r:.2e}")
        assert r <= 1e-6
        fm.set_block_product_arithmetic(fm.ACC_FP8)
        try:
            r8 = rel(fm.block_products(*args).cpu().numpy(), want)
        finally:
            fm.set_block_product_arithmetic(fm.ACC_BF16)
        say(f"[parity] every-code products {fmt}: FP8 matrix instructions rel {r8:.2e}")
        assert r8 <= 1e-3


@pytest.mark.parametrize("batch,Mb,Nb,Kb", [
    (96, 300, 260, 384),   # ragged in both directions, several tiles per workgroup
    (70, 256, 128, 128),   # exactly one tile and one K step per product
    (9, 512, 256, 1024),   # interior tiles only, eight K steps
    (12, 200, 130, 256),   # a row length not a multiple of 4 (element stores)
    (5, 72, 80, 96),       # inner length not a multiple of 128
    # the wide-wave kernel (512 x 128 tiles, K steps of 64):
    (5, 512, 128, 64),     # one tile and one K step per product
    (40, 512, 128, 192),   # three K steps: a ring turn per tile; 40 tiles
    (7, 1536, 384, 128),   # 63 tiles (not a multiple of 8)
    (30, 1024, 640, 128),  # 300 tiles: several per workgroup
    (3, 1024, 640, 3456),  # the three-level projection shape's products
])
def test_block_products_tilings(batch, Mb, Nb, Kb):
    """Batched block products over tilings that exercise the persistent
    pipelined kernels (ring wrap-around, tile changes inside the ring, ragged
    edges) against the exact sums rounded once."""
    say(f"[parity] block products batch {batch} {Mb}x{Nb}x{Kb}")
    rng = np.random.default_rng(batch * 7 + Kb)
    vals = oracle.fp8_decode(np.arange(256, dtype=np.uint8), oracle.E4M3)
    finite = np.nonzero(np.isfinite(vals) & (np.abs(vals) <= 64))[0].astype(np.uint8)
    Tq = rng.choice(finite, size=(batch, Mb, Kb)).astype(np.uint8)
    Sq = rng.choice(finite, size=(batch, Nb, Kb)).astype(np.uint8)
    dT = (rng.random(batch) + 0.5).astype(np.float32)
    dS = (rng.random(batch) + 0.5).astype(np.float32)
    got = fm.block_products(gpu(Tq), gpu(Sq), gpu(dT), gpu(dS), fm.E4M3).cpu().numpy()
    for b in sorted({0, 1, batch // 2, batch - 1}):
        want = oracle.block_product(Tq[b], Sq[b].T, dT[b], dS[b], oracle.E4M3)
        assert rel(got[b], want) <= 1e-6, f"product {b}: rel {rel(got[b], want):.2e}"


def test_block_products_rowcol_scales_wide_tiles():
    """Per-row and per-column scales through the wide-wave kernel's epilogue
    (512 x 128 tiles) against the oracle's scaled exact sums."""
    rng = np.random.default_rng(17)
    vals = oracle.fp8_decode(np.arange(256, dtype=np.uint8), oracle.E4M3)
    finite = np.nonzero(np.isfinite(vals))[0].astype(np.uint8)
    batch, Mb, Nb, Kb = 4, 512, 256, 256
    Tq = rng.choice(finite, size=(batch, Mb, Kb)).astype(np.uint8)
    Sq = rng.choice(finite, size=(batch, Nb, Kb)).astype(np.uint8)
    dT = (rng.random((batch, Mb)) + 0.5).astype(np.float32)
    dS = (rng.random((batch, Nb)) + 0.5).astype(np.float32)
    got = fm.block_products(gpu(Tq), gpu(Sq), gpu(dT), gpu(dS), fm.E4M3,
                            scale_mode=fm.SCALE_ROWCOL).cpu().numpy()
    for b in range(batch):
        want = oracle.block_product_rc(Tq[b], Sq[b].T, dT[b], dS[b], oracle.E4M3)
        assert rel(got[b], want) <= 1e-6, f"product {b}: rel {rel(got[b], want):.2e}"


# ---------------------------------------------------------- edge cases
def test_zero_operand_and_single_tile():
    say("[parity] zero operand")
    A = np.zeros((64, 64), np.float32)
    B = np.random.default_rng(1).standard_normal((64, 64)).astype(np.float32)
    h = fm.Scheme.base("strassen")
    Tq, Sq, dT, dS = fm.form_operands(h, gpu(A), gpu(B))
    assert not Tq.cpu().numpy().any() and np.all(dT.cpu().numpy() == 1.0)
    C = fm.matmul_lowp(h, gpu(A), gpu(B)).cpu().numpy()
    assert not C.any()
    Cref = fm.reference_f64(gpu(A), gpu(B))
    errs = fm.orbit_eval([h], gpu(A), gpu(B), Cref)
    assert errs[0] == 0.0


def test_nonfinite_input_is_reported():
    say("[parity] non-finite input")
    rng = np.random.default_rng(2)
    A = rng.standard_normal((64, 64)).astype(np.float32)
    B = rng.standard_normal((64, 64)).astype(np.float32)
    A[5, 7] = np.inf
    h = fm.Scheme.base("strassen")
    Cref = fm.reference_f64(gpu(A), gpu(B))
    with pytest.raises(fm.FmError) as e:
        fm.orbit_eval([h], gpu(A), gpu(B), Cref)
    assert e.value.name == "FM_E_NONFINITE"
    ws = fm.workspace(fm.workspace_size(h, 64, 64, 64))
    fm.matmul_lowp(h, gpu(A), gpu(B), ws=ws)
    with pytest.raises(fm.FmError):
        fm.status(ws)
    fm.status(ws)  # cleared


def test_orbit_mixing_sign_variants_and_other_family_members():
    """Sign variants of two-level Strassen take the compile-time coefficient
    formation; a diagonal gauge with a non-unit entry has the same nonzero
    structure but is no sign variant, so a chunk holding it is formed by the
    generic kernels.  Every chunking gives the one-chunk bits, and both kinds
    of gauge match the oracle's errors."""
    say("[parity] sign variants beside other family members")
    w = sy.scaled(sy.WORKLOADS["strassen2_2048x4096x4096_sign512"], 256, 512, 256, G=5)
    A, B = sy.operands(w)
    At, Bt = gpu(A), gpu(B)
    gauges = sy.gauges(w)
    odd = (np.diag([2.0, 1.0, 1.0, -1.0]), np.diag([1.0, -1.0, 0.5, 1.0]), np.eye(4))
    gauges = gauges[:3] + [odd] + gauges[3:]
    hips, orcs, levels = schemes_for(w, gauges)
    assert hips[0].sign_variant(levels, 0)[0] and not hips[3].sign_variant(levels, 0)[0]
    Cref = fm.reference_f64(At, Bt)
    e1 = fm.orbit_eval(hips, At, Bt, Cref, levels)
    for ch in (1, 2, 4):
        ws = fm.workspace(fm.workspace_size(hips[0], w.M, w.N, w.K, levels, len(hips), ch))
        e2 = fm.orbit_eval(hips, At, Bt, Cref, levels, ws=ws)
        assert np.array_equal(e1.view(np.uint64), e2.view(np.uint64)), ch
    Cref_o = oracle.reference_f64(A, B)
    for gi in (2, 3, 4):
        check_operands(hips[gi], orcs[gi], levels, A, B, At, Bt, "e4m3")
        Co = oracle.lowp_matmul(A, B, *oracle.flatten_f32(orcs[gi]))
        assert abs(e1[gi] / oracle.rel_fro(Co, Cref_o) - 1) <= 1e-2, gi


def test_chunked_orbit_equals_single_launch_and_is_deterministic():
    say("[parity] chunking and determinism")
    w = sy.scaled(sy.WORKLOADS["strassen2_2048x4096x4096_sign512"], 256, 256, 256, G=24)
    A, B = sy.operands(w)
    At, Bt = gpu(A), gpu(B)
    hips, _, levels = schemes_for(w, sy.gauges(w))
    Cref = fm.reference_f64(At, Bt)
    e1 = fm.orbit_eval(hips, At, Bt, Cref, levels)
    e2 = fm.orbit_eval(hips, At, Bt, Cref, levels)
    assert np.array_equal(e1.view(np.uint64), e2.view(np.uint64))
    # chunks of 6 and 3 (halving 24) with two product buffers: the
    # reconstruction runs on the second stream and each buffer is reused;
    # a workspace sized for chunks of 5 takes chunks of 6 with one buffer,
    # one sized for 7 (not reached by halving) chunks of 6 with two
    for ch in (6, 3, 5, 7):
        ws = fm.workspace(fm.workspace_size(hips[0], w.M, w.N, w.K, levels, len(hips), ch))
        e3 = fm.orbit_eval(hips, At, Bt, Cref, levels, ws=ws)
        assert np.array_equal(e1.view(np.uint64), e3.view(np.uint64)), ch
    c1 = fm.matmul_lowp(hips[3], At, Bt, levels).cpu().numpy()
    c2 = fm.matmul_lowp(hips[3], At, Bt, levels).cpu().numpy()
    assert np.array_equal(c1.view(np.uint32), c2.view(np.uint32))
    # chunks whose kernel families differ (the identity's sparse Strassen
    # beside dense GL-gauged copies, and a chunk mixing both, formed by the
    # generic kernels): the codes of one chunk and the maxima of the next
    # are then formed in separate passes; same bits as one chunk
    wg = sy.scaled(sy.WORKLOADS["strassen1_256_gl64"], 192, 256, 160, G=11)
    A, B = sy.operands(wg)
    At, Bt = gpu(A), gpu(B)
    hips, _, levels = schemes_for(wg, [sy.identity_gauge(wg)] + sy.gauges(wg))
    Cref = fm.reference_f64(At, Bt)
    e1 = fm.orbit_eval(hips, At, Bt, Cref, levels)
    for ch in (1, 3):
        ws = fm.workspace(fm.workspace_size(hips[0], wg.M, wg.N, wg.K, levels, len(hips), ch))
        e3 = fm.orbit_eval(hips, At, Bt, Cref, levels, ws=ws)
        assert np.array_equal(e1.view(np.uint64), e3.view(np.uint64)), ch
    # blocks of whole 256 x 128 tiles: the orbit passes its products to the
    # reconstruction in the tiled layout; its errors equal those of the
    # stand-alone row-major path (the same output bits, sums in another order)
    # (blocks of 256 rows: 256 x 128 tiles; of 512 rows: the wide-wave
    # kernel's 512 x 128 tiles; three-level Strassen: one position per
    # thread of the reconstruction)
    for (name, M, K, N) in (("strassen1_256_gl64", 512, 512, 256),
                            ("strassen1_256_gl64", 1024, 256, 512),
                            ("strassen3_8192x27648x5120_sign512", 4096, 512, 1024)):
        wt = sy.scaled(sy.WORKLOADS[name], M, K, N, G=6 if name.startswith("strassen1") else 3)
        A, B = sy.operands(wt)
        At, Bt = gpu(A), gpu(B)
        hips, _, levels = schemes_for(wt, sy.gauges(wt))
        Cref = fm.reference_f64(At, Bt)
        for ch in (0, 2):
            ws = None if ch == 0 else fm.workspace(
                fm.workspace_size(hips[0], wt.M, wt.N, wt.K, levels, len(hips), ch))
            errs = fm.orbit_eval(hips, At, Bt, Cref, levels, ws=ws)
            for gi, h in enumerate(hips):
                st = fm.error_stats(fm.matmul_lowp(h, At, Bt, levels), Cref)
                assert abs(errs[gi] / st["rel_fro"] - 1) <= 1e-9, (name, M, ch, gi, errs[gi], st["rel_fro"])


def test_full_size_strassen2_workload_sampled():
    """Two-level Strassen at 2048 x 4096 x 4096, all 512 sign variants in the
    schedule the benchmark uses (32 gauges per launch at two levels, so
    gauges after the first chunk go through the second set of maxima, scales
    and product buffers and the two-stream overlap); the oracle checks the identity
    variant's operands bit for bit and the errors of three variants (first,
    a middle and the last chunk) from its whole output."""
    w = sy.WORKLOADS["strassen2_2048x4096x4096_sign512"]
    say(f"[parity] {w.name} full size")
    A, B = sy.operands(w)
    At, Bt = gpu(A), gpu(B)
    gauges = sy.gauges(w)
    hips, orcs, levels = schemes_for(w, gauges)
    Cref = fm.reference_f64(At, Bt)
    errs = fm.orbit_eval(hips, At, Bt, Cref, levels, chunk=default_chunk(w))
    check_operands(hips[0], orcs[0], levels, A, B, At, Bt, "e4m3")
    Cref_o = oracle.reference_f64(A, B)
    for gi in (0, 137, 511):
        Co = oracle.lowp_matmul(A, B, *oracle.flatten_f32(orcs[gi]))
        e_want = oracle.rel_fro(Co, Cref_o)
        say(f"[parity] gauge {gi}: gpu {errs[gi]:.6e} oracle {e_want:.6e}")
        assert abs(errs[gi] / e_want - 1) <= 1e-2


FULL_SIZE = [("laderman1_3072x4608x12288_gl512", "e4m3"), ("laderman1_3072x4608x12288_gl512", "e5m2"),
             ("strassen2_4096x4096x14336_sign512", "e4m3"),
             ("strassen3_8192x27648x5120_sign512", "e4m3")]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,fmt", FULL_SIZE)
def test_full_size_workloads_sampled(name, fmt):
    """The other full-size workloads (the last is the benchmark's headline),
    every gauge of the orbit in the launch configuration the benchmark times
    (`bench.default_chunk`: 16 gauges per launch at three levels, 32
    otherwise; two sets of buffers, two streams).  For gauge 1
    (first chunk) and the last gauge (last chunk) the oracle checks the
    operands bit for bit over the whole tensors and the output at sampled
    positions of every output block (the block products at those positions,
    then the reconstruction); the orbit's error of each must equal the error
    of the stand-alone output against the same reference.  For the last
    gauge the orbit error is also checked against the oracle's error of its
    whole output against the oracle's own float64 reference (within 1%).
    The float64 reference is checked at sampled entries."""
    w = sy.WORKLOADS[name]
    say(f"[parity] {name} fmt={fmt} full size")
    A, B = sy.operands(w)
    At, Bt = gpu(A), gpu(B)
    gauges = sy.gauges(w)
    hips, orcs, levels = schemes_for(w, gauges)
    Cref = fm.reference_f64(At, Bt)
    errs = fm.orbit_eval(hips, At, Bt, Cref, levels, FMT[fmt], chunk=default_chunk(w))
    assert errs.shape == (w.G,) and np.all(np.isfinite(errs)) and np.all(errs > 0)
    say(f"[parity] orbit done: errors {errs.min():.4e} .. {errs.max():.4e}")

    ri, rj = sy.ratio_sample_positions(w.M, w.N, 48, seed=11)
    want = np.array([oracle.reference_f64_at(A, B, int(i), int(j)) for i, j in zip(ri, rj)])
    got = Cref[torch.from_numpy(ri).to(DEV), torch.from_numpy(rj).to(DEV)].cpu().numpy()
    assert rel(got, want) <= 1e-12

    last = w.G - 1
    for gi in (1, last):
        _, _, _, _, tq, sq, dt, ds = check_operands(hips[gi], orcs[gi], levels, A, B, At, Bt, fmt)
        say(f"[parity] gauge {gi}: operands bit-exact")
        tabs, dims = oracle.flatten_f32(orcs[gi])
        gm, gk, gn, R = dims
        Mb, Nb = w.M // gm, w.N // gn
        rng = np.random.default_rng(5 + gi)
        xs, zs = rng.integers(0, Mb, 24), rng.integers(0, Nb, 24)
        C_o = oracle.lowp_matmul_at(tq, dt, sq, ds, tabs[2], gm, gn, xs, zs, OFMT[fmt])
        del tq, sq
        C = fm.matmul_lowp(hips[gi], At, Bt, levels, FMT[fmt])
        rows = (np.arange(gm)[:, None, None] * Mb + xs[None, None, :]).repeat(gn, 1)
        cols = (np.arange(gn)[None, :, None] * Nb + zs[None, None, :]).repeat(gm, 0)
        C_s = C[torch.from_numpy(rows.ravel()).to(DEV), torch.from_numpy(cols.ravel()).to(DEV)]
        r_c = rel(C_s.cpu().numpy(), C_o.ravel())
        st = fm.error_stats(C, Cref)
        del C
        say(f"[parity] gauge {gi}: sampled C rel {r_c:.3e}; orbit error {errs[gi]:.6e}, "
            f"stand-alone {st['rel_fro']:.6e}")
        assert r_c <= 1e-5
        assert abs(errs[gi] / st["rel_fro"] - 1) <= 1e-6

    say(f"[parity] gauge {last}: the oracle's whole output and float64 reference")
    Co = oracle.lowp_matmul(A, B, *oracle.flatten_f32(orcs[last]), OFMT[fmt])
    Cref_o = oracle.reference_f64(A, B)
    e_want = oracle.rel_fro(Co, Cref_o)
    say(f"[parity] gauge {last}: orbit {errs[last]:.6e} oracle {e_want:.6e}")
    assert abs(errs[last] / e_want - 1) <= 1e-2
