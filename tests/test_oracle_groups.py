"""Pins of the group-scale granularity on the CPU oracle (App. B.1: the
models' schedule rounds the block sums of a layer's input to e4m3 with one
scale for every 128 consecutive entries of a row, those of its weight, first
stored in bf16, with one scale for every 128 x 128 block; the products come
back in bf16 and are combined in fp32).

What pins it:
  * the bf16 rounding against torch's bfloat16 cast (a library routine) on
    random values, exact ties and the largest finite values;
  * the whole schedule against an independent computation: block sums in
    float32 arithmetic (coefficients +-1), scales as correctly rounded
    rationals, codes by nearest-value search, bf16 by torch, every group's
    exact sum as a rational rounded once, fused multiply-adds in exact
    rationals, reconstruction the same way -- codes, scales, products and C
    bit for bit;
  * the fp32 accumulation rule itself (before the bf16 rounding, which
    would hide a changed rule) against exact rationals;
  * structure: with one group per block-sum row, A's group scales are the
    per-row scales; every product is a bf16 value; App. C.3's row map and
    Sec. 4.2's 48 of 496 pairs hold as under the per-row form; a power of two
    on the rows at one block offset scales exactly those output rows.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import scheme_ops as so
from oracle import schemes

from test_oracle_numerics import fmaf_exact, nearest_code, round_to_f32

torch = pytest.importorskip("torch")
E4M3 = oracle.E4M3
GRP = oracle.GROUP
SG = oracle.SCALE_GROUP


def bf16_torch(x):
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).float().numpy()


def bits(x):
    return np.ascontiguousarray(x, np.float32).view(np.uint32)


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(4000) * 10.0 ** rng.integers(-30, 30, 4000)).astype(np.float32)
    # exact ties between bf16 neighbours, both parities, and the top of the range
    base = rng.integers(0, 1 << 15, 200, dtype=np.uint32) << 16
    ties = (base | 0x8000).view(np.float32)
    top = np.array([3.3895314e38, 3.38e38, -3.3895314e38, 1e-40, -1e-45], np.float32)
    for v in (x, ties, top):
        v = v[np.isfinite(v)]
        assert np.array_equal(bits(oracle.bf16_round(v)), bits(bf16_torch(v)))


def independent_group_schedule(A, B, U, V, W, dims):
    """The group-scale schedule written independently of the oracle."""
    gm, gk, gn, R = dims
    M, K = A.shape
    N = B.shape[1]
    br, bk, bc = M // gm, K // gk, N // gn
    fmax = Fraction(448)
    vals = {c: Fraction(float(v)) for c, v in
            enumerate(oracle.fp8_decode(np.arange(256, dtype=np.uint8), E4M3)) if np.isfinite(v)}

    def block_sum(X, gr, gc, coef, rows, cols):
        assert set(np.unique(coef)) <= {-1.0, 0.0, 1.0}
        T = np.zeros((rows, cols), np.float32)
        for p in range(gr):
            for q in range(gc):
                u = coef[p * gc + q]
                if u != 0:  # fmaf(+-1, x, acc) is the rounded sum acc +- x
                    T = (T + np.float32(u) * X[p * rows:(p + 1) * rows, q * cols:(q + 1) * cols]
                         ).astype(np.float32)
        return T

    def scale(values):
        amax = max(abs(Fraction(float(t))) for t in values.reshape(-1))
        if amax == 0:
            return np.float32(1), np.float32(1)
        return round_to_f32(fmax / amax), round_to_f32(amax / fmax)

    Mr, Tqs, Sqs, dTs, dSs = [], [], [], [], []
    for r in range(R):
        T = block_sum(A, gm, gk, U[r], br, bk)
        Tq = np.zeros((br, bk), np.uint8)
        dT = np.zeros((bk // GRP, br), np.float32)
        for x in range(br):
            for kg in range(bk // GRP):
                seg = T[x, kg * GRP:(kg + 1) * GRP]
                q, d = scale(seg)
                dT[kg, x] = d
                for y in range(GRP):
                    Tq[x, kg * GRP + y] = nearest_code(np.float32(seg[y] * q), E4M3)
        S = bf16_torch(block_sum(B, gk, gn, V[r], bk, bc))
        Sq = np.zeros((bk, bc), np.uint8)
        dS = np.zeros((bk // GRP, bc // GRP), np.float32)
        for kg in range(bk // GRP):
            for zb in range(bc // GRP):
                blk = S[kg * GRP:(kg + 1) * GRP, zb * GRP:(zb + 1) * GRP]
                q, d = scale(blk)
                dS[kg, zb] = d
                for y in range(GRP):
                    for z in range(GRP):
                        Sq[kg * GRP + y, zb * GRP + z] = nearest_code(np.float32(blk[y, z] * q), E4M3)
        P = np.zeros((br, bc), np.float32)
        for x in range(br):
            for z in range(bc):
                acc = np.float32(0.0)
                for kg in range(bk // GRP):
                    ex = sum(vals[int(Tq[x, y])] * vals[int(Sq[y, z])]
                             for y in range(kg * GRP, (kg + 1) * GRP))
                    acc = fmaf_exact(round_to_f32(ex), np.float32(dT[kg, x] * dS[kg, z // GRP]), acc)
                P[x, z] = acc
        Mr.append(bf16_torch(P))
        Tqs.append(Tq), Sqs.append(Sq), dTs.append(dT), dSs.append(dS)
    C = np.zeros((M, N), np.float32)
    for i in range(gm):
        for j in range(gn):
            for x in range(br):
                for z in range(bc):
                    acc = np.float32(0.0)
                    for r in range(R):
                        w = np.float32(W[r, i * gn + j])
                        if w != 0:
                            acc = fmaf_exact(w, Mr[r][x, z], acc)
                    C[i * br + x, j * bc + z] = acc
    return dict(C=C, Tq=np.array(Tqs), Sq=np.array(Sqs), dT=np.array(dTs), dS=np.array(dSs),
                Mr=np.array(Mr))


def test_group_schedule_matches_independent_computation():
    rng = np.random.default_rng(21)
    A = rng.standard_normal((4, 512)).astype(np.float32)
    A[1, :200] *= 300.0  # groups of very different magnitude within a row
    B = (0.02 * rng.standard_normal((512, 256))).astype(np.float32)
    B[:, 5] *= 40.0
    tabs, dims = oracle.flatten_f32(schemes.strassen())
    got = oracle.lowp_matmul(A, B, tabs, dims, E4M3, keep=True, scale_mode=SG)
    want = independent_group_schedule(A, B, *tabs, dims)
    assert got["dT"].shape == (7, 2, 2) and got["dS"].shape == (7, 2, 1)
    for key in ("Tq", "Sq"):
        assert np.array_equal(got[key], want[key]), key
    for key in ("dT", "dS", "Mr", "C"):
        assert np.array_equal(bits(got[key]), bits(want[key])), key


def test_group_accumulation_rule_before_bf16():
    """The fp32 accumulator of the group rule, before the bf16 rounding hides
    its last bits: acc = fmaf(exact group sum rounded once, fl(dT dS), acc)
    from +0 in ascending groups, against exact rationals."""
    rng = np.random.default_rng(24)
    finite = [c for c in range(256) if np.isfinite(oracle.fp8_decode([c], E4M3)[0])]
    Tq = rng.choice(finite, size=(3, 3 * GRP)).astype(np.uint8)
    Sq = rng.choice(finite, size=(3 * GRP, GRP)).astype(np.uint8)
    dT = (rng.random((3, 3)) * 1e-2 + 1e-3).astype(np.float32)
    dS = (rng.random((3, 1)) * 1e-2 + 1e-3).astype(np.float32)
    got = oracle.block_product_groups(Tq, Sq, dT, dS, E4M3, bf16=False)
    vt = oracle.fp8_decode(Tq, E4M3)
    vs = oracle.fp8_decode(Sq, E4M3)
    for x in range(3):
        for z in range(0, GRP, 9):
            acc = np.float32(0.0)
            for kg in range(3):
                ex = sum(Fraction(float(vt[x, y])) * Fraction(float(vs[y, z]))
                         for y in range(kg * GRP, (kg + 1) * GRP))
                acc = fmaf_exact(round_to_f32(ex), np.float32(dT[kg, x] * dS[kg, 0]), acc)
            assert got[x, z].view(np.uint32) == acc.view(np.uint32)
    rounded = oracle.block_product_groups(Tq, Sq, dT, dS, E4M3)
    assert np.array_equal(bits(rounded), bits(bf16_torch(got)))


def test_one_group_per_row_gives_the_row_scales_on_a():
    rng = np.random.default_rng(22)
    A = rng.standard_normal((64, 256)).astype(np.float32)
    U = oracle.flatten_f32(schemes.strassen())[0][0]
    t2, d2 = oracle.form_operands(A, 2, 2, U, scale_mode=SG, side=0)
    t1, d1 = oracle.form_operands(A, 2, 2, U, scale_mode=oracle.SCALE_ROWCOL, side=0)
    assert np.array_equal(t2, t1) and np.array_equal(bits(d2[:, 0, :]), bits(d1))


def test_products_are_bf16_values():
    rng = np.random.default_rng(23)
    A = rng.standard_normal((64, 512)).astype(np.float32)
    B = rng.standard_normal((512, 256)).astype(np.float32)
    got = oracle.lowp_matmul(A, B, *oracle.flatten_f32(schemes.strassen()), E4M3, keep=True,
                             scale_mode=SG)
    assert np.all(bits(got["Mr"]) & 0xffff == 0)


def changed_rows(C0, C1):
    return [int(r) for r in np.nonzero(np.any(C0 != C1, axis=1))[0]]


def test_row_map_and_prefix_pairs(golden):
    """App. C.3 and Sec. 4.2 under group scales (one group per block-sum row
    at inner length 512 with two levels): the same rows move as under the
    per-row form."""
    tabs, dims = oracle.flatten_f32(so.power(schemes.strassen(), 2))
    rng = np.random.default_rng(40)
    A = np.zeros((48, 512), np.float32)
    A[:40] = rng.standard_normal((40, 512))
    B = rng.standard_normal((512, 512)).astype(np.float32)
    A1 = A.copy()
    A1[39] = rng.standard_normal(512)
    C0 = oracle.lowp_matmul(A, B, tabs, dims, scale_mode=SG)
    C1 = oracle.lowp_matmul(A1, B, tabs, dims, scale_mode=SG)
    assert [r + 1 for r in changed_rows(C0, C1)] == golden["rowmap_changed_rows_1based"]["value"]
    rng = np.random.default_rng(32)
    A = rng.standard_normal((32, 512)).astype(np.float32)
    B = rng.standard_normal((512, 512)).astype(np.float32)
    base = oracle.lowp_matmul(A, B, tabs, dims, scale_mode=SG)
    rng2 = np.random.default_rng(33)
    moved = set()
    for j in range(1, 32):
        A1 = A.copy()
        A1[j] = rng2.standard_normal(512)
        C1 = oracle.lowp_matmul(A1, B, tabs, dims, scale_mode=SG)
        moved |= {(i, j) for i in range(j) if np.any(base[i] != C1[i])}
    assert len(moved) == golden["prefix_pairs_moved_fp8"]["value"]
    assert moved == {(i, j) for j in range(32) for i in range(j) if i % 8 == j % 8}


def test_power_of_two_on_one_block_offset():
    tabs, dims = oracle.flatten_f32(so.power(schemes.strassen(), 2))
    rng = np.random.default_rng(41)
    A = rng.standard_normal((32, 512)).astype(np.float32)
    B = rng.standard_normal((512, 512)).astype(np.float32)
    rows = [3, 11, 19, 27]  # offset 3 in each of the four row blocks
    A2 = A.copy()
    A2[rows] *= np.float32(8.0)
    C0 = oracle.lowp_matmul(A, B, tabs, dims, scale_mode=SG)
    C2 = oracle.lowp_matmul(A2, B, tabs, dims, scale_mode=SG)
    other = [r for r in range(32) if r not in rows]
    assert np.array_equal(bits(C2[rows]), bits(C0[rows] * np.float32(8.0)))
    assert np.array_equal(bits(C2[other]), bits(C0[other]))
