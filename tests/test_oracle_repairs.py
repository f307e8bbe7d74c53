"""Pins of the repairs on the CPU oracle (App. C, the repair rules), as
options of the group-scale schedule: the outside power-of-two row scaling of
A and the joint rounding of B's block sums.

What pins them:
  * the row exponent against an exactly rounded float64 definition (math.fsum)
    on rows of many scales, on rows whose RMS is exactly a power of two or
    one unit above it, and on zero and tiny rows (the 1e-3 floor);
  * row scaling makes the output covariant with a power of two on any single
    row of A (that row's output scales exactly, the others do not move), and
    equals the plain schedule when every row has the same exponent;
  * joint rounding: with H the identity (the classical 2 x 2 x 2 scheme) it is
    the ordinary nearest rounding; on Strassen it never raises the exact
    quadratic error e^T H e of a position above the nearest rounding's, and
    leaves no single flip that lowers it by more than the fp32 decision noise;
    H's entries for two-level Strassen against exact integer inner products;
  * no flags: the plain group-scale schedule bit for bit.
The repaired errors on the workloads are parity unpinned (the paper's are on
model layers).
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import scheme_ops as so
from oracle import schemes

E4M3 = oracle.E4M3


def bits(x):
    return np.ascontiguousarray(x, np.float32).view(np.uint32)


def exponent_by_definition(row):
    m2 = math.fsum(float(v) * float(v) for v in row) / len(row)
    if m2 == 0:
        return -9
    rms = Fraction(m2) ** 1  # exact value of the float64 mean of squares
    # least k with 4^k >= m2, at least -9
    k = -9
    while Fraction(4) ** k < rms:
        k += 1
    while k > -9 and Fraction(4) ** (k - 1) >= rms:
        k -= 1
    return k


def test_row_exponent_definition():
    rng = np.random.default_rng(1)
    rows = [rng.standard_normal(300).astype(np.float32) * np.float32(10.0 ** e)
            for e in rng.uniform(-5, 6, 40)]
    K = 256
    for j in (-12, -3, 0, 5):
        rows.append(np.full(K, 2.0 ** j, np.float32))             # RMS exactly 2^j
        up = np.full(K, 2.0 ** j, np.float32)
        up[0] = np.nextafter(up[0], np.float32(np.inf))
        rows.append(up)                                            # just above 2^j
    rows += [np.zeros(K, np.float32), np.full(K, 1e-6, np.float32)]
    for row in rows:
        assert oracle.row_exponents(row[None, :])[0] == exponent_by_definition(row)
    k = oracle.row_exponents(np.stack([np.full(K, 2.0 ** j, np.float32) for j in (-12, -3, 0, 5)]))
    assert list(k) == [-9, -3, 0, 5]


def strassen2():
    return oracle.flatten_f32(so.power(schemes.strassen(), 2))


def test_no_flags_is_the_plain_group_schedule():
    tabs, dims = strassen2()
    rng = np.random.default_rng(2)
    A = rng.standard_normal((32, 512)).astype(np.float32)
    B = rng.standard_normal((512, 512)).astype(np.float32)
    C0 = oracle.lowp_matmul(A, B, tabs, dims, scale_mode=oracle.SCALE_GROUP)
    C1 = oracle.lowp_matmul_repaired(A, B, tabs, dims, flags=0)
    assert np.array_equal(bits(C0), bits(C1))


def test_row_scaling_makes_single_rows_covariant():
    tabs, dims = strassen2()
    rng = np.random.default_rng(3)
    A = rng.standard_normal((32, 512)).astype(np.float32)
    A[::5] *= np.float32(30.0)
    B = rng.standard_normal((512, 512)).astype(np.float32)
    C = oracle.lowp_matmul_repaired(A, B, tabs, dims, flags=oracle.REPAIR_ROWS)
    for t, p in ((3, 4.0), (17, 0.125), (30, 64.0)):
        A2 = A.copy()
        A2[t] *= np.float32(p)
        C2 = oracle.lowp_matmul_repaired(A2, B, tabs, dims, flags=oracle.REPAIR_ROWS)
        others = [r for r in range(32) if r != t]
        assert np.array_equal(bits(C2[t]), bits(C[t] * np.float32(p)))
        assert np.array_equal(bits(C2[others]), bits(C[others]))
    # the plain schedule is not covariant: its block-sum rows mix row t with others
    P = oracle.lowp_matmul(A, B, tabs, dims, scale_mode=oracle.SCALE_GROUP)
    A2 = A.copy()
    A2[3] *= np.float32(64.0)
    P2 = oracle.lowp_matmul(A2, B, tabs, dims, scale_mode=oracle.SCALE_GROUP)
    assert not np.array_equal(bits(P2[[11, 19, 27]]), bits(P[[11, 19, 27]]))


def test_row_scaling_with_one_common_exponent_changes_nothing():
    tabs, dims = strassen2()
    rng = np.random.default_rng(4)
    A = np.sign(rng.standard_normal((32, 512))).astype(np.float32) * np.float32(8.0)  # RMS 8
    B = rng.standard_normal((512, 512)).astype(np.float32)
    got = oracle.lowp_matmul_repaired(A, B, tabs, dims, flags=oracle.REPAIR_ROWS, keep=True)
    assert set(got["rowexp"].tolist()) == {3}
    C0 = oracle.lowp_matmul(A, B, tabs, dims, scale_mode=oracle.SCALE_GROUP)
    assert np.array_equal(bits(got["C"]), bits(C0))


def test_gram_of_two_level_strassen():
    (U, V, W), dims = strassen2()
    H = oracle.repair_gram(U, W)
    Ui, Wi = U.astype(np.int64), W.astype(np.int64)
    assert np.array_equal(H.astype(np.int64), (Wi @ Wi.T) * (Ui @ Ui.T))
    assert np.array_equal(H, H.T) and np.all(np.diag(H) > 0)


def test_identity_gram_gives_the_nearest_rounding():
    """The classical 2 x 2 x 2 scheme has H = I: each coordinate is rounded
    alone, to the code whose value is nearest the bf16 entry (checked in
    exact rationals wherever the two distances differ beyond fp32 noise)."""
    c = schemes.classical(2, 2, 2)
    tabs, dims = oracle.flatten_f32(c)
    H = oracle.repair_gram(tabs[0], tabs[2])
    assert np.array_equal(H, np.eye(8, dtype=np.float32))
    rng = np.random.default_rng(5)
    checked = 0
    for _ in range(300):
        s = oracle.bf16_round(rng.standard_normal(8).astype(np.float32))
        amax = np.float32(np.abs(s).max() * rng.uniform(1.0, 2.0))
        q = np.full(8, np.float32(448.0) / amax, np.float32)
        d = np.full(8, amax / np.float32(448.0), np.float32)
        codes, sweeps = oracle.joint_round_position(s, q, d, H)
        assert sweeps == 1  # nothing to improve after the start
        for r in range(8):
            y = np.float32(s[r] * q[r])
            c0 = int(oracle.fp8_encode(np.array([y], np.float32))[0])
            cands = {c0, c0 + 1 if abs(float(oracle.fp8_decode([c0])[0])) < abs(float(y)) else c0 - 1}
            dist = {cc: abs(Fraction(float(np.float32(np.float32(oracle.fp8_decode([cc])[0]) * d[r])))
                            - Fraction(float(s[r]))) for cc in cands if 0 <= (cc & 0x7f) <= 0x7e}
            best = min(dist, key=dist.get)
            others = [v for cc, v in dist.items() if cc != best]
            if others and abs(others[0] - dist[best]) > Fraction(float(d[r])) * Fraction(1, 10 ** 6):
                assert codes[r] == best
                checked += 1
    assert checked > 1000


def exact_energy(codes, s, d, H):
    vals = oracle.fp8_decode(codes, E4M3)
    e = [Fraction(float(np.float32(np.float32(v) * dd))) - Fraction(float(ss))
         for v, dd, ss in zip(vals, d, s)]
    Hf = [[Fraction(float(h)) for h in row] for row in H]
    return sum(e[r] * Hf[r][t] * e[t] for r in range(len(e)) for t in range(len(e)))


def bracket(y):
    """The codes whose values bracket y (one or two)."""
    c0 = int(oracle.fp8_encode(np.array([y], np.float32))[0])
    v0 = float(oracle.fp8_decode([c0])[0])
    if v0 == float(y):
        return {c0}
    step = 1 if abs(float(y)) > abs(v0) else -1
    c1 = (c0 & 0x80) | ((c0 & 0x7f) + step)
    return {c0, c1} if 0 <= (c0 & 0x7f) + step <= 0x7e else {c0}


def test_joint_rounding_lowers_the_quadratic_error():
    """On two-level Strassen: every code is one of the two that bracket its
    scaled value; the exact quadratic error e^T H e never exceeds the nearest
    rounding's; when the sweeps stop on their own, no single flip lowers it
    beyond fp32 decision noise; and the sweeps usually improve on nearest."""
    (U, V, W), dims = strassen2()
    H = oracle.repair_gram(U, W)
    R = H.shape[0]
    rng = np.random.default_rng(6)
    improved = 0
    for _ in range(12):
        s = oracle.bf16_round(rng.standard_normal(R).astype(np.float32) * np.float32(0.05))
        amax = np.abs(s).max() * rng.uniform(1.0, 3.0)
        q = np.full(R, np.float32(448.0) / np.float32(amax), np.float32)
        d = np.full(R, np.float32(amax) / np.float32(448.0), np.float32)
        rne = oracle.fp8_encode((s * q).astype(np.float32))
        codes, sweeps = oracle.joint_round_position(s, q, d, H)
        assert 1 <= sweeps <= oracle.REPAIR_SWEEPS
        for r in range(R):
            assert int(codes[r]) in bracket(np.float32(s[r] * q[r]))
        noise = float(np.sum(np.abs(H))) * float(d[0]) ** 2 * 1e-5
        E0, E1 = exact_energy(rne, s, d, H), exact_energy(codes, s, d, H)
        assert float(E1) <= float(E0) + noise
        if sweeps < oracle.REPAIR_SWEEPS:
            for r in range(R):
                others = bracket(np.float32(s[r] * q[r])) - {int(codes[r])}
                for o in others:
                    c2 = codes.copy()
                    c2[r] = o
                    assert float(exact_energy(c2, s, d, H)) >= float(E1) - noise
        improved += int(float(E1) < float(E0) - noise)
    assert improved >= 6


def test_joint_rounding_sweeps_in_ascending_order_hand_example():
    """App. C's joint rounding sweeps r = 1, ..., R in order.  A hand-worked
    position (E4M3, q = d = 1, so values are codes' values) where the sweep
    order decides the outcome:

      s = (343/256, 151/128, 103/64), H = [[6, -6, 0], [-6, 9, 0], [0, 0, 8]].

    Brackets: s0 in (5/4, 11/8), s1 in (9/8, 5/4), s2 in (3/2, 13/8); the
    nearer values start: (11/8, 9/8, 13/8), e = (9, -14, 4)/256, so
    g = H e = (138, -180, 32)/256.  Sweep 1, r = 0: delta = -1/8, change =
    2 delta g0 + delta^2 H00 = -276/2048 + 6/64 < 0, flip to 5/4; g becomes
    (-54, 12, 32)/256.  r = 1: delta = 1/8, change = 24/2048 + 9/64 > 0.
    r = 2: delta = -1/8, change = -64/2048 + 8/64 > 0.  Sweep 2 changes
    nothing (r = 0: 2 (1/8)(-54/256) + 6/64 > 0), so two sweeps end at
    (5/4, 9/8, 13/8) = codes (0x3A, 0x39, 0x3D).

    Swept in reverse (r = 2, 1, 0) the same start flips product 1 first
    (change 2 (1/8)(-180/256) + 9/64 < 0), after which g0 = -54/256 keeps
    product 0 at 11/8: (11/8, 5/4, 13/8) = (0x3B, 0x3A, 0x3D).  Every value
    here is exact in fp32 and no decision is within 1/64 of zero, so the
    fp32 arithmetic cannot change a decision."""
    s = np.array([343 / 256, 151 / 128, 103 / 64], np.float32)
    H = np.array([[6, -6, 0], [-6, 9, 0], [0, 0, 8]], np.float32)
    one = np.ones(3, np.float32)
    codes, sweeps = oracle.joint_round_position(s, one, one, H)
    assert [int(c) for c in codes] == [0x3A, 0x39, 0x3D]
    assert sweeps == 2
    assert list(oracle.fp8_decode(codes)) == [1.25, 1.125, 1.625]
    # the reversed sweep's result, from the oracle on the mirrored problem
    # (reverse the product order, so that its ascending sweep visits the
    # original products from the last): it must differ
    p = [2, 1, 0]
    rcodes, rsweeps = oracle.joint_round_position(s[p], one, one, H[np.ix_(p, p)])
    assert [int(c) for c in rcodes[p]] == [0x3B, 0x3A, 0x3D]
    assert rsweeps == 2
