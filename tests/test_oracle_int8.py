"""Pins of the integer path on the CPU oracle: the quantization
specification of App. D, the classical int8 operator (Sec. 2.2) and the
certified fast realization of Sec. 4.2 (Prop. 1), for two-level Strassen at
code bound 31, groups of 128 and blocks of inner length 32.

What pins it:
  * the quantizer's definition on constructed groups (unit scales, ties to
    even, the largest entry reaching the code bound, all-zero groups);
  * the classical operator reduces to an exact integer matrix product when
    every scale is 1, and is row-local;
  * Prop. 1: the fast realization equals classical int8 bit for bit on 200
    random problems and for every one of the 512 sign variants, with no
    block sum outside int8 and no partial sum outside int32; the sign
    variants give one distinct integer product, and rounding the block sums
    to FP8 instead leaves none of them exact;
  * the certificate's conditions (the printed L_A, L_B, L_W and h_max), the
    sharpness of condition (i) (codes following the coefficient signs reach
    L_A b, so b = 32 leaves int8);
  * prefix invariance: 0 of 496 pairs of token rows move.
"""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import scheme_ops as so
from oracle import schemes
import synthetic as sy

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))
G, B_CODE, H = 128, 31, 32


def strassen2():
    return so.power(schemes.strassen(), 2)


def tabs(s):
    return oracle.flatten_f32(s)


def quantized(rng, M, K, N, b=B_CODE):
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = rng.standard_normal((K, N)).astype(np.float32)
    Ac, dA = oracle.int8_quantize_a(A, G, b)
    Bc, dB = oracle.int8_quantize_b(B, G, b)
    return Ac, dA, Bc, dB


def test_quantizer_definition():
    """d = max|x| / b; codes x / d rounded to nearest, ties to even."""
    # a group whose largest magnitude is b has d = 1, so codes are the
    # values rounded to nearest even
    row = np.zeros(G, np.float32)
    row[:8] = [31.0, 2.5, 3.5, -2.5, -3.5, 0.49999997, 7.5, -0.5]
    codes, d = oracle.int8_quantize_a(row[None, :], G, 31)
    assert d[0, 0] == np.float32(1.0)
    assert list(codes[0, :8]) == [31, 2, 4, -2, -4, 0, 8, 0]
    # general groups: the largest entry maps to +-b, every code within b,
    # reconstruction within half a step
    rng = np.random.default_rng(0)
    X = (rng.standard_normal((16, 4 * G)) * rng.uniform(0.01, 100, (16, 1))).astype(np.float32)
    codes, d = oracle.int8_quantize_a(X, G, 31)
    for t in range(16):
        for gi in range(4):
            x = X[t, gi * G:(gi + 1) * G].astype(np.float64)
            c = codes[t, gi * G:(gi + 1) * G].astype(np.float64)
            assert np.max(np.abs(c)) == 31 and np.abs(c[np.argmax(np.abs(x))]) == 31
            assert np.all(np.abs(x - c * d[t, gi]) <= 0.5 * d[t, gi] * (1 + 1e-6))
    # an all-zero group has d = 1 and zero codes; B's groups run down columns
    Z = np.zeros((G, 3), np.float32)
    Z[:, 1] = rng.standard_normal(G)
    cb, db = oracle.int8_quantize_b(Z, G, 31)
    assert db[0, 0] == 1.0 and db[0, 2] == 1.0 and not cb[:, 0].any()
    assert np.max(np.abs(cb[:, 1])) == 31


def test_classical_operator_with_unit_scales_is_the_integer_product():
    """With every group's largest magnitude equal to b the scales are 1, the
    codes are the inputs, and the operator returns the exact integer product
    (all partial sums are integers below 2^24)."""
    rng = np.random.default_rng(1)
    M, K, N = 12, 3 * G, 10
    A = rng.integers(-31, 32, (M, K)).astype(np.float32)
    B = rng.integers(-31, 32, (K, N)).astype(np.float32)
    for gi in range(3):
        A[:, gi * G] = 31
        B[gi * G, :] = -31
    Ac, dA = oracle.int8_quantize_a(A, G, 31)
    Bc, dB = oracle.int8_quantize_b(B, G, 31)
    assert np.all(dA == 1) and np.all(dB == 1)
    out = oracle.int8_classical(Ac, dA, Bc, dB, G)
    assert np.array_equal(out.astype(np.int64), A.astype(np.int64) @ B.astype(np.int64))


def test_classical_operator_is_row_local():
    rng = np.random.default_rng(2)
    M, K, N = 16, 2 * G, 8
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = rng.standard_normal((K, N)).astype(np.float32)
    Bc, dB = oracle.int8_quantize_b(B, G, 31)
    Ac, dA = oracle.int8_quantize_a(A, G, 31)
    base = oracle.int8_classical(Ac, dA, Bc, dB, G)
    A[5] = rng.standard_normal(K)
    Ac, dA = oracle.int8_quantize_a(A, G, 31)
    out = oracle.int8_classical(Ac, dA, Bc, dB, G)
    changed = np.nonzero(np.any(out != base, axis=1))[0]
    assert list(changed) == [5]


def test_certificate_of_two_level_strassen():
    """Sec. 4.2: L_A = L_B = 4, L_W = 16, so code bound 31 satisfies (i);
    blocks of 32 with groups of 128 satisfy (ii) and (iii); int32 stays exact
    up to inner length 8729."""
    s2 = strassen2()
    c = oracle.certificate(s2, 31, 31, H, G, 4)
    assert (c["L_A"], c["L_B"], c["L_W"]) == (GOLD["strassen2_L_A"]["value"],
                                               GOLD["strassen2_L_B"]["value"],
                                               GOLD["strassen2_L_W"]["value"])
    assert c["certified"]
    assert not oracle.certificate(s2, 32, 32, H, G, 4)["i"]      # 4 * 32 = 128 leaves int8
    assert not oracle.certificate(s2, 127, 127, H, G, 4)["i"]
    h_max = GOLD["strassen2_h_max_int32"]["value"]
    assert oracle.certificate(s2, 31, 31, h_max, G, 4)["ii"]
    assert not oracle.certificate(s2, 31, 31, h_max + 1, G, 4)["ii"]
    assert not oracle.certificate(s2, 31, 31, H, 96, 4)["iii"]   # a call of 128 spans two groups


def test_fast_realization_equals_classical_on_random_problems():
    """Prop. 1 on 200 random problems (the paper's 200 random tiles): output
    bits identical, no condition violated on the way."""
    s2 = tabs(strassen2())
    rng = np.random.default_rng(3)
    trials = GOLD["int8_exact_trials"]["value"]
    for _ in range(trials):
        Ac, dA, Bc, dB = quantized(rng, 16, G, 8)
        fast, v1, v2 = oracle.int8_fast(Ac, dA, Bc, dB, *s2, G, H)
        assert v1 == 0 and v2 == 0
        assert np.array_equal(fast.view(np.uint32),
                              oracle.int8_classical(Ac, dA, Bc, dB, G).view(np.uint32))


def test_every_sign_variant_gives_the_classical_bits():
    """All 512 sign variants on one problem of two groups: one distinct
    integer product per group, output bits equal to classical int8."""
    rng = np.random.default_rng(4)
    Ac, dA, Bc, dB = quantized(rng, 32, 2 * G, 32)
    want = oracle.int8_classical(Ac, dA, Bc, dB, G).view(np.uint32)
    P0 = oracle.int8_group_product(Ac, Bc, G, 0).astype(np.float64)
    s2 = strassen2()
    distinct = set()
    for d, e, f in sy.sign_orbit(4, 4, 4):
        t = tabs(so.gauge(s2, np.diag(d), np.diag(e), np.diag(f)))
        out, v1, v2 = oracle.int8_fast(Ac, dA, Bc, dB, *t, G, H)
        assert v1 == 0 and v2 == 0
        assert np.array_equal(out.view(np.uint32), want)
        P, _, _ = oracle.int8_group_product_fast(Ac, Bc, *t, G, 0, H)
        distinct.add(P.tobytes())
        assert np.array_equal(P, P0)
    assert len(distinct) == GOLD["int8_sign_variants_distinct_products"]["value"]


def test_fp8_rounded_block_sums_leave_no_variant_exact():
    """Sec. 4.2: on a tile of codes at bound 31, rounding the block sums to
    E4M3 (integers above 16 are not all representable) leaves none of the
    512 sign variants with the exact integer product."""
    rng = np.random.default_rng(5)
    Ac = rng.integers(-31, 32, (32, G)).astype(np.int8)
    Bc = rng.integers(-31, 32, (G, 32)).astype(np.int8)
    exact = oracle.int8_group_product(Ac, Bc, G, 0).astype(np.float64)
    s2 = strassen2()
    n_exact, worst = 0, []
    for d, e, f in sy.sign_orbit(4, 4, 4):
        t = tabs(so.gauge(s2, np.diag(d), np.diag(e), np.diag(f)))
        P, _, _ = oracle.int8_group_product_fast(Ac, Bc, *t, G, 0, H, round_fp8=True)
        n_exact += int(np.array_equal(P, exact))
        worst.append(np.max(np.abs(P - exact)))
    assert n_exact == GOLD["int8_fp8_rounded_exact_variants"]["value"]
    assert max(worst) / min(worst) > 1.2  # the variants' largest errors differ


def test_condition_i_is_sharp():
    """Codes whose signs follow a product's coefficients reach L_A * b in that
    block sum: at b = 31 that is 124, within int8; at b = 32 it is 128, and
    the realization leaves int8 (condition (i) fails)."""
    (U, V, W), dims = tabs(strassen2())
    r = int(np.argmax(np.abs(U).sum(1)))  # a product reading L_A = 4 blocks
    Ur = U[r].reshape(4, 4)
    assert np.abs(Ur).sum() == 4
    for b, expect_violation in ((31, False), (32, True)):
        Ac = np.zeros((8, G), np.int8)  # block rows of 2
        for p in range(4):
            for q in range(4):
                if Ur[p, q] != 0:
                    Ac[p * 2:(p + 1) * 2, q * H:(q + 1) * H] = int(b * np.sign(Ur[p, q]))
        Bc = np.ones((G, 4), np.int8)
        _, v1, _ = oracle.int8_group_product_fast(Ac, Bc, (U, V, W), dims, G, 0, H)
        assert (v1 > 0) == expect_violation, (b, v1)


def test_no_prefix_pair_moves_under_the_certified_realization():
    """Sec. 4.2: 32 token rows in four blocks, one group of 128; changing one
    later row at a time moves 0 of the 496 pairs."""
    rng = np.random.default_rng(32)
    A = rng.standard_normal((32, G)).astype(np.float32)
    B = rng.standard_normal((G, 128)).astype(np.float32)
    Bc, dB = oracle.int8_quantize_b(B, G, 31)
    t = tabs(strassen2())

    def run(X):
        Ac, dA = oracle.int8_quantize_a(X, G, 31)
        return oracle.int8_fast(Ac, dA, Bc, dB, *t, G, H)[0]

    base = run(A)
    moved = set()
    rng2 = np.random.default_rng(33)
    for j in range(1, 32):
        A1 = A.copy()
        A1[j] = rng2.standard_normal(G)
        out = run(A1)
        moved |= {(i, j) for i in range(j) if np.any(out[i] != base[i])}
    assert 32 * 31 // 2 == GOLD["prefix_pairs_total"]["value"]
    assert len(moved) == GOLD["int8_prefix_pairs_moved"]["value"]
