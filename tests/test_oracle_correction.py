"""Pins of the overflow correction on the CPU oracle (Sec. 4.3, eq. (2);
App. D, the corrected computation's certificate; App. E, the correction's
multiplication counts), for two-level Strassen at code bound 127, groups of
128 and blocks of inner length 32.

What pins it:
  * the split of an exact block sum s = s0 + 256 q over every value two-level
    Strassen can produce at code bound 127 (|s| <= 508): s0 within int8,
    |q| <= 2, q = 0 exactly when s is itself within int8;
  * the printed bounds (508, |R| <= 2, h (128 + 512)^2 = 13,107,200 per
    reconstructed product entry, 16 of them below 2^31, group products below
    2^24) and the oracle's measured term sums on adversarial codes (signs
    following the coefficients) staying within them;
  * the corrected realization equals classical int8 at code bound 127 bit for
    bit on random Gaussian and heavy-tailed problems and under every one of
    the 512 sign variants, with overflows actually corrected, while the
    uncorrected block sums leave int8 (condition (i) fails at 127);
  * a deliberately flipped decoding weight is caught by the bit comparison
    (App. E's control);
  * the multiplication counts: with no overflow (code bound 31) the
    correction costs nothing and the total is 49/64 of classical int8; the
    sparse count never exceeds the gathered one, which never exceeds three
    dense products.  The counts on the heavy-tailed slices themselves are
    parity unpinned (the paper's values come from model layers).
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
G, H, BFULL = 128, 32, 127


def strassen2_tabs():
    return oracle.flatten_f32(so.power(schemes.strassen(), 2))


def quantize(A, B, b):
    Ac, dA = oracle.int8_quantize_a(A, G, b)
    Bc, dB = oracle.int8_quantize_b(B, G, b)
    return Ac, dA, Bc, dB


def bits(x):
    return np.ascontiguousarray(x, np.float32).view(np.uint32)


def test_split_of_every_reachable_block_sum():
    bound = GOLD["correction_block_sum_bound"]["value"]
    assert 4 * 127 == bound  # L_A * 127 for two-level Strassen
    qmax = 0
    for s in range(-bound, bound + 1):
        s0, q = oracle.int8_split(s)
        assert s == s0 + 256 * q
        assert -128 <= s0 <= 127
        assert (q == 0) == (-128 <= s <= 127)
        qmax = max(qmax, abs(q))
    assert qmax == GOLD["correction_remainder_bound"]["value"]


def test_printed_bounds():
    term = GOLD["correction_term_bound"]["value"]
    assert H * (128 + 256 * 2) ** 2 == term
    assert 16 * term < 2 ** 31
    grp = GOLD["correction_group_product_bound"]["value"]
    assert G * 127 ** 2 == grp and grp < 2 ** 24


def test_adversarial_codes_stay_within_the_bound():
    """Codes at +-127 whose signs follow one product's coefficients drive its
    block sums to 508: the oracle's largest sum of absolute weighted terms
    per output entry stays below L_W times the printed per-product bound."""
    (U, V, W), dims = strassen2_tabs()
    gm, gk, gn, R = dims
    r = int(np.argmax(np.abs(U).sum(1)))
    Ur = U[r].reshape(gm, gk)
    Vr = V[r].reshape(gk, gn)
    M, N, K = 4 * gm, 4 * gn, G
    Ac = np.zeros((M, K), np.int8)
    Bc = np.zeros((K, N), np.int8)
    br, bc = M // gm, N // gn
    for p in range(gm):
        for q in range(gk):
            Ac[p * br:(p + 1) * br, q * H:(q + 1) * H] = 127 * int(np.sign(Ur[p, q]) or 1)
    for p in range(gk):
        for q in range(gn):
            Bc[p * H:(p + 1) * H, q * bc:(q + 1) * bc] = 127 * int(np.sign(Vr[p, q]) or 1)
    dA = np.ones((M, K // G), np.float32)
    dB = np.ones((K // G, N), np.float32)
    out, st = oracle.int8_fast_corrected(Ac, dA, Bc, dB, (U, V, W), dims, G, H)
    assert st["split_violations"] == 0 and st["overflows"] > 0
    assert st["term_bound"] <= 16 * GOLD["correction_term_bound"]["value"]
    assert np.array_equal(bits(out), bits(oracle.int8_classical(Ac, dA, Bc, dB, G)))


@pytest.mark.parametrize("dist", ["normal", "t3"])
def test_corrected_equals_classical_at_127(dist):
    tabs, dims = strassen2_tabs()
    rng = np.random.default_rng(11 if dist == "normal" else 12)
    for M, K, N in ((64, 256, 96), (128, 384, 64)):
        A = (rng.standard_normal((M, K)) if dist == "normal"
             else rng.standard_t(3, (M, K))).astype(np.float32)
        B = rng.standard_normal((K, N)).astype(np.float32)
        Ac, dA, Bc, dB = quantize(A, B, BFULL)
        want = oracle.int8_classical(Ac, dA, Bc, dB, G)
        out, st = oracle.int8_fast_corrected(Ac, dA, Bc, dB, tabs, dims, G, H)
        assert np.array_equal(bits(out), bits(want))
        assert st["split_violations"] == 0 and st["overflows"] > 0
        # without the split the block sums leave int8: condition (i) fails
        _, viol_i, _ = oracle.int8_fast(Ac, dA, Bc, dB, tabs, dims, G, H)
        assert viol_i > 0


def test_every_sign_variant_corrected():
    s2 = so.power(schemes.strassen(), 2)
    rng = np.random.default_rng(13)
    A = rng.standard_normal((32, G)).astype(np.float32)
    B = rng.standard_normal((G, 32)).astype(np.float32)
    Ac, dA, Bc, dB = quantize(A, B, BFULL)
    want = bits(oracle.int8_classical(Ac, dA, Bc, dB, G))
    n = 0
    for d, e, f in sy.sign_orbit(4, 4, 4):
        tabs, dims = oracle.flatten_f32(so.gauge(s2, np.diag(d), np.diag(e), np.diag(f)))
        out, st = oracle.int8_fast_corrected(Ac, dA, Bc, dB, tabs, dims, G, H)
        assert np.array_equal(bits(out), want) and st["split_violations"] == 0
        n += 1
    assert n == 512


def test_flipped_weight_is_caught():
    """App. E: the bit check must reject a deliberate sign flip in one
    decoding coefficient."""
    (U, V, W), dims = strassen2_tabs()
    rng = np.random.default_rng(14)
    A = rng.standard_normal((32, G)).astype(np.float32)
    B = rng.standard_normal((G, 32)).astype(np.float32)
    Ac, dA, Bc, dB = quantize(A, B, BFULL)
    want = bits(oracle.int8_classical(Ac, dA, Bc, dB, G))
    r, c = np.argwhere(W != 0)[7]
    W2 = W.copy()
    W2[r, c] = -W2[r, c]
    out, _ = oracle.int8_fast_corrected(Ac, dA, Bc, dB, (U, V, W2), dims, G, H)
    assert not np.array_equal(bits(out), want)


def test_counts_without_overflow_and_their_order():
    tabs, dims = strassen2_tabs()
    rng = np.random.default_rng(15)
    A = rng.standard_normal((64, 256)).astype(np.float32)
    B = rng.standard_normal((256, 64)).astype(np.float32)
    Ac, dA, Bc, dB = quantize(A, B, 31)
    _, st = oracle.int8_fast_corrected(Ac, dA, Bc, dB, tabs, dims, G, H)
    assert st["overflows"] == 0 and st["sparse"] == 0 and st["gathered"] == 0
    assert st["main"] / st["classical"] == pytest.approx(49 / 64, abs=0)
    Ac, dA, Bc, dB = quantize(A, B, BFULL)
    _, st = oracle.int8_fast_corrected(Ac, dA, Bc, dB, tabs, dims, G, H)
    assert 0 < st["sparse"] <= st["gathered"] <= 3 * st["main"]


def test_counts_on_a_heavy_tailed_slice():
    """The correction's counts on a reduced heavy-tailed slice (parity
    unpinned: reported, with the invariants that must hold)."""
    w = sy.scaled(sy.CORRECTION_SLICES["down_512x13824x1024"], 128, 512, 256)
    A, B = sy.operands(w)
    tabs, dims = strassen2_tabs()
    Ac, dA, Bc, dB = quantize(A, B, BFULL)
    out, st = oracle.int8_fast_corrected(Ac, dA, Bc, dB, tabs, dims, G, H)
    assert np.array_equal(bits(out), bits(oracle.int8_classical(Ac, dA, Bc, dB, G)))
    assert 0 < st["sparse"] <= st["gathered"]
    assert st["main"] / st["classical"] == pytest.approx(49 / 64, abs=0)
