"""Pins of the oracle's coefficient side: tables, Kronecker power, gauges.

Each check is against something the paper or the mathematics fixes, not a
retyping of the oracle's own formula: the Brent equations (eq. (1) computes
AB for every input iff they hold), numbers the paper prints, the structure
of its Strassen table, and exactness of the product under gauges (Sec. 2.1).
"""
import numpy as np
import pytest

from oracle import scheme_ops as so
from oracle import schemes
import synthetic as sy


def test_strassen_table_satisfies_brent_exactly():
    assert so.brent_residual(schemes.strassen()) == 0.0


def test_laderman_table_satisfies_brent_exactly():
    s = schemes.laderman()
    assert s.R == 23
    assert so.brent_residual(s) == 0.0


def test_classical_scheme_brent_and_count():
    s = schemes.classical(2, 3, 4)
    assert s.R == 24
    assert so.brent_residual(s) == 0.0


def test_strassen_reads_and_feeds_rows_as_printed(golden):
    """App. A.1's table: which block rows of A each product reads and which
    block rows of C it feeds.  Pins U's row support and W's row support."""
    s = schemes.strassen()
    table = golden["strassen_reads_feeds"]["value"]
    for r in range(7):
        reads = sorted({i + 1 for i in range(2) for l in range(2) if s.U[r, i * 2 + l] != 0})
        feeds = sorted({i + 1 for i in range(2) for j in range(2) if s.W[r, i * 2 + j] != 0})
        assert reads == table[f"M{r + 1}"]["reads"]
        assert feeds == table[f"M{r + 1}"]["feeds"]


def test_two_level_strassen_printed_quantities(golden):
    s2 = so.power(schemes.strassen(), 2)
    c = so.criteria(s2)
    assert (s2.m, s2.k, s2.n, s2.R) == (4, 4, 4, golden["strassen2_products"]["value"])
    assert c["phi"] == golden["strassen2_phi"]["value"]
    assert c["nnz"] == golden["strassen2_nnz"]["value"]
    assert c["maxabs"] == golden["strassen2_maxabs"]["value"]
    assert c["L_A"] == golden["strassen2_L_A"]["value"]
    assert c["L_B"] == golden["strassen2_L_B"]["value"]
    assert c["L_W"] == golden["strassen2_L_W"]["value"]
    assert c["b_A"] == c["b_B"] == golden["strassen2_code_bound"]["value"]
    assert c["h_max_int32"] == golden["strassen2_h_max_int32"]["value"]
    ratio = s2.R / golden["strassen2_classical_products"]["value"]
    assert round(ratio, 4) == golden["strassen2_mult_ratio"]["value"]
    assert round(127 / c["b_A"], 4) == golden["step_ratio_127_over_31"]["value"]
    assert so.brent_residual(s2) == 0.0


def test_three_level_strassen_is_exact():
    s3 = so.power(schemes.strassen(), 3)
    assert (s3.m, s3.R) == (8, 343)
    assert int((s3.U != 0).sum()) == 12 ** 3
    assert so.brent_residual(s3) == 0.0


def test_kron_index_map_is_block_recursive():
    """Two-level Strassen applied to a matrix equals one-level Strassen whose
    block products are themselves computed with one-level Strassen: both
    evaluated in float64 give the exact product, and the flattened grid
    uses contiguous blocks (i = i1*m + i2)."""
    rng = np.random.default_rng(1)
    A = rng.integers(-3, 4, size=(8, 8)).astype(np.float64)
    B = rng.integers(-3, 4, size=(8, 8)).astype(np.float64)
    s2 = so.power(schemes.strassen(), 2)
    assert np.array_equal(so.evaluate_f64(s2, A, B), A @ B)


def test_sign_orbit_size_and_criteria_constant(golden):
    """Sec. 2.1 and Sec. 3.3: 512 sign variants of two-level Strassen, all
    exact, and every coefficient criterion takes one value on all of them."""
    s2 = so.power(schemes.strassen(), 2)
    orbit = sy.sign_orbit(4, 4, 4)
    assert len(orbit) == golden["strassen2_sign_variants"]["value"]
    assert orbit[0] == ((1.0,) * 4,) * 3
    ref = so.criteria(s2)
    for d, e, f in orbit[::37]:
        g = so.sign_gauge(s2, d, e, f)
        assert so.brent_residual(g) == 0.0
        assert so.criteria(g) == ref


def test_sign_variant_matches_paper_coefficient_rule():
    """Sec. 2.1: absorbing D, E, F gives d_i e_l u, e_l f_j v, d_i f_j w."""
    s = schemes.strassen()
    d, e, f = (1.0, -1.0), (1.0, -1.0), (1.0, 1.0)
    g = so.sign_gauge(s, d, e, f)
    for r in range(s.R):
        for i in range(2):
            for l in range(2):
                assert g.U[r, i * 2 + l] == d[i] * e[l] * s.U[r, i * 2 + l]
        for l in range(2):
            for j in range(2):
                assert g.V[r, l * 2 + j] == e[l] * f[j] * s.V[r, l * 2 + j]
        for i in range(2):
            for j in range(2):
                assert g.W[r, i * 2 + j] == d[i] * f[j] * s.W[r, i * 2 + j]


@pytest.mark.parametrize("base", ["strassen", "laderman"])
def test_gl_gauge_keeps_the_product_exact(base):
    """A gauged scheme computes the same product in exact arithmetic: in
    float64 it reproduces AB to rounding level, and satisfies Brent to 1e-12."""
    s = schemes.BASE_SCHEMES[base]()
    rng = np.random.default_rng(7)
    A = rng.standard_normal((s.m * 3, s.k * 2))
    B = rng.standard_normal((s.k * 2, s.n * 4))
    for P, Q, S in sy.gl_gauges(s.m, s.k, s.n, 8, seed=3):
        g = so.gauge(s, P, Q, S)
        assert so.brent_residual(g) < 1e-12
        C = so.evaluate_f64(g, A, B)
        assert np.linalg.norm(C - A @ B) / np.linalg.norm(A @ B) < 1e-12


def test_identity_gauge_round_trip_is_bit_identical():
    for s in (schemes.strassen(), schemes.laderman(), so.power(schemes.strassen(), 2)):
        g = so.gauge(s, np.eye(s.m), np.eye(s.k), np.eye(s.n))
        assert np.array_equal(g.U, s.U) and np.array_equal(g.V, s.V) and np.array_equal(g.W, s.W)


def test_gauge_composition_acts_as_a_group():
    """Applying (P1,Q1,S1) then (P2,Q2,S2) equals applying (P1 P2, Q2 Q1, S2 S1):
    the second gauge runs the first gauged scheme on P2 A Q2 and Q2^-1 B S2,
    i.e. the base scheme on (P1 P2) A (Q2 Q1) and (Q2 Q1)^-1 B (S2 S1)."""
    s = schemes.strassen()
    (P1, Q1, S1), (P2, Q2, S2) = sy.gl_gauges(2, 2, 2, 2, seed=11)
    g12 = so.gauge(so.gauge(s, P1, Q1, S1), P2, Q2, S2)
    gc = so.gauge(s, P1 @ P2, Q2 @ Q1, S2 @ S1)
    for a, b in ((g12.U, gc.U), (g12.V, gc.V), (g12.W, gc.W)):
        assert np.allclose(a, b, rtol=1e-12, atol=1e-12)


def test_single_sign_flip_is_rejected():
    """The paper checks its kernels reject a deliberate sign flip in one
    decoding coefficient (App. E, timings paragraph); the Brent equations
    catch every such flip."""
    s = schemes.strassen()
    for r in range(s.R):
        for ij in np.nonzero(s.W[r])[0]:
            W = s.W.copy()
            W[r, ij] = -W[r, ij]
            bad = schemes.Scheme(s.U, s.V, W, s.m, s.k, s.n, s.R)
            assert so.brent_residual(bad) >= 1.0


def test_inverse_formulas():
    rng = np.random.default_rng(5)
    for n in (1, 2, 3, 4, 6):
        P = rng.uniform(-2, 2, size=(n, n)) + 3 * np.eye(n)
        Pi = np.array(so.inverse(P.tolist()))
        assert np.allclose(Pi @ P, np.eye(n), atol=1e-12)
    D = np.diag([1.0, -1.0, -1.0, 1.0])
    assert np.array_equal(np.array(so.inverse(D.tolist())), D)
