"""GPU parity of the integer path through the C ABI: the quantizer and the
classical int8 operator bit for bit against the CPU oracle, and the
certified fast realization (Sec. 4.2, Prop. 1) bit for bit against the
classical operator -- for two-level Strassen at code bound 31 (blocks of 32,
groups of 128), every one of its 512 sign variants, and one-level Strassen
at code bound 63.  Uncertified configurations are rejected before any
kernel runs; codes beyond the certified bound are reported.
"""
import sys

import numpy as np
import pytest

import oracle
from oracle import scheme_ops as so
from oracle import schemes as osch
import synthetic as sy

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU-only machines, never run
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2609_39816_amd import fm  # noqa: E402

DEV = torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def gpu(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def bits(x):
    return np.ascontiguousarray(x, np.float32).view(np.uint32)


def quantize_both(A, B, g, b):
    """Device codes and scales (B through its transpose) and the oracle's."""
    Ac, dA = fm.int8_quantize(gpu(A), g, b)
    BTc, dB = fm.int8_quantize(gpu(np.ascontiguousarray(B.T)), g, b)
    oAc, odA = oracle.int8_quantize_a(A, g, b)
    oBc, odB = oracle.int8_quantize_b(B, g, b)
    return (Ac, dA, BTc, dB), (oAc, odA, oBc, odB)


@pytest.mark.parametrize("M,K,N,g,b", [(96, 384, 80, 128, 31), (64, 512, 200, 256, 127),
                                       (300, 256, 132, 128, 63)])
def test_quantizer_and_classical_operator_bit_exact(M, K, N, g, b):
    say(f"[int8] classical {M}x{K}x{N} g={g} b={b}")
    rng = np.random.default_rng(M + K + N)
    A = (rng.standard_normal((M, K)) * rng.uniform(0.1, 10, (M, 1))).astype(np.float32)
    B = rng.standard_normal((K, N)).astype(np.float32)
    (Ac, dA, BTc, dB), (oAc, odA, oBc, odB) = quantize_both(A, B, g, b)
    assert np.array_equal(Ac.cpu().numpy(), oAc)
    assert np.array_equal(BTc.cpu().numpy(), oBc.T)
    assert np.array_equal(bits(dA.cpu().numpy()), bits(odA.T))
    assert np.array_equal(bits(dB.cpu().numpy()), bits(odB))
    out = fm.int8_matmul_classical(Ac, dA, BTc, dB, g).cpu().numpy()
    want = oracle.int8_classical(oAc, odA, oBc, odB, g)
    assert np.array_equal(bits(out), bits(want))


def fast_vs_classical(s, levels, M, K, N, g, h, b, seed, variants=None):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = rng.standard_normal((K, N)).astype(np.float32)
    (Ac, dA, BTc, dB), (oAc, odA, oBc, odB) = quantize_both(A, B, g, b)
    cl = fm.int8_matmul_classical(Ac, dA, BTc, dB, g).cpu().numpy()
    assert np.array_equal(bits(cl), bits(oracle.int8_classical(oAc, odA, oBc, odB, g)))
    schemes = [s] if variants is None else variants
    ws = fm.workspace(fm.int8_workspace_size(schemes[0], M, N, K, levels, g, h))
    for sc in schemes:
        out = fm.int8_matmul_fast(sc, Ac, dA, BTc, dB, levels, g, h, b, b, ws=ws).cpu().numpy()
        fm.status(ws)  # no block sum left int8
        assert np.array_equal(bits(out), bits(cl))
    return cl


def test_two_level_strassen_equals_classical():
    say("[int8] fast two-level Strassen 256x512x384")
    fast_vs_classical(fm.Scheme.base("strassen"), 2, 256, 512, 384, 128, 32, 31, 1)


def test_two_level_strassen_groups_of_256_and_ragged_tiles():
    say("[int8] fast two-level Strassen 400x768x208, g=256")
    fast_vs_classical(fm.Scheme.base("strassen"), 2, 400, 768, 208, 256, 32, 31, 2)


def test_one_level_strassen_at_code_bound_63():
    say("[int8] fast one-level Strassen b=63 h=64")
    fast_vs_classical(fm.Scheme.base("strassen"), 1, 192, 384, 136, 128, 64, 63, 3)


def test_every_sign_variant_equals_classical():
    """All 512 sign variants of two-level Strassen on one problem: every
    output bit equals classical int8's (Sec. 4.2: one distinct output)."""
    say("[int8] 512 sign variants 64x256x64")
    s2 = fm.Scheme.base("strassen").kron(2)
    orbit = s2.gauge_orbit([(np.diag(d), np.diag(e), np.diag(f)) for d, e, f in sy.sign_orbit(4, 4, 4)])
    fast_vs_classical(None, 1, 64, 256, 64, 128, 32, 31, 4, variants=orbit)


def test_larger_problem_equals_classical():
    say("[int8] fast two-level Strassen 2048x2048x2048")
    fast_vs_classical(fm.Scheme.base("strassen"), 2, 2048, 2048, 2048, 128, 32, 31, 5)


def test_uncertified_configurations_are_rejected():
    """Prop. 1 is checked before any kernel: code bound 32 (block sums can
    reach 128), a call spanning two groups, GL-gauged coefficients."""
    s = fm.Scheme.base("strassen")
    z8 = torch.zeros((64, 256), dtype=torch.int8, device=DEV)
    d = torch.ones((2, 64), dtype=torch.float32, device=DEV)
    ws = fm.workspace(fm.int8_workspace_size(s, 64, 64, 256, 2, 128, 32))
    with pytest.raises(fm.FmError) as e:
        fm.int8_matmul_fast(s, z8, d, z8, d, 2, 128, 32, 32, 32, ws=ws)
    assert e.value.name == "FM_E_UNCERTIFIED"
    with pytest.raises(fm.FmError) as e:
        fm.int8_matmul_fast(s, z8, d, z8, d, 2, 128, 64, 31, 31, ws=ws)  # a call of 256 > 128
    assert e.value.name in ("FM_E_UNCERTIFIED", "FM_E_WORKSPACE")


def test_codes_beyond_the_bound_are_reported():
    """Codes quantized at 127 but claimed to be within 31: some block sums
    leave int8; the device flags it and fm_status reports FM_E_RANGE."""
    rng = np.random.default_rng(6)
    A = rng.standard_normal((64, 128)).astype(np.float32)
    B = rng.standard_normal((128, 64)).astype(np.float32)
    (Ac, dA, BTc, dB), _ = quantize_both(A, B, 128, 127)
    s = fm.Scheme.base("strassen")
    ws = fm.workspace(fm.int8_workspace_size(s, 64, 64, 128, 2, 128, 32))
    fm.int8_matmul_fast(s, Ac, dA, BTc, dB, 2, 128, 32, 31, 31, ws=ws)
    with pytest.raises(fm.FmError) as e:
        fm.status(ws)
    assert e.value.name == "FM_E_RANGE"


def test_prepared_plan_runs_new_codes():
    """A plan made once serves later calls: two runs on different codes of the
    planned shapes give the classical operator's bits; other shapes are
    rejected by the binding."""
    say("[int8] plan: two-level Strassen 256x512x384, two runs")
    s = fm.Scheme.base("strassen")
    M, K, N, g, h, b = 256, 512, 384, 128, 32, 31
    plan = fm.Int8Plan(s, M, N, K, 2, g, h, b, b, device=DEV)
    for seed in (7, 8):
        rng = np.random.default_rng(seed)
        A = rng.standard_normal((M, K)).astype(np.float32)
        B = rng.standard_normal((K, N)).astype(np.float32)
        (Ac, dA, BTc, dB), (oAc, odA, oBc, odB) = quantize_both(A, B, g, b)
        out = plan.run(Ac, dA, BTc, dB).cpu().numpy()
        fm.status(plan.ws)
        assert np.array_equal(bits(out), bits(oracle.int8_classical(oAc, odA, oBc, odB, g)))
    with pytest.raises(ValueError):
        plan.run(Ac[:128].contiguous(), dA[:, :128].contiguous(), BTc, dB)


def corrected_vs_classical(s, levels, M, K, N, seed, variants=None, dist="normal", b=127):
    rng = np.random.default_rng(seed)
    A = (rng.standard_normal((M, K)) if dist == "normal"
         else rng.standard_t(3, (M, K))).astype(np.float32)
    B = rng.standard_normal((K, N)).astype(np.float32)
    (Ac, dA, BTc, dB), (oAc, odA, oBc, odB) = quantize_both(A, B, 128, b)
    cl = fm.int8_matmul_classical(Ac, dA, BTc, dB, 128).cpu().numpy()
    assert np.array_equal(bits(cl), bits(oracle.int8_classical(oAc, odA, oBc, odB, 128)))
    schemes = [s] if variants is None else variants
    ws = fm.workspace(fm.int8_workspace_size(schemes[0], M, N, K, levels, 128, 32, correct=True))
    for sc in schemes:
        out = fm.int8_matmul_corrected(sc, Ac, dA, BTc, dB, levels, 128, 32, b, b, ws=ws)
        fm.status(ws)
        assert np.array_equal(bits(out.cpu().numpy()), bits(cl))
    return (oAc, odA, oBc, odB), cl


def test_corrected_two_level_at_code_bound_127():
    """Sec. 4.3: with the overflow correction two-level Strassen computes
    classical int8 at code bound 127 bit for bit (blocks of 32, groups of
    128), as the oracle's corrected realization does."""
    say("[int8] corrected two-level Strassen 256x512x384, b=127")
    (oAc, odA, oBc, odB), cl = corrected_vs_classical(fm.Scheme.base("strassen"), 2, 256, 512,
                                                      384, 21)
    (U, V, W), dims = oracle.flatten_f32(so.power(osch.strassen(), 2))
    want, st = oracle.int8_fast_corrected(oAc, odA, oBc, odB, (U, V, W), dims, 128, 32)
    assert st["overflows"] > 0
    assert np.array_equal(bits(cl), bits(want))


def test_corrected_ragged_tiles_and_heavy_tails():
    say("[int8] corrected two-level Strassen 400x768x208, t(3), b=127")
    corrected_vs_classical(fm.Scheme.base("strassen"), 2, 400, 768, 208, 22, dist="t3")


def test_corrected_every_sign_variant():
    say("[int8] corrected: 512 sign variants 64x256x64, b=127")
    s2 = fm.Scheme.base("strassen").kron(2)
    orbit = s2.gauge_orbit([(np.diag(d), np.diag(e), np.diag(f)) for d, e, f in sy.sign_orbit(4, 4, 4)])
    corrected_vs_classical(None, 1, 64, 256, 64, 23, variants=orbit)


def test_corrected_layer_slice_at_full_size():
    """App. E's slice shape (512 token rows, 1024 output channels, inner
    dimension 13824, groups of 128, blocks of 32) on the heavy-tailed
    stand-in: corrected output equals classical int8 on every bit."""
    say("[int8] corrected slice down_512x13824x1024, b=127")
    w = sy.CORRECTION_SLICES["down_512x13824x1024"]
    A, B = sy.operands(w)
    s = fm.Scheme.base("strassen")
    Ac, dA = fm.int8_quantize(gpu(A), 128, 127)
    BTc, dB = fm.int8_quantize(gpu(np.ascontiguousarray(B.T)), 128, 127)
    cl = fm.int8_matmul_classical(Ac, dA, BTc, dB, 128)
    plan = fm.Int8Plan(s, w.M, w.N, w.K, 2, 128, 32, 127, 127, correct=True, device=DEV)
    out = plan.run(Ac, dA, BTc, dB)
    fm.status(plan.ws)
    assert torch.equal(out.view(torch.int32), cl.view(torch.int32))


def test_corrected_split_beyond_its_bound_is_reported():
    """Codes quantized at 127 but declared within 63: the certificate allows
    split parts |q| <= 1, block sums reach 2; the device reports FM_E_RANGE."""
    rng = np.random.default_rng(24)
    A = rng.standard_normal((64, 128)).astype(np.float32)
    B = rng.standard_normal((128, 64)).astype(np.float32)
    (Ac, dA, BTc, dB), _ = quantize_both(A, B, 128, 127)
    s = fm.Scheme.base("strassen")
    c = fm.int8_certify_corrected(s, 2, 63, 63, 32, 128)
    assert c["certified"] and c["qmax_A"] == 1
    ws = fm.workspace(fm.int8_workspace_size(s, 64, 64, 128, 2, 128, 32, correct=True))
    fm.int8_matmul_corrected(s, Ac, dA, BTc, dB, 2, 128, 32, 63, 63, ws=ws)
    with pytest.raises(fm.FmError) as e:
        fm.status(ws)
    assert e.value.name == "FM_E_RANGE"
