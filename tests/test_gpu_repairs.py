"""GPU parity of the repairs (App. C, the repair rules) on the group-scale
schedule, through the C ABI (FM_REPAIR_ROWS, FM_REPAIR_WEIGHTS OR-ed into
FM_SCALE_GROUP), against the CPU oracle on the same seeded inputs.

Bars as for the group scales: codes and scales bit-exact (with row scaling
the codes of the rescaled rows; with joint rounding the jointly chosen
codes), C within 5e-4 relative Frobenius of the oracle's (bf16 products),
orbit errors within 1%.  Row scaling's covariance with a power of two on a
single row of A holds bit for bit on the device.
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
SG = fm.SCALE_GROUP
TOL = 5e-4
FLAGS = {"rows": (fm.REPAIR_ROWS, oracle.REPAIR_ROWS),
         "weights": (fm.REPAIR_WEIGHTS, oracle.REPAIR_WEIGHTS),
         "both": (fm.REPAIR_ROWS | fm.REPAIR_WEIGHTS, oracle.REPAIR_ROWS | oracle.REPAIR_WEIGHTS)}


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


def operands(M, K, N, seed):
    rng = np.random.default_rng(seed)
    A = rng.standard_t(3, (M, K)).astype(np.float32)
    A[rng.choice(M, M // 4, replace=False)] *= np.float32(20.0)   # rows of mixed magnitude
    A[:, rng.choice(K, 4, replace=False)] *= np.float32(30.0)     # outlier channels
    B = (0.02 * rng.standard_normal((K, N))).astype(np.float32)
    return A, B


CASES = [
    # name, base, levels, gauge, M, K, N, fmt, which.  Kronecker powers and
    # sign gauges keep a family's structure (the kernel specialized for it);
    # a GL gauge on A's side alone leaves B's lists as they were but not A's
    # and C's, so the joint rounding takes the generic kernel
    ("strassen2_rows", "strassen", 2, None, 256, 512, 512, "e4m3", "rows"),
    ("strassen2_weights", "strassen", 2, None, 256, 512, 512, "e4m3", "weights"),
    ("strassen2_both_two_groups", "strassen", 2, None, 128, 1024, 512, "e4m3", "both"),
    ("strassen1_both", "strassen", 1, None, 192, 256, 256, "e4m3", "both"),
    ("strassen2_sign_weights_e5m2", "strassen", 2, "sign", 128, 512, 512, "e5m2", "weights"),
    ("laderman_both", "laderman", 1, None, 192, 384, 384, "e4m3", "both"),
    ("strassen1_gl_on_a_generic", "strassen", 1, "gl_a", 128, 256, 512, "e4m3", "weights"),
]
FMT = {"e4m3": (fm.E4M3, oracle.E4M3), "e5m2": (fm.E5M2, oracle.E5M2)}


def schemes_for(base, levels, gauge, seed):
    """The library's scheme and the oracle's, flattened when gauged by signs
    (then evaluated at one level)."""
    hb, ob = fm.Scheme.base(base), osch.BASE_SCHEMES[base]()
    if gauge is None:
        return hb, so.power(ob, levels), levels
    if gauge == "sign":
        g = 2 ** levels
        d, e, f = sy.sample_sign_orbit(g, g, g, 3, seed=seed)[-1]  # not the identity
        D, E, F = np.diag(d), np.diag(e), np.diag(f)
        return hb.kron(levels).gauge(D, E, F), so.gauge(so.power(ob, levels), D, E, F), 1
    X = sy.gl_gauges(2, 2, 2, 1, seed=seed)[0][0]
    I2 = np.eye(2)
    assert levels == 1
    return hb.gauge(X, I2, I2), so.gauge(ob, X, I2, I2), 1


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_repair_parity(case):
    name, base, levels, gauge, M, K, N, fmt, which = case
    fh, fo = FLAGS[which]
    th, to = FMT[fmt]
    say(f"[repairs] {name} {M}x{K}x{N} {fmt}")
    A, B = operands(M, K, N, sum(name.encode()))
    At, Bt = gpu(A), gpu(B)
    s, o, lv = schemes_for(base, levels, gauge, seed=sum(name.encode()))
    fam = s.kernel_family(lv)
    assert (fam == "generic") == (gauge == "gl_a"), fam
    tabs, dims = oracle.flatten_f32(o)
    want = oracle.lowp_matmul_repaired(A, B, tabs, dims, fmt=to, flags=fo, keep=True)
    Tq, Sq, dT, dS = fm.form_operands(s, At, Bt, lv, th, scale_mode=SG | fh)
    assert np.array_equal(Tq.cpu().numpy(), want["Tq"]), "Tq"
    assert np.array_equal(bits(dT.cpu().numpy()), bits(want["dT"])), "dT"
    assert np.array_equal(Sq.cpu().numpy(), want["Sq"].transpose(0, 2, 1)), "Sq"
    assert np.array_equal(bits(dS.cpu().numpy()), bits(want["dS"])), "dS"
    C = fm.matmul_lowp(s, At, Bt, lv, th, scale_mode=SG | fh).cpu().numpy()
    assert rel(C, want["C"]) <= TOL, f"C: {rel(C, want['C']):.2e}"
    # the orbit path (errors fused in the reconstruction) agrees with C
    Cref = fm.reference_f64(At, Bt)
    err = fm.orbit_eval([s.kron(lv) if lv > 1 else s], At, Bt, Cref, 1, th,
                        scale_mode=SG | fh)[0]
    assert abs(err / oracle.rel_fro(want["C"], oracle.reference_f64(A, B)) - 1) <= 1e-2


def test_row_scaling_covariance_on_the_device():
    s = fm.Scheme.base("strassen")
    A, B = operands(64, 512, 512, 5)
    Bt = gpu(B)
    mode = SG | fm.REPAIR_ROWS
    C = fm.matmul_lowp(s, gpu(A), Bt, 2, scale_mode=mode).cpu().numpy()
    for t, p in ((5, 8.0), (40, 0.25)):
        A2 = A.copy()
        A2[t] *= np.float32(p)
        C2 = fm.matmul_lowp(s, gpu(A2), Bt, 2, scale_mode=mode).cpu().numpy()
        others = [r for r in range(64) if r != t]
        assert np.array_equal(bits(C2[t]), bits(C[t] * np.float32(p)))
        assert np.array_equal(bits(C2[others]), bits(C[others]))


def test_repairs_need_the_group_schedule():
    s = fm.Scheme.base("strassen")
    A, B = operands(64, 512, 512, 6)
    with pytest.raises(fm.FmError) as e:
        fm.matmul_lowp(s, gpu(A), gpu(B), 2, scale_mode=fm.SCALE_ROWCOL | fm.REPAIR_ROWS,
                       ws=fm.workspace(1 << 26))
    assert e.value.name == "FM_E_ARG"
