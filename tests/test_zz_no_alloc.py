"""The allocation-free error statistics (fm_error_stats_noalloc) against
fm_error_stats with a caller's workspace: the same kernels and sums, so the
results must agree bit for bit.  Two calls in a row, the second on a
smaller output, so the second reuses the static scratch the first left
behind (and a third on a large output uses every partial slot)."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU-only machines, never run
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2609_39816_amd import fm  # noqa: E402

DEV = torch.device("cuda:0")


def same_bits(a, b):
    return np.float64(a).view(np.uint64) == np.float64(b).view(np.uint64)


def case(M, N, seed):
    print(f"[noalloc] M={M} N={N} seed={seed}", flush=True)
    sys.stdout.flush()
    rng = np.random.default_rng(seed)
    ref = rng.standard_normal((M, N))
    C = (ref + 1e-3 * rng.standard_normal((M, N))).astype(np.float32)
    Ct = torch.from_numpy(C).to(DEV)
    Rt = torch.from_numpy(ref).to(DEV)
    want = fm.error_stats(Ct, Rt)
    got = fm.error_stats_noalloc(Ct, Rt)
    for k in ("err_sq", "ref_sq", "max_abs", "rel_fro"):
        assert same_bits(got[k], want[k]), (M, N, k, got[k], want[k])
    # an independent float64 check of the definition (App. B.1's error)
    d = C.astype(np.float64) - ref
    e = float(np.sqrt((d * d).sum()) / np.sqrt((ref * ref).sum()))
    assert abs(got["rel_fro"] / e - 1) <= 1e-12
    assert got["max_abs"] == float(np.abs(d).max())
    return got


def test_noalloc_error_stats_matches_workspace_version():
    case(1536, 2304, 1)   # more than 1024 x 256 entries: every partial slot used
    case(96, 80, 2)       # smaller, right after: partial slots of the first call remain
    case(1, 1, 3)         # one entry: one partial


def test_noalloc_error_stats_rejects_bad_arguments():
    C = torch.zeros((4, 4), dtype=torch.float32, device=DEV)
    R = torch.zeros((4, 4), dtype=torch.float64, device=DEV)
    st = fm._Stats()
    rc = fm.lib.fm_error_stats_noalloc(None, fm._dptr(R), 4, 4, fm.ct.byref(st), None)
    assert fm.ERRORS[rc] == "FM_E_ARG"
    rc = fm.lib.fm_error_stats_noalloc(fm._dptr(C), fm._dptr(R), 0, 4, fm.ct.byref(st), None)
    assert fm.ERRORS[rc] == "FM_E_ARG"
    # an all-zero reference: error 0 relative by convention, sums exact
    got = fm.error_stats_noalloc(C, R)
    assert got["rel_fro"] == 0.0 and got["err_sq"] == 0.0 and got["ref_sq"] == 0.0
