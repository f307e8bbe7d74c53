"""The Python binding checks the shapes of the tensors it passes: the C ABI
sees only pointers and sizes, so a B with fewer rows than A has columns, an
output or reference of the wrong shape, or block products that do not match
M and N would otherwise be read or written out of bounds on the device.
Every case here is refused with ValueError before any library call."""
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU-only machines, never run
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2609_39816_amd import fm  # noqa: E402

DEV = torch.device("cuda:0")


def z(shape, dtype=torch.float32):
    return torch.zeros(shape, dtype=dtype, device=DEV)


def test_mismatched_shapes_are_refused():
    s = fm.Scheme.base("strassen")
    A, B_bad, B = z((64, 64)), z((48, 64)), z((64, 64))
    for call in (lambda: fm.reference_f64(A, B_bad),
                 lambda: fm.matmul_lowp(s, A, B_bad),
                 lambda: fm.form_operands(s, A, B_bad),
                 lambda: fm.reference_f64(A, B, out=z((64, 8), torch.float64)),
                 lambda: fm.matmul_lowp(s, A, B, out=z((32, 64))),
                 lambda: fm.orbit_eval([s], A, B, z((64, 8), torch.float64)),
                 lambda: fm.orbit_eval([], A, B, z((64, 64), torch.float64)),
                 lambda: fm.error_stats(z((64, 64)), z((64, 8), torch.float64)),
                 lambda: fm.error_stats_noalloc(z((64, 16)), z((16, 64), torch.float64)),
                 lambda: fm.block_products(z((2, 16, 32), torch.uint8), z((2, 16, 16), torch.uint8),
                                           z(2) + 1, z(2) + 1),
                 lambda: fm.block_products(z((2, 16, 32), torch.uint8), z((2, 16, 32), torch.uint8),
                                           z(2) + 1, z(2) + 1, out=z((2, 16, 8))),
                 # one level of Strassen on 64 x 64: 7 products of 32 x 32
                 lambda: fm.reconstruct(s, z((7, 32, 16)), 64, 64),
                 lambda: fm.matmul_lowp(s, A, B, ws=z((1024, 1024)).t())):
        with pytest.raises(ValueError):
            call()


def test_matching_shapes_still_run():
    s = fm.Scheme.base("strassen")
    g = torch.Generator(device=DEV)
    g.manual_seed(3)
    A = torch.randn((64, 64), device=DEV, generator=g)
    B = torch.randn((64, 64), device=DEV, generator=g)
    Cref = fm.reference_f64(A, B, out=z((64, 64), torch.float64))
    C = fm.matmul_lowp(s, A, B, out=z((64, 64)))
    assert fm.error_stats(C, Cref)["rel_fro"] < 0.2
    errs = fm.orbit_eval([s], A, B, Cref)
    assert errs.shape == (1,) and 0 < errs[0] < 0.2
