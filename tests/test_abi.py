"""The C ABI on the host (no GPU needed): the library loads, exports every symbol
include/kred.h declares, and rejects bad arguments before touching a device."""
import ctypes

import pytest

from paper_2004_11127_amd import kred

OK, INVALID, UNSUPPORTED, NO_DEVICE = 0, 1, 2, 5


@pytest.fixture(scope="module")
def lib():
    return kred.load()


def test_exports_every_declared_symbol(lib):
    names = kred.header_symbols()
    assert set(names) >= {"kred_create", "kred_destroy", "kred_run", "kred_validate",
                          "kred_scratch_bytes", "kred_profile_collect", "kred_strerror",
                          "kred_version"}
    for n in names:
        assert hasattr(lib, n), n


def test_version_and_strerror(lib):
    assert kred.version() == 1
    for code in range(6):
        assert kred.strerror(code)
    assert kred.strerror(0) == "success"
    assert kred.strerror(999) == "unknown status"


def test_create_rejects_bad_device(lib):
    h = ctypes.c_void_p()
    assert lib.kred_create(ctypes.byref(h), 4096) == NO_DEVICE
    assert lib.kred_create(None, 0) == INVALID
    assert lib.kred_destroy(None) == OK


def test_run_rejects_null_context(lib):
    p = kred.make_params(sigma=1.0)
    assert lib.kred_run(None, 0, 0, ctypes.byref(p), 4, 4, 3, 1, 16, 16, 16, 16, None) == INVALID


V = kred.validate


@pytest.mark.parametrize("formula,reduction,E,kw", [
    ("gauss", "sum", 1, dict(sigma=0.1)), ("gauss", "sum", 64, dict(sigma=2.0)),
    ("laplace", "sum", 3, dict(sigma=1.0)), ("sqdist", "sum", 7, {}),
    ("gauss_gradx", "sum", 1, dict(sigma=0.05)), ("sinkhorn", "lse", 1, dict(eps=0.01)),
])
def test_valid_pairs(lib, formula, reduction, E, kw):
    assert V(formula, reduction, 100, 200, 3, E, **kw) == OK


def test_valid_argkmin(lib):
    assert V("sqdist", "argkmin", 100, 200, 3, 0, b=None, K=10) == OK
    assert V("sqdist", "argkmin", 100, 64, 16, 0, b=None, K=64) == OK


@pytest.mark.parametrize("formula,reduction", [
    ("gauss", "kmin"), ("gauss", "argkmin"), ("laplace", "argkmin"), ("sinkhorn", "sum"),
    ("gauss_gradx", "lse"), ("sqdist", "lse")])
def test_unsupported_pairs(lib, formula, reduction):
    b = None if reduction in ("argkmin", "kmin") else 16
    assert V(formula, reduction, 10, 10, 3, 1, b=b, K=1, sigma=1.0, eps=1.0) == UNSUPPORTED


def test_invalid_arguments(lib):
    g = dict(sigma=1.0)
    assert V("gauss", "sum", -1, 10, 3, 1, **g) == INVALID          # M < 0
    assert V("gauss", "sum", 10, -1, 3, 1, **g) == INVALID          # N < 0
    assert V("gauss", "sum", 2**31, 10, 3, 1, **g) == INVALID       # M too large
    assert V("gauss", "sum", 10, 10, 0, 1, **g) == INVALID          # D < 1
    assert V("gauss", "sum", 10, 10, 257, 1, **g) == INVALID        # D > 256
    assert V("gauss", "sum", 10, 10, 3, 0, **g) == INVALID          # E < 1
    assert V("gauss", "sum", 10, 10, 3, 65, **g) == INVALID         # E > 64
    assert V("gauss", "sum", 10, 10, 3, 1, sigma=0.0) == INVALID    # sigma <= 0
    assert V("gauss", "sum", 10, 10, 3, 1, sigma=float("nan")) == INVALID
    assert V("laplace", "sum", 10, 10, 3, 1, sigma=-1.0) == INVALID
    assert V("gauss_gradx", "sum", 10, 10, 3, 2, **g) == INVALID    # gradient needs E = 1
    assert V("sinkhorn", "lse", 10, 10, 3, 1, eps=0.0) == INVALID
    assert V("sinkhorn", "lse", 10, 10, 3, 1, eps=float("inf")) == INVALID
    assert V("sinkhorn", "lse", 10, 10, 3, 2, eps=1.0) == INVALID
    assert V("sqdist", "argkmin", 10, 10, 3, 0, b=None, K=0) == INVALID
    assert V("sqdist", "argkmin", 10, 10, 3, 0, b=None, K=11) == INVALID   # K > N
    assert V("sqdist", "argkmin", 10, 100, 3, 0, b=None, K=65) == INVALID  # K > 64
    assert V("sqdist", "argkmin", 10, 10, 3, 0, b=16, K=3) == INVALID      # b must be NULL
    assert V("gauss", "sum", 10, 10, 3, 1, col_blocks=-1, **g) == INVALID
    assert V("gauss", "sum", 10, 10, 3, 1, col_blocks=257, **g) == INVALID
    assert V(7, "sum", 10, 10, 3, 1, **g) == INVALID                       # unknown formula
    assert V("gauss", 9, 10, 10, 3, 1, **g) == INVALID                     # unknown reduction


def test_pointer_rules(lib):
    g = dict(sigma=1.0)
    assert V("gauss", "sum", 10, 10, 3, 1, x=None, **g) == INVALID
    assert V("gauss", "sum", 10, 10, 3, 1, out=None, **g) == INVALID
    assert V("gauss", "sum", 10, 10, 3, 1, y=None, **g) == INVALID
    assert V("gauss", "sum", 10, 10, 3, 1, b=None, **g) == INVALID
    assert V("gauss", "sum", 10, 10, 3, 1, x=18, **g) == INVALID             # misaligned
    assert V("gauss", "sum", 10, 0, 3, 1, y=None, b=None, **g) == OK         # N = 0 needs no y, b
    assert V("gauss", "sum", 0, 10, 3, 1, x=None, y=None, b=None, out=None, **g) == OK  # M = 0


def test_unsupported_sizes_are_reported(lib):
    # pairs the library has no kernel for at this D report UNSUPPORTED, not a crash
    st = V("gauss_gradx", "sum", 10, 10, 200, 1, sigma=1.0)
    assert st in (OK, UNSUPPORTED)


def test_scratch_is_linear_not_quadratic(lib):
    # No M x N buffer: scratch grows linearly in M and N (Sec. 2 linear memory footprint).
    s1 = kred.scratch_bytes("gauss", "sum", 100_000, 100_000, 3, 1, sigma=0.1)
    s2 = kred.scratch_bytes("gauss", "sum", 1_000_000, 1_000_000, 3, 1, sigma=0.1)
    assert 0 < s1 and 0 < s2
    assert s2 < 40 * s1                       # 10x the points, far less than 100x the bytes
    assert s2 < 1_000_000 * 1_000_000 * 4 / 1000
    assert kred.scratch_bytes("gauss", "sum", 10, 10, 3, 0, sigma=0.1) == -1
    assert kred.scratch_bytes("gauss", "sum", 0, 10, 3, 1, sigma=0.1) == 0


# ------------------------------------------------------- Gaussian backward

VB = kred.validate_backward


def test_backward_declared_and_null_context(lib):
    assert {"kred_gauss_backward", "kred_validate_backward"} <= set(kred.header_symbols())
    p = kred.make_params(sigma=1.0)
    assert lib.kred_gauss_backward(None, ctypes.byref(p), 4, 4, 3, 1, 16, 16, 16, 16,
                                   16, 16, 16, None) == INVALID


def test_backward_valid_arguments(lib):
    assert VB(100, 200, 3, 1, sigma=0.1) == OK
    assert VB(100, 200, 16, 64, sigma=2.0) == OK
    assert VB(100, 200, 3, 5, gy=None, gb=None, sigma=0.1) == OK     # gx only
    assert VB(100, 200, 3, 5, gx=None, gy=None, b=None, sigma=0.1) == OK   # gb reads no b
    assert VB(100, 200, 3, 5, gx=None, gy=None, gb=None, x=None, y=None, b=None, e=None,
              sigma=0.1) == OK   # nothing requested
    # empty reductions read no input: the outputs are zero-filled
    assert VB(0, 200, 3, 2, x=None, y=None, b=None, e=None, sigma=0.1) == OK
    assert VB(100, 0, 3, 2, x=None, y=None, b=None, e=None, sigma=0.1) == OK


def test_backward_invalid_arguments(lib):
    assert VB(100, 200, 3, 1, sigma=0.0) == INVALID
    assert VB(100, 200, 3, 1, sigma=float("inf")) == INVALID
    assert VB(100, 200, 0, 1, sigma=1.0) == INVALID
    assert VB(100, 200, 3, 0, sigma=1.0) == INVALID
    assert VB(100, 200, 3, 65, sigma=1.0) == INVALID
    assert VB(-1, 200, 3, 1, sigma=1.0) == INVALID
    assert VB(100, 2 ** 31, 3, 1, sigma=1.0) == INVALID
    assert VB(100, 200, 3, 1, sigma=1.0, col_blocks=257) == INVALID
    assert VB(100, 200, 3, 1, b=None, sigma=1.0) == INVALID          # gx, gy need b
    assert VB(100, 200, 3, 1, e=None, sigma=1.0) == INVALID
    assert VB(100, 200, 3, 1, x=None, gx=None, gy=None, sigma=1.0) == INVALID   # gb needs x
    assert VB(100, 200, 3, 1, gx=18, sigma=1.0) == INVALID           # misaligned output
    assert VB(100, 200, 3, 1, e=2, sigma=1.0) == INVALID             # misaligned input


def test_backward_large_d(lib):
    # 16 < D <= 256 on the matrix cores, any E
    assert VB(100, 200, 17, 1, sigma=1.0) == OK
    assert VB(100, 200, 256, 1, sigma=1.0) == OK
    assert VB(100, 200, 64, 8, gx=None, gy=None, sigma=1.0) == OK
    assert VB(100, 200, 64, 8, sigma=1.0) == OK
    assert VB(100, 200, 256, 64, sigma=1.0) == OK
    assert VB(100, 200, 257, 1, sigma=1.0) == INVALID


def test_gradx_large_d(lib):
    V = kred.validate
    assert V("gauss_gradx", "sum", 100, 200, 17, 1, sigma=1.0) == OK
    assert V("gauss_gradx", "sum", 100, 200, 256, 1, sigma=1.0) == OK
    assert V("gauss_gradx", "sum", 100, 200, 64, 2, sigma=1.0) == INVALID
    assert kred.scratch_bytes("gauss_gradx", "sum", 1000, 2000, 128, 1, sigma=1.0) > \
        kred.scratch_bytes("gauss", "sum", 1000, 2000, 128, 1, sigma=1.0)


# ------------------------------------------------ min / max / arg-min / K-min

@pytest.mark.parametrize("red", ["min", "max", "argmin", "argmax"])
def test_extreme_pairs(lib, red):
    assert V("gauss", red, 100, 200, 3, 4, sigma=0.3) == OK
    assert V("laplace", red, 100, 200, 16, 64, sigma=0.3) == OK
    assert V("sqdist", red, 100, 200, 3, 2) == OK                  # with b
    assert V("sqdist", red, 100, 200, 3, 0, b=None) == OK          # F = d, E ignored
    assert V("sinkhorn", red, 100, 200, 3, 1, eps=0.1) == OK
    assert V("sinkhorn", red, 100, 200, 3, 2, eps=0.1) == INVALID  # one column
    assert V("gauss", red, 100, 200, 3, 4, b=None, sigma=0.3) == INVALID
    assert V("gauss", red, 100, 200, 3, 0, sigma=0.3) == INVALID
    assert V("gauss", red, 100, 200, 3, 1, sigma=0.0) == INVALID
    assert V("gauss_gradx", red, 100, 200, 3, 1, sigma=0.3) == UNSUPPORTED
    # D > 16: every min / max on the matrix cores
    assert V("gauss", red, 100, 200, 17, 1, sigma=0.3) == OK
    assert V("sqdist", red, 100, 200, 64, 0, b=None) == OK
    assert V("sinkhorn", red, 100, 200, 256, 1, eps=0.3) == OK
    assert V("gauss_gradx", red, 100, 200, 64, 1, sigma=0.3) == UNSUPPORTED


def test_kmin_pairs(lib):
    assert V("sqdist", "kmin", 100, 200, 3, 0, b=None, K=10) == OK
    assert V("sqdist", "kmin", 100, 200, 128, 0, b=None, K=64) == OK
    assert V("sqdist", "kmin", 100, 200, 3, 0, K=10) == INVALID          # b must be NULL
    assert V("sqdist", "kmin", 100, 5, 3, 0, b=None, K=10) == INVALID    # K > N
    assert V("sqdist", "kmin", 100, 0, 3, 0, b=None, K=1) == INVALID     # N = 0
    assert V("gauss", "kmin", 100, 200, 3, 0, b=None, K=10, sigma=1.0) == UNSUPPORTED
    assert V("sqdist", 8, 100, 200, 3, 0, b=None, K=10) == INVALID       # unknown reduction


def test_extreme_output_shapes(lib):
    assert kred.output_shape("gauss", "max", 10, 3, 4) == (10, 4)
    assert kred.output_shape("sqdist", "argmin", 10, 3, 0) == (10, 1)
    assert kred.output_shape("sinkhorn", "max", 10, 3, 1) == (10, 1)
    assert kred.output_shape("sqdist", "kmin", 10, 3, 0, K=7) == (10, 7)
    assert kred.scratch_bytes("sqdist", "min", 1000, 2000, 64, 0) > 0
    assert kred.scratch_bytes("sqdist", "argmax", 1000, 2000, 64, 0) > 0   # the farthest point, served at D > 16


def test_kernel_lse_pairs(lib):
    assert V("gauss", "lse", 100, 200, 3, 1, sigma=0.1) == OK
    assert V("laplace", "lse", 100, 200, 16, 1, sigma=0.1) == OK
    assert V("gauss", "lse", 100, 200, 3, 2, sigma=0.1) == INVALID
    assert V("laplace", "lse", 100, 200, 3, 1, sigma=0.0) == INVALID
    assert V("gauss", "lse", 100, 200, 3, 1, sigma=0.1, b=None) == INVALID
    assert V("sqdist", "lse", 100, 200, 3, 1) == UNSUPPORTED
    # 16 < D <= 256: every log-sum-exp on the matrix cores; the min / max family
    # beyond the nearest squared distance is not served there
    assert V("gauss", "lse", 100, 200, 17, 1, sigma=0.1) == OK
    assert V("sinkhorn", "lse", 100, 200, 256, 1, eps=0.1) == OK
    assert V("laplace", "lse", 100, 200, 17, 1, sigma=0.1) == OK
    assert V("sinkhorn", "max", 100, 200, 17, 1, eps=0.1) == OK
    assert V("gauss", "max", 100, 200, 17, 1, sigma=0.1) == OK
    assert V("sqdist", "lse", 100, 200, 17, 1) == UNSUPPORTED


def test_ranges_validation(lib):
    VR = kred.validate_ranges
    assert "kred_run_ranges" in kred.header_symbols()
    assert VR("gauss", "sum", 100, 200, 3, 1, 5, sigma=1.0) == OK
    assert VR("sqdist", "argkmin", 100, 200, 3, 0, 5, b=None, K=4) == OK
    assert VR("gauss", "sum", 100, 200, 3, 1, 0, rr=None, cp=None, cr=None, sigma=1.0) == OK
    assert VR("gauss", "sum", 100, 200, 3, 1, 5, cr=None, sigma=1.0) == INVALID
    assert VR("gauss", "sum", 100, 200, 3, 1, -1, sigma=1.0) == INVALID
    assert VR("gauss", "sum", 100, 200, 3, 1, 5, rr=2, sigma=1.0) == INVALID   # misaligned
    # the matrix-core path (16 < D <= 256) takes patterns for what kred_run accepts there
    assert VR("gauss", "sum", 100, 200, 17, 1, 5, sigma=1.0) == OK
    assert VR("sqdist", "argkmin", 100, 200, 64, 0, 5, b=None, K=10) == OK
    assert VR("gauss", "lse", 100, 200, 17, 1, 5, sigma=1.0) == OK
    assert VR("laplace", "lse", 100, 200, 17, 1, 5, sigma=1.0) == OK
    assert VR("gauss", "min", 100, 200, 17, 1, 5, sigma=1.0) == OK
    assert VR("gauss", "sum", 100, 200, 257, 1, 5, sigma=1.0) == INVALID        # as kred_run
    assert VR("gauss", "sum", 100, 200, 3, 1, 5, sigma=0.0) == INVALID         # as kred_run


def test_backward_ranges_validation(lib):
    VBR = kred.validate_backward_ranges
    assert {"kred_gauss_backward_ranges", "kred_validate_backward_ranges"} <= set(kred.header_symbols())
    p = kred.make_params(sigma=1.0)
    assert lib.kred_gauss_backward_ranges(None, ctypes.byref(p), 4, 4, 3, 1, 16, 16, 16, 16, 16, 16,
                                          16, 1, 16, 16, 16, 1, 16, 16, 16, None) == INVALID
    assert VBR(100, 200, 3, 1, 5, 7, sigma=0.1) == OK
    assert VBR(100, 200, 16, 40, 5, 7, sigma=0.1) == OK
    # a pattern's arrays are only needed by the outputs it serves
    assert VBR(100, 200, 3, 1, 5, 7, cc=None, rp=None, rt=None, gy=None, gb=None, sigma=0.1) == OK
    assert VBR(100, 200, 3, 1, 5, 7, rr=None, cp=None, cr=None, gx=None, sigma=0.1) == OK
    assert VBR(100, 200, 3, 1, 0, 0, rr=None, cp=None, cr=None, cc=None, rp=None, rt=None,
               sigma=0.1) == OK
    assert VBR(100, 200, 3, 1, 5, 7, cr=None, sigma=0.1) == INVALID
    assert VBR(100, 200, 3, 1, 5, 7, rt=None, gy=None, sigma=0.1) == INVALID    # gb needs it
    assert VBR(100, 200, 3, 1, -1, 7, sigma=0.1) == INVALID
    assert VBR(100, 200, 3, 1, 5, -1, sigma=0.1) == INVALID
    assert VBR(100, 200, 3, 1, 5, 7, rp=2, sigma=0.1) == INVALID                # misaligned
    # the dense backward's rules
    assert VBR(100, 200, 3, 1, 5, 7, sigma=0.0) == INVALID
    assert VBR(100, 200, 17, 4, 5, 7, sigma=1.0) == OK
    assert VBR(100, 200, 3, 1, 5, 7, b=None, sigma=1.0) == INVALID
