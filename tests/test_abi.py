"""The C-ABI library loads and exports every symbol ``include/ltlt.h``
declares; host-side argument checks reject bad calls before any GPU work.
No compute call is made here (no GPU needed)."""
import ctypes
import os
import re

import pytest

import paper_2005_06410_amd as lt
from paper_2005_06410_amd import build as ltbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ltlt.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(ltlt_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(lt.LIB_PATH):
        ltbuild.build()
    return lt.load()


def test_header_declares_the_entry_points():
    names = declared_functions()
    for must in ["ltlt_factor", "ltlt_factor_nb", "ltlt_pfaffian", "ltlt_factor_batched",
                 "ltlt_skew_update", "ltlt_device_status", "ltlt_profile_enable",
                 "ltlt_profile_read", "ltlt_release_workspace", "ltlt_mfma_probe",
                 "ltlt_pfaffian_direct", "ltlt_solve", "ltlt_pfaffian_complex",
                 "ltlt_set_cooperative_panels"]:
        assert must in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert isinstance(getattr(lib, name), ctypes._CFuncPtr)


def test_binding_covers_every_declared_symbol():
    assert set(declared_functions()) == set(lt._SYMBOLS)


def test_library_is_built_for_gfx950_only():
    out = os.popen(f"/opt/rocm/llvm/bin/clang-offload-bundler --list --type=o --input={lt.LIB_PATH} 2>/dev/null"
                   ).read()
    if not out.strip():
        pytest.skip("offload bundle listing unavailable")
    assert "gfx950" in out


NULL = None


@pytest.mark.parametrize("args,code", [
    ((-1, 1, 1, 0, 1, 128, NULL), -1),          # n < 0
    ((4, NULL, 4, 0, 1, 128, NULL), -2),        # A null
    ((4, 1, 3, 0, 1, 128, NULL), -3),           # lda < n
    ((4, 1, 4, 7, 1, 128, NULL), -4),           # bad dtype
    ((4, 1, 4, 0, NULL, 128, NULL), -5),        # ipiv null
    ((4, 1, 4, 0, 1, 0, NULL), -6),             # nb < 1
    ((4, 1, 4, 0, 1, 257, NULL), -6),           # nb too wide
    ((0, NULL, 1, 0, NULL, 128, NULL), 0),      # n = 0 is a no-op
    ((4, 1, 4, 4, 1, 64, NULL), -4),            # no such dtype
    ((4, 1, 4, 2, 1, 129, NULL), -6),           # complex panel holds at most 128 steps
    ((4, 1, 4, 3, 1, 0, NULL), -6),
    ((0, NULL, 1, 2, NULL, 64, NULL), 0),       # complex n = 0
])
def test_factor_argument_checks(lib, args, code):
    assert lib.ltlt_factor_nb(*args) == code


@pytest.mark.parametrize("args,code", [
    ((65, 1, 1, 65, 65 * 65, 0, 1, 65, 1, 1, NULL), -1),     # n above the batched limit
    ((4, -1, 1, 4, 16, 0, 1, 4, 1, 1, NULL), -2),            # batch < 0
    ((4, 2, NULL, 4, 16, 0, 1, 4, 1, 1, NULL), -3),          # A null
    ((4, 2, 1, 3, 16, 0, 1, 4, 1, 1, NULL), -4),             # lda < n
    ((4, 2, 1, 4, 15, 0, 1, 4, 1, 1, NULL), -5),             # overlapping matrices
    ((4, 2, 1, 4, 16, 2, 1, 4, 1, 1, NULL), -6),             # bad dtype
    ((4, 2, 1, 4, 16, 0, NULL, 4, 1, 1, NULL), -7),          # ipiv null
    ((4, 2, 1, 4, 16, 0, 1, 3, 1, 1, NULL), -8),             # pivot stride < n
    ((4, 2, 1, 4, 16, 0, 1, 4, NULL, 1, NULL), -9),          # logabs null
    ((4, 2, 1, 4, 16, 0, 1, 4, 1, NULL, NULL), -10),         # sign null
    ((4, 0, NULL, 4, 16, 0, NULL, 4, NULL, NULL, NULL), 0),  # empty batch
])
def test_batched_argument_checks(lib, args, code):
    assert lib.ltlt_factor_batched(*args) == code


@pytest.mark.parametrize("args,code", [
    ((-1, 1, 1, 0, 1, NULL, NULL, NULL), -1),
    ((4, NULL, 4, 0, 1, 1, 1, NULL), -2),
    ((4, 1, 2, 0, 1, 1, 1, NULL), -3),
    ((4, 1, 4, 3, 1, 1, 1, NULL), -4),
    ((4, 1, 4, 0, NULL, 1, 1, NULL), -5),
    ((4, 1, 4, 0, 1, NULL, 1, NULL), -6),
    ((4, 1, 4, 0, 1, 1, NULL, NULL), -7),
])
def test_pfaffian_argument_checks(lib, args, code):
    assert lib.ltlt_pfaffian(*args) == code


@pytest.mark.parametrize("args,code", [
    ((-1, 1, 1, 2, 1, 1, 1, NULL), -1),
    ((4, NULL, 4, 2, 1, 1, 1, NULL), -2),
    ((4, 1, 2, 2, 1, 1, 1, NULL), -3),
    ((4, 1, 4, 0, 1, 1, 1, NULL), -4),          # real dtype: ltlt_pfaffian's job
    ((4, 1, 4, 2, NULL, 1, 1, NULL), -5),
    ((4, 1, 4, 3, 1, NULL, 1, NULL), -6),
    ((4, 1, 4, 3, 1, 1, NULL, NULL), -7),
])
def test_pfaffian_complex_argument_checks(lib, args, code):
    assert lib.ltlt_pfaffian_complex(*args) == code


@pytest.mark.parametrize("dtype", [2, 3])
def test_complex_dtypes_refused_where_not_supported(lib, dtype):
    assert lib.ltlt_pfaffian(4, 1, 4, dtype, 1, 1, 1, NULL) == -4
    assert lib.ltlt_pfaffian_direct(4, 1, 4, dtype, 1, 0, 1, 1, NULL) == -4
    assert lib.ltlt_solve(4, 1, 4, dtype, 1, 1, 1, 4, NULL) == -4
    assert lib.ltlt_factor_batched(4, 2, 1, 4, 16, dtype, 1, 4, 1, 1, NULL) == -6
    assert lib.ltlt_skew_update(5, 1, 5, NULL, 2, 1, 5, 1, 5, dtype, NULL) == -10


@pytest.mark.parametrize("args,code", [
    ((-1, 1, 1, NULL, 1, 1, 1, 1, 1, 0, NULL), -1),
    ((5, NULL, 5, NULL, 1, 1, 5, 1, 5, 0, NULL), -2),
    ((5, 1, 4, NULL, 1, 1, 5, 1, 5, 0, NULL), -3),
    ((5, 1, 5, NULL, -1, 1, 5, 1, 5, 0, NULL), -5),
    ((5, 1, 5, NULL, 2, NULL, 5, 1, 5, 0, NULL), -6),
    ((5, 1, 5, NULL, 2, 1, 4, 1, 5, 0, NULL), -7),
    ((5, 1, 5, NULL, 2, 1, 5, NULL, 5, 0, NULL), -8),
    ((5, 1, 5, NULL, 2, 1, 5, 1, 4, 0, NULL), -9),
    ((5, 1, 5, NULL, 2, 1, 5, 1, 5, 9, NULL), -10),
    ((1, 1, 1, NULL, 2, 1, 1, 1, 1, 0, NULL), 0),            # m < 2: nothing to update
])
def test_skew_update_argument_checks(lib, args, code):
    assert lib.ltlt_skew_update(*args) == code


@pytest.mark.parametrize("args,code", [
    ((7, 10, "ok"), -1),           # bad dtype
    ((0, 0, "ok"), -2),            # iters < 1
    ((0, 100000001, "ok"), -2),    # iters > 1e8
    ((1, 10, None), -3),           # tflops NULL
])
def test_mfma_probe_argument_checks(lib, args, code):
    dtype, iters, ptr = args
    out = ctypes.c_double(0.0)
    assert lib.ltlt_mfma_probe(dtype, iters, ctypes.addressof(out) if ptr else None, None) == code


@pytest.mark.parametrize("args,code", [
    ((-1, 1, 1, 0, 1, 0, 1, 1, NULL), -1),
    ((4, NULL, 4, 0, 1, 0, 1, 1, NULL), -2),
    ((4, 1, 3, 0, 1, 0, 1, 1, NULL), -3),
    ((4, 1, 4, 5, 1, 0, 1, 1, NULL), -4),
    ((4, 1, 4, 0, NULL, 0, 1, 1, NULL), -5),
    ((4, 1, 4, 0, 1, 3, 1, 1, NULL), -6),       # odd nb
    ((4, 1, 4, 0, 1, 258, 1, 1, NULL), -6),     # nb above the widest panel
    ((4, 1, 4, 0, 1, -2, 1, 1, NULL), -6),
    ((4, 1, 4, 0, 1, 0, NULL, 1, NULL), -7),
    ((4, 1, 4, 0, 1, 0, 1, NULL, NULL), -8),
])
def test_pfaffian_direct_argument_checks(lib, args, code):
    assert lib.ltlt_pfaffian_direct(*args) == code


@pytest.mark.parametrize("args,code", [
    ((-1, 1, 1, 0, 1, 1, 1, 1, NULL), -1),
    ((4, NULL, 4, 0, 1, 1, 1, 4, NULL), -2),
    ((4, 1, 3, 0, 1, 1, 1, 4, NULL), -3),
    ((4, 1, 4, 9, 1, 1, 1, 4, NULL), -4),
    ((4, 1, 4, 0, NULL, 1, 1, 4, NULL), -5),
    ((4, 1, 4, 0, 1, -1, 1, 4, NULL), -6),
    ((4, 1, 4, 0, 1, 1, NULL, 4, NULL), -7),
    ((4, 1, 4, 0, 1, 1, 1, 3, NULL), -8),
    ((5, 1, 5, 0, 1, 1, 1, 5, NULL), -4000),     # odd order: singular
    ((0, NULL, 1, 0, NULL, 1, NULL, 1, NULL), 0),  # nothing to solve
    ((4, 1, 4, 0, 1, 0, NULL, 4, NULL), 0),        # no right-hand side
])
def test_solve_argument_checks(lib, args, code):
    assert lib.ltlt_solve(*args) == code


def test_error_messages():
    assert "argument 3" in str(lt.LtltError("f", -3))
    assert "HIP runtime error 2" in str(lt.LtltError("f", -1002))
    assert "not supported" in str(lt.LtltError("f", -2000))
    assert "bounded wait" in str(lt.LtltError("f", -3000))


def test_profile_enable_is_host_only(lib):
    assert lib.ltlt_set_cooperative_panels(2) == -1
    assert lib.ltlt_set_cooperative_panels(1) == 0
    assert lib.ltlt_set_cooperative_panels(0) == 0   # back to the default
    assert lib.ltlt_profile_enable(1) == 0
    assert lib.ltlt_profile_enable(2) == 0          # trailing updates only
    assert lib.ltlt_profile_enable(0) == 0
    assert lib.ltlt_profile_enable(3) == -1
    assert lib.ltlt_profile_enable(-1) == -1
