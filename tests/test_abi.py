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
HEADERS = [os.path.join(ROOT, "include", h) for h in sorted(os.listdir(os.path.join(ROOT, "include")))
           if h.endswith(".h")]


def declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*((?:ltlt|convgemm)_\w+)\s*\(", text, flags=re.M))
    return sorted(names)


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
                 "ltlt_set_cooperative_panels", "convgemm_f32", "convgemm_out_size"]:
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


# convgemm_f32(kn, kh, kw, ci, hi, wi, b, stride, pad, F, I, O, accumulate, path, mt, nt, stream)
CG_OK = (8, 3, 3, 2, 9, 9, 2, 1, 1, 1, 1, 1, 0, 0, 0, 0, NULL)


def _cg(**kw):
    names = ["kn", "kh", "kw", "ci", "hi", "wi", "b", "s", "p", "F", "I", "O", "acc", "path", "mt", "nt",
             "stream"]
    args = dict(zip(names, CG_OK))
    args.update(kw)
    return tuple(args[n] for n in names)


@pytest.mark.parametrize("args,code", [
    (_cg(kn=0), -1),
    (_cg(kh=0), -2),
    (_cg(kw=-1), -3),
    (_cg(ci=0), -4),
    (_cg(hi=0), -5),
    (_cg(wi=0), -6),
    (_cg(b=-1), -7),
    (_cg(s=0), -8),
    (_cg(p=-1), -9),
    (_cg(hi=1, kh=4, p=1), -5),                  # window taller than the padded input
    (_cg(wi=2, kw=5, p=1), -6),
    (_cg(hi=50000, wi=50000, ci=1), -5),         # input sample beyond 2^31 floats
    (_cg(kh=2, kw=1, ci=1 << 30, hi=1, wi=1, p=1), -2),  # kh kw ci = 2^31
    (_cg(hi=4000, wi=4000, kh=1, kw=1, ci=1, b=200), -7),  # ho wo b beyond 2^31
    (_cg(kn=2, kh=1, kw=1, ci=1 << 29, hi=1, wi=1, b=1, p=0), -1),  # filter tensor 2^30 elements
    (_cg(acc=2), -13),
    (_cg(path=3), -14),
    (_cg(path=-1), -14),
    (_cg(path=0, mt=64, nt=64), -14),           # automatic path takes no tile
    (_cg(path=2, p=1), -14),                    # register-direct: no padding
    (_cg(path=2, p=0, kh=3, kw=3, ci=1821, hi=9, wi=9), -14),   # register-direct: K <= 16384
    (_cg(path=1, mt=128, nt=64), -15),
    (_cg(path=1, mt=96, nt=128), -15),
    (_cg(path=2, p=0, mt=64, nt=256), -15),
    (_cg(path=2, p=0, mt=192, nt=128), -15),
    (_cg(F=NULL), -10),
    (_cg(I=NULL), -11),
    (_cg(O=NULL), -12),
    (_cg(b=0, F=NULL, I=NULL, O=NULL), 0),       # empty batch: nothing to do
])
def test_convgemm_argument_checks(lib, args, code):
    assert lib.convgemm_f32(*args) == code


def test_convgemm_out_size_matches_oracle():
    from oracle import conv as oc
    for h in range(1, 12):
        for k in range(1, 6):
            for s in range(1, 4):
                for p in range(0, 3):
                    try:
                        want = oc.out_size(h, k, s, p)
                    except ValueError:
                        want = -1
                    assert lib_out_size(h, k, s, p) == want
    assert lib_out_size(5, 0, 1, 0) == -1 and lib_out_size(5, 3, 0, 0) == -1 and lib_out_size(5, 3, 1, -1) == -1


def lib_out_size(h, k, s, p):
    return lt.load().convgemm_out_size(h, k, s, p)
