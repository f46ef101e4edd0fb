"""Host-side checks of the C ABI: exports, the host coefficient function, argument validation.

Nothing here launches a kernel: validation failures return before any HIP call, and
zo_probe_coeffs is host code.
"""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
import paper_2609_38095_amd as zo

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(zo.LIB_PATH):
        pytest.fail("libzo.so is not built (run __graft_entry__.build())")
    return zo.library()


def _declared_functions(header="zo.h"):
    text = open(os.path.join(ROOT, "include", header)).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(zo_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared_functions()
    for must in ("zo_perturb", "zo_update", "zo_probe_coeffs"):
        assert must in names


def test_library_exports_every_declared_symbol(lib):
    for name in _declared_functions():
        assert hasattr(lib, name), name
    assert set(zo.EXPORTS) == set(_declared_functions())


def test_calibration_library_exports_its_header():
    path = os.path.join(os.path.dirname(zo.LIB_PATH), "libzo_calib.so")
    if not os.path.exists(path):
        pytest.fail("libzo_calib.so is not built (run __graft_entry__.build())")
    calib = ctypes.CDLL(path)
    names = _declared_functions("zo_calib.h")
    assert names == ["zo_calib_rmw", "zo_calib_rmw_shape"]
    calib.zo_calib_rmw.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p]
    calib.zo_calib_rmw_shape.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32,
                                         ctypes.c_void_p]
    # validation returns before any HIP call
    assert calib.zo_calib_rmw(None, 0, 1, None) == 0
    assert calib.zo_calib_rmw(None, 16, 1, None) == -1
    assert calib.zo_calib_rmw(ctypes.c_void_p(0x1008), 16, 1, None) == -2
    assert calib.zo_calib_rmw(ctypes.c_void_p(0x1000), 24, 1, None) == -2
    assert calib.zo_calib_rmw_shape(None, 16, 1, 7, None) == -1
    assert calib.zo_calib_rmw_shape(ctypes.c_void_p(0x1000), 16, 1, 8, None) == -2
    assert calib.zo_calib_rmw_shape(ctypes.c_void_p(0x1000), 1 << 41, 1, 0, None) == -2


def test_header_constants_match_binding():
    text = open(os.path.join(ROOT, "include", "zo.h")).read()
    assert int(re.search(r"#define ZO_K_MAX (\d+)u", text).group(1)) == zo.ZO_K_MAX
    assert 1 << int(re.search(r"#define ZO_N_MAX \(1ull << (\d+)\)", text).group(1)) == zo.ZO_N_MAX
    for name, val in [("ZO_ERR_NULL", zo.ZO_ERR_NULL), ("ZO_ERR_ARG", zo.ZO_ERR_ARG),
                      ("ZO_ERR_NONFINITE", zo.ZO_ERR_NONFINITE), ("ZO_ERR_HIP", zo.ZO_ERR_HIP)]:
        assert int(re.search(name + r"\s*=\s*(-?\d+)", text).group(1)) == val


def _coeff_cases():
    rng = np.random.default_rng(0)
    cases = []
    for K in (1, 2, 4, 16, 64, 257):
        cases.append((rng.normal(2, 0.05, K), rng.normal(2, 0.05, K), 2.0 + 0.01 * rng.standard_normal(), 1e-3, 0.1, 1.0))
    cases.append((rng.normal(2, 0.05, 60), rng.normal(2, 0.05, 60), 1.99, 1e-4, 0.1, 1.0))  # paper's eps = lr = 1e-4
    cases.append(([52.0], [50.0], 1.0, 1e-3, 0.1, 1.0))                 # |chat| = 1e8
    cases.append(([1.0 + 1e-7], [1.0 - 1e-7], 1.0, 1e-3, 0.1, 1.0))     # |chat| ~ 0
    cases.append(([3.0, -1.0], [2.0, 5.0], 1.0, 0.5, 0.0, 1.0))         # alpha 0
    cases.append(([3.0, -1.0], [2.0, 5.0], 1.0, 0.5, 1.0, 1.0))         # alpha 1
    cases.append(([3.0, -1.0], [2.0, 5.0], 1.0, 0.5, 0.5, 2.5))         # lambda_reg 2.5
    cases.append(([1e300, -1e300], [-1e300, 1e300], 0.0, 1e-3, 0.1, 1.0))  # overflow to inf inside
    cases.append(([2.0], [1.0], 1.0, 1e-170, 0.1, 1.0))                 # eps^2 underflows
    cases.append(([1.0], [1.0], 1.0, 1e-3, 0.1, 1.0))                   # chat exactly 1 -> w 1
    return cases


@pytest.mark.parametrize("case", _coeff_cases())
def test_probe_coeffs_bit_exact_vs_oracle(lib, case):
    lp, lm, l0, eps, alpha, lam = case
    with np.errstate(all="ignore"):
        want = oracle.probe_coeffs(lp, lm, l0, eps, alpha, lam)
        got = zo.zo_probe_coeffs_ex(lp, lm, l0, eps, alpha, lam)
    for key in ("c", "c64", "curv", "w"):
        a, b = got[key], want[key]
        assert a.dtype == b.dtype
        np.testing.assert_array_equal(a.view(np.uint8), b.view(np.uint8), err_msg=key)
    if alpha == 0.1 and lam == 1.0:
        np.testing.assert_array_equal(zo.zo_probe_coeffs(lp, lm, l0, eps), want["c"])


def test_probe_coeffs_errors(lib):
    ok = dict(L_plus=[1.0], L_minus=[0.9], L_clean=1.0, eps=1e-3, alpha=0.1, lambda_reg=1.0)
    bad = [(dict(eps=0.0), zo.ZO_ERR_ARG), (dict(eps=-1.0), zo.ZO_ERR_ARG), (dict(alpha=1.5), zo.ZO_ERR_ARG),
           (dict(alpha=-0.5), zo.ZO_ERR_ARG), (dict(lambda_reg=0.0), zo.ZO_ERR_ARG),
           (dict(eps=float("nan")), zo.ZO_ERR_NONFINITE), (dict(L_plus=[float("inf")]), zo.ZO_ERR_NONFINITE),
           (dict(L_clean=float("nan")), zo.ZO_ERR_NONFINITE), (dict(L_plus=[], L_minus=[]), zo.ZO_ERR_ARG)]
    for change, code in bad:
        args = dict(ok, **change)
        with pytest.raises(zo.ZoError) as ei:
            zo.zo_probe_coeffs_ex(**args)
        assert ei.value.status == code, change
    # a NULL output array is refused and nothing is written
    d = (ctypes.c_double * 1)(1.0)
    assert lib.zo_probe_coeffs(d, d, 1, 1.0, 1e-3, None) == zo.ZO_ERR_NULL
    assert lib.zo_probe_coeffs_ex(None, d, 1, 1.0, 1e-3, 0.1, 1.0, None, None, None, None) == zo.ZO_ERR_NULL


def test_probe_coeffs_outputs_untouched_on_error(lib):
    d = (ctypes.c_double * 2)(1.0, float("nan"))
    out = (ctypes.c_float * 2)(7.0, 7.0)
    assert lib.zo_probe_coeffs(d, d, 2, 1.0, 1e-3, out) == zo.ZO_ERR_NONFINITE
    assert list(out) == [7.0, 7.0]


def test_sweep_validation_returns_before_launch(lib):
    """Invalid sweep arguments are refused synchronously (no device is touched here)."""
    c1 = (ctypes.c_float * 1)(1.0)
    big = (ctypes.c_float * (zo.ZO_K_MAX + 1))()
    cnan = (ctypes.c_float * 1)(float("nan"))
    fake = ctypes.c_void_p(0x10000)  # never dereferenced: every call below fails validation
    odd = ctypes.c_void_p(0x10001)
    assert lib.zo_perturb(None, 0, 0, 10, 0, 0, 0, 1e-3, None) == zo.ZO_ERR_NULL
    assert lib.zo_perturb(fake, 7, 0, 10, 0, 0, 0, 1e-3, None) == zo.ZO_ERR_ARG
    assert lib.zo_perturb(odd, zo.ZO_F32, 0, 10, 0, 0, 0, 1e-3, None) == zo.ZO_ERR_ARG
    assert lib.zo_perturb(odd, zo.ZO_BF16, 0, 10, 0, 0, 0, 1e-3, None) == zo.ZO_ERR_ARG
    assert lib.zo_perturb(fake, zo.ZO_F32, 2 ** 64 - 5, 10, 0, 0, 0, 1e-3, None) == zo.ZO_ERR_ARG
    assert lib.zo_perturb(fake, zo.ZO_BF16, 0, zo.ZO_N_MAX, 0, 0, 0, 1e-3, None) == zo.ZO_ERR_ARG
    assert lib.zo_update(fake, zo.ZO_BF16, zo.ZO_N_MAX, 0, 0, 1, c1, 1e-3, None) == zo.ZO_ERR_ARG
    assert lib.zo_perturb(fake, zo.ZO_F32, 0, 10, 0, 0, 0, float("inf"), None) == zo.ZO_ERR_NONFINITE
    assert lib.zo_perturb(None, zo.ZO_F32, 0, 0, 0, 0, 0, 1e-3, None) == zo.ZO_OK  # n = 0: no-op
    assert lib.zo_update(fake, zo.ZO_F32, 10, 0, 0, zo.ZO_K_MAX + 1, big, 1e-3, None) == zo.ZO_ERR_ARG
    assert lib.zo_update(fake, zo.ZO_F32, 10, 0, 0, 1, None, 1e-3, None) == zo.ZO_ERR_NULL
    assert lib.zo_update(fake, zo.ZO_F32, 10, 0, 0, 1, cnan, 1e-3, None) == zo.ZO_ERR_NONFINITE
    assert lib.zo_update(fake, zo.ZO_F32, 10, 0, 0, 1, c1, float("nan"), None) == zo.ZO_ERR_NONFINITE
    assert lib.zo_update(None, zo.ZO_BF16, 10, 0, 0, 1, c1, 1e-3, None) == zo.ZO_ERR_NULL
    assert lib.zo_update_ex(fake, zo.ZO_F32, 0, 10, 0, 0, 2 ** 32 - 1, 2, (ctypes.c_float * 2)(), 1e-3, None) == zo.ZO_ERR_ARG
    assert lib.zo_update(fake, zo.ZO_F32, 10, 0, 0, 0, None, 1e-3, None) == zo.ZO_OK  # K = 0: no-op
    assert lib.zo_gen_bits(None, 0, 4, 0, 0, 0, None) == zo.ZO_ERR_NULL
    assert lib.zo_gen_bits(ctypes.c_void_p(0x10008), 0, 4, 0, 0, 0, None) == zo.ZO_ERR_ARG
    assert lib.zo_gen_bits(fake, 2 ** 60, 1, 0, 0, 0, None) == zo.ZO_ERR_ARG
    assert lib.zo_gen_bits(None, 0, 0, 0, 0, 0, None) == zo.ZO_OK


def test_segments_validation_returns_before_launch(lib):
    Seg = zo.ZoSegment
    c1 = (ctypes.c_float * 1)(1.0)

    def arr(*segs):
        a = (Seg * len(segs))()
        for i, sg in enumerate(segs):
            a[i] = Seg(*sg)
        return a
    ok = arr((0x10000, 0, 100), (0x20000, 100, 50))
    assert lib.zo_perturb_segments(None, 3, zo.ZO_F32, 0, 0, 0, 1e-3, 1, 1e-3, None) == zo.ZO_ERR_NULL
    assert lib.zo_perturb_segments(ok, 2, 9, 0, 0, 0, 1e-3, 1, 1e-3, None) == zo.ZO_ERR_ARG
    assert lib.zo_perturb_segments(arr((None, 0, 5)), 1, zo.ZO_F32, 0, 0, 0, 1e-3, 1, 1e-3, None) == zo.ZO_ERR_NULL
    assert lib.zo_perturb_segments(arr((0x10002, 0, 5)), 1, zo.ZO_F32, 0, 0, 0, 1e-3, 1, 1e-3, None) == zo.ZO_ERR_ARG
    assert lib.zo_perturb_segments(arr((0x10000, 2 ** 64 - 2, 5)), 1, zo.ZO_F32, 0, 0, 0, 1e-3, 1, 1e-3, None) == zo.ZO_ERR_ARG
    too_big = arr((0x10000, 0, 100), (0x20000, 100, zo.ZO_N_MAX))
    assert lib.zo_perturb_segments(too_big, 2, zo.ZO_BF16, 0, 0, 0, 1e-3, 1, 1e-3, None) == zo.ZO_ERR_ARG
    # overlapping memory (the second starts inside the first)
    overl = arr((0x10000, 0, 100), (0x10000 + 4 * 99, 100, 10))
    assert lib.zo_perturb_segments(overl, 2, zo.ZO_F32, 0, 0, 0, 1e-3, 1, 1e-3, None) == zo.ZO_ERR_ARG
    overl_bf16 = arr((0x10000, 0, 100), (0x10000 + 2 * 50, 100, 10))
    assert lib.zo_update_segments(overl_bf16, 2, zo.ZO_BF16, 0, 0, 0, 1, c1, 1e-3, 0, 0.0, None) == zo.ZO_ERR_ARG
    assert lib.zo_perturb_segments(ok, 2, zo.ZO_F32, 0, 0, 0, float("nan"), 1, 1e-3, None) == zo.ZO_ERR_NONFINITE
    big = (ctypes.c_float * (zo.ZO_K_MAX + 1))()
    assert lib.zo_update_segments(ok, 2, zo.ZO_F32, 0, 0, 0, zo.ZO_K_MAX + 1, big, 1e-3, 0, 0.0, None) == zo.ZO_ERR_ARG
    assert lib.zo_update_segments(ok, 2, zo.ZO_F32, 0, 0, 0, 1, c1, float("inf"), 0, 0.0, None) == zo.ZO_ERR_NONFINITE
    # empty lists and empty segments are no-ops
    assert lib.zo_perturb_segments(None, 0, zo.ZO_F32, 0, 0, 0, 1e-3, 1, 1e-3, None) == zo.ZO_OK
    assert lib.zo_update_segments(arr((None, 0, 0)), 1, zo.ZO_F32, 0, 0, 0, 0, None, 1e-3, 0, 0.0, None) == zo.ZO_OK


def test_strerror_and_version(lib):
    for s in (0, -1, -2, -3, -4, 99):
        assert lib.zo_strerror(s)
    assert b"gfx950" in lib.zo_version()


def test_binding_refuses_cpu_tensors(lib):
    import torch
    with pytest.raises(TypeError):
        zo.zo_perturb(torch.zeros(4), 0, 1e-3, 0, 0)


def test_plain_c_consumer(tmp_path):
    """The header compiles as C99 with warnings as errors, and a C program linked against
    libzo.so gets the documented host results and validation codes (no GPU needed)."""
    import shutil
    cc = shutil.which("gcc")
    if cc is None:
        pytest.skip("no C compiler")
    exe = tmp_path / "abi_c_check"
    src = os.path.join(ROOT, "tests", "helpers", "abi_c_check.c")
    libdir = os.path.dirname(zo.LIB_PATH)
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"), src,
                        "-o", str(exe), "-L", libdir, "-lzo", "-Wl,-rpath," + libdir, "-lm"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.count("ok ") == 15 and "FAIL" not in r.stdout, r.stdout


def test_missing_library_raises_and_nothing_falls_back():
    """Without libzo.so every call raises ZoLibraryMissing (the host coefficient function
    included); the package imports no other implementation of the method."""
    code = (
        "import sys\n"
        "import paper_2609_38095_amd as zo\n"
        "zo.LIB_PATH = '/nonexistent/libzo.so'\n"
        "zo._LIB = None\n"
        "calls = [zo.library, zo.zo_version, lambda: zo.zo_probe_coeffs([2.0], [2.0], 2.0, 1e-3),\n"
        "         lambda: zo.zo_probe_coeffs_ex([2.0], [2.0], 2.0, 1e-3), lambda: zo.zo_set_max_blocks(0)]\n"
        "for call in calls:\n"
        "    try:\n"
        "        call()\n"
        "    except zo.ZoLibraryMissing:\n"
        "        continue\n"
        "    sys.exit('a call succeeded without the library')\n"
        "assert 'oracle' not in sys.modules, 'the binding imported the oracle'\n"
        "print('ok')\n")
    r = subprocess.run([os.sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stderr
    src = open(os.path.join(ROOT, "paper_2609_38095_amd", "__init__.py")).read()
    assert not re.search(r"^\s*(from|import)\s+(oracle|\.\.oracle)", src, flags=re.M)
