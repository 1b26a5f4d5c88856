"""Host-side checks of the C ABI: symbols, argument errors, error strings.

None of these make a compute call, so they run without a GPU: every argument
error is returned before the library touches the HIP runtime.
"""
import ctypes
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mi355fft.h")


@pytest.fixture(scope="module")
def L():
    from paper_2609_32237_amd import _lib

    return _lib


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_][a-z0-9_]*)\s*\([^;{]*\)\s*;", text)))


def test_header_declares_the_abi():
    assert declared_functions() == sorted(
        ["fft_plan_create", "fft_plan_create_ex", "fft_execute", "fft_plan_destroy", "sar_workspace_bytes", "sar_form_image_ex",
         "sar_form_image", "sar_form_image_noalloc", "sar_rd_workspace_bytes", "sar_rd_form_image", "fft_strerror"])


def test_library_exports_every_declared_symbol(L):
    out = subprocess.run(["nm", "-D", "--defined-only", L.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r" T (\w+)$", out, flags=re.M))
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(L.lib, name)
    assert set(L.EXPORTS) == set(declared_functions())


def test_header_compiles_as_c():
    """The header is plain C: it compiles with gcc against the HIP runtime headers."""
    src = f'#include "{HEADER}"\nint main(void) {{ return FFT_OK; }}\n'
    res = subprocess.run(["gcc", "-x", "c", "-std=c11", "-fsyntax-only", "-D__HIP_PLATFORM_AMD__",
                          "-I/opt/rocm/include", "-"], input=src, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr


def test_strerror_covers_every_code(L):
    codes = [L.FFT_OK, L.FFT_EINVAL, L.FFT_EUNSUPPORTED, L.FFT_ENOMEM, L.FFT_EALIGN, L.FFT_EHIP]
    msgs = [L.fft_strerror(c) for c in codes]
    assert len(set(msgs)) == len(codes)
    assert "unknown" not in " ".join(msgs)
    assert L.fft_strerror(12345) == "unknown error code"


def create(L, *args):
    p = ctypes.c_void_p()
    return L.lib.fft_plan_create(*args, ctypes.byref(p)), p


@pytest.mark.parametrize("args, code", [
    ((1000, 1, 1, 1000, 0, -1), "FFT_EUNSUPPORTED"),   # not a power of two
    ((512, 1, 1, 512, 0, -1), "FFT_EUNSUPPORTED"),     # below 1024
    ((1 << 29, 1, 1, 1 << 29, 0, -1), "FFT_EUNSUPPORTED"),  # above 2^28
    ((32768, 2, 2, 1, 0, -1), "FFT_EUNSUPPORTED"),     # long transforms: contiguous only
    ((0, 1, 1, 1, 0, -1), "FFT_EINVAL"),
    ((4096, 0, 1, 4096, 0, -1), "FFT_EINVAL"),         # empty batch
    ((4096, -3, 1, 4096, 0, -1), "FFT_EINVAL"),
    ((4096, 2, 0, 4096, 0, -1), "FFT_EINVAL"),         # stride 0
    ((4096, 2, 1, 0, 0, -1), "FFT_EINVAL"),            # dist 0
    ((4096, 2, 1, 4095, 0, -1), "FFT_EINVAL"),         # rows overlap
    ((4096, 8, 4, 1, 0, -1), "FFT_EINVAL"),            # columns overlap (stride < batch)
    ((4096, 3, 2, 2, 0, -1), "FFT_EINVAL"),            # neither blocks nor interleaved
    ((4096, 1, 1, 4096, 2, -1), "FFT_EINVAL"),         # bad storage
    ((4096, 1, 1, 4096, 0, 0), "FFT_EINVAL"),          # bad direction
    ((4096, 1 << 30, 1, 1 << 30, 0, -1), "FFT_EINVAL"),  # layout beyond 2^40 elements
])
def test_plan_argument_errors(L, args, code):
    rc, p = create(L, *args)
    assert rc == getattr(L, code)
    assert p.value is None


def test_plan_null_out(L):
    assert L.lib.fft_plan_create(4096, 1, 1, 4096, 0, -1, None) == L.FFT_EINVAL


def test_execute_and_destroy_null(L):
    assert L.lib.fft_execute(None, 256, 256, None) == L.FFT_EINVAL
    assert L.lib.fft_plan_destroy(None) == L.FFT_OK


def test_sar_argument_errors(L):
    f = L.lib.sar_form_image_ex
    ok = 1 << 20
    assert f(4096, 4096, 0, None, ok, ok, ok, ok, None) == L.FFT_EINVAL
    assert f(4096, 4096, 3, ok, ok, ok, ok, ok, None) == L.FFT_EINVAL
    assert f(4000, 4096, 0, ok, ok, ok, ok, ok, None) == L.FFT_EUNSUPPORTED
    assert f(4096, 32768, 0, ok, ok, ok, ok, ok, None) == L.FFT_EUNSUPPORTED
    assert f(4096, 4096, 0, ok + 4, ok, ok, 1 << 40, 1 << 41, None) == L.FFT_EALIGN
    assert f(4096, 4096, 0, ok, ok, ok, 1 << 40, (1 << 41) + 8, None) == L.FFT_EALIGN  # workspace 256 B
    # out overlapping raw
    assert f(4096, 4096, 0, 1 << 30, ok, ok, (1 << 30) + 4096, 1 << 40, None) == L.FFT_EINVAL
    # a reference inside the workspace (the range pass writes the spectra there)
    ws = 1 << 41
    assert f(4096, 4096, 0, 1 << 30, ws + 8, ok, 1 << 40, ws, None) == L.FFT_EINVAL
    assert f(4096, 4096, 0, 1 << 30, ok, ws + (1 << 20), 1 << 40, ws, None) == L.FFT_EINVAL
    assert L.lib.sar_form_image(None, ok, ok, ok, None) == L.FFT_EINVAL


def test_sar_noalloc_argument_errors(L):
    """Every argument error, and an intermediate beyond the fixed array's
    128 MiB, comes back before any HIP call."""
    f = L.lib.sar_form_image_noalloc
    ok = 1 << 20
    assert f(4096, 4096, 0, None, ok, ok, ok, None) == L.FFT_EINVAL
    assert f(4096, 4096, 3, ok, ok, ok, 1 << 40, None) == L.FFT_EINVAL
    assert f(4000, 4096, 0, ok, ok, ok, 1 << 40, None) == L.FFT_EUNSUPPORTED
    assert f(4096, 4096, 0, ok + 4, ok, ok, 1 << 40, None) == L.FFT_EALIGN
    assert f(4096, 4096, 0, 1 << 30, ok, ok, (1 << 30) + 4096, None) == L.FFT_EINVAL
    # the largest intermediates the array holds are 128 MiB; one beyond is refused
    assert f(8192, 4096, 0, 1 << 30, ok, ok, 1 << 40, None) == L.FFT_EUNSUPPORTED
    assert f(8192, 8192, 1, 1 << 30, ok, ok, 1 << 40, None) == L.FFT_EUNSUPPORTED
    assert f(16384, 16384, 0, 1 << 30, ok, ok, 1 << 40, None) == L.FFT_EUNSUPPORTED


def test_sar_workspace_bytes(L):
    # both spectra, the 256-byte flag slot of the range pass, the intermediate
    assert L.sar_workspace_bytes(4096, 4096, 0) == (4096 + 4096) * 8 + 256 + 4096 * 4096 * 8
    assert L.sar_workspace_bytes(4096, 4096, 1) == (4096 + 4096) * 8 + 256 + 4096 * 4096 * 4
    assert L.sar_workspace_bytes(1024, 16384, 1) == (1024 + 16384) * 8 + 256 + 1024 * 16384 * 4
    assert L.sar_workspace_bytes(4096, 4000, 0) == 0
    assert L.sar_workspace_bytes(4096, 4096, 5) == 0


def test_forced_allocation_failure_reports_enomem():
    """MI355FFT_TEST_FAIL_ALLOC=1 makes the first device allocation fail."""
    code = ("import ctypes\n"
            "from paper_2609_32237_amd import _lib as L\n"
            "p = ctypes.c_void_p()\n"
            "print(L.lib.fft_plan_create(4096, 2, 1, 4096, 0, -1, ctypes.byref(p)), p.value)\n")
    env = dict(os.environ, MI355FFT_TEST_FAIL_ALLOC="1")
    res = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                         timeout=120)
    assert res.returncode == 0, res.stderr
    rc, val = res.stdout.split()
    assert int(rc) == -3 and val == "None"


@pytest.mark.parametrize("var, value", [("MI355FFT_ROW_VARIANT", "99"), ("MI355FFT_ROW_VARIANT", "x"),
                                        ("MI355FFT_COL_VARIANT", "-1")])
def test_out_of_range_variant_is_rejected_before_any_hip_call(var, value):
    stride, dist = (1, 4096) if var == "MI355FFT_ROW_VARIANT" else (8, 1)
    code = ("import ctypes\n"
            "from paper_2609_32237_amd import _lib as L\n"
            "p = ctypes.c_void_p()\n"
            f"print(L.lib.fft_plan_create(4096, 2, {stride}, {dist}, 0, -1, ctypes.byref(p)))\n")
    env = dict(os.environ, **{var: value})
    res = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                         timeout=120)
    assert res.returncode == 0, res.stderr
    assert int(res.stdout.split()[0]) == -1


def test_sar_rd_workspace_bytes(L):
    def up(x):
        return (x + 255) // 256 * 256
    tables = up(4096 * 16) + up(4096 * 8) + up(129 * 8 * 8)
    assert L.sar_rd_workspace_bytes(4096, 4096, 0) == 4096 * 8 + 256 + tables + 4096 * 4096 * 8
    assert L.sar_rd_workspace_bytes(4096, 4096, 1) == 4096 * 8 + 256 + tables + 4096 * 4096 * 4
    assert L.sar_rd_workspace_bytes(16384, 8192, 0) == 8192 * 8 + 256 + up(16384 * 16) + up(8192 * 8) + up(129 * 64) + \
        16384 * 8192 * 8
    assert L.sar_rd_workspace_bytes(16384, 16384, 0) == 0  # beyond 2^27 points
    assert L.sar_rd_workspace_bytes(4096, 4000, 0) == 0
    assert L.sar_rd_workspace_bytes(4096, 4096, 2) == 0


def test_sar_rd_argument_errors(L):
    f = L.lib.sar_rd_form_image
    geo = L.geometry(dict(wavelength=0.24, speed=200.0, prf=500.0, range_bin=1.249, r_near=17500.0))
    g = ctypes.byref(geo)
    ok = 1 << 20
    ws = 1 << 40
    assert f(4096, 4096, 0, None, ok, ok, 1 << 36, ws, None) == L.FFT_EINVAL        # no geometry
    assert f(4096, 4096, 0, g, None, ok, 1 << 36, ws, None) == L.FFT_EINVAL         # no echo
    assert f(4096, 4096, 2, g, ok, ok, 1 << 36, ws, None) == L.FFT_EINVAL           # bad storage
    for field, bad in (("wavelength", 0.0), ("speed", -1.0), ("prf", float("nan")), ("range_bin", float("inf")),
                       ("r_near", 0.0), ("prf", 3400.0)):  # prf 3400: lambda prf / 4v >= 1
        b = L.geometry(dict(wavelength=0.24, speed=200.0, prf=500.0, range_bin=1.249, r_near=17500.0))
        setattr(b, field, bad)
        assert f(4096, 4096, 0, ctypes.byref(b), ok, ok, 1 << 36, ws, None) == L.FFT_EINVAL, field
    wide_band = L.geometry(dict(wavelength=0.24, speed=200.0, prf=1400.0, range_bin=1.249, r_near=17500.0))
    assert f(4096, 4096, 0, ctypes.byref(wide_band), ok, ok, 1 << 36, ws, None) == L.FFT_EUNSUPPORTED  # 0.42 > 1/3
    assert f(4000, 4096, 0, g, ok, ok, 1 << 36, ws, None) == L.FFT_EUNSUPPORTED
    assert f(16384, 16384, 0, g, ok, ok, 1 << 36, ws, None) == L.FFT_EUNSUPPORTED   # beyond 2^27 points
    assert f(4096, 4096, 0, g, ok + 4, ok, 1 << 36, ws, None) == L.FFT_EALIGN
    assert f(4096, 4096, 0, g, ok, ok, 1 << 36, ws + 8, None) == L.FFT_EALIGN       # workspace 256 B
    assert f(4096, 4096, 0, g, 1 << 30, ok, (1 << 30) + 4096, ws, None) == L.FFT_EINVAL  # out overlaps raw
    assert f(4096, 4096, 0, g, ok, ok, ws + 4096, ws, None) == L.FFT_EINVAL         # out inside workspace
    assert f(4096, 4096, 0, g, ok, ws + 256, 1 << 36, ws, None) == L.FFT_EINVAL     # reference inside workspace
    assert f(4096, 4096, 0, g, ok, (1 << 36) + 64, 1 << 36, ws, None) == L.FFT_EINVAL  # reference inside out


def test_long_transform_plans_are_accepted(L):
    """Lengths above 16384 (four-step) plan without a GPU call beyond the
    twiddle tables, so only check the argument path here: the plan either
    succeeds (a GPU is present) or fails in the HIP runtime, never EINVAL."""
    for n in (1 << 15, 1 << 20, 1 << 28):
        rc, p = create(L, n, 1, 1, n, 0, -1)
        assert rc in (L.FFT_OK, L.FFT_EHIP, L.FFT_ENOMEM), (n, rc)
        if rc == L.FFT_OK:
            L.lib.fft_plan_destroy(p)


@pytest.mark.parametrize("args, code", [
    ((4096, 1, 1, 4096, 0, -1, -1, 0), "FFT_EINVAL"),       # negative shift
    ((4096, 1, 1, 4096, 0, -1, 61, 0), "FFT_EINVAL"),       # shift beyond 60
    ((4096, 1, 1, 4096, 1, -1, 0, 4), "FFT_EINVAL"),        # unknown flag
    ((4096, 1, 1, 4096, 0, -1, 0, 2), "FFT_EINVAL"),        # matrix units need FP16 storage
    ((4096, 1, 1, 4096, 1, -1, 0, 3), "FFT_EINVAL"),        # two exclusive options
    ((8192, 1, 1, 8192, 1, -1, 0, 2), "FFT_EUNSUPPORTED"),  # matrix units: 4096 and 16384
    ((4096, 2, 2, 1, 1, -1, 0, 2), "FFT_EUNSUPPORTED"),     # matrix units: rows only
    ((4096, 1, 1, 4096, 1, -1, 3, 2), "FFT_EUNSUPPORTED"),  # matrix units: no output scale
    ((4096, 1, 1, 4096, 0, -1, 0, 1), "FFT_EINVAL"),        # FP16 exchange needs FP16 storage
    ((4096, 2, 2, 1, 1, -1, 0, 1), "FFT_EUNSUPPORTED"),     # FP16 exchange: rows only
    ((32768, 1, 1, 32768, 1, -1, 0, 1), "FFT_EUNSUPPORTED"),  # FP16 exchange: single pass only
    ((1000, 1, 1, 1000, 0, -1, 3, 0), "FFT_EUNSUPPORTED"),
])
def test_plan_ex_argument_errors(L, args, code):
    p = ctypes.c_void_p()
    assert L.lib.fft_plan_create_ex(*args, ctypes.byref(p)) == getattr(L, code)
    assert p.value is None
