"""The oracle's pins are strong enough to catch plausible mistakes.

Each case copies ``oracle/oracle.c`` to a temporary directory, plants one
mistake there (a flipped sign, a dropped scale, a missing conjugate, a wrong
index, swapped image axes), compiles the copy, and checks that at least one of
the pins in ``test_oracle.py`` fails against it.  The committed oracle is never
modified; everything happens on the CPU.
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle
import test_oracle as pins

MUTANTS = {
    "twiddle_sign": ("w[2 * m + 1] = (double)sign * sin(ang);",
                     "w[2 * m + 1] = -(double)sign * sin(ang);"),
    "direct_index": ("int64_t m = (j * k) % n;", "int64_t m = (j * k + k) % n;"),
    "butterfly_index": ("const double *tw = w + 2 * (k * step);",
                        "const double *tw = w + 2 * ((k * step) / 2);"),
    "butterfly_sign": ("v[0] = u[0] - vr;", "v[0] = u[0] + vr;"),
    "bit_reversal": ("if (i < j) {", "if (i < j && i > 1) {"),
    "dropped_scale": ("double inv_len = 1.0 / (double)len;", "double inv_len = 1.0;"),
    "missing_conj": ("double hr = job->spec[2 * k], hi = -job->spec[2 * k + 1];",
                     "double hr = job->spec[2 * k], hi = job->spec[2 * k + 1];"),
    "swapped_axes": ("rc = sar_axis(n_az, n_rg, 1, mid, out, az_ref, nthreads);",
                     "rc = sar_axis(n_az, n_rg, 1, mid, out, range_ref, nthreads);"),
    "xcorr_conj": ("double har = az_ref[2 * ta], hai = -az_ref[2 * ta + 1];",
                   "double har = az_ref[2 * ta], hai = az_ref[2 * ta + 1];"),
    "xcorr_index": ("const double *x = row + 2 * ((pr[p] + tr) % n_rg);",
                    "const double *x = row + 2 * ((pr[p] + n_rg - tr) % n_rg);"),
}


def _battery(mod):
    """Run a compact set of pins; return the names of those that fail."""
    failed = []
    checks = [
        ("direct_closed_forms", lambda: pins.test_direct_dft_closed_forms(mod, 12)),
        ("fft_vs_bruteforce", lambda: pins.test_fft_vs_bruteforce(mod, 64)),
        ("fft_closed_forms", lambda: pins.test_fft_closed_forms(mod, 1024)),
        ("fft_vs_numpy", lambda: pins.test_fft_vs_numpy(mod, 1024)),
        ("sar_vs_direct", lambda: pins.test_sar_chain_vs_direct_definition_tiny(mod)),
        ("lone_target_value", lambda: pins.test_xcorr_direct_single_target_value(mod)),
        ("lone_target_closed_form", lambda: pins.test_sar_single_target_closed_form(mod, (256, 128))),
    ]
    for name, fn in checks:
        try:
            with np.errstate(all="ignore"):
                fn()
        except (AssertionError, RuntimeError, ValueError, IndexError):
            failed.append(name)
    return failed


def test_committed_oracle_passes_battery():
    oracle._load()
    assert _battery(oracle) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, monkeypatch, name):
    old, new = MUTANTS[name]
    src = open(os.path.join(os.path.dirname(oracle.__file__), "oracle.c")).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    mutated = tmp_path / "oracle_mut.c"
    mutated.write_text(src.replace(old, new))
    so = tmp_path / "liboracle_mut.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-pthread", "-o", str(so),
                    str(mutated), "-lm"], check=True)
    lib = ctypes.CDLL(str(so))
    real = oracle._load()
    for fname in ("oracle_dft_direct", "oracle_fft", "oracle_sar_chain", "oracle_xcorr2d_points"):
        f, g = getattr(lib, fname), getattr(real, fname)
        f.argtypes, f.restype = g.argtypes, g.restype
    monkeypatch.setattr(oracle, "_lib", lib)
    failed = _battery(oracle)
    assert failed, f"planted mistake {name!r} passed every pin"
