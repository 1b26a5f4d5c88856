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
import test_oracle_rd as rd_pins
import workloads

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

# Mistakes in the full range-Doppler chain (caught by the pins in test_oracle_rd.py).
RD_MUTANTS = {
    "rcmc_direction": ("int64_t base = n + (int64_t)fl - 3;", "int64_t base = n - (int64_t)fl - 3;"),
    "rcmc_tap_offset": ("int64_t base = n + (int64_t)fl - 3;", "int64_t base = n + (int64_t)fl - 4;"),
    "rcmc_skipped": ("double dn = r0 * inv_d_minus_1 / job->range_bin;",
                     "double dn = 0.0 * r0 * inv_d_minus_1 / job->range_bin;"),
    "blend_reversed": ("double g = (1.0 - a) * job->tab[q * RD_TAPS + j] + a * job->tab[(q + 1) * RD_TAPS + j];",
                       "double g = a * job->tab[q * RD_TAPS + j] + (1.0 - a) * job->tab[(q + 1) * RD_TAPS + j];"),
    "blend_nearest": ("double a = qf - (double)q;", "double a = qf - (double)q >= 0.5 ? 1.0 : 0.0;"),
    "sinc_argument": ("double x = (double)(j - 3) - mu;", "double x = (double)(j - 3) + mu;"),
    "filter_sign": ("double ang = OR_TWO_PI * (cyc - nearbyint(cyc));",
                    "double ang = -OR_TWO_PI * (cyc - nearbyint(cyc));"),
    "filter_not_baseband": ("double cyc = 2.0 * r0 * d_minus_1 / job->wavelength;",
                            "double cyc = 2.0 * r0 * (d_minus_1 + 1.0) / job->wavelength;"),
    "doppler_wrap": ("return (double)(k < n_az / 2 ? k : k - n_az) * prf / (double)n_az;",
                     "return (double)k * prf / (double)n_az;"),
    "azimuth_scale": ("const double s = 1.0 / (double)n_az;", "const double s = 1.0;"),
}


def _rd_battery(mod):
    """The range-Doppler pins on the 1024 x 1024 scene; names of those that fail."""
    failed = []
    try:
        sc = workloads.rd_scene_small(sigma=0.0)
        small = (sc, {s: mod.rd_chain(sc.raw, sc.range_ref, sc.geometry, stop_after=s) for s in (1, 2, 3, 4, 5)})
    except RuntimeError:
        return ["chain"]
    checks = [
        ("range_compression", lambda: rd_pins.test_range_compression_is_the_circular_correlation(small)),
        ("azimuth_fft", lambda: rd_pins.test_azimuth_fft_is_scaled_by_one_over_n_az(small)),
        ("migration_curve", lambda: rd_pins.test_migration_follows_r0_over_d_before_correction(small)),
        ("rcmc_straight", lambda: rd_pins.test_rcmc_straightens_every_target(small)),
        ("interp_tones", lambda: rd_pins.test_interpolator_reproduces_band_limited_signals(mod)),
        ("interp_continuous", lambda: rd_pins.test_rcmc_output_is_continuous_in_the_shift(mod)),
        ("interp_table", lambda: rd_pins.test_interpolator_table_properties(mod)),
        ("filter_fm_rate", lambda: rd_pins.test_azimuth_filter_phase_tends_to_the_fm_rate(small)),
        ("baseband", lambda: rd_pins.test_baseband_filter_keeps_the_range_spectrum_in_band((sc, small[1][5]))),
        ("focus", lambda: rd_pins.test_noisy_scene_focuses_every_target(mod)),
    ]
    for name, fn in checks:
        try:
            with np.errstate(all="ignore"):
                fn()
        except (AssertionError, RuntimeError, ValueError, IndexError):
            failed.append(name)
    return failed


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
    assert _rd_battery(oracle) == []


def _load_mutant(tmp_path, monkeypatch, old, new):
    src = open(os.path.join(os.path.dirname(oracle.__file__), "oracle.c")).read()
    assert src.count(old) == 1, f"mutation anchor {old!r} not found exactly once"
    mutated = tmp_path / "oracle_mut.c"
    mutated.write_text(src.replace(old, new))
    so = tmp_path / "liboracle_mut.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-pthread", "-o", str(so),
                    str(mutated), "-lm"], check=True)
    lib = ctypes.CDLL(str(so))
    real = oracle._load()
    for fname in ("oracle_dft_direct", "oracle_fft", "oracle_sar_chain", "oracle_xcorr2d_points",
                  "oracle_rd_chain", "oracle_rd_interp_table"):
        f, g = getattr(lib, fname), getattr(real, fname)
        f.argtypes, f.restype = g.argtypes, g.restype
    monkeypatch.setattr(oracle, "_lib", lib)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, monkeypatch, name):
    _load_mutant(tmp_path, monkeypatch, *MUTANTS[name])
    failed = _battery(oracle)
    assert failed, f"planted mistake {name!r} passed every pin"


@pytest.mark.parametrize("name", sorted(RD_MUTANTS))
def test_planted_range_doppler_mistake_is_caught(tmp_path, monkeypatch, name):
    _load_mutant(tmp_path, monkeypatch, *RD_MUTANTS[name])
    failed = _rd_battery(oracle)
    print(name, "caught by", failed)
    assert failed, f"planted mistake {name!r} passed every pin"
