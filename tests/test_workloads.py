"""Seeded input generators: determinism, value sets and scene structure."""
import numpy as np
import pytest

import workloads


def test_uniform_is_deterministic_and_exact():
    a = workloads.uniform_complex(4, 256, 1)
    b = workloads.uniform_complex(4, 256, 1)
    c = workloads.uniform_complex(4, 256, 2)
    assert a.dtype == np.complex64 and a.shape == (4, 256)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert not np.array_equal(a, c)
    parts = a.view(np.float32)
    assert parts.min() >= -1.0 and parts.max() < 1.0
    # 2u - 1 with u = k / 2^24: every value is a multiple of 2^-23
    scaled = parts.astype(np.float64) * 2.0**23
    assert np.array_equal(scaled, np.round(scaled))


def test_fp16_is_rne_of_fp32_draw():
    x16 = workloads.uniform_complex(3, 128, 3, "fp16")
    x32 = workloads.uniform_complex(3, 128, 3, "fp32")
    assert x16.dtype == np.float16 and x16.shape == (3, 128, 2)
    assert np.array_equal(x16, x32.view(np.float32).reshape(3, 128, 2).astype(np.float16))


def test_named_workloads_small_and_sampled_rows():
    x = workloads.fft_workload("fft_n1024_b64_fp32")
    assert x.shape == (64, 1024)
    assert np.array_equal(x, workloads.uniform_complex(64, 1024, 0))
    rows = np.array([0, 5, 63])
    assert np.array_equal(workloads.fft_workload_rows("fft_n1024_b64_fp32", rows), x[rows])


@pytest.mark.parametrize("name", ["fft_n8192_b16384_fp32", "fft_n16384_b8192_fp32"])
def test_sampled_rows_match_prefix_of_full_draw(name):
    """Row sampling by generator advance agrees with a full C-ordered draw."""
    w = workloads.FFT_WORKLOADS[name]
    full = workloads.uniform_complex(6, w["n"], w["seed"])
    got = workloads.fft_workload_rows(name, [0, 2, 5])
    assert np.array_equal(got, full[[0, 2, 5]])


def test_sampled_rows_fp16():
    full = workloads.uniform_complex(4, 16384, 3, "fp16")
    got = workloads.fft_workload_rows("fft_n16384_b16384_fp16", [1, 3])
    assert np.array_equal(got, full[[1, 3]])


def test_chirp_support_and_magnitude():
    h = workloads.centred_chirp(4096, 1024, 0.8)
    nz = np.flatnonzero(h)
    assert nz.size == 1024
    assert set(nz) == set(range(0, 512)) | set(range(4096 - 512, 4096))
    np.testing.assert_allclose(abs(h[nz]), 1.0, rtol=1e-15)
    # centred: h(t) = h(-t)
    t = np.arange(1, 512)
    np.testing.assert_allclose(h[t], h[4096 - t], rtol=1e-15)
    # instantaneous frequency beta t / L -> phase difference between neighbours
    dphi = np.angle(h[101] * np.conj(h[100])) / (2 * np.pi)
    np.testing.assert_allclose(dphi, 0.8 * 100.5 / 1024, rtol=1e-12)


def test_sar_scene_structure():
    sc = workloads.sar_scene()
    assert sc.raw.shape == (4096, 4096) and sc.raw.dtype == np.complex64
    assert sc.range_ref.shape == (4096,) and sc.az_ref.shape == (4096,)
    assert len(sc.targets_az) == 32
    assert sc.targets_az.min() >= 256 and sc.targets_az.max() < 3840
    assert sc.targets_rg.min() >= 512 and sc.targets_rg.max() < 3584
    da = np.abs(sc.targets_az[:, None] - sc.targets_az[None, :])
    dr = np.abs(sc.targets_rg[:, None] - sc.targets_rg[None, :])
    off = ~np.eye(32, dtype=bool)
    assert da[off].min() >= 32 and dr[off].min() >= 32
    assert sc.amplitudes.min() >= 0.5 and sc.amplitudes.max() <= 1.0
    sc2 = workloads.sar_scene()
    assert np.array_equal(sc.raw.view(np.uint32), sc2.raw.view(np.uint32))


def test_sar_scene_noise_level():
    sc = workloads.sar_scene(n_az=512, n_rg=512, n_targets=1, len_rg=64, len_az=32, min_sep=1,
                             targets=[(100, 100, 1.0)])
    quiet = sc.raw[200:, 200:]  # far from the single echo
    np.testing.assert_allclose(quiet.real.std(), 0.01, rtol=0.05)
    np.testing.assert_allclose(quiet.imag.std(), 0.01, rtol=0.05)


def test_rd_scene_matches_the_papers_geometry():
    """Section X: 600 m synthetic aperture (1500 pulses at 500 Hz) at 20 km,
    about 1.8 range bins of migration across it, 1200-sample pulses, every
    echo inside the frame; deterministic for a seed."""
    sc = workloads.rd_scene(sigma=0.0)
    g, p = sc.geometry, sc.params
    assert g["range_bin"] == pytest.approx(299_792_458.0 / 240e6)
    r0 = 20_000.0
    aperture = g["wavelength"] * r0 / p["antenna"]
    assert aperture == pytest.approx(600.0)
    assert aperture / g["speed"] * g["prf"] == pytest.approx(1500.0)
    migration = (np.hypot(r0, aperture / 2) - r0) / g["range_bin"]
    assert 1.7 < migration < 1.9
    assert p["pulse_samples"] == 1200 and np.count_nonzero(sc.range_ref) == 1200
    assert len(sc.targets_az) == 6
    # a lone target's echo is lit on its aperture only (about 1360-1580 pulses)
    for a_i, n_i, _ in workloads.RD_TARGETS:
        lone = workloads.rd_scene(sigma=0.0, targets=((a_i, n_i, 1.0),))
        r0_i = g["r_near"] + n_i * g["range_bin"]
        half = g["wavelength"] * r0_i / (2 * p["antenna"]) * g["prf"] / g["speed"]
        lit = np.nonzero(abs(lone.raw[:, n_i + 600]) > 0.5)[0]
        assert abs(lit.min() - (a_i - half)) <= 1 and abs(lit.max() - (a_i + half)) <= 1
    noisy = workloads.rd_scene_small()
    again = workloads.rd_scene_small()
    assert np.array_equal(noisy.raw, again.raw)
    assert noisy.raw.dtype == np.complex64 and noisy.range_ref.dtype == np.complex64
