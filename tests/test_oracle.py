"""Pins for the fp64 oracle, independent of the oracle's own formulas.

Each test checks the oracle against something fixed by the mathematics or by
the paper: closed-form transforms, brute force on tiny inputs, Parseval's
identity, linearity, the shift theorem, round trips, an independent FFT
library (numpy's pocketfft), the separable closed form of a single focused
point target, and the focus quality the paper prints for its SAR scene
(Section X).  A dropped term, a wrong sign, a wrong index, a missing conjugate,
a missing scale or swapped image axes in the oracle fails at least one test.
"""
import json
import os

import numpy as np
import pytest

import workloads

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")

SIZES = [1024, 2048, 4096, 8192, 16384]
LONG = [1 << 15, 1 << 17, 1 << 20]  # four-step lengths (the oracle's radix-2 takes any power of two)
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rel(a, b):
    return np.linalg.norm(a - b) / np.linalg.norm(b)


def rand_c(rng, *shape):
    return rng.standard_normal(shape) + 1j * rng.standard_normal(shape)


# --------------------------------------------------------------------------
# The definition (O(N^2)) against closed forms, any N
# --------------------------------------------------------------------------


@pytest.mark.parametrize("n", [1, 2, 3, 5, 12, 64])
def test_direct_dft_closed_forms(oracle_mod, n):
    k = np.arange(n)
    for n0 in {0, 1 % n, n - 1}:
        x = np.zeros(n, complex)
        x[n0] = 1.0
        # impulse at n0 -> exp(-2 pi i k n0 / N)
        np.testing.assert_allclose(oracle_mod.dft_direct(x), np.exp(-2j * np.pi * k * n0 / n), atol=1e-13)
        np.testing.assert_allclose(oracle_mod.dft_direct(x, +1), np.exp(2j * np.pi * k * n0 / n), atol=1e-13)
    for f in {0, 1 % n, n // 2}:
        # tone exp(+2 pi i f n / N) -> N delta[k - f]
        x = np.exp(2j * np.pi * ((f * k) % n) / n)
        want = np.zeros(n, complex)
        want[f] = n
        np.testing.assert_allclose(oracle_mod.dft_direct(x), want, atol=1e-12 * n)


def test_direct_dft_vs_numpy(oracle_mod):
    rng = np.random.default_rng(10)
    for n in (7, 16, 100, 256):
        x = rand_c(rng, 2, n)
        assert rel(oracle_mod.dft_direct(x), np.fft.fft(x)) < 1e-13
        assert rel(oracle_mod.dft_direct(x, +1), np.fft.ifft(x) * n) < 1e-13


# --------------------------------------------------------------------------
# The radix-2 FFT
# --------------------------------------------------------------------------


@pytest.mark.parametrize("n", [1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024])
def test_fft_vs_bruteforce(oracle_mod, n):
    rng = np.random.default_rng(n)
    for batch in (1, 3):
        x = rand_c(rng, batch, n)
        for sign in (-1, 1):
            assert rel(oracle_mod.fft(x, sign), oracle_mod.dft_direct(x, sign)) < 1e-12


@pytest.mark.parametrize("n", SIZES + LONG)
def test_fft_closed_forms(oracle_mod, n):
    k = np.arange(n)
    rng = np.random.default_rng(n + 1)
    n0 = int(rng.integers(1, n))
    f = int(rng.integers(1, n))
    x = np.zeros((4, n), complex)
    x[0, n0] = 1.0  # impulse
    x[1] = np.exp(2j * np.pi * ((f * k) % n) / n)  # tone, argument reduced exactly
    x[2] = 1.0  # constant
    x[3, 0] = 1.0  # impulse at the origin
    y = oracle_mod.fft(x)
    np.testing.assert_allclose(y[0], np.exp(-2j * np.pi * ((k * n0) % n) / n), atol=1e-13)
    tone = np.zeros(n, complex)
    tone[f] = n
    np.testing.assert_allclose(y[1], tone, atol=1e-12 * n)
    const = np.zeros(n, complex)
    const[0] = n
    np.testing.assert_allclose(y[2], const, atol=1e-12 * n)
    np.testing.assert_allclose(y[3], np.ones(n), atol=0)
    yi = oracle_mod.fft(x[:1], +1)
    np.testing.assert_allclose(yi[0], np.exp(2j * np.pi * ((k * n0) % n) / n), atol=1e-13)


@pytest.mark.parametrize("n", SIZES)
def test_fft_parseval_linearity_shift_roundtrip(oracle_mod, n):
    rng = np.random.default_rng(2 * n)
    x = rand_c(rng, 2, n)
    y = oracle_mod.fft(x)
    # Parseval: sum |X|^2 = N sum |x|^2
    np.testing.assert_allclose((abs(y) ** 2).sum(1), n * (abs(x) ** 2).sum(1), rtol=1e-12)
    # linearity
    a, b = 0.3 - 1.1j, 2.0 + 0.5j
    np.testing.assert_allclose(oracle_mod.fft(a * x[0] + b * x[1]), a * y[0] + b * y[1], atol=1e-9)
    # shift theorem: x[(n - s) mod N] -> X[k] exp(-2 pi i k s / N)
    s = 37
    k = np.arange(n)
    ys = oracle_mod.fft(np.roll(x[0], s))
    np.testing.assert_allclose(ys, y[0] * np.exp(-2j * np.pi * ((k * s) % n) / n), atol=1e-9)
    # round trip: IFFT(FFT(x)) = N x
    np.testing.assert_allclose(oracle_mod.fft(y, +1), n * x, atol=1e-9)


@pytest.mark.parametrize("n", SIZES + LONG)
def test_fft_vs_numpy(oracle_mod, n):
    rng = np.random.default_rng(3 * n)
    x = rand_c(rng, 3, n)
    assert rel(oracle_mod.fft(x), np.fft.fft(x)) < 1e-13
    assert rel(oracle_mod.fft(x, +1), np.fft.ifft(x) * n) < 1e-13


def test_fft_on_float32_and_float16_storage(oracle_mod):
    """Stored inputs are widened exactly (complex64 and (re, im) binary16 pairs)."""
    x16 = workloads.uniform_complex(2, 1024, 3, "fp16")
    x = x16.astype(np.float64)
    xc = x[..., 0] + 1j * x[..., 1]
    assert rel(oracle_mod.fft(x16), np.fft.fft(xc)) < 1e-13
    x32 = workloads.uniform_complex(2, 1024, 0)
    assert rel(oracle_mod.fft(x32), np.fft.fft(x32.astype(np.complex128))) < 1e-13


def test_fft_layouts(oracle_mod):
    """Advanced layout: element j of transform b at b*dist + j*stride."""
    rng = np.random.default_rng(5)
    n, batch = 64, 10
    # columns of a (n, 16) row-major matrix: stride 16, dist 1, untouched column 10..15
    m = rand_c(rng, n, 16)
    y = oracle_mod.fft_layout(m.reshape(-1), n, batch, 16, 1).reshape(n, 16)
    assert rel(y[:, :batch], np.fft.fft(m[:, :batch], axis=0)) < 1e-13
    np.testing.assert_array_equal(y[:, batch:], m[:, batch:])
    # padded rows: stride 1, dist 80, gaps untouched
    buf = rand_c(rng, batch * 80)
    y = oracle_mod.fft_layout(buf, n, batch, 1, 80, sign=+1).reshape(batch, 80)
    assert rel(y[:, :n], np.fft.ifft(buf.reshape(batch, 80)[:, :n], axis=1) * n) < 1e-13
    np.testing.assert_array_equal(y[:, n:], buf.reshape(batch, 80)[:, n:])
    # strided blocks: stride 3, dist 3n
    buf = rand_c(rng, batch * 3 * n)
    y = oracle_mod.fft_layout(buf, n, batch, 3, 3 * n).reshape(batch, n, 3)
    assert rel(y[:, :, 0], np.fft.fft(buf.reshape(batch, n, 3)[:, :, 0], axis=1)) < 1e-13
    # the direct definition honours the same layout
    yd = oracle_mod.fft_layout(m.reshape(-1), n, batch, 16, 1, direct=True).reshape(n, 16)
    assert rel(yd[:, :batch], np.fft.fft(m[:, :batch], axis=0)) < 1e-13


# --------------------------------------------------------------------------
# SAR chain
# --------------------------------------------------------------------------


def small_scene(seed=7, sigma=0.01, **kw):
    args = dict(n_az=64, n_rg=32, n_targets=3, len_rg=16, beta_rg=0.8, len_az=8, beta_az=0.8,
                sigma=sigma, seed=seed, min_sep=4)
    args.update(kw)
    return workloads.sar_scene(**args)


def test_sar_chain_vs_direct_definition_tiny(oracle_mod):
    """The FFT chain equals the direct 2-D circular cross-correlation (64 x 32)."""
    sc = small_scene()
    out = oracle_mod.sar_chain(sc.raw, sc.range_ref, sc.az_ref)
    aa, rr = np.meshgrid(np.arange(64), np.arange(32), indexing="ij")
    direct = oracle_mod.xcorr2d_points(sc.raw, sc.range_ref, sc.az_ref, aa.ravel(), rr.ravel())
    assert rel(out.ravel(), direct) < 1e-12


def test_xcorr_direct_single_target_value(oracle_mod):
    """Direct sum at a lone target equals A * L_r * L_a (|h| = 1 on its support;
    complex64 storage of the chirps perturbs |h|^2 by at most a few 1e-8)."""
    sc = small_scene(sigma=0.0, targets=[(20, 11, 0.75)])
    v = oracle_mod.xcorr2d_points(sc.raw, sc.range_ref, sc.az_ref, [20], [11])
    np.testing.assert_allclose(v, 0.75 * 16 * 8, rtol=1e-6)


def _autocorr(h):
    """R[m] = sum_t h[(t + m) mod n] conj(h[t]), by direct summation."""
    n = h.size
    return np.array([np.sum(np.roll(h, -m) * np.conj(h)) for m in range(n)])


@pytest.mark.parametrize("shape", [(256, 128), (128, 512)])
def test_sar_single_target_closed_form(oracle_mod, shape):
    """Noiseless lone target: the image is A R_a(a - a0) R_r(r - r0), peak A L_r L_a.

    Built in complex128 (no storage rounding) so the identity holds to fp64."""
    n_az, n_rg = shape
    la, lr = 32, 64
    a0, r0, amp = n_az // 2 + 5, n_rg // 2 - 7, 0.625
    h_a = workloads.centred_chirp(n_az, la, 0.5)
    h_r = workloads.centred_chirp(n_rg, lr, 0.8)
    raw = amp * np.outer(np.roll(h_a, a0), np.roll(h_r, r0))
    out = oracle_mod.sar_chain(raw, h_r, h_a)
    want = amp * np.outer(np.roll(_autocorr(h_a), a0), np.roll(_autocorr(h_r), r0))
    np.testing.assert_allclose(out[a0, r0], amp * la * lr, rtol=1e-13)
    assert np.abs(out - want).max() < 1e-12 * amp * la * lr
    assert np.unravel_index(np.argmax(abs(out)), out.shape) == (a0, r0)


def test_sar_chain_full_size_sampled(oracle_mod):
    """4096 x 4096 scene: chain vs the direct definition at peaks and random points."""
    sc = workloads.sar_scene()
    out = oracle_mod.sar_chain(sc.raw, sc.range_ref, sc.az_ref)
    rng = np.random.default_rng(11)
    pa = np.concatenate([sc.targets_az[:4], rng.integers(0, 4096, 4)])
    pr = np.concatenate([sc.targets_rg[:4], rng.integers(0, 4096, 4)])
    direct = oracle_mod.xcorr2d_points(sc.raw, sc.range_ref, sc.az_ref, pa, pr)
    scale = 1024 * 512
    assert np.abs(out[pa, pr] - direct).max() < 1e-9 * scale
    # every target focuses on its own bin
    for a, r in zip(sc.targets_az, sc.targets_rg):
        win = abs(out[a - 8:a + 9, r - 8:r + 9])
        assert np.unravel_index(np.argmax(win), win.shape) == (8, 8)


def _irw_pslr(cut, up=16):
    """-3 dB width (input bins) and peak sidelobe ratio (dB) of a 1-D response,
    after band-limited upsampling by ``up`` (zero padding in frequency)."""
    n = cut.size
    spec = np.fft.fft(cut)
    pad = np.zeros(n * up, complex)
    pad[: n // 2] = spec[: n // 2]
    pad[-n // 2:] = spec[-n // 2:]
    mag = abs(np.fft.ifft(pad)) * up
    mag = np.roll(mag, n * up // 2 - int(np.argmax(mag)))
    c = n * up // 2
    p = mag[c]
    half = p / np.sqrt(2.0)
    i = c
    while mag[i] > half:
        i += 1
    right = i - 1 + (mag[i - 1] - half) / (mag[i - 1] - mag[i])
    i = c
    while mag[i] > half:
        i -= 1
    left = i + 1 - (mag[i + 1] - half) / (mag[i + 1] - mag[i])
    irw = (right - left) / up
    # main lobe ends at the first local minimum on each side
    i = c
    while mag[i + 1] < mag[i]:
        i += 1
    j = c
    while mag[j - 1] < mag[j]:
        j -= 1
    side = max(mag[i:c + n * up // 4].max(), mag[c - n * up // 4:j + 1].max())
    return irw, 20 * np.log10(side / p)


def test_sar_focus_quality_matches_paper(oracle_mod):
    """Section X scene parameters -> the printed theory IRW and PSLR."""
    g = json.load(open(os.path.join(GOLDEN, "paper_sar_focus.json")))
    s = g["scene"]
    beta_r = s["range_bandwidth_hz"] / s["range_sampling_hz"]
    len_r = s["range_pulse_samples"]
    beta_a = (2 * s["platform_speed_mps"] / s["antenna_length_m"]) / s["prf_hz"]
    len_a = int(round(s["synthetic_aperture_m"] / s["platform_speed_mps"] * s["prf_hz"]))
    assert (len_a, round(beta_a, 6)) == (1500, 0.1)
    n = 2048
    sc = workloads.sar_scene(n_az=n, n_rg=n, len_rg=len_r, beta_rg=beta_r, len_az=len_a,
                             beta_az=beta_a, sigma=0.0, targets=[(1024, 1024, 1.0)])
    out = oracle_mod.sar_chain(sc.raw, sc.range_ref, sc.az_ref)
    irw_r, pslr_r = _irw_pslr(out[1024, :])
    irw_a, pslr_a = _irw_pslr(out[:, 1024])
    th = g["theory"]
    assert abs(irw_r - th["irw_range_bins"]) < 0.02 * th["irw_range_bins"]
    assert abs(irw_a - th["irw_azimuth_bins"]) < 0.02 * th["irw_azimuth_bins"]
    assert abs(pslr_r - th["pslr_db"]) < 0.3
    assert abs(pslr_a - th["pslr_db"]) < 0.3
