"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This module holds input synthesis only: random batches for the batched FFT
workloads and the simulated point-target SAR scene.  It contains none of the
method's arithmetic (no transform, no matched filtering); the HIP library and
the oracle each do that on their own.

Batched FFT inputs (paper, Section III "Platform and Methodology": uniform
random inputs on [-1, 1]).  Real and imaginary parts are drawn as float32 from
``numpy.random.default_rng(seed)``: ``u = rng.random((B, N, 2), float32)``,
``x = 2u - 1``.  ``rng.random`` returns k / 2**24, so ``2u - 1`` is exact in
float32 and lies in [-1, 1).  The fp16-storage workload draws the same way and
rounds to IEEE binary16 with round-to-nearest-even (``astype(float16)``).

SAR scene (paper, Section X "End to End: Range-Doppler SAR", re-parameterised
for the 4096 x 4096 image with 32 point targets): rows are pulses (azimuth),
columns are range samples.  Each target is a separable product of a centred
linear-FM range chirp and a centred azimuth quadratic-phase chirp, circularly
placed at its (azimuth, range) bin, plus complex Gaussian noise.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

# Workload table: (name, N, batch, storage, seed).  The two fp32 workloads at
# N = 8192 and N = 16384 each use a fresh generator seeded with 2.
FFT_WORKLOADS = {
    "fft_n1024_b64_fp32": dict(n=1024, batch=64, storage="fp32", seed=0),
    "fft_n4096_b32768_fp32": dict(n=4096, batch=32768, storage="fp32", seed=1),
    "fft_n8192_b16384_fp32": dict(n=8192, batch=16384, storage="fp32", seed=2),
    "fft_n16384_b8192_fp32": dict(n=16384, batch=8192, storage="fp32", seed=2),
    "fft_n16384_b16384_fp16": dict(n=16384, batch=16384, storage="fp16", seed=3),
}


def uniform_complex(batch: int, n: int, seed: int, storage: str = "fp32") -> np.ndarray:
    """Return a (batch, n) complex batch with iid uniform[-1, 1) parts.

    ``storage == "fp32"`` gives complex64.  ``storage == "fp16"`` gives a
    (batch, n, 2) float16 array holding interleaved (re, im) pairs: the fp32
    draw rounded to binary16 (round to nearest even).
    """
    rng = np.random.default_rng(seed)
    u = rng.random((batch, n, 2), dtype=np.float32)
    u *= np.float32(2.0)
    u -= np.float32(1.0)
    if storage == "fp32":
        return u.view(np.complex64).reshape(batch, n)
    if storage == "fp16":
        return u.astype(np.float16)
    raise ValueError(f"unknown storage {storage!r}")


def fft_workload(name: str) -> np.ndarray:
    """Input batch of one of the named FFT workloads in ``FFT_WORKLOADS``."""
    w = FFT_WORKLOADS[name]
    return uniform_complex(w["batch"], w["n"], w["seed"], w["storage"])


def fft_workload_rows(name: str, rows: np.ndarray) -> np.ndarray:
    """Selected transforms of a named workload, generated without the rest.

    ``rng.random`` fills a C-ordered array, so transform b consumes the
    generator's draws [2nb, 2n(b+1)).  The generator is advanced to each
    transform's offset (PCG64 ``advance``) so that a sample of a 1 GiB batch can
    be produced for the host-side checks without building the whole batch.
    Float32 draws consume one 32-bit half of a 64-bit output each, so the
    advance happens on 64-bit boundaries; transforms start at an even draw
    index because 2n is even.
    """
    w = FFT_WORKLOADS[name]
    n, seed, storage = w["n"], w["seed"], w["storage"]
    rows = np.asarray(rows, dtype=np.int64)
    out = np.empty((rows.size, n, 2), dtype=np.float32)
    for i, b in enumerate(rows):
        bitgen = np.random.PCG64(seed)
        bitgen.advance(int(b) * n)  # 2n float32 draws = n 64-bit outputs
        rng = np.random.Generator(bitgen)
        u = rng.random((n, 2), dtype=np.float32)
        out[i] = u * np.float32(2.0) - np.float32(1.0)
    if storage == "fp32":
        return out.view(np.complex64).reshape(rows.size, n)
    return out.astype(np.float16)


# --------------------------------------------------------------------------
# SAR scene
# --------------------------------------------------------------------------


@dataclass
class SarScene:
    """Simulated raw echo and the two time-domain reference chirps."""

    raw: np.ndarray  # (n_az, n_rg) complex64, rows = pulses
    range_ref: np.ndarray  # (n_rg,) complex64, chirp centred and wrapped
    az_ref: np.ndarray  # (n_az,) complex64
    targets_az: np.ndarray  # (K,) int64 azimuth bins
    targets_rg: np.ndarray  # (K,) int64 range bins
    amplitudes: np.ndarray  # (K,) float64
    params: dict = field(default_factory=dict)


def centred_chirp(n: int, length: int, beta: float) -> np.ndarray:
    """Centred quadratic-phase chirp h(t) = exp(+j pi beta t^2 / L), wrapped.

    t runs over the integers in [-L/2, L/2); h(t) is stored at index t mod n
    and the array is zero elsewhere.  The instantaneous frequency beta t / L
    spans [-beta/2, beta/2) cycles per sample, a bandwidth of beta times the
    sampling rate.  Returned in complex128; callers cast once.
    """
    if length > n or length % 2:
        raise ValueError("chirp length must be even and at most n")
    t = np.arange(-length // 2, length // 2, dtype=np.float64)
    h = np.zeros(n, dtype=np.complex128)
    h[np.mod(t.astype(np.int64), n)] = np.exp(1j * np.pi * beta * t * t / length)
    return h


def _place_targets(rng, k, lo_az, hi_az, lo_rg, hi_rg, min_sep):
    """Rejection-sample k bins with pairwise |da| >= min_sep and |dr| >= min_sep."""
    az, rg = [], []
    tries = 0
    while len(az) < k:
        tries += 1
        if tries > 1_000_000:
            raise RuntimeError("could not place targets with the requested separation")
        a = int(rng.integers(lo_az, hi_az))
        r = int(rng.integers(lo_rg, hi_rg))
        if all(abs(a - a2) >= min_sep and abs(r - r2) >= min_sep for a2, r2 in zip(az, rg)):
            az.append(a)
            rg.append(r)
    return np.array(az, dtype=np.int64), np.array(rg, dtype=np.int64)


def sar_scene(
    n_az: int = 4096,
    n_rg: int = 4096,
    n_targets: int = 32,
    len_rg: int = 1024,
    beta_rg: float = 0.8,
    len_az: int = 512,
    beta_az: float = 0.8,
    sigma: float = 0.01,
    seed: int = 4,
    min_sep: int = 32,
    amp_range=(0.5, 1.0),
    targets=None,
) -> SarScene:
    """Build the point-target scene.

    Targets lie in azimuth [L_a/2, n_az - L_a/2) and range [L_r/2, n_rg - L_r/2)
    so that no echo wraps.  One generator seeded with ``seed`` draws, in order,
    the target positions, the amplitudes (uniform on ``amp_range``) and the
    noise (each of re and im normal with standard deviation ``sigma``).
    ``targets`` may instead give explicit ((a, r, A), ...) triples.  The echo is
    summed in complex128 and cast once to complex64.
    """
    rng = np.random.default_rng(seed)
    h_r = centred_chirp(n_rg, len_rg, beta_rg)
    h_a = centred_chirp(n_az, len_az, beta_az)
    if targets is None:
        ta, tr = _place_targets(
            rng, n_targets, len_az // 2, n_az - len_az // 2, len_rg // 2, n_rg - len_rg // 2, min_sep
        )
        amp = rng.uniform(amp_range[0], amp_range[1], size=n_targets)
    else:
        ta = np.array([t[0] for t in targets], dtype=np.int64)
        tr = np.array([t[1] for t in targets], dtype=np.int64)
        amp = np.array([t[2] for t in targets], dtype=np.float64)
    raw = np.zeros((n_az, n_rg), dtype=np.complex128)
    t_a = np.arange(-len_az // 2, len_az // 2)
    t_r = np.arange(-len_rg // 2, len_rg // 2)
    ha_seg = h_a[np.mod(t_a, n_az)]
    hr_seg = h_r[np.mod(t_r, n_rg)]
    for a, r, amplitude in zip(ta, tr, amp):
        rows = np.mod(a + t_a, n_az)
        cols = np.mod(r + t_r, n_rg)
        raw[np.ix_(rows, cols)] += amplitude * np.outer(ha_seg, hr_seg)
    if sigma > 0:
        noise = rng.normal(0.0, sigma, size=(n_az, n_rg, 2))
        raw += noise[..., 0] + 1j * noise[..., 1]
    params = dict(
        n_az=n_az, n_rg=n_rg, n_targets=len(ta), len_rg=len_rg, beta_rg=beta_rg,
        len_az=len_az, beta_az=beta_az, sigma=sigma, seed=seed, min_sep=min_sep,
    )
    return SarScene(
        raw=raw.astype(np.complex64),
        range_ref=h_r.astype(np.complex64),
        az_ref=h_a.astype(np.complex64),
        targets_az=ta,
        targets_rg=tr,
        amplitudes=amp,
        params=params,
    )


# --------------------------------------------------------------------------
# Range-Doppler scene: the paper's L-band stripmap geometry
# --------------------------------------------------------------------------

SPEED_OF_LIGHT = 299_792_458.0

# Six point targets as (pulse of closest approach, range bin of closest
# approach, amplitude): spread over the frame so that every synthetic
# aperture (about 1500 pulses) and every echo (1200 samples plus 2 bins of
# migration) lies inside it.
RD_TARGETS = ((1024, 512, 1.0), (1024, 2304, 1.0), (2048, 1280, 1.0),
              (2048, 2816, 1.0), (3072, 256, 1.0), (3072, 1792, 1.0))


@dataclass
class RdScene:
    """Simulated stripmap echo, the transmitted pulse replica and the geometry."""

    raw: np.ndarray  # (n_az, n_rg) complex64, rows = pulses
    range_ref: np.ndarray  # (n_rg,) complex64, the pulse replica from index 0
    geometry: dict  # wavelength, speed, prf, range_bin, r_near (the processor's inputs)
    targets_az: np.ndarray  # (K,) int64 pulse of closest approach
    targets_rg: np.ndarray  # (K,) int64 range bin of closest approach
    amplitudes: np.ndarray  # (K,) float64
    params: dict = field(default_factory=dict)


def rd_scene(
    n_az: int = 4096,
    n_rg: int = 4096,
    wavelength: float = 0.24,
    bandwidth: float = 100e6,
    fs: float = 120e6,
    speed: float = 200.0,
    prf: float = 500.0,
    antenna: float = 8.0,
    pulse_samples: int = 1200,
    r_near: float = 17500.0,
    targets=RD_TARGETS,
    sigma: float = 0.01,
    seed: int = 5,
) -> RdScene:
    """Stripmap echo of point targets (paper, Section X: lambda 0.24 m,
    B 100 MHz, fs 120 MHz, v 200 m/s, PRF 500 Hz, 8 m antenna, six targets and
    complex Gaussian noise; the pulse lasts ``pulse_samples`` samples).

    Broadside geometry, start-stop approximation.  Pulse a is sent at slow time
    a / PRF; target i is closest at pulse a_i, at slant range
    R0_i = r_near + n_i * dr with dr = c / (2 fs) the range bin spacing, so
    R_i(a) = sqrt(R0_i^2 + (v (a - a_i) / PRF)^2).  The antenna beam (width
    lambda / L) lights the target while |v (a - a_i) / PRF| <= lambda R0_i / (2L),
    which is its synthetic aperture (600 m at 20 km).  Range sample m is taken
    at fast time tau_m = 2 r_near / c + m / fs, and the baseband echo is

        A_i p(tau_m - 2 R_i(a) / c) exp(-j 4 pi R_i(a) / lambda),

    with p(u) = exp(j pi K (u - T/2)^2) for 0 <= u < T (T = pulse_samples / fs,
    K = B / T: an up-chirp spanning -B/2 .. B/2) and zero elsewhere.  The
    replica is p sampled at m / fs, m = 0 .. pulse_samples - 1.  The echo is
    summed in complex128, noise (re and im each normal with standard deviation
    ``sigma``, from ``default_rng(seed)``) added, and cast once to complex64.
    """
    dr = SPEED_OF_LIGHT / (2.0 * fs)
    t_p = pulse_samples / fs
    k_r = bandwidth / t_p
    raw = np.zeros((n_az, n_rg), dtype=np.complex128)
    ta = np.array([t[0] for t in targets], dtype=np.int64)
    tr = np.array([t[1] for t in targets], dtype=np.int64)
    amp = np.array([t[2] for t in targets], dtype=np.float64)
    m_all = np.arange(n_rg, dtype=np.float64)
    for a_i, n_i, amp_i in zip(ta, tr, amp):
        r0 = r_near + n_i * dr
        half = wavelength * r0 / (2.0 * antenna)
        a_lo = int(np.ceil(a_i - half * prf / speed))
        a_hi = int(np.floor(a_i + half * prf / speed))
        if a_lo < 0 or a_hi >= n_az:
            raise ValueError("a target's synthetic aperture leaves the frame")
        pulses = np.arange(a_lo, a_hi + 1)
        x = speed * (pulses - a_i) / prf
        r = np.sqrt(r0 * r0 + x * x)
        delay = (r - r_near) / dr  # echo start in (fractional) range samples
        lo = int(np.floor(delay.min()))
        hi = int(np.ceil(delay.max())) + pulse_samples + 1
        if lo < 0 or hi > n_rg:
            raise ValueError("a target's echo leaves the range window")
        m = m_all[lo:hi]
        u = (m[None, :] - delay[:, None]) / fs
        inside = (u >= 0.0) & (u < t_p)
        echo = np.where(inside, np.exp(1j * np.pi * k_r * (u - t_p / 2) ** 2), 0.0)
        echo *= (amp_i * np.exp(-4j * np.pi * r / wavelength))[:, None]
        raw[a_lo:a_hi + 1, lo:hi] += echo
    if sigma > 0:
        rng = np.random.default_rng(seed)
        noise = rng.normal(0.0, sigma, size=(n_az, n_rg, 2))
        raw += noise[..., 0] + 1j * noise[..., 1]
    u = np.arange(pulse_samples) / fs
    ref = np.zeros(n_rg, dtype=np.complex128)
    ref[:pulse_samples] = np.exp(1j * np.pi * k_r * (u - t_p / 2) ** 2)
    geometry = dict(wavelength=wavelength, speed=speed, prf=prf, range_bin=dr, r_near=r_near)
    params = dict(n_az=n_az, n_rg=n_rg, bandwidth=bandwidth, fs=fs, antenna=antenna,
                  pulse_samples=pulse_samples, sigma=sigma, seed=seed, **geometry)
    return RdScene(raw=raw.astype(np.complex64), range_ref=ref.astype(np.complex64), geometry=geometry,
                   targets_az=ta, targets_rg=tr, amplitudes=amp, params=params)


def rd_scene_small(**kw) -> RdScene:
    """A 1024 x 1024 version of the same scene for quick checks: PRF 125 Hz
    keeps the 600 m aperture (375 pulses) and the 1.8-bin migration, and a
    300-sample (2.5 us) pulse fits the shorter range window."""
    args = dict(n_az=1024, n_rg=1024, prf=125.0, pulse_samples=300,
                targets=((256, 128, 1.0), (512, 640, 1.0), (768, 384, 1.0), (768, 700, 0.7)))
    args.update(kw)
    return rd_scene(**args)
