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
