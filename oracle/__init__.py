"""fp64 CPU oracle for the batched FFT and the SAR chains -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never calls it and
shares no code with it.  The arithmetic lives in ``oracle.c`` (plain C, fp64);
this module only loads the compiled library and marshals numpy arrays.

Every function takes and returns complex128 numpy arrays.  Inputs stored in
complex64 or binary16 are widened exactly before the call.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build() -> str:
    """Compile oracle.c into liboracle.so with gcc (fp64, no fast-math)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", "-fno-fast-math",
           "-ffp-contract=off", "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    i64, dp, ip = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    lib.oracle_dft_direct.argtypes = [i64, i64, i64, i64, ip, dp, dp]
    lib.oracle_fft.argtypes = [i64, i64, i64, i64, ip, dp, dp, ip]
    lib.oracle_sar_chain.argtypes = [i64, i64, dp, dp, dp, dp, ip]
    lib.oracle_xcorr2d_points.argtypes = [i64, i64, dp, dp, dp, i64, dp, dp, dp]
    lib.oracle_rd_chain.argtypes = [i64, i64, dp, dp, dp, ip, dp, ip]
    lib.oracle_rd_interp_table.argtypes = [dp]
    for f in (lib.oracle_dft_direct, lib.oracle_fft, lib.oracle_sar_chain, lib.oracle_xcorr2d_points,
              lib.oracle_rd_chain, lib.oracle_rd_interp_table):
        f.restype = ctypes.c_int
    _lib = lib
    return lib


def default_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _c128(x) -> np.ndarray:
    x = np.asarray(x)
    if x.dtype == np.float16:
        # binary16 storage holds interleaved (re, im) pairs: widen exactly
        if not x.shape or x.shape[-1] != 2:
            raise ValueError("binary16 input must end in an (re, im) axis of length 2")
        x = x.astype(np.float64)
        x = x[..., 0] + 1j * x[..., 1]
    return np.ascontiguousarray(x, dtype=np.complex128)


def _check(rc: int, what: str):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with code {rc}")


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def fft_layout(buf, n: int, batch: int, stride: int, dist: int, sign: int = -1,
               direct: bool = False, nthreads: int | None = None) -> np.ndarray:
    """Transform a flat buffer in the advanced layout (element j of transform b
    at index b*dist + j*stride).  Entries outside the transforms are copied
    through unchanged.  ``direct`` selects the O(N^2) definition."""
    x = _c128(buf).reshape(-1)
    y = x.copy()
    lib = _load()
    if direct:
        rc = lib.oracle_dft_direct(n, batch, stride, dist, sign, _ptr(x), _ptr(y))
    else:
        rc = lib.oracle_fft(n, batch, stride, dist, sign, _ptr(x), _ptr(y),
                            nthreads or default_threads())
    _check(rc, "fft")
    return y


def fft(x, sign: int = -1, nthreads: int | None = None) -> np.ndarray:
    """Unnormalised DFT of each row of a (batch, n) array (radix-2, fp64)."""
    x = _c128(x)
    if x.ndim == 1:
        return fft(x[None], sign, nthreads)[0]
    b, n = x.shape
    return fft_layout(x, n, b, 1, n, sign, nthreads=nthreads).reshape(b, n)


def dft_direct(x, sign: int = -1) -> np.ndarray:
    """Unnormalised DFT of each row by the O(N^2) definition (fp64)."""
    x = _c128(x)
    if x.ndim == 1:
        return dft_direct(x[None], sign)[0]
    b, n = x.shape
    return fft_layout(x, n, b, 1, n, sign, direct=True).reshape(b, n)


def sar_chain(raw, range_ref, az_ref, nthreads: int | None = None) -> np.ndarray:
    """Range compression then azimuth compression of an (n_az, n_rg) echo."""
    raw = _c128(raw)
    n_az, n_rg = raw.shape
    hr = _c128(range_ref).reshape(-1)
    ha = _c128(az_ref).reshape(-1)
    if hr.size != n_rg or ha.size != n_az:
        raise ValueError("reference lengths must match the image axes")
    out = np.empty_like(raw)
    rc = _load().oracle_sar_chain(n_az, n_rg, _ptr(raw), _ptr(hr), _ptr(ha), _ptr(out),
                                  nthreads or default_threads())
    _check(rc, "sar_chain")
    return out


def xcorr2d_points(raw, range_ref, az_ref, pts_az, pts_rg) -> np.ndarray:
    """2-D circular cross-correlation of the echo with both references, by
    direct summation, at the listed (azimuth, range) points."""
    raw = _c128(raw)
    n_az, n_rg = raw.shape
    hr = _c128(range_ref).reshape(-1)
    ha = _c128(az_ref).reshape(-1)
    pa = np.ascontiguousarray(pts_az, dtype=np.int64).reshape(-1)
    pr = np.ascontiguousarray(pts_rg, dtype=np.int64).reshape(-1)
    if pa.size != pr.size:
        raise ValueError("point lists differ in length")
    out = np.empty(pa.size, dtype=np.complex128)
    rc = _load().oracle_xcorr2d_points(n_az, n_rg, _ptr(raw), _ptr(hr), _ptr(ha), pa.size,
                                       _ptr(pa), _ptr(pr), _ptr(out))
    _check(rc, "xcorr2d_points")
    return out


RD_TAPS = 8
RD_SUB = 128
GEOMETRY_KEYS = ("wavelength", "speed", "prf", "range_bin", "r_near")


def rd_interp_table() -> np.ndarray:
    """The range-cell migration interpolator's table, (RD_SUB + 1, RD_TAPS)."""
    tab = np.empty((RD_SUB + 1, RD_TAPS), dtype=np.float64)
    _check(_load().oracle_rd_interp_table(_ptr(tab)), "rd_interp_table")
    return tab


def rd_chain(raw, range_ref, geometry: dict, stop_after: int = 5, nthreads: int | None = None) -> np.ndarray:
    """The full range-Doppler chain on an (n_az, n_rg) echo (rows = pulses).

    ``geometry`` holds wavelength [m], speed [m/s], prf [Hz], range_bin [m]
    (slant-range spacing of the range samples) and r_near [m] (slant range of
    range bin 0).  ``stop_after`` returns the image after step 1 (range
    compression), 2 (azimuth FFT / n_az), 3 (RCMC), 4 (azimuth filter) or 5
    (azimuth inverse FFT: the focused image)."""
    raw = _c128(raw)
    n_az, n_rg = raw.shape
    hr = _c128(range_ref).reshape(-1)
    if hr.size != n_rg:
        raise ValueError("range reference length must match the range axis")
    geo = np.array([float(geometry[k]) for k in GEOMETRY_KEYS], dtype=np.float64)
    out = np.empty_like(raw)
    rc = _load().oracle_rd_chain(n_az, n_rg, _ptr(raw), _ptr(hr), _ptr(geo), int(stop_after), _ptr(out),
                                 nthreads or default_threads())
    _check(rc, "rd_chain")
    return out
