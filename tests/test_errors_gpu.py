"""Error contract of the C ABI on the GPU.

* A launch's status is its own: an earlier, unrelated HIP error left pending on
  the calling thread (here a failed hipSetDevice on an ordinal no machine has)
  is neither returned by the next library call nor cleared by it.
* fft_execute rejects input and output extents that partly overlap; in place
  and adjacent extents are accepted.
* The fixed-shift (block-floating-point) output scale of Section VII also
  protects the intermediates of the split forms: with FP16 storage, inputs of
  magnitude about 1000 and scale_log2 = log2 n, the four-step, three-pass,
  small-batch and long-column forms stay finite and match the oracle (and,
  where the single-pass kernel applies, its in-place result).  Without the
  split of the scale over the passes, their first pass would store up to
  n1 = 128 times the input, past binary16's 65504.
"""
import ctypes

import numpy as np
import pytest

import oracle
import workloads
from gpu_util import log, rel_rows, to_dev, to_host, widen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    import torch

    assert torch.cuda.is_available()
    from paper_2609_32237_amd import _lib

    return _lib


def test_launch_status_ignores_an_earlier_pending_error(lib):
    import torch

    hip = ctypes.CDLL("libamdhip64.so.7")  # the runtime this process already loaded
    hip.hipSetDevice.argtypes = [ctypes.c_int]
    n, batch = 4096, 8
    x = workloads.uniform_complex(batch, n, 31)
    xd = to_dev(x)
    out = torch.empty_like(xd)
    p = lib.fft_plan_create(n, batch, 1, n, 0, -1)
    try:
        torch.cuda.synchronize()
        bad = hip.hipSetDevice(9999)  # a host-side argument error, left pending
        rc = lib.lib.fft_execute(p, xd.data_ptr(), out.data_ptr(), None)
        pending = hip.hipGetLastError()  # read and clear before torch runs again
        log(f"hipSetDevice(9999) -> {bad}; fft_execute -> {rc}; hipGetLastError afterwards -> {pending}")
        assert bad != 0
        assert rc == lib.FFT_OK
        torch.cuda.synchronize()
    finally:
        lib.fft_plan_destroy(p)
    assert rel_rows(widen(to_host(out)), oracle.fft(x)).max() < 1e-5


def test_partly_overlapping_extents_are_rejected(lib):
    import torch

    n = 4096
    buf = torch.zeros(3 * n, dtype=torch.complex64, device="cuda")
    base = buf.data_ptr()
    p = lib.fft_plan_create(n, 1, 1, n, 0, -1)
    try:
        for shift in (8, 1, n - 1):
            assert lib.lib.fft_execute(p, base, base + 8 * shift, None) == lib.FFT_EINVAL, shift
            assert lib.lib.fft_execute(p, base + 8 * shift, base, None) == lib.FFT_EINVAL, shift
        assert lib.lib.fft_execute(p, base, base + 8 * n, None) == lib.FFT_OK  # adjacent
        assert lib.lib.fft_execute(p, base, base, None) == lib.FFT_OK  # in place
        torch.cuda.synchronize()
    finally:
        lib.fft_plan_destroy(p)
    # a strided layout: extent (n - 1) * stride + batch elements
    q = lib.fft_plan_create(1024, 2, 2, 1, 0, -1)
    try:
        assert lib.lib.fft_execute(q, base, base + 8 * 2000, None) == lib.FFT_EINVAL
        assert lib.lib.fft_execute(q, base, base + 8 * 2048, None) == lib.FFT_OK
        torch.cuda.synchronize()
    finally:
        lib.fft_plan_destroy(q)


def loud_inputs(n, rows, seed):
    """FP16 pairs of magnitude about 1000: a constant, a tone, uniform noise."""
    k = np.arange(n)
    rng = np.random.default_rng(seed)
    sig = [np.full(n, 1000.0 + 0j), 1000.0 * np.exp(2j * np.pi * ((29 * k) % n) / n)]
    sig.append(1000.0 * (rng.random(n) * 2 - 1 + 1j * (rng.random(n) * 2 - 1)))
    x = np.stack(sig[:rows])
    return np.stack([x.real, x.imag], -1).astype(np.float16)


def run_ex(lib, xd, od, n, batch, stride, dist, direction, s):
    import torch

    p = lib.fft_plan_create_ex(n, batch, stride, dist, 1, direction, s, 0)
    try:
        lib.fft_execute(p, xd.data_ptr(), od.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
    finally:
        lib.fft_plan_destroy(p)
    return to_host(od)


@pytest.mark.parametrize("n", [16384, 1 << 17, 1 << 23])
def test_fp16_shift_protects_split_intermediates(lib, n):
    import torch

    rows = 3 if n <= (1 << 17) else 1
    s = int(np.log2(n))
    x = loud_inputs(n, rows, 40 + s)
    ref = oracle.fft(x) * 2.0 ** -s
    xd = to_dev(x)
    for direction in (-1, 1):
        r = ref if direction == -1 else oracle.fft(x, 1) * 2.0 ** -s
        y = widen(run_ex(lib, xd, torch.empty_like(xd), n, rows, 1, n, direction, s))
        log(f"fp16 shift n={n} dir={direction}: finite {np.isfinite(y).all()}")
        assert np.isfinite(y).all()
        err = rel_rows(y, r)
        assert err.max() < 3e-3, err
        if n <= 16384:  # in place the single-pass kernel runs
            z = widen(run_inplace(lib, x, n, rows, direction, s))
            assert rel_rows(y, z).max() < 3e-3


def run_inplace(lib, x, n, rows, direction, s):
    xd = to_dev(x)
    return run_ex(lib, xd, xd, n, rows, 1, n, direction, s)


@pytest.mark.parametrize("n", [8192, 16384])
def test_fp16_shift_protects_long_column_intermediates(lib, n):
    """Columns of 8192 / 16384 points out of place: the two-pass column form."""
    import torch

    cols = 3
    s = int(np.log2(n))
    x = loud_inputs(n, cols, 50 + s)          # (cols, n, 2)
    m = np.ascontiguousarray(np.transpose(x, (1, 0, 2)))  # (n, cols, 2): column c is transform c
    md = to_dev(m)
    y = run_ex(lib, md, torch.empty_like(md), n, cols, cols, 1, -1, s)
    got = widen(np.ascontiguousarray(np.transpose(y, (1, 0, 2))))
    assert np.isfinite(got).all()
    assert rel_rows(got, oracle.fft(x) * 2.0 ** -s).max() < 3e-3
    inpl = to_dev(m)
    zi = widen(np.ascontiguousarray(np.transpose(run_ex(lib, inpl, inpl, n, cols, cols, 1, -1, s), (1, 0, 2))))
    assert rel_rows(got, zi).max() < 3e-3
