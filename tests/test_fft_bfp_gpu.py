"""FP16 robustness options of fft_plan_create_ex (paper, Section VII and
Section X), through the C ABI:

* the fixed-shift output scale 2^-s, the block-floating-point schedule the
  paper applies to FP16 storage of coherent data (outputs grow up to N for
  coherent inputs and overflow binary16 without it).  The scale is exact in
  FP32, so scaled FP32 outputs must equal the unscaled ones times 2^-s bit for
  bit; FP16 outputs of coherent inputs must match the oracle within the FP16
  bound instead of overflowing;
* the binary16 exchange between stages (Section VII: about 6 dB less
  accurate than the FP32 exchange): within the FP16 bound of 3e-3, and
  measurably less accurate than the default, which shows the flag is in
  effect.
"""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import log, rel_rows, to_dev, to_host, widen

pytestmark = pytest.mark.gpu

SIZES = [1024, 2048, 4096, 8192, 16384]


@pytest.fixture(scope="module")
def lib():
    import torch

    assert torch.cuda.is_available()
    from paper_2609_32237_amd import _lib

    return _lib


def run(lib, x, n, batch, stride, dist, storage, direction, scale_log2=0, flags=0):
    import torch

    xd = to_dev(x)
    out = xd.clone()
    p = lib.fft_plan_create_ex(n, batch, stride, dist, storage, direction, scale_log2, flags)
    try:
        lib.fft_execute(p, xd.data_ptr(), out.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
    finally:
        lib.fft_plan_destroy(p)
    return to_host(out)


@pytest.mark.parametrize("n", SIZES + [1 << 17])
def test_fp32_scale_is_exact(lib, n):
    """Rows (and the four-step form beyond 16384) and columns: scaled output
    == unscaled output * 2^-s, bit for bit."""
    s = int(np.log2(n))
    x = workloads.uniform_complex(3, n, 970)
    a = run(lib, x, n, 3, 1, n, 0, -1)
    b = run(lib, x, n, 3, 1, n, 0, -1, scale_log2=s)
    assert np.array_equal(b, (a * np.float32(2.0 ** -s)).astype(np.complex64))
    if n <= 16384:
        m = workloads.uniform_complex(n, 9, 971)
        a = run(lib, m, n, 9, 9, 1, 0, 1)
        b = run(lib, m, n, 9, 9, 1, 0, 1, scale_log2=5)
        assert np.array_equal(b, (a * np.float32(2.0 ** -5)).astype(np.complex64))


def coherent_inputs(n):
    """Constant, a pure tone and a linear-FM chirp of amplitude 8: their
    spectra peak at 8n, 8n and about 8 sqrt(n / 0.8), beyond binary16 for the
    first two from n = 8192 on."""
    k = np.arange(n)
    tone = 8 * np.exp(2j * np.pi * ((37 * k) % n) / n)
    t = k - n / 2
    chirp = 8 * np.exp(1j * np.pi * 0.8 * t * t / n)
    rows = np.stack([np.full(n, 8.0 + 0j), tone, chirp])
    pairs = np.stack([rows.real, rows.imag], -1).astype(np.float16)
    return pairs


@pytest.mark.parametrize("n", SIZES)
def test_fp16_coherent_inputs_need_the_shift(lib, n):
    x = coherent_inputs(n)
    s = int(np.log2(n))
    ref = oracle.fft(x) * 2.0 ** -s
    log(f"bfp n={n}")
    y = widen(run(lib, x, n, 3, 1, n, 1, -1, scale_log2=s))
    assert np.isfinite(y).all()
    assert rel_rows(y, ref).max() < 3e-3
    if n >= 8192:  # unscaled, the constant's and the tone's peaks (8n) overflow binary16
        raw = widen(run(lib, x, n, 3, 1, n, 1, -1))
        assert not np.isfinite(raw[:2]).all()
    # block exponent kept by the caller: the inverse of the scaled spectrum,
    # unnormalised, returns the input
    back = widen(run(lib, run(lib, x, n, 3, 1, n, 1, -1, scale_log2=s), n, 3, 1, n, 1, 1))
    assert rel_rows(back, widen(x)).max() < 3e-3


@pytest.mark.parametrize("n", SIZES)
def test_fp16_exchange_flag(lib, n):
    x = workloads.uniform_complex(6, n, 980, "fp16")
    ref = oracle.fft(x)
    e_std = rel_rows(widen(run(lib, x, n, 6, 1, n, 1, -1)), ref)
    e_half = rel_rows(widen(run(lib, x, n, 6, 1, n, 1, -1, flags=lib.FFT_FLAG_FP16_EXCHANGE)), ref)
    log(f"fp16 exchange n={n}: rel {e_std.mean():.2e} (FP32 exchange) vs {e_half.mean():.2e} "
        f"({20 * np.log10(e_half.mean() / e_std.mean()):.1f} dB)")
    assert e_half.max() < 3e-3
    assert e_half.mean() > 1.2 * e_std.mean()
    inv = rel_rows(widen(run(lib, x, n, 6, 1, n, 1, 1, flags=lib.FFT_FLAG_FP16_EXCHANGE)), oracle.fft(x, 1))
    assert inv.max() < 3e-3


def test_every_fp16_exchange_shape(lib):
    """Both binary16-exchange shapes at 16384 (MI355FFT_HALF_VARIANT)."""
    import os

    n = 16384
    x = workloads.uniform_complex(4, n, 990, "fp16")
    ref = oracle.fft(x)
    for v in range(2):
        os.environ["MI355FFT_HALF_VARIANT"] = str(v)
        try:
            y = widen(run(lib, x, n, 4, 1, n, 1, -1, flags=lib.FFT_FLAG_FP16_EXCHANGE))
        finally:
            os.environ.pop("MI355FFT_HALF_VARIANT", None)
        assert rel_rows(y, ref).max() < 3e-3, v



@pytest.mark.parametrize("n", [4096, 16384])
def test_matrix_unit_transforms(lib, n):
    """FFT_FLAG_MATRIX_UNITS: radix-16 stages as MFMA products (binary16 data,
    FP32 accumulation).  Within the FP16 bound, both directions, in place too;
    its accuracy is reported beside the vector kernel's."""
    import torch

    x = workloads.uniform_complex(9, n, 995, "fp16")
    f = lib.FFT_FLAG_MATRIX_UNITS
    for direction in (-1, 1):
        ref = oracle.fft(x, direction)
        e_mm = rel_rows(widen(run(lib, x, n, 9, 1, n, 1, direction, flags=f)), ref)
        e_v = rel_rows(widen(run(lib, x, n, 9, 1, n, 1, direction)), ref)
        log(f"matrix units n={n} dir={direction}: rel {e_mm.mean():.2e} (vector {e_v.mean():.2e}), "
            f"SQNR {-20 * np.log10(e_mm.mean()):.1f} dB")
        assert e_mm.max() < 3e-3
    # closed form: an impulse at n0 gives exp(-2 pi i k n0 / n) up to binary16 rounding
    n0 = 77
    imp = np.zeros((1, n, 2), np.float16)
    imp[0, n0, 0] = 1.0
    k = np.arange(n)
    y = widen(run(lib, imp, n, 1, 1, n, 1, -1, flags=f))[0]
    assert abs(y - np.exp(-2j * np.pi * ((k * n0) % n) / n)).max() < 2e-3
    # in place
    xd = to_dev(x)
    p = lib.fft_plan_create_ex(n, 9, 1, n, 1, -1, 0, f)
    try:
        lib.fft_execute(p, xd.data_ptr(), xd.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
    finally:
        lib.fft_plan_destroy(p)
    assert rel_rows(widen(to_host(xd)), oracle.fft(x)).max() < 3e-3
