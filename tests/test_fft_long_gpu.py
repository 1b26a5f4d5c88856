"""Transforms longer than 16384 points: the two-pass four-step form (Section VI:
once the transform no longer fits on chip it takes a second pass through
memory), n = n1 * n2, through the C ABI against the oracle.

Bounds as for the single-pass transforms: per-transform relative L2 error
<= 1e-5 with FP32 storage and <= 3e-3 with FP16 storage (the FP16 form also
rounds the intermediate it keeps in the output buffer).
"""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import log, rel_rows, to_dev, to_host, widen

pytestmark = pytest.mark.gpu

TOL = {0: 1e-5, 1: 3e-3}


@pytest.fixture(scope="module")
def lib():
    import torch

    assert torch.cuda.is_available()
    from paper_2609_32237_amd import _lib

    return _lib


def run(lib, x, n, batch, dist, storage, direction, out=None):
    import torch

    xd = to_dev(x)
    od = torch.zeros_like(xd) if out is None else out
    p = lib.fft_plan_create(n, batch, 1, dist, storage, direction)
    try:
        lib.fft_execute(p, xd.data_ptr(), od.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
    finally:
        lib.fft_plan_destroy(p)
    return to_host(od)


@pytest.mark.parametrize("log2n", [15, 16, 17, 18, 19, 20, 21, 22, 23])
@pytest.mark.parametrize("storage", [0, 1])
def test_long_transforms_match_oracle(lib, log2n, storage):
    n = 1 << log2n
    batch = 3 if log2n <= 18 else 1
    st = "fp32" if storage == 0 else "fp16"
    x = workloads.uniform_complex(batch, n, 900 + log2n, st)
    for direction in (-1, 1):
        log(f"long n=2^{log2n} {st} dir={direction}")
        y = widen(run(lib, x, n, batch, n, storage, direction))
        err = rel_rows(y, oracle.fft(x, direction))
        assert err.max() < TOL[storage], (log2n, storage, direction, err.max())


def test_padded_batch_distance(lib):
    """dist > n: the gaps between transforms are neither read nor written."""
    n, batch, dist = 1 << 16, 3, (1 << 16) + 96
    rng = np.random.default_rng(5)
    buf = (rng.standard_normal(batch * dist) + 1j * rng.standard_normal(batch * dist)).astype(np.complex64)
    import torch

    out = torch.full((batch * dist,), 7 + 7j, dtype=torch.complex64, device="cuda")
    y = run(lib, buf, n, batch, dist, 0, -1, out=out)
    ref = oracle.fft_layout(buf, n, batch, 1, dist, -1)
    for b in range(batch):
        seg = slice(b * dist, b * dist + n)
        assert rel_rows(y[seg][None].astype(np.complex128), ref[seg][None]).max() < 1e-5
        gap = y[b * dist + n:(b + 1) * dist]
        assert np.all(gap == np.complex64(7 + 7j))


def test_2_pow_24_matches_oracle(lib):
    n = 1 << 24
    x = workloads.uniform_complex(1, n, 924)
    log("long n=2^24")
    y = run(lib, x, n, 1, n, 0, -1)
    err = rel_rows(y.astype(np.complex128), oracle.fft(x))
    assert err.max() < 1e-5, err


@pytest.mark.parametrize("storage", [0, 1])
def test_three_pass_lengths_match_oracle(lib, storage):
    """Beyond 2^24 the transform takes three passes (n1 x na x nb, columns of
    at most 1024 points); 2^25 = 256 x 256 x 512, two transforms in both
    directions, and a scaled inverse."""
    import torch

    n, batch = 1 << 25, 2
    st = "fp32" if storage == 0 else "fp16"
    x = workloads.uniform_complex(batch, n, 925, st)
    for direction in (-1, 1):
        log(f"three-pass n=2^25 {st} dir={direction}")
        y = widen(run(lib, x, n, batch, n, storage, direction))
        err = rel_rows(y, oracle.fft(x, direction))
        assert err.max() < TOL[storage], (storage, direction, err.max())
    if storage == 0:
        xd = to_dev(x)
        yd = torch.empty_like(xd)
        p = lib.fft_plan_create_ex(n, batch, 1, n, 0, 1, 25, 0)
        try:
            lib.fft_execute(p, xd.data_ptr(), yd.data_ptr(), torch.cuda.current_stream().cuda_stream)
            torch.cuda.synchronize()
        finally:
            lib.fft_plan_destroy(p)
        err = rel_rows(widen(to_host(yd)), oracle.fft(x, 1) / n)
        assert err.max() < TOL[0], err.max()


def test_largest_length_closed_forms(lib):
    """n = 2^28 (2 GiB per FP32 transform): an impulse at n0 transforms to
    exp(-2 pi i k n0 / n); sampled outputs against that closed form in double,
    and Parseval over the whole output."""
    import torch

    n = 1 << 28
    n0 = 123457
    x = torch.zeros(n, dtype=torch.complex64, device="cuda")
    x[n0] = 1.0 + 0.0j
    y = torch.empty_like(x)
    p = lib.fft_plan_create(n, 1, 1, n, 0, -1)
    try:
        log("long n=2^28 impulse")
        lib.fft_execute(p, x.data_ptr(), y.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
    finally:
        lib.fft_plan_destroy(p)
    del x
    k = np.unique(np.r_[0, 1, n - 1, n // 2, np.random.default_rng(6).integers(0, n, 4096)])
    got = y[torch.from_numpy(k).cuda()].cpu().numpy().astype(np.complex128)
    want = np.exp(-2j * np.pi * ((k * n0) % n) / n)
    assert abs(got - want).max() < 2e-5
    energy = float((y.real.double() ** 2 + y.imag.double() ** 2).sum())
    assert abs(energy / n - 1.0) < 1e-5


def test_batch_beyond_one_grid_dimension(lib):
    """More than 65535 transforms: the host splits the batch across launches;
    transforms on both sides of each split against the oracle."""
    import torch

    n, batch = 1 << 15, 65539
    g = torch.Generator(device="cuda").manual_seed(7)
    x = (torch.rand(batch, n, 2, device="cuda", generator=g) * 2 - 1).half()
    y = torch.empty_like(x)
    p = lib.fft_plan_create(n, batch, 1, n, 1, -1)
    try:
        log(f"long n=2^15 batch={batch} fp16")
        lib.fft_execute(p, x.data_ptr(), y.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
    finally:
        lib.fft_plan_destroy(p)
    rows = np.array([0, 1, 65533, 65534, 65535, 65536, batch - 1])
    xs = x[torch.from_numpy(rows).cuda()].cpu().numpy()
    ys = widen(y[torch.from_numpy(rows).cuda()].cpu().numpy())
    assert rel_rows(ys, oracle.fft(xs)).max() < 3e-3


def test_in_place_is_rejected_for_long_transforms(lib):
    import torch

    n = 1 << 15
    x = torch.zeros(n, dtype=torch.complex64, device="cuda")
    p = lib.fft_plan_create(n, 1, 1, n, 0, -1)
    try:
        with pytest.raises(lib.FFTError) as e:
            lib.fft_execute(p, x.data_ptr(), x.data_ptr(), 0)
        assert e.value.code == lib.FFT_EINVAL
    finally:
        lib.fft_plan_destroy(p)


@pytest.mark.parametrize("batch", [1, 3, 16, 17])
def test_small_batches_at_16384_split_out_of_place(lib, batch):
    """Up to 16 out-of-place transforms of 16384 points run as 128 x 128
    four-step (Section VI: split one transform over several workgroups when
    the batch is small); in place, and from 17 on, they stay single-pass.
    Both against the oracle."""
    import torch

    n = 16384
    x = workloads.uniform_complex(batch, n, 950 + batch)
    ref = oracle.fft(x)
    log(f"split n=16384 batch={batch}")
    y = widen(run(lib, x, n, batch, n, 0, -1))
    assert rel_rows(y, ref).max() < 1e-5
    xd = to_dev(x)
    p = lib.fft_plan_create(n, batch, 1, n, 0, -1)
    try:
        lib.fft_execute(p, xd.data_ptr(), xd.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
    finally:
        lib.fft_plan_destroy(p)
    assert rel_rows(widen(to_host(xd)), ref).max() < 1e-5


def test_every_short_column_shape(lib):
    """The 512-point column kernels (both strip widths) as both passes of a
    2^18-point transform, forced through MI355FFT_COL_VARIANT."""
    import os

    n = 1 << 18
    x = workloads.uniform_complex(2, n, 960)
    ref = oracle.fft(x)
    for v in range(2):
        os.environ["MI355FFT_COL_VARIANT"] = str(v)
        try:
            log(f"long n=2^18 column variant {v}")
            y = widen(run(lib, x, n, 2, n, 0, -1))
        finally:
            os.environ.pop("MI355FFT_COL_VARIANT", None)
        assert rel_rows(y, ref).max() < 1e-5, v
