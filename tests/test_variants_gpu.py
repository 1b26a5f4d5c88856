"""Every kernel variant computes the same transform (the paper's regression test
that forces N = 8192 through its two-half exchange path, Section VI, applied to
every exchange / twiddle / persistence variant here).

Variants are forced with MI355FFT_ROW_VARIANT / MI355FFT_COL_VARIANT, which
plan creation and the SAR entry points read; an index the size does not have
makes them return FFT_EINVAL, which is how the count is found.
"""
import os

import numpy as np
import pytest

import oracle
import workloads
from gpu_util import log, rel_rows, to_dev, to_host, widen

pytestmark = pytest.mark.gpu

SIZES = [1024, 2048, 4096, 8192, 16384]
TOL = {0: 1e-5, 1: 3e-3}


@pytest.fixture(scope="module")
def lib():
    import torch

    assert torch.cuda.is_available()
    from paper_2609_32237_amd import _lib

    return _lib


def env_var(layout):
    return "MI355FFT_ROW_VARIANT" if layout == "rows" else "MI355FFT_COL_VARIANT"


def count_variants(lib, n, layout):
    k = 0
    try:
        while True:
            os.environ[env_var(layout)] = str(k)
            try:
                p = lib.fft_plan_create(n, 8, 1 if layout == "rows" else 8, n if layout == "rows" else 1, 0, -1)
            except lib.FFTError as e:
                assert e.code == lib.FFT_EINVAL
                return k
            lib.fft_plan_destroy(p)
            k += 1
    finally:
        os.environ.pop(env_var(layout), None)


def run(lib, x, n, batch, stride, dist, storage, direction):
    import torch

    xd = to_dev(x)
    out = xd.clone()
    p = lib.fft_plan_create(n, batch, stride, dist, storage, direction)
    try:
        lib.fft_execute(p, xd.data_ptr(), out.data_ptr(), torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
    finally:
        lib.fft_plan_destroy(p)
    return to_host(out)


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("layout", ["rows", "cols"])
def test_every_variant_matches_oracle(lib, n, layout):
    nv = count_variants(lib, n, layout)
    assert nv >= 2
    for v in range(nv):
        os.environ[env_var(layout)] = str(v)
        try:
            for storage in (0, 1):
                for direction in (-1, 1):
                    log(f"variant {layout} n={n} v={v} storage={storage} dir={direction}")
                    st = "fp32" if storage == 0 else "fp16"
                    if layout == "rows":
                        x = (workloads.uniform_complex(5, n, 600 + v) if storage == 0
                             else workloads.uniform_complex(5, n, 600 + v, "fp16"))
                        y = widen(run(lib, x, n, 5, 1, n, storage, direction))
                        err = rel_rows(y, oracle.fft(x, direction))
                    else:
                        m = (workloads.uniform_complex(n, 13, 700 + v) if storage == 0
                             else workloads.uniform_complex(n, 13, 700 + v, "fp16"))
                        y = run(lib, m, n, 11, 13, 1, storage, direction)
                        ref = oracle.fft_layout(m, n, 11, 13, 1, direction).reshape(n, 13)
                        err = rel_rows(widen(y).T[:11], ref.T[:11])
                        assert np.array_equal(y[:, 11:], m[:, 11:])
                    assert err.max() < TOL[storage], (v, storage, direction, err.max())
        finally:
            os.environ.pop(env_var(layout), None)


@pytest.mark.parametrize("n", SIZES)
def test_every_row_variant_on_a_batch_larger_than_the_device(lib, n):
    """Enough transforms that persistent variants loop several times per workgroup:
    a CU holds at most 2048 threads, so at most 256 * 2048 / THREADS workgroups of
    C transforms are resident; these batches exceed that by 1.5x or more."""
    batch = {1024: 24581, 2048: 12293, 4096: 6149, 8192: 3077, 16384: 1541}[n]
    x = workloads.uniform_complex(batch, n, 800)
    rows = np.unique(np.r_[0, batch - 1, batch - 2, np.random.default_rng(1).integers(0, batch, 24)])
    ref = oracle.fft(x[rows])
    for v in range(count_variants(lib, n, "rows")):
        log(f"large batch rows n={n} v={v} batch={batch}")
        os.environ["MI355FFT_ROW_VARIANT"] = str(v)
        try:
            y = run(lib, x, n, batch, 1, n, 0, -1)
        finally:
            os.environ.pop("MI355FFT_ROW_VARIANT", None)
        assert rel_rows(widen(y[rows]), ref).max() < 1e-5, v


def test_every_sar_variant(lib):
    """SAR with every (row, column) variant pair at 4096 x 4096 on a small echo
    window, both intermediate precisions."""
    import torch

    from paper_2609_32237_amd import torch_api

    sc = workloads.sar_scene(n_targets=8, seed=9)
    ref = oracle.sar_chain(sc.raw, sc.range_ref, sc.az_ref)
    raw, hr, ha = to_dev(sc.raw), to_dev(sc.range_ref), to_dev(sc.az_ref)
    for vr in range(count_variants(lib, 4096, "rows")):
        for vc in range(count_variants(lib, 4096, "cols")):
            for inter in (0, 1):
                log(f"sar variants row={vr} col={vc} inter={inter}")
                os.environ["MI355FFT_ROW_VARIANT"] = str(vr)
                os.environ["MI355FFT_COL_VARIANT"] = str(vc)
                try:
                    img = torch_api.sar_form_image(raw, hr, ha, inter)
                    torch.cuda.synchronize()
                finally:
                    os.environ.pop("MI355FFT_ROW_VARIANT", None)
                    os.environ.pop("MI355FFT_COL_VARIANT", None)
                got = to_host(img).astype(np.complex128)
                e = np.linalg.norm(got - ref) / np.linalg.norm(ref)
                assert e < TOL[inter], (vr, vc, inter, e)

