"""The allocation-free SAR entry point against sar_form_image_ex, through the
C ABI: two calls in a row on one device, the second with a smaller image and
the other intermediate precision, each compared with the entry point that
takes a caller workspace (and with the oracle's plain definition at the
targets, as the other SAR parity tests do); the device's free memory does not
change across the calls after the first."""
import ctypes

import numpy as np
import pytest

import oracle
import workloads
from gpu_util import log, to_dev, to_host

pytestmark = pytest.mark.gpu

TOL = {0: 1e-5, 1: 3e-3}


@pytest.fixture(scope="module")
def lib():
    import torch

    assert torch.cuda.is_available()
    from paper_2609_32237_amd import _lib

    return _lib


def free_bytes():
    hip = ctypes.CDLL("libamdhip64.so.7")
    free, total = ctypes.c_size_t(), ctypes.c_size_t()
    assert hip.hipMemGetInfo(ctypes.byref(free), ctypes.byref(total)) == 0
    return free.value


def one_image(lib, sc, inter):
    import torch

    n_az, n_rg = sc.raw.shape
    raw, hr, ha = to_dev(sc.raw), to_dev(sc.range_ref), to_dev(sc.az_ref)
    ref_out = torch.empty_like(raw)
    ws = torch.empty(lib.sar_workspace_bytes(n_az, n_rg, inter), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    lib.sar_form_image_ex(n_az, n_rg, inter, raw.data_ptr(), hr.data_ptr(), ha.data_ptr(), ref_out.data_ptr(),
                          ws.data_ptr(), stream)
    out = torch.full_like(raw, float("nan"))
    torch.cuda.synchronize()
    before = free_bytes()
    lib.sar_form_image_noalloc(n_az, n_rg, inter, raw.data_ptr(), hr.data_ptr(), ha.data_ptr(), out.data_ptr(),
                               stream)
    torch.cuda.synchronize()
    after = free_bytes()
    return to_host(out), to_host(ref_out), before, after


def test_noalloc_matches_the_workspace_entry_point(lib):
    first = workloads.sar_scene()  # 4096 x 4096, FP32 intermediate: the array's largest image
    second = workloads.sar_scene(n_az=1024, n_rg=2048, n_targets=4, len_rg=256, len_az=128, min_sep=32, seed=21)
    frees = []
    for sc, inter in ((first, 0), (second, 1)):
        n_az, n_rg = sc.raw.shape
        log(f"noalloc {n_az}x{n_rg} inter={inter}")
        got, ref, before, after = one_image(lib, sc, inter)
        frees.append((before, after))
        assert np.isfinite(got).all()
        rel = np.linalg.norm((got - ref).astype(np.complex128)) / np.linalg.norm(ref.astype(np.complex128))
        log(f"  rel to sar_form_image_ex {rel:.3e}, max |diff| {np.abs(got - ref).max():.3e}")
        assert rel < TOL[inter]
        # the oracle's plain definition at the targets and at random points
        rng = np.random.default_rng(7)
        pa = np.concatenate([sc.targets_az, rng.integers(0, n_az, 16)])
        pr = np.concatenate([sc.targets_rg, rng.integers(0, n_rg, 16)])
        want = oracle.xcorr2d_points(sc.raw, sc.range_ref, sc.az_ref, pa, pr)
        have = got[pa, pr].astype(np.complex128)
        assert np.linalg.norm(have - want) / np.linalg.norm(want) < TOL[inter]
    # after the first call (which loads the array and copies the tables in),
    # a call changes no device allocation
    assert frees[1][1] == frees[1][0], frees
