"""Tensor conveniences over the C ABI (device pointers and streams only).

PyTorch provides device memory and the current stream; every transform runs
in the library's HIP kernels through ``_lib``.  Complex FP32 data is a
complex64 tensor; complex FP16 data is a float16 tensor whose last axis holds
the (re, im) pair.
"""
from __future__ import annotations

import torch

from . import _lib
from ._lib import FFT_FORWARD, FFT_INVERSE, FFT_STORAGE_FP16, FFT_STORAGE_FP32  # noqa: F401


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _storage_of(t: torch.Tensor) -> int:
    if t.dtype == torch.complex64:
        return FFT_STORAGE_FP32
    if t.dtype == torch.float16 and t.shape[-1] == 2:
        return FFT_STORAGE_FP16
    raise TypeError("expected complex64, or float16 with a trailing (re, im) axis")


class Plan:
    """A plan for ``batch`` transforms of ``n`` points in an advanced layout."""

    def __init__(self, n: int, batch: int, stride: int = 1, dist: int | None = None,
                 storage: int = FFT_STORAGE_FP32, direction: int = FFT_FORWARD, scale_log2: int = 0,
                 flags: int = 0):
        self.n, self.batch, self.stride = n, batch, stride
        self.dist = n if dist is None else dist
        self.storage, self.direction = storage, direction
        self.handle = _lib.fft_plan_create_ex(n, batch, stride, self.dist, storage, direction, scale_log2, flags)

    def execute(self, inp: torch.Tensor, out: torch.Tensor, stream=None) -> torch.Tensor:
        for t in (inp, out):
            if not t.is_cuda or _storage_of(t) != self.storage:
                raise TypeError("tensors must live on the GPU in the plan's storage format")
        _lib.fft_execute(self.handle, inp.data_ptr(), out.data_ptr(), _stream(stream))
        return out

    def close(self):
        if self.handle:
            _lib.fft_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def fft(x: torch.Tensor, direction: int = FFT_FORWARD, out: torch.Tensor | None = None,
        stream=None) -> torch.Tensor:
    """Unnormalised transform of each row of a contiguous (batch, n) batch."""
    storage = _storage_of(x)
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    n = x.shape[-2] if storage == FFT_STORAGE_FP16 else x.shape[-1]
    batch = x.numel() // (n * (2 if storage == FFT_STORAGE_FP16 else 1))
    out = torch.empty_like(x) if out is None else out
    plan = Plan(n, batch, 1, n, storage, direction)
    plan.execute(x, out, stream)
    plan.close()
    return out


def sar_form_image(raw: torch.Tensor, range_ref: torch.Tensor, az_ref: torch.Tensor,
                   inter_storage: int = FFT_STORAGE_FP32, out: torch.Tensor | None = None,
                   workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Range-Doppler image of a (n_az, n_rg) complex64 echo."""
    n_az, n_rg = raw.shape
    for t in (raw, range_ref, az_ref):
        if t.dtype != torch.complex64 or not t.is_cuda or not t.is_contiguous():
            raise TypeError("raw and references must be contiguous complex64 GPU tensors")
    out = torch.empty_like(raw) if out is None else out
    nbytes = _lib.sar_workspace_bytes(n_az, n_rg, inter_storage)
    if nbytes == 0:
        raise _lib.FFTError(_lib.FFT_EUNSUPPORTED, "sar_workspace_bytes")
    if workspace is None:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=raw.device)
    _lib.sar_form_image_ex(n_az, n_rg, inter_storage, raw.data_ptr(), range_ref.data_ptr(),
                           az_ref.data_ptr(), out.data_ptr(), workspace.data_ptr(), _stream(stream))
    return out


def sar_rd_form_image(raw: torch.Tensor, range_ref: torch.Tensor, geometry,
                      inter_storage: int = FFT_STORAGE_FP32, out: torch.Tensor | None = None,
                      workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Focused image of a (n_az, n_rg) complex64 stripmap echo by the full
    range-Doppler chain; ``geometry`` maps wavelength, speed, prf, range_bin
    and r_near to their values."""
    n_az, n_rg = raw.shape
    for t in (raw, range_ref):
        if t.dtype != torch.complex64 or not t.is_cuda or not t.is_contiguous():
            raise TypeError("raw and range_ref must be contiguous complex64 GPU tensors")
    out = torch.empty_like(raw) if out is None else out
    nbytes = _lib.sar_rd_workspace_bytes(n_az, n_rg, inter_storage)
    if nbytes == 0:
        raise _lib.FFTError(_lib.FFT_EUNSUPPORTED, "sar_rd_workspace_bytes")
    if workspace is None:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=raw.device)
    _lib.sar_rd_form_image(n_az, n_rg, inter_storage, geometry, raw.data_ptr(), range_ref.data_ptr(),
                           out.data_ptr(), workspace.data_ptr(), _stream(stream))
    return out
