"""ctypes binding of libmi355fft.so: the C ABI of include/mi355fft.h, same names.

Argument marshalling only: every transform runs in the HIP kernels of the
library.  Device pointers are plain integers (``tensor.data_ptr()``) and
streams are ``hipStream_t`` handles (``torch.cuda.current_stream().cuda_stream``).
There is no fallback: if the library is missing, importing this module fails.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmi355fft.so")

FFT_STORAGE_FP32 = 0
FFT_STORAGE_FP16 = 1
FFT_FORWARD = -1
FFT_INVERSE = 1
FFT_OK = 0
FFT_EINVAL = -1
FFT_EUNSUPPORTED = -2
FFT_ENOMEM = -3
FFT_EALIGN = -4
FFT_EHIP = -5

# every symbol include/mi355fft.h declares
FFT_FLAG_FP16_EXCHANGE = 1
FFT_FLAG_MATRIX_UNITS = 2

EXPORTS = ("fft_plan_create", "fft_plan_create_ex", "fft_execute", "fft_plan_destroy", "sar_workspace_bytes",
           "sar_form_image_ex", "sar_form_image", "sar_form_image_noalloc", "sar_rd_workspace_bytes",
           "sar_rd_form_image", "fft_strerror")


class SarGeometry(ctypes.Structure):
    """struct sar_geometry: broadside stripmap acquisition (metres, Hz, m/s)."""

    _fields_ = [("wavelength", ctypes.c_double), ("speed", ctypes.c_double), ("prf", ctypes.c_double),
                ("range_bin", ctypes.c_double), ("r_near", ctypes.c_double)]

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'` "
        "(there is no CPU fallback)")

lib = ctypes.CDLL(LIB_PATH)
_i64, _vp, _int = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
lib.fft_plan_create.argtypes = [_i64, _i64, _i64, _i64, _int, _int, ctypes.POINTER(_vp)]
lib.fft_plan_create.restype = _int
lib.fft_plan_create_ex.argtypes = [_i64, _i64, _i64, _i64, _int, _int, _int, ctypes.c_uint, ctypes.POINTER(_vp)]
lib.fft_plan_create_ex.restype = _int
lib.fft_execute.argtypes = [_vp, _vp, _vp, _vp]
lib.fft_execute.restype = _int
lib.fft_plan_destroy.argtypes = [_vp]
lib.fft_plan_destroy.restype = _int
lib.sar_workspace_bytes.argtypes = [_i64, _i64, _int]
lib.sar_workspace_bytes.restype = ctypes.c_size_t
lib.sar_form_image_ex.argtypes = [_i64, _i64, _int, _vp, _vp, _vp, _vp, _vp, _vp]
lib.sar_form_image_ex.restype = _int
lib.sar_form_image.argtypes = [_vp, _vp, _vp, _vp, _vp]
lib.sar_form_image.restype = _int
lib.sar_form_image_noalloc.argtypes = [_i64, _i64, _int, _vp, _vp, _vp, _vp, _vp]
lib.sar_form_image_noalloc.restype = _int
lib.sar_rd_workspace_bytes.argtypes = [_i64, _i64, _int]
lib.sar_rd_workspace_bytes.restype = ctypes.c_size_t
lib.sar_rd_form_image.argtypes = [_i64, _i64, _int, ctypes.POINTER(SarGeometry), _vp, _vp, _vp, _vp, _vp]
lib.sar_rd_form_image.restype = _int
lib.fft_strerror.argtypes = [_int]
lib.fft_strerror.restype = ctypes.c_char_p


class FFTError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {fft_strerror(code)} ({code})")
        self.code = code


def _check(code: int, what: str) -> int:
    if code != FFT_OK:
        raise FFTError(code, what)
    return code


def fft_strerror(code: int) -> str:
    return lib.fft_strerror(code).decode()


def fft_plan_create(n: int, batch: int, stride: int, dist: int, storage: int, dir: int) -> int:
    """Returns an opaque plan handle (int); raises FFTError on failure."""
    p = _vp()
    _check(lib.fft_plan_create(n, batch, stride, dist, storage, dir, ctypes.byref(p)), "fft_plan_create")
    return p.value


def fft_plan_create_ex(n: int, batch: int, stride: int, dist: int, storage: int, dir: int, scale_log2: int = 0,
                       flags: int = 0) -> int:
    """fft_plan_create with the output scale 2^-scale_log2 and plan flags."""
    p = _vp()
    _check(lib.fft_plan_create_ex(n, batch, stride, dist, storage, dir, scale_log2, flags, ctypes.byref(p)),
           "fft_plan_create_ex")
    return p.value


def fft_execute(plan: int, in_ptr: int, out_ptr: int, stream: int = 0) -> None:
    _check(lib.fft_execute(plan, in_ptr, out_ptr, stream), "fft_execute")


def fft_plan_destroy(plan) -> None:
    _check(lib.fft_plan_destroy(plan), "fft_plan_destroy")


def sar_workspace_bytes(n_az: int, n_rg: int, inter_storage: int) -> int:
    return int(lib.sar_workspace_bytes(n_az, n_rg, inter_storage))


def sar_form_image_ex(n_az: int, n_rg: int, inter_storage: int, raw: int, range_ref: int, az_ref: int,
                      out: int, workspace: int, stream: int = 0) -> None:
    _check(lib.sar_form_image_ex(n_az, n_rg, inter_storage, raw, range_ref, az_ref, out, workspace, stream),
           "sar_form_image_ex")


def sar_form_image(raw: int, range_ref: int, az_ref: int, out: int, stream: int = 0) -> None:
    _check(lib.sar_form_image(raw, range_ref, az_ref, out, stream), "sar_form_image")


def sar_form_image_noalloc(n_az: int, n_rg: int, inter_storage: int, raw: int, range_ref: int, az_ref: int,
                           out: int, stream: int = 0) -> None:
    """sar_form_image_ex with the library's fixed device array as workspace."""
    _check(lib.sar_form_image_noalloc(n_az, n_rg, inter_storage, raw, range_ref, az_ref, out, stream),
           "sar_form_image_noalloc")


def sar_rd_workspace_bytes(n_az: int, n_rg: int, inter_storage: int) -> int:
    return int(lib.sar_rd_workspace_bytes(n_az, n_rg, inter_storage))


def geometry(g) -> SarGeometry:
    """A SarGeometry from a mapping with the struct's field names (or itself)."""
    if isinstance(g, SarGeometry):
        return g
    return SarGeometry(*(float(g[k]) for k, _ in SarGeometry._fields_))


def sar_rd_form_image(n_az: int, n_rg: int, inter_storage: int, geo, raw: int, range_ref: int, out: int,
                      workspace: int, stream: int = 0) -> None:
    g = geometry(geo)
    _check(lib.sar_rd_form_image(n_az, n_rg, inter_storage, ctypes.byref(g), raw, range_ref, out, workspace,
                                 stream), "sar_rd_form_image")
