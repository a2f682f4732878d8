"""Thin ctypes binding of libwino.so: the C-ABI's names, argument marshalling only.

Every function here takes the same arguments as its C counterpart in
``include/wino.h`` and returns its status / size unchanged.  Device buffers may
be given as torch CUDA tensors (fp32, contiguous; their data pointers are
passed) or as raw integer addresses; ``None`` passes NULL.  ``stream=None``
passes torch's current stream when a GPU is present, else NULL.  All compute
happens in the HIP kernels of libwino.so; nothing here computes.  If the library
has not been built, loading raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libwino.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "wino.h")

WINO_OK = 0
WINO_ERR_INVALID_ARG = -1
WINO_ERR_UNSUPPORTED = -2
WINO_ERR_WORKSPACE = -3
WINO_ERR_HIP = -4

WINO_FLAG_RELU = 0x001
WINO_ALGO_AUTO = 0x000
WINO_ALGO_FUSED = 0x100
WINO_ALGO_STAGED = 0x200
WINO_ALGO_SPLIT = 0x300
WINO_ALGO_LOWC = 0x400
WINO_ALGO_MASK = 0xF00


WINO_BLOCK_1x16 = 0x1000
WINO_BLOCK_4x4 = 0x2000


def WINO_CSPLIT(n: int) -> int:
    return (n & 0xF) << 16


def WINO_CSLICES(n: int) -> int:
    return (n & 0xF) << 20


class WinoError(RuntimeError):
    def __init__(self, status: int, where: str = ""):
        self.status = status
        super().__init__(f"{where}: {wino_status_string(status)} ({status})")


_lib = None

_c_int, _c_uint, _c_size, _vp = ctypes.c_int, ctypes.c_uint, ctypes.c_size_t, ctypes.c_void_p
_SIGS = {
    "wino_status_string": ([_c_int], ctypes.c_char_p),
    "wino_version": ([], _c_int),
    "wino_filter_bytes": ([_c_int] * 3, _c_size),
    "wino_input_tf_bytes": ([_c_int] * 6, _c_size),
    "wino_gemm_out_bytes": ([_c_int] * 6, _c_size),
    "wino_workspace_bytes": ([_c_int] * 7 + [_c_uint], _c_size),
    "wino_filter_transform": ([_vp, _vp] + [_c_int] * 3 + [_vp], _c_int),
    "wino_conv2d": ([_vp, _vp, _vp] + [_c_int] * 7 + [_c_uint, _vp, _c_size, _vp], _c_int),
    "wino_input_transform": ([_vp, _vp] + [_c_int] * 6 + [_vp], _c_int),
    "wino_batched_gemm": ([_vp, _vp, _vp] + [_c_int] * 7 + [_vp], _c_int),
    "wino_output_transform": ([_vp, _vp] + [_c_int] * 6 + [_c_uint, _vp], _c_int),
    "wino_maxpool2x2": ([_vp, _vp] + [_c_int] * 4 + [_vp], _c_int),
    "wino_probe_mfma_f32": ([_c_int, _vp, _vp], _c_int),
    "wino_plan_r": ([_c_int] * 8 + [_c_uint, _vp, _vp], _c_int),
    "wino_probe_mfma_f32_flops": ([_c_int], _c_size),
    "wino_filter_bytes_r": ([_c_int] * 4, _c_size),
    "wino_filter_transform_r": ([_vp, _vp] + [_c_int] * 4 + [_vp], _c_int),
    "wino_workspace_bytes_r": ([_c_int] * 8 + [_c_uint], _c_size),
    "wino_conv2d_r": ([_vp, _vp, _vp] + [_c_int] * 8 + [_c_uint, _vp, _c_size, _vp], _c_int),
    "wino_input_tf_bytes_r": ([_c_int] * 7, _c_size),
    "wino_gemm_out_bytes_r": ([_c_int] * 7, _c_size),
    "wino_input_transform_r": ([_vp, _vp] + [_c_int] * 7 + [_vp], _c_int),
    "wino_batched_gemm_r": ([_vp, _vp, _vp] + [_c_int] * 8 + [_vp], _c_int),
    "wino_output_transform_r": ([_vp, _vp] + [_c_int] * 7 + [_c_uint, _vp], _c_int),
    "wino_filter_bytes_1d": ([_c_int] * 4, _c_size),
    "wino_filter_transform_1d": ([_vp, _vp] + [_c_int] * 4 + [_vp], _c_int),
    "wino_workspace_bytes_1d": ([_c_int] * 9 + [_c_uint], _c_size),
    "wino_conv2d_1d": ([_vp, _vp, _vp] + [_c_int] * 9 + [_c_uint, _vp, _c_size, _vp], _c_int),
    "wino_workspace_bytes_nhwc": ([_c_int] * 7 + [_c_uint], _c_size),
    "wino_filter_bytes_p": ([_c_int] * 3 + [_c_uint], _c_size),
    "wino_filter_transform_p": ([_vp, _vp] + [_c_int] * 3 + [_c_uint, _vp], _c_int),
    "wino_conv2d_nhwc": ([_vp, _vp, _vp] + [_c_int] * 7 + [_c_uint, _vp, _c_size, _vp], _c_int),
    "wino_conv2d_noalloc": ([_vp, _vp, _vp] + [_c_int] * 7 + [_c_uint, _vp], _c_int),
}

WINO_NOALLOC_SCRATCH_BYTES = 64 << 20


def lib() -> ctypes.CDLL:
    """Load libwino.so (built in-tree).  Raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_1903_01521_amd.build` "
                               "or __graft_entry__.build() first")
        so = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            fn = getattr(so, name)
            fn.argtypes = args
            fn.restype = res
        _lib = so
    return _lib


def header_functions() -> list[str]:
    """Names of the functions include/wino.h declares."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(wino_\w+)\s*\(", text, flags=re.M)))


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    # torch tensor
    if not t.is_cuda:
        raise ValueError("device buffers must be CUDA (HIP) tensors")
    if not t.is_contiguous():
        raise ValueError("device buffers must be contiguous")
    return t.data_ptr()


def _fptr(t):
    if t is not None and not isinstance(t, int):
        import torch
        if t.dtype != torch.float32:
            raise ValueError("tensors must be float32")
    return _ptr(t)


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    try:
        import torch
        if torch.cuda.is_available():
            return torch.cuda.current_stream().cuda_stream
    except Exception:
        pass
    return None


def wino_status_string(status: int) -> str:
    return lib().wino_status_string(int(status)).decode()


def wino_version() -> int:
    return lib().wino_version()


def wino_filter_bytes(C, K, m) -> int:
    return lib().wino_filter_bytes(C, K, m)


def wino_input_tf_bytes(N, C, H, W, pad, m) -> int:
    return lib().wino_input_tf_bytes(N, C, H, W, pad, m)


def wino_gemm_out_bytes(N, K, H, W, pad, m) -> int:
    return lib().wino_gemm_out_bytes(N, K, H, W, pad, m)


def wino_workspace_bytes(N, C, H, W, K, pad, m, flags=0) -> int:
    return lib().wino_workspace_bytes(N, C, H, W, K, pad, m, flags)


def wino_filter_transform(g, U, C, K, m, stream=None) -> int:
    return lib().wino_filter_transform(_fptr(g), _fptr(U), C, K, m, _stream(stream))


def wino_conv2d(x, U, y, N, C, H, W, K, pad, m, flags=0, workspace=None, workspace_bytes=0,
                stream=None) -> int:
    return lib().wino_conv2d(_fptr(x), _fptr(U), _fptr(y), N, C, H, W, K, pad, m, flags,
                             _ptr(workspace), workspace_bytes, _stream(stream))


def wino_conv2d_noalloc(x, U, y, N, C, H, W, K, pad, m, flags=0, stream=None) -> int:
    return lib().wino_conv2d_noalloc(_fptr(x), _fptr(U), _fptr(y), N, C, H, W, K, pad, m, flags,
                                     _stream(stream))


def wino_input_transform(x, V, N, C, H, W, pad, m, stream=None) -> int:
    return lib().wino_input_transform(_fptr(x), _fptr(V), N, C, H, W, pad, m, _stream(stream))


def wino_batched_gemm(U, V, M, N, C, H, W, K, pad, m, stream=None) -> int:
    return lib().wino_batched_gemm(_fptr(U), _fptr(V), _fptr(M), N, C, H, W, K, pad, m, _stream(stream))


def wino_output_transform(M, y, N, K, H, W, pad, m, flags=0, stream=None) -> int:
    return lib().wino_output_transform(_fptr(M), _fptr(y), N, K, H, W, pad, m, flags, _stream(stream))


def wino_maxpool2x2(x, y, N, C, H, W, stream=None) -> int:
    return lib().wino_maxpool2x2(_fptr(x), _fptr(y), N, C, H, W, _stream(stream))


def wino_plan_r(N, C, H, W, K, pad, m, r, flags=0):
    """(status, algo, slices): the planner's choice, given the workspace it asks for."""
    algo, slices = ctypes.c_uint(0), ctypes.c_int(0)
    st = lib().wino_plan_r(N, C, H, W, K, pad, m, r, flags, ctypes.byref(algo), ctypes.byref(slices))
    return st, algo.value, slices.value


def wino_probe_mfma_f32(iters, out, stream=None) -> int:
    return lib().wino_probe_mfma_f32(iters, _fptr(out), _stream(stream))


def wino_probe_mfma_f32_flops(iters) -> int:
    return lib().wino_probe_mfma_f32_flops(iters)


def wino_filter_bytes_r(C, K, m, r) -> int:
    return lib().wino_filter_bytes_r(C, K, m, r)


def wino_filter_transform_r(g, U, C, K, m, r, stream=None) -> int:
    return lib().wino_filter_transform_r(_fptr(g), _fptr(U), C, K, m, r, _stream(stream))


def wino_workspace_bytes_r(N, C, H, W, K, pad, m, r, flags=0) -> int:
    return lib().wino_workspace_bytes_r(N, C, H, W, K, pad, m, r, flags)


def wino_conv2d_r(x, U, y, N, C, H, W, K, pad, m, r, flags=0, workspace=None, workspace_bytes=0,
                  stream=None) -> int:
    return lib().wino_conv2d_r(_fptr(x), _fptr(U), _fptr(y), N, C, H, W, K, pad, m, r, flags,
                               _ptr(workspace), workspace_bytes, _stream(stream))


def wino_input_tf_bytes_r(N, C, H, W, pad, m, r) -> int:
    return lib().wino_input_tf_bytes_r(N, C, H, W, pad, m, r)


def wino_gemm_out_bytes_r(N, K, H, W, pad, m, r) -> int:
    return lib().wino_gemm_out_bytes_r(N, K, H, W, pad, m, r)


def wino_input_transform_r(x, V, N, C, H, W, pad, m, r, stream=None) -> int:
    return lib().wino_input_transform_r(_fptr(x), _fptr(V), N, C, H, W, pad, m, r, _stream(stream))


def wino_batched_gemm_r(U, V, M, N, C, H, W, K, pad, m, r, stream=None) -> int:
    return lib().wino_batched_gemm_r(_fptr(U), _fptr(V), _fptr(M), N, C, H, W, K, pad, m, r, _stream(stream))


def wino_output_transform_r(M, y, N, K, H, W, pad, m, r, flags=0, stream=None) -> int:
    return lib().wino_output_transform_r(_fptr(M), _fptr(y), N, K, H, W, pad, m, r, flags, _stream(stream))


WINO_PREC_F16 = 0x010
WINO_PREC_BF16 = 0x020
WINO_PREC_MASK = 0x030


def wino_filter_bytes_p(C, K, m, prec) -> int:
    return lib().wino_filter_bytes_p(C, K, m, prec)


def wino_filter_transform_p(g, U, C, K, m, prec, stream=None) -> int:
    return lib().wino_filter_transform_p(_fptr(g), _ptr(U), C, K, m, prec, _stream(stream))


WINO_AXIS_W = 1
WINO_AXIS_H = 2


def wino_filter_bytes_1d(C, K, m, r) -> int:
    return lib().wino_filter_bytes_1d(C, K, m, r)


def wino_filter_transform_1d(g, U, C, K, m, r, stream=None) -> int:
    return lib().wino_filter_transform_1d(_fptr(g), _fptr(U), C, K, m, r, _stream(stream))


def wino_workspace_bytes_1d(N, C, H, W, K, pad, m, r, axis, flags=0) -> int:
    return lib().wino_workspace_bytes_1d(N, C, H, W, K, pad, m, r, axis, flags)


def wino_conv2d_1d(x, U, y, N, C, H, W, K, pad, m, r, axis, flags=0, workspace=None, workspace_bytes=0,
                   stream=None) -> int:
    return lib().wino_conv2d_1d(_fptr(x), _fptr(U), _fptr(y), N, C, H, W, K, pad, m, r, axis, flags,
                                _ptr(workspace), workspace_bytes, _stream(stream))


def wino_workspace_bytes_nhwc(N, C, H, W, K, pad, m, flags=0) -> int:
    return lib().wino_workspace_bytes_nhwc(N, C, H, W, K, pad, m, flags)


def wino_conv2d_nhwc(x, U, y, N, C, H, W, K, pad, m, flags=0, workspace=None, workspace_bytes=0,
                     stream=None) -> int:
    return lib().wino_conv2d_nhwc(_fptr(x), _fptr(U), _fptr(y), N, C, H, W, K, pad, m, flags,
                                  _ptr(workspace), workspace_bytes, _stream(stream))


def check(status: int, where: str = "wino") -> None:
    """Raise WinoError for a non-zero status."""
    if status != WINO_OK:
        raise WinoError(status, where)
