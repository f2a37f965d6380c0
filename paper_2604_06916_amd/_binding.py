"""Thin ctypes binding of libsolfp4.so (declared in include/solfp4.h).

Argument marshalling only: torch supplies device memory and the current
stream; every step of the computation runs in the library's HIP kernels.
Loading fails loudly if the library has not been built.
"""
from __future__ import annotations

import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsolfp4.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2604_06916_amd.build`")

lib = ctypes.CDLL(LIB_PATH)

_p = ctypes.c_void_p
_i64 = ctypes.c_int64
_sz = ctypes.c_size_t

lib.solfp4_strerror.restype = ctypes.c_char_p
lib.solfp4_strerror.argtypes = [ctypes.c_int]
lib.solfp4_version.restype = ctypes.c_int
lib.solfp4_version.argtypes = []
lib.nvfp4_quantize_workspace_bytes.restype = _sz
lib.nvfp4_quantize_workspace_bytes.argtypes = [_i64, _i64]
lib.nvfp4_quantize.restype = ctypes.c_int
lib.nvfp4_quantize.argtypes = [_p, _i64, _i64, _p, _p, _p, _p, _sz, _p]
lib.nvfp4_gemm.restype = ctypes.c_int
lib.nvfp4_gemm.argtypes = [_p, _p, _p, _p, _p, _p, _p, _p, _p, _sz, _i64, _i64, _i64, _p]
lib.nvfp4_gemm_workspace_bytes.restype = _sz
lib.nvfp4_gemm_workspace_bytes.argtypes = [_i64, _i64, _i64]
lib.nvfp4_linear_workspace_bytes.restype = _sz
lib.nvfp4_linear_workspace_bytes.argtypes = [_i64, _i64, _i64]
lib.nvfp4_linear.restype = ctypes.c_int
lib.nvfp4_linear.argtypes = [_p, _p, _p, _p, _p, _p, _p, _sz, _i64, _i64, _i64, _p]

lib.mxfp4_quantize.restype = ctypes.c_int
lib.mxfp4_quantize.argtypes = [_p, _i64, _i64, _p, _p, _p]
lib.mxfp4_gemm.restype = ctypes.c_int
lib.mxfp4_gemm.argtypes = [_p, _p, _p, _p, _p, _p, _i64, _i64, _i64, _p]
lib.mxfp4_linear_workspace_bytes.restype = _sz
lib.mxfp4_linear_workspace_bytes.argtypes = [_i64, _i64]
lib.mxfp4_linear.restype = ctypes.c_int
lib.mxfp4_linear.argtypes = [_p, _p, _p, _p, _p, _p, _sz, _i64, _i64, _i64, _p]

EXPORTED = ["solfp4_strerror", "solfp4_version", "nvfp4_quantize_workspace_bytes",
            "nvfp4_quantize", "nvfp4_gemm", "nvfp4_gemm_workspace_bytes",
            "nvfp4_linear_workspace_bytes", "nvfp4_linear",
            "mxfp4_quantize", "mxfp4_gemm", "mxfp4_linear_workspace_bytes", "mxfp4_linear"]


class Solfp4Error(RuntimeError):
    def __init__(self, status: int):
        self.status = status
        super().__init__(f"solfp4 status {status}: {lib.solfp4_strerror(status).decode()}")


def _check(status: int):
    if status != 0:
        raise Solfp4Error(status)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _need(t, dtype, shape, name):
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous() or not t.is_cuda:
        raise ValueError(f"{name}: expected contiguous CUDA {dtype} {tuple(shape)}, "
                         f"got {t.dtype} {tuple(t.shape)} on {t.device}")


def nvfp4_quantize_workspace_bytes(rows: int, K: int) -> int:
    return lib.nvfp4_quantize_workspace_bytes(rows, K)


def nvfp4_gemm_workspace_bytes(M: int, N: int, K: int) -> int:
    return lib.nvfp4_gemm_workspace_bytes(M, N, K)


def nvfp4_linear_workspace_bytes(M: int, N: int, K: int) -> int:
    return lib.nvfp4_linear_workspace_bytes(M, N, K)


def nvfp4_quantize(x, codes=None, scales=None, global_scale=None, workspace=None, stream=None):
    """x: BF16 [rows, K] -> (codes uint8 [rows, K/2], scales uint8 [rows, K/16],
    global_scale float32 [1]).  Outputs may be passed in to avoid allocation."""
    rows, K = x.shape
    dev = x.device
    if codes is None:
        codes = torch.empty((rows, K // 2), dtype=torch.uint8, device=dev)
    if scales is None:
        scales = torch.empty((rows, K // 16), dtype=torch.uint8, device=dev)
    if global_scale is None:
        global_scale = torch.empty(1, dtype=torch.float32, device=dev)
    if workspace is None:
        workspace = torch.empty(max(nvfp4_quantize_workspace_bytes(rows, K), 256),
                                dtype=torch.uint8, device=dev)
    _need(x, torch.bfloat16, (rows, K), "x")
    _check(lib.nvfp4_quantize(_ptr(x), rows, K, _ptr(codes), _ptr(scales), _ptr(global_scale),
                              _ptr(workspace), workspace.numel(), _stream(stream)))
    return codes, scales, global_scale


def nvfp4_gemm(a_codes, a_scales, a_global_scale, b_codes, b_scales, b_global_scale,
               bias=None, out=None, workspace=None, stream=None, split=True):
    """Block-scaled NVFP4 GEMM: A [M, K] (packed), B [N, K] (packed) -> BF16 [M, N].
    `workspace` (uint8, at least nvfp4_gemm_workspace_bytes(M, N, K)) is
    allocated when needed and not given; split=False passes none (no split
    of the last round's tiles)."""
    M, N = a_codes.shape[0], b_codes.shape[0]
    K = a_codes.shape[1] * 2
    if b_codes.shape[1] * 2 != K:
        raise ValueError("A and B disagree on K")
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=a_codes.device)
    _need(out, torch.bfloat16, (M, N), "out")
    if bias is not None:
        _need(bias, torch.bfloat16, (N,), "bias")
    if not split:
        workspace = None
    elif workspace is None:
        need = nvfp4_gemm_workspace_bytes(M, N, K)
        if need:
            workspace = torch.empty(need, dtype=torch.uint8, device=a_codes.device)
    _check(lib.nvfp4_gemm(_ptr(a_codes), _ptr(a_scales), _ptr(a_global_scale), _ptr(b_codes),
                          _ptr(b_scales), _ptr(b_global_scale), _ptr(bias), _ptr(out),
                          _ptr(workspace), 0 if workspace is None else workspace.numel(),
                          M, N, K, _stream(stream)))
    return out


def nvfp4_linear(x, w_codes, w_scales, w_global_scale, bias=None, out=None, workspace=None,
                 stream=None):
    """NVFP4 linear: quantize BF16 x [M, K] on the fly, GEMM with the packed
    weight [N, K], add bias -> BF16 [M, N]."""
    M, K = x.shape
    N = w_codes.shape[0]
    _need(x, torch.bfloat16, (M, K), "x")
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    _need(out, torch.bfloat16, (M, N), "out")
    if bias is not None:
        _need(bias, torch.bfloat16, (N,), "bias")
    if workspace is None:
        workspace = torch.empty(nvfp4_linear_workspace_bytes(M, N, K), dtype=torch.uint8,
                                device=x.device)
    _check(lib.nvfp4_linear(_ptr(x), _ptr(w_codes), _ptr(w_scales), _ptr(w_global_scale),
                            _ptr(bias), _ptr(out), _ptr(workspace), workspace.numel(),
                            M, N, K, _stream(stream)))
    return out


def mxfp4_linear_workspace_bytes(M: int, K: int) -> int:
    return lib.mxfp4_linear_workspace_bytes(M, K)


def mxfp4_quantize(x, codes=None, scales=None, stream=None):
    """x: BF16 [rows, K] (K % 32 == 0) -> (codes uint8 [rows, K/2],
    scales uint8 [rows, K/32], E8M0)."""
    rows, K = x.shape
    _need(x, torch.bfloat16, (rows, K), "x")
    if codes is None:
        codes = torch.empty((rows, K // 2), dtype=torch.uint8, device=x.device)
    if scales is None:
        scales = torch.empty((rows, K // 32), dtype=torch.uint8, device=x.device)
    _check(lib.mxfp4_quantize(_ptr(x), rows, K, _ptr(codes), _ptr(scales), _stream(stream)))
    return codes, scales


def mxfp4_gemm(a_codes, a_scales, b_codes, b_scales, bias=None, out=None, stream=None):
    """MXFP4 GEMM: A [M, K] (packed), B [N, K] (packed) -> BF16 [M, N]."""
    M, N = a_codes.shape[0], b_codes.shape[0]
    K = a_codes.shape[1] * 2
    if b_codes.shape[1] * 2 != K:
        raise ValueError("A and B disagree on K")
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=a_codes.device)
    _need(out, torch.bfloat16, (M, N), "out")
    if bias is not None:
        _need(bias, torch.bfloat16, (N,), "bias")
    _check(lib.mxfp4_gemm(_ptr(a_codes), _ptr(a_scales), _ptr(b_codes), _ptr(b_scales),
                          _ptr(bias), _ptr(out), M, N, K, _stream(stream)))
    return out


def mxfp4_linear(x, w_codes, w_scales, bias=None, out=None, workspace=None, stream=None):
    """MXFP4 linear: quantize BF16 x [M, K] on the fly, GEMM with the packed
    weight [N, K], add bias -> BF16 [M, N]."""
    M, K = x.shape
    N = w_codes.shape[0]
    _need(x, torch.bfloat16, (M, K), "x")
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    _need(out, torch.bfloat16, (M, N), "out")
    if bias is not None:
        _need(bias, torch.bfloat16, (N,), "bias")
    if workspace is None:
        workspace = torch.empty(mxfp4_linear_workspace_bytes(M, K), dtype=torch.uint8,
                                device=x.device)
    _check(lib.mxfp4_linear(_ptr(x), _ptr(w_codes), _ptr(w_scales), _ptr(bias), _ptr(out),
                            _ptr(workspace), workspace.numel(), M, N, K, _stream(stream)))
    return out
