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
lib.nvfp4_quantize_amax.restype = ctypes.c_int
lib.nvfp4_quantize_amax.argtypes = [_p, _i64, _i64, _p, _sz, _p]
lib.nvfp4_quantize_encode.restype = ctypes.c_int
lib.nvfp4_quantize_encode.argtypes = [_p, _i64, _i64, _p, _p, _p, _p, _sz, _p]
lib.nvfp4_quantize_noalloc.restype = ctypes.c_int
lib.nvfp4_quantize_noalloc.argtypes = [_p, _i64, _i64, _p, _p, _p, _p]
lib.nvfp4_gemm.restype = ctypes.c_int
lib.nvfp4_gemm.argtypes = [_p, _p, _p, _p, _p, _p, _p, _p, _p, _sz, _i64, _i64, _i64, _p]
lib.nvfp4_gemm_workspace_bytes.restype = _sz
lib.nvfp4_gemm_workspace_bytes.argtypes = [_i64, _i64, _i64]
lib.nvfp4_linear_workspace_bytes.restype = _sz
lib.nvfp4_linear_workspace_bytes.argtypes = [_i64, _i64, _i64]
lib.nvfp4_linear.restype = ctypes.c_int
lib.nvfp4_linear.argtypes = [_p, _p, _p, _p, _p, _p, _p, _sz, _i64, _i64, _i64, _p]

lib.solfp4_gemm_plan.restype = ctypes.c_int
lib.solfp4_gemm_plan.argtypes = [ctypes.c_int, _i64, _i64, _i64, ctypes.c_int,
                                 ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int),
                                 ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int)]

lib.mxfp4_quantize.restype = ctypes.c_int
lib.mxfp4_quantize.argtypes = [_p, _i64, _i64, _p, _p, _p]
lib.mxfp4_gemm.restype = ctypes.c_int
lib.mxfp4_gemm.argtypes = [_p, _p, _p, _p, _p, _p, _i64, _i64, _i64, _p]
lib.mxfp4_linear_workspace_bytes.restype = _sz
lib.mxfp4_linear_workspace_bytes.argtypes = [_i64, _i64]
lib.mxfp4_linear.restype = ctypes.c_int
lib.mxfp4_linear.argtypes = [_p, _p, _p, _p, _p, _p, _sz, _i64, _i64, _i64, _p]

EXPORTED = ["solfp4_strerror", "solfp4_version", "solfp4_gemm_plan",
            "nvfp4_quantize_workspace_bytes", "nvfp4_quantize", "nvfp4_quantize_amax",
            "nvfp4_quantize_encode", "nvfp4_quantize_noalloc",
            "nvfp4_gemm",
            "nvfp4_gemm_workspace_bytes", "nvfp4_linear_workspace_bytes", "nvfp4_linear",
            "mxfp4_quantize", "mxfp4_gemm", "mxfp4_linear_workspace_bytes", "mxfp4_linear"]

FORMAT_NVFP4, FORMAT_MXFP4 = 0, 1
KERNEL_NAMES = {0: None, 1: "nvfp4_gemm_lane_kernel", 2: "nvfp4_gemm_kernel",
                3: "mxfp4_gemm_kernel", 4: "nvfp4_gemm_small_kernel", 5: "nvfp4_gemm_wavek_kernel",
                6: "mxfp4_gemm_wavek_kernel"}


class Solfp4Error(RuntimeError):
    def __init__(self, status: int):
        self.status = status
        super().__init__(f"solfp4 status {status}: {lib.solfp4_strerror(status).decode()}")


def _check(status: int):
    if status != 0:
        raise Solfp4Error(status)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream, device):
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream


def _alloc(shape, dtype, device, stream):
    """A temporary or output on `device`, allocated under `stream` so the
    caching allocator does not hand its memory to other work before the
    library's kernels on that stream are done with it."""
    with torch.cuda.stream(stream):
        return torch.empty(shape, dtype=dtype, device=device)


def _is_gpu(t):
    return t.is_cuda


def _need(t, dtype, shape, name, device=None):
    """Every tensor crossing the boundary: contiguous, on the GPU (on the
    same device as the call's other tensors), of the dtype and shape the
    C-ABI expects for these sizes; else ValueError before any launch."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
    if (t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous() or not _is_gpu(t)
            or (device is not None and t.device != device)):
        want = f"contiguous CUDA {dtype} {tuple(shape)}" + (f" on {device}" if device is not None else "")
        raise ValueError(f"{name}: expected {want}, got {t.dtype} {tuple(t.shape)} on {t.device}"
                         f"{'' if t.is_contiguous() else ' (not contiguous)'}")


def _need_workspace(t, nbytes, name, device):
    if not isinstance(t, torch.Tensor) or t.dtype != torch.uint8 or t.dim() != 1 \
            or not t.is_contiguous() or not _is_gpu(t) or t.device != device:
        raise ValueError(f"{name}: expected a contiguous 1-D CUDA uint8 tensor on {device}")
    if t.numel() < nbytes:
        raise ValueError(f"{name}: {t.numel()} bytes, at least {nbytes} needed")


def _dims(x, name, block):
    if not isinstance(x, torch.Tensor) or x.dim() != 2:
        raise ValueError(f"{name}: expected a 2-D tensor")
    rows, K = x.shape
    if K % block:
        raise ValueError(f"{name}: K = {K} is not a multiple of {block}")
    return rows, K


def nvfp4_quantize_workspace_bytes(rows: int, K: int) -> int:
    return lib.nvfp4_quantize_workspace_bytes(rows, K)


def nvfp4_gemm_workspace_bytes(M: int, N: int, K: int) -> int:
    return lib.nvfp4_gemm_workspace_bytes(M, N, K)


def nvfp4_linear_workspace_bytes(M: int, N: int, K: int) -> int:
    return lib.nvfp4_linear_workspace_bytes(M, N, K)


def gemm_plan(M: int, N: int, K: int, fmt: int = FORMAT_NVFP4, with_workspace: bool = True) -> dict:
    """The library's own account of how a GEMM of this shape runs (host
    only): kernel name, output tile edge, workgroups, K ranges per tile of
    the last round."""
    kernel, tile, splits = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    wgs = ctypes.c_int64()
    _check(lib.solfp4_gemm_plan(fmt, M, N, K, int(with_workspace), ctypes.byref(kernel),
                                ctypes.byref(tile), ctypes.byref(wgs), ctypes.byref(splits)))
    return {"kernel": KERNEL_NAMES.get(kernel.value, f"kernel {kernel.value}"), "tile": tile.value,
            "workgroups": wgs.value, "splits": splits.value}


def nvfp4_quantize(x, codes=None, scales=None, global_scale=None, workspace=None, stream=None):
    """x: BF16 [rows, K] -> (codes uint8 [rows, K/2], scales uint8 [rows, K/16],
    global_scale float32 [1]).  Outputs may be passed in to avoid allocation."""
    rows, K = _dims(x, "x", 16)
    dev = x.device
    _need(x, torch.bfloat16, (rows, K), "x")
    need = nvfp4_quantize_workspace_bytes(rows, K)
    if codes is not None:
        _need(codes, torch.uint8, (rows, K // 2), "codes", dev)
    if scales is not None:
        _need(scales, torch.uint8, (rows, K // 16), "scales", dev)
    if global_scale is not None:
        _need(global_scale, torch.float32, (1,), "global_scale", dev)
    if workspace is not None:
        _need_workspace(workspace, need, "workspace", dev)
    st = _stream(stream, dev)
    if codes is None:
        codes = _alloc((rows, K // 2), torch.uint8, dev, st)
    if scales is None:
        scales = _alloc((rows, K // 16), torch.uint8, dev, st)
    if global_scale is None:
        global_scale = _alloc((1,), torch.float32, dev, st)
    if workspace is None:
        workspace = _alloc((max(need, 256),), torch.uint8, dev, st)
    _check(lib.nvfp4_quantize(_ptr(x), rows, K, _ptr(codes), _ptr(scales), _ptr(global_scale),
                              _ptr(workspace), workspace.numel(), ctypes.c_void_p(st.cuda_stream)))
    return codes, scales, global_scale


def nvfp4_quantize_amax(x, workspace, stream=None):
    """The first pass of nvfp4_quantize: x's partial maxima into `workspace`
    (uint8, at least nvfp4_quantize_workspace_bytes(rows, K))."""
    rows, K = _dims(x, "x", 16)
    dev = x.device
    _need(x, torch.bfloat16, (rows, K), "x")
    _need_workspace(workspace, nvfp4_quantize_workspace_bytes(rows, K), "workspace", dev)
    st = _stream(stream, dev)
    _check(lib.nvfp4_quantize_amax(_ptr(x), rows, K, _ptr(workspace), workspace.numel(),
                                   ctypes.c_void_p(st.cuda_stream)))


def nvfp4_quantize_encode(x, codes, scales, global_scale, workspace, stream=None):
    """The second pass of nvfp4_quantize (after nvfp4_quantize_amax on the
    same x and workspace): codes, scales and alpha."""
    rows, K = _dims(x, "x", 16)
    dev = x.device
    _need(x, torch.bfloat16, (rows, K), "x")
    _need(codes, torch.uint8, (rows, K // 2), "codes", dev)
    _need(scales, torch.uint8, (rows, K // 16), "scales", dev)
    _need(global_scale, torch.float32, (1,), "global_scale", dev)
    _need_workspace(workspace, nvfp4_quantize_workspace_bytes(rows, K), "workspace", dev)
    st = _stream(stream, dev)
    _check(lib.nvfp4_quantize_encode(_ptr(x), rows, K, _ptr(codes), _ptr(scales), _ptr(global_scale),
                                     _ptr(workspace), workspace.numel(), ctypes.c_void_p(st.cuda_stream)))
    return codes, scales, global_scale


def nvfp4_quantize_noalloc(x, codes, scales, global_scale, stream=None):
    """nvfp4_quantize into caller-provided outputs with no workspace: the
    library's fixed per-device scratch holds the partial maxima, so this
    call allocates nothing (usable where allocation is not allowed).  Calls
    that may overlap on one device race on that scratch."""
    rows, K = _dims(x, "x", 16)
    dev = x.device
    _need(x, torch.bfloat16, (rows, K), "x")
    _need(codes, torch.uint8, (rows, K // 2), "codes", dev)
    _need(scales, torch.uint8, (rows, K // 16), "scales", dev)
    _need(global_scale, torch.float32, (1,), "global_scale", dev)
    st = _stream(stream, dev)
    _check(lib.nvfp4_quantize_noalloc(_ptr(x), rows, K, _ptr(codes), _ptr(scales),
                                      _ptr(global_scale), ctypes.c_void_p(st.cuda_stream)))
    return codes, scales, global_scale


def nvfp4_gemm(a_codes, a_scales, a_global_scale, b_codes, b_scales, b_global_scale,
               bias=None, out=None, workspace=None, stream=None, split=True):
    """Block-scaled NVFP4 GEMM: A [M, K] (packed), B [N, K] (packed) -> BF16 [M, N].
    `workspace` (uint8, at least nvfp4_gemm_workspace_bytes(M, N, K)) is
    allocated when needed and not given; split=False passes none (no split
    of the last round's tiles)."""
    M, Kh = _dims(a_codes, "a_codes", 1)
    N = _dims(b_codes, "b_codes", 1)[0]
    K = 2 * Kh
    if K % 16:
        raise ValueError(f"K = {K} is not a multiple of 16")
    dev = a_codes.device
    _need(a_codes, torch.uint8, (M, K // 2), "a_codes")
    _need(a_scales, torch.uint8, (M, K // 16), "a_scales", dev)
    _need(a_global_scale, torch.float32, (1,), "a_global_scale", dev)
    _need(b_codes, torch.uint8, (N, K // 2), "b_codes (A and B must agree on K)", dev)
    _need(b_scales, torch.uint8, (N, K // 16), "b_scales", dev)
    _need(b_global_scale, torch.float32, (1,), "b_global_scale", dev)
    if bias is not None:
        _need(bias, torch.bfloat16, (N,), "bias", dev)
    if out is not None:
        _need(out, torch.bfloat16, (M, N), "out", dev)
    if split and workspace is not None:
        _need_workspace(workspace, nvfp4_gemm_workspace_bytes(M, N, K), "workspace", dev)
    st = _stream(stream, dev)
    if out is None:
        out = _alloc((M, N), torch.bfloat16, dev, st)
    if not split:
        workspace = None
    elif workspace is None:
        need = nvfp4_gemm_workspace_bytes(M, N, K)
        if need:
            workspace = _alloc((need,), torch.uint8, dev, st)
    _check(lib.nvfp4_gemm(_ptr(a_codes), _ptr(a_scales), _ptr(a_global_scale), _ptr(b_codes),
                          _ptr(b_scales), _ptr(b_global_scale), _ptr(bias), _ptr(out),
                          _ptr(workspace), 0 if workspace is None else workspace.numel(),
                          M, N, K, ctypes.c_void_p(st.cuda_stream)))
    return out


def nvfp4_linear(x, w_codes, w_scales, w_global_scale, bias=None, out=None, workspace=None,
                 stream=None):
    """NVFP4 linear: quantize BF16 x [M, K] on the fly, GEMM with the packed
    weight [N, K], add bias -> BF16 [M, N]."""
    M, K = _dims(x, "x", 16)
    dev = x.device
    _need(x, torch.bfloat16, (M, K), "x")
    N = _dims(w_codes, "w_codes", 1)[0]
    _need(w_codes, torch.uint8, (N, K // 2), "w_codes (x and w must agree on K)", dev)
    _need(w_scales, torch.uint8, (N, K // 16), "w_scales", dev)
    _need(w_global_scale, torch.float32, (1,), "w_global_scale", dev)
    if bias is not None:
        _need(bias, torch.bfloat16, (N,), "bias", dev)
    if out is not None:
        _need(out, torch.bfloat16, (M, N), "out", dev)
    need = nvfp4_linear_workspace_bytes(M, N, K)
    if workspace is not None:
        _need_workspace(workspace, need, "workspace", dev)
    st = _stream(stream, dev)
    if out is None:
        out = _alloc((M, N), torch.bfloat16, dev, st)
    if workspace is None:
        workspace = _alloc((need,), torch.uint8, dev, st)
    _check(lib.nvfp4_linear(_ptr(x), _ptr(w_codes), _ptr(w_scales), _ptr(w_global_scale),
                            _ptr(bias), _ptr(out), _ptr(workspace), workspace.numel(),
                            M, N, K, ctypes.c_void_p(st.cuda_stream)))
    return out


def mxfp4_linear_workspace_bytes(M: int, K: int) -> int:
    return lib.mxfp4_linear_workspace_bytes(M, K)


def mxfp4_quantize(x, codes=None, scales=None, stream=None):
    """x: BF16 [rows, K] (K % 32 == 0) -> (codes uint8 [rows, K/2],
    scales uint8 [rows, K/32], E8M0)."""
    rows, K = _dims(x, "x", 32)
    dev = x.device
    _need(x, torch.bfloat16, (rows, K), "x")
    if codes is not None:
        _need(codes, torch.uint8, (rows, K // 2), "codes", dev)
    if scales is not None:
        _need(scales, torch.uint8, (rows, K // 32), "scales", dev)
    st = _stream(stream, dev)
    if codes is None:
        codes = _alloc((rows, K // 2), torch.uint8, dev, st)
    if scales is None:
        scales = _alloc((rows, K // 32), torch.uint8, dev, st)
    _check(lib.mxfp4_quantize(_ptr(x), rows, K, _ptr(codes), _ptr(scales),
                              ctypes.c_void_p(st.cuda_stream)))
    return codes, scales


def mxfp4_gemm(a_codes, a_scales, b_codes, b_scales, bias=None, out=None, stream=None):
    """MXFP4 GEMM: A [M, K] (packed), B [N, K] (packed) -> BF16 [M, N]."""
    M, Kh = _dims(a_codes, "a_codes", 1)
    N = _dims(b_codes, "b_codes", 1)[0]
    K = 2 * Kh
    if K % 32:
        raise ValueError(f"K = {K} is not a multiple of 32")
    dev = a_codes.device
    _need(a_codes, torch.uint8, (M, K // 2), "a_codes")
    _need(a_scales, torch.uint8, (M, K // 32), "a_scales", dev)
    _need(b_codes, torch.uint8, (N, K // 2), "b_codes (A and B must agree on K)", dev)
    _need(b_scales, torch.uint8, (N, K // 32), "b_scales", dev)
    if bias is not None:
        _need(bias, torch.bfloat16, (N,), "bias", dev)
    if out is not None:
        _need(out, torch.bfloat16, (M, N), "out", dev)
    st = _stream(stream, dev)
    if out is None:
        out = _alloc((M, N), torch.bfloat16, dev, st)
    _check(lib.mxfp4_gemm(_ptr(a_codes), _ptr(a_scales), _ptr(b_codes), _ptr(b_scales),
                          _ptr(bias), _ptr(out), M, N, K, ctypes.c_void_p(st.cuda_stream)))
    return out


def mxfp4_linear(x, w_codes, w_scales, bias=None, out=None, workspace=None, stream=None):
    """MXFP4 linear: quantize BF16 x [M, K] on the fly, GEMM with the packed
    weight [N, K], add bias -> BF16 [M, N]."""
    M, K = _dims(x, "x", 32)
    dev = x.device
    _need(x, torch.bfloat16, (M, K), "x")
    N = _dims(w_codes, "w_codes", 1)[0]
    _need(w_codes, torch.uint8, (N, K // 2), "w_codes (x and w must agree on K)", dev)
    _need(w_scales, torch.uint8, (N, K // 32), "w_scales", dev)
    if bias is not None:
        _need(bias, torch.bfloat16, (N,), "bias", dev)
    if out is not None:
        _need(out, torch.bfloat16, (M, N), "out", dev)
    need = mxfp4_linear_workspace_bytes(M, K)
    if workspace is not None:
        _need_workspace(workspace, need, "workspace", dev)
    st = _stream(stream, dev)
    if out is None:
        out = _alloc((M, N), torch.bfloat16, dev, st)
    if workspace is None:
        workspace = _alloc((need,), torch.uint8, dev, st)
    _check(lib.mxfp4_linear(_ptr(x), _ptr(w_codes), _ptr(w_scales), _ptr(bias), _ptr(out),
                            _ptr(workspace), workspace.numel(), M, N, K,
                            ctypes.c_void_p(st.cuda_stream)))
    return out
