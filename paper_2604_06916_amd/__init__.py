"""solfp4: NVFP4 linear layer (quantize, block-scaled GEMM, linear) for
AMD MI355X, plus its MXFP4 variant on the native scaled FP4 matrix
instructions, as a C-ABI HIP library with a thin Python binding.

The binding (and so libsolfp4.so) loads on first use of any name below and
raises ImportError if the library has not been built.
"""
_NAMES = ("EXPORTED", "LIB_PATH", "Solfp4Error", "lib", "gemm_plan", "FORMAT_NVFP4",
          "FORMAT_MXFP4", "nvfp4_gemm",
          "nvfp4_gemm_workspace_bytes", "nvfp4_linear", "nvfp4_linear_workspace_bytes",
          "nvfp4_quantize", "nvfp4_quantize_amax", "nvfp4_quantize_encode", "nvfp4_quantize_noalloc", "nvfp4_quantize_workspace_bytes", "mxfp4_gemm", "mxfp4_linear", "mxfp4_linear_workspace_bytes", "mxfp4_quantize")
__all__ = list(_NAMES)


def __getattr__(name):
    if name in _NAMES:
        from . import _binding
        return getattr(_binding, name)
    raise AttributeError(name)
