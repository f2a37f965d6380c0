"""The Python binding's argument checks, without a GPU: every operand of
every call is checked for dtype, shape, contiguity and device before the
library is called, so a wrong tensor (an MXFP4 scale tensor passed to the
NVFP4 GEMM, a host scalar as the tensor scale, a transposed view) raises
ValueError instead of handing the kernels a buffer smaller than the sizes
they derive from M, N and K.  Tensors live on torch's "meta" device, which
has shapes and dtypes but no storage; the binding's GPU test is patched to
accept it, and the call is stopped where it would pick its stream."""
import pytest

torch = pytest.importorskip("torch")

from paper_2604_06916_amd import _binding as B  # noqa: E402


class Reached(Exception):
    """Validation passed: the binding went on to pick its stream."""


@pytest.fixture(autouse=True)
def meta_device(monkeypatch):
    monkeypatch.setattr(B, "_is_gpu", lambda t: t.device.type == "meta")

    def stop(stream, device):
        raise Reached()
    monkeypatch.setattr(B, "_stream", stop)


def T(shape, dtype=torch.uint8):
    return torch.empty(shape, dtype=dtype, device="meta")


M, N, K = 48, 80, 256


def gemm_args():
    return dict(a_codes=T((M, K // 2)), a_scales=T((M, K // 16)), a_global_scale=T((1,), torch.float32),
                b_codes=T((N, K // 2)), b_scales=T((N, K // 16)), b_global_scale=T((1,), torch.float32),
                bias=T((N,), torch.bfloat16), out=T((M, N), torch.bfloat16))


def call_gemm(**kw):
    a = gemm_args()
    a.update(kw)
    B.nvfp4_gemm(a["a_codes"], a["a_scales"], a["a_global_scale"], a["b_codes"], a["b_scales"],
                 a["b_global_scale"], a["bias"], a["out"])


def test_valid_gemm_reaches_the_library():
    with pytest.raises(Reached):
        call_gemm()


@pytest.mark.parametrize("name,bad", [
    ("a_scales", T((M, K // 32))),                      # MXFP4-shaped scales
    ("b_scales", T((N, K // 32))),
    ("a_scales", T((M, K // 16), torch.int8)),
    ("a_global_scale", torch.empty(1, dtype=torch.float32)),   # host tensor
    ("b_global_scale", T((2,), torch.float32)),
    ("b_global_scale", T((1,), torch.float64)),
    ("b_codes", T((N, K // 2 + 8))),                    # K disagrees
    ("b_codes", T((K // 2, N)).t()),                    # transposed view
    ("bias", T((N + 1,), torch.bfloat16)),
    ("out", T((M, N), torch.float16)),
    ("out", T((N, M), torch.bfloat16)),
])
def test_gemm_rejects_each_wrong_operand(name, bad):
    with pytest.raises(ValueError):
        call_gemm(**{name: bad})


def test_quantize_checks_every_output():
    x = T((M, K), torch.bfloat16)
    with pytest.raises(Reached):
        B.nvfp4_quantize(x, T((M, K // 2)), T((M, K // 16)), T((1,), torch.float32), T((4096,)))
    for bad in [dict(codes=T((M, K // 4))), dict(scales=T((M, K // 32))),
                dict(global_scale=T((1,), torch.float16)), dict(workspace=T((2,))),
                dict(workspace=T((64, 64)))]:
        kw = dict(codes=T((M, K // 2)), scales=T((M, K // 16)), global_scale=T((1,), torch.float32),
                  workspace=T((4096,)))
        kw.update(bad)
        with pytest.raises(ValueError):
            B.nvfp4_quantize(x, **kw)
    with pytest.raises(ValueError):
        B.nvfp4_quantize(T((M, 40), torch.bfloat16))      # K % 16


def test_linear_checks_weight_and_workspace():
    x = T((M, K), torch.bfloat16)
    w = (T((N, K // 2)), T((N, K // 16)), T((1,), torch.float32))
    with pytest.raises(Reached):
        B.nvfp4_linear(x, *w, out=T((M, N), torch.bfloat16), workspace=T((1 << 20,)))
    with pytest.raises(ValueError):
        B.nvfp4_linear(x, w[0], T((N, K // 32)), w[2])
    with pytest.raises(ValueError):
        B.nvfp4_linear(x, T((N, K // 4)), w[1], w[2])
    with pytest.raises(ValueError):
        B.nvfp4_linear(x, *w, workspace=T((16,)))


def test_mxfp4_checks():
    x = T((M, K), torch.bfloat16)
    with pytest.raises(Reached):
        B.mxfp4_gemm(T((M, K // 2)), T((M, K // 32)), T((N, K // 2)), T((N, K // 32)),
                     out=T((M, N), torch.bfloat16))
    with pytest.raises(ValueError):      # NVFP4-shaped scales to the MXFP4 GEMM
        B.mxfp4_gemm(T((M, K // 2)), T((M, K // 16)), T((N, K // 2)), T((N, K // 32)))
    with pytest.raises(ValueError):
        B.mxfp4_quantize(x, scales=T((M, K // 16)))
    with pytest.raises(ValueError):
        B.mxfp4_linear(x, T((N, K // 2)), T((N, K // 16)))


def test_gemm_plan_names_the_kernels():
    # FLUX QKV: 2560 whole 256 x 256 tiles, then the last 32 as 128 quadrants
    # of 128 x 128, each in two K halves (without a workspace, whole)
    p = B.gemm_plan(18432, 9216, 3072)
    assert p == {"kernel": "nvfp4_gemm_lane_kernel", "tile": 256, "workgroups": 2560 + 2 * 128,
                 "splits": 2}
    assert B.gemm_plan(18432, 9216, 3072, with_workspace=False) == {
        "kernel": "nvfp4_gemm_lane_kernel", "tile": 256, "workgroups": 2560 + 128, "splits": 1}
    # FLUX out: 864 tiles, the last 96 each in two K halves
    assert B.gemm_plan(18432, 3072, 3072)["workgroups"] == 768 + 2 * 96
    assert B.gemm_plan(128, 1152, 1152) == {"kernel": "nvfp4_gemm_wavek_kernel", "tile": 32,
                                            "workgroups": 144, "splits": 1}
    assert B.gemm_plan(256, 3072, 1152) == {"kernel": "nvfp4_gemm_small_kernel", "tile": 64,
                                            "workgroups": 192, "splits": 1}
    assert B.gemm_plan(300, 1000, 512)["kernel"] == "nvfp4_gemm_small_kernel"
    assert B.gemm_plan(128, 12288, 3072)["kernel"] == "nvfp4_gemm_lane_kernel"
    assert B.gemm_plan(128, 1152, 1120)["tile"] == 128      # K % 128 != 0
    assert B.gemm_plan(4096, 4096, 320)["kernel"] == "nvfp4_gemm_kernel"
    # MXFP4 FLUX QKV: 2560 whole tiles, then the last 32 as 128 quadrants
    assert B.gemm_plan(18432, 9216, 3072, B.FORMAT_MXFP4) == {"kernel": "mxfp4_gemm_kernel",
                                                              "tile": 256, "workgroups": 2560 + 128,
                                                              "splits": 1}
    assert B.gemm_plan(18432, 3072, 3072, B.FORMAT_MXFP4)["workgroups"] == 864
    # MXFP4 tiles by token count (on a host without a device the library
    # plans for 256 CUs): the wave-K kernel's 32 x 32 tiles while they fit
    # one per CU and K spans more than one stage, 64 x 64 while those take
    # at most two rounds and 128 x 128 tiles one, 128 x 128 beyond
    mx = lambda M, N, K: B.gemm_plan(M, N, K, B.FORMAT_MXFP4)
    assert mx(128, 1152, 1152) == {"kernel": "mxfp4_gemm_wavek_kernel", "tile": 32,
                                   "workgroups": 144, "splits": 1}
    assert mx(7, 33, 128)["tile"] == 64                      # one stage
    assert mx(128, 1152, 1120)["tile"] == 64                 # K % 128 != 0
    assert mx(128, 3072, 3072)["tile"] == 64                 # 384 tiles of 32 x 32
    assert mx(384, 3072, 3072)["tile"] == 64 and mx(512, 2240, 2240)["workgroups"] == 280
    assert mx(1024, 3072, 3072)["tile"] == 128 and mx(1000, 3000, 256)["tile"] == 128
    assert mx(2100, 9000, 3072)["tile"] == 256
    assert B.gemm_plan(0, 16, 16)["kernel"] is None
    with pytest.raises(B.Solfp4Error):
        B.gemm_plan(16, 16, 24)
