"""The library's operations around the layer, on the GPU, against plain
numpy: ReLU and 2x2 max-pooling (exact: both only select values), the
float64 direct convolution (the reference of the error studies; against the
oracle's float64 convolution, equal up to float64 summation order), and the
float64 error sums."""
import numpy as np
import pytest
import torch

from gpu_helpers import TORCH, to_dev, to_np
from oracle import conv as OC
from oracle import fp as OF
from paper_1905_05233_amd import workloads as WL

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("pool", [False, True])
@pytest.mark.parametrize("shape", [(2, 8, 6, 64), (3, 7, 9, 5), (1, 224, 224, 64), (1, 1, 1, 8)])
def test_relu_pool_exact(dtype, pool, shape):
    from paper_1905_05233_amd.layer_ops import relu_pool
    rng = np.random.default_rng(sum(shape))
    x = OF.to_dtype(rng.standard_normal(shape).astype(np.float32), dtype)
    y = to_np(relu_pool(to_dev(x, dtype), pool))
    r = np.maximum(x, 0)
    if pool:
        N, H, W, C = shape
        Ho, Wo = H // 2, W // 2
        r = r[:, :2 * Ho, :2 * Wo, :].reshape(N, Ho, 2, Wo, 2, C).max(axis=(2, 4))
    assert y.shape == r.shape
    assert np.array_equal(y, r)


def test_relu_pool_rejects_overlap_and_bad_shapes():
    from paper_1905_05233_amd._native import WinogradError
    from paper_1905_05233_amd.layer_ops import relu_pool
    x = torch.zeros((1, 4, 4, 8), device="cuda")
    with pytest.raises(WinogradError, match="ARG"):
        relu_pool(x, False, out=x)
    with pytest.raises(WinogradError, match="ARG"):
        relu_pool(x, True, out=torch.zeros((1, 4, 4, 8), device="cuda"))


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", [(2, 9, 11, 5, 7), (1, 32, 32, 64, 64)])
def test_direct_conv_f64(dtype, shape):
    from paper_1905_05233_amd.layer_ops import direct_conv_f64
    N, H, W, C, K = shape
    x, w = WL.draw_inputs(N, H, W, C, K, "halfnormal", seed=C + K)
    x, w = OF.to_dtype(x, dtype), OF.to_dtype(w, dtype)
    y = direct_conv_f64(to_dev(x, dtype), to_dev(w, dtype)).cpu().numpy()
    ref = OC.direct_f64(x, w)
    mag = OC.direct_f64(np.abs(x), np.abs(w))
    assert np.all(np.abs(y - ref) <= 1e-14 * (9 * C) * mag + 1e-300)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_direct_conv_f64_1d(dtype):
    from paper_1905_05233_amd.layer_ops import direct_conv_f64
    x4, w4 = WL.draw_inputs(3, 1, 37, 12, 10, "uniform", seed=4)
    x, w = OF.to_dtype(x4[:, 0], dtype), OF.to_dtype(w4[:, 1], dtype)
    y = direct_conv_f64(to_dev(x[:, None], dtype), to_dev(w[:, None], dtype)).cpu().numpy()[:, 0]
    ref = OC.direct1d_f64(x, w)
    mag = OC.direct1d_f64(np.abs(x), np.abs(w))
    assert np.all(np.abs(y - ref) <= 1e-14 * 36 * mag + 1e-300)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("n", [1, 1000, 3_000_001])
def test_error_sums(dtype, n):
    from paper_1905_05233_amd.layer_ops import error_sums, rel_l2
    rng = np.random.default_rng(n)
    ref = rng.standard_normal(n)
    y = OF.to_dtype((ref + 1e-3 * rng.standard_normal(n)).astype(np.float32), dtype)
    yd = torch.from_numpy(y).to(TORCH[dtype]).cuda()
    rd = torch.from_numpy(ref).cuda()
    e2, r2 = error_sums(yd, rd)
    d = y.astype(np.float64) - ref
    assert e2 == pytest.approx(float(np.sum(d * d)), rel=1e-12)
    assert r2 == pytest.approx(float(np.sum(ref * ref)), rel=1e-12)
    assert rel_l2(yd, rd) == pytest.approx(OC.rel_l2(y, ref), rel=1e-10)
    assert error_sums(yd, rd) == (e2, r2)          # fixed order: the same bits again
