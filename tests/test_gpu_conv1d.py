"""1D F(m, 3) on the GPU (winograd_conv1d) against the oracle's 1D path.

  * The 1D kernels run the oracle's operations (one fp32 pass of ascending
    fused multiply-adds per transform, dtype roundings of U, V and y), so y
    lies within ``pair_bound_1d`` of the oracle's y (the paths differ only in
    the order of the fp32 channel sums; a U or V that differed would break
    the bound, not hide in it), and the rel-L2 error against float64 direct
    convolution is at most twice the oracle's.
  * Dyadic plans on small integers are bit-exact against direct convolution.
  * Every compiled (input tile, alpha') shape, all three dtypes, ragged
    lengths, one-element layers and channel counts over 64.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import ALL_SHAPES, TORCH, pair_bound_1d
from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP
from paper_1905_05233_amd import workloads as WL

pytestmark = pytest.mark.gpu


def _inputs(N, L, C, K, dtype, dist, seed):
    x4, w4 = WL.draw_inputs(N, 1, L, C, K, dist, seed=seed)
    return OF.to_dtype(x4[:, 0], dtype), OF.to_dtype(w4[:, 1], dtype)


def _dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(TORCH[dtype]).cuda()


@pytest.mark.parametrize("spec,m", ALL_SHAPES, ids=[f"t{m + 2}-{s}" for s, m in ALL_SHAPES])
@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", [(3, 53, 24, 40), (1, 1, 1, 1), (2, 17, 72, 136)], ids=["ragged", "one", "wide"])
def test_conv1d_parity(spec, m, dtype, shape):
    from paper_1905_05233_amd.winograd import Plan
    N, L, C, K = shape
    print(f"[conv1d] {spec} m={m} {dtype} {shape}", flush=True)
    x, w = _inputs(N, L, C, K, dtype, "uniform", seed=m + L)
    p = Plan(spec, m=m, dtype=dtype)
    y = p.conv1d(_dev(x, dtype), _dev(w, dtype)).float().cpu().numpy().astype(np.float64)
    op = OP.build_plan(spec, n_o=m)
    st = OC.winograd1d_emulated_stages(x, w, op, dtype)
    b = pair_bound_1d(st, op, dtype, y)
    err = np.abs(y - st["y"])
    assert np.all(err <= b), (int(np.sum(err > b)), float(np.max(err / b)))
    y64 = OC.direct1d_f64(x, w)
    e_gpu, e_or = OC.rel_l2(y, y64), OC.rel_l2(st["y"], y64)
    print(f"[conv1d] err gpu {e_gpu:.3e} oracle {e_or:.3e}; max err/pair bound {np.max(err / b):.3g}", flush=True)
    if np.all(np.isfinite(st["y"])):
        assert e_gpu <= 2 * e_or or e_gpu == 0.0


@pytest.mark.parametrize("spec,m", [(WL.F2_LINEAR, 2), (WL.F4_A2P1, 4), ("0,a^2+1,inf", 2)])
@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_conv1d_bit_exact_dyadic(spec, m, dtype):
    from paper_1905_05233_amd.winograd import Plan
    x, w = _inputs(3, 41, 20, 9, dtype, "ternary" if dtype == "bf16" else "int2", seed=m)
    y = Plan(spec, m=m, dtype=dtype).conv1d(_dev(x, dtype), _dev(w, dtype)).float().cpu().numpy()
    assert np.array_equal(y.astype(np.float64), OC.direct1d_f64(x, w))


def test_conv1d_rejects_bad_shapes():
    from paper_1905_05233_amd._native import WinogradError
    from paper_1905_05233_amd.winograd import Plan
    p = Plan(WL.F4_LINEAR, m=4, dtype="f32")
    x = torch.zeros((2, 10, 4), device="cuda")
    with pytest.raises(ValueError):
        p.conv1d(x, torch.zeros((3, 3, 5), device="cuda"))
    p.bind_workspace(torch.empty(256, dtype=torch.uint8, device="cuda"))
    with pytest.raises(WinogradError, match="WORKSPACE"):
        p.conv1d(x, torch.zeros((3, 3, 4), device="cuda"), workspace=torch.empty(256, dtype=torch.uint8,
                                                                                  device="cuda"))
