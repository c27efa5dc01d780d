"""Pairwise summation over the channels (plan option channel_sum="pairwise",
the method the related work of Section 4 names after Barabasz et al. 2018)
on the GPU.

  * The contraction stage: M within the pairwise rounding bound
    (leaf + ceil(log2 leaves) + 2) u32 sum |V||U| of the exact channel sum,
    on random data of every dtype, short and long channel rows.
  * Its error against the exact sum, measured next to the matrix-core chains
    on a long fp32 reduction (C = 4096): pairwise is the more accurate.
  * conv2d with the option: U and V bit-equal to the oracle's, y within the
    pair bound of the oracle's pairwise evaluation, the 2x rule; the rel-L2
    against fp64 direct convolution is printed for both channel sums.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import check_layer, to_dev, to_np
from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP
from paper_1905_05233_amd import workloads as WL

pytestmark = pytest.mark.gpu
U32 = 2.0 ** -24


def _depth_terms(C, dtype):
    leaf = OC.leaf_channels(dtype)
    n = -(-C // leaf)
    return leaf + (n - 1).bit_length() + 2


def _contract(channel_sum, dtype, V, U, C):
    from paper_1905_05233_amd.winograd import Plan
    p = Plan(WL.F4_A2P1, m=4, dtype=dtype, channel_sum=channel_sum, path="separate")
    return to_np(p.contract(to_dev(V, dtype), to_dev(U, dtype), C))


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("T,C,K", [(1, 1, 1), (97, 5, 40), (130, 300, 70), (33, 2048, 17), (64, 520, 136)])
def test_pairwise_contraction_bound(dtype, T, C, K):
    a2 = 49
    Cp = -(-C // 8) * 8
    rng = np.random.Generator(np.random.PCG64(T + C + K))
    V = np.zeros((a2, T, Cp), np.float32)
    U = np.zeros((a2, K, Cp), np.float32)
    V[:, :, :C] = OF.to_dtype(rng.standard_normal((a2, T, C)).astype(np.float32), dtype)
    U[:, :, :C] = OF.to_dtype(rng.standard_normal((a2, K, C)).astype(np.float32), dtype)
    M = _contract("pairwise", dtype, V, U, C)[:, :, :K].astype(np.float64)
    ex = np.einsum("xtc,xkc->xtk", V.astype(np.float64), U.astype(np.float64))
    mag = np.einsum("xtc,xkc->xtk", np.abs(V).astype(np.float64), np.abs(U).astype(np.float64))
    assert np.all(np.abs(M - ex) <= 1.1 * _depth_terms(C, dtype) * U32 * mag)


def test_pairwise_more_accurate_on_long_fp32_sums():
    """C = 4096 half-normal products in fp32: the rel-L2 error of M against
    the exact sum, pairwise against the matrix-core chains."""
    a2, T, C, K = 49, 64, 4096, 64
    rng = np.random.Generator(np.random.PCG64(5))
    V = np.abs(rng.standard_normal((a2, T, C))).astype(np.float32)
    U = np.abs(rng.standard_normal((a2, K, C))).astype(np.float32)
    ex = np.einsum("xtc,xkc->xtk", V.astype(np.float64), U.astype(np.float64))
    e_pw = OC.rel_l2(_contract("pairwise", "f32", V, U, C)[:, :, :K], ex)
    e_mf = OC.rel_l2(_contract("mfma", "f32", V, U, C)[:, :, :K], ex)
    print(f"[pairwise] fp32 C={C}: rel-L2 of M, pairwise {e_pw:.3e}, MFMA chains {e_mf:.3e}", flush=True)
    assert e_pw < e_mf


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("spec,m", [(WL.F4_LINEAR, 4), (WL.F6_TWO_QUAD, 6)])
def test_pairwise_conv_parity(spec, m, dtype):
    from paper_1905_05233_amd.winograd import Plan
    N, H, W, C, K = 1, 18, 14, 1024, 48
    x, w = WL.draw_inputs(N, H, W, C, K, "halfnormal", seed=m + C)
    x, w = OF.to_dtype(x, dtype), OF.to_dtype(w, dtype)
    op = OP.build_plan(spec, n_o=m)
    p = Plan(spec, m=m, dtype=dtype, channel_sum="pairwise")
    assert p.conv_path(N, H, W, C, K) == "separate"
    y = to_np(p.conv2d(to_dev(x, dtype), to_dev(w, dtype))).astype(np.float64)
    st = OC.winograd_emulated_stages(x, w, op, dtype, channel_sum="pairwise")
    check_layer(p, op, x, w, dtype, y, label=f"pairwise {spec} {dtype}", st=st, sum_terms=_depth_terms(C, dtype))
    y64 = OC.direct_f64(x, w)
    e_gpu, e_or = OC.rel_l2(y, y64), OC.rel_l2(st["y"], y64)
    y_mfma = to_np(Plan(spec, m=m, dtype=dtype).conv2d(to_dev(x, dtype), to_dev(w, dtype)))
    print(f"[pairwise] {spec} {dtype} C={C}: rel-L2 pairwise {e_gpu:.3e} (oracle {e_or:.3e}), "
          f"MFMA chains {OC.rel_l2(y_mfma, y64):.3e}", flush=True)
    assert e_gpu <= 2 * e_or


def test_pairwise_rejects_fused_paths():
    from paper_1905_05233_amd._native import WinogradError
    from paper_1905_05233_amd.winograd import Plan
    with pytest.raises(WinogradError, match="ARG"):
        Plan(WL.F4_A2P1, m=4, dtype="bf16", channel_sum="pairwise", path="fused")
