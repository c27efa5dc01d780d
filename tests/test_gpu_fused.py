"""Parity of the fused path: the channel contraction and the output transform
of eq. (2) in one kernel, with M kept in registers.

Checks, on seeded inputs:
  * the 2x rule, and element by element U and V bit-equal to the oracle's
    and y within ``pair_bound`` of the oracle's y, for every compiled (input
    tile, alpha') shape of the fused kernel, in fp32, fp16 and bf16, on
    shapes with ragged tiles, channel counts that are not multiples of 16 and
    rows longer than one 128-byte slice;
  * the fused and the separate path agree element by element within
    ``pair_bound`` taken between the two (they read the same U and V and
    differ only in the order of the fp32 channel sums), for every compiled
    shape and for the VGG-16 layers the automatic rule sends to the fused
    kernel;
  * the stage entry point gives the same bits as conv2d on the fused path;
  * dyadic plans on small integers are bit-exact (every rounding is exact).
"""
import numpy as np
import pytest
import torch

from gpu_helpers import check_layer, elementwise_bound, pair_bound, to_dev, to_np
from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP
from paper_1905_05233_amd import workloads as WL

pytestmark = pytest.mark.gpu

# one plan per compiled (input tile, alpha') shape of the fused kernel
FUSED_PLANS = [
    (WL.F2_LINEAR, 2),                       # t 4, alpha' 4
    ("0,a^2+1,inf", 2),                      # t 4, alpha' 5
    ("a^2+1,a^2-2", 2),                      # t 4, alpha' 6 (no infinity)
    (WL.F4_LINEAR, 4),                       # t 6, alpha' 6
    (WL.F4_A2P1, 4),                         # t 6, alpha' 7
    ("0,a^2+1,a^2-2,inf", 4),                # t 6, alpha' 8
    ("a^2+1,a^2-2,a^2+2", 4),                # t 6, alpha' 9
    (WL.F6_LINEAR, 6),                       # t 8, alpha' 8
    (WL.F6_ONE_A2P1, 6),                     # t 8, alpha' 9
    (WL.F6_TWO_QUAD, 6),                     # t 8, alpha' 10
    ("0,a^2+1,a^2-2,a^2+2,inf", 6),          # t 8, alpha' 11
    ("a^2+1,a^2-2,a^2+2,a^2+a+1", 6),        # t 8, alpha' 12
]


def _plan(spec, m, dtype, path):
    from paper_1905_05233_amd.winograd import Plan
    return Plan(spec, m=m, dtype=dtype, path=path)


def _inputs(shape, dtype, seed):
    N, H, W, C, K = shape
    x, w = WL.draw_inputs(N, H, W, C, K, "halfnormal", seed=seed)
    return OF.to_dtype(x, dtype), OF.to_dtype(w, dtype)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("spec,m", FUSED_PLANS, ids=[f"{s}-m{m}" for s, m in FUSED_PLANS])
@pytest.mark.parametrize("shape", [(2, 26, 30, 24, 40), (1, 19, 17, 200, 70)], ids=["ragged", "long-rows"])
def test_fused_parity(spec, m, dtype, shape):
    print(f"[fused] {spec} m={m} {dtype} {shape}", flush=True)
    x, w = _inputs(shape, dtype, seed=7 * m + shape[3])
    p = _plan(spec, m, dtype, "fused")
    N, H, W, C, K = shape
    assert p.conv_path(N, H, W, C, K) == "fused"
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    y1 = p.conv2d(xd, wd)
    y2 = p.conv2d(xd, wd)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    y = to_np(y1).astype(np.float64)
    op = OP.build_plan(spec, n_o=m)
    y64 = OC.direct_f64(x, w)
    st = check_layer(p, op, x, w, dtype, y, label=f"fused {spec} {dtype} {shape}")
    err_gpu, err_or = OC.rel_l2(y, y64), OC.rel_l2(st["y"], y64)
    print(f"[fused] err_gpu={err_gpu:.3e} err_oracle={err_or:.3e}", flush=True)
    assert np.all(np.isfinite(y))
    assert err_gpu <= 2 * err_or
    if dtype == "f32":
        assert np.all(np.abs(y - y64) <= elementwise_bound(x, w, op, dtype, y64))


def _fused_vs_separate(spec, m, dtype, shape, seed, label):
    x, w = _inputs(shape, dtype, seed=seed)
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    pf, ps = _plan(spec, m, dtype, "fused"), _plan(spec, m, dtype, "separate")
    N, H, W, C, K = shape
    assert ps.conv_path(N, H, W, C, K) == "separate"
    assert pf.workspace_bytes(N, H, W, C, K) < ps.workspace_bytes(N, H, W, C, K)   # no M
    yf = to_np(pf.conv2d(xd, wd)).astype(np.float64)
    ys = to_np(ps.conv2d(xd, wd)).astype(np.float64)
    op = OP.build_plan(spec, n_o=m)
    st = check_layer(ps, op, x, w, dtype, ys, label=f"{label} separate")
    check_layer(pf, op, x, w, dtype, yf, label=f"{label} fused", st=st)
    b = pair_bound(st, op, dtype, yf, H, W, y_ref=ys)
    diff = np.abs(yf - ys)
    print(f"[fused-vs-separate] {label}: max |diff| {np.max(diff):.3e}, max diff/bound {np.max(diff / b):.3g}, "
          f"median bound/|y| {np.median(b / np.maximum(np.abs(ys), 1e-30)):.3g}", flush=True)
    assert np.all(diff <= b)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("spec,m", FUSED_PLANS, ids=[f"{s}-m{m}" for s, m in FUSED_PLANS])
def test_fused_matches_separate(spec, m, dtype):
    """Every compiled fused shape, fused against separate, element by element."""
    _fused_vs_separate(spec, m, dtype, (3, 40, 36, 64, 96), 3 * m, f"{spec} {dtype}")


# VGG-16 layers that the automatic rule sends to the fused kernel (N = 1)
VGG_FUSED = [(224, 3, 64), (224, 64, 64), (112, 64, 128), (112, 128, 128), (56, 128, 256)]


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("hw,C,K", VGG_FUSED, ids=[f"{h}x{h}-{c}-{k}" for h, c, k in VGG_FUSED])
def test_fused_matches_separate_vgg_layers(hw, C, K, dtype):
    from paper_1905_05233_amd.winograd import Plan
    assert Plan(WL.F4_A2P1, m=4, dtype=dtype).conv_path(32, hw, hw, C, K) == "fused"
    _fused_vs_separate(WL.F4_A2P1, 4, dtype, (1, hw, hw, C, K), hw + C, f"VGG {hw}x{hw} {C}->{K} {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_stage_entry_point(dtype):
    """winograd_contract_output on the transforms' outputs is conv2d's fused path."""
    shape = (2, 23, 29, 40, 52)
    x, w = _inputs(shape, dtype, seed=11)
    p = _plan(WL.F4_A2P1, 4, dtype, "fused")
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    N, H, W, C, K = shape
    U = p.kernel_transform(wd)
    V = p.input_transform(xd)
    y_stage = p.contract_output(V, U, C, N, H, W)
    y_conv = p.conv2d(xd, wd)
    torch.cuda.synchronize()
    assert torch.equal(y_stage, y_conv)


@pytest.mark.parametrize("spec,m", [(WL.F2_LINEAR, 2), (WL.F4_A2P1, 4), ("0,a^2+1,inf", 2)])
@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", [(1, 16, 16, 8, 8), (2, 7, 11, 3, 5), (1, 1, 1, 1, 1), (3, 13, 6, 28, 130),
                                   (1, 9, 9, 160, 3)])
def test_fused_bit_exact_dyadic(spec, m, dtype, shape):
    N, H, W, C, K = shape
    print(f"[fused-exact] {spec} m={m} {dtype} {shape}", flush=True)
    dist = "ternary" if dtype == "bf16" else "int2"
    x, w = WL.draw_inputs(N, H, W, C, K, dist, seed=N + H + W + C + K)
    p = _plan(spec, m, dtype, "fused")
    y = to_np(p.conv2d(to_dev(x, dtype), to_dev(w, dtype))).astype(np.float64)
    ref = OC.direct_f64(x, w)
    op = OP.build_plan(spec, n_o=m)
    assert np.array_equal(OC.winograd_emulated(x, w, op, dtype).astype(np.float64), ref)
    assert np.array_equal(y, ref)


def test_fused_unsupported_shape_raises():
    """Input tiles over 8 have no fused kernel: a plan that asks for the fused
    path reports WG_ERR_UNSUPPORTED instead of falling back."""
    from paper_1905_05233_amd._native import WinogradError
    p = _plan("0,-1,1,-1/2,2,1/2,-2,a^2+1,inf", 8, "f32", "fused")
    x, w = _inputs((1, 16, 16, 8, 8), "f32", seed=1)
    with pytest.raises(WinogradError, match="UNSUPPORTED"):
        p.conv2d(to_dev(x, "f32"), to_dev(w, "f32"))


# layers whose fused kernel also computes V (rows of at most 32 bytes, K > 32)
FUSE_INPUT = [
    (WL.F2_LINEAR, 2, "f32", (2, 26, 30, 3, 40)),        # 32-byte rows: 4 domain points per step
    (WL.F4_LINEAR, 4, "f32", (1, 19, 17, 8, 70)),
    (WL.F4_A2P1, 4, "bf16", (2, 26, 30, 3, 40)),         # 16-byte rows: 8 per step
    (WL.F4_A2P1, 4, "f16", (1, 19, 17, 8, 70)),
    (WL.F6_LINEAR, 6, "bf16", (2, 23, 29, 5, 96)),
    (WL.F4_LINEAR, 4, "bf16", (1, 21, 22, 16, 48)),      # 32-byte rows in 16-bit storage
]


@pytest.mark.parametrize("spec,m,dtype,shape", FUSE_INPUT,
                         ids=[f"{s}-m{m}-{d}-{sh}" for s, m, d, sh in FUSE_INPUT])
def test_fused_input_transform(spec, m, dtype, shape):
    """The input transform in the fused kernel's prologue gives the same bits as
    the input-transform kernel followed by the fused kernel, and conv2d on the
    fused_input path is that kernel; against the oracle, the 2x rule and the
    pair bound."""
    N, H, W, C, K = shape
    print(f"[fused-input] {spec} m={m} {dtype} {shape}", flush=True)
    x, w = _inputs(shape, dtype, seed=m + C + K)
    p = _plan(spec, m, dtype, "fused_input")
    assert p.conv_path(N, H, W, C, K) == "fused_input"
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    U = p.kernel_transform(wd)
    y_two = p.contract_output(p.input_transform(xd), U, C, N, H, W)
    y_one = p.input_contract_output(xd, U)
    y_conv = p.conv2d(xd, wd)
    torch.cuda.synchronize()
    assert torch.equal(y_one, y_two)
    assert torch.equal(y_conv, y_two)
    y = to_np(y_conv).astype(np.float64)
    op = OP.build_plan(spec, n_o=m)
    y64 = OC.direct_f64(x, w)
    st = check_layer(p, op, x, w, dtype, y, label=f"fused-input {spec} {dtype} {shape}")
    assert OC.rel_l2(y, y64) <= 2 * OC.rel_l2(st["y"], y64)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_fused_input_transform_bit_exact_dyadic(dtype):
    """Small integers through a dyadic plan: every rounding exact, so the
    fused-input kernel equals direct convolution bit for bit."""
    N, H, W, C, K = 2, 30, 27, 3, 64
    dist = "ternary" if dtype == "bf16" else "int2"
    x, w = WL.draw_inputs(N, H, W, C, K, dist, seed=17)
    spec, m = (WL.F2_LINEAR, 2) if dtype == "f32" else (WL.F4_A2P1, 4)
    p = _plan(spec, m, dtype, "fused_input")
    assert p.conv_path(N, H, W, C, K) == "fused_input"
    y = to_np(p.conv2d(to_dev(x, dtype), to_dev(w, dtype))).astype(np.float64)
    assert np.array_equal(y, OC.direct_f64(x, w))


def test_fused_input_transform_unsupported_raises():
    from paper_1905_05233_amd._native import WinogradError
    p = _plan(WL.F4_A2P1, 4, "bf16", "fused")
    x, w = _inputs((1, 16, 16, 24, 64), "bf16", seed=2)       # 48-byte rows
    U = p.kernel_transform(to_dev(w, "bf16"))
    with pytest.raises(WinogradError, match="UNSUPPORTED"):
        p.input_contract_output(to_dev(x, "bf16"), U)
