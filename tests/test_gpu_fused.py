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
VGG_FUSED = [(224, 3, 64), (224, 64, 64), (112, 64, 128), (112, 128, 128), (56, 128, 256), (56, 256, 256),
             (28, 256, 512)]


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("hw,C,K", VGG_FUSED, ids=[f"{h}x{h}-{c}-{k}" for h, c, k in VGG_FUSED])
def test_fused_matches_separate_vgg_layers(hw, C, K, dtype):
    from paper_1905_05233_amd.winograd import Plan
    assert Plan(WL.F4_A2P1, m=4, dtype=dtype).conv_path(32, hw, hw, C, K) == "fused"
    _fused_vs_separate(WL.F4_A2P1, 4, dtype, (1, hw, hw, C, K), hw + C, f"VGG {hw}x{hw} {C}->{K} {dtype}")


# The unrolled fused kernel: channel rows of 65 .. 256 bytes (one or two
# 128-byte slices per step), m <= 4, more than 32 output channels and enough
# blocks of 64 channels x 32 tiles to give every CU two (the launcher's rule).
# One plan per compiled instance: built-in plans (constant coefficients) and
# plans with run-time coefficients.
UNROLLED_PLANS = [
    (WL.F2_LINEAR, 2, False),              # t 4, alpha' 4, built-in
    (WL.F2_LINEAR, 2, True),               # the same shape, run-time coefficients
    ("0,a^2+1,inf", 2, False),             # t 4, alpha' 5
    ("a^2+1,a^2-2", 2, False),             # t 4, alpha' 6
    (WL.F4_LINEAR, 4, False),              # t 6, alpha' 6, built-in
    (WL.F4_A2P1, 4, False),                # t 6, alpha' 7, built-in
    (WL.F4_A2P1, 4, True),                 # the same shape, run-time coefficients
    ("0,a^2+1,a^2-2,inf", 4, False),       # t 6, alpha' 8
    ("a^2+1,a^2-2,a^2+2", 4, False),       # t 6, alpha' 9
]


def _unrolled_shape(m, dtype, ragged_k, slices=1, C=None):
    """A layer the launcher sends to the unrolled kernel: rows that leave the
    last pieces of a 128-byte slice empty, or fill it; ragged tiles; with
    ``ragged_k`` an output-channel count whose rows end mid 16-byte chunk (the
    epilogue's direct stores) and a partial block of 64 channels."""
    if C is not None:
        pass
    elif slices == 1:
        C = {"f32": 20, "f16": 48, "bf16": 64}[dtype]
    else:
        C = {"f32": 48, "f16": 100, "bf16": 128}[dtype]
    K = 250 if ragged_k else 256
    hw = 254 if m == 4 else 129
    return 1, hw, hw, C, K


def _selects_unrolled(m, C, K, T, dtype):
    rb = -(-C // 8) * 8 * (4 if dtype == "f32" else 2)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    return m <= 4 and K > 32 and (-(-K // 64)) * (-(-T // 32)) >= 2 * cus


def _gpu_stages(p, V, U, M, C, K, N, H, W):
    """The library's own U, V and M in the oracle's stage layout."""
    al, m = p.alpha, p.m
    th, tw = -(-H // m), -(-W // m)
    return {"V": to_np(V)[:, :, :C].reshape(al, al, N, th, tw, C),
            "U": to_np(U)[:, :, :C].reshape(al, al, K, C),
            "M": to_np(M)[:, :, :K].reshape(al, al, N, th, tw, K)}


def _unrolled_vs_separate(spec, m, generic, dtype, slices, C=None):
    from paper_1905_05233_amd.winograd import Plan
    N, H, W, C, K = _unrolled_shape(m, dtype, ragged_k=generic, slices=slices, C=C)
    print(f"[unrolled] {spec} m={m} generic={generic} {dtype} {(N, H, W, C, K)}", flush=True)
    x, w = _inputs((N, H, W, C, K), dtype, seed=5 * m + C)
    p = Plan(spec, m=m, dtype=dtype, path="fused", generic_transforms=generic)
    assert (p.builtin >= 0) == (not generic and spec in (WL.F2_LINEAR, WL.F4_LINEAR, WL.F4_A2P1))
    g = p.geometry(N, H, W, C, K)
    assert _selects_unrolled(m, C, K, g["T"], dtype)
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    U, V = p.kernel_input_transform(wd, xd)
    yf = p.contract_output(V, U, C, N, H, W)
    M = p.contract(V, U, C)
    ys = p.output_transform(M, N, H, W, K)
    y_conv = p.conv2d(xd, wd)
    torch.cuda.synchronize()
    assert torch.equal(y_conv, yf)
    st = _gpu_stages(p, V, U, M, C, K, N, H, W)
    yf64, ys64 = to_np(yf).astype(np.float64), to_np(ys).astype(np.float64)
    op = OP.build_plan(spec, n_o=m)
    b = pair_bound(st, op, dtype, yf64, H, W, y_ref=ys64)
    diff = np.abs(yf64 - ys64)
    print(f"[unrolled] max |diff| {np.max(diff):.3e}, max diff/bound {np.max(diff / b):.3g}, "
          f"median bound/|y| {np.median(b / np.maximum(np.abs(ys64), 1e-30)):.3g}", flush=True)
    assert np.all(np.isfinite(yf64))
    assert np.all(diff <= b)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("spec,m,generic", UNROLLED_PLANS,
                         ids=[f"{s}-m{m}" + ("-runtime" if g else "") for s, m, g in UNROLLED_PLANS])
def test_unrolled_matches_separate(spec, m, generic, dtype):
    """Fused (unrolled instance, one slice per step) against the separate path
    on the same U and V, element by element within the bound between two
    evaluations that differ only in the order of the fp32 channel sums
    (``pair_bound`` with the separate path as the reference)."""
    _unrolled_vs_separate(spec, m, generic, dtype, slices=1)


UNROLLED_TWO_SLICES = [(WL.F2_LINEAR, 2, False), (WL.F4_A2P1, 4, False), (WL.F4_A2P1, 4, True),
                       ("0,a^2+1,a^2-2,inf", 4, False)]


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("spec,m,generic", UNROLLED_TWO_SLICES,
                         ids=[f"{s}-m{m}" + ("-runtime" if g else "") for s, m, g in UNROLLED_TWO_SLICES])
def test_unrolled_two_slices_matches_separate(spec, m, generic, dtype):
    """The same with channel rows of two slices (a step contracts both)."""
    _unrolled_vs_separate(spec, m, generic, dtype, slices=2)


# long rows: two slices per step; rows of three or four slices take two
# unrolled steps per domain point, longer ones run the steps in a loop
UNROLLED_LONG = [
    (WL.F4_A2P1, 4, False, "bf16", 256),     # 512-byte rows: 2 steps per domain point
    (WL.F4_A2P1, 4, False, "f16", 256),      # the same in fp16
    (WL.F4_A2P1, 4, True, "f16", 200),       # 400-byte rows: the last step's second slice partly empty
    (WL.F2_LINEAR, 2, False, "f32", 100),    # 400-byte rows in fp32
    ("0,a^2+1,a^2-2,inf", 4, False, "bf16", 160),   # 320-byte rows: the second step's second slice empty
    ("0,a^2+1,a^2-2,inf", 4, False, "bf16", 520),   # 1040-byte rows: 5 steps in a loop, the last one's second slice empty
    (WL.F2_LINEAR, 2, True, "f32", 200),     # 800-byte rows: 4 steps in a loop, run-time coefficients
]


@pytest.mark.parametrize("spec,m,generic,dtype,C", UNROLLED_LONG,
                         ids=[f"{s}-m{m}-{d}-C{c}" + ("-runtime" if g else "") for s, m, g, d, c in UNROLLED_LONG])
def test_unrolled_long_rows_matches_separate(spec, m, generic, dtype, C):
    """The same with rows longer than two slices."""
    _unrolled_vs_separate(spec, m, generic, dtype, slices=1, C=C)


# narrow rows: 128 / row bytes domain points share a step (8, 4 or 2)
UNROLLED_NARROW = [
    (WL.F4_A2P1, 4, False, "bf16", 3),       # 16-byte rows (the RGB layer): 8 per step
    (WL.F4_A2P1, 4, True, "f16", 16),        # 32-byte rows: 4 per step
    (WL.F2_LINEAR, 2, False, "f32", 12),     # 12 channels padded to 16: 64-byte rows, 2 per step
    ("0,a^2+1,a^2-2,inf", 4, False, "bf16", 24),   # 48-byte rows: the last piece of each half empty
    (WL.F4_LINEAR, 4, False, "f32", 4),      # 32-byte rows in fp32
]


@pytest.mark.parametrize("spec,m,generic,dtype,C", UNROLLED_NARROW,
                         ids=[f"{s}-m{m}-{d}-C{c}" + ("-runtime" if g else "") for s, m, g, d, c in UNROLLED_NARROW])
def test_unrolled_narrow_matches_separate(spec, m, generic, dtype, C):
    """The same with rows of at most 64 bytes, several domain points per step."""
    _unrolled_vs_separate(spec, m, generic, dtype, slices=1, C=C)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("spec,m", [(WL.F2_LINEAR, 2), (WL.F4_A2P1, 4)])
def test_unrolled_builtin_equals_runtime_coefficients(spec, m, dtype):
    """The constant-coefficient instance of a built-in plan drops the zero terms
    of the fold; for finite data the sums are unchanged, so it gives the same
    bits as the run-time-coefficient instance."""
    from paper_1905_05233_amd.winograd import Plan
    N, H, W, C, K = _unrolled_shape(m, dtype, ragged_k=False)
    x, w = _inputs((N, H, W, C, K), dtype, seed=m)
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    pb = Plan(spec, m=m, dtype=dtype, path="fused")
    pr = Plan(spec, m=m, dtype=dtype, path="fused", generic_transforms=True)
    assert pb.builtin >= 0 and pr.builtin < 0
    U, V = pb.kernel_input_transform(wd, xd)
    yb = pb.contract_output(V, U, C, N, H, W)
    yr = pr.contract_output(V, U, C, N, H, W)
    torch.cuda.synchronize()
    assert torch.equal(yb, yr)


@pytest.mark.parametrize("N,H,W,C,K,dtype", [(9, 224, 224, 64, 64, "bf16"), (32, 224, 224, 64, 64, "bf16"),
                                              (9, 222, 222, 60, 70, "bf16"), (9, 222, 218, 60, 70, "f16")])
def test_conv2d_in_chunks_equals_one_launch(N, H, W, C, K, dtype):
    """A batch whose V exceeds the chunk budget (224x224x64 -> 64: 19.7 MB of V
    per image in 16-bit) runs as launch pairs over chunks of images (N = 9:
    5 + 4, N = 32: four of 8), with a workspace for one chunk's V; the output is
    the fused kernel's over the whole batch, bit for bit.  The ragged cases
    (a partial last tile row and column, C and K off the 64-channel blocks)
    take the same split."""
    from paper_1905_05233_amd.winograd import Plan
    x, w = _inputs((N, H, W, C, K), dtype, seed=N + C)
    p = Plan(WL.F4_A2P1, m=4, dtype=dtype)
    assert p.conv_path(N, H, W, C, K) == "fused"
    n_chunks, chunk = p.conv_chunks(N, H, W, C, K)
    assert n_chunks > 1 and chunk == -(-N // n_chunks)
    v_all = 49 * N * (-(-H // 4)) * (-(-W // 4)) * (-(-C // 8) * 8) * 2
    assert p.workspace_bytes(N, H, W, C, K) < v_all        # one chunk's V, not the batch's
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    y = p.conv2d(xd, wd)
    U, V = p.kernel_input_transform(wd, xd)
    y_one = p.contract_output(V, U, C, N, H, W)
    torch.cuda.synchronize()
    assert torch.equal(y, y_one)


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
