"""Per-kernel parity on the GPU through the C ABI stage entry points.

Bit-exact where every rounding is exact (dyadic transforms, small-integer
data): this pins tile indexing, the Winograd-domain index xi = i*alpha' + j,
the channel padding and the GEMM lane layouts.  Elsewhere each stage is held
to the rounding bound of its own arithmetic against the oracle.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import ALL_SHAPES, TORCH, to_dev, to_np
from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP
from paper_1905_05233_amd import workloads as WL

pytestmark = pytest.mark.gpu

DYADIC = [(WL.F2_LINEAR, 2), (WL.F4_A2P1, 4), ("0,a^2+1,inf", 2)]
DTYPES = ["f32", "f16", "bf16"]


def _plan(spec, m, dtype, inner="0,-1,inf"):
    from paper_1905_05233_amd.winograd import Plan
    print(f"[stage] plan {spec} m={m} dtype={dtype}", flush=True)
    return Plan(spec, m=m, dtype=dtype, inner=inner), OP.build_plan(spec, n_o=m, inner=inner)


@pytest.mark.parametrize("spec,m", DYADIC)
@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("shape", [(2, 9, 7, 5), (1, 1, 1, 3), (3, 16, 13, 40)])
def test_input_transform_bit_exact(spec, m, dtype, shape):
    p, op = _plan(spec, m, dtype)
    N, H, W, C = shape
    dist = "ternary" if dtype == "bf16" else "int2"
    x, _ = WL.draw_inputs(N, H, W, C, 1, dist, seed=H * 31 + W)
    V = to_np(p.input_transform(to_dev(x, dtype)))
    torch.cuda.synchronize()
    ref = OC.input_transform_emulated(x, op, dtype)
    al = op.alpha
    ref = ref.reshape(al * al, -1, C)
    assert V.shape[:2] == ref.shape[:2]
    assert np.array_equal(V[:, :, :C], ref)
    assert np.all(V[:, :, C:] == 0)


@pytest.mark.parametrize("spec,m,dtype,shape", [(WL.F4_A2P1, 4, "bf16", (3, 186, 250, 64)),
                                                 (WL.F2_LINEAR, 2, "f16", (5, 130, 130, 128)),
                                                 (WL.F4_A2P1, 4, "f32", (5, 130, 130, 128))])
def test_input_transform_multi_tile_bit_exact(spec, m, dtype, shape):
    """Layers with 8192 or more (tile, 64-channel) units run workgroups that walk
    four tiles in turn; tile counts that are not a multiple of four leave a
    ragged last workgroup.  Exact data: V equals the oracle bit for bit."""
    p, op = _plan(spec, m, dtype)
    N, H, W, C = shape
    T = N * (-(-H // m)) * (-(-W // m))
    assert T * (-(-C // 64)) >= 8192 and T % 4 != 0
    dist = "ternary" if dtype == "bf16" else "int2"
    x, _ = WL.draw_inputs(N, H, W, C, 1, dist, seed=H + W + C)
    V = to_np(p.input_transform(to_dev(x, dtype)))
    torch.cuda.synchronize()
    ref = OC.input_transform_emulated(x, op, dtype).reshape(op.alpha ** 2, T, C)
    assert np.array_equal(V[:, :, :C], ref)


SHAPE_IDS = [f"t{m + 2}-{s}" for s, m in ALL_SHAPES]


@pytest.mark.parametrize("spec,m", ALL_SHAPES, ids=SHAPE_IDS)
@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("C", [72, 5])
def test_input_transform_bit_exact_random(spec, m, dtype, C):
    """Every compiled (input tile, alpha') shape on random half-normal data:
    the kernel runs the oracle's operations (ascending-index fused
    multiply-adds, one dtype rounding), so V is equal bit for bit.  C = 72
    spans two 64-channel columns (ragged second), C = 5 the narrow layout."""
    p, op = _plan(spec, m, dtype)
    N, H, W = 2, 2 * m + 3, 3 * m - 1
    x, _ = WL.draw_inputs(N, H, W, C, 1, "halfnormal", seed=5 * m + C)
    x = OF.to_dtype(x, dtype)
    V = to_np(p.input_transform(to_dev(x, dtype)))
    ref = OC.input_transform_emulated(x, op, dtype).reshape(op.alpha ** 2, -1, C)
    assert np.array_equal(V[:, :, :C], ref, equal_nan=True)
    assert np.all(V[:, :, C:] == 0)


@pytest.mark.parametrize("spec,m,dtype,shape", [(WL.F4_A2P1, 4, "bf16", (3, 150, 170, 128)),
                                                 (WL.F6_TWO_QUAD, 6, "f16", (6, 170, 160, 128)),
                                                 (WL.F4_LINEAR, 4, "f32", (3, 150, 170, 128))])
def test_input_transform_walking_instance_bit_exact_random(spec, m, dtype, shape):
    """The instance whose workgroups walk four tiles (built-in plans, layers
    of 8192 or more (tile, 64-channel) units, a ragged last workgroup) on
    random data: V equal to the oracle bit for bit."""
    p, op = _plan(spec, m, dtype)
    N, H, W, C = shape
    T = N * (-(-H // m)) * (-(-W // m))
    assert T * (-(-C // 64)) >= 8192 and T % 4 != 0
    x, _ = WL.draw_inputs(N, H, W, C, 1, "halfnormal", seed=H + C)
    x = OF.to_dtype(x, dtype)
    V = to_np(p.input_transform(to_dev(x, dtype)))
    ref = OC.input_transform_emulated(x, op, dtype).reshape(op.alpha ** 2, T, C)
    assert np.array_equal(V[:, :, :C], ref, equal_nan=True)


@pytest.mark.parametrize("spec,m", ALL_SHAPES, ids=SHAPE_IDS)
@pytest.mark.parametrize("dtype", DTYPES)
def test_kernel_transform_bit_exact_random(spec, m, dtype):
    p, op = _plan(spec, m, dtype)
    K, C = 9, 21
    _, w = WL.draw_inputs(1, 1, 1, C, K, "halfnormal", seed=K + C + m)
    w = OF.to_dtype(w, dtype)
    U = to_np(p.kernel_transform(to_dev(w, dtype)))
    ref = OC.kernel_transform_emulated(w, op, dtype).reshape(op.alpha ** 2, K, C)
    assert np.array_equal(U[:, :, :C], ref, equal_nan=True)
    assert np.all(U[:, :, C:] == 0)


@pytest.mark.parametrize("spec,m", ALL_SHAPES, ids=SHAPE_IDS)
@pytest.mark.parametrize("dtype", DTYPES)
def test_output_transform_bit_exact_random(spec, m, dtype):
    """y = A^T M A from random fp32 M: two passes of fused multiply-adds and
    one dtype rounding, equal to the oracle bit for bit; 70 output channels
    span two 64-channel workgroups, H and W leave partial tiles."""
    p, op = _plan(spec, m, dtype)
    N, H, W, K = 2, 2 * m + 1, m + 3, 70
    g = p.geometry(N, H, W, 1, K)
    al = op.alpha
    rng = np.random.Generator(np.random.PCG64(7 + m))
    Mx = np.zeros((al * al, g["T"], g["Kp"]), np.float32)
    Mx[:, :, :K] = rng.standard_normal((al * al, g["T"], K))
    y = to_np(p.output_transform(torch.from_numpy(Mx).cuda(), N, H, W, K))
    Mo = Mx[:, :, :K].reshape(al, al, N, g["th"], g["tw"], K)
    ref = OC.output_transform_emulated(Mo, op, dtype, H, W)
    assert np.array_equal(y, ref, equal_nan=True)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("T,C,K", [(1, 1, 1), (37, 8, 5), (129, 40, 130), (300, 264, 96), (130, 320, 257),
                                   (1568, 128, 128)])
def test_contract_bit_exact_on_integers(dtype, T, C, K):
    p, _ = _plan(WL.F4_A2P1, 4, dtype)
    a2 = p.alpha ** 2
    Cp = -(-C // 8) * 8
    rng = np.random.Generator(np.random.PCG64(T + C + K))
    V = np.zeros((a2, T, Cp), np.float32)
    U = np.zeros((a2, K, Cp), np.float32)
    V[:, :, :C] = rng.integers(-3, 4, size=(a2, T, C))
    U[:, :, :C] = rng.integers(-3, 4, size=(a2, K, C))
    M = to_np(p.contract(to_dev(V, dtype), to_dev(U, dtype), C))
    ref = np.einsum("xtc,xkc->xtk", V.astype(np.float64), U.astype(np.float64))
    assert np.array_equal(M[:, :, :K].astype(np.float64), ref)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("T,C,K", [(200, 256, 72), (150, 520, 136), (97, 136, 40)])
def test_contract_random_within_bound(dtype, T, C, K):
    """Random data; C = 520 (and C = 136 in fp32) gives rows over 512 bytes,
    which run the 128 x 128 block kernel."""
    p, _ = _plan(WL.F6_TWO_QUAD, 6, dtype)
    a2 = p.alpha ** 2
    rng = np.random.Generator(np.random.PCG64(3))
    Cp = -(-C // 8) * 8
    V = np.zeros((a2, T, Cp), np.float32)
    U = np.zeros((a2, K, Cp), np.float32)
    V[:, :, :C] = OF.to_dtype(rng.standard_normal((a2, T, C)).astype(np.float32), dtype)
    U[:, :, :C] = OF.to_dtype(rng.standard_normal((a2, K, C)).astype(np.float32), dtype)
    M = to_np(p.contract(to_dev(V, dtype), to_dev(U, dtype), C))[:, :, :K]
    V, U = V[:, :, :C], U[:, :, :C]
    ref = np.einsum("xtc,xkc->xtk", V.astype(np.float64), U.astype(np.float64))
    mag = np.einsum("xtc,xkc->xtk", np.abs(V).astype(np.float64), np.abs(U).astype(np.float64))
    u32 = 2.0 ** -24
    # fp32 products (exact for fp16/bf16) and a C-term fp32 sum
    assert np.all(np.abs(M - ref) <= (C + 1) * u32 * 1.1 * mag)


@pytest.mark.parametrize("spec,m", [(WL.F2_LINEAR, 2), (WL.F4_A2P1, 4), (WL.F6_TWO_QUAD, 6),
                                    ("0,-1,1,-1/2,2,1/2,-2,a^2+1,inf", 8)])
@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("shape", [(2, 9, 7, 5, 6), (1, 30, 26, 64, 40), (1, 1, 1, 1, 1)])
def test_kernel_input_transform_matches_separate_calls(spec, m, dtype, shape):
    """The combined launch (conv2d's first kernel) gives U and V bit-equal to
    the two separate stage kernels, including C not a multiple of the run."""
    p, _ = _plan(spec, m, dtype)
    N, H, W, C, K = shape
    x, w = WL.draw_inputs(N, H, W, C, K, "halfnormal", seed=C + K)
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    U2, V2 = p.kernel_input_transform(wd, xd)
    U1, V1 = p.kernel_transform(wd), p.input_transform(xd)
    torch.cuda.synchronize()
    assert torch.equal(U1, U2)
    assert torch.equal(V1, V2)


BUILTIN = [(WL.F2_LINEAR, 2), (WL.F4_LINEAR, 4), (WL.F4_A2P1, 4), (WL.F6_LINEAR, 6), (WL.F6_TWO_QUAD, 6),
           (WL.F6_ONE_A2P1, 6)]


@pytest.mark.parametrize("spec,m", BUILTIN)
@pytest.mark.parametrize("dtype", DTYPES)
def test_builtin_transforms_equal_generic(spec, m, dtype):
    """Constant-coefficient transform kernels (zero terms dropped) against the
    kernels that read the same tables at run time: V and y equal value for
    value (finite data), on a shape with ragged tiles and channels."""
    from paper_1905_05233_amd.winograd import Plan
    pb, pg = Plan(spec, m=m, dtype=dtype, path="separate"), Plan(spec, m=m, dtype=dtype, path="separate",
                                                                  generic_transforms=True)
    assert pb.builtin >= 0 and pg.builtin == -1
    N, H, W, C, K = 2, 23, 19, 20, 36
    x, w = WL.draw_inputs(N, H, W, C, K, "halfnormal", seed=m + C)
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    Ub, Vb = pb.kernel_input_transform(wd, xd)
    Ug, Vg = pg.kernel_input_transform(wd, xd)
    assert torch.equal(Ub, Ug) and torch.equal(Vb, Vg)
    assert torch.equal(pb.input_transform(xd), Vg)
    M = pb.contract(Vb, Ub, C)
    assert torch.equal(pb.output_transform(M, N, H, W, K), pg.output_transform(M, N, H, W, K))
    assert torch.equal(pb.conv2d(xd, wd), pg.conv2d(xd, wd))
