"""End-to-end parity of winograd_conv2d on the GPU against the oracle.

For every workload and plan (seeded synthetic inputs, sizes as configured):
  * rel-L2 error against fp64 direct convolution of the dtype-rounded inputs
    is at most min(2 x the oracle's same-algorithm, same-dtype error, cap);
  * element by element: U and V equal the oracle's bit for bit, and y lies
    within ``pair_bound`` of the oracle's y (the two differ only in the order
    of the fp32 channel sums, so the bound is about one unit in the last
    place of y in fp16/bf16); in fp32 also within the a-priori rounding bound
    of the exact value;
  * two runs are bitwise identical.
Bit-exact end-to-end checks use dyadic plans with small-integer inputs, where
every rounding is exact and the result must equal direct convolution.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import check_layer, elementwise_bound, oracle_plan, rounded_inputs, to_dev, to_np
from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP
from paper_1905_05233_amd import workloads as WL

pytestmark = pytest.mark.gpu

CASES = [(name, i) for name in ("cfg1", "cfg2", "cfg3", "cfg4") for i in range(len(WL.CONFIGS[name].plans))]


def _plan(ps, dtype):
    from paper_1905_05233_amd.winograd import Plan
    return Plan(ps.moduli, m=ps.m, dtype=dtype, inner=ps.inner)


@pytest.mark.parametrize("name,idx", CASES, ids=[f"{n}-plan{i}" for n, i in CASES])
def test_workload_parity(name, idx):
    wl = WL.CONFIGS[name]
    ps = wl.plans[idx]
    print(f"[conv] {name} plan {ps.moduli} m={ps.m} {wl.dtype} N={wl.N} H={wl.H} C={wl.C} K={wl.K}", flush=True)
    x, w = rounded_inputs(wl.draw(), wl.dtype)
    p = _plan(ps, wl.dtype)
    xd, wd = to_dev(x, wl.dtype), to_dev(w, wl.dtype)
    y1 = p.conv2d(xd, wd)
    y2 = p.conv2d(xd, wd)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)                       # deterministic
    y = to_np(y1).astype(np.float64)
    op = oracle_plan(ps)
    y64 = OC.direct_f64(x, w)
    st = check_layer(p, op, x, w, wl.dtype, y, label=f"{name} plan{idx}")
    err_gpu = OC.rel_l2(y, y64)
    err_oracle = OC.rel_l2(st["y"], y64)
    print(f"[conv] {name} plan{idx}: err_gpu={err_gpu:.3e} err_oracle={err_oracle:.3e} cap={wl.cap}", flush=True)
    assert np.all(np.isfinite(y))
    assert err_gpu <= min(2 * err_oracle, wl.cap)
    if wl.dtype == "f32":
        assert np.all(np.abs(y - y64) <= elementwise_bound(x, w, op, wl.dtype, y64))


@pytest.mark.parametrize("spec,m", [(WL.F2_LINEAR, 2), (WL.F4_A2P1, 4), ("0,a^2+1,inf", 2)])
@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", [(1, 16, 16, 8, 8), (2, 7, 11, 3, 5), (1, 1, 1, 1, 1), (3, 13, 6, 28, 130)])
def test_bit_exact_dyadic(spec, m, dtype, shape):
    from paper_1905_05233_amd.winograd import Plan
    N, H, W, C, K = shape
    print(f"[conv-exact] {spec} m={m} {dtype} {shape}", flush=True)
    dist = "ternary" if dtype == "bf16" else "int2"
    x, w = WL.draw_inputs(N, H, W, C, K, dist, seed=N + H + W + C + K)
    p = Plan(spec, m=m, dtype=dtype)
    y = to_np(p.conv2d(to_dev(x, dtype), to_dev(w, dtype))).astype(np.float64)
    ref = OC.direct_f64(x, w)
    # every intermediate is exactly representable: check that premise on the oracle
    op = OP.build_plan(spec, n_o=m)
    assert np.array_equal(OC.winograd_emulated(x, w, op, dtype).astype(np.float64), ref)
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("spec,m", [(WL.F4_LINEAR, 4), (WL.F6_TWO_QUAD, 6), (WL.F6_ONE_A2P1, 6), (WL.F6_LINEAR, 6)])
@pytest.mark.parametrize("shape", [(1, 1, 1, 1, 1), (2, 5, 9, 3, 7), (1, 14, 14, 64, 64)])
def test_edge_shapes(dtype, spec, m, shape):
    """Empty-ish, ragged and padded shapes: tiles beyond H/W, C and K not
    multiples of 8, a single pixel, one channel."""
    from paper_1905_05233_amd.winograd import Plan
    N, H, W, C, K = shape
    print(f"[conv-edge] {spec} m={m} {dtype} {shape}", flush=True)
    x, w = WL.draw_inputs(N, H, W, C, K, "halfnormal", seed=H * W + C)
    x, w = OF.to_dtype(x, dtype), OF.to_dtype(w, dtype)
    p = Plan(spec, m=m, dtype=dtype)
    y = to_np(p.conv2d(to_dev(x, dtype), to_dev(w, dtype))).astype(np.float64)
    op = OP.build_plan(spec, n_o=m)
    check_layer(p, op, x, w, dtype, y, label=f"edge {spec} {dtype} {shape}")
    if dtype == "f32":
        y64 = OC.direct_f64(x, w)
        assert np.all(np.abs(y - y64) <= elementwise_bound(x, w, op, dtype, y64))


def test_workspace_reuse_and_external_binding():
    from paper_1905_05233_amd.winograd import Plan
    p = Plan(WL.F4_LINEAR, m=4, dtype="f32")
    x, w = WL.draw_inputs(2, 20, 20, 16, 24, "uniform", seed=9)
    ws = torch.empty(p.workspace_bytes(2, 20, 20, 16, 24), dtype=torch.uint8, device="cuda")
    y1 = p.conv2d(to_dev(x, "f32"), to_dev(w, "f32"), workspace=ws)
    xs, ws_ = WL.draw_inputs(1, 8, 8, 16, 24, "uniform", seed=10)
    y_small = p.conv2d(to_dev(xs, "f32"), to_dev(ws_, "f32"), workspace=ws)   # smaller call, same workspace
    y2 = p.conv2d(to_dev(x, "f32"), to_dev(w, "f32"), workspace=ws)
    assert torch.equal(y1, y2)
    ref = OC.direct_f64(xs, ws_)
    assert OC.rel_l2(to_np(y_small), ref) < 1e-5


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("spec,m", [(WL.F2_LINEAR, 2), (WL.F4_LINEAR, 4), (WL.F4_A2P1, 4), (WL.F6_TWO_QUAD, 6)])
def test_factors_in_g_parity(spec, m, dtype):
    """Plans with the CRT factors on the kernel side: the 2x rule, U and V
    bit-equal to the oracle's emulation of the same plan and y within the
    pair bound."""
    from paper_1905_05233_amd.winograd import Plan
    N, H, W, C, K = 2, 26, 30, 24, 40
    x, w = WL.draw_inputs(N, H, W, C, K, "halfnormal", seed=5 * m)
    x, w = OF.to_dtype(x, dtype), OF.to_dtype(w, dtype)
    op = OP.build_plan(spec, n_o=m, factors="G")
    pg = Plan(spec, m=m, dtype=dtype, factors="G")
    yg = to_np(pg.conv2d(to_dev(x, dtype), to_dev(w, dtype)))
    y64 = OC.direct_f64(x, w)
    st = check_layer(pg, op, x, w, dtype, yg, label=f"factors-G {spec} {dtype}")
    yo = st["y"]
    err_gpu, err_or = OC.rel_l2(yg, y64), OC.rel_l2(yo, y64)
    err_b = OC.rel_l2(OC.winograd_emulated(x, w, OP.build_plan(spec, n_o=m), dtype), y64)
    print(f"[factors-G] {spec} {dtype}: gpu {err_gpu:.3e} oracle {err_or:.3e} (factors in B: {err_b:.3e})",
          flush=True)
    assert err_gpu <= 2 * err_or


def test_factors_in_g_bit_exact_dyadic():
    """F(2,3) with the factors in G has entries 0, +-1, +-1/2: on small
    integers every rounding is exact and the result is direct convolution."""
    from paper_1905_05233_amd.winograd import Plan
    x, w = WL.draw_inputs(2, 9, 13, 5, 7, "int2", seed=21)
    op = OP.build_plan(WL.F2_LINEAR, n_o=2, factors="G")
    ref = OC.direct_f64(x, w)
    assert np.array_equal(OC.winograd_emulated(x, w, op, "f32").astype(np.float64), ref)
    y = to_np(Plan(WL.F2_LINEAR, m=2, dtype="f32", factors="G").conv2d(to_dev(x, "f32"), to_dev(w, "f32")))
    assert np.array_equal(y.astype(np.float64), ref)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("spec,m", [(WL.F4_LINEAR, 4), (WL.F4_A2P1, 4), (WL.F6_TWO_QUAD, 6),
                                    ("0,-1,1,-1/2,2,1/2,-2,-1/4,4,inf", 8)])
@pytest.mark.parametrize("path", ["separate", "fused"])
def test_scaled_plan_parity(spec, m, dtype, path):
    """Plans with the rows of G and A scaled to unit 1-norm (compensated in
    B): U and V bit-equal to the oracle's emulation of the scaled plan, y
    within the pair bound, and the 2x rule against fp64 direct convolution.
    In fp16 the scaling keeps F(8x8)'s transforms in range (rel-L2 about 0.07
    where the unscaled plan overflows)."""
    from paper_1905_05233_amd.winograd import Plan
    if path == "fused" and m > 6:
        pytest.skip("the fused kernel takes input tiles up to 8")
    N, H, W, C, K = 2, 26, 30, 24, 40
    x, w = WL.draw_inputs(N, H, W, C, K, "halfnormal", seed=9 * m)
    x, w = OF.to_dtype(x, dtype), OF.to_dtype(w, dtype)
    op = OP.build_plan(spec, n_o=m, scaling="l1")
    p = Plan(spec, m=m, dtype=dtype, scaling="l1", path=path)
    y = to_np(p.conv2d(to_dev(x, dtype), to_dev(w, dtype))).astype(np.float64)
    st = check_layer(p, op, x, w, dtype, y, label=f"scaled {spec} {dtype} {path}")
    y64 = OC.direct_f64(x, w)
    err_gpu, err_or = OC.rel_l2(y, y64), OC.rel_l2(st["y"], y64)
    err_plain = OC.rel_l2(OC.winograd_emulated(x, w, OP.build_plan(spec, n_o=m), dtype), y64)
    print(f"[scaled] {spec} {dtype} {path}: gpu {err_gpu:.3e} oracle {err_or:.3e} (unscaled oracle {err_plain:.3e})",
          flush=True)
    assert np.all(np.isfinite(y))
    assert err_gpu <= 2 * err_or
