"""Pins of the oracle's convolution references and rounding emulation (CPU only).

* fp64 direct convolution against PyTorch's CPU conv2d in float64 (a library
  routine for the same definition) and against the exact definition;
* eq. (2) in exact rationals equals direct convolution bit for bit, on inputs
  with partial tiles, for every workload modulus set and the worked example;
* the rounding-emulated Winograd: exact on dyadic plans with small-integer
  inputs (every rounding is then exact), inside the a-priori error bound
  otherwise, and with every storage rounding actually applied;
* the superlinear plan's error is below the linear plan's at fp16 (the
  direction the paper reports, Section 3.2); magnitudes are parity unpinned
  because the paper's Fig. 3 values are not in its text.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP
from paper_1905_05233_amd import workloads as WL

ALL_SETS = [
    (WL.F2_LINEAR, 2), (WL.F4_LINEAR, 4), (WL.F4_A2P1, 4),
    (WL.F6_LINEAR, 6), (WL.F6_TWO_QUAD, 6), (WL.F6_ONE_A2P1, 6),
]


def _torch_direct(x, w):
    xt = torch.from_numpy(np.asarray(x, np.float64)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(np.asarray(w, np.float64)).permute(0, 3, 1, 2)
    return torch.nn.functional.conv2d(xt, wt, padding=1).permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("shape", [(2, 7, 9, 3, 5), (1, 1, 1, 1, 1), (3, 12, 5, 16, 4)])
def test_direct_f64_matches_torch(shape):
    N, H, W, C, K = shape
    x, w = WL.draw_inputs(N, H, W, C, K, "uniform", seed=3)
    np.testing.assert_allclose(OC.direct_f64(x, w), _torch_direct(x, w), rtol=1e-13, atol=1e-13)


def test_direct_exact_matches_f64_on_integers():
    x, w = WL.draw_inputs(1, 5, 6, 3, 2, "int2", seed=4)
    ye = OC.direct_exact(x.tolist(), w.tolist())
    assert np.array_equal(np.array(ye, dtype=np.float64), OC.direct_f64(x, w))


def _frac_inputs(N, H, W, C, K, seed):
    """Small rational inputs (eighths) so exact arithmetic stays fast."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = [[[[Fraction(int(v), 8) for v in rng.integers(-8, 9, size=C)] for _ in range(W)]
          for _ in range(H)] for _ in range(N)]
    w = [[[[Fraction(int(v), 8) for v in rng.integers(-8, 9, size=C)] for _ in range(3)]
          for _ in range(3)] for _ in range(K)]
    return x, w


@pytest.mark.parametrize("spec,m", ALL_SETS)
def test_exact_winograd_equals_direct(spec, m):
    pl = OP.build_plan(spec, n_o=m)
    for hw in [(m, m + 1), (2 * m - 1, m)]:
        x, w = _frac_inputs(1, hw[0], hw[1], 2, 2, seed=m + hw[0])
        assert OC.winograd_exact(x, w, pl) == OC.direct_exact(x, w)


@pytest.mark.parametrize("spec,m", ALL_SETS)
def test_exact_winograd_equals_direct_with_factors_in_g(spec, m):
    """The CRT factors on the kernel side give the same exact convolution."""
    pl = OP.build_plan(spec, n_o=m, factors="G")
    x, w = _frac_inputs(1, 2 * m - 1, m + 1, 2, 2, seed=3 * m)
    assert OC.winograd_exact(x, w, pl) == OC.direct_exact(x, w)


def test_exact_winograd_worked_example_plan():
    for b, c in [(0, 1), (1, 1), (0, -2)]:
        pl = OP.build_plan(["0", (Fraction(c), Fraction(b), Fraction(1)), "inf"], n_o=2, inner="0,1,inf")
        x, w = _frac_inputs(2, 3, 5, 2, 1, seed=b + 7)
        assert OC.winograd_exact(x, w, pl) == OC.direct_exact(x, w)


@pytest.mark.parametrize("spec,m,dtype,dist", [
    (WL.F2_LINEAR, 2, "f32", "int2"),
    (WL.F2_LINEAR, 2, "f16", "int2"),
    (WL.F4_A2P1, 4, "f32", "int2"),
    (WL.F4_A2P1, 4, "f16", "int2"),
    (WL.F4_A2P1, 4, "bf16", "ternary"),
    (WL.F2_LINEAR, 2, "bf16", "ternary"),
])
def test_emulation_exact_on_dyadic_plans(spec, m, dtype, dist):
    """Dyadic matrices and small integers: every rounding is exact, so the
    emulation must reproduce the direct result bit for bit (tiling check)."""
    pl = OP.build_plan(spec, n_o=m)
    for (N, H, W, C, K) in [(2, 9, 7, 8, 3), (1, m, m, 3, 2), (1, 1, 2 * m + 1, 5, 4)]:
        x, w = WL.draw_inputs(N, H, W, C, K, dist, seed=H * W)
        y = OC.winograd_emulated(x, w, pl, dtype)
        assert np.array_equal(y.astype(np.float64), OC.direct_f64(x, w))


@pytest.mark.parametrize("spec,m", ALL_SETS)
@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_emulation_within_error_bound(spec, m, dtype):
    pl = OP.build_plan(spec, n_o=m)
    N, H, W, C, K = 1, 2 * m + 3, m + 1, 16, 4
    x, w = WL.draw_inputs(N, H, W, C, K, "uniform", seed=11)
    x, w = OF.to_dtype(x, dtype), OF.to_dtype(w, dtype)
    y = OC.winograd_emulated(x, w, pl, dtype).astype(np.float64)
    y64 = OC.direct_f64(x, w)
    bound = OC.error_bound_coefficient(pl, C, dtype) * OC.abs_bound(x, w, pl) \
        + OF.UNIT_ROUNDOFF[dtype] * np.abs(y64)
    assert np.all(np.abs(y - y64) <= bound)
    # the bound is not vacuous: it stays far below the magnitudes involved
    assert np.max(bound) < 0.2 * np.max(np.abs(y64)) or dtype != "f32"


def test_abs_bound_dominates():
    pl = OP.build_plan(WL.F4_LINEAR, n_o=4)
    x, w = WL.draw_inputs(1, 9, 9, 3, 2, "uniform", seed=1)
    assert np.all(np.abs(OC.direct_f64(x, w)) <= OC.abs_bound(x, w, pl) * (1 + 1e-12))
    xp, wp = np.abs(x), np.abs(w)
    # with non-negative data and a non-negative plan the two coincide exactly
    pln = OP.build_plan("0,inf,a^2+1", n_o=2)   # entries 0, +-1; |.| keeps a valid bound
    assert np.all(OC.abs_bound(xp, wp, pln) >= OC.direct_f64(xp, wp) - 1e-12)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_storage_roundings_are_applied(dtype):
    pl = OP.build_plan(WL.F4_A2P1, n_o=4)
    x, w = WL.draw_inputs(1, 8, 8, 4, 3, "uniform", seed=2)
    x, w = OF.to_dtype(x, dtype), OF.to_dtype(w, dtype)
    V = OC.input_transform_emulated(x, pl, dtype)
    U = OC.kernel_transform_emulated(w, pl, dtype)
    assert np.array_equal(OF.to_dtype(V, dtype), V)
    assert np.array_equal(OF.to_dtype(U, dtype), U)
    V32 = OC.input_transform_emulated(x, pl, "f32")
    assert not np.array_equal(V32, V)
    y = OC.winograd_emulated(x, w, pl, dtype)
    assert np.array_equal(OF.to_dtype(y, dtype), y)


def test_superlinear_more_accurate_fp16():
    """Section 3.2: at fp16 the a^2+1 plan is more accurate than Toom-Cook
    F(4x4) on the same data (direction only)."""
    wl = WL.CONFIGS["cfg3"]
    x, w = wl.draw()
    x, w = OF.to_dtype(x, "f16"), OF.to_dtype(w, "f16")
    y64 = OC.direct_f64(x, w)
    errs = [OC.rel_l2(OC.winograd_emulated(x, w, OP.build_plan(p.moduli, n_o=p.m), "f16"), y64)
            for p in wl.plans]
    assert errs[1] < errs[0]


def test_rel_l2():
    a = np.array([3.0, 4.0])
    assert OC.rel_l2(a, a) == 0.0
    assert OC.rel_l2(np.array([3.0, 4.0 + 5.0]), a) == pytest.approx(1.0)


def test_pairwise_contraction_tree_shape():
    """The pairwise channel sum of the oracle against hand-built trees: with
    leaf = 1 channel and values chosen so that fp32 addition order shows,
    5 leaves sum as ((l0 + l1) + (l2 + l3)) + l4 (padded to 8 leaves) and 3
    as (l0 + l1) + l2; the plain left-to-right sum differs."""
    big, tiny = np.float32(2.0 ** 24), np.float32(1.0)
    for vals, want in (([big, tiny, tiny, tiny, -big], np.float32((big + tiny) + (tiny + tiny)) + (-big)),
                       ([big, tiny, tiny], np.float32(big + tiny) + tiny)):
        C = len(vals)
        V = np.array(vals, np.float32).reshape(1, 1, 1, C)
        U = np.ones((1, 1, 1, C), np.float32)
        got = OC.contraction_emulated_pairwise(V, U, leaf=1)
        assert got.shape == (1, 1, 1, 1)
        assert got[0, 0, 0, 0] == np.float32(want)
    seq = np.float32(0)
    for v in [big, tiny, tiny, tiny, -big]:
        seq = np.float32(seq + v)
    assert seq != OC.contraction_emulated_pairwise(np.array([big, tiny, tiny, tiny, -big], np.float32)
                                                   .reshape(1, 1, 1, 5), np.ones((1, 1, 1, 5), np.float32), 1)[0, 0, 0, 0]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_pairwise_contraction_close_to_exact_sum(dtype):
    """On random data the pairwise sum differs from the exact channel sum by
    at most its bound (leaf + ceil(log2 leaves) + 2) u32 sum |V||U|."""
    rng = np.random.default_rng(2)
    C, leaf = 300, OC.leaf_channels(dtype)
    V = OF.to_dtype(rng.standard_normal((2, 2, 7, C)).astype(np.float32), dtype)
    U = OF.to_dtype(rng.standard_normal((2, 2, 5, C)).astype(np.float32), dtype)
    M = OC.contraction_emulated_pairwise(V, U, leaf).astype(np.float64)
    ex = np.einsum("abtc,abkc->abtk", V.astype(np.float64), U.astype(np.float64))
    mag = np.einsum("abtc,abkc->abtk", np.abs(V).astype(np.float64), np.abs(U).astype(np.float64))
    n = -(-C // leaf)
    depth = (n - 1).bit_length()
    assert np.all(np.abs(M - ex) <= 1.1 * (leaf + depth + 2) * 2.0 ** -24 * mag)
