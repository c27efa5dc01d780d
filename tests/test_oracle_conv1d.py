"""The oracle's 1D F(m, 3) against what fixes it independently: exact
Winograd equals the definition of the 1D convolution on tiny rational inputs
(full and partial tiles, every kind of plan); Lavin & Gray's published 1D
F(2,3) and F(4,3) matrices (the fixture) compute the same convolution; the
rounding emulation is exact on dyadic plans with small integers and, in
fp16, the a^2+1 plan is the more accurate one (the direction Section 3.1
reports)."""
from fractions import Fraction

import numpy as np
import pytest

from conftest import frac_matrix, load_golden
from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP
from paper_1905_05233_amd import workloads as WL

PLANS = [("0,1,-1,inf", 2, "0,-1,inf"), ("0,1,-1,1/2,-1/2,inf", 4, "0,-1,inf"), ("0,1,-1,a^2+1,inf", 4, "0,-1,inf"),
         ("0,-1,1,a^2+1,a^2-2,inf", 6, "0,-1,inf"), ("a^2+1,a^2+2", 2, "0,-1,inf"),
         ("0,-1,a^3+2,inf", 4, "0,-1,1,-2,inf"), ("0,1,-1,1/2", 2, "0,1,inf")]


def _rand_rational(rng, shape):
    out = np.empty(shape, dtype=object)
    for idx in np.ndindex(*shape):
        out[idx] = Fraction(int(rng.integers(-9, 10)), int(rng.integers(1, 5)))
    return out.tolist()


@pytest.mark.parametrize("spec,m,inner", PLANS)
def test_exact_1d_winograd_equals_direct(spec, m, inner):
    pl = OP.build_plan(spec, n_o=m, inner=inner)
    rng = np.random.default_rng(m)
    for (N, L, C, K) in [(1, m, 2, 1), (2, 2 * m + 1, 3, 2), (1, 1, 1, 1)]:
        x, w = _rand_rational(rng, (N, L, C)), _rand_rational(rng, (K, 3, C))
        assert OC.winograd1d_exact(x, w, pl) == OC.direct1d_exact(x, w)


@pytest.mark.parametrize("name,m", [("F(2,3)", 2), ("F(4,3)", 4)])
def test_lavin_gray_1d_matrices_compute_the_convolution(name, m):
    """The published matrices, run through the oracle's 1D Winograd, give the
    1D convolution exactly; the oracle's plan with the CRT factors in G is
    those matrices (F(4,3)) or equal up to single-row signs (F(2,3))."""
    gold = load_golden("lavin_gray_2016.json")[name]
    G, BT, AT = frac_matrix(gold["G"]), frac_matrix(gold["BT"]), frac_matrix(gold["AT"])
    lav = OP.build_plan(gold["points"], n_o=m, factors="G")
    lav.G, lav.B, lav.A = G, [list(r) for r in zip(*BT)], [list(r) for r in zip(*AT)]
    rng = np.random.default_rng(3)
    x, w = _rand_rational(rng, (2, 3 * m + 1, 2)), _rand_rational(rng, (3, 3, 2))
    assert OC.winograd1d_exact(x, w, lav) == OC.direct1d_exact(x, w)


@pytest.mark.parametrize("spec,m", [(WL.F2_LINEAR, 2), (WL.F4_A2P1, 4), ("0,a^2+1,inf", 2)])
@pytest.mark.parametrize("dtype,dist", [("f32", "int2"), ("f16", "int2"), ("bf16", "ternary")])
def test_1d_emulation_exact_on_dyadic_plans(spec, m, dtype, dist):
    pl = OP.build_plan(spec, n_o=m)
    x4, w4 = WL.draw_inputs(3, 1, 5 * m + 1, 6, 4, dist, seed=m)
    x, w = x4[:, 0], w4[:, 1]
    y = OC.winograd1d_emulated(x, w, pl, dtype)
    assert np.array_equal(y.astype(np.float64), OC.direct1d_f64(x, w))


def test_1d_direct_f64_matches_exact():
    rng = np.random.default_rng(1)
    x = rng.integers(-5, 6, size=(2, 9, 3)).astype(np.float64)
    w = rng.integers(-5, 6, size=(4, 3, 3)).astype(np.float64)
    ex = OC.direct1d_exact(x.tolist(), w.tolist())
    assert np.array_equal(OC.direct1d_f64(x, w), np.array(ex, dtype=np.float64))


def test_1d_superlinear_more_accurate_fp16():
    """F(4,3) in fp16: {0, 1, -1, a^2+1, inf} beats the linear points
    {0, 1, -1, 1/2, -1/2, inf} on the same data (direction only)."""
    x4, w4 = WL.draw_inputs(4, 1, 256, 32, 32, "halfnormal", seed=5)
    x, w = OF.to_dtype(x4[:, 0], "f16"), OF.to_dtype(w4[:, 1], "f16")
    y64 = OC.direct1d_f64(x, w)
    e_lin = OC.rel_l2(OC.winograd1d_emulated(x, w, OP.build_plan(WL.F4_LINEAR, n_o=4), "f16"), y64)
    e_quad = OC.rel_l2(OC.winograd1d_emulated(x, w, OP.build_plan(WL.F4_A2P1, n_o=4), "f16"), y64)
    assert e_quad < e_lin
