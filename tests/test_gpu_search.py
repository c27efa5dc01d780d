"""The polynomial-set search on the GPU (Section 3.1's error-versus-ratio sweep
on seeded synthetic data).

* The search's reference, the fp32 F(2x2,3x3) plan, is within 1e-6 of fp64
  direct convolution on the sweep data, so it can rank errors of 1e-6 and up.
* Every set's GPU error obeys the parity rule against the oracle's emulation
  of the same set (at most twice the oracle's same-algorithm error).
* The paper's finding holds: for F(4x4) and F(6x6) the most accurate set with
  degree-2 moduli is several times more accurate than the most accurate set
  of linear points, in fp32 and in bf16.
* Plan selection returns the most accurate candidate, or the fastest one
  within an error cap.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import to_np
from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP
from paper_1905_05233_amd import search as S
from paper_1905_05233_amd import workloads as WL

pytestmark = pytest.mark.gpu

SHAPE = (1, 24, 24, 32, 32)


def test_reference_is_accurate():
    for dtype in ("f32", "bf16"):
        x, w = S.layer_inputs(*SHAPE, dtype=dtype, seed=0)
        ref = to_np(S.reference(x, w)).astype(np.float64)
        x64, w64 = to_np(x).astype(np.float64), to_np(w).astype(np.float64)
        assert OC.rel_l2(ref, OC.direct_f64(x64, w64)) < 1e-6


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("m", [4, 6])
def test_sweep_parity_and_superlinear_advantage(m, dtype):
    sets = S.candidate_sets(m, max_quadratic=2)
    print(f"[search] m={m} {dtype}: {len(sets)} sets", flush=True)
    rows = S.sweep(sets, m, dtype, shape=SHAPE, seed=0)
    x, w = WL.draw_inputs(*SHAPE, "halfnormal", 0)
    x, w = OF.to_dtype(x, dtype), OF.to_dtype(w, dtype)
    y64 = OC.direct_f64(x, w)
    for r in rows:
        e_or = OC.rel_l2(OC.winograd_emulated(x, w, OP.build_plan(r.moduli, n_o=m), dtype), y64)
        # the sweep's error is measured against the fp32 F(2x2) reference, itself ~1e-7 off
        assert r.rel_l2 <= 2 * e_or + 2e-7, (r.moduli, r.rel_l2, e_or)
    best_lin = min(r.rel_l2 for r in rows if "a^2" not in r.moduli)
    best_quad = min(r.rel_l2 for r in rows if "a^2" in r.moduli)
    print(f"[search] m={m} {dtype}: best linear {best_lin:.2e}, best with quadratics {best_quad:.2e} "
          f"({rows[0].moduli})", flush=True)
    assert best_quad * 2 < best_lin
    assert [r.rel_l2 for r in rows] == sorted(r.rel_l2 for r in rows)


def test_best_plan_policies():
    cands = WL.VGG_CANDIDATES
    choice, rows = S.best_plan(28, 28, 64, 64, "bf16", cands, policy="accuracy")
    assert choice == min(rows, key=lambda r: r[1])[0]
    cap = 3e-2
    fast, rows = S.best_plan(28, 28, 64, 64, "bf16", cands, policy="speed", cap=cap, time_reps=3)
    ok = [r for r in rows if r[1] <= cap]
    assert fast in [r[0] for r in ok]
    assert all(np.isfinite(r[2]) for r in rows)
    with pytest.raises(ValueError):
        S.best_plan(28, 28, 64, 64, "bf16", cands, policy="speed", cap=1e-9, time_reps=1)
