"""Polynomial-set search on the GPU.

Section 3.1 of Barabasz & Gregg (arXiv 1905.05233) compares the floating-point
error of Winograd convolutions built from different modulus sets, on random
data, against the ratio alpha'^2 / m^2 of multiplications per output; and it
picks, for each CNN layer, the plan that suits it.  This module runs both on
the library's own kernels:

* ``candidate_sets(m)`` enumerates modulus sets for F(m x m, 3 x 3): the first
  linear points of a fixed list of well-conditioned points (0, -1, 1, -1/2, 2,
  1/2, -2, ...), plus up to ``max_quadratic`` irreducible quadratics, plus the
  pseudo-point infinity, with degrees summing to m + r - 1 (Algorithms 1 and 2, Table 1).
* ``sweep(...)`` convolves one seeded synthetic layer with every set and ranks
  them by relative L2 error.  The reference is the same layer, on the same
  dtype-rounded inputs, computed in fp32 by the F(2 x 2, 3 x 3) plan on points
  {0, 1, -1, inf}, whose own error on such data is about 1e-7 (the test suite
  pins it against fp64 direct convolution) -- far below the 1e-6 .. 1e-1
  errors being ranked.  Everything, reference included, runs through the
  library on the GPU; torch only holds memory and reduces the error norms.
* ``best_plan(...)`` picks a plan for a layer shape: the most accurate
  candidate, or the fastest one whose error stays within a cap.
"""
import itertools
from dataclasses import dataclass
from fractions import Fraction

import numpy as np
import torch

from .winograd import Plan
from .workloads import F2_LINEAR, INNER_DEFAULT, PlanSpec, draw_inputs

# linear points in the order the paper's experiments add them (small
# magnitudes and their reciprocals first)
LINEAR_POINTS = ("0", "-1", "1", "-1/2", "2", "1/2", "-2", "-1/4", "4", "1/4", "-4", "-3/4", "4/3")
# irreducible over Q, pairwise coprime
QUADRATICS = ("a^2+1", "a^2-2", "a^2+2", "a^2+a+1", "a^2-a+1")

TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def candidate_sets(m, max_quadratic=2, with_inf=True, quadratics=QUADRATICS, r=3):
    """Modulus-set spec strings for F(m x m, r x r), fewest quadratics first."""
    need = m + r - 1 - (1 if with_inf else 0)   # finite degree sum
    out = []
    for q in range(0, max_quadratic + 1):
        n_lin = need - 2 * q
        if n_lin < 0 or n_lin > len(LINEAR_POINTS):
            continue
        for quads in itertools.combinations(quadratics, q):
            parts = list(LINEAR_POINTS[:n_lin]) + list(quads) + (["inf"] if with_inf else [])
            out.append(",".join(parts))
    return out


@dataclass
class SweepResult:
    moduli: str
    m: int
    alpha: int
    ratio: Fraction
    rel_l2: float
    us: float = float("nan")


def _rel_l2(y, ref):
    d = (y.double() - ref.double()).pow(2).sum().sqrt()
    return float(d / ref.double().pow(2).sum().sqrt())


def _time_us(fn, reps):
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return 1e3 * e0.elapsed_time(e1) / reps


def layer_inputs(N, H, W, C, K, dtype, seed=0, x_dist="halfnormal", device="cuda"):
    """Seeded layer inputs rounded to ``dtype`` on the device."""
    x, w = draw_inputs(N, H, W, C, K, x_dist, seed)
    td = TORCH_DTYPES[dtype]
    return (torch.from_numpy(x).to(device).to(td), torch.from_numpy(w).to(device).to(td))


def reference(x, w):
    """The fp32 F(2x2,3x3) result on the same (already rounded) inputs."""
    return Plan(F2_LINEAR, m=2, dtype="f32").conv2d(x.float().contiguous(), w.float().contiguous())


def sweep(sets, m, dtype, shape=(1, 32, 32, 64, 64), seed=0, inner=INNER_DEFAULT, time_reps=0):
    """Rank modulus sets for F(m x m, 3 x 3) by error on one seeded layer.

    ``sets`` are spec strings; ``shape`` is (N, H, W, C, K).  Returns
    SweepResult records sorted by rel_l2 (most accurate first); with
    ``time_reps`` > 0 each record also carries the mean conv2d time in us.
    """
    x, w = layer_inputs(*shape, dtype=dtype, seed=seed)
    ref = reference(x, w)
    out = []
    for spec in sets:
        p = Plan(spec, m=m, dtype=dtype, inner=inner)
        y = p.conv2d(x, w)
        rec = SweepResult(spec, m, p.alpha, p.ratio, _rel_l2(y, ref))
        if time_reps:
            rec.us = _time_us(lambda: p.conv2d(x, w, y=y), time_reps)
        out.append(rec)
        p.close()
    out.sort(key=lambda r: r.rel_l2)
    return out


def best_plan(H, W, C, K, dtype, candidates, policy="accuracy", cap=None, seed=0, sample_hw=32, time_reps=5):
    """Choose a plan for a layer of shape (H, W, C, K).

    Every candidate (a PlanSpec) is run on one seeded image of the layer's
    channel counts, cropped to at most ``sample_hw`` pixels a side.  Policy
    ``accuracy`` returns the most accurate candidate; ``speed`` the fastest
    (timed at the full layer size, N = 1) among those whose error is at most
    ``cap``.  Returns (PlanSpec, list of (PlanSpec, rel_l2, us)).
    """
    if policy not in ("accuracy", "speed"):
        raise ValueError("policy must be 'accuracy' or 'speed'")
    hs, ws = min(H, sample_hw), min(W, sample_hw)
    x, w = layer_inputs(1, hs, ws, C, K, dtype, seed=seed)
    ref = reference(x, w)
    rows = []
    for cand in candidates:
        p = Plan(cand.moduli, m=cand.m, dtype=dtype, inner=cand.inner)
        err = _rel_l2(p.conv2d(x, w), ref)
        us = float("nan")
        if policy == "speed":
            xf, wf = layer_inputs(1, H, W, C, K, dtype, seed=seed)
            yf = p.conv2d(xf, wf)
            us = _time_us(lambda: p.conv2d(xf, wf, y=yf), time_reps)
        rows.append((cand, err, us))
        p.close()
    if policy == "accuracy":
        return min(rows, key=lambda r: r[1])[0], rows
    ok = [r for r in rows if cap is None or r[1] <= cap]
    if not ok:
        raise ValueError("no candidate meets the error cap")
    return min(ok, key=lambda r: r[2])[0], rows


def spec_of(moduli, m, inner=INNER_DEFAULT):
    return PlanSpec(moduli, m, inner)


def _main(argv=None):
    import argparse
    ap = argparse.ArgumentParser(description="error-versus-ratio sweep of modulus sets on the GPU")
    ap.add_argument("--m", type=int, default=4)
    ap.add_argument("--dtype", default="f32", choices=sorted(TORCH_DTYPES))
    ap.add_argument("--max-quadratic", type=int, default=2)
    ap.add_argument("--shape", default="1,32,32,64,64", help="N,H,W,C,K")
    ap.add_argument("--time-reps", type=int, default=0)
    a = ap.parse_args(argv)
    shape = tuple(int(v) for v in a.shape.split(","))
    rows = sweep(candidate_sets(a.m, a.max_quadratic), a.m, a.dtype, shape, time_reps=a.time_reps)
    for r in rows:
        t = "" if np.isnan(r.us) else f"  {r.us:8.2f} us"
        print(f"{r.rel_l2:10.3e}  alpha'={r.alpha:2d}  ratio={float(r.ratio):5.3f}  {r.moduli}{t}")


if __name__ == "__main__":
    _main()
