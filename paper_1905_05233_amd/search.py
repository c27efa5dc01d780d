"""Polynomial-set search on the GPU: the random-data error study of Section
3.1 of Barabasz & Gregg (arXiv 1905.05233) and the choice of a plan per CNN
layer.

Every error here is measured against a float64 direct convolution of the
same (storage-rounded) inputs computed by the library's own float64 kernel
(``layer_ops.direct_conv_f64``), never against another Winograd result; the
error sums are reduced on the device.

* ``candidate_sets(m)`` enumerates modulus sets for F(m, 3): the first linear
  points of the paper's list of good points (0, -1, 1, -1/2, 2, 1/2, -2,
  -1/4, 4, then 1/4, -4, -3/4, 4/3 where more are needed), plus up to
  ``max_quadratic`` degree-2 moduli and the pseudo-point infinity, degrees
  summing to m + r - 1 (Algorithms 1 and 2, Table 1).  Section 3.1 considers
  the quadratics with coefficients in {0, -1, 1} that are coprime with the
  linear ones: a^2 + 1, a^2 + a + 1 and a^2 - a + 1.
* ``x1_experiment(...)`` is the study itself: for output tiles m = 2 .. 8, in
  1D and 2D, every candidate set is run on ``loops`` random convolutions of
  one tile with one 3-tap (3x3) kernel, inputs and kernels drawn from the
  standard normal distribution restricted to (-1, 1), and its error against
  float64 direct convolution is recorded; ``best_per_ratio`` keeps the most
  accurate set for each ratio of multiplications per output and each number
  of quadratic moduli, as the paper's Figure 3 plots them.
* ``sweep(...)`` ranks sets on seeded CNN-layer-shaped data, averaged over
  several draws.
* ``best_plan(...)`` picks a plan for a layer from its own input: the most
  accurate candidate (ties within 1% go to the lower ratio), or the fastest
  one within an error cap.
"""
import itertools
import math
from dataclasses import dataclass
from fractions import Fraction

import numpy as np
import torch

from . import layer_ops
from .winograd import Plan
from .workloads import INNER_DEFAULT, PlanSpec, draw_inputs

# linear points in the order of Section 3.1's list of good points, then more
# of the same kind for the largest tiles
LINEAR_POINTS = ("0", "-1", "1", "-1/2", "2", "1/2", "-2", "-1/4", "4", "1/4", "-4", "-3/4", "4/3")
# the degree-2 moduli Section 3.1 considers
QUADRATICS_X1 = ("a^2+1", "a^2+a+1", "a^2-a+1")
# a wider list for the per-layer search (irreducible over Q, pairwise coprime)
QUADRATICS = ("a^2+1", "a^2-2", "a^2+2", "a^2+a+1", "a^2-a+1")

TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def candidate_sets(m, max_quadratic=2, with_inf=True, quadratics=QUADRATICS, r=3):
    """Modulus-set spec strings for F(m, r), fewest quadratics first."""
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


def n_quadratics(spec):
    return sum(1 for s in spec.split(",") if "a^2" in s)


@dataclass
class SweepResult:
    moduli: str
    m: int
    alpha: int
    ratio: Fraction
    rel_l2: float
    us: float = float("nan")
    dims: int = 2
    tile_l2: float = float("nan")   # mean Euclidean error of one output tile

    @property
    def quadratics(self):
        return n_quadratics(self.moduli)


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
    """float64 direct convolution of the (already rounded) inputs, on the GPU."""
    return layer_ops.direct_conv_f64(x, w)


def sweep(sets, m, dtype, shape=(1, 32, 32, 64, 64), seeds=(0, 1, 2), inner=INNER_DEFAULT, time_reps=0):
    """Rank modulus sets for F(m x m, 3 x 3) by the relative L2 error against
    float64 direct convolution, pooled over one seeded layer per seed
    (sqrt of the summed squared errors over the summed squared references).

    ``sets`` are spec strings; ``shape`` is (N, H, W, C, K).  Returns
    SweepResult records sorted by rel_l2 (most accurate first); with
    ``time_reps`` > 0 each record also carries the mean conv2d time in us.
    """
    draws = []
    for s in seeds:
        x, w = layer_inputs(*shape, dtype=dtype, seed=s)
        draws.append((x, w, reference(x, w)))
    out = []
    for spec in sets:
        p = Plan(spec, m=m, dtype=dtype, inner=inner)
        e2 = r2 = 0.0
        for x, w, ref in draws:
            a, b = layer_ops.error_sums(p.conv2d(x, w), ref)
            e2, r2 = e2 + a, r2 + b
        rec = SweepResult(spec, m, p.alpha, p.ratio, math.sqrt(e2 / r2))
        if time_reps:
            x, w, _ = draws[0]
            y = p.conv2d(x, w)
            rec.us = _time_us(lambda: p.conv2d(x, w, y=y), time_reps)
        out.append(rec)
        p.close()
    out.sort(key=lambda r: r.rel_l2)
    return out


def x1_inputs(dims, m, loops, dtype, seed, kernels=8, tiles_per_side=8):
    """The random convolutions of the Section 3.1 study as one layer: C = 1
    channel, ``kernels`` output channels (one random kernel each) and enough
    images of ``tiles_per_side`` tiles a side (a row of as many tiles in 1D)
    for at least ``loops`` (tile, kernel) convolutions.  Values ~ N(0, 1)
    restricted to (-1, 1), rounded to ``dtype``.  Returns x, w on the device
    (1D: x [N][1][L][1], w [K][1][3][1])."""
    side = m * tiles_per_side
    per_image = (tiles_per_side ** dims) * kernels
    N = max(1, -(-loops // per_image))
    H = side if dims == 2 else 1
    x, w = draw_inputs(N, H, side, 1, kernels, "normal_clip1", seed)
    if dims == 1:
        w = w[:, 1:2]                                # [K][1][3][1]: one row of taps
    td = TORCH_DTYPES[dtype]
    return torch.from_numpy(np.ascontiguousarray(x)).cuda().to(td), \
        torch.from_numpy(np.ascontiguousarray(w)).cuda().to(td)


def x1_experiment(dims=2, m_values=range(2, 9), dtype="f32", loops=5000, max_quadratic=1,
                  quadratics=QUADRATICS_X1, seed=0, inner=INNER_DEFAULT):
    """Section 3.1's random-data study.  For each output tile m and each
    candidate set, the error of ``loops`` random one-tile convolutions
    (``x1_inputs``) against float64 direct convolution: ``rel_l2`` pooled over
    all of them and ``tile_l2`` the root mean square Euclidean error of one
    output tile.  Returns SweepResult records (``dims`` 1 or 2)."""
    out = []
    for m in m_values:
        x, w = x1_inputs(dims, m, loops, dtype, seed + m)
        ref = reference(x, w)
        tiles = x.shape[0] * (x.shape[1] // m if dims == 2 else 1) * (x.shape[2] // m) * w.shape[0]
        for spec in candidate_sets(m, max_quadratic, quadratics=quadratics):
            p = Plan(spec, m=m, dtype=dtype, inner=inner)
            if dims == 2:
                y = p.conv2d(x, w)
                ratio = p.ratio
            else:
                y = p.conv1d(x[:, 0], w[:, 0]).unsqueeze(1)
                ratio = Fraction(p.alpha, p.m)
            e2, r2 = layer_ops.error_sums(y, ref)
            out.append(SweepResult(spec, m, p.alpha, ratio, math.sqrt(e2 / r2), dims=dims,
                                   tile_l2=math.sqrt(e2 / tiles)))
            p.close()
    return out


def best_per_ratio(records):
    """{(ratio, number of quadratics): the most accurate record}."""
    best = {}
    for r in records:
        key = (r.ratio, r.quadratics)
        if key not in best or r.rel_l2 < best[key].rel_l2:
            best[key] = r
    return best


def best_plan(x, w, candidates, policy="accuracy", cap=None, time_reps=5, x_full=None):
    """Choose a plan for a layer from its own input.

    ``x`` (a few images of the layer's input, NHWC) and ``w`` are device
    tensors in the storage dtype.  Each candidate (a PlanSpec) convolves them
    and is scored by its relative L2 error against the float64 direct
    convolution of the same tensors.  Policy ``accuracy`` returns the most
    accurate candidate, ties within 1% going to the lower ratio; ``speed`` the
    fastest (timed on ``x_full`` if given, else on ``x``) among those whose
    error is at most ``cap``.  Returns (PlanSpec, list of (PlanSpec, rel_l2, us)).
    """
    if policy not in ("accuracy", "speed"):
        raise ValueError("policy must be 'accuracy' or 'speed'")
    dtype = {v: k for k, v in TORCH_DTYPES.items()}[x.dtype]
    ref = reference(x, w)
    rows = []
    for cand in candidates:
        p = Plan(cand.moduli, m=cand.m, dtype=dtype, inner=cand.inner)
        err = layer_ops.rel_l2(p.conv2d(x, w), ref)
        us = float("nan")
        if policy == "speed":
            xt = x if x_full is None else x_full
            yt = p.conv2d(xt, w)
            us = _time_us(lambda: p.conv2d(xt, w, y=yt), time_reps)
        rows.append((cand, err, us, p.ratio))
        p.close()
    if policy == "accuracy":
        lo = min(r[1] for r in rows)
        near = [r for r in rows if r[1] <= 1.01 * lo]
        pick = min(near, key=lambda r: (r[3], r[1]))[0]
        return pick, [r[:3] for r in rows]
    ok = [r for r in rows if cap is None or r[1] <= cap]
    if not ok:
        raise ValueError("no candidate meets the error cap")
    return min(ok, key=lambda r: r[2])[0], [r[:3] for r in rows]


def spec_of(moduli, m, inner=INNER_DEFAULT):
    return PlanSpec(moduli, m, inner)


def _main(argv=None):
    import argparse
    ap = argparse.ArgumentParser(description="the random-data error study of Section 3.1 on the GPU")
    ap.add_argument("--dims", type=int, default=2, choices=(1, 2))
    ap.add_argument("--m", default="2,3,4,5,6,7,8", help="output tile sizes")
    ap.add_argument("--dtype", default="f32", choices=sorted(TORCH_DTYPES))
    ap.add_argument("--loops", type=int, default=5000)
    ap.add_argument("--max-quadratic", type=int, default=1)
    a = ap.parse_args(argv)
    recs = x1_experiment(a.dims, [int(v) for v in a.m.split(",")], a.dtype, a.loops, a.max_quadratic)
    for (ratio, q), r in sorted(best_per_ratio(recs).items(), key=lambda kv: (kv[0][0], kv[0][1])):
        print(f"ratio {float(ratio):6.3f}  quadratics {q}  m={r.m:2d}  alpha'={r.alpha:2d}  rel-L2 {r.rel_l2:10.3e}  "
              f"tile L2 {r.tile_l2:10.3e}  {{{r.moduli}}}")


if __name__ == "__main__":
    _main()
