"""The wider plan family on the GPU: larger output tiles with one degree-2
modulus (alpha' = m + 3, the sweep of Section 3.2, Table 3), point sets without the
pseudo-point infinity (Table 1's zero-linear columns), a degree-3 modulus, and
layers whose channel counts span several 64-channel and 128-column blocks.

Each case checks, on seeded half-normal data, that U and V equal the
oracle's bit for bit, that every output lies within ``pair_bound`` of the
oracle's (and, in fp32, within the a-priori rounding bound of the exact
convolution), and that the rel-L2 error against fp64 direct convolution is at
most twice the oracle's same-algorithm, same-dtype error.
"""
import numpy as np
import pytest

from gpu_helpers import check_layer, elementwise_bound, to_dev, to_np
from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP
from paper_1905_05233_amd import workloads as WL

pytestmark = pytest.mark.gpu

# (moduli, m, inner points)
WIDE = [
    ("0,1,-1,1/2,-1/2,2,-2,a^2+1,inf", 8, "0,-1,inf"),                  # alpha' 11, tile 10
    ("0,1,-1,1/2,-1/2,2,-2,1/4,-4,a^2+1,inf", 10, "0,-1,inf"),          # alpha' 13, tile 12
    ("0,1,-1,1/2,-1/2,2,-2,1/4,-4,4,-1/4,a^2+1,inf", 12, "0,-1,inf"),   # alpha' 15, tile 14
    ("0,1,-1,1/2", 2, "0,-1,inf"),                                      # no infinity
    ("0,1,-1,1/2,-1/2,2", 4, "0,-1,inf"),                               # no infinity
    ("a^2+1,a^2+2", 2, "0,-1,inf"),                                     # two quadratics, no infinity
    ("0,-1,a^3+2,inf", 4, "0,-1,1,-2,inf"),                             # a degree-3 modulus
]
SHAPES = [(1, 26, 30, 24, 40), (2, 20, 18, 72, 136)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("spec,m,inner", WIDE, ids=[f"m{m}-{s}" for s, m, _ in WIDE])
def test_wide_plan_parity(spec, m, inner, dtype, shape):
    from paper_1905_05233_amd.winograd import Plan
    N, H, W, C, K = shape
    print(f"[wide] {spec} m={m} inner={inner} {dtype} {shape}", flush=True)
    x, w = WL.draw_inputs(N, H, W, C, K, "halfnormal", seed=7 * m + C)
    x, w = OF.to_dtype(x, dtype), OF.to_dtype(w, dtype)
    p = Plan(spec, m=m, dtype=dtype, inner=inner)
    op = OP.build_plan(spec, n_o=m, inner=inner)
    assert p.alpha == op.alpha
    y = to_np(p.conv2d(to_dev(x, dtype), to_dev(w, dtype))).astype(np.float64)
    y64 = OC.direct_f64(x, w)
    st = check_layer(p, op, x, w, dtype, y, label=f"wide {spec} {dtype} {shape}")
    err_gpu, err_oracle = OC.rel_l2(y, y64), OC.rel_l2(st["y"], y64)
    print(f"[wide] alpha'={op.alpha} err_gpu={err_gpu:.3e} err_oracle={err_oracle:.3e}", flush=True)
    assert np.all(np.isfinite(y))
    assert err_gpu <= 2 * err_oracle
    if dtype == "f32":
        assert np.all(np.abs(y - y64) <= elementwise_bound(x, w, op, dtype, y64))
