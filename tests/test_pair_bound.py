"""The element-wise criterion the GPU tests use (``pair_bound``), checked on
the CPU with the oracle alone.

Two evaluations of eq. (2) that share U and V bit for bit but sum the
channels of M in different orders must stay within the bound; the bound must
be of the order of one unit in the last place of y in fp16 and bf16 (not the
loose a-priori bound of the whole algorithm); and a wrong output channel in
one tile, or one output off by a fifth of its value, must break it.
"""
import numpy as np
import pytest

from gpu_helpers import pair_bound
from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP
from paper_1905_05233_amd import workloads as WL

CASES = [(WL.F4_LINEAR, 4, "f32"), (WL.F4_A2P1, 4, "f16"), (WL.F6_LINEAR, 6, "bf16"),
         (WL.F6_TWO_QUAD, 6, "bf16"), (WL.F6_ONE_A2P1, 6, "f16")]


def _second_evaluation(st, op, dtype, H, W, how):
    """Same U and V, M summed another way, then the same output transform."""
    V, U = st["V"], st["U"]
    al, C, K = V.shape[0], V.shape[-1], U.shape[2]
    Vf = V.reshape(al, al, -1, C)
    if how == "fp64":          # the exact-ish sum, rounded once
        M = np.einsum("abtc,abkc->abtk", Vf.astype(np.float64), U.astype(np.float64)).astype(np.float32)
    else:                      # fp32, channels in descending order
        M = np.zeros(Vf.shape[:3] + (K,), np.float32)
        for c in reversed(range(C)):
            M = M + Vf[..., c:c + 1] * U[:, :, None, :, c]
    M = M.reshape(st["M"].shape)
    return OC.output_transform_emulated(M, op, dtype, H, W)


@pytest.mark.parametrize("spec,m,dtype", CASES)
def test_pair_bound_holds_is_tight_and_catches_local_errors(spec, m, dtype):
    N, H, W, C, K = 1, 4 * m + 3, 3 * m + 1, 40, 24
    x, w = WL.draw_inputs(N, H, W, C, K, "halfnormal", seed=13 * m)
    x, w = OF.to_dtype(x, dtype), OF.to_dtype(w, dtype)
    op = OP.build_plan(spec, n_o=m)
    st = OC.winograd_emulated_stages(x, w, op, dtype)
    yo = st["y"].astype(np.float64)
    for how in ("fp64", "fp32-reversed"):
        y2 = _second_evaluation(st, op, dtype, H, W, how).astype(np.float64)
        b = pair_bound(st, op, dtype, y2, H, W)
        assert np.all(np.abs(y2 - yo) <= b), how
    ratio = b / np.maximum(np.abs(yo), 1e-30)
    med = float(np.median(ratio))
    # of the order of an ulp of the storage type (2 u_d = 2^-10 fp16, 2^-7 bf16)
    print(f"{spec} {dtype}: median bound/|y| {med:.3g}")
    assert med < {"f32": 2e-3, "f16": 1e-2, "bf16": 5e-2}[dtype], med
    # a wrong output channel in one tile: channel 3's values where channel 5's belong
    bad = y2.copy()
    bad[0, m:2 * m, m:2 * m, 5] = bad[0, m:2 * m, m:2 * m, 3]
    assert np.any(np.abs(bad - yo) > pair_bound(st, op, dtype, bad, H, W))
    # one output off by a fifth of its value, at an ordinary (median-ratio) element
    i = np.unravel_index(np.argsort(ratio, axis=None)[ratio.size // 2], ratio.shape)
    bad = y2.copy()
    bad[i] += 0.2 * abs(bad[i])
    assert np.abs(bad - yo)[i] > pair_bound(st, op, dtype, bad, H, W)[i]


def test_a_priori_bound_is_attained_within_a_factor_in_16_bit():
    """The a-priori bound kappa * Yabs + u_d |y| (``error_bound_coefficient``,
    ``abs_bound``) is a worst case: on one-channel, one-tile layers with
    inputs in [-2, 2] the largest error over 150 draws reaches at least 2%
    of it in fp16 and bf16 (measured 6-9%), so it is not loose by orders of
    magnitude.  It is still far above typical errors on whole layers, which
    is why the GPU tests compare with the oracle through ``pair_bound``."""
    for spec, m in ((WL.F4_LINEAR, 4), (WL.F6_TWO_QUAD, 6)):
        pl = OP.build_plan(spec, n_o=m)
        for dtype in ("f16", "bf16"):
            rng = np.random.default_rng(0)
            best = 0.0
            for _ in range(150):
                x = OF.to_dtype(rng.uniform(-2, 2, size=(1, m, m, 1)).astype(np.float32), dtype)
                w = OF.to_dtype(rng.uniform(-2, 2, size=(1, 3, 3, 1)).astype(np.float32), dtype)
                y = OC.winograd_emulated(x, w, pl, dtype).astype(np.float64)
                y64 = OC.direct_f64(x, w)
                b = OC.error_bound_coefficient(pl, 1, dtype) * OC.abs_bound(x, w, pl) \
                    + OF.UNIT_ROUNDOFF[dtype] * np.abs(y64)
                assert np.all(np.abs(y - y64) <= b)
                best = max(best, float(np.max(np.abs(y - y64) / b)))
            assert best >= 0.02, (spec, dtype, best)
