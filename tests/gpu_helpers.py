"""Shared helpers for the GPU parity tests: device transfer and the
tolerances derived from the arithmetic of eq. (2)."""
import numpy as np
import torch

from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP

TORCH = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def to_dev(a, dtype):
    """float32 numpy -> device tensor in the storage dtype (torch RNE cast)."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(TORCH[dtype]).cuda()


def to_np(t):
    return t.float().cpu().numpy()


def oracle_plan(plan_spec):
    return OP.build_plan(plan_spec.moduli, n_o=plan_spec.m, inner=plan_spec.inner)


def rounded_inputs(wl_or_arrays, dtype):
    x, w = wl_or_arrays
    return OF.to_dtype(x, dtype), OF.to_dtype(w, dtype)


def elementwise_bound(x, w, oplan, dtype, y_ref):
    """|y_hat - y_exact| <= kappa * Yabs + u_d |y| for any evaluation of eq. (2)
    with the library's rounding points (first-order analysis with margin)."""
    C = x.shape[-1]
    kappa = OC.error_bound_coefficient(oplan, C, dtype)
    return kappa * OC.abs_bound(x, w, oplan) + OF.UNIT_ROUNDOFF[dtype] * np.abs(y_ref)


def sampled_tile_check(x, w, y, oplan, dtype, tiles):
    """Check whole output tiles of a large layer against the exact convolution.

    For each sampled tile (n, ty, tx) the m x m outputs (inside the image) are
    computed in float64 directly from the (dtype-rounded) inputs, and the GPU
    values must lie within the a-priori rounding bound kappa * Yabs + u_d |y|,
    with Yabs evaluated for that tile alone.  x, w, y are float64 numpy arrays
    (NHWC, [K][3][3][C], NHWK).  Returns the largest |error| / bound seen.
    """
    N, H, W, C = x.shape
    K = w.shape[0]
    m, t = oplan.n_o, oplan.tile_in
    G = np.abs(np.array([[float(v) for v in r] for r in oplan.G]))
    A = np.abs(np.array([[float(v) for v in r] for r in oplan.A]))
    B = np.abs(np.array([[float(v) for v in r] for r in oplan.B]))
    Uabs = np.einsum("ai,kijc,bj->abkc", G, np.abs(w), G, optimize=True)
    kappa = OC.error_bound_coefficient(oplan, C, dtype)
    ud = OF.UNIT_ROUNDOFF[dtype]
    worst = 0.0
    for n, ty, tx in tiles:
        h0, w0 = ty * m - 1, tx * m - 1
        d = np.zeros((t, t, C))
        hs, ws = max(h0, 0), max(w0, 0)
        he, we = min(h0 + t, H), min(w0 + t, W)
        d[hs - h0:he - h0, ws - w0:we - w0, :] = x[n, hs:he, ws:we, :]
        exact = np.zeros((m, m, K))
        for i in range(3):
            for j in range(3):
                exact += np.einsum("opc,kc->opk", d[i:i + m, j:j + m, :], w[:, i, j, :], optimize=True)
        Vabs = np.einsum("ua,uvc,vb->abc", B, np.abs(d), B, optimize=True)
        Mabs = np.einsum("abc,abkc->abk", Vabs, Uabs, optimize=True)
        Yabs = np.einsum("ao,abk,bp->opk", A, Mabs, A, optimize=True)
        ho, wo = min(m, H - ty * m), min(m, W - tx * m)
        got = y[n, ty * m:ty * m + ho, tx * m:tx * m + wo, :]
        ex = exact[:ho, :wo]
        bound = kappa * Yabs[:ho, :wo] + ud * np.abs(ex)
        err = np.abs(got - ex)
        assert np.all(err <= bound), (n, ty, tx, float(np.max(err - bound)))
        worst = max(worst, float(np.max(err / np.maximum(bound, 1e-300))))
    return worst
