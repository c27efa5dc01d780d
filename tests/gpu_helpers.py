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
