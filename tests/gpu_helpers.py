"""Shared helpers for the GPU parity tests: device transfer and the
tolerances derived from the arithmetic of eq. (2)."""
import numpy as np
import torch

from oracle import conv as OC
from oracle import fp as OF
from oracle import plan as OP
from paper_1905_05233_amd import workloads as WL

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


# Plans that reach every compiled (input tile, alpha') shape of the transform
# kernels: (moduli, m).  alpha' = m + 2 + (number of degree-2 moduli); the
# sets without infinity hold one more degree.  Tile 4 with alpha' 7 needs a
# degree-4 modulus, which plans do not take.
ALL_SHAPES = [
    (WL.F2_LINEAR, 2),                                              # t 4, alpha' 4
    ("0,a^2+1,inf", 2),                                             # t 4, alpha' 5
    ("a^2+1,a^2-2", 2),                                             # t 4, alpha' 6
    (WL.F4_LINEAR, 4),                                              # t 6, alpha' 6
    (WL.F4_A2P1, 4),                                                # t 6, alpha' 7
    ("0,a^2+1,a^2-2,inf", 4),                                       # t 6, alpha' 8
    ("a^2+1,a^2-2,a^2+2", 4),                                       # t 6, alpha' 9
    (WL.F6_LINEAR, 6),                                              # t 8, alpha' 8
    (WL.F6_ONE_A2P1, 6),                                            # t 8, alpha' 9
    (WL.F6_TWO_QUAD, 6),                                            # t 8, alpha' 10
    ("0,a^2+1,a^2-2,a^2+2,inf", 6),                                 # t 8, alpha' 11
    ("a^2+1,a^2-2,a^2+2,a^2+a+1", 6),                               # t 8, alpha' 12
    ("0,-1,1,-1/2,2,1/2,-2,-1/4,4,inf", 8),                         # t 10, alpha' 10
    ("0,-1,1,-1/2,2,1/2,-2,a^2+1,inf", 8),                          # t 10, alpha' 11
    ("0,-1,1,-1/2,2,a^2+1,a^2-2,inf", 8),                           # t 10, alpha' 12
    ("0,-1,1,a^2+1,a^2-2,a^2+2,inf", 8),                            # t 10, alpha' 13
    ("0,-1,1,-1/2,2,1/2,-2,-1/4,4,1/4,-4,inf", 10),                 # t 12, alpha' 12
    ("0,-1,1,-1/2,2,1/2,-2,-1/4,4,a^2+1,inf", 10),                  # t 12, alpha' 13
    ("0,-1,1,-1/2,2,1/2,-2,a^2+1,a^2-2,inf", 10),                   # t 12, alpha' 14
    ("0,-1,1,-1/2,2,a^2+1,a^2-2,a^2+2,inf", 10),                    # t 12, alpha' 15
    ("0,-1,1,-1/2,2,1/2,-2,-1/4,4,1/4,-4,-3/4,4/3,inf", 12),        # t 14, alpha' 14
    ("0,-1,1,-1/2,2,1/2,-2,-1/4,4,1/4,-4,a^2+1,inf", 12),           # t 14, alpha' 15
    ("0,-1,1,-1/2,2,1/2,-2,-1/4,4,a^2+1,a^2-2,inf", 12),            # t 14, alpha' 16
    # odd output tiles (separate path only): the tile sizes of Section 3.1's study
    ("0,-1,1,-1/2,inf", 3),                                         # t 5, alpha' 5
    ("0,-1,a^2+1,inf", 3),                                          # t 5, alpha' 6
    ("0,-1,1,-1/2,2,1/2,inf", 5),                                   # t 7, alpha' 7
    ("0,-1,1,-1/2,a^2+1,inf", 5),                                   # t 7, alpha' 8
    ("0,-1,1,-1/2,2,1/2,-2,-1/4,inf", 7),                           # t 9, alpha' 9
    ("0,-1,1,-1/2,2,1/2,a^2+1,inf", 7),                             # t 9, alpha' 10
]

# smallest positive value of each storage type (the spacing of its subnormals)
_TINY = {"f32": 0.0, "f16": 2.0 ** -24, "bf16": 2.0 ** -133}


def stages_on_device_layout(st):
    """The oracle's U and V in the library's layouts: U [alpha'^2][K][C],
    V [alpha'^2][T][C] with t = (n * th + ty) * tw + tx."""
    al = st["U"].shape[0]
    U = st["U"].reshape(al * al, st["U"].shape[2], st["U"].shape[3])
    V = st["V"].reshape(al * al, -1, st["V"].shape[-1])
    return U, V


def pair_bound(st, oplan, dtype, y_other, H, W, y_ref=None, sum_terms=None):
    """Element-wise bound on |y_other - y_oracle| for another evaluation of
    eq. (2) with the library's rounding points that holds the same U and V
    bit for bit (the tests check that first, stage by stage).

    The two then differ only in the fp32 channel sums of M (summation order)
    and in whatever that changes downstream:
      * each M is within 1.1 (C + 2) u32 Mabs of the exact sum, Mabs =
        sum_c |V| |U|, so |dM| <= 2.2 (C + 2) u32 Mabs;
      * the output transform (fp32 tables identical on both sides, two passes
        of alpha' fused multiply-adds) adds at most 1.1 (2 alpha' + 2) u32
        |A^T| |M| |A| per side, with |M_other| <= |M_oracle| + dM;
      * the final rounding to the storage type moves each side by at most
        u_d |y| (plus the subnormal spacing), so the two may land one unit in
        the last place apart.
    Hence |dy| <= 1.1 |A^T| (dM + 1.1 (2 alpha' + 2) u32 (2 |M| + dM)) |A|
    + 2.01 u_d max(|y_other|, |y_oracle|) + tiny, with u_d = 0 for fp32 (no
    rounding after the fp32 result).  Unlike the a-priori bound, this one is
    of the order of one unit in the last place of y in fp16 and bf16.

    ``y_ref`` replaces the oracle's y by a third evaluation with the same U
    and V (two GPU paths compared with each other): the same argument holds,
    since each path's M is within 1.1 (C + 2) u32 Mabs of the exact sum.
    ``sum_terms`` replaces C + 2 for sums of another depth (pairwise sums:
    leaf + ceil(log2 leaves) + 2).
    """
    V, U, M = st["V"], st["U"], st["M"]
    yo = st["y"] if y_ref is None else y_ref
    al = V.shape[0]
    C = V.shape[-1]
    K = U.shape[2]
    N, th, tw = V.shape[2:5]
    m = oplan.n_o
    Va = np.abs(V.reshape(al * al, -1, C).astype(np.float64))
    Ua = np.abs(U.reshape(al * al, K, C).astype(np.float64))
    Mabs = np.matmul(Va, np.transpose(Ua, (0, 2, 1)))
    Mo = np.abs(M.reshape(al * al, -1, K).astype(np.float64))
    u32 = 2.0 ** -24
    dM = 2.2 * ((C + 2) if sum_terms is None else sum_terms) * u32 * Mabs
    inner = (dM + 1.1 * (2 * al + 2) * u32 * (2 * Mo + dM)).reshape(al, al, N, th, tw, K)
    A = np.abs(np.array([[float(v) for v in r] for r in oplan.A]))
    Y = np.einsum("ao,abnxyk,bp->nxoypk", A, inner, A, optimize=True).reshape(N, th * m, tw * m, K)
    D = 1.1 * Y[:, :H, :W, :]
    ud = 0.0 if dtype == "f32" else OF.UNIT_ROUNDOFF[dtype]
    big = np.maximum(np.abs(np.asarray(yo, np.float64)), np.abs(np.asarray(y_other, np.float64)))
    return D + 2.01 * ud * big + _TINY[dtype]


def check_against_oracle(y, st, oplan, dtype, H, W, label="", sum_terms=None):
    """Assert |y - y_oracle| <= pair_bound element by element; print how
    tight the bound is (median bound / |y| and the largest error / bound)."""
    y = np.asarray(y, np.float64)
    yo = np.asarray(st["y"], np.float64)
    b = pair_bound(st, oplan, dtype, y, H, W, sum_terms=sum_terms)
    err = np.abs(y - yo)
    nz = np.abs(yo) > 0
    med = float(np.median(b[nz] / np.abs(yo[nz]))) if np.any(nz) else 0.0
    worst = float(np.max(err / np.maximum(b, 1e-300)))
    print(f"[pair-bound] {label} median bound/|y| {med:.3g}, max error/bound {worst:.3g}", flush=True)
    bad = err > b
    assert not np.any(bad), (label, int(np.sum(bad)), np.argwhere(bad)[:5].tolist())
    return med, worst


def check_layer(p, op, x, w, dtype, y_gpu, label="", st=None, sum_terms=None):
    """The GPU layer against the oracle's same-algorithm evaluation, element
    by element and tight: the plan's transform kernels (run here through
    the stage entry point that conv2d's first launch uses) give U and V equal
    to the oracle's bit for bit, and y is within ``pair_bound`` of the
    oracle's y.  Returns the oracle's stages."""
    N, H, W, C = x.shape
    if st is None:
        st = OC.winograd_emulated_stages(x, w, op, dtype)
    Ug, Vg = p.kernel_input_transform(to_dev(w, dtype), to_dev(x, dtype))
    Uo, Vo = stages_on_device_layout(st)
    assert np.array_equal(to_np(Ug)[:, :, :C], Uo, equal_nan=True), f"{label}: U differs from the oracle"
    assert np.array_equal(to_np(Vg)[:, :, :C], Vo, equal_nan=True), f"{label}: V differs from the oracle"
    check_against_oracle(y_gpu, st, op, dtype, H, W, label, sum_terms=sum_terms)
    return st


def pair_bound_1d(st, oplan, dtype, y_other, y_ref=None):
    """``pair_bound`` for the 1D path (stages of winograd1d_emulated_stages):
    the same argument with one output pass of alpha' fused multiply-adds."""
    V, U, M = st["V"], st["U"], st["M"]
    yo = st["y"] if y_ref is None else y_ref
    al, C, K = V.shape[0], V.shape[-1], U.shape[1]
    N, tl = V.shape[1:3]
    m = oplan.n_o
    Va = np.abs(V.reshape(al, -1, C).astype(np.float64))
    Ua = np.abs(U.astype(np.float64))
    Mabs = np.matmul(Va, np.transpose(Ua, (0, 2, 1)))
    Mo = np.abs(M.reshape(al, -1, K).astype(np.float64))
    u32 = 2.0 ** -24
    dM = 2.2 * (C + 2) * u32 * Mabs
    inner = (dM + 1.1 * (al + 1) * u32 * (2 * Mo + dM)).reshape(al, N, tl, K)
    A = np.abs(np.array([[float(v) for v in r] for r in oplan.A]))
    Y = np.einsum("ao,antk->ntok", A, inner, optimize=True).reshape(N, tl * m, K)
    L = np.asarray(yo).shape[1]
    D = 1.1 * Y[:, :L, :]
    ud = 0.0 if dtype == "f32" else OF.UNIT_ROUNDOFF[dtype]
    big = np.maximum(np.abs(np.asarray(yo, np.float64)), np.abs(np.asarray(y_other, np.float64)))
    return D + 2.01 * ud * big + _TINY[dtype]
