"""Convolution references (oracle; test infrastructure only).

Problem statement (Section 2.1 and eq. (2) of Barabasz & Gregg): a DNN layer
convolves each 3x3 kernel with an input that is split into overlapping tiles
(Section 2.3, following Lavin & Gray).  The layer computed here is the usual
DNN "convolution": stride 1, zero padding 1, cross-correlation (no kernel
flip), NHWC activations x[N][H][W][C], weights w[K][3][3][C], output
y[N][H][W][K] with

    y[n, h, v, k] = sum_{i, j, c} w[k, i, j, c] * x[n, h + i - 1, v + j - 1, c].

eq. (2)'s matrix-exchange form A^T [(G g G^T) (.) (B^T d B)] A computes exactly
this cross-correlation on one (m+2) x (m+2) input tile d: the 1D form is
y_j = sum_i g_i d_(i+j) because sum_xi B[k,xi] G[xi,i] A[xi,j] = [k == i + j].

Functions:

* ``direct_exact``      the definition above in exact rationals (tiny inputs);
* ``direct_f64``        the definition in float64 (9 shifted matrix products);
* ``winograd_exact``    eq. (2) tile by tile in exact rationals (tiny inputs);
* ``winograd_emulated`` eq. (2) with the rounding points of the GPU library:
  matrices rounded once to fp32; B^T d B and G g G^T as two 1D passes in fp32
  with ascending-index sums of fused multiply-adds (one rounding per term),
  then rounded to the storage dtype; the channel sum in fp32 of
  storage-dtype products; A^T M A as two such passes, rounded to the dtype;
* ``abs_bound``         the magnitude sum |A^T| sum_c (|G||g||G^T|) (.)
  (|B^T||d||B|) |A| that bounds every rounding error of the algorithm;
* ``rel_l2``            ||y - y_ref||_2 / ||y_ref||_2 in float64.
"""
from fractions import Fraction

import numpy as np

from . import fp


def _check_shapes(x_shape, w_shape):
    if len(x_shape) != 4 or len(w_shape) != 4:
        raise ValueError("x must be [N][H][W][C], w must be [K][3][3][C]")
    if tuple(w_shape[1:3]) != (3, 3) or w_shape[3] != x_shape[3]:
        raise ValueError("w must be [K][3][3][C] with the input's C")


# ---------------------------------------------------------------------------
# Direct convolution
# ---------------------------------------------------------------------------

def direct_exact(x, w):
    """Definition of the layer in exact rationals; x, w nested lists."""
    N, H, W, C = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    K = len(w)
    y = [[[[Fraction(0)] * K for _ in range(W)] for _ in range(H)] for _ in range(N)]
    for n in range(N):
        for h in range(H):
            for v in range(W):
                for k in range(K):
                    acc = Fraction(0)
                    for i in range(3):
                        for j in range(3):
                            hh, vv = h + i - 1, v + j - 1
                            if 0 <= hh < H and 0 <= vv < W:
                                for c in range(C):
                                    acc += Fraction(w[k][i][j][c]) * Fraction(x[n][hh][vv][c])
                    y[n][h][v][k] = acc
    return y


def direct_f64(x, w, chunk=4):
    """The layer in float64: 9 shifted [N*H*W x C] @ [C x K] products per chunk."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    _check_shapes(x.shape, w.shape)
    N, H, W, C = x.shape
    K = w.shape[0]
    y = np.zeros((N, H, W, K), dtype=np.float64)
    for n0 in range(0, N, chunk):
        xs = x[n0:n0 + chunk]
        xp = np.zeros((xs.shape[0], H + 2, W + 2, C), dtype=np.float64)
        xp[:, 1:H + 1, 1:W + 1, :] = xs
        acc = np.zeros((xs.shape[0], H, W, K), dtype=np.float64)
        for i in range(3):
            for j in range(3):
                acc += xp[:, i:i + H, j:j + W, :] @ w[:, i, j, :].T
        y[n0:n0 + chunk] = acc
    return y


# ---------------------------------------------------------------------------
# Tiling (Section 2.3): output tiles m x m, input tiles (m+2) x (m+2)
# ---------------------------------------------------------------------------

def tile_counts(H, W, m):
    return -(-H // m), -(-W // m)


def _padded(x, m):
    """Zero-padded input so that every tile's (m+2)^2 window is in range."""
    N, H, W, C = x.shape
    th, tw = tile_counts(H, W, m)
    xp = np.zeros((N, th * m + 2, tw * m + 2, C), dtype=x.dtype)
    xp[:, 1:H + 1, 1:W + 1, :] = x
    return xp


def _windows(x, m):
    """d[n, ty, tx, u, v, c] = x[n, ty*m - 1 + u, tx*m - 1 + v, c] (0 outside)."""
    N, H, W, C = x.shape
    t = m + 2
    th, tw = tile_counts(H, W, m)
    xp = _padded(x, m)
    d = np.empty((N, th, tw, t, t, C), dtype=x.dtype)
    for u in range(t):
        for v in range(t):
            d[:, :, :, u, v, :] = xp[:, u:u + th * m:m, v:v + tw * m:m, :]
    return d


# ---------------------------------------------------------------------------
# Winograd, exact
# ---------------------------------------------------------------------------

def winograd_exact(x, w, plan):
    """eq. (2) on every tile and channel pair, exact; x, w nested lists."""
    m, t, al = plan.n_o, plan.tile_in, plan.alpha
    if plan.n_h != 3:
        raise ValueError("the layer uses 3x3 kernels")
    G, A, B = plan.G, plan.A, plan.B
    N, H, W, C = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    K = len(w)
    th, tw = tile_counts(H, W, m)

    def xin(n, h, v, c):
        return Fraction(x[n][h][v][c]) if 0 <= h < H and 0 <= v < W else Fraction(0)

    # U[k][c] = G g G^T
    U = [[None] * C for _ in range(K)]
    for k in range(K):
        for c in range(C):
            g = [[Fraction(w[k][i][j][c]) for j in range(3)] for i in range(3)]
            Gg = [[sum((G[a][i] * g[i][j] for i in range(3)), Fraction(0)) for j in range(3)] for a in range(al)]
            U[k][c] = [[sum((Gg[a][j] * G[b][j] for j in range(3)), Fraction(0)) for b in range(al)] for a in range(al)]
    y = [[[[Fraction(0)] * K for _ in range(W)] for _ in range(H)] for _ in range(N)]
    for n in range(N):
        for ty in range(th):
            for tx in range(tw):
                Vs = []
                for c in range(C):
                    d = [[xin(n, ty * m - 1 + u, tx * m - 1 + v, c) for v in range(t)] for u in range(t)]
                    Bd = [[sum((B[u][a] * d[u][v] for u in range(t)), Fraction(0)) for v in range(t)] for a in range(al)]
                    Vs.append([[sum((Bd[a][v] * B[v][b] for v in range(t)), Fraction(0)) for b in range(al)] for a in range(al)])
                for k in range(K):
                    Mx = [[sum((U[k][c][a][b] * Vs[c][a][b] for c in range(C)), Fraction(0)) for b in range(al)] for a in range(al)]
                    AM = [[sum((A[a][o] * Mx[a][b] for a in range(al)), Fraction(0)) for b in range(al)] for o in range(m)]
                    for o1 in range(m):
                        for o2 in range(m):
                            h, v = ty * m + o1, tx * m + o2
                            if h < H and v < W:
                                y[n][h][v][k] = sum((AM[o1][b] * A[b][o2] for b in range(al)), Fraction(0))
    return y


# ---------------------------------------------------------------------------
# Winograd, same algorithm and dtype with rounding emulation
# ---------------------------------------------------------------------------

def plan_f32(plan):
    """The plan's matrices rounded once, exact rational -> fp32 RNE."""
    G = np.array([[fp.fraction_to_f32(v) for v in row] for row in plan.G], dtype=np.float32)
    A = np.array([[fp.fraction_to_f32(v) for v in row] for row in plan.A], dtype=np.float32)
    B = np.array([[fp.fraction_to_f32(v) for v in row] for row in plan.B], dtype=np.float32)
    return G, A, B


def _left(Mt, d, axis):
    """out[..., i, ...] = sum_k Mt[i, k] * d[..., k, ...] in fp32: from zero,
    ascending k, each term added by one fused multiply-add (one rounding)."""
    d = np.moveaxis(d, axis, 0)
    out = np.empty((Mt.shape[0],) + d.shape[1:], dtype=np.float32)
    for i in range(Mt.shape[0]):
        acc = np.zeros(d.shape[1:], dtype=np.float32)
        for k in range(Mt.shape[1]):
            acc = fp.fma_f32(Mt[i, k], d[k], acc)
        out[i] = acc
    return np.moveaxis(out, 0, axis)


def kernel_transform_emulated(w, plan, dtype, mats=None):
    """U[a, b, k, c] = round_dtype(G g G^T) computed in fp32 (two 1D passes)."""
    G, _, _ = mats or plan_f32(plan)
    w = np.asarray(w, dtype=np.float32)         # [K][3][3][C]
    Gg = _left(G, w, axis=1)                     # [K][al][3][C]
    U = _left(G, Gg, axis=2)                     # [K][al][al][C]
    U = fp.to_dtype(U, dtype)
    return np.ascontiguousarray(np.transpose(U, (1, 2, 0, 3)))  # [al][al][K][C]


def input_transform_emulated(x, plan, dtype, mats=None):
    """V[a, b, n, ty, tx, c] = round_dtype(B^T d B) in fp32 (columns, then rows)."""
    _, _, B = mats or plan_f32(plan)
    BT = np.ascontiguousarray(B.T)
    d = _windows(np.asarray(x, dtype=np.float32), plan.n_o)   # [N][th][tw][t][t][C]
    Bd = _left(BT, d, axis=3)                                  # [N][th][tw][al][t][C]
    V = _left(BT, Bd, axis=4)                                  # [N][th][tw][al][al][C]
    V = fp.to_dtype(V, dtype)
    return np.ascontiguousarray(np.transpose(V, (3, 4, 0, 1, 2, 5)))


def contraction_emulated(V, U):
    """M[a, b, tiles, k] = sum_c V[a, b, tiles, c] U[a, b, k, c] in fp32."""
    al = V.shape[0]
    shp = V.shape[2:-1]
    C = V.shape[-1]
    K = U.shape[2]
    Vf = V.reshape(al, al, -1, C)
    M = np.empty((al, al, Vf.shape[2], K), dtype=np.float32)
    for a in range(al):
        for b in range(al):
            M[a, b] = Vf[a, b] @ U[a, b].T
    return M.reshape((al, al) + shp + (K,))


def leaf_channels(dtype):
    """Channels per leaf of the pairwise channel sum: 64 bytes of a channel
    row (16 fp32, 32 fp16/bf16 values)."""
    return 16 if dtype == "f32" else 32


def contraction_emulated_pairwise(V, U, leaf):
    """M[a, b, tiles, k] = sum_c V U with the channels summed pairwise (the
    pairwise summation over channels that Section 4 names): leaves of
    ``leaf`` consecutive channels, each summed in fp32, then the complete
    binary tree over the leaves in channel order, the leaf list padded with
    empty leaves to a power of two (an empty subtree passes its sibling
    through unchanged), every addition rounded to fp32."""
    al = V.shape[0]
    shp = V.shape[2:-1]
    C = V.shape[-1]
    K = U.shape[2]
    Vf = V.reshape(al, al, -1, C)
    n = -(-C // leaf)
    leaves = []
    for i in range(n):
        sl = slice(i * leaf, min(C, (i + 1) * leaf))
        Mi = np.empty((al, al, Vf.shape[2], K), dtype=np.float32)
        for a in range(al):
            for b in range(al):
                Mi[a, b] = Vf[a, b, :, sl] @ U[a, b, :, sl].T
        leaves.append(Mi)
    size = 1
    while size < n:
        size *= 2
    leaves += [None] * (size - n)

    def tree(lo, hi):
        if hi - lo == 1:
            return leaves[lo]
        mid = (lo + hi) // 2
        left, right = tree(lo, mid), tree(mid, hi)
        if right is None:
            return left
        return (left + right).astype(np.float32)

    return tree(0, size).reshape((al, al) + shp + (K,))


def output_transform_emulated(M, plan, dtype, H, W, mats=None):
    """y = round_dtype(A^T M A) in fp32, cropped to H x W, NHWC."""
    _, A, _ = mats or plan_f32(plan)
    AT = np.ascontiguousarray(A.T)
    m = plan.n_o
    Z = _left(AT, M, axis=0)        # [m][al][N][th][tw][K]
    Y = _left(AT, Z, axis=1)        # [m][m][N][th][tw][K]
    Y = fp.to_dtype(Y, dtype)
    N, th, tw, K = Y.shape[2:]
    y = np.transpose(Y, (2, 3, 0, 4, 1, 5)).reshape(N, th * m, tw * m, K)
    return np.ascontiguousarray(y[:, :H, :W, :])


def winograd_emulated_stages(x, w, plan, dtype, channel_sum="mfma"):
    """Full layer by eq. (2) with the library's rounding points (see module
    doc), returning every stage: U [al][al][K][C], V [al][al][N][th][tw][C],
    M [al][al][N][th][tw][K] (fp32) and y [N][H][W][K].  ``channel_sum``
    "pairwise" sums M's channels pairwise (contraction_emulated_pairwise).

    ``x`` and ``w`` must already hold values representable in ``dtype``.
    """
    x = np.asarray(x, dtype=np.float32)
    w = np.asarray(w, dtype=np.float32)
    _check_shapes(x.shape, w.shape)
    mats = plan_f32(plan)
    U = kernel_transform_emulated(w, plan, dtype, mats)
    V = input_transform_emulated(x, plan, dtype, mats)
    if channel_sum == "pairwise":
        M = contraction_emulated_pairwise(V, U, leaf_channels(dtype))
    else:
        M = contraction_emulated(V, U)
    y = output_transform_emulated(M, plan, dtype, x.shape[1], x.shape[2], mats)
    return {"U": U, "V": V, "M": M, "y": y}


def winograd_emulated(x, w, plan, dtype):
    """Full layer by eq. (2) with the library's rounding points; y only."""
    return winograd_emulated_stages(x, w, plan, dtype)["y"]


# ---------------------------------------------------------------------------
# Error measures
# ---------------------------------------------------------------------------

def abs_bound(x, w, plan):
    """Yabs = |A^T| sum_c (|G||g||G^T|) (.) (|B^T||d||B|) |A| in float64.

    Every rounding error of the algorithm is a small multiple of the unit
    roundoff times this magnitude sum (standard dot-product error analysis).
    """
    G = np.abs(np.array([[float(v) for v in r] for r in plan.G]))
    A = np.abs(np.array([[float(v) for v in r] for r in plan.A]))
    B = np.abs(np.array([[float(v) for v in r] for r in plan.B]))
    x = np.abs(np.asarray(x, dtype=np.float64))
    w = np.abs(np.asarray(w, dtype=np.float64))
    N, H, W, C = x.shape
    m = plan.n_o
    d = _windows(x, m)                                        # [N][th][tw][t][t][C]
    V = np.einsum("ua,nxyuvc,vb->abnxyc", B, d, B, optimize=True)
    U = np.einsum("ai,kijc,bj->abkc", G, w, G, optimize=True)
    al = V.shape[0]
    Mx = np.einsum("abnxyc,abkc->abnxyk", V, U, optimize=True)
    Y = np.einsum("ao,abnxyk,bp->opnxyk", A, Mx, A, optimize=True)
    th, tw = Y.shape[3], Y.shape[4]
    K = Y.shape[-1]
    y = np.transpose(Y, (2, 3, 0, 4, 1, 5)).reshape(N, th * m, tw * m, K)
    del al
    return np.ascontiguousarray(y[:, :H, :W, :])


def error_bound_coefficient(plan, C, dtype):
    """First-order coefficient kappa with |y_hat - y| <= kappa * Yabs + u_d |y|.

    Sources (u32 = 2^-24, u_d = the storage dtype's unit roundoff, t = m + 2):
    matrix entries rounded to fp32 (2 u32 per transform), the two 1D passes of
    t (input), 3 (kernel) and alpha' (output) terms (gamma_n = n u32 each),
    the storage roundings of V and U (u_d each), fp32 products (u32) and the
    C-term fp32 channel sum (gamma_C).  A 10% margin covers second-order terms.
    """
    u32 = 2.0 ** -24
    ud = fp.UNIT_ROUNDOFF[dtype]
    t, al = plan.tile_in, plan.alpha
    k = 2 * ud + (2 * t + 2) * u32 + (2 * 3 + 2) * u32 + u32 + C * u32 + (2 * al + 2) * u32
    return 1.1 * k


def rel_l2(y, y_ref):
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    den = np.sqrt(np.sum(y_ref * y_ref))
    num = np.sqrt(np.sum((y - y_ref) ** 2))
    return float(num / den) if den > 0 else float(num)


# ---------------------------------------------------------------------------
# 1D convolution F(m, 3) (Section 2.1's polynomial product on one row;
# Section 3.1 studies its error beside the 2D form).  Layouts: x [N][L][C],
# w [K][3][C], y [N][L][K]; y[n, l, k] = sum_{j, c} w[k, j, c] x[n, l+j-1, c]
# with zero padding 1.  Output tiles of m values, input windows of m + 2
# values starting at tx*m - 1.
# ---------------------------------------------------------------------------

def _check_shapes_1d(x_shape, w_shape):
    if len(x_shape) != 3 or len(w_shape) != 3 or w_shape[1] != 3 or w_shape[2] != x_shape[2]:
        raise ValueError("x must be [N][L][C], w must be [K][3][C] with the input's C")


def direct1d_exact(x, w):
    """The 1D layer by its definition in exact rationals; nested lists."""
    N, L, C = len(x), len(x[0]), len(x[0][0])
    K = len(w)
    y = [[[Fraction(0)] * K for _ in range(L)] for _ in range(N)]
    for n in range(N):
        for l in range(L):
            for k in range(K):
                acc = Fraction(0)
                for j in range(3):
                    ll = l + j - 1
                    if 0 <= ll < L:
                        for c in range(C):
                            acc += Fraction(w[k][j][c]) * Fraction(x[n][ll][c])
                y[n][l][k] = acc
    return y


def direct1d_f64(x, w):
    """The 1D layer in float64: 3 shifted [N*L x C] @ [C x K] products."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    _check_shapes_1d(x.shape, w.shape)
    N, L, C = x.shape
    xp = np.zeros((N, L + 2, C))
    xp[:, 1:L + 1, :] = x
    y = np.zeros((N, L, w.shape[0]))
    for j in range(3):
        y += xp[:, j:j + L, :] @ w[:, j, :].T
    return y


def winograd1d_exact(x, w, plan):
    """A^T [(G g) (.) (B^T d)] on every tile and channel pair, exact."""
    m, t, al = plan.n_o, plan.tile_in, plan.alpha
    G, A, B = plan.G, plan.A, plan.B
    N, L, C = len(x), len(x[0]), len(x[0][0])
    K = len(w)
    tl = -(-L // m)
    U = [[[sum((G[a][i] * Fraction(w[k][i][c]) for i in range(3)), Fraction(0)) for a in range(al)]
          for c in range(C)] for k in range(K)]
    y = [[[Fraction(0)] * K for _ in range(L)] for _ in range(N)]
    for n in range(N):
        for tx in range(tl):
            Vs = []
            for c in range(C):
                d = [Fraction(x[n][tx * m - 1 + u][c]) if 0 <= tx * m - 1 + u < L else Fraction(0) for u in range(t)]
                Vs.append([sum((B[u][a] * d[u] for u in range(t)), Fraction(0)) for a in range(al)])
            for k in range(K):
                Mx = [sum((U[k][c][a] * Vs[c][a] for c in range(C)), Fraction(0)) for a in range(al)]
                for o in range(m):
                    if tx * m + o < L:
                        y[n][tx * m + o][k] = sum((A[a][o] * Mx[a] for a in range(al)), Fraction(0))
    return y


def winograd1d_emulated_stages(x, w, plan, dtype):
    """The 1D layer with the library's rounding points: U = G g and V = B^T d
    as one fp32 pass each (ascending index, fused multiply-adds), rounded to
    the dtype; M the fp32 channel sum; y = A^T M in one fp32 pass, rounded to
    the dtype.  Returns U [al][K][C], V [al][N][tl][C], M [al][N][tl][K] and
    y [N][L][K]."""
    x = np.asarray(x, dtype=np.float32)
    w = np.asarray(w, dtype=np.float32)
    _check_shapes_1d(x.shape, w.shape)
    G, A, B = plan_f32(plan)
    m, t = plan.n_o, plan.tile_in
    N, L, C = x.shape
    tl = -(-L // m)
    U = fp.to_dtype(_left(G, np.transpose(w, (1, 0, 2)), axis=0), dtype)           # [al][K][C]
    xp = np.zeros((N, tl * m + 2, C), dtype=np.float32)
    xp[:, 1:L + 1, :] = x
    d = np.empty((t, N, tl, C), dtype=np.float32)
    for u in range(t):
        d[u] = xp[:, u:u + tl * m:m, :]
    V = fp.to_dtype(_left(np.ascontiguousarray(B.T), d, axis=0), dtype)             # [al][N][tl][C]
    al = V.shape[0]
    M = np.empty((al, N, tl, w.shape[0]), dtype=np.float32)
    for a in range(al):
        M[a] = V[a] @ U[a].T
    Y = fp.to_dtype(_left(np.ascontiguousarray(A.T), M, axis=0), dtype)             # [m][N][tl][K]
    y = np.transpose(Y, (1, 2, 0, 3)).reshape(N, tl * m, -1)[:, :L, :]
    return {"U": U, "V": V, "M": M, "y": np.ascontiguousarray(y)}


def winograd1d_emulated(x, w, plan, dtype):
    return winograd1d_emulated_stages(x, w, plan, dtype)["y"]
