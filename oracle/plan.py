"""Exact Winograd transform construction by the polynomial CRT (oracle; test
infrastructure only).

Follows Section 2 of Barabasz & Gregg (arXiv 1905.05233):

* eq. (1): s(a) = sum_i s_i(a) N_i(a) M_i(a) mod M(a), with M = prod m_i,
  M_i = M / m_i and N_i M_i + n_i m_i = 1 from the extended Euclidean algorithm;
* Algorithm 1: the kernel and Hadamard-result transforms G^W (alpha' x n_h) and
  A^W (alpha' x n_o).  A linear modulus a - p contributes the Toom-Cook rows
  [p^0 .. p^(n_h-1)] and [p^0 .. p^(n_o-1)]; a degree-d modulus contributes
  G^(T-C) G' and A^(T-C) A', where G', A' map into the "polynomials' Winograd
  domain" (columns vec(R_m[a^k])) and G^(T-C), A^(T-C) belong to the inner
  Toom-Cook algorithm F_T-C(d x d, d x d); the pseudo-point infinity adds the
  rows [0 .. 0 1];
* Algorithm 2: the input transform B^W = [E C | vec(M)], with C block-diagonal
  (a linear modulus gives [1], a degree-d modulus gives the columns
  vec(R_m[b_j]) of the inner B^(T-C)) and E_i = [vec(R_M[a^k N_i M_i])]_{k<d},
  stacked over a zero row;
* Section 2.3 / Table 1: the number of elementwise multiplications per output
  point, ratio = alpha'^2 / n_o^2.

Readings where the paper is silent or garbled (each is listed in the design
notes of the repository):

* The inner Toom-Cook algorithm uses the scaling the worked example shows
  (Section 2.2): its G^(T-C) rows carry the Lagrange factor N_q, its A^(T-C)
  rows are plain powers, its B^(T-C) columns are vec(M_in / (a - q)) and, for
  the pseudo-point, vec(M_in).  The outer linear rows are not scaled (the
  outer N_i live in B^W through E), as the paper states.
* The worked example prints A_2 and A^W with four columns although n_o = 2;
  Algorithm 1 is followed (A' has n_o columns).
* The printed N_1 = 1, N_2 = -a (and hence E, EC, B^W of the example) hold only
  for b = 0, c = 1; N_i is always computed by the extended Euclidean algorithm.
* Degree rule: with the pseudo-point, sum(deg m_i) = n_h + n_o - 2
  (Algorithms 1 and 2); without it, sum(deg m_i) = n_h + n_o - 1, which is what
  Table 1's all-quadratic columns require.  Then E has no zero row and
  B^W = E C.
* Domain row order: modulus list order, 2d - 1 rows per degree-d modulus in
  inner-point order, the pseudo-point last.
* Moduli are made monic; they must be irreducible and pairwise coprime
  (Section 2.1).

Option (an accuracy variant the paper's related work names as complementary, Section 4):
``factors="G"`` moves each CRT factor N_i from the input side to the kernel
side.  Eq. (1) multiplies the residue product s_i = (g d) mod m_i by N_i; since
(N_i g mod m_i)(d mod m_i) = N_i g d (mod m_i), the factor may multiply the
kernel residue instead: G' gets the columns vec(R_m[N_i a^k]) (for a linear
modulus the row [p^0 .. p^(r-1)] times the scalar N_i(p)) and E the columns
vec(R_M[a^k M_i]).  The exact algorithm is unchanged; the rounding is not.
"""
from dataclasses import dataclass, field
from fractions import Fraction

from . import polynomials as P

INF = "inf"


# ---------------------------------------------------------------------------
# Modulus-set parsing
# ---------------------------------------------------------------------------

def parse_modulus(item):
    """One modulus: ``inf``, a point p (meaning a - p), a polynomial in a given
    as text, or a coefficient tuple (low to high)."""
    if isinstance(item, tuple):
        return P.monic(P.poly(item))
    s = str(item).strip()
    if s.lower() in ("inf", "infinity", "∞"):
        return INF
    if "a" in s:
        return P.monic(P.parse(s))
    p = Fraction(s)
    return P.poly([-p, 1])


def parse_modulus_set(spec):
    """``"0,1,-1,a^2+1,inf"`` -> (list of monic finite moduli, has_inf)."""
    items = spec.split(",") if isinstance(spec, str) else list(spec)
    finite, has_inf = [], False
    for it in items:
        m = parse_modulus(it)
        if m == INF:
            if has_inf:
                raise ValueError("pseudo-point infinity given twice")
            has_inf = True
        else:
            finite.append(m)
    return finite, has_inf


def parse_points(spec):
    """Inner Toom-Cook points, e.g. ``"0,-1,inf"`` -> (finite points, has_inf)."""
    items = spec.split(",") if isinstance(spec, str) else list(spec)
    pts, has_inf = [], False
    for it in items:
        s = str(it).strip()
        if s.lower() in ("inf", "infinity", "∞"):
            has_inf = True
        else:
            pts.append(Fraction(s))
    return pts, has_inf


# ---------------------------------------------------------------------------
# Validity (Section 2.1: irreducible, pairwise coprime moduli)
# ---------------------------------------------------------------------------

def _rational_roots(p):
    """All rational roots of p (rational root theorem); p has rational coeffs."""
    from math import gcd
    den = 1
    for c in p:
        den = den * c.denominator // gcd(den, c.denominator)
    ints = [int(c * den) for c in p]
    # strip a factor a^k (root 0)
    roots = set()
    k = 0
    while ints and ints[0] == 0:
        ints.pop(0)
        k += 1
    if k:
        roots.add(Fraction(0))
    if len(ints) <= 1:
        return roots

    def divisors(n):
        n = abs(n)
        return [d for d in range(1, n + 1) if n % d == 0]

    for pn in divisors(ints[0]):
        for qd in divisors(ints[-1]):
            for sgn in (1, -1):
                cand = Fraction(sgn * pn, qd)
                if P.evaluate(p, cand) == 0:
                    roots.add(cand)
    return roots


def is_irreducible(m):
    d = P.deg(m)
    if d <= 0:
        return False
    if d == 1:
        return True
    if d == 2:
        c0, c1, c2 = m
        return not P.is_square_rational(c1 * c1 - 4 * c0 * c2)
    if d == 3:
        return not _rational_roots(m)
    raise NotImplementedError("irreducibility is only decided for degree <= 3")


# ---------------------------------------------------------------------------
# Inner Toom-Cook algorithm F_T-C(d x d, d x d) for a degree-d modulus
# ---------------------------------------------------------------------------

@dataclass
class ToomCook:
    G: list  # (2d-1) x d
    A: list  # (2d-1) x d
    B: list  # (2d-1) x (2d-1); columns are the reconstruction polynomials


def inner_toom_cook(d, points, with_inf):
    """F_T-C(d x d, d x d): product of two degree-(d-1) polynomials, 2d-1 mults.

    ``points`` are the finite evaluation points in order; with the pseudo-point
    2d-2 of them are used, without it 2d-1.  Row order: the finite points, then
    infinity.  Scaling as in the paper's worked example: G rows carry N_q.
    """
    nfin = 2 * d - 1 - (1 if with_inf else 0)
    if len(points) < nfin:
        raise ValueError(f"a degree-{d} modulus needs {nfin} finite inner points")
    pts = list(points[:nfin])
    if len(set(pts)) != len(pts):
        raise ValueError("inner points must be distinct")
    M_in = P.product([P.poly([-q, 1]) for q in pts])
    L = 2 * d - 1
    G, A, Bcols = [], [], []
    for q in pts:
        lin = P.poly([-q, 1])
        Mq = P.exact_div(M_in, lin)
        Nq = P.inverse_mod(Mq, lin)           # a constant: 1 / Mq(q)
        nq = Nq[0] if Nq else Fraction(0)
        G.append([nq * q ** k for k in range(d)])
        A.append([q ** k for k in range(d)])
        Bcols.append(P.vec(Mq, L))
    if with_inf:
        G.append([Fraction(0)] * (d - 1) + [Fraction(1)])
        A.append([Fraction(0)] * (d - 1) + [Fraction(1)])
        Bcols.append(P.vec(M_in, L))
    B = [[Bcols[j][k] for j in range(L)] for k in range(L)]
    return ToomCook(G=G, A=A, B=B)


# ---------------------------------------------------------------------------
# Algorithms 1 and 2
# ---------------------------------------------------------------------------

def _matmul(X, Y):
    return [[sum((X[i][k] * Y[k][j] for k in range(len(Y))), Fraction(0))
             for j in range(len(Y[0]))] for i in range(len(X))]


@dataclass
class ExactPlan:
    n_o: int
    n_h: int
    moduli: list            # monic finite moduli, in order
    has_inf: bool
    inner_points: list
    inner_inf: bool
    G: list = field(default_factory=list)     # alpha' x n_h
    A: list = field(default_factory=list)     # alpha' x n_o
    B: list = field(default_factory=list)     # (n+1) x alpha'
    C: list = field(default_factory=list)
    E: list = field(default_factory=list)
    N: list = field(default_factory=list)     # N_i polynomials
    M: tuple = ()
    Mi: list = field(default_factory=list)
    blocks: list = field(default_factory=list)  # per modulus: dict of G_i, A_i, C_i, E_i

    @property
    def alpha(self):
        return len(self.G)

    @property
    def n(self):
        return self.n_h + self.n_o - 2

    @property
    def tile_in(self):
        return self.n + 1

    @property
    def ratio(self):
        return Fraction(self.alpha ** 2, self.n_o ** 2)

    @property
    def BT(self):
        return [list(r) for r in zip(*self.B)]


def residue_map(m, ncols, factor=None):
    """[vec(R_m[f a^0]) ... vec(R_m[f a^(ncols-1)])]: deg(m) x ncols
    (Algorithm 1's G' and A' with f = 1; f = N_i moves the CRT factor)."""
    d = P.deg(m)
    f = P.ONE if factor is None else factor
    cols = [P.vec(P.rem(P.mul(f, P.power_of_a(k)), m), d) for k in range(ncols)]
    return [[cols[j][i] for j in range(ncols)] for i in range(d)]


def build_plan(moduli_spec, n_o, n_h=3, inner="0,-1,inf", factors="B", scaling="none"):
    """Build G^W, A^W, B^W exactly for F(n_o, n_h) from a modulus set.

    ``factors`` places the CRT factors N_i: "B" (the paper's matrices, inside
    E) or "G" (multiplying the kernel residues).  ``scaling`` "l1" applies the
    diagonal scaling of G and A^T that Section 4 cites (Vincent et al.): each
    domain row of G and of A divided by its 1-norm, B's column multiplied by
    both, which leaves every domain row's rank-1 term unchanged."""
    if factors not in ("B", "G"):
        raise ValueError("factors must be 'B' or 'G'")
    if scaling not in ("none", "l1"):
        raise ValueError("scaling must be 'none' or 'l1'")
    finite, has_inf = parse_modulus_set(moduli_spec)
    inner_pts, inner_inf = parse_points(inner)
    n = n_h + n_o - 2
    if n_o < 1 or n_h < 1:
        raise ValueError("sizes must be positive")
    if not finite:
        raise ValueError("at least one finite modulus is needed")
    degsum = sum(P.deg(m) for m in finite)
    want = n if has_inf else n + 1
    if degsum != want:
        raise ValueError(f"sum of degrees is {degsum}, F({n_o},{n_h}) needs {want}")
    for m in finite:
        if not is_irreducible(m):
            raise ValueError(f"modulus {m} is reducible")
    for i in range(len(finite)):
        for j in range(i + 1, len(finite)):
            g, _, _ = P.ext_euclid(finite[i], finite[j])
            if g != P.ONE:
                raise ValueError("moduli are not pairwise coprime")

    plan = ExactPlan(n_o=n_o, n_h=n_h, moduli=finite, has_inf=has_inf,
                     inner_points=inner_pts, inner_inf=inner_inf)

    # CRT factors of eq. (1): M = prod m_i, M_i = M / m_i, N_i M_i = 1 mod m_i
    Mpoly = P.product(finite)
    Mi = [P.exact_div(Mpoly, m) for m in finite]
    N = [P.inverse_mod(Mi_, m) for m, Mi_ in zip(finite, Mi)]

    # ---- Algorithm 1: G^W and A^W -----------------------------------------
    G, A, blocks = [], [], []
    for m, Ni in zip(finite, N):
        d = P.deg(m)
        blk = {"m": m, "d": d}
        kf = Ni if factors == "G" else None
        if d == 1:
            p = -m[0]                      # root of the monic a - p
            s_ = Ni[0] if factors == "G" else Fraction(1)   # N_i is the constant 1 / M_i(p)
            Gi = [[s_ * p ** k for k in range(n_h)]]
            Ai = [[p ** k for k in range(n_o)]]
        else:
            tc = inner_toom_cook(d, inner_pts, inner_inf)
            Gp = residue_map(m, n_h, kf)  # G'
            Ap = residue_map(m, n_o)      # A'
            Gi = _matmul(tc.G, Gp)
            Ai = _matmul(tc.A, Ap)
            blk.update(tc=tc, Gp=Gp, Ap=Ap)
        blk.update(G=Gi, A=Ai)
        G.extend(Gi)
        A.extend(Ai)
        blocks.append(blk)
    if has_inf:
        G.append([Fraction(0)] * (n_h - 1) + [Fraction(1)])
        A.append([Fraction(0)] * (n_o - 1) + [Fraction(1)])

    # ---- Algorithm 2: B^W = [E C | vec(M)] -------------------------------
    # block-diagonal C
    Cblocks = []
    for blk in blocks:
        d = blk["d"]
        if d == 1:
            Ci = [[Fraction(1)]]
        else:
            Btc = blk["tc"].B
            L = 2 * d - 1
            cols = []
            for j in range(L):
                bj = P.poly([Btc[k][j] for k in range(L)])
                cols.append(P.vec(P.rem(bj, blk["m"]), d))
            Ci = [[cols[j][i] for j in range(L)] for i in range(d)]
        blk["C"] = Ci
        Cblocks.append(Ci)
    nrowsC = sum(len(b) for b in Cblocks)
    ncolsC = sum(len(b[0]) for b in Cblocks)
    C = [[Fraction(0)] * ncolsC for _ in range(nrowsC)]
    r0 = c0 = 0
    for b in Cblocks:
        for i, row in enumerate(b):
            for j, v in enumerate(row):
                C[r0 + i][c0 + j] = v
        r0 += len(b)
        c0 += len(b[0])
    # E: columns vec(R_M[a^k N_i M_i]) (vec(R_M[a^k M_i]) with the factors in G), k < d,
    # padded to n + 1 rows
    Ecols = []
    for bi, (m, Mi_, Ni) in enumerate(zip(finite, Mi, N)):
        f = Mi_ if factors == "G" else P.mul(Ni, Mi_)
        for k in range(P.deg(m)):
            Ecols.append(P.vec(P.rem(P.mul(P.power_of_a(k), f), Mpoly), n + 1))
        blocks[bi]["E"] = Ecols[-P.deg(m):]
    E = [[Ecols[j][i] for j in range(len(Ecols))] for i in range(n + 1)]
    EC = _matmul(E, C)
    if has_inf:
        vM = P.vec(Mpoly, n + 1)
        B = [EC[i] + [vM[i]] for i in range(n + 1)]
    else:
        B = EC

    if scaling == "l1":
        for x in range(len(G)):
            # a zero row (a domain point the output never uses) stays as it is
            sg = sum((abs(v) for v in G[x]), Fraction(0)) or Fraction(1)
            sa = sum((abs(v) for v in A[x]), Fraction(0)) or Fraction(1)
            G[x] = [v / sg for v in G[x]]
            A[x] = [v / sa for v in A[x]]
            for k in range(n + 1):
                B[k][x] = B[k][x] * sg * sa

    plan.G, plan.A, plan.B = G, A, B
    plan.C, plan.E, plan.N, plan.M, plan.Mi = C, E, N, Mpoly, Mi
    plan.blocks = blocks
    return plan


# ---------------------------------------------------------------------------
# Exact identities the construction must satisfy
# ---------------------------------------------------------------------------

def trilinear_defect(plan):
    """Max |sum_xi B[k,xi] G[xi,i] A[xi,j] - [k == i + j]| (0 for a valid plan).

    This is the CRT reconstruction identity: B^W (G^W h (.) A^W x) equals the
    coefficient vector of h(a) x(a) for every h, x (Section 2.1).
    """
    worst = Fraction(0)
    al = plan.alpha
    for k in range(plan.n + 1):
        for i in range(plan.n_h):
            for j in range(plan.n_o):
                s = sum((plan.B[k][x] * plan.G[x][i] * plan.A[x][j] for x in range(al)), Fraction(0))
                worst = max(worst, abs(s - (1 if k == i + j else 0)))
    return worst


def crt_idempotent_defect(plan):
    """Max over (i, j) of the coefficients of R_{m_j}[N_i M_i] - delta_ij."""
    worst = Fraction(0)
    for i, (Ni, Mi_) in enumerate(zip(plan.N, plan.Mi)):
        e = P.mul(Ni, Mi_)
        for j, mj in enumerate(plan.moduli):
            r = P.rem(e, mj)
            target = P.ONE if i == j else P.ZERO
            diff = P.sub(r, target)
            for c in diff:
                worst = max(worst, abs(c))
    return worst
