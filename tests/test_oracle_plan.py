"""Pins of the oracle's exact transform construction (CPU only).

Each check ties the oracle to something other than itself: matrices the paper
prints (Section 2.2 worked example), the ratios of Table 1 and Section 3.2,
published Toom-Cook matrices (Lavin & Gray 2016) and closed-form identities
(the CRT reconstruction identity and the CRT idempotents, eq. (1)).
"""
from fractions import Fraction

import pytest

from conftest import frac_matrix, load_golden
from oracle import conv as OC
from oracle import plan as OP
from oracle import polynomials as P

# modulus sets of the library's parity workloads (domain row order = list order)
CONFIG_SETS = [
    ("0,1,-1,inf", 2),                      # F(2x2) Toom-Cook
    ("0,1,-1,1/2,-1/2,inf", 4),             # F(4x4) Toom-Cook
    ("0,1,-1,a^2+1,inf", 4),                # F(4x4) with a^2+1
    ("0,-1,1,-1/2,2,1/2,-2,inf", 6),        # F(6x6) Toom-Cook
    ("0,-1,1,a^2+1,a^2-2,inf", 6),          # F(6x6) with two quadratics
    ("0,-1,1,-1/2,2,a^2+1,inf", 6),         # F(6x6) with one a^2+1 (ratio 2.25)
]


def example_plan(b, c):
    m2 = (Fraction(c), Fraction(b), Fraction(1))
    return OP.build_plan(["0", m2, "inf"], n_o=2, inner="0,1,inf")


BC_VALUES = [(0, 1), (1, 1), (-1, 1), (0, -2), (2, 3), (Fraction(1, 2), 5)]


@pytest.mark.parametrize("b,c", BC_VALUES)
def test_worked_example_general_entries(b, c):
    """Section 2.2 worked example: entries printed in terms of (b, c)."""
    gold = load_golden("worked_example_sec2_2.json")["general"]
    env = {"b": Fraction(b), "c": Fraction(c)}
    pl = example_plan(b, c)
    blk = pl.blocks[1]
    assert blk["tc"].G == frac_matrix(gold["G_TC"], env)
    assert blk["tc"].A == frac_matrix(gold["A_TC"], env)
    assert blk["tc"].B == frac_matrix(gold["B_TC"], env)
    assert blk["Gp"] == frac_matrix(gold["G_prime"], env)
    assert blk["G"] == frac_matrix(gold["G_2"], env)
    # the printed A' / A_2 use four columns (a^0..a^3): the residue map itself
    A4 = OP.residue_map(blk["m"], 4)
    assert A4 == frac_matrix(gold["A_prime_4col"], env)
    assert OP._matmul(blk["tc"].A, A4) == frac_matrix(gold["A_2_4col"], env)
    assert pl.G == frac_matrix(gold["G_W"], env)
    assert blk["C"] == frac_matrix(gold["C_2"], env)
    assert pl.C == frac_matrix(gold["C"], env)
    assert [row[-1] for row in pl.B] == frac_matrix([gold["B_W_last_column"]], env)[0]


def test_worked_example_at_b0_c1():
    """E, EC, B^W and N_i as printed; they are valid at b = 0, c = 1."""
    gold = load_golden("worked_example_sec2_2.json")["b0c1"]
    env = {"b": Fraction(0), "c": Fraction(1)}
    pl = example_plan(0, 1)
    assert list(pl.N[0]) == frac_matrix([gold["N_1"]], env)[0]
    assert list(pl.N[1]) == frac_matrix([gold["N_2"]], env)[0]
    Ecols1 = pl.blocks[0]["E"]
    Ecols2 = pl.blocks[1]["E"]
    # the printed E_i stack the deg(M) = 3 coefficients (no zero row yet)
    assert [[col[i] for col in Ecols1] for i in range(3)] == frac_matrix(gold["E_1"], env)
    assert [[col[i] for col in Ecols2] for i in range(3)] == frac_matrix(gold["E_2"], env)
    assert pl.E == frac_matrix(gold["E"], env)
    assert OP._matmul(pl.E, pl.C) == frac_matrix(gold["EC"], env)
    assert pl.B == frac_matrix(gold["B_W"], env)
    # the corrected A^W (Algorithm 1: A' has n_o = 2 columns)
    assert pl.A == [[1, 0], [1, 0], [1, 1], [0, 1], [0, 1]]


@pytest.mark.parametrize("b,c", [(1, 1), (0, -2)])
def test_printed_N_is_specific_to_b0_c1(b, c):
    """Away from b=0, c=1 the printed N_1 = 1, N_2 = -a are not inverses;
    the oracle's Euclid-derived N_i are, and its B^W satisfies the identity."""
    pl = example_plan(b, c)
    m1, m2 = pl.moduli
    M1, M2 = pl.Mi
    assert P.rem(P.mul(P.poly([1]), M1), m1) != P.ONE or P.rem(P.mul(P.poly([0, -1]), M2), m2) != P.ONE
    assert P.rem(P.mul(pl.N[0], M1), m1) == P.ONE
    assert P.rem(P.mul(pl.N[1], M2), m2) == P.ONE
    assert OP.trilinear_defect(pl) == 0


def _table1_set(n_o, deg1, deg2):
    pts = load_golden("table1_ratios.json")["good_points_sec3_1"]
    quads = ["a^2+1", "a^2+a+1", "a^2-a+1", "a^2-2"]
    items = []
    has_inf = deg1 > 0
    nfin = deg1 - (1 if has_inf else 0)
    items += pts[:nfin]
    items += quads[:deg2]
    if has_inf:
        items.append("inf")
    return ",".join(items)


@pytest.mark.parametrize("row", load_golden("table1_ratios.json")["table1"],
                         ids=lambda r: f"m{r['n_o']}-l{r['deg1']}-q{r['deg2']}")
def test_table1_ratios(row):
    """Table 1: build each modulus mix and compare alpha'^2/m^2 with the print."""
    spec = _table1_set(row["n_o"], row["deg1"], row["deg2"])
    pl = OP.build_plan(spec, n_o=row["n_o"])
    assert OP.trilinear_defect(pl) == 0
    assert round(float(pl.ratio), 2) == float(row["ratio"])


@pytest.mark.parametrize("opt", load_golden("table1_ratios.json")["f2x2_options_sec2_3"],
                         ids=lambda o: o["moduli"])
def test_f2x2_option_list(opt):
    """Section 2.3's list of F(2x2,3x3) constructions and their ratios."""
    pl = OP.build_plan(opt["moduli"], n_o=2, inner=opt.get("inner", "0,-1,inf"))
    assert OP.trilinear_defect(pl) == 0
    assert float(pl.ratio) == float(opt["ratio"])


def test_section3_2_ratio_lists():
    gold = load_golden("table1_ratios.json")
    pts = gold["good_points_sec3_1"] + ["1/4", "-4"]
    for row in gold["toom_cook_sec3_2"]:
        m = row["n_o"]
        pl = OP.build_plan(",".join(pts[:m + 1] + ["inf"]), n_o=m)
        assert OP.trilinear_defect(pl) == 0
        assert round(float(pl.ratio), 2) == float(row["ratio"])
    for row in gold["winograd_one_a2p1_sec3_2"]:
        m = row["n_o"]
        # linear points of F_W(m) are those of F_T-C(m - 2): m - 1 finite points
        pl = OP.build_plan(",".join(pts[:m - 1] + ["a^2+1", "inf"]), n_o=m)
        assert OP.trilinear_defect(pl) == 0
        assert round(float(pl.ratio), 2) == float(row["ratio"])


@pytest.mark.parametrize("spec,m", CONFIG_SETS)
def test_crt_identities(spec, m):
    pl = OP.build_plan(spec, n_o=m)
    assert OP.trilinear_defect(pl) == 0
    assert OP.crt_idempotent_defect(pl) == 0
    assert len(pl.G) == pl.alpha and len(pl.A) == pl.alpha
    assert len(pl.B) == m + 2 and all(len(r) == pl.alpha for r in pl.B)


def test_config_alphas():
    want = {0: 4, 1: 6, 2: 7, 3: 8, 4: 10, 5: 9}
    for i, (spec, m) in enumerate(CONFIG_SETS):
        assert OP.build_plan(spec, n_o=m).alpha == want[i]


def _triples(G, A, BT):
    al = len(G)
    out = []
    for x in range(al):
        out.append([[[A[x][j] * G[x][i] * BT[x][k] for k in range(len(BT[x]))]
                     for i in range(len(G[x]))] for j in range(len(A[x]))])
    return out


@pytest.mark.parametrize("name", ["F(2,3)", "F(4,3)"])
def test_linear_points_reproduce_lavin(name):
    """Linear-only sets are Toom-Cook: each domain row's rank-1 term
    A_xi (x) G_xi (x) B^T_xi equals the published matrices' (Lavin & Gray)."""
    gold = load_golden("lavin_gray_2016.json")[name]
    G = frac_matrix(gold["G"])
    BT = frac_matrix(gold["BT"])
    AT = frac_matrix(gold["AT"])
    A = [list(r) for r in zip(*AT)]
    m = len(AT)
    # the published set itself satisfies the reconstruction identity
    B = [list(r) for r in zip(*BT)]
    for k in range(m + 2):
        for i in range(3):
            for j in range(m):
                s = sum(B[k][x] * G[x][i] * A[x][j] for x in range(len(G)))
                assert s == (1 if k == i + j else 0)
    pl = OP.build_plan(gold["points"], n_o=m)
    assert _triples(pl.G, pl.A, pl.BT) == _triples(G, A, BT)


def test_linear_rows_are_powers():
    """Algorithm 1: a linear modulus a - p gives rows [p^0 .. p^(n-1)]."""
    pl = OP.build_plan("0,1,-1,1/2,-1/2,inf", n_o=4)
    for x, p in enumerate([0, 1, -1, Fraction(1, 2), Fraction(-1, 2)]):
        assert pl.G[x] == [Fraction(p) ** k for k in range(3)]
        assert pl.A[x] == [Fraction(p) ** k for k in range(4)]
    assert pl.G[-1] == [0, 0, 1] and pl.A[-1] == [0, 0, 0, 1]


def test_inner_points_default_matches_section3():
    """Section 3.1 solves the degree-2 sub-problem with points 0, -1, infinity."""
    pl = OP.build_plan("0,1,-1,a^2+1,inf", n_o=4)
    tc = pl.blocks[3]["tc"]
    assert tc.A == [[1, 0], [1, -1], [0, 1]]


@pytest.mark.parametrize("spec,m,err", [
    ("0,1,inf", 4, "sum of degrees"),
    ("0,1,-1,a^2-1,inf", 4, "reducible"),
    ("0,1,-1,a^2+1,a^2+1,inf", 6, "coprime"),
    ("0,0,1,-1,1/2,inf", 4, "coprime"),
])
def test_invalid_sets_rejected(spec, m, err):
    with pytest.raises(ValueError, match=err):
        OP.build_plan(spec, n_o=m)


def test_polynomial_helpers_against_brute_force():
    """divmod, Euclid and the inverse against direct expansion."""
    import random
    rng = random.Random(5)
    for _ in range(50):
        p = P.poly([Fraction(rng.randint(-5, 5), rng.randint(1, 4)) for _ in range(rng.randint(1, 7))])
        q = P.poly([Fraction(rng.randint(-5, 5), rng.randint(1, 4)) for _ in range(rng.randint(1, 4))] + [1])
        quo, r = P.divmod_poly(p, q)
        assert P.add(P.mul(quo, q), r) == p
        assert P.deg(r) < P.deg(q)
        for x in range(-3, 4):
            assert P.evaluate(p, x) == P.evaluate(quo, x) * P.evaluate(q, x) + P.evaluate(r, x)
    m = P.parse("a^2+1")
    inv = P.inverse_mod(P.parse("a+2"), m)
    assert P.rem(P.mul(inv, P.parse("a+2")), m) == P.ONE
    assert P.parse("a^2-a+1") == P.poly([1, -1, 1])
    assert P.parse("2a^3-1/2") == P.poly([Fraction(-1, 2), 0, 0, 2])


# ---------------------------------------------------------------------------
# CRT factors on the kernel side (factors="G")
# ---------------------------------------------------------------------------

def test_factors_in_g_reproduce_lavin_f43_exactly():
    """With the CRT factors N_i moved onto the kernel residues, the points
    {0, 1, -1, 2, -2, inf} give exactly the F(4,3) matrices Lavin & Gray
    published: G (with its 1/4, -1/6, 1/24 ... rows), B^T and A^T."""
    gold = load_golden("lavin_gray_2016.json")["F(4,3)"]
    pl = OP.build_plan(gold["points"], n_o=4, factors="G")
    assert pl.G == frac_matrix(gold["G"])
    assert pl.BT == frac_matrix(gold["BT"])
    assert [list(r) for r in zip(*pl.A)] == frac_matrix(gold["AT"])


def test_factors_in_g_reproduce_lavin_f23_up_to_row_signs():
    """F(2,3) on {0, 1, -1, inf}: Lavin & Gray's matrices up to the signs of
    single domain rows (G and B^T entries equal in magnitude, and each row's
    rank-1 term A (x) G (x) B^T is the published one)."""
    gold = load_golden("lavin_gray_2016.json")["F(2,3)"]
    pl = OP.build_plan(gold["points"], n_o=2, factors="G")
    G, BT, AT = frac_matrix(gold["G"]), frac_matrix(gold["BT"]), frac_matrix(gold["AT"])
    assert [[abs(v) for v in r] for r in pl.G] == [[abs(v) for v in r] for r in G]
    assert [[abs(v) for v in r] for r in pl.BT] == [[abs(v) for v in r] for r in BT]
    A = [list(r) for r in zip(*AT)]
    assert _triples(pl.G, pl.A, pl.BT) == _triples(G, A, BT)


@pytest.mark.parametrize("spec,m,inner", [
    ("0,1,-1,1/2,-1/2,inf", 4, "0,-1,inf"), ("0,1,-1,a^2+1,inf", 4, "0,-1,inf"),
    ("0,-1,1,a^2+1,a^2-2,inf", 6, "0,-1,inf"), ("a^2+1,a^2+2", 2, "0,-1,inf"),
    ("0,-1,a^3+2,inf", 4, "0,-1,1,-2,inf"), ("0,a^2+a+1,inf", 2, "0,1,inf"),
])
def test_factors_in_g_move_exactly_the_crt_factors(spec, m, inner):
    """eq. (1): moving N_i from B to G leaves the reconstruction identity and
    A unchanged; a linear modulus's G row is multiplied, and its B column
    divided, by the constant N_i = 1 / M_i(p); a degree-d block's kernel
    residues are multiplied by N_i mod m_i."""
    pb = OP.build_plan(spec, n_o=m, inner=inner)
    pg = OP.build_plan(spec, n_o=m, inner=inner, factors="G")
    assert OP.trilinear_defect(pg) == 0
    assert pg.A == pb.A and pg.alpha == pb.alpha
    x = 0
    for blk, Ni, Mi in zip(pb.blocks, pb.N, pb.Mi):
        d = blk["d"]
        rows = 1 if d == 1 else 2 * d - 1
        if d == 1:
            c = Ni[0]
            p_ = -blk["m"][0]
            assert c * P.evaluate(Mi, p_) == 1
            assert pg.G[x] == [c * v for v in pb.G[x]]
            assert [r[x] for r in pg.B] == [v / c for v in (r[x] for r in pb.B)]
        else:
            Gp = OP.residue_map(blk["m"], 3, Ni)
            want = [[sum((blk["tc"].G[i][k] * Gp[k][j] for k in range(d)), Fraction(0)) for j in range(3)]
                    for i in range(rows)]
            assert pg.G[x:x + rows] == want
        x += rows


# ---------------------------------------------------------------------------
# The exact checkers must see a broken plan (values computed by hand)
# ---------------------------------------------------------------------------

def _f23():
    """F(2x2) on {0, 1, -1, inf}: G = [[1,0,0],[1,1,1],[1,-1,1],[0,0,1]],
    A = [[1,0],[1,1],[1,-1],[0,1]], B^T = [[1,0,-1,0],[0,1/2,1/2,0],
    [0,-1/2,1/2,0],[0,-1,0,1]] (Algorithms 1 and 2)."""
    import copy
    return copy.deepcopy(OP.build_plan("0,1,-1,inf", n_o=2))


def test_trilinear_defect_sees_a_perturbed_g_entry():
    """G[1][2] += 1/2 changes sum_xi B[k,xi] G[xi,2] A[xi,j] by
    B[k,1] * 1/2 * A[1,j]; the largest such change is (1/2)(1/2)(1) = 1/4."""
    pl = _f23()
    assert OP.trilinear_defect(pl) == 0
    pl.G[1][2] += Fraction(1, 2)
    assert OP.trilinear_defect(pl) == Fraction(1, 4)


def test_trilinear_defect_sees_a_perturbed_a_entry():
    """A[2][0] += 1: the change B[k,2] G[2,i] is largest at |B^T[2][k]| = 1/2,
    |G[2][i]| = 1."""
    pl = _f23()
    pl.A[2][0] += 1
    assert OP.trilinear_defect(pl) == Fraction(1, 2)


def test_trilinear_defect_sees_a_perturbed_b_entry():
    """B[3][3] += 1 (B^T[3][3] = 1 becomes 2): the (k, i, j) = (3, 2, 1) sum,
    G[3][2] A[3][1] = 1 times the new entry, becomes 2 against a target of 1."""
    pl = _f23()
    pl.B[3][3] += 1
    assert OP.trilinear_defect(pl) == 1


def test_crt_idempotent_defect_sees_a_wrong_linear_factor():
    """For the modulus a, M_0 = a^2 - 1 and N_0 = 1 / M_0(0) = -1.  Doubling
    N_0 makes R_a[N_0 M_0] = 2 instead of 1: defect 1."""
    pl = _f23()
    assert pl.N[0] == (Fraction(-1),)
    assert OP.crt_idempotent_defect(pl) == 0
    pl.N[0] = (Fraction(-2),)
    assert OP.crt_idempotent_defect(pl) == 1


def test_crt_idempotent_defect_sees_a_wrong_quadratic_factor():
    """For a^2 + 1 in {0, 1, -1, a^2+1, inf}: M_3 = a^3 - a = -2a mod a^2+1,
    so N_3 = a/2 (since -2a * a/2 = -a^2 = 1).  With N_3 = a instead,
    R[a (a^3 - a)] = -2a^2 = 2: defect 1."""
    import copy
    pl = copy.deepcopy(OP.build_plan("0,1,-1,a^2+1,inf", n_o=4))
    assert pl.N[3] == (Fraction(0), Fraction(1, 2))
    assert OP.crt_idempotent_defect(pl) == 0
    pl.N[3] = (Fraction(0), Fraction(1))
    assert OP.crt_idempotent_defect(pl) == 1


@pytest.mark.parametrize("poly", ["a^3-1", "a^3-3a^2+3a-1", "a^3+2a^2+a+2", "a^3-1/2a^2+a-1/2", "a^3+a"])
def test_reducible_cubics_rejected(poly):
    """(a-1)(a^2+a+1), (a-1)^3, (a+2)(a^2+1), (a-1/2)(a^2+1) and a(a^2+1) have
    a rational root, so they factor over Q (Section 2.1 asks for irreducible
    moduli)."""
    assert not OP.is_irreducible(P.monic(P.parse(poly)))
    with pytest.raises(ValueError, match="reducible"):
        OP.build_plan(f"0,-1,{poly},inf", n_o=4, inner="0,-1,1,-2,inf")


@pytest.mark.parametrize("poly", ["a^3+2", "a^3-2", "a^3+a+1", "a^3-1/3a^2+1"])
def test_irreducible_cubics_accepted(poly):
    """No rational root: +-2 and +-1 are not roots of a^3 + 2, a^3 - 2 or
    a^3 + a + 1 (values 10, 6, -6, ... 3, -1), nor is any +-p/q of 3a^3 - a^2 + 3."""
    assert OP.is_irreducible(P.monic(P.parse(poly)))
    pl = OP.build_plan(f"0,-1,{poly},inf", n_o=4, inner="0,-1,1,-2,inf")
    assert OP.trilinear_defect(pl) == 0


# ---------------------------------------------------------------------------
# Diagonal scaling of G and A^T (scaling="l1")
# ---------------------------------------------------------------------------

def test_l1_scaling_of_f2x2_by_hand():
    """{0, 1, -1, inf}: G rows [1,1,1] and [1,-1,1] have 1-norm 3, A rows
    [1,1] and [1,-1] have 1-norm 2; those rows become thirds and halves and
    the B columns 1 and 2 (B^T rows [0,1/2,1/2,0] and [0,-1/2,1/2,0]) are
    multiplied by 6; rows 0 and 3 have norm 1 and stay."""
    pl = OP.build_plan("0,1,-1,inf", n_o=2, scaling="l1")
    t, h = Fraction(1, 3), Fraction(1, 2)
    assert pl.G == [[1, 0, 0], [t, t, t], [t, -t, t], [0, 0, 1]]
    assert pl.A == [[1, 0], [h, h], [h, -h], [0, 1]]
    assert pl.BT == [[1, 0, -1, 0], [0, 3, 3, 0], [0, -3, 3, 0], [0, -1, 0, 1]]


@pytest.mark.parametrize("spec,m,inner", [
    ("0,1,-1,1/2,-1/2,inf", 4, "0,-1,inf"), ("0,1,-1,a^2+1,inf", 4, "0,-1,inf"),
    ("0,-1,1,a^2+1,a^2-2,inf", 6, "0,-1,inf"), ("0,-1,1,-1/2,2,1/2,-2,-1/4,4,inf", 8, "0,-1,inf"),
    ("a^2+1,a^2+2", 2, "0,-1,inf"), ("0,-1,a^3+2,inf", 4, "0,-1,1,-2,inf"),
    ("0,a^3+2", 2, "0,-1,1,-2,inf"),    # its cubic block has a zero A row: left unscaled
])
def test_l1_scaling_keeps_each_rank_one_term(spec, m, inner):
    """Scaling moves magnitude between the three factors of every domain
    point's term A[xi] (x) G[xi] (x) B[:, xi], never the term itself; G and A
    rows end with 1-norm 1; exact Winograd still equals direct convolution."""
    pl = OP.build_plan(spec, n_o=m, inner=inner)
    ps = OP.build_plan(spec, n_o=m, inner=inner, scaling="l1")
    assert _triples(ps.G, ps.A, ps.BT) == _triples(pl.G, pl.A, pl.BT)
    assert OP.trilinear_defect(ps) == 0
    for row in ps.G + ps.A:
        assert sum(abs(v) for v in row) in (0, 1)
    x = [[[[Fraction((3 * i + 5 * j + c) % 7 - 3, 2) for c in range(2)] for j in range(m + 1)]
          for i in range(m + 2)]]
    w = [[[[Fraction((i - j + 2 * c + k) % 5 - 2) for c in range(2)] for j in range(3)] for i in range(3)]
         for k in range(2)]
    assert OC.winograd_exact(x, w, ps) == OC.direct_exact(x, w)
