// Winograd transform construction by the polynomial Chinese Remainder Theorem.
//
// Barabasz & Gregg, arXiv 1905.05233:
//   Section 2.1, eq. (1): s = sum_i s_i N_i M_i mod M with M = prod m_i,
//     M_i = M / m_i and N_i M_i + n_i m_i = 1 (extended Euclid); the
//     "modified" algorithm adds the pseudo-point infinity so that deg M = deg s.
//   Algorithm 1: G^W and A^W.  A linear modulus a - p gives the Toom-Cook rows
//     [p^0 .. p^(r-1)] and [p^0 .. p^(m-1)] (not scaled by N_i); a degree-d
//     modulus gives G^(T-C) G' and A^(T-C) A', where G', A' reduce a
//     polynomial mod m_i (columns vec(R_m[a^k])) and G^(T-C), A^(T-C) belong
//     to the inner Toom-Cook F_T-C(d x d, d x d); infinity gives [0 .. 0 1].
//   Algorithm 2: B^W = [E C | vec(M)], C block-diagonal with [1] for linear
//     moduli and the columns vec(R_m[b_j]) of the inner B^(T-C) otherwise,
//     E_i = [vec(R_M[a^k N_i M_i])]_{k<d} above a zero row.
//
// Readings of the paper that the implementation fixes:
//   - inner Toom-Cook scaling as in the Section 2.2 example: the Lagrange
//     factor of each inner point sits in G^(T-C); B^(T-C) columns are
//     vec(M_in / (a - q)) and vec(M_in) for infinity;
//   - A' has m columns (Algorithm 1; the example prints four);
//   - N_i always from extended Euclid (the example's N_i assume b=0, c=1);
//   - without the pseudo-point the degree sum is m + r - 1, E has no zero
//     row and B^W = E C (Table 1's all-quadratic columns);
//   - Winograd-domain rows: modulus order, 2d-1 rows per degree-d modulus
//     in inner-point order, infinity last.
// Option: the CRT factors N_i may instead multiply the kernel residues
// ((N_i g mod m_i)(d mod m_i) = N_i g d mod m_i), giving G' = [vec(R_m[N_i
// a^k])] and E_i = [vec(R_M[a^k M_i])]: the same exact algorithm with other
// roundings (an accuracy variant of the kind the related work of Section 4 names as complementary).
#include "plan.hpp"

#include <algorithm>
#include <cctype>
#include <cerrno>
#include <cstdlib>

namespace wg {

namespace {

// ---------------------------------------------------------------- parsing

Rat parse_rational(const std::string& s) {
    if (s.empty()) throw PlanError(kErrArg, "empty number");
    const size_t slash = s.find('/');
    auto parse_int = [](const std::string& t) -> int64_t {
        if (t.empty()) throw PlanError(kErrArg, "bad number");
        size_t i = 0;
        if (t[0] == '+' || t[0] == '-') i = 1;
        if (i >= t.size()) throw PlanError(kErrArg, "bad number '" + t + "'");
        for (size_t j = i; j < t.size(); ++j)
            if (!std::isdigit(static_cast<unsigned char>(t[j]))) throw PlanError(kErrArg, "bad number '" + t + "'");
        errno = 0;
        const long long v = std::strtoll(t.c_str(), nullptr, 10);
        if (errno != 0) throw PlanError(kErrOverflow, "number out of range '" + t + "'");
        return static_cast<int64_t>(v);
    };
    if (slash == std::string::npos) return Rat(parse_int(s));
    const int64_t d = parse_int(s.substr(slash + 1));
    if (d == 0) throw PlanError(kErrArg, "zero denominator in '" + s + "'");
    return Rat(parse_int(s.substr(0, slash)), d);
}

// A polynomial in a: terms like "a^2", "-3/2a", "+1", separated by + or -.
Poly parse_poly(const std::string& text) {
    std::string s;
    for (char ch : text)
        if (!std::isspace(static_cast<unsigned char>(ch)) && ch != '*') s += ch;
    if (s.empty()) throw PlanError(kErrArg, "empty polynomial");
    std::vector<std::string> terms;
    std::string cur;
    for (size_t i = 0; i < s.size(); ++i) {
        const char ch = s[i];
        if ((ch == '+' || ch == '-') && !cur.empty() && cur.back() != '^') {
            terms.push_back(cur);
            cur.clear();
        }
        cur += ch;
    }
    terms.push_back(cur);
    std::vector<Rat> coef;
    for (std::string t : terms) {
        bool neg = false;
        if (!t.empty() && (t[0] == '+' || t[0] == '-')) {
            neg = t[0] == '-';
            t = t.substr(1);
        }
        Rat c(1);
        int k = 0;
        const size_t pa = t.find('a');
        if (pa == std::string::npos) {
            c = parse_rational(t);
        } else {
            if (pa > 0) c = parse_rational(t.substr(0, pa));
            const std::string e = t.substr(pa + 1);
            if (e.empty()) k = 1;
            else if (e[0] == '^' && e.size() > 1) k = static_cast<int>(parse_rational(e.substr(1)).num());
            else throw PlanError(kErrArg, "bad term '" + t + "'");
            if (k < 0 || k > 8) throw PlanError(kErrUnsupported, "exponent out of range in '" + t + "'");
        }
        if (neg) c = -c;
        if (coef.size() <= static_cast<size_t>(k)) coef.resize(static_cast<size_t>(k) + 1);
        coef[static_cast<size_t>(k)] += c;
    }
    return Poly(coef);
}

std::vector<std::string> split_commas(const std::string& text) {
    std::vector<std::string> out;
    std::string cur;
    for (char ch : text) {
        if (ch == ',') { out.push_back(cur); cur.clear(); }
        else if (!std::isspace(static_cast<unsigned char>(ch))) cur += ch;
    }
    out.push_back(cur);
    return out;
}

bool is_inf_token(const std::string& t) {
    std::string l;
    for (char ch : t) l += static_cast<char>(std::tolower(static_cast<unsigned char>(ch)));
    return l == "inf" || l == "infinity";
}

// ------------------------------------------------------------ validation

// Rational roots of a polynomial with rational coefficients (rational root
// theorem on the integer-scaled polynomial); used to decide irreducibility of
// cubics.
bool has_rational_root(const Poly& p) {
    if (p.coef(0).is_zero()) return true;
    i128 lcm = 1;
    for (const Rat& c : p.coeffs()) lcm = lcm / gcd128(lcm, c.den()) * c.den();
    if (lcm > (static_cast<i128>(1) << 40)) throw PlanError(kErrUnsupported, "modulus coefficients too large");
    const i128 a0 = static_cast<i128>(p.coef(0).num()) * (lcm / p.coef(0).den());
    const i128 an = static_cast<i128>(p.lead().num()) * (lcm / p.lead().den());
    const i128 A0 = a0 < 0 ? -a0 : a0, AN = an < 0 ? -an : an;
    if (A0 > 1000000 || AN > 1000000) throw PlanError(kErrUnsupported, "modulus coefficients too large");
    for (int64_t u = 1; u <= static_cast<int64_t>(A0); ++u) {
        if (A0 % u != 0) continue;
        for (int64_t v = 1; v <= static_cast<int64_t>(AN); ++v) {
            if (AN % v != 0) continue;
            for (int sgn = -1; sgn <= 1; sgn += 2)
                if (p.eval(Rat(sgn * u, v)).is_zero()) return true;
        }
    }
    return false;
}

bool irreducible(const Poly& m) {
    const int d = m.deg();
    if (d == 1) return true;
    if (d == 2) {
        const Rat disc = m.coef(1) * m.coef(1) - Rat(4) * m.coef(0) * m.coef(2);
        return !is_rational_square(disc);
    }
    if (d == 3) return !has_rational_root(m);
    throw PlanError(kErrUnsupported, "moduli of degree above 3 are not supported");
}

// ------------------------------------------------------------ matrices

using Mat = std::vector<std::vector<Rat>>;  // row-major

Mat matmul(const Mat& X, const Mat& Y) {
    const size_t rows = X.size(), inner = Y.size(), cols = Y.empty() ? 0 : Y[0].size();
    Mat Z(rows, std::vector<Rat>(cols));
    for (size_t i = 0; i < rows; ++i)
        for (size_t k = 0; k < inner; ++k) {
            if (X[i][k].is_zero()) continue;
            for (size_t j = 0; j < cols; ++j) Z[i][j] += X[i][k] * Y[k][j];
        }
    return Z;
}

// d x ncols matrix whose column k is vec(R_m[a^k])  (G' / A' of Algorithm 1).
// [vec(R_mod[f a^0]) .. vec(R_mod[f a^(ncols-1)])]: Algorithm 1's G' and A'
// with f = 1; f = N_i carries the CRT factor on the kernel side.
Mat residue_columns(const Poly& mod, int ncols, const Poly& f = Poly::constant(Rat(1))) {
    const int d = mod.deg();
    Mat R(static_cast<size_t>(d), std::vector<Rat>(static_cast<size_t>(ncols)));
    for (int k = 0; k < ncols; ++k) {
        const std::vector<Rat> v = (f * Poly::monomial(k)).rem(mod).vec(d);
        for (int i = 0; i < d; ++i) R[static_cast<size_t>(i)][static_cast<size_t>(k)] = v[static_cast<size_t>(i)];
    }
    return R;
}

// Inner Toom-Cook F_T-C(d x d, d x d) on the given points.
struct InnerTC {
    Mat G, A;  // (2d-1) x d
    Mat B;     // (2d-1) x (2d-1), column j = reconstruction polynomial of row j
};

InnerTC inner_toom_cook(int d, const std::vector<Rat>& pts_all, bool with_inf) {
    const int L = 2 * d - 1;
    const int nfin = with_inf ? L - 1 : L;
    if (static_cast<int>(pts_all.size()) < nfin)
        throw PlanError(kErrArg, "a degree-" + std::to_string(d) + " modulus needs " + std::to_string(nfin) +
                                     " finite inner points");
    std::vector<Rat> pts(pts_all.begin(), pts_all.begin() + nfin);
    for (int i = 0; i < nfin; ++i)
        for (int j = i + 1; j < nfin; ++j)
            if (pts[static_cast<size_t>(i)] == pts[static_cast<size_t>(j)]) throw PlanError(kErrArg, "inner points must be distinct");
    Poly Min = Poly::constant(Rat(1));
    for (const Rat& q : pts) Min = Min * Poly(std::vector<Rat>{-q, Rat(1)});
    InnerTC tc;
    tc.B.assign(static_cast<size_t>(L), std::vector<Rat>(static_cast<size_t>(L)));
    int col = 0;
    for (const Rat& q : pts) {
        // Lagrange basis numerator M_in / (a - q) and its value at q
        const Poly lin(std::vector<Rat>{-q, Rat(1)});
        const Poly Mq = Min.exact_div(lin);
        const Rat Nq = Rat(1) / Mq.eval(q);
        std::vector<Rat> grow, arow;
        Rat pw(1);
        for (int k = 0; k < d; ++k) {
            grow.push_back(Nq * pw);
            arow.push_back(pw);
            pw = pw * q;
        }
        tc.G.push_back(grow);
        tc.A.push_back(arow);
        const std::vector<Rat> bc = Mq.vec(L);
        for (int k = 0; k < L; ++k) tc.B[static_cast<size_t>(k)][static_cast<size_t>(col)] = bc[static_cast<size_t>(k)];
        ++col;
    }
    if (with_inf) {
        std::vector<Rat> e(static_cast<size_t>(d), Rat(0));
        e.back() = Rat(1);
        tc.G.push_back(e);
        tc.A.push_back(e);
        const std::vector<Rat> bc = Min.vec(L);
        for (int k = 0; k < L; ++k) tc.B[static_cast<size_t>(k)][static_cast<size_t>(col)] = bc[static_cast<size_t>(k)];
    }
    return tc;
}

}  // namespace

std::vector<Modulus> parse_moduli(const std::string& text) {
    std::vector<Modulus> out;
    for (const std::string& tok : split_commas(text)) {
        if (tok.empty()) throw PlanError(kErrArg, "empty modulus in '" + text + "'");
        Modulus md;
        if (is_inf_token(tok)) {
            md.inf = true;
        } else if (tok.find('a') != std::string::npos) {
            md.p = parse_poly(tok);
        } else {
            md.p = Poly(std::vector<Rat>{-parse_rational(tok), Rat(1)});
        }
        out.push_back(md);
    }
    return out;
}

void parse_points(const std::string& text, std::vector<Rat>* pts, bool* with_inf) {
    pts->clear();
    *with_inf = false;
    for (const std::string& tok : split_commas(text)) {
        if (tok.empty()) throw PlanError(kErrArg, "empty inner point");
        if (is_inf_token(tok)) *with_inf = true;
        else pts->push_back(parse_rational(tok));
    }
}

Transforms build_transforms(const std::vector<Modulus>& moduli_in, const std::vector<Rat>& inner_pts,
                            bool inner_inf, int m, int r, bool factors_in_g, bool scale_rows) {
    if (m < 1 || r < 1) throw PlanError(kErrArg, "tile sizes must be positive");
    const int n = m + r - 2;  // degree of the product polynomial s(a)
    std::vector<Poly> mods;
    bool has_inf = false;
    for (const Modulus& md : moduli_in) {
        if (md.inf) {
            if (has_inf) throw PlanError(kErrArg, "the pseudo-point infinity appears twice");
            has_inf = true;
            continue;
        }
        if (md.p.deg() < 1) throw PlanError(kErrArg, "a modulus must have degree >= 1");
        mods.push_back(md.p.monic());
    }
    if (mods.empty()) throw PlanError(kErrArg, "no finite modulus");
    int degsum = 0;
    for (const Poly& p : mods) degsum += p.deg();
    const int want = has_inf ? n : n + 1;
    if (degsum != want)
        throw PlanError(kErrDegreeSum, "sum of modulus degrees is " + std::to_string(degsum) + ", F(" +
                                           std::to_string(m) + "," + std::to_string(r) + ") needs " +
                                           std::to_string(want));
    for (const Poly& p : mods)
        if (!irreducible(p)) throw PlanError(kErrReducible, "a modulus is reducible over Q");
    for (size_t i = 0; i < mods.size(); ++i)
        for (size_t j = i + 1; j < mods.size(); ++j)
            if (poly_gcd(mods[i], mods[j], nullptr).deg() != 0)
                throw PlanError(kErrNotCoprime, "moduli are not pairwise coprime");

    // eq. (1): M = prod m_i, M_i = M / m_i, N_i M_i = 1 (mod m_i)
    Poly M = Poly::constant(Rat(1));
    for (const Poly& p : mods) M = M * p;
    std::vector<Poly> Mis, Nis;
    for (const Poly& mi : mods) {
        Mis.push_back(M.exact_div(mi));
        Nis.push_back(inverse_mod(Mis.back(), mi));
    }

    // ---- Algorithm 1 -------------------------------------------------------
    // factors_in_g: the kernel residues carry N_i (rows scaled by the constant
    // N_i(p) for a linear modulus, G' = [vec(R_m[N_i a^k])] otherwise)
    Mat G, A;
    std::vector<InnerTC> tcs(mods.size());
    for (size_t i = 0; i < mods.size(); ++i) {
        const Poly& mi = mods[i];
        const int d = mi.deg();
        const Poly kf = factors_in_g ? Nis[i] : Poly::constant(Rat(1));
        if (d == 1) {
            const Rat p = -mi.coef(0);
            const Rat sc = kf.coef(0);   // N_i is the constant 1 / M_i(p)
            std::vector<Rat> g, a;
            Rat pw(1);
            for (int k = 0; k < std::max(r, m); ++k) {
                if (k < r) g.push_back(sc * pw);
                if (k < m) a.push_back(pw);
                pw = pw * p;
            }
            G.push_back(g);
            A.push_back(a);
        } else {
            tcs[i] = inner_toom_cook(d, inner_pts, inner_inf);
            const Mat Gi = matmul(tcs[i].G, residue_columns(mi, r, kf));
            const Mat Ai = matmul(tcs[i].A, residue_columns(mi, m));
            G.insert(G.end(), Gi.begin(), Gi.end());
            A.insert(A.end(), Ai.begin(), Ai.end());
        }
    }
    if (has_inf) {
        std::vector<Rat> g(static_cast<size_t>(r), Rat(0)), a(static_cast<size_t>(m), Rat(0));
        g.back() = Rat(1);
        a.back() = Rat(1);
        G.push_back(g);
        A.push_back(a);
    }
    const int alpha = static_cast<int>(G.size());

    // ---- Algorithm 2 -------------------------------------------------------
    const int rowsB = n + 1;
    // E C computed block by block: for modulus i, E_i (rowsB x d) times C_i
    // (d x (2d-1)) fills the columns of that modulus' domain rows.
    Mat B(static_cast<size_t>(rowsB), std::vector<Rat>(static_cast<size_t>(alpha)));
    int col0 = 0;
    for (size_t i = 0; i < mods.size(); ++i) {
        const Poly& mi = mods[i];
        const int d = mi.deg();
        // E_i = [vec(R_M[a^k N_i M_i])], or [vec(R_M[a^k M_i])] with the factors in G
        const Poly NiMi = factors_in_g ? Mis[i] : Nis[i] * Mis[i];
        Mat Ei(static_cast<size_t>(rowsB), std::vector<Rat>(static_cast<size_t>(d)));
        for (int k = 0; k < d; ++k) {
            const std::vector<Rat> v = (Poly::monomial(k) * NiMi).rem(M).vec(rowsB);
            for (int row = 0; row < rowsB; ++row) Ei[static_cast<size_t>(row)][static_cast<size_t>(k)] = v[static_cast<size_t>(row)];
        }
        Mat Ci;
        if (d == 1) {
            Ci = Mat{{Rat(1)}};
        } else {
            const int L = 2 * d - 1;
            Ci.assign(static_cast<size_t>(d), std::vector<Rat>(static_cast<size_t>(L)));
            for (int j = 0; j < L; ++j) {
                std::vector<Rat> bj(static_cast<size_t>(L));
                for (int k = 0; k < L; ++k) bj[static_cast<size_t>(k)] = tcs[i].B[static_cast<size_t>(k)][static_cast<size_t>(j)];
                const std::vector<Rat> v = Poly(bj).rem(mi).vec(d);
                for (int k = 0; k < d; ++k) Ci[static_cast<size_t>(k)][static_cast<size_t>(j)] = v[static_cast<size_t>(k)];
            }
        }
        const Mat EiCi = matmul(Ei, Ci);
        for (int row = 0; row < rowsB; ++row)
            for (size_t j = 0; j < EiCi[0].size(); ++j)
                B[static_cast<size_t>(row)][static_cast<size_t>(col0) + j] = EiCi[static_cast<size_t>(row)][j];
        col0 += static_cast<int>(EiCi[0].size());
    }
    if (has_inf) {
        const std::vector<Rat> vM = M.vec(rowsB);
        for (int row = 0; row < rowsB; ++row) B[static_cast<size_t>(row)][static_cast<size_t>(col0)] = vM[static_cast<size_t>(row)];
        ++col0;
    }
    if (col0 != alpha) throw PlanError(kErrInternal, "inconsistent domain size");

    // scale_rows: every domain row of G and of A divided by its 1-norm, the
    // matching column of B multiplied by both norms.  Each domain row's
    // rank-1 term B[:, xi] G[xi] A[xi] is unchanged, so the algorithm stays
    // exact; only the roundings move (the diagonal scaling of G and A^T that
    // the related work of Section 4 cites).
    if (scale_rows) {
        auto absr = [](const Rat& v) { return v.num() < 0 ? -v : v; };
        for (int x = 0; x < alpha; ++x) {
            Rat sg(0), sa(0);
            for (const Rat& v : G[static_cast<size_t>(x)]) sg += absr(v);
            for (const Rat& v : A[static_cast<size_t>(x)]) sa += absr(v);
            // a zero row (a domain point the output never uses) stays as it is
            if (sg.is_zero()) sg = Rat(1);
            if (sa.is_zero()) sa = Rat(1);
            for (Rat& v : G[static_cast<size_t>(x)]) v = v / sg;
            for (Rat& v : A[static_cast<size_t>(x)]) v = v / sa;
            for (int row = 0; row < rowsB; ++row) {
                Rat& b = B[static_cast<size_t>(row)][static_cast<size_t>(x)];
                b = b * sg * sa;
            }
        }
    }

    // ---- exact self-check: sum_xi B[k][xi] G[xi][i] A[xi][j] == [k == i+j] ----
    for (int k = 0; k < rowsB; ++k)
        for (int i = 0; i < r; ++i)
            for (int j = 0; j < m; ++j) {
                Rat s(0);
                for (int x = 0; x < alpha; ++x)
                    s += B[static_cast<size_t>(k)][static_cast<size_t>(x)] * G[static_cast<size_t>(x)][static_cast<size_t>(i)] *
                         A[static_cast<size_t>(x)][static_cast<size_t>(j)];
                if (s != Rat(k == i + j ? 1 : 0))
                    throw PlanError(kErrInternal, "built transforms fail the CRT reconstruction identity");
            }

    Transforms t;
    t.m = m;
    t.r = r;
    t.alpha = alpha;
    t.tile_in = rowsB;
    for (const auto& row : G) for (const Rat& v : row) { t.G.push_back(v); t.Gf.push_back(v.to_f32()); }
    for (const auto& row : A) for (const Rat& v : row) { t.A.push_back(v); t.Af.push_back(v.to_f32()); }
    for (const auto& row : B) for (const Rat& v : row) { t.B.push_back(v); t.Bf.push_back(v.to_f32()); }
    return t;
}

}  // namespace wg
