// Exact rational and polynomial arithmetic (host only).  See rational.hpp.
#include "rational.hpp"

#include <cmath>

namespace wg {

static int bit_length(unsigned __int128 v) {
    int b = 0;
    while (v != 0) { v >>= 1; ++b; }
    return b;
}

float Rat::to_f32() const {
    if (n_ == 0) return 0.0f;
    using u128 = unsigned __int128;
    const bool neg = n_ < 0;
    const u128 num = static_cast<u128>(neg ? -static_cast<i128>(n_) : static_cast<i128>(n_));
    const u128 den = static_cast<u128>(d_);
    // e = floor(log2(num / den)); num, den < 2^63 so every shift fits 128 bits
    int e = bit_length(num) - bit_length(den);
    const bool below = e >= 0 ? num < (den << e) : (num << -e) < den;
    if (below) e -= 1;
    // quantum of the result: 2^(e-23) for normals, 2^-149 for subnormals
    const int qe = (e > -126 ? e : -126) - 23;
    // q = floor(num / (den * 2^qe)), r = the remainder over divisor dd
    u128 q, r, dd;
    if (qe >= 0) {
        dd = den << qe;                   // qe <= 39
        q = num / dd;
        r = num % dd;
    } else {
        dd = den;
        q = num / den;
        r = num % den;
        for (int i = 0; i < -qe; ++i) {   // long division, one bit at a time
            r <<= 1;
            q <<= 1;
            if (r >= den) { r -= den; q |= 1; }
        }
    }
    const u128 twice = r << 1;
    if (twice > dd || (twice == dd && (q & 1) != 0)) q += 1;   // nearest, ties to even
    // q <= 2^24 and qe >= -149: the value is exactly representable
    const double v = std::ldexp(static_cast<double>(static_cast<uint64_t>(q)), qe);
    const float f = v > 3.4028234663852886e38 ? INFINITY : static_cast<float>(v);
    return neg ? -f : f;
}

void Poly::divmod(const Poly& b, Poly* q, Poly* r) const {
    if (b.is_zero()) throw std::domain_error("division by the zero polynomial");
    std::vector<Rat> rem(c_);
    const int db = b.deg();
    const Rat lb = b.lead();
    std::vector<Rat> quo(rem.size() > static_cast<size_t>(db) ? rem.size() - static_cast<size_t>(db) : 0);
    while (!rem.empty() && static_cast<int>(rem.size()) - 1 >= db) {
        const int shift = static_cast<int>(rem.size()) - 1 - db;
        const Rat f = rem.back() / lb;
        quo[static_cast<size_t>(shift)] = f;
        for (int i = 0; i <= db; ++i) rem[static_cast<size_t>(shift + i)] -= f * b.coef(i);
        rem.pop_back();
        while (!rem.empty() && rem.back().is_zero()) rem.pop_back();
    }
    if (q) *q = Poly(quo);
    if (r) *r = Poly(rem);
}

Poly Poly::exact_div(const Poly& b) const {
    Poly q, r;
    divmod(b, &q, &r);
    if (!r.is_zero()) throw std::logic_error("polynomial division is not exact");
    return q;
}

std::vector<Rat> Poly::vec(int n) const {
    if (deg() >= n) throw std::logic_error("polynomial does not fit the vector length");
    std::vector<Rat> v(static_cast<size_t>(n), Rat(0));
    for (size_t i = 0; i < c_.size(); ++i) v[i] = c_[i];
    return v;
}

Poly poly_gcd(const Poly& f, const Poly& g, Poly* s_out) {
    Poly r0 = f, r1 = g;
    Poly s0 = Poly::constant(Rat(1)), s1;
    while (!r1.is_zero()) {
        Poly q, r;
        r0.divmod(r1, &q, &r);
        r0 = r1;
        r1 = r;
        Poly s2 = s0 - q * s1;
        s0 = s1;
        s1 = s2;
    }
    if (r0.is_zero()) throw std::domain_error("gcd of zero polynomials");
    const Rat inv = Rat(1) / r0.lead();
    if (s_out) *s_out = s0.scaled(inv);
    return r0.scaled(inv);
}

Poly inverse_mod(const Poly& f, const Poly& m) {
    Poly s;
    Poly g = poly_gcd(f, m, &s);
    if (g.deg() != 0) throw std::domain_error("not coprime");
    return s.rem(m);
}

static bool is_square_u(int64_t v) {
    if (v < 0) return false;
    int64_t r = static_cast<int64_t>(std::sqrt(static_cast<double>(v)));
    while (r > 0 && r * r > v) --r;
    while ((r + 1) * (r + 1) <= v) ++r;
    return r * r == v;
}

bool is_rational_square(const Rat& q) {
    if (q.num() < 0) return false;
    return is_square_u(q.num()) && is_square_u(q.den());
}

}  // namespace wg
