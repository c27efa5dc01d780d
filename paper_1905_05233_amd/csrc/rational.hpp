// Exact rational numbers and polynomials over Q for the host-side plan builder.
//
// Section 2.1 of Barabasz & Gregg (arXiv 1905.05233) builds the Winograd
// transforms in the ring of polynomials over a field; the library does that in
// exact rationals with int64 numerator/denominator, 128-bit intermediates and
// an overflow check on every operation (an OverflowError surfaces as
// WG_ERR_OVERFLOW at the C ABI, never as a wrapped value).
#pragma once

#include <cstdint>
#include <stdexcept>
#include <string>
#include <vector>

namespace wg {

struct OverflowError : std::runtime_error {
    OverflowError() : std::runtime_error("exact rational arithmetic overflowed int64") {}
};

using i128 = __int128;

inline i128 gcd128(i128 a, i128 b) {
    if (a < 0) a = -a;
    if (b < 0) b = -b;
    while (b != 0) {
        i128 t = a % b;
        a = b;
        b = t;
    }
    return a;
}

class Rat {
public:
    Rat() : n_(0), d_(1) {}
    Rat(int64_t n) : n_(n), d_(1) {}  // NOLINT(google-explicit-constructor)
    Rat(int64_t n, int64_t d) { set(n, d); }

    static Rat from128(i128 n, i128 d) {
        if (d == 0) throw std::domain_error("zero denominator");
        if (d < 0) { n = -n; d = -d; }
        i128 g = gcd128(n, d);
        if (g > 1) { n /= g; d /= g; }
        if (n > INT64_MAX || n < -INT64_MAX || d > INT64_MAX) throw OverflowError();
        Rat r;
        r.n_ = static_cast<int64_t>(n);
        r.d_ = static_cast<int64_t>(d);
        return r;
    }

    int64_t num() const { return n_; }
    int64_t den() const { return d_; }
    bool is_zero() const { return n_ == 0; }

    friend Rat operator+(const Rat& a, const Rat& b) {
        return from128(static_cast<i128>(a.n_) * b.d_ + static_cast<i128>(b.n_) * a.d_,
                       static_cast<i128>(a.d_) * b.d_);
    }
    friend Rat operator-(const Rat& a, const Rat& b) {
        return from128(static_cast<i128>(a.n_) * b.d_ - static_cast<i128>(b.n_) * a.d_,
                       static_cast<i128>(a.d_) * b.d_);
    }
    friend Rat operator*(const Rat& a, const Rat& b) {
        return from128(static_cast<i128>(a.n_) * b.n_, static_cast<i128>(a.d_) * b.d_);
    }
    friend Rat operator/(const Rat& a, const Rat& b) {
        if (b.n_ == 0) throw std::domain_error("division by zero");
        return from128(static_cast<i128>(a.n_) * b.d_, static_cast<i128>(a.d_) * b.n_);
    }
    Rat operator-() const { return from128(-static_cast<i128>(n_), d_); }
    Rat& operator+=(const Rat& b) { return *this = *this + b; }
    Rat& operator-=(const Rat& b) { return *this = *this - b; }
    friend bool operator==(const Rat& a, const Rat& b) { return a.n_ == b.n_ && a.d_ == b.d_; }
    friend bool operator!=(const Rat& a, const Rat& b) { return !(a == b); }

    // Nearest fp32 value, ties to even (exact long division, no double rounding).
    float to_f32() const;

    std::string str() const {
        return d_ == 1 ? std::to_string(n_) : std::to_string(n_) + "/" + std::to_string(d_);
    }

private:
    void set(int64_t n, int64_t d) { *this = from128(n, d); }
    int64_t n_, d_;
};

// Polynomial over Q, coefficients lowest power first, no trailing zeros
// (the zero polynomial is empty).  This is the paper's vec() order.
class Poly {
public:
    Poly() = default;
    explicit Poly(std::vector<Rat> c) : c_(std::move(c)) { trim(); }
    static Poly monomial(int k) {
        std::vector<Rat> c(static_cast<size_t>(k) + 1, Rat(0));
        c[static_cast<size_t>(k)] = Rat(1);
        return Poly(c);
    }
    static Poly constant(Rat v) { return Poly(std::vector<Rat>{v}); }

    int deg() const { return static_cast<int>(c_.size()) - 1; }
    bool is_zero() const { return c_.empty(); }
    Rat coef(int i) const { return i >= 0 && i < static_cast<int>(c_.size()) ? c_[static_cast<size_t>(i)] : Rat(0); }
    Rat lead() const { return c_.back(); }
    const std::vector<Rat>& coeffs() const { return c_; }

    friend Poly operator+(const Poly& a, const Poly& b) {
        size_t n = std::max(a.c_.size(), b.c_.size());
        std::vector<Rat> c(n);
        for (size_t i = 0; i < n; ++i) c[i] = a.coef(static_cast<int>(i)) + b.coef(static_cast<int>(i));
        return Poly(c);
    }
    friend Poly operator-(const Poly& a, const Poly& b) {
        size_t n = std::max(a.c_.size(), b.c_.size());
        std::vector<Rat> c(n);
        for (size_t i = 0; i < n; ++i) c[i] = a.coef(static_cast<int>(i)) - b.coef(static_cast<int>(i));
        return Poly(c);
    }
    friend Poly operator*(const Poly& a, const Poly& b) {
        if (a.is_zero() || b.is_zero()) return Poly();
        std::vector<Rat> c(a.c_.size() + b.c_.size() - 1);
        for (size_t i = 0; i < a.c_.size(); ++i)
            for (size_t j = 0; j < b.c_.size(); ++j) c[i + j] += a.c_[i] * b.c_[j];
        return Poly(c);
    }
    Poly scaled(const Rat& s) const {
        std::vector<Rat> c(c_);
        for (auto& v : c) v = v * s;
        return Poly(c);
    }

    // Division with remainder: *this = q * b + r, deg r < deg b.
    void divmod(const Poly& b, Poly* q, Poly* r) const;
    Poly rem(const Poly& m) const { Poly q, r; divmod(m, &q, &r); return r; }
    Poly exact_div(const Poly& b) const;
    Poly monic() const { return scaled(Rat(1) / lead()); }
    Rat eval(const Rat& x) const {
        Rat acc(0);
        for (size_t i = c_.size(); i-- > 0;) acc = acc * x + c_[i];
        return acc;
    }
    // vec() padded with zeros to length n.
    std::vector<Rat> vec(int n) const;

    friend bool operator==(const Poly& a, const Poly& b) { return a.c_ == b.c_; }

private:
    void trim() { while (!c_.empty() && c_.back().is_zero()) c_.pop_back(); }
    std::vector<Rat> c_;
};

// gcd (monic) and Bezout coefficient s with s*f + t*g = gcd.
Poly poly_gcd(const Poly& f, const Poly& g, Poly* s_out);
// N with N*f = 1 (mod m), deg N < deg m  (the N_i of eq. (1)); throws if not coprime.
Poly inverse_mod(const Poly& f, const Poly& m);
// True iff the rational q is the square of a rational.
bool is_rational_square(const Rat& q);

}  // namespace wg
