"""Exact polynomial arithmetic over the rationals (oracle; test infrastructure only).

A polynomial is a tuple of ``fractions.Fraction`` coefficients, lowest degree
first, with no trailing zeros (the zero polynomial is ``()``).  This is the
coefficient order of the paper's vec(.) map (Section 2.2: vec(m(a)) lists
m_1 .. m_n for m(a) = m_1 + m_2 a + ... + m_n a^(n-1)).

Everything here is textbook algebra in the ring Q[a] (Section 2.1): products,
division with remainder, the remainder R_m[p] and the extended Euclidean
algorithm that yields the CRT coefficients N_i with N_i M_i + n_i m_i = 1
(eq. (1)).
"""
from fractions import Fraction


def poly(coeffs):
    """Build a normalised polynomial from low-to-high coefficients."""
    c = [Fraction(v) for v in coeffs]
    while c and c[-1] == 0:
        c.pop()
    return tuple(c)


ZERO = ()
ONE = (Fraction(1),)
X = (Fraction(0), Fraction(1))


def deg(p):
    """Degree; the zero polynomial has degree -1."""
    return len(p) - 1


def add(p, q):
    n = max(len(p), len(q))
    return poly([(p[i] if i < len(p) else 0) + (q[i] if i < len(q) else 0) for i in range(n)])


def neg(p):
    return tuple(-v for v in p)


def sub(p, q):
    return add(p, neg(q))


def scale(p, s):
    return poly([v * Fraction(s) for v in p])


def mul(p, q):
    if not p or not q:
        return ZERO
    out = [Fraction(0)] * (len(p) + len(q) - 1)
    for i, a in enumerate(p):
        for j, b in enumerate(q):
            out[i + j] += a * b
    return poly(out)


def power_of_a(k):
    """The monomial a^k."""
    return poly([0] * k + [1])


def divmod_poly(p, q):
    """Long division: p = quo*q + rem with deg rem < deg q."""
    if not q:
        raise ZeroDivisionError("division by the zero polynomial")
    rem = list(p)
    dq = deg(q)
    lead = q[-1]
    quo = [Fraction(0)] * max(len(p) - dq, 0)
    while len(rem) - 1 >= dq and rem:
        shift = len(rem) - 1 - dq
        f = rem[-1] / lead
        quo[shift] = f
        for i, c in enumerate(q):
            rem[shift + i] -= f * c
        # the leading term is now exactly zero
        rem.pop()
        while rem and rem[-1] == 0:
            rem.pop()
    return poly(quo), poly(rem)


def rem(p, m):
    """R_m[p]: the remainder of p on division by m (Section 2.2)."""
    return divmod_poly(p, m)[1]


def exact_div(p, q):
    quo, r = divmod_poly(p, q)
    if r:
        raise ValueError("division is not exact")
    return quo


def monic(p):
    if not p:
        raise ValueError("zero polynomial has no monic form")
    return scale(p, 1 / p[-1])


def vec(p, n):
    """vec(p) padded with zeros to length n (Section 2.2); error if deg p >= n."""
    if len(p) > n:
        raise ValueError(f"polynomial of degree {deg(p)} does not fit a length-{n} vector")
    return [Fraction(v) for v in p] + [Fraction(0)] * (n - len(p))


def evaluate(p, x):
    acc = Fraction(0)
    for c in reversed(p):
        acc = acc * x + c
    return acc


def ext_euclid(f, g):
    """Extended Euclid over Q: returns (d, s, t) with s*f + t*g = d, d = monic gcd."""
    r0, r1 = f, g
    s0, s1 = ONE, ZERO
    t0, t1 = ZERO, ONE
    while r1:
        q, r = divmod_poly(r0, r1)
        r0, r1 = r1, r
        s0, s1 = s1, sub(s0, mul(q, s1))
        t0, t1 = t1, sub(t0, mul(q, t1))
    if not r0:
        raise ValueError("gcd of two zero polynomials")
    inv = 1 / r0[-1]
    return scale(r0, inv), scale(s0, inv), scale(t0, inv)


def inverse_mod(f, m):
    """N with N*f = 1 (mod m), deg N < deg m; from N f + n m = 1 (eq. (1))."""
    d, s, _ = ext_euclid(f, m)
    if d != ONE:
        raise ValueError("polynomials are not coprime")
    return rem(s, m)


def product(polys):
    out = ONE
    for p in polys:
        out = mul(out, p)
    return out


def is_square_rational(q):
    """True iff the rational q >= 0 is the square of a rational."""
    q = Fraction(q)
    if q < 0:
        return False
    from math import isqrt
    n, d = q.numerator, q.denominator
    rn, rd = isqrt(n), isqrt(d)
    return rn * rn == n and rd * rd == d


def parse(text):
    """Parse a polynomial in ``a`` such as ``a^2+1``, ``a^2-a+1``, ``2a-1/2``."""
    s = text.replace(" ", "").replace("**", "^").replace("*", "")
    if not s:
        raise ValueError("empty polynomial")
    terms = []
    cur = ""
    for ch in s:
        if ch in "+-" and cur and cur[-1] != "^":
            terms.append(cur)
            cur = ch
        else:
            cur += ch
    terms.append(cur)
    coeffs = {}
    for t in terms:
        sign = 1
        if t.startswith("+"):
            t = t[1:]
        elif t.startswith("-"):
            sign, t = -1, t[1:]
        if "a" in t:
            c, _, e = t.partition("a")
            coef = Fraction(c) if c else Fraction(1)
            if e:
                if not e.startswith("^"):
                    raise ValueError(f"bad term {t!r}")
                k = int(e[1:])
            else:
                k = 1
        else:
            coef, k = Fraction(t), 0
        coeffs[k] = coeffs.get(k, Fraction(0)) + sign * coef
    top = max(coeffs)
    return poly([coeffs.get(i, 0) for i in range(top + 1)])
