// Host-side construction of the Winograd transforms by the polynomial CRT
// (Barabasz & Gregg, arXiv 1905.05233, Section 2.2, Algorithms 1 and 2).
#pragma once

#include <stdexcept>
#include <string>
#include <vector>

#include "rational.hpp"

namespace wg {

// Error with a wg_status code (values of the C enum in winograd_crt.h).
struct PlanError : std::runtime_error {
    PlanError(int code, const std::string& msg) : std::runtime_error(msg), status(code) {}
    int status;
};

enum : int {
    kErrArg = 1, kErrDegreeSum = 2, kErrNotCoprime = 3, kErrReducible = 4,
    kErrUnsupported = 5, kErrOverflow = 6, kErrInternal = 9
};

// One modulus m_i(a) or the pseudo-point infinity.
struct Modulus {
    bool inf = false;
    Poly p;  // monic for finite moduli
};

struct Transforms {
    int m = 0, r = 0, alpha = 0, tile_in = 0;
    // exact matrices, row-major: G alpha x r, A alpha x m, B tile_in x alpha
    std::vector<Rat> G, A, B;
    // the same rounded once to fp32, nearest even
    std::vector<float> Gf, Af, Bf;
};

// Parse "0,1,-1,1/2,a^2+1,inf" (points mean a - p).  Throws PlanError(kErrArg).
std::vector<Modulus> parse_moduli(const std::string& text);
// Parse "0,-1,inf" into finite points and the infinity flag.
void parse_points(const std::string& text, std::vector<Rat>* pts, bool* with_inf);

// Algorithms 1 and 2 for F(m x m, r x r) plus the exact reconstruction check.
// factors_in_g moves the CRT factors N_i of eq. (1) from B (the paper's
// matrices) to the kernel transform G; scale_rows divides every domain row of
// G and of A by its 1-norm and compensates in B.
Transforms build_transforms(const std::vector<Modulus>& moduli, const std::vector<Rat>& inner_pts,
                            bool inner_inf, int m, int r, bool factors_in_g = false, bool scale_rows = false);

}  // namespace wg
