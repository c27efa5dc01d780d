// Transform coefficients on the device, shared by the transform kernels and
// the fused contraction: read from the kernel-argument tables (any plan) or,
// for the built-in plans, compile-time constants, with which the compiler
// drops every term whose coefficient is zero.  Dropping a zero term leaves the
// sum unchanged for finite data (up to the sign of a zero result).
#pragma once

#include "builtin_plans.hpp"
#include "kernels.hpp"

namespace wg {

struct RuntimeCoefs {
    static constexpr bool kConst = false;
    static __device__ __forceinline__ float bt(const InputTable& t, int i) { return t.bt[i]; }
    static __device__ __forceinline__ float at(const OutputTable& t, int i) { return t.at[i]; }
};
template <class P> struct ConstCoefs {
    static constexpr bool kConst = true;
    static __device__ __forceinline__ constexpr float bt(const InputTable&, int i) { return P::bt[i]; }
    static __device__ __forceinline__ constexpr float at(const OutputTable&, int i) { return P::at[i]; }
};
// acc + c * x as one fused multiply-add; skipped for a compile-time zero c
template <class CO> __device__ __forceinline__ float term(float c, float x, float acc) {
    if (CO::kConst && c == 0.0f) return acc;
    return __builtin_fmaf(c, x, acc);
}

}  // namespace wg
