// Device-side storage types and conversions (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace wg {

// bf16 kept as its 16 raw bits; arithmetic is always done in fp32.
struct bf16_t { uint16_t bits; };

template <typename T> struct Storage;

template <> struct Storage<float> {
    static __device__ __forceinline__ float to_f32(float v) { return v; }
    static __device__ __forceinline__ float from_f32(float f) { return f; }
};

template <> struct Storage<_Float16> {
    static __device__ __forceinline__ float to_f32(_Float16 v) { return static_cast<float>(v); }
    // IEEE conversion, round to nearest even (the default rounding mode), of
    // the value as rounded to fp32.  The empty asm keeps the compiler from
    // folding a preceding fp32 fma into the conversion (v_fma_mix*_f16, one
    // rounding straight to fp16), which would skip the fp32 rounding.
    static __device__ __forceinline__ _Float16 from_f32(float f) {
        asm("" : "+v"(f));
        return static_cast<_Float16>(f);
    }
};

template <> struct Storage<bf16_t> {
    static __device__ __forceinline__ float to_f32(bf16_t v) {
        return __uint_as_float(static_cast<uint32_t>(v.bits) << 16);
    }
    // Round to nearest even (v_cvt_pk_bf16_f32 on gfx950); NaN stays a NaN.
    static __device__ __forceinline__ bf16_t from_f32(float f) {
        bf16_t r;
        r.bits = __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
        return r;
    }
};

template <int D> struct DTypeOf;
template <> struct DTypeOf<0> { using type = float; };
template <> struct DTypeOf<1> { using type = _Float16; };
template <> struct DTypeOf<2> { using type = bf16_t; };

// Buffer descriptors (gfx950): loads at an offset past the record count return
// zero and stores there are dropped, which clips ragged tails without branches.
constexpr uint32_t kRsrcWord3 = 0x00020000u;   // raw 32-bit buffer, gfx9 family
constexpr uint32_t kOob = 0xfffffff0u;         // an offset beyond every record count used here

// Buffer descriptor over [base, base + bytes), bytes clipped to [0, 2^32 - 1].
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
    const int64_t n = bytes < 0 ? 0 : (bytes > 0xffffffffLL ? 0xffffffffLL : bytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                             static_cast<int>(static_cast<uint32_t>(n)),
                                             static_cast<int>(kRsrcWord3));
}

// --- LDS fragment reads issued from inline assembly ------------------------
// The compiler inserts its waits for LDS reads it issues itself, and cannot
// tell the buffers of a software pipeline apart; reads issued from inline
// assembly are waited for explicitly with lds_settle*, whose in/out operands
// tie the values to the wait.  LDS reads of a wave complete in issue order,
// so lgkmcnt(n) means every read except the last n issued has arrived (scalar
// loads in flight only lower that count).  Every operand of one wait must be
// a different variable: one bound twice gets a copy made before the wait,
// which reads the register while its load is still in flight.
typedef unsigned int lds_u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ lds_u32x4 lds_read16(const unsigned char* p) {
    const uint32_t a = static_cast<uint32_t>(
        reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const unsigned char*)p));
    lds_u32x4 v;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a) : "memory");
    return v;
}

// wait for every LDS read of this wave
__device__ __forceinline__ void lds_settle(lds_u32x4& a, lds_u32x4& b) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b) : : "memory");
}
__device__ __forceinline__ void lds_settle(lds_u32x4& a, lds_u32x4& b, lds_u32x4& c) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b), "+v"(c) : : "memory");
}
__device__ __forceinline__ void lds_settle(lds_u32x4& a, lds_u32x4& b, lds_u32x4& c, lds_u32x4& d) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d) : : "memory");
}
__device__ __forceinline__ void lds_settle(lds_u32x4& a, lds_u32x4& b, lds_u32x4& c, lds_u32x4& d, lds_u32x4& e,
                                           lds_u32x4& f) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d), "+v"(e), "+v"(f) : : "memory");
}
// wait for all but the last two LDS reads of this wave
__device__ __forceinline__ void lds_settle_but2(lds_u32x4& a, lds_u32x4& b) {
    asm volatile("s_waitcnt lgkmcnt(2)" : "+v"(a), "+v"(b) : : "memory");
}

}  // namespace wg
