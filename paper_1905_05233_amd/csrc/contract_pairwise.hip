// Winograd-domain contraction with pairwise summation over the channels.
//
// The channel sum M[xi][t][k] = sum_c V[xi][t][c] U[xi][k][c] of eq. (2)
// (Barabasz & Gregg, arXiv 1905.05233) accumulates C products.  The related
// work of Section 4 names pairwise summation over the channels as a way to
// shrink its floating-point error: the sum's rounding error then grows with
// log2 C instead of C.  This kernel is that option of the library.
//
// One wavefront computes a 16 x 16 block (16 tiles x 16 output channels) of
// one domain point.  The channel rows are cut into leaves of 64 bytes (16
// fp32 or 32 fp16/bf16 channels; each lane group of 16 lanes loads one
// 16-byte piece of every row): a leaf's products are summed by the matrix
// core into a fresh fp32 accumulator (one 16x16x32 MFMA, or four chained
// 16x16x4 f32 MFMAs), and the leaves are added pairwise in channel order with
// a binary counter: level j holds the sum of a complete block of 2^j leaves,
// and a new leaf carries up through the occupied levels (earlier block on the
// left); at the end the occupied levels are added from the lowest up.  This is
// the pairwise tree over the leaves padded with zero leaves to a power of two
// (adding a zero changes nothing).  It favours accuracy over speed: fragments
// come straight from memory and nothing is staged.
#include <algorithm>

#include "device_common.hpp"
#include "kernels.hpp"

namespace wg {

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kPwWaves = 4;      // waves (items) per workgroup
constexpr int kLevels = 24;      // leaves per row below 2^24 (checked at launch)
constexpr int kLeafBytes = 64;   // four lane groups x 16 bytes

// the products of one leaf summed into a fresh fp32 accumulator
template <int D>
__device__ __forceinline__ f32x4 leaf_sum(const u32x4& a, const u32x4& b) {
    const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    if constexpr (D == 0) {
        const f32x4 av = __builtin_bit_cast(f32x4, a);
        const f32x4 bv = __builtin_bit_cast(f32x4, b);
        f32x4 c = __builtin_amdgcn_mfma_f32_16x16x4f32(av[0], bv[0], z, 0, 0, 0);
#pragma unroll
        for (int e = 1; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], bv[e], c, 0, 0, 0);
        return c;
    } else if constexpr (D == 1) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), z, 0,
                                                      0, 0);
    } else {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), z,
                                                       0, 0, 0);
    }
}

// MFMA rows are tiles (A = V), columns output channels (B = U): lane l holds
// M of tiles 4 (l / 16) + q, q < 4, for the output channel l % 16.
template <int D>
__global__ __launch_bounds__(kPwWaves * 64) void contract_pairwise_kernel(
    const unsigned char* __restrict__ V, const unsigned char* __restrict__ U, float* __restrict__ M, int64_t T,
    int64_t K, int64_t rb, int64_t Kp, int64_t num_tb, int64_t num_kb, int64_t n_items) {
    const int lane = threadIdx.x & 63;
    const int64_t item = static_cast<int64_t>(blockIdx.x) * kPwWaves + (threadIdx.x >> 6);
    if (item >= n_items) return;   // the same for every lane of the wave
    const int64_t kb = item % num_kb;
    const int64_t tb = (item / num_kb) % num_tb;
    const int64_t xi = item / (num_kb * num_tb);
    const int l16 = lane & 15, grp = lane >> 4;
    const int64_t t = tb * 16 + l16, k = kb * 16 + l16;
    const bool tin = t < T, kin = k < K;
    const unsigned char* vrow = V + (xi * T + (tin ? t : 0)) * rb;
    const unsigned char* urow = U + (xi * K + (kin ? k : 0)) * rb;
    const int64_t n_leaf = (rb + kLeafBytes - 1) / kLeafBytes;

    f32x4 lev[kLevels];
    for (int64_t i = 0; i < n_leaf; ++i) {
        const int64_t off = i * kLeafBytes + grp * 16;
        u32x4 a = {0u, 0u, 0u, 0u}, b = {0u, 0u, 0u, 0u};
        if (off < rb) {
            if (tin) a = *reinterpret_cast<const u32x4*>(vrow + off);
            if (kin) b = *reinterpret_cast<const u32x4*>(urow + off);
        }
        f32x4 v = leaf_sum<D>(a, b);
        // carry through the occupied levels: bit j of i set = level j occupied
        bool placed = false;
#pragma unroll
        for (int j = 0; j < kLevels; ++j) {
            if (!placed) {
                if ((i >> j) & 1) {
                    v = lev[j] + v;
                } else {
                    lev[j] = v;
                    placed = true;
                }
            }
        }
    }
    // the occupied levels (the bits of n_leaf), lowest first; later leaves on the right
    f32x4 r = {0.0f, 0.0f, 0.0f, 0.0f};
    bool any = false;
#pragma unroll
    for (int j = 0; j < kLevels; ++j) {
        if ((n_leaf >> j) & 1) {
            r = any ? lev[j] + r : lev[j];
            any = true;
        }
    }
    if (!kin) return;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int64_t tt = tb * 16 + 4 * grp + q;
        if (tt < T) M[(xi * T + tt) * Kp + k] = r[q];
    }
}

}  // namespace

template <int D>
hipError_t launch_contract_pairwise_t(const Geometry& g, const void* V, const void* U, float* M, hipStream_t stream) {
    const int64_t rb = g.Cp * (D == 0 ? 4 : 2);
    if ((rb + kLeafBytes - 1) / kLeafBytes >= (int64_t(1) << kLevels)) return hipErrorInvalidValue;
    const int64_t num_tb = (g.T + 15) / 16, num_kb = (g.K + 15) / 16;
    const int64_t n_items = g.planes * num_tb * num_kb;
    const int64_t blocks = (n_items + kPwWaves - 1) / kPwWaves;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL(contract_pairwise_kernel<D>, dim3(static_cast<unsigned>(blocks)), dim3(kPwWaves * 64), 0,
                       stream, static_cast<const unsigned char*>(V), static_cast<const unsigned char*>(U), M, g.T, g.K,
                       rb, g.Kp, num_tb, num_kb, n_items);
    return hipGetLastError();
}

template hipError_t launch_contract_pairwise_t<0>(const Geometry&, const void*, const void*, float*, hipStream_t);
template hipError_t launch_contract_pairwise_t<1>(const Geometry&, const void*, const void*, float*, hipStream_t);
template hipError_t launch_contract_pairwise_t<2>(const Geometry&, const void*, const void*, float*, hipStream_t);

}  // namespace wg
