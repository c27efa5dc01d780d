// Winograd-domain contraction on the gfx950 matrix cores.
//
// eq. (2) of Barabasz & Gregg (arXiv 1905.05233) multiplies the transformed
// kernel and input tiles elementwise (the Hadamard product, Section 2.3: the
// "elementwise multiplications" that dominate the run time).  Summed over the
// C input channels of a DNN layer, each of the alpha'^2 domain points xi is an
// independent GEMM:
//
//     M[xi][t][k] = sum_c V[xi][t][c] * U[xi][k][c]      ([T x C] . [C x K])
//
// Both operands are channel-contiguous, so both MFMA operands stream along the
// reduction dimension.  A 256-thread workgroup computes a 128 x 128 block of
// one xi with four wavefronts of 64 x 64 (2 x 2 MFMA tiles of 32 x 32);
// k-tiles of 128 bytes per row are staged through double-buffered LDS (rows
// padded to 144 bytes, which keeps the 16-byte fragment reads conflict-free),
// with the next k-tile's global loads in flight during the current MFMAs.
// fp32 uses v_mfma_f32_32x32x2_f32; fp16 and bf16 use
// v_mfma_f32_32x32x16_{f16,bf16}; the accumulator is fp32 for every dtype.
//
// Inside a k-tile each lane half (lanes 0-31 / 32-63) owns one contiguous half
// of the k range, so every fragment is a 16-byte LDS read; the reduction order
// differs from the textbook lane layout but covers each k exactly once with
// the same (row, k) / (col, k) pairing on both operands.
#include "device_common.hpp"
#include "kernels.hpp"

namespace wg {

namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kBM = 128;                 // rows (tiles) per workgroup
constexpr int kBN = 128;                 // columns (output channels) per workgroup
constexpr int kRowChunks = 8;            // 16-byte chunks per k-tile row (128 bytes)
constexpr int kLdsChunks = kRowChunks + 1;   // + one chunk of padding

template <int D> __device__ __forceinline__ void mma_chunk(const u32x4& a, const u32x4& b, f32x16& c);

template <> __device__ __forceinline__ void mma_chunk<0>(const u32x4& a, const u32x4& b, f32x16& c) {
    const f32x4 av = __builtin_bit_cast(f32x4, a);
    const f32x4 bv = __builtin_bit_cast(f32x4, b);
#pragma unroll
    for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_32x32x2f32(av[e], bv[e], c, 0, 0, 0);
}

template <> __device__ __forceinline__ void mma_chunk<1>(const u32x4& a, const u32x4& b, f32x16& c) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                               0, 0);
}

template <> __device__ __forceinline__ void mma_chunk<2>(const u32x4& a, const u32x4& b, f32x16& c) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                0, 0, 0);
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void contract_kernel(const unsigned char* __restrict__ V,
                                                              const unsigned char* __restrict__ U,
                                                              float* __restrict__ M, int64_t T, int64_t K,
                                                              int64_t row_bytes, int64_t Kp, int num_mb,
                                                              int num_nb) {
    __shared__ u32x4 lds[2][(kBM + kBN) * kLdsChunks];

    int bid = blockIdx.x;
    const int nb = bid % num_nb;
    bid /= num_nb;
    const int mb = bid % num_mb;
    const int xi = bid / num_mb;
    const unsigned char* Vb = V + static_cast<int64_t>(xi) * T * row_bytes;
    const unsigned char* Ub = U + static_cast<int64_t>(xi) * K * row_bytes;
    float* Mb = M + static_cast<int64_t>(xi) * T * Kp;
    const int64_t m0 = static_cast<int64_t>(mb) * kBM;
    const int64_t n0 = static_cast<int64_t>(nb) * kBN;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1;
    const int wn = wave & 1;
    const int half = lane >> 5;
    const int r32 = lane & 31;

    // global -> register staging: 4 chunks of A and 4 of B per thread
    const int lrow = tid >> 3;          // 0..31, + 32 p
    const int lcol = tid & 7;
    u32x4 ra[4], rb[4];
    const u32x4 zero = {0u, 0u, 0u, 0u};

    auto gload = [&](int kt) {
        const int64_t byte = static_cast<int64_t>(kt) * (kRowChunks * 16) + lcol * 16;
        const bool kin = byte < row_bytes;  // row_bytes is a multiple of 16
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const int64_t gm = m0 + lrow + 32 * p;
            const int64_t gn = n0 + lrow + 32 * p;
            ra[p] = (kin && gm < T) ? *reinterpret_cast<const u32x4*>(Vb + gm * row_bytes + byte) : zero;
            rb[p] = (kin && gn < K) ? *reinterpret_cast<const u32x4*>(Ub + gn * row_bytes + byte) : zero;
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            lds[buf][(lrow + 32 * p) * kLdsChunks + lcol] = ra[p];
            lds[buf][(kBM + lrow + 32 * p) * kLdsChunks + lcol] = rb[p];
        }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    const int nk = static_cast<int>((row_bytes + kRowChunks * 16 - 1) / (kRowChunks * 16));
    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) gload(kt + 1);
        const u32x4* L = lds[buf];
        const int arow0 = (wm * 64 + r32) * kLdsChunks;
        const int arow1 = (wm * 64 + 32 + r32) * kLdsChunks;
        const int brow0 = (kBM + wn * 64 + r32) * kLdsChunks;
        const int brow1 = (kBM + wn * 64 + 32 + r32) * kLdsChunks;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int ch = half * 4 + q;
            const u32x4 a0 = L[arow0 + ch];
            const u32x4 a1 = L[arow1 + ch];
            const u32x4 b0 = L[brow0 + ch];
            const u32x4 b1 = L[brow1 + ch];
            mma_chunk<D>(a0, b0, acc[0][0]);
            mma_chunk<D>(a0, b1, acc[0][1]);
            mma_chunk<D>(a1, b0, acc[1][0]);
            mma_chunk<D>(a1, b1, acc[1][1]);
        }
        if (kt + 1 < nk) sstore(buf ^ 1);
        __syncthreads();
    }

    // 32x32 accumulator layout: lane holds column r32, rows 8*(r/4) + 4*half + r%4
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t col = n0 + wn * 64 + j * 32 + r32;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
                if (row < T && col < K) Mb[row * Kp + col] = acc[i][j][r];
            }
        }
}

}  // namespace

template <int D>
hipError_t launch_contract_t(const Geometry& g, const void* V, const void* U, float* M, hipStream_t stream) {
    const int64_t es = D == 0 ? 4 : 2;
    const int64_t row_bytes = g.Cp * es;
    const int num_mb = static_cast<int>((g.T + kBM - 1) / kBM);
    const int num_nb = static_cast<int>((g.K + kBN - 1) / kBN);
    const int64_t blocks = static_cast<int64_t>(num_mb) * num_nb * g.alpha * g.alpha;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL(contract_kernel<D>, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream,
                       static_cast<const unsigned char*>(V), static_cast<const unsigned char*>(U), M, g.T, g.K,
                       row_bytes, g.Kp, num_mb, num_nb);
    return hipGetLastError();
}

template hipError_t launch_contract_t<0>(const Geometry&, const void*, const void*, float*, hipStream_t);
template hipError_t launch_contract_t<1>(const Geometry&, const void*, const void*, float*, hipStream_t);
template hipError_t launch_contract_t<2>(const Geometry&, const void*, const void*, float*, hipStream_t);

}  // namespace wg
