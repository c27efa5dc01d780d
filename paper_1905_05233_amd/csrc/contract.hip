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
// reduction dimension.  Short reductions (a row of C within 512 bytes) use the
// streaming kernel further down.  For longer ones a 256-thread workgroup
// computes a 128 x 128 block of one xi with four wavefronts of 64 x 64 (2 x 2 MFMA tiles of 32 x 32);
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
#include <algorithm>

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


// ---------------------------------------------------------------------------
// Streaming variant for short reductions (one row of C fits 512 bytes: fp32
// C <= 128, fp16/bf16 C <= 256), the common DNN case.
//
// One persistent 512-thread workgroup per CU walks a contiguous range of work
// items; an item is 32 rows (tiles) x 128 columns (output channels) of one
// domain point xi, with the whole reduction.  Items are ordered xi-major, so a
// workgroup's consecutive items share U[xi]; workgroup ids are remapped so
// that the ranges of the workgroups of one XCD are adjacent (the hardware
// hands out consecutive ids round-robin across the 8 XCDs), which keeps each
// U[xi] in a single L2.  The 8 waves split the item into 2 row halves x 4
// groups of 32 columns; each wave runs the whole reduction on 16x16 MFMA
// tiles with four independent accumulators and keeps its U fragments in
// registers while xi and the column block stay the same (the U block of the
// next item, when it changes, is fetched one item ahead and parked in LDS).
// Only the V tile streams: loaded one item ahead into registers and parked in
// double-buffered LDS, its wait falling after a full MFMA phase.  The 32 x 128
// block of M is staged in LDS and written with full-row 16-byte stores.
constexpr int kStreamThreads = 512;
constexpr int kStreamRows = 32;
constexpr int kStreamCols = 128;

template <int D> __device__ __forceinline__ void mma16_chunk(const u32x4& a, const u32x4& b, f32x4& c);

template <> __device__ __forceinline__ void mma16_chunk<0>(const u32x4& a, const u32x4& b, f32x4& c) {
    const f32x4 av = __builtin_bit_cast(f32x4, a);
    const f32x4 bv = __builtin_bit_cast(f32x4, b);
#pragma unroll
    for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], bv[e], c, 0, 0, 0);
}

template <> __device__ __forceinline__ void mma16_chunk<1>(const u32x4& a, const u32x4& b, f32x4& c) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                               0, 0);
}

template <> __device__ __forceinline__ void mma16_chunk<2>(const u32x4& a, const u32x4& b, f32x4& c) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                0, 0, 0);
}

// One 16-byte chunk of A against the same chunk of two B column blocks.
template <int D>
__device__ __forceinline__ void mma16_chunk2(const u32x4& x, const u32x4& y0, const u32x4& y1, f32x4& c0,
                                             f32x4& c1) {
    if constexpr (D == 0) {
        const f32x4 a = __builtin_bit_cast(f32x4, x);
        const f32x4 b0 = __builtin_bit_cast(f32x4, y0), b1 = __builtin_bit_cast(f32x4, y1);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            c0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b0[e], c0, 0, 0, 0);
            c1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b1[e], c1, 0, 0, 0);
        }
    } else {
        mma16_chunk<D>(x, y0, c0);
        mma16_chunk<D>(x, y1, c1);
    }
}

template <int NCH>
struct StreamLds {
    // NCH = 16-byte chunks per lane per 16-row block: the k range of a row is
    // 64 * NCH bytes, split over the four 16-lane groups of a wave.
    static constexpr int kRowBytes = 64 * NCH + 16;                   // + padding: conflict-free reads
    static constexpr int kABytes = kStreamRows * kRowBytes;           // one V tile (32 rows)
    static constexpr int kBBytes = kStreamCols * kRowBytes;           // one U block (128 columns)
    static constexpr int kORowFloats = kStreamCols + 4;               // output staging row (+ padding)
    static constexpr int kOBytes = kStreamRows * kORowFloats * 4;     // one 32 x 128 fp32 tile of M
    static constexpr int kUsed = 2 * kABytes + kBBytes + 2 * kOBytes;
    // at least 84 KB: more than half of a CU's 160 KB, so one workgroup per CU
    static constexpr int kBytes = kUsed > 84 * 1024 ? kUsed : 84 * 1024;
    static_assert(kUsed <= 160 * 1024, "LDS layout");
};


template <int D, int NCH>
__global__ __launch_bounds__(kStreamThreads, 1) void contract_stream_kernel(
    const unsigned char* __restrict__ V, const unsigned char* __restrict__ U, float* __restrict__ M, int64_t T,
    int64_t K, int64_t row_bytes, int64_t Kp, int num_mb, int num_nb, int64_t n_items) {
    using L = StreamLds<NCH>;
    __shared__ __attribute__((aligned(16))) unsigned char smem[L::kBytes];
    unsigned char* const abuf = smem;                   // [2][32 rows][kRowBytes]
    unsigned char* const bbuf = smem + 2 * L::kABytes;  // [128 cols][kRowBytes]
    float* const obuf = reinterpret_cast<float*>(smem + 2 * L::kABytes + L::kBBytes);  // [2][32][132]

    // XCD-aware contiguous item range of this workgroup
    const int64_t G = gridDim.x;
    const int64_t bid = blockIdx.x;
    const int64_t v = (G % 8 == 0) ? (bid % 8) * (G / 8) + bid / 8 : bid;
    const int64_t it0 = v * n_items / G;
    const int64_t it1 = (v + 1) * n_items / G;
    if (it0 >= it1) return;
    const int n_mine = static_cast<int>(it1 - it0);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int rh = wave >> 2;              // 16-row half of the item
    const int cg = wave & 3;               // 32-column group
    const int grp = lane >> 4;
    const int l16 = lane & 15;
    const int kbyte0 = grp * (16 * NCH);   // each 16-lane group owns a quarter of the k range
    const u32x4 zero = {0u, 0u, 0u, 0u};

    // staging map: chunk ci -> (row, 16-byte column) of a tile row of 64*NCH bytes
    constexpr int kRowChunks = 4 * NCH;
    constexpr int kAChunks = kStreamRows * kRowChunks;
    constexpr int kAPer = (kAChunks + kStreamThreads - 1) / kStreamThreads;
    constexpr int kBChunks = kStreamCols * kRowChunks;
    constexpr int kBPer = (kBChunks + kStreamThreads - 1) / kStreamThreads;

    int xi = static_cast<int>(it0 / (static_cast<int64_t>(num_mb) * num_nb));
    int nb = static_cast<int>((it0 / num_mb) % num_nb);
    int mb = static_cast<int>(it0 % num_mb);

    // U block of (xi, nb): global -> registers, registers -> LDS (all threads;
    // the caller synchronises around the LDS write)
    u32x4 breg[kBPer];
    auto load_b = [&](int bxi, int bnb) {
        const unsigned char* src = U + static_cast<int64_t>(bxi) * K * row_bytes;
#pragma unroll
        for (int p = 0; p < kBPer; ++p) {
            const int ci = tid + p * kStreamThreads;
            const int col = ci / kRowChunks;
            const int c16 = ci % kRowChunks;
            const int64_t gcol = static_cast<int64_t>(bnb) * kStreamCols + col;
            const bool ok = ci < kBChunks && gcol < K && c16 * 16 < row_bytes;
            breg[p] = ok ? *reinterpret_cast<const u32x4*>(src + gcol * row_bytes + c16 * 16) : zero;
        }
    };
    auto store_b = [&]() {
#pragma unroll
        for (int p = 0; p < kBPer; ++p) {
            const int ci = tid + p * kStreamThreads;
            if (ci < kBChunks)
                *reinterpret_cast<u32x4*>(bbuf + (ci / kRowChunks) * L::kRowBytes + (ci % kRowChunks) * 16) =
                    breg[p];
        }
    };
    // V tile rows [mb*32, mb*32+32) of xi -> registers
    u32x4 areg[kAPer];
    auto load_a = [&](int axi, int amb) {
        const unsigned char* src = V + static_cast<int64_t>(axi) * T * row_bytes;
#pragma unroll
        for (int p = 0; p < kAPer; ++p) {
            const int ci = tid + p * kStreamThreads;
            const int row = ci / kRowChunks;
            const int c16 = ci % kRowChunks;
            const int64_t grow = static_cast<int64_t>(amb) * kStreamRows + row;
            const bool ok = ci < kAChunks && grow < T && c16 * 16 < row_bytes;
            areg[p] = ok ? *reinterpret_cast<const u32x4*>(src + grow * row_bytes + c16 * 16) : zero;
        }
    };
    auto store_a = [&](int slot) {
#pragma unroll
        for (int p = 0; p < kAPer; ++p) {
            const int ci = tid + p * kStreamThreads;
            if (ci < kAChunks)
                *reinterpret_cast<u32x4*>(abuf + slot * L::kABytes + (ci / kRowChunks) * L::kRowBytes +
                                          (ci % kRowChunks) * 16) = areg[p];
        }
    };

    // prologue: first U block and V tile in LDS (loads issued together), the
    // second V tile in flight
    load_b(xi, nb);
    load_a(xi, mb);
    store_b();
    store_a(0);
    int nxi = xi, nnb = nb, nmb = mb;
    auto advance = [&](int& a, int& b, int& c) {
        if (++c == num_mb) {
            c = 0;
            if (++b == num_nb) {
                b = 0;
                ++a;
            }
        }
    };
    advance(nxi, nnb, nmb);
    if (n_mine > 1) load_a(nxi, nmb);
    __syncthreads();

    // this wave's U fragments (two 16-column blocks), refreshed from LDS when
    // the U block changes
    u32x4 fy0[NCH], fy1[NCH];
    auto frag_b = [&]() {
        const unsigned char* b0 = bbuf + (cg * 32 + l16) * L::kRowBytes + kbyte0;
        const unsigned char* b1 = b0 + 16 * L::kRowBytes;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            fy0[c] = *reinterpret_cast<const u32x4*>(b0 + c * 16);
            fy1[c] = *reinterpret_cast<const u32x4*>(b1 + c * 16);
        }
    };
    frag_b();

    int slot = 0;
    for (int i = 0; i < n_mine; ++i) {
        // the next item's U block, if it changes, is fetched during this item
        const bool new_b = i + 1 < n_mine && (nxi != xi || nnb != nb);
        if (new_b) load_b(nxi, nnb);
        // 16 rows x 32 columns of this wave: four accumulators (two column
        // blocks x even/odd chunks) so consecutive MFMAs are independent
        f32x4 acc[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[q] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        const unsigned char* arow = abuf + slot * L::kABytes + (rh * 16 + l16) * L::kRowBytes + kbyte0;
        u32x4 fx[NCH];
#pragma unroll
        for (int c = 0; c < NCH; ++c) fx[c] = *reinterpret_cast<const u32x4*>(arow + c * 16);
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int q = c & 1;
            mma16_chunk2<D>(fx[c], fy0[c], fy1[c], acc[q], acc[2 + q]);
        }
        const bool has_next = i + 1 < n_mine;
        // park the next item's V tile (in flight since the previous item)
        if (has_next) store_a(slot ^ 1);
        // stage the 32 x 128 block of M in LDS (16x16 accumulator layout: lane
        // holds column l16, rows 4*grp + r of each 16-row block)
        float* ob = obuf + slot * (L::kOBytes / 4);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float* orow = ob + (rh * 16 + 4 * grp + r) * L::kORowFloats + cg * 32 + l16;
            orow[0] = acc[0][r] + acc[1][r];
            orow[16] = acc[2][r] + acc[3][r];
        }
        __syncthreads();
        // full-row 16-byte stores: 32 rows x 32 chunks of 4 floats
        {
            float* Mx = M + static_cast<int64_t>(xi) * T * Kp;
            const int64_t col0 = static_cast<int64_t>(nb) * kStreamCols;
#pragma unroll
            for (int p = 0; p < 2; ++p) {
                const int ci = tid + p * kStreamThreads;
                const int row = ci >> 5;
                const int c4 = (ci & 31) * 4;
                const int64_t grow = static_cast<int64_t>(mb) * kStreamRows + row;
                const int64_t gcol = col0 + c4;
                if (grow < T && gcol < K) {
                    const f32x4 val = *reinterpret_cast<const f32x4*>(ob + row * L::kORowFloats + c4);
                    float* dst = Mx + grow * Kp + gcol;
                    if (gcol + 4 <= Kp) {
                        *reinterpret_cast<f32x4*>(dst) = val;
                    } else {
                        for (int e = 0; e < 4 && gcol + e < K; ++e) dst[e] = val[e];
                    }
                }
            }
        }
        if (has_next) {
            xi = nxi;
            nb = nnb;
            mb = nmb;
            advance(nxi, nnb, nmb);
            if (new_b) {
                // all waves are past their reads of the old block (barrier above)
                store_b();
                __syncthreads();
                frag_b();
            }
            if (i + 2 < n_mine) load_a(nxi, nmb);
        }
        slot ^= 1;
    }
}

int device_cu_count() {
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cache[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        cache[dev] = n;
    }
    return cache[dev];
}

template <int D, int NCH>
hipError_t launch_stream(const Geometry& g, const void* V, const void* U, float* M, int64_t row_bytes,
                         hipStream_t stream) {
    const int num_mb = static_cast<int>((g.T + kStreamRows - 1) / kStreamRows);
    const int num_nb = static_cast<int>((g.K + kStreamCols - 1) / kStreamCols);
    const int64_t n_items = static_cast<int64_t>(num_mb) * num_nb * g.alpha * g.alpha;
    const int64_t grid = std::min<int64_t>(n_items, device_cu_count());
    hipLaunchKernelGGL((contract_stream_kernel<D, NCH>), dim3(static_cast<unsigned>(grid)), dim3(kStreamThreads), 0,
                       stream, static_cast<const unsigned char*>(V), static_cast<const unsigned char*>(U), M, g.T,
                       g.K, row_bytes, g.Kp, num_mb, num_nb, n_items);
    return hipGetLastError();
}

}  // namespace

template <int D>
hipError_t launch_contract_t(const Geometry& g, const void* V, const void* U, float* M, hipStream_t stream) {
    const int64_t es = D == 0 ? 4 : 2;
    const int64_t row_bytes = g.Cp * es;
    if (row_bytes <= 64) return launch_stream<D, 1>(g, V, U, M, row_bytes, stream);
    if (row_bytes <= 128) return launch_stream<D, 2>(g, V, U, M, row_bytes, stream);
    if (row_bytes <= 256) return launch_stream<D, 4>(g, V, U, M, row_bytes, stream);
    if (row_bytes <= 512) return launch_stream<D, 8>(g, V, U, M, row_bytes, stream);
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
