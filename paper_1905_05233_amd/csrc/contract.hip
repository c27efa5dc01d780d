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

    // XCD-aware numbering: the hardware deals workgroup ids round-robin over
    // the 8 XCDs, each with its own L2; giving each XCD a contiguous run of
    // blocks keeps the column blocks of one row block (same V rows) and the
    // row blocks of one domain point (same U plane) in one L2, instead of V
    // being fetched from HBM once per XCD that needs it
    const int64_t G = gridDim.x;
    const int64_t b0 = blockIdx.x;
    const int64_t xcd = b0 % 8;
    int bid = static_cast<int>(xcd * (G / 8) + std::min<int64_t>(xcd, G % 8) + b0 / 8);
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

    // global -> register staging: 4 chunks of A and 4 of B per thread, in two
    // register sets, so that two k-tiles are in flight while one is computed
    const int lrow = tid >> 3;          // 0..31, + 32 p
    const int lcol = tid & 7;
    u32x4 ra[2][4], rb[2][4];
    // buffer descriptors over the block's own rows: rows past T or K and
    // bytes past the row read zero, with no branch (a branch per load would
    // make the compiler wait for every load in flight where the paths join);
    // the launcher checks that 128 rows stay below the out-of-range offset
    const auto rv = make_rsrc(Vb + m0 * row_bytes, (T - m0 < kBM ? T - m0 : kBM) * row_bytes);
    const auto ru = make_rsrc(Ub + n0 * row_bytes, (K - n0 < kBN ? K - n0 : kBN) * row_bytes);

    auto gload = [&](int set, int kt) __attribute__((always_inline)) {
        const int64_t byte = static_cast<int64_t>(kt) * (kRowChunks * 16) + lcol * 16;
        const bool kin = byte < row_bytes;  // row_bytes is a multiple of 16
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const uint32_t off = static_cast<uint32_t>((lrow + 32 * p) * row_bytes + byte);
            ra[set][p] = __builtin_amdgcn_raw_buffer_load_b128(rv, kin ? off : kOob, 0, 0);
            rb[set][p] = __builtin_amdgcn_raw_buffer_load_b128(ru, kin ? off : kOob, 0, 0);
        }
    };
    auto sstore = [&](int set, int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            lds[buf][(lrow + 32 * p) * kLdsChunks + lcol] = ra[set][p];
            lds[buf][(kBM + lrow + 32 * p) * kLdsChunks + lcol] = rb[set][p];
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
    // k-tile kt is loaded into register set kt % 2 two k-tiles ahead and
    // parked in LDS buffer kt % 2 one k-tile ahead
    auto compute = [&](int buf) __attribute__((always_inline)) {
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
    };
    // the loads are issued unconditionally (k-tiles past the row read zero):
    // a load behind a branch would make the compiler drain every load in
    // flight where the paths join
    gload(0, 0);
    gload(1, 1);
    sstore(0, 0);
    __syncthreads();
    for (int kt = 0; kt < nk; kt += 2) {
        // even k-tile: computed from buffer 0, its set refilled with kt + 2
        gload(0, kt + 2);
        compute(0);
        if (kt + 1 < nk) sstore(1, 1);
        __syncthreads();
        if (kt + 1 >= nk) break;
        // odd k-tile: buffer 1, set 1 refilled with kt + 3
        gload(1, kt + 3);
        compute(1);
        if (kt + 2 < nk) sstore(0, 0);
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
// One persistent workgroup per CU walks a contiguous range of work items; an
// item is 32 rows (tiles) x 128 columns (output channels) of one domain point
// xi, with the whole reduction.  Items are ordered xi-major, so consecutive
// items share U[xi]; workgroup ids are remapped so that the ranges of the
// workgroups of one XCD are adjacent (the hardware hands out consecutive ids
// round-robin across the 8 XCDs), which keeps each U[xi] in a single L2.
//
// The workgroup is split by role.  The loader waves (wave 8, and wave 9 for
// rows of up to 256 bytes) stream V tiles through registers into
// double-buffered LDS, two or four tiles in flight; they issue nothing but
// loads, so each of their waits covers exactly the tile they need.
// Waves 0-7 each own 32 rows x 16 columns of the item: their U fragments stay
// in registers while the block is unchanged (the next block is fetched one
// item ahead), A fragments come from LDS, and the finished block of M is
// stored straight from the accumulators.  These waves issue no global load in
// the steady state, so their stores are never waited on.  All global accesses
// go through buffer descriptors whose record counts clip the ragged tails
// (out-of-range loads return zero, out-of-range stores are dropped).
constexpr int kStreamMmaWaves = 8;
// Loader waves and the V tiles each keeps in flight (register sets), by row
// length: short rows make short MFMA phases and need a deeper prefetch; for
// 512-byte rows a second loader (a third wave on two SIMDs) measured slower.
constexpr int stream_loaders(int nch) { return nch >= 8 ? 1 : 2; }
constexpr int stream_sets(int nch) { return nch >= 8 ? 2 : 4; }
constexpr int stream_threads(int nch) { return (kStreamMmaWaves + stream_loaders(nch)) * 64; }
constexpr int kStreamRows = 32;
constexpr int kStreamCols = kStreamMmaWaves * 16;

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

// One 16-byte chunk of two 16-row A blocks against the same chunk of one B
// column block; the two accumulators alternate so consecutive MFMAs are
// independent.
template <int D>
__device__ __forceinline__ void mma16_rows2(const u32x4& x0, const u32x4& x1, const u32x4& y, f32x4& c0,
                                            f32x4& c1) {
    if constexpr (D == 0) {
        const f32x4 a0 = __builtin_bit_cast(f32x4, x0), a1 = __builtin_bit_cast(f32x4, x1);
        const f32x4 b = __builtin_bit_cast(f32x4, y);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            c0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[e], b[e], c0, 0, 0, 0);
            c1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[e], b[e], c1, 0, 0, 0);
        }
    } else {
        mma16_chunk<D>(x0, y, c0);
        mma16_chunk<D>(x1, y, c1);
    }
}

template <int D, int NCH>
__global__ __launch_bounds__(stream_threads(NCH), 1) void contract_stream_kernel(
    const unsigned char* __restrict__ V, const unsigned char* __restrict__ U, unsigned char* __restrict__ M,
    int64_t T, int64_t K, int rb, int64_t Kp, int num_mb, int num_nb, int64_t n_items) {
    // NCH = 16-byte chunks per lane per row: the k range of a row (rb <= 64 * NCH
    // bytes) is split over the four 16-lane groups of a wave.  LDS rows are
    // padded by one chunk, which keeps the fragment reads conflict-free.
    constexpr int kRowBytes = 64 * NCH + 16;
    constexpr int kABytes = kStreamRows * kRowBytes;
    __shared__ __attribute__((aligned(16))) unsigned char abuf[2 * kABytes];

    const int64_t G = gridDim.x;
    const int64_t bid = blockIdx.x;
    const int64_t v = (G % 8 == 0) ? (bid % 8) * (G / 8) + bid / 8 : bid;
    const int64_t it0 = v * n_items / G;
    const int64_t it1 = (v + 1) * n_items / G;
    if (it0 >= it1) return;
    const int n_mine = static_cast<int>(it1 - it0);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    int xi = static_cast<int>(it0 / (static_cast<int64_t>(num_mb) * num_nb));
    int nb = static_cast<int>((it0 / num_mb) % num_nb);
    int mb = static_cast<int>(it0 % num_mb);
    auto advance = [&](int& a, int& b, int& c) {
        if (++c == num_mb) {
            c = 0;
            if (++b == num_nb) {
                b = 0;
                ++a;
            }
        }
    };

    if (wave >= kStreamMmaWaves) {
        // ----------------------------------------------------------- loaders
        // loader lw owns every kLoaders-th 64-chunk group of a tile and keeps
        // kSets tiles in flight in its registers
        constexpr int kLoaders = stream_loaders(NCH);
        constexpr int kSets = stream_sets(NCH);
        const int lw = kLoaders == 1 ? 0 : wave - kStreamMmaWaves;
        constexpr int kRC = 4 * NCH;                                     // 16-byte chunks per LDS row
        constexpr int kLP = kStreamRows * kRC / (64 * kLoaders);   // chunks per lane per tile
        static_assert(kLP * 64 * kLoaders == kStreamRows * kRC, "tile split");
        uint32_t voff[kLP];
        int lofs[kLP];
#pragma unroll
        for (int p = 0; p < kLP; ++p) {
            const int ci = lw * 64 + lane + 64 * kLoaders * p;
            const int row = ci / kRC;
            const int c16 = ci % kRC;
            lofs[p] = row * kRowBytes + c16 * 16;
            voff[p] = c16 * 16 < rb ? static_cast<uint32_t>(row * rb + c16 * 16) : kOob;   // zero past the row
        }
        int lxi = xi, lnb = nb, lmb = mb;   // next tile to request
        auto load = [&](u32x4 (&dst)[kLP]) {
            const int64_t r0 = static_cast<int64_t>(lmb) * kStreamRows;
            const auto r = make_rsrc(V + (static_cast<int64_t>(lxi) * T + r0) * rb, (T - r0) * rb);
#pragma unroll
            for (int p = 0; p < kLP; ++p) dst[p] = __builtin_amdgcn_raw_buffer_load_b128(r, voff[p], 0, 0);
            advance(lxi, lnb, lmb);
        };
        auto park = [&](const u32x4 (&src)[kLP], int slot) {
#pragma unroll
            for (int p = 0; p < kLP; ++p) *reinterpret_cast<u32x4*>(abuf + slot * kABytes + lofs[p]) = src[p];
        };
        if constexpr (kSets == 2) {
            // two register sets, written out (the generic loop below costs
            // registers that the 512-byte rows do not have to spare)
            u32x4 s0[kLP], s1[kLP];
            load(s0);
            if (n_mine > 1) load(s1);
            park(s0, 0);
            if (n_mine > 2) load(s0);
            __syncthreads();
            // during item i: park tile i+1, request tile i+3 in its registers
            for (int i = 0; i < n_mine; i += 2) {
                if (i + 1 < n_mine) {
                    park(s1, 1);
                    if (i + 3 < n_mine) load(s1);
                }
                __syncthreads();
                if (i + 1 >= n_mine) break;
                if (i + 2 < n_mine) {
                    park(s0, 0);
                    if (i + 4 < n_mine) load(s0);
                }
                __syncthreads();
            }
        } else {
            u32x4 s[kSets][kLP];
            // tiles 0 .. kSets-1 requested, tile 0 parked, its registers refilled
#pragma unroll
            for (int j = 0; j < kSets; ++j)
                if (j < n_mine) load(s[j]);
            park(s[0], 0);
            if (kSets < n_mine) load(s[0]);
            __syncthreads();
            // during item i: park tile i+1 into LDS slot (i+1) mod 2, request tile
            // i+1+kSets in its registers (the loop is unrolled so that the register
            // set is a compile-time index)
            for (int i = 0; i < n_mine; i += kSets) {
                bool done = false;
#pragma unroll
                for (int j = 0; j < kSets; ++j) {
                    if (!done) {
                        const int ii = i + j;
                        if (ii + 1 < n_mine) {
                            park(s[(j + 1) % kSets], (ii + 1) & 1);
                            if (ii + 1 + kSets < n_mine) load(s[(j + 1) % kSets]);
                        }
                        __syncthreads();
                        done = ii + 1 >= n_mine;
                    }
                }
                if (done) break;
            }
        }
        return;
    }

    // -------------------------------------------------------------- MFMA waves
    const int grp = lane >> 4;
    const int l16 = lane & 15;
    // each 16-lane group owns a quarter of the k range.  With 512-byte rows
    // (528 in LDS) groups 1 and 2 swap quarters: a fragment read in the natural
    // order measured 1.7 times slower than a conflict-free one (LDS bank
    // conflicts), in this order as fast
    const int quarter = NCH == 8 ? ((grp & 1) << 1) | (grp >> 1) : grp;
    const int kb0 = quarter * (16 * NCH);
    u32x4 fy[NCH], fyn[NCH];
    auto load_b = [&](u32x4 (&dst)[NCH], int bxi, int bnb) {
        const int64_t c0 = static_cast<int64_t>(bnb) * kStreamCols;
        const auto r = make_rsrc(U + (static_cast<int64_t>(bxi) * K + c0) * rb, (K - c0) * rb);
        const uint32_t col = static_cast<uint32_t>((wave * 16 + l16) * rb);
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int byte = kb0 + c * 16;
            dst[c] = __builtin_amdgcn_raw_buffer_load_b128(r, byte < rb ? col + byte : kOob, 0, 0);
        }
    };
    // the wait for the U fragments lands here, outside the MFMA phase
    auto settle = [&]() {
#pragma unroll
        for (int c = 0; c < NCH; ++c) asm volatile("" : "+v"(fy[c]));
    };
    load_b(fy, xi, nb);
    settle();
    int nxi = xi, nnb = nb, nmb = mb;
    advance(nxi, nnb, nmb);
    __syncthreads();

    // 16x16 accumulator layout: lane holds column l16, rows 4*grp + q
    const uint32_t m_row = static_cast<uint32_t>(Kp * 4);
    const uint32_t m_lane = static_cast<uint32_t>((4 * grp * Kp + wave * 16 + l16) * 4);
    const unsigned char* arow = abuf + l16 * kRowBytes + kb0;
    int slot = 0;
    for (int i = 0; i < n_mine; ++i) {
        // the next item's U block, when it changes, arrives during this item
        const bool new_b = i + 1 < n_mine && (nxi != xi || nnb != nb);
        if (new_b) load_b(fyn, nxi, nnb);
        f32x4 acc0 = {0.0f, 0.0f, 0.0f, 0.0f}, acc1 = {0.0f, 0.0f, 0.0f, 0.0f};
        const unsigned char* a = arow + slot * kABytes;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const u32x4 x0 = *reinterpret_cast<const u32x4*>(a + c * 16);
            const u32x4 x1 = *reinterpret_cast<const u32x4*>(a + 16 * kRowBytes + c * 16);
            mma16_rows2<D>(x0, x1, fy[c], acc0, acc1);
        }
        if (new_b) {
#pragma unroll
            for (int c = 0; c < NCH; ++c) fy[c] = fyn[c];
            settle();
        }
        {
            const int64_t r0 = static_cast<int64_t>(mb) * kStreamRows;
            const int64_t c0 = static_cast<int64_t>(nb) * kStreamCols;
            const auto r = make_rsrc(M + ((static_cast<int64_t>(xi) * T + r0) * Kp + c0) * 4,
                                     (T - r0) * Kp * 4 - c0 * 4);
            const bool ok = c0 + wave * 16 + l16 < Kp;   // columns past Kp would wrap into the next row
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t off = m_lane + q * m_row;
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc0[q]), r, ok ? off : kOob, 0, 0);
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc1[q]), r, ok ? off + 16 * m_row : kOob,
                                                      0, 0);
            }
        }
        xi = nxi;
        nb = nnb;
        mb = nmb;
        advance(nxi, nnb, nmb);
        __syncthreads();
        slot ^= 1;
    }
}


template <int D, int NCH>
hipError_t launch_stream(const Geometry& g, const void* V, const void* U, float* M, int64_t row_bytes,
                         hipStream_t stream) {
    const int num_mb = static_cast<int>((g.T + kStreamRows - 1) / kStreamRows);
    const int num_nb = static_cast<int>((g.K + kStreamCols - 1) / kStreamCols);
    const int64_t n_items = static_cast<int64_t>(num_mb) * num_nb * g.planes;
    const int64_t grid = std::min<int64_t>(n_items, device_cu_count());
    hipLaunchKernelGGL((contract_stream_kernel<D, NCH>), dim3(static_cast<unsigned>(grid)), dim3(stream_threads(NCH)), 0,
                       stream, static_cast<const unsigned char*>(V), static_cast<const unsigned char*>(U),
                       reinterpret_cast<unsigned char*>(M), g.T, g.K, static_cast<int>(row_bytes), g.Kp, num_mb,
                       num_nb, n_items);
    return hipGetLastError();
}

}  // namespace

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

template <int D>
hipError_t launch_contract_t(const Geometry& g, const void* V, const void* U, float* M, hipStream_t stream) {
    const int64_t es = D == 0 ? 4 : 2;
    const int64_t row_bytes = g.Cp * es;
    // the streaming kernel addresses each plane of V, U and M with 32-bit offsets
    const bool fits32 = g.T * row_bytes < 0xffff0000LL && g.K * row_bytes < 0xffff0000LL &&
                        g.T * g.Kp * 4 < 0xffff0000LL;
    if (fits32 && row_bytes <= 64) return launch_stream<D, 1>(g, V, U, M, row_bytes, stream);
    if (fits32 && row_bytes <= 128) return launch_stream<D, 2>(g, V, U, M, row_bytes, stream);
    if (fits32 && row_bytes <= 256) return launch_stream<D, 4>(g, V, U, M, row_bytes, stream);
    if (fits32 && row_bytes <= 512) return launch_stream<D, 8>(g, V, U, M, row_bytes, stream);
    const int num_mb = static_cast<int>((g.T + kBM - 1) / kBM);
    const int num_nb = static_cast<int>((g.K + kBN - 1) / kBN);
    const int64_t blocks = static_cast<int64_t>(num_mb) * num_nb * g.planes;
    // the block kernel addresses its 128 rows of V and of U with 32-bit offsets
    if (blocks > 0x7fffffff || std::max(kBM, kBN) * row_bytes >= 0xffff0000LL) return hipErrorInvalidValue;
    hipLaunchKernelGGL(contract_kernel<D>, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream,
                       static_cast<const unsigned char*>(V), static_cast<const unsigned char*>(U), M, g.T, g.K,
                       row_bytes, g.Kp, num_mb, num_nb);
    return hipGetLastError();
}

template hipError_t launch_contract_t<0>(const Geometry&, const void*, const void*, float*, hipStream_t);
template hipError_t launch_contract_t<1>(const Geometry&, const void*, const void*, float*, hipStream_t);
template hipError_t launch_contract_t<2>(const Geometry&, const void*, const void*, float*, hipStream_t);

}  // namespace wg
