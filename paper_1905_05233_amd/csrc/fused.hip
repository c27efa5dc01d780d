// Contraction fused with the output transform (gfx950 matrix cores).
//
// eq. (2) of Barabasz & Gregg (arXiv 1905.05233) gives an output tile as
// A^T [ sum_c (G g_c G^T) . (B^T d_c B) ] A, the product taken elementwise.
// The separate path writes the channel sums M[xi][t][k] of all alpha'^2 domain
// points xi to memory and reads them back in the output transform.  Here a
// workgroup owns a block of (output channel, tile) pairs for every xi: the
// MFMAs leave M of one xi = (a, b) in the accumulators, and it is folded into
// the output tile at once,
//
//     Z[o]     = sum_a A^T[o][a] M[a][b]      (a ascending: the xi loop runs a fastest)
//     Y[o][p] += Z[o] A^T[p][b]               (after the last a of column b; b ascending)
//
// which is the order of operations of the stand-alone output transform, so
// M never reaches memory.  The MFMA rows are output channels (U) and its
// columns are tiles (V): a lane's accumulator then holds four consecutive
// channels of one tile, written as one 8- or 16-byte NHWC store per pixel.
//
// Workgroup: four waves of 16 channels x 16*WT tiles each, kw waves side by
// side along the channels and 4/kw along the tiles.  A step covers one
// 128-byte slice of the channel rows of one xi: the block's U and V rows are
// staged in double-buffered LDS (rows padded to 144 bytes, so the 16-byte
// fragment reads are conflict-free), with the next step's global loads in
// flight during the current MFMAs.  Global loads go through buffer
// descriptors clipped to the plane, so rows past T or K and bytes past a row
// read as zero.
#include <algorithm>
#include <cstring>
#include <type_traits>
#include <utility>

#include "coefs.hpp"
#include "device_common.hpp"
#include "kernels.hpp"

#ifndef WG_DTYPE
#error "compile once per storage dtype with -DWG_DTYPE=0 (fp32), 1 (fp16) or 2 (bf16)"
#endif

namespace wg {

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kSlice = 128;                          // bytes of each channel row per step
// LDS rows per stage: 16 kw channel rows + 16 WT (4 / kw) tile rows, at most
// 96 (kw >= 2 when WT = 2), filled by 12 DMA instructions of 8 rows
constexpr int kStageRows = 96;
constexpr int kDmaPerWave = kStageRows / 8 / 4;      // per wave and step
constexpr int kStageBytes = kStageRows * kSlice;

// One 16-byte fragment pair: lanes of group g hold the same slice of the
// channel range on both operands, so every channel meets its partner.
template <int D>
__device__ __forceinline__ void mma(const u32x4& a, const u32x4& b, f32x4& c) {
    if constexpr (D == 0) {
        const f32x4 av = __builtin_bit_cast(f32x4, a);
        const f32x4 bv = __builtin_bit_cast(f32x4, b);
#pragma unroll
        for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], bv[e], c, 0, 0, 0);
    } else if constexpr (D == 1) {
        c = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c,
                                                   0, 0, 0);
    } else {
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                    c, 0, 0, 0);
    }
}

template <typename Elem> __device__ __forceinline__ uint32_t bits16(Elem v) {
    if constexpr (sizeof(Elem) == 2 && __is_same(Elem, bf16_t)) return v.bits;
    else return __builtin_bit_cast(uint16_t, v);
}

// four consecutive output channels of one pixel, rounded to the storage dtype
template <typename Elem>
__device__ __forceinline__ void store4(Elem* dst, float v0, float v1, float v2, float v3) {
    using S = Storage<Elem>;
    if constexpr (sizeof(Elem) == 4) {
        *reinterpret_cast<f32x4*>(dst) = f32x4{v0, v1, v2, v3};
    } else {
        const uint32_t lo = bits16(S::from_f32(v0)) | (bits16(S::from_f32(v1)) << 16);
        const uint32_t hi = bits16(S::from_f32(v2)) | (bits16(S::from_f32(v3)) << 16);
        *reinterpret_cast<u32x2*>(dst) = u32x2{lo, hi};
    }
}

// 16 bytes per lane from a buffer straight into LDS (no registers): lane l
// lands at dst + 16 l; offsets past the record count write zeros
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, unsigned char* dst, uint32_t voff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)dst, 16, voff, 0, 0, 0);
}

// Workgroup barrier without the release fence of __syncthreads (which would
// wait for every DMA in flight): the LDS the waves read next was filled by
// DMAs that each wave has already waited for.  The empty asm statements keep
// the compiler from moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// s_waitcnt immediate that waits until at most n vector-memory operations of
// this wave are outstanding (gfx9 encoding; expcnt and lgkmcnt not waited on)
constexpr int vm_wait(int n) { return (n & 0xf) | (0x7 << 4) | (0xf << 8) | (((n >> 4) & 0x3) << 14); }

// K1 (input transform in the prologue): 0 = off (V comes from HBM); else the
// kernel computes the V rows of its 32 tiles itself, for every domain point,
// into LDS before the loop, and K1 = xp (8 or 4) domain points per step.
// Bytes of that buffer: alpha'^2 x 32 tiles x (128 / K1)-byte rows.
template <int ALPHA, int K1> constexpr int k1_vbuf_bytes() { return K1 ? ALPHA * ALPHA * 32 * (128 / K1) : 16; }

// ONE: every channel row fits one step (narrow rows, or rows of at most 128
// bytes), so a step's MFMA results are M of its domain point and the
// two-level channel sum is skipped.
template <int D, int MM, int ALPHA, int WT, bool NARROW, int K1, bool ONE>
__global__ __launch_bounds__(kThreads, 2) void contract_output_kernel(
    const unsigned char* __restrict__ V, const unsigned char* __restrict__ U, typename DTypeOf<D>::type* __restrict__ y,
    OutputTable tab, Geometry geo, int kw, int n_kb, int rb, int n_slices, int xp,
    const typename DTypeOf<D>::type* __restrict__ x, InputTable itab) {
    using Elem = typename DTypeOf<D>::type;
    using S = Storage<Elem>;
    static_assert(K1 == 0 || NARROW, "the input transform is fused only into the narrow-row variant");
    // four LDS stages (one step each, three steps in flight), separate arrays
    // so that the compiler can tell the stage being read from the ones being
    // filled; with K1 they hold only the 64 channel rows (U)
    constexpr int kSB = K1 ? 64 * kSlice : kStageBytes;
    __shared__ __attribute__((aligned(1024))) unsigned char st0[kSB];
    __shared__ __attribute__((aligned(1024))) unsigned char st1[kSB];
    __shared__ __attribute__((aligned(1024))) unsigned char st2[kSB];
    __shared__ __attribute__((aligned(1024))) unsigned char st3[kSB];
    __shared__ __attribute__((aligned(16))) unsigned char vbuf[k1_vbuf_bytes<ALPHA, K1>()];
    constexpr int kRB = K1 ? 128 / K1 : 16;   // bytes of a V row in vbuf
    constexpr int kDma = K1 ? 2 : kDmaPerWave;   // DMA instructions per wave and step

    // XCD-aware numbering: the hardware deals consecutive workgroup ids
    // round-robin over the 8 XCDs; give each XCD a contiguous run of units, so
    // the channel blocks of one tile block share an L2
    const int64_t G = gridDim.x;
    const int64_t bid = blockIdx.x;
    const int64_t xcd = bid % 8;
    const int64_t unit = xcd * (G / 8) + std::min<int64_t>(xcd, G % 8) + bid / 8;
    const int kb = static_cast<int>(unit % n_kb);
    const int64_t tb = unit / n_kb;

    const int krows = 16 * kw;              // channel rows of the block
    const int vrows = 16 * WT * (4 / kw);   // tile rows of the block
    const int rows = krows + vrows;         // <= kStageRows
    const int64_t k0 = static_cast<int64_t>(kb) * krows;
    const int64_t t0 = tb * vrows;
    const int64_t T = geo.T, K = geo.K;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wk = wave % kw;               // channel block of this wave
    const int wt = wave / kw;               // tile block of this wave
    const int grp = lane >> 4;
    const int l16 = lane & 15;

    // DMA map: instruction j of wave w fills stage rows 8 (w + 4 j) .. + 7
    // (channel rows first, then tile rows; whole instructions, since both
    // counts are multiples of 16, so the choice of operand is uniform).  Lane l
    // lands at row 8 (w + 4 j) + l / 8, 16-byte column l % 8, and fetches the
    // row's piece lp = (l % 8) ^ (l / 8): an XOR swizzle that keeps the
    // fragment reads conflict-free without padding.  Instructions past the
    // block's rows write zeros (every wave issues the same count, so one
    // vmcnt fits all).
    //
    // Narrow rows (xp > 1, a row of at most 64 bytes): a step holds xp domain
    // points, each in ppr = 8 / xp consecutive pieces of the slice, so the
    // DMAs and barriers per domain point drop xp-fold.  Piece lp then belongs
    // to the step's domain point lp / ppr, byte 16 (lp % ppr) of its row.
    const int ppr = 8 / xp;
    const int lp = (lane & 7) ^ (lane >> 3);
    const int lxi = lp / ppr;                   // domain point of the piece within the step (0 if wide)
    const int piece = (lp % ppr) * 16;          // byte offset of the piece within its row
    uint32_t roff[kDmaPerWave];
    bool live[kDmaPerWave], isu[kDmaPerWave];
#pragma unroll
    for (int j = 0; j < kDma; ++j) {
        const int r8 = 8 * (wave + 4 * j);
        live[j] = r8 < rows;
        isu[j] = r8 < krows;
        const int row = r8 + (lane >> 3);
        roff[j] = static_cast<uint32_t>((row < krows ? row : row - krows) * rb + piece);
    }
    // wide: the block's rows in plane 0, the plane strides and the
    // loop-invariant record counts of the buffer descriptors (rows past K or T
    // of a plane read zero), so that a request only multiplies its small plane
    // index by a stride
    const unsigned char* bu = U + k0 * rb;
    const unsigned char* bv = V + t0 * rb;
    const uint64_t plane_u = static_cast<uint64_t>(K * rb), plane_v = static_cast<uint64_t>(T * rb);
    const int64_t rec_u64 = (K - k0) * rb, rec_v64 = (T - t0) * rb;
    const int rec_u = static_cast<int>(static_cast<uint32_t>(rec_u64 > 0xffffffffLL ? 0xffffffffLL : rec_u64));
    const int rec_v = static_cast<int>(static_cast<uint32_t>(rec_v64 > 0xffffffffLL ? 0xffffffffLL : rec_v64));
    // wide: the request is (xi, slice); narrow: the step's first domain point
    // in visiting order (a fastest), each lane's plane found from its lxi
    auto issue = [&](unsigned char* st, int xi, int sl, int q0, bool any) __attribute__((always_inline)) {
        if constexpr (!NARROW) {
            const uint64_t ux = static_cast<uint32_t>(xi);   // 0 <= xi < alpha'^2
            const auto ru = __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned char*>(bu + ux * plane_u),
                                                              static_cast<short>(0), rec_u,
                                                              static_cast<int>(kRsrcWord3));
            const auto rv = __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned char*>(bv + ux * plane_v),
                                                              static_cast<short>(0), rec_v,
                                                              static_cast<int>(kRsrcWord3));
            const int sb = sl * kSlice;
            const bool in = any && sb + piece < rb;   // zero past the row
#pragma unroll
            for (int j = 0; j < kDmaPerWave; ++j)
                dma16(isu[j] ? ru : rv, st + (wave + 4 * j) * 1024, live[j] && in ? roff[j] + sb : kOob);
        } else {
            // descriptors over every plane (checked to fit 32-bit offsets at
            // launch); rows past T or K read other planes' rows, which only
            // reach (channel, tile) pairs that are never stored
            const auto ru = make_rsrc(U + k0 * rb, (static_cast<int64_t>(ALPHA) * ALPHA * K - k0) * rb);
            const auto rv = make_rsrc(V + t0 * rb, (static_cast<int64_t>(ALPHA) * ALPHA * T - t0) * rb);
            const int q = q0 + lxi;                         // this lane's domain point, in visiting order
            const int pxi = (q % ALPHA) * ALPHA + q / ALPHA;  // its index xi = a alpha' + b
            const bool in = any && q < ALPHA * ALPHA && piece < rb;
            const uint32_t pu = static_cast<uint32_t>(pxi * K * rb), pv = static_cast<uint32_t>(pxi * T * rb);
#pragma unroll
            for (int j = 0; j < kDma; ++j)
                dma16(isu[j] ? ru : rv, st + (wave + 4 * j) * 1024,
                      live[j] && in ? roff[j] + (isu[j] ? pu : pv) : kOob);
        }
    };

    f32x4 acc[WT];
    float Z[WT][MM][4];
    float Y[WT][MM][MM][4];
#pragma unroll
    for (int w = 0; w < WT; ++w) {
        acc[w] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int o = 0; o < MM; ++o)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                Z[w][o][r] = 0.0f;
#pragma unroll
                for (int q = 0; q < MM; ++q) Y[w][o][q][r] = 0.0f;
            }
    }

    // fragment addresses (row & 7 = l16 & 7 for both operands)
    const int swz = l16 & 7;
    const int a_row = (wk * 16 + l16) * kSlice;
    const int b_row = (krows + wt * 16 * WT + l16) * kSlice;
    const int col0 = ((grp) ^ swz) * 16;       // slice half 0: pieces 0..3
    const int col1 = ((grp + 4) ^ swz) * 16;   // slice half 1: pieces 4..7
    const int nsteps = NARROW ? (ALPHA * ALPHA + xp - 1) / xp : ALPHA * ALPHA * n_slices;
    // step order: slices fastest, then a (M row), then b (M column)
    int a = 0, bc = 0, sl = 0;      // step being computed (the next domain point to fold when narrow)
    int na = 0, nb = 0, ns = 0;     // next step to request (wide)
    int nq = 0;                     // first domain point of the next step to request (narrow)
    auto advance = [&](int& a_, int& b_, int& s_) {
        if (++s_ == n_slices) {
            s_ = 0;
            if (++a_ == ALPHA) {
                a_ = 0;
                ++b_;
            }
        }
    };
    auto request = [&](unsigned char* st) __attribute__((always_inline)) {
        // past the last step the group is issued anyway (all zeros), which
        // keeps the outstanding count per step constant
        if constexpr (!NARROW) {
            const bool any = nb < ALPHA;
            issue(st, any ? na * ALPHA + nb : 0, any ? ns : 0, 0, any);
            if (any) advance(na, nb, ns);
        } else {
            issue(st, 0, 0, nq, nq < ALPHA * ALPHA);
            nq += xp;
        }
    };

    // two-level channel sum: each step's slice goes into a fresh accumulator
    // `part`, added to the running sum `acc` (a sequential chain over C would
    // be C/4 deep).  The fold of a step into Z and Y runs one step later,
    // while the next step's LDS reads are in flight, and consumes the MFMA
    // results only then.
    f32x4 part[WT];
#pragma unroll
    for (int w = 0; w < WT; ++w) part[w] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    // the output-transform coefficients of the step being folded, A^T[o][a]
    // and A^T[o][bc], are loaded into scalar registers before its LDS reads
    // are issued (a wait for them afterwards would also wait for those reads)
    float cz[MM], cy[MM];
    auto coefs = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int o = 0; o < MM; ++o) {
            cz[o] = tab.at[o * ALPHA + a];
            cy[o] = tab.at[o * ALPHA + bc];
        }
    };
    auto fold = [&]() __attribute__((always_inline)) {   // the step (a, bc, sl)
        if constexpr (!ONE) {
#pragma unroll
            for (int w = 0; w < WT; ++w) acc[w] += part[w];
        }
        if (ONE || sl == n_slices - 1) {
            // M[a][bc] of this block is complete: fold it into Z (pass 1)
            const f32x4* mv = ONE ? part : acc;
#pragma unroll
            for (int o = 0; o < MM; ++o) {
                const float c = cz[o];
#pragma unroll
                for (int w = 0; w < WT; ++w)
#pragma unroll
                    for (int r = 0; r < 4; ++r) Z[w][o][r] = __builtin_fmaf(c, mv[w][r], Z[w][o][r]);
            }
            if constexpr (!ONE) {
#pragma unroll
                for (int w = 0; w < WT; ++w) acc[w] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            }
            if (a == ALPHA - 1) {
                // column bc done: pass 2 into the output tile
#pragma unroll
                for (int q = 0; q < MM; ++q) {
                    const float c = cy[q];
#pragma unroll
                    for (int w = 0; w < WT; ++w)
#pragma unroll
                        for (int o = 0; o < MM; ++o)
#pragma unroll
                            for (int r = 0; r < 4; ++r) Y[w][o][q][r] = __builtin_fmaf(Z[w][o][r], c, Y[w][o][q][r]);
                }
#pragma unroll
                for (int w = 0; w < WT; ++w)
#pragma unroll
                    for (int o = 0; o < MM; ++o)
#pragma unroll
                        for (int r = 0; r < 4; ++r) Z[w][o][r] = 0.0f;
            }
        }
        advance(a, bc, sl);
    };

    bool have_prev = false;
    int sq = 0;   // first domain point of the step being computed (narrow)
    auto step = [&](const unsigned char* cur, unsigned char* nxt) __attribute__((always_inline)) {
        // this wave's DMAs for `cur` are done once at most two groups remain;
        // the barrier makes every wave's visible and frees `nxt` (read in the
        // previous step) for the next request
        coefs();
        __builtin_amdgcn_s_waitcnt(vm_wait(2 * kDma));
        lds_barrier();
        request(nxt);
        // the coefficients must be in registers before the LDS reads go out
#pragma unroll
        for (int o = 0; o < MM; ++o) asm volatile("" : "+s"(cz[o]), "+s"(cy[o]));
        if constexpr (!NARROW) {
            u32x4 fa0 = lds_read16(cur + a_row + col0);
            u32x4 fa1 = lds_read16(cur + a_row + col1);
            u32x4 fb[WT][2];
#pragma unroll
            for (int w = 0; w < WT; ++w) {
                fb[w][0] = lds_read16(cur + b_row + w * 16 * kSlice + col0);
                fb[w][1] = lds_read16(cur + b_row + w * 16 * kSlice + col1);
            }
            if (have_prev) fold();
            have_prev = true;
            if constexpr (WT == 2) lds_settle(fa0, fa1, fb[0][0], fb[0][1], fb[1][0], fb[1][1]);
            else lds_settle(fa0, fa1, fb[0][0], fb[0][1]);
#pragma unroll
            for (int w = 0; w < WT; ++w) {
                part[w] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                mma<D>(fa0, fb[w][0], part[w]);
                mma<D>(fa1, fb[w][1], part[w]);
            }
        } else {
        // narrow: domain point i of the step sits in pieces [i ppr, i ppr + ppr)
        // of one slice half; lane groups outside them contribute zeros
        for (int i = 0; i < xp; ++i) {
            if (sq + i >= ALPHA * ALPHA) break;
            if (i > 0) {
                // the coefficients loaded at the end of the last iteration,
                // in registers before this iteration's LDS reads go out
#pragma unroll
                for (int o = 0; o < MM; ++o) asm volatile("" : "+s"(cz[o]), "+s"(cy[o]));
            }
            const int p0 = i * ppr;
            const int col = (((p0 & 4) + grp) ^ swz) * 16;
            u32x4 fa = lds_read16(cur + a_row + col);
            u32x4 fb[WT];
            if constexpr (K1 != 0) {
                // this lane group's piece of domain point sq + i in vbuf (any
                // piece for the groups that are masked below)
                const int pc = (grp - (p0 & 3)) & (ppr - 1);
#pragma unroll
                for (int w = 0; w < WT; ++w)
                    fb[w] = lds_read16(vbuf + ((sq + i) * 32 + wt * 16 * WT + w * 16 + l16) * kRB + pc * 16);
            } else {
#pragma unroll
                for (int w = 0; w < WT; ++w) fb[w] = lds_read16(cur + b_row + w * 16 * kSlice + col);
            }
            if (have_prev) fold();
            have_prev = true;
            coefs();   // for the fold of this domain point, in the next iteration
            if constexpr (WT == 2) lds_settle(fa, fb[0], fb[1]);
            else lds_settle(fa, fb[0]);
            if (static_cast<unsigned>(grp - (p0 & 3)) >= static_cast<unsigned>(ppr)) fa = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
            for (int w = 0; w < WT; ++w) {
                part[w] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                mma<D>(fa, fb[w], part[w]);
            }
        }
        sq += xp;
        }
    };

    // prologue: steps 0, 1, 2 requested into stages 0, 1, 2
    request(st0);
    request(st1);
    request(st2);
    if constexpr (K1 != 0) {
        // The V rows of this block's 32 tiles (kw = 4), every domain point,
        // into vbuf at [q][tile][kRB bytes], q = b alpha' + a the visiting
        // order of the loop; the first U requests are already in flight.
        // Each (tile, channel) pair runs the input transform of eq. (2) in the
        // order of the stand-alone kernel: pass 1 W = B^T d in ascending u,
        // pass 2 in ascending v, fp32 fused multiply-adds from zero, rounded
        // once to the storage type (the same values bit for bit); padding
        // channels and tiles past T hold zeros.  Tile coordinates are carried
        // from the block's first tile (T < 2^28 here, so 32-bit arithmetic).
        constexpr int TT = MM + 2;
        constexpr int kNE = kRB / static_cast<int>(sizeof(Elem));   // channels of a vbuf row
        const int tw = static_cast<int>(geo.tw), th = static_cast<int>(geo.th);
        const int tx0 = static_cast<int>(t0 % geo.tw);
        const int ty0 = static_cast<int>((t0 / geo.tw) % geo.th);
        const int n0 = static_cast<int>(t0 / (geo.tw * geo.th));
        const int H = static_cast<int>(geo.H), Wd = static_cast<int>(geo.W), C = static_cast<int>(geo.C);
        for (int pr = tid; pr < 32 * kNE; pr += kThreads) {
            const int r = pr / kNE, c = pr % kNE;
            int tx = tx0 + r, ty = ty0, n = n0;
            while (tx >= tw) {
                tx -= tw;
                if (++ty == th) {
                    ty = 0;
                    ++n;
                }
            }
            const bool live_t = t0 + r < T && c < C;
            float d[TT][TT];
#pragma unroll
            for (int u = 0; u < TT; ++u) {
                const int hr = ty * geo.m - 1 + u;
                const int wc0 = tx * geo.m - 1;
                const Elem* row = x + ((static_cast<int64_t>(n) * H + hr) * Wd + wc0) * C + c;
#pragma unroll
                for (int v = 0; v < TT; ++v) {
                    const bool in = live_t && hr >= 0 && hr < H && wc0 + v >= 0 && wc0 + v < Wd;
                    d[u][v] = in ? S::to_f32(row[v * C]) : 0.0f;
                }
            }
#pragma unroll
            for (int a = 0; a < ALPHA; ++a) {
                float w1[TT];
#pragma unroll
                for (int v = 0; v < TT; ++v) {
                    float acc = 0.0f;
#pragma unroll
                    for (int u = 0; u < TT; ++u) acc = __builtin_fmaf(itab.bt[a * TT + u], d[u][v], acc);
                    w1[v] = acc;
                }
#pragma unroll
                for (int b = 0; b < ALPHA; ++b) {
                    float acc = 0.0f;
#pragma unroll
                    for (int v = 0; v < TT; ++v) acc = __builtin_fmaf(itab.bt[b * TT + v], w1[v], acc);
                    *reinterpret_cast<Elem*>(vbuf + ((b * ALPHA + a) * 32 + r) * kRB + c * sizeof(Elem)) =
                        S::from_f32(acc);
                }
            }
        }
        // this wave's vbuf writes done, then every wave's (no wait for the
        // U requests in flight)
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        lds_barrier();
    }

    // step s reads stage s % 4 and requests step s + 3 into stage (s + 3) % 4
    for (int s0 = 0; s0 < nsteps; s0 += 4) {
        step(st0, st3);
        if (s0 + 1 >= nsteps) break;
        step(st1, st0);
        if (s0 + 2 >= nsteps) break;
        step(st2, st1);
        if (s0 + 3 >= nsteps) break;
        step(st3, st2);
    }
    coefs();
    fold();   // the last step
    // the trailing zero groups must land before the wave ends (the LDS of
    // the workgroup is then handed to the next one)
    __builtin_amdgcn_s_waitcnt(vm_wait(0));

    // epilogue: masked NHWC store, four consecutive channels per lane
    const int64_t k = k0 + wk * 16 + 4 * grp;
    if (k >= K) return;
    const bool vec = (K & 3) == 0;
#pragma unroll
    for (int w = 0; w < WT; ++w) {
        const int64_t tile = t0 + (wt * WT + w) * 16 + l16;
        if (tile >= T) continue;
        const int64_t tx = tile % geo.tw;
        const int64_t ty = (tile / geo.tw) % geo.th;
        const int64_t n = tile / (geo.tw * geo.th);
#pragma unroll
        for (int o = 0; o < MM; ++o) {
            const int64_t hr = ty * MM + o;
            if (hr >= geo.H) break;
#pragma unroll
            for (int q = 0; q < MM; ++q) {
                const int64_t wc = tx * MM + q;
                if (wc >= geo.W) break;
                Elem* dst = y + ((n * geo.H + hr) * geo.W + wc) * K + k;
                if (vec) {
                    store4(dst, Y[w][o][q][0], Y[w][o][q][1], Y[w][o][q][2], Y[w][o][q][3]);
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (k + r < K) dst[r] = S::from_f32(Y[w][o][q][r]);
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Whole channel rows per step, with the domain-point loop unrolled.
//
// When a channel row fits NSL 128-byte slices (NSL = 1: C <= 64 in fp16/bf16,
// C <= 32 in fp32; NSL = 2: twice that) and the block is 64 output channels x
// 32 tiles (WT = 2), the contraction of a domain point is a single step of NSL
// slices; rows of at most 64 bytes share one slice between XP = 128 / row
// bytes domain points, as in the looped kernel's narrow steps; rows of three
// or four slices take NCK = 2 steps of two slices per domain point, unrolled
// like the rest; longer rows (CH) take n_ch steps of two slices per domain
// point in a loop at run time.  In both, the MFMA chains of a domain point
// accumulate over its steps.  This variant unrolls the
// domain points at compile time: the
// output-transform coefficients of every fold are constants (for a built-in
// plan the zero terms disappear; for any other plan they are read from the
// kernel arguments once), and no step bookkeeping is left.  Each step's U and
// V rows are staged in LDS by buffer-to-LDS loads in the layout of the looped
// kernel (rows of 128 bytes per slice, XOR-swizzled 16-byte pieces), NST
// stages deep; each wave loads whole rows with 8 lanes per row, so its
// requests are coalesced.  The output tile leaves through LDS: each wave
// parks its channels of every pixel there, and the block's pixels are then
// written with 16 contiguous bytes per lane (whole 64-channel runs of each
// pixel) instead of 4 channels per lane.  Folds, rounding and the order of
// every sum are those of the looped kernel.

// f(std::integral_constant<int, S>) for S = 0 .. N-1, in order
template <class F, int... S>
__device__ __forceinline__ void unroll_seq(F& f, std::integer_sequence<int, S...>) {
    (f(std::integral_constant<int, S>{}), ...);
}
template <int N, class F> __device__ __forceinline__ void unroll(F&& f) {
    unroll_seq(f, std::make_integer_sequence<int, N>{});
}

// Stages of the unrolled kernel and LDS bytes of one stage (NSL slices of 96
// rows: 64 channel rows, then 32 tile rows)
template <int NSL> constexpr int unrolled_stages() { return NSL == 1 ? 4 : 3; }
template <int NSL> constexpr int unrolled_stage_bytes() { return NSL * kStageBytes; }
// LDS of the output tile in the epilogue: 16 tiles x m^2 pixels x 64 channels
template <int MM, class Elem> constexpr int unrolled_out_bytes() {
    return 16 * MM * MM * 64 * static_cast<int>(sizeof(Elem));
}

// Vector-memory groups (one per step) a wave has issued after that of step s
// when step s begins: the prologue requests steps 0 .. NST-2, and step s'
// requests step s' + NST - 1.
template <int NSTEPS, int NST>
constexpr int groups_after(int s) {
    const int issued = (s + NST - 1 < NSTEPS) ? s + NST - 1 : NSTEPS;
    return issued - (s + 1);
}

template <int D, int MM, int ALPHA, class CO, int NSL, int XP, bool CH, int NCK>
__global__ __launch_bounds__(kThreads, 2) void contract_output_unrolled_kernel(
    const unsigned char* __restrict__ V, const unsigned char* __restrict__ U, typename DTypeOf<D>::type* __restrict__ y,
    OutputTable tab, Geometry geo, int n_kb, int rb, int n_ch) {
    using Elem = typename DTypeOf<D>::type;
    using S = Storage<Elem>;
    constexpr int WT = 2;                  // two 16-tile blocks per wave
    constexpr int NPTS = ALPHA * ALPHA;    // domain points
    constexpr int NSTEPS = NCK * ((NPTS + XP - 1) / XP);
    constexpr int PPR = 8 / XP;            // 16-byte pieces of a domain point's row in a slice
    static_assert(XP == 1 || NSL == 1, "narrow rows fit one slice");
    static_assert(!CH || (NSL == 2 && XP == 1 && NCK == 1), "long rows go in steps of two slices");
    static_assert(NCK == 1 || (NSL == 2 && XP == 1 && !CH), "unrolled chunks are steps of two slices");
    constexpr int NST = unrolled_stages<NSL>();
    constexpr int kSB = unrolled_stage_bytes<NSL>();
    constexpr int kKD = 3 * NSL;           // DMA instructions per wave and step
    constexpr int kOut = unrolled_out_bytes<MM, Elem>();
    constexpr int kLds = NST * kSB > kOut ? NST * kSB : kOut;
    static_assert(kKD * (NST - 2) < 64, "vmcnt holds 6 bits");
    static_assert(2 * kLds <= 160 * 1024, "two workgroups per CU");
    __shared__ __attribute__((aligned(1024))) unsigned char lds[kLds];

    // XCD-aware numbering, as in contract_output_kernel
    const int64_t G = gridDim.x;
    const int64_t bid = blockIdx.x;
    const int64_t xcd = bid % 8;
    const int64_t unit = xcd * (G / 8) + std::min<int64_t>(xcd, G % 8) + bid / 8;
    const int kb = static_cast<int>(unit % n_kb);
    const int64_t tb = unit / n_kb;
    const int64_t k0 = static_cast<int64_t>(kb) * 64;
    const int64_t t0 = tb * 32;
    const int64_t T = geo.T, K = geo.K;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // 16 output channels each
    const int grp = lane >> 4;
    const int l16 = lane & 15;

    // DMA map (the looped kernel's): instruction j of wave w fills stage rows
    // 8 (w + 4 j) .. + 7 of each slice, channel rows 0 .. 63 first, then tile
    // rows; lane l lands at row 8 (w + 4 j) + l / 8, 16-byte column l % 8, and
    // fetches piece lp = (l % 8) ^ (l / 8) of the slice; pieces past the row
    // read zero.  Narrow rows: piece lp holds byte 16 (lp % PPR) of the row of
    // the step's domain point lp / PPR.
    const int lp = (lane & 7) ^ (lane >> 3);
    const int lxi = lp / PPR;
    const int piece = (lp % PPR) * 16;
    uint32_t roff[3];
#pragma unroll
    for (int j = 0; j < 3; ++j) {
        const int row = 8 * (wave + 4 * j) + (lane >> 3);
        roff[j] = static_cast<uint32_t>((row < 64 ? row : row - 64) * rb + piece);
    }
    // descriptors over one plane's rows of the block (rows past K or T read zero)
    const unsigned char* bu = U + k0 * rb;
    const unsigned char* bv = V + t0 * rb;
    const uint64_t plane_u = static_cast<uint64_t>(K * rb), plane_v = static_cast<uint64_t>(T * rb);
    const int64_t rec_u64 = (K - k0) * rb, rec_v64 = (T - t0) * rb;
    const int rec_u = static_cast<int>(static_cast<uint32_t>(rec_u64 > 0xffffffffLL ? 0xffffffffLL : rec_u64));
    const int rec_v = static_cast<int>(static_cast<uint32_t>(rec_v64 > 0xffffffffLL ? 0xffffffffLL : rec_v64));

    // domain point q is (a, b) = (q % alpha', q / alpha'), xi = a alpha' + b;
    // step s holds q = s XP .. s XP + XP - 1
    // narrow: descriptors over every plane (the launcher checks that they fit
    // 32-bit offsets); rows past T or K then read other planes' rows, which
    // only reach (channel, tile) pairs that are never stored
    const auto ru_all = make_rsrc(bu, (static_cast<int64_t>(NPTS) * K - k0) * rb);
    const auto rv_all = make_rsrc(bv, (static_cast<int64_t>(NPTS) * T - t0) * rb);
    auto issue = [&](auto sc) __attribute__((always_inline)) {
        constexpr int s = decltype(sc)::value;
        if constexpr (XP > 1) {
            const int q = s * XP + lxi;
            const int pxi = (q % ALPHA) * ALPHA + q / ALPHA;
            const bool in = q < NPTS && piece < rb;
            const uint32_t pu = static_cast<uint32_t>(pxi) * static_cast<uint32_t>(plane_u);
            const uint32_t pv = static_cast<uint32_t>(pxi) * static_cast<uint32_t>(plane_v);
            unsigned char* st = lds + (s % NST) * kSB;
#pragma unroll
            for (int j = 0; j < 3; ++j)
                dma16(j < 2 ? ru_all : rv_all, st + (wave + 4 * j) * 1024,
                      in ? roff[j] + (j < 2 ? pu : pv) : kOob);
            return;
        }
        // step s is chunk s % NCK (slices NSL (s % NCK) ..) of domain point s / NCK
        constexpr int q = s / NCK, ck = s % NCK;
        constexpr uint64_t xi = (q % ALPHA) * ALPHA + q / ALPHA;
        const auto ru = __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned char*>(bu + xi * plane_u),
                                                          static_cast<short>(0), rec_u, static_cast<int>(kRsrcWord3));
        const auto rv = __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned char*>(bv + xi * plane_v),
                                                          static_cast<short>(0), rec_v, static_cast<int>(kRsrcWord3));
        unsigned char* st = lds + (s % NST) * kSB;
#pragma unroll
        for (int sl = 0; sl < NSL; ++sl) {
            constexpr int sb0 = ck * NSL * kSlice;
            const bool in = sb0 + sl * kSlice + piece < rb;
#pragma unroll
            for (int j = 0; j < 3; ++j)
                dma16(j < 2 ? ru : rv, st + sl * kStageBytes + (wave + 4 * j) * 1024,
                      in ? roff[j] + sb0 + sl * kSlice : kOob);
        }
    };

    f32x4 part[WT];
    float Z[WT][MM][4];
    float Y[WT][MM][MM][4];
#pragma unroll
    for (int w = 0; w < WT; ++w)
#pragma unroll
        for (int o = 0; o < MM; ++o)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                Z[w][o][r] = 0.0f;
#pragma unroll
                for (int q = 0; q < MM; ++q) Y[w][o][q][r] = 0.0f;
            }

    // M of step s (in part) into Z, and Z into the output tile after a column
    auto fold = [&](auto sc) __attribute__((always_inline)) {
        constexpr int s = decltype(sc)::value;
        constexpr int a = s % ALPHA, bc = s / ALPHA;
#pragma unroll
        for (int o = 0; o < MM; ++o) {
            const float c = CO::at(tab, o * ALPHA + a);
#pragma unroll
            for (int w = 0; w < WT; ++w)
#pragma unroll
                for (int r = 0; r < 4; ++r) Z[w][o][r] = term<CO>(c, part[w][r], Z[w][o][r]);
        }
        if constexpr (a == ALPHA - 1) {
#pragma unroll
            for (int q = 0; q < MM; ++q) {
                const float c = CO::at(tab, q * ALPHA + bc);
#pragma unroll
                for (int w = 0; w < WT; ++w)
#pragma unroll
                    for (int o = 0; o < MM; ++o)
#pragma unroll
                        for (int r = 0; r < 4; ++r) Y[w][o][q][r] = term<CO>(c, Z[w][o][r], Y[w][o][q][r]);
            }
#pragma unroll
            for (int w = 0; w < WT; ++w)
#pragma unroll
                for (int o = 0; o < MM; ++o)
#pragma unroll
                    for (int r = 0; r < 4; ++r) Z[w][o][r] = 0.0f;
        }
        if constexpr (CH) {
            // the fold happens here: the compiler would otherwise sink it past
            // the run-time loops of later domain points, keeping every
            // domain point's M live
#pragma unroll
            for (int w = 0; w < WT; ++w)
#pragma unroll
                for (int o = 0; o < MM; ++o)
#pragma unroll
                    for (int r = 0; r < 4; ++r) asm volatile("" : "+v"(Z[w][o][r]));
            if constexpr (a == ALPHA - 1) {
#pragma unroll
                for (int w = 0; w < WT; ++w)
#pragma unroll
                    for (int o = 0; o < MM; ++o)
#pragma unroll
                        for (int q = 0; q < MM; ++q)
#pragma unroll
                            for (int r = 0; r < 4; ++r) asm volatile("" : "+v"(Y[w][o][q][r]));
            }
        }
    };

    // fragments: A = channel row 16 wave + l16, B = tile row 16 w + l16 of
    // each slice, pieces grp and grp + 4 (row & 7 = l16 & 7 for both)
    const int swz = l16 & 7;
    const int a_row = (wave * 16 + l16) * kSlice;
    const int b_row = (64 + l16) * kSlice;
    const int col0 = (grp ^ swz) * 16;
    const int col1 = ((grp + 4) ^ swz) * 16;
    auto step = [&](auto sc) __attribute__((always_inline)) {
        constexpr int s = decltype(sc)::value;
        // each step is scheduled on its own (else the scheduler interleaves the
        // straight-line steps and runs out of registers)
        __builtin_amdgcn_sched_barrier(0);
        // this wave's requests of step s have landed once at most the later
        // groups are outstanding; the barrier makes every wave's visible and
        // frees the stage read in the previous step for the next request
        __builtin_amdgcn_s_waitcnt(vm_wait(kKD * groups_after<NSTEPS, NST>(s)));
        lds_barrier();
        if constexpr (s + NST - 1 < NSTEPS) issue(std::integral_constant<int, s + NST - 1>{});
        const unsigned char* cur = lds + (s % NST) * kSB;
        if constexpr (XP > 1) {
            // domain point q of the step sits in pieces [i PPR, i PPR + PPR) of
            // one slice half; lane groups outside them contribute zeros
            unroll<XP>([&](auto ic) __attribute__((always_inline)) {
                constexpr int i = decltype(ic)::value;
                constexpr int q = s * XP + i;
                if constexpr (q < NPTS) {
                    constexpr int p0 = i * PPR;
                    const int col = (((p0 & 4) + grp) ^ swz) * 16;
                    u32x4 fa = lds_read16(cur + a_row + col);
                    u32x4 fb0 = lds_read16(cur + b_row + col);
                    u32x4 fb1 = lds_read16(cur + b_row + 16 * kSlice + col);
                    if constexpr (q > 0) fold(std::integral_constant<int, q - 1>{});
                    lds_settle(fa, fb0, fb1);
                    if (static_cast<unsigned>(grp - (p0 & 3)) >= static_cast<unsigned>(PPR)) fa = u32x4{0u, 0u, 0u, 0u};
                    part[0] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                    part[1] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                    mma<D>(fa, fb0, part[0]);
                    mma<D>(fa, fb1, part[1]);
                }
            });
            return;
        }
        // NCK > 1: the first chunk of a domain point folds the previous one
        constexpr int q = s / NCK, ck = s % NCK;
        u32x4 fa0 = lds_read16(cur + a_row + col0);
        u32x4 fa1 = lds_read16(cur + a_row + col1);
        u32x4 fb00 = lds_read16(cur + b_row + col0);
        u32x4 fb01 = lds_read16(cur + b_row + col1);
        u32x4 fb10 = lds_read16(cur + b_row + 16 * kSlice + col0);
        u32x4 fb11 = lds_read16(cur + b_row + 16 * kSlice + col1);
        if constexpr (ck == 0 && q > 0) fold(std::integral_constant<int, q - 1>{});
        lds_settle(fa0, fa1, fb00, fb01, fb10, fb11);
        if constexpr (ck == 0) {
            part[0] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            part[1] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        }
        mma<D>(fa0, fb00, part[0]);
        mma<D>(fa0, fb10, part[1]);
        mma<D>(fa1, fb01, part[0]);
        mma<D>(fa1, fb11, part[1]);
        if constexpr (NSL == 2) {
            // the second slice, its fragments read after the first slice's
            // MFMAs have taken theirs (the register sets are reused)
            cur += kStageBytes;
            fa0 = lds_read16(cur + a_row + col0);
            fa1 = lds_read16(cur + a_row + col1);
            fb00 = lds_read16(cur + b_row + col0);
            fb01 = lds_read16(cur + b_row + col1);
            fb10 = lds_read16(cur + b_row + 16 * kSlice + col0);
            fb11 = lds_read16(cur + b_row + 16 * kSlice + col1);
            lds_settle(fa0, fa1, fb00, fb01, fb10, fb11);
            mma<D>(fa0, fb00, part[0]);
            mma<D>(fa0, fb10, part[1]);
            mma<D>(fa1, fb01, part[0]);
            mma<D>(fa1, fb11, part[1]);
        }
    };

    if constexpr (CH) {
        // Long rows: step (q, c) is chunk c (slices 2c and 2c + 1) of domain
        // point q, steps in the order q n_ch + c.  The request for the step NST - 1
        // ahead is tracked by counters (rq, rc) and its stage rs; past the last
        // step a group of out-of-range requests (zero fills) keeps one group
        // per step, so every step waits for the same count.
        int rq = 0, rc = 0, rs = 0, cs = 0;
        auto issue_next = [&]() __attribute__((always_inline)) {
            const bool live = rq < NPTS;
            const uint64_t xi = live ? static_cast<uint64_t>((rq % ALPHA) * ALPHA + rq / ALPHA) : 0;
            const auto ru = __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned char*>(bu + xi * plane_u),
                                                              static_cast<short>(0), rec_u,
                                                              static_cast<int>(kRsrcWord3));
            const auto rv = __builtin_amdgcn_make_buffer_rsrc(const_cast<unsigned char*>(bv + xi * plane_v),
                                                              static_cast<short>(0), rec_v,
                                                              static_cast<int>(kRsrcWord3));
            unsigned char* st = lds + rs * kSB;
#pragma unroll
            for (int sl = 0; sl < NSL; ++sl) {
                const int sb = (rc * NSL + sl) * kSlice;
                const bool in = live && sb + piece < rb;
#pragma unroll
                for (int j = 0; j < 3; ++j)
                    dma16(j < 2 ? ru : rv, st + sl * kStageBytes + (wave + 4 * j) * 1024, in ? roff[j] + sb : kOob);
            }
            if (++rc == n_ch) {
                rc = 0;
                ++rq;
            }
            rs = rs + 1 == NST ? 0 : rs + 1;
        };
        // one step: wait for this wave's group of the step, barrier, request
        // the group NST - 1 ahead, contract both slices into part
        auto chunk = [&](auto qc, bool first) __attribute__((always_inline)) {
            constexpr int q = decltype(qc)::value;
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_waitcnt(vm_wait(kKD * (NST - 2)));
            lds_barrier();
            issue_next();
            const unsigned char* cur = lds + cs * kSB;
            cs = cs + 1 == NST ? 0 : cs + 1;
            u32x4 fa0 = lds_read16(cur + a_row + col0);
            u32x4 fa1 = lds_read16(cur + a_row + col1);
            u32x4 fb00 = lds_read16(cur + b_row + col0);
            u32x4 fb01 = lds_read16(cur + b_row + col1);
            u32x4 fb10 = lds_read16(cur + b_row + 16 * kSlice + col0);
            u32x4 fb11 = lds_read16(cur + b_row + 16 * kSlice + col1);
            if (first) {
                if constexpr (q > 0) fold(std::integral_constant<int, q - 1>{});
            }
            lds_settle(fa0, fa1, fb00, fb01, fb10, fb11);
            if (first) {
                part[0] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                part[1] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            }
            mma<D>(fa0, fb00, part[0]);
            mma<D>(fa0, fb10, part[1]);
            mma<D>(fa1, fb01, part[0]);
            mma<D>(fa1, fb11, part[1]);
            // the second slice, its fragments read after the first slice's
            // MFMAs have taken theirs (the register sets are reused)
            cur += kStageBytes;
            fa0 = lds_read16(cur + a_row + col0);
            fa1 = lds_read16(cur + a_row + col1);
            fb00 = lds_read16(cur + b_row + col0);
            fb01 = lds_read16(cur + b_row + col1);
            fb10 = lds_read16(cur + b_row + 16 * kSlice + col0);
            fb11 = lds_read16(cur + b_row + 16 * kSlice + col1);
            lds_settle(fa0, fa1, fb00, fb01, fb10, fb11);
            mma<D>(fa0, fb00, part[0]);
            mma<D>(fa0, fb10, part[1]);
            mma<D>(fa1, fb01, part[0]);
            mma<D>(fa1, fb11, part[1]);
        };
        for (int i = 0; i < NST - 1; ++i) issue_next();
        unroll<NPTS>([&](auto qc) __attribute__((always_inline)) {
            chunk(qc, true);   // the first chunk folds the previous domain point
            for (int c = 1; c < n_ch; ++c) chunk(qc, false);
        });
        fold(std::integral_constant<int, NPTS - 1>{});
        // the trailing zero-fill groups land before the LDS is reused
        __builtin_amdgcn_s_waitcnt(vm_wait(0));
    } else {
        // prologue: steps 0 .. NST-2 requested
        unroll<NST - 1>([&](auto sc) __attribute__((always_inline)) {
            if constexpr (decltype(sc)::value < NSTEPS) issue(sc);
        });
        unroll<NSTEPS>(step);
        fold(std::integral_constant<int, NPTS - 1>{});
    }
    // the output tile is complete here: without this, the compiler sinks the
    // folds of every step into the (conditional) store code after the loop
#pragma unroll
    for (int w = 0; w < WT; ++w)
#pragma unroll
        for (int o = 0; o < MM; ++o)
#pragma unroll
            for (int q = 0; q < MM; ++q)
#pragma unroll
                for (int r = 0; r < 4; ++r) asm volatile("" : "+v"(Y[w][o][q][r]));

    // epilogue, one 16-tile block at a time: each lane parks its four
    // channels of every pixel in LDS (records of 64 channels per pixel, the
    // 16-byte chunks XOR-swizzled by tile), then the block's records go out
    // with 16 contiguous bytes per lane.  Channel counts that are not a
    // multiple of a 16-byte chunk take the direct per-lane store instead.
    constexpr int ES = static_cast<int>(sizeof(Elem));
    constexpr int kRec = 64 * ES;               // bytes of a pixel record
    constexpr int kPx = MM * MM;                // pixels of a tile
    constexpr int kLanesPerRec = kRec / 16;
    constexpr int kRecPerIns = 64 / kLanesPerRec;
    constexpr int kInsPerWave = 16 * kPx / kRecPerIns / 4;
    const bool staged = (K * ES) % 16 == 0;
    if (staged) {
        unsigned char* ybytes = reinterpret_cast<unsigned char*>(y);
        const int chunk = lane % kLanesPerRec;
        // coordinates of the block's first tile; a later tile of the block is
        // reached by stepping (T < 2^31 here, so 32-bit arithmetic)
        const int tw = static_cast<int>(geo.tw), th = static_cast<int>(geo.th);
        const int H = static_cast<int>(geo.H), W = static_cast<int>(geo.W);
        const int tx0 = static_cast<int>(t0 % geo.tw);
        const int ty0 = static_cast<int>((t0 / geo.tw) % geo.th);
        const int n0 = static_cast<int>(t0 / (geo.tw * geo.th));
#pragma unroll
        for (int w = 0; w < WT; ++w) {
            // every wave is done with the LDS (the stages, or the previous block's records)
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            lds_barrier();
#pragma unroll
            for (int o = 0; o < MM; ++o)
#pragma unroll
                for (int q = 0; q < MM; ++q) {
                    const int rec = l16 * kPx + o * MM + q;
                    const int byte = (wave * 16 + 4 * grp) * ES;      // within the record
                    const int phys = (((byte >> 4) ^ (l16 & 7)) << 4) | (byte & 15);
                    unsigned char* dst = lds + rec * kRec + phys;
                    if constexpr (ES == 4) {
                        *reinterpret_cast<f32x4*>(dst) = f32x4{Y[w][o][q][0], Y[w][o][q][1], Y[w][o][q][2], Y[w][o][q][3]};
                    } else {
                        const uint32_t lo = bits16(S::from_f32(Y[w][o][q][0])) | (bits16(S::from_f32(Y[w][o][q][1])) << 16);
                        const uint32_t hi = bits16(S::from_f32(Y[w][o][q][2])) | (bits16(S::from_f32(Y[w][o][q][3])) << 16);
                        *reinterpret_cast<u32x2*>(dst) = u32x2{lo, hi};
                    }
                }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the records are in LDS
            lds_barrier();
#pragma unroll
            for (int i = 0; i < kInsPerWave; ++i) {
                const int rec = (wave * kInsPerWave + i) * kRecPerIns + lane / kLanesPerRec;
                const int tl = rec / kPx, px = rec % kPx;
                const u32x4 v = *reinterpret_cast<const u32x4*>(lds + rec * kRec + ((chunk ^ (tl & 7)) << 4));
                int tx = tx0 + w * 16 + tl, ty = ty0, n = n0;
                while (tx >= tw) {
                    tx -= tw;
                    if (++ty == th) {
                        ty = 0;
                        ++n;
                    }
                }
                const int hr = ty * MM + px / MM, wc = tx * MM + px % MM;
                const int64_t ch = k0 + chunk * (16 / ES);
                // non-temporal: y is written once and read by the next kernel, and
                // as a streaming store it does not push out of L2 the U and V rows
                // that the other blocks of this XCD are still reading
                if (t0 + w * 16 + tl < T && hr < H && wc < W && ch < K)
                    __builtin_nontemporal_store(
                        v, reinterpret_cast<u32x4*>(ybytes + ((static_cast<int64_t>(n * H + hr) * W + wc) * K + ch) * ES));
            }
        }
        return;
    }
    const int64_t k = k0 + wave * 16 + 4 * grp;
    if (k >= K) return;
#pragma unroll
    for (int w = 0; w < WT; ++w) {
        const int64_t tile = t0 + w * 16 + l16;
        if (tile >= T) continue;
        const int64_t tx = tile % geo.tw;
        const int64_t ty = (tile / geo.tw) % geo.th;
        const int64_t n = tile / (geo.tw * geo.th);
#pragma unroll
        for (int o = 0; o < MM; ++o) {
            const int64_t hr = ty * MM + o;
            if (hr >= geo.H) break;
#pragma unroll
            for (int q = 0; q < MM; ++q) {
                const int64_t wc = tx * MM + q;
                if (wc >= geo.W) break;
                Elem* dst = y + ((n * geo.H + hr) * geo.W + wc) * K + k;
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (k + r < K) dst[r] = S::from_f32(Y[w][o][q][r]);
            }
        }
    }
}

// tile blocks per wave: as many as the output-tile registers allow (Y holds
// m^2 values per channel-tile pair); with 64-channel blocks two (the unrolled
// kernel's block), else fewer when that leaves CUs idle
int pick_wt(const Geometry& g, int kw) {
    if (g.m > 4) return 1;
    if (kw == 4) return 2;   // the unrolled kernel's block: 64 output channels x 32 tiles
    const int64_t n_kb = (g.K + 16 * kw - 1) / (16 * kw);
    const int64_t n_tb2 = (g.T + 16 * 2 * (4 / kw) - 1) / (16 * 2 * (4 / kw));
    return n_kb * n_tb2 >= 2 * device_cu_count() ? 2 : 1;
}

}  // namespace

template <>
bool contract_output_supported_t<WG_DTYPE>(const Geometry& g) {
    const int64_t rb = g.Cp * (WG_DTYPE == 0 ? 4 : 2);
    if (g.t > 8 || (g.t & 1) != 0 || !transform_shape_supported(g.t, g.alpha)) return false;
    // 32-bit buffer offsets: within a plane, and for every staged row of a block
    return g.T * rb < 0xffff0000LL && g.K * rb < 0xffff0000LL && rb <= (1 << 20);
}

// the input transform fused into the prologue: rows of at most 32 bytes (8 or
// 4 domain points per step), more than 32 output channels (so a block has
// 32 tiles whatever its shape) and the block's V rows within 48 KB of LDS (two
// workgroups per CU)
template <>
bool input_contract_output_supported_t<WG_DTYPE>(const Geometry& g) {
    const int64_t rb = g.Cp * (WG_DTYPE == 0 ? 4 : 2);
    const int64_t a2 = static_cast<int64_t>(g.alpha) * g.alpha;
    if (!contract_output_supported_t<WG_DTYPE>(g) || rb > 32 || g.K <= 32) return false;
    const int64_t vrow = rb <= 16 ? 16 : 32;
    return a2 * g.K * rb < 0xffff0000LL && a2 * 32 * vrow <= 49152;
}

namespace {

struct CoArgs {
    const unsigned char* V;
    const unsigned char* U;
    void* y;
    OutputTable tab;
    Geometry g;
    int kw, n_kb, rb, n_slices, xp;
    const void* x;
    InputTable itab;
    unsigned nb;
};

template <int D, int TT, int A, int W, bool NAR, int K1, bool ONE>
hipError_t launch_co_instance(const CoArgs& c, hipStream_t stream) {
    using Elem = typename DTypeOf<D>::type;
    if constexpr (k1_vbuf_bytes<A, K1>() <= 49152) {
        hipLaunchKernelGGL((contract_output_kernel<D, TT - 2, A, W, NAR, K1, ONE>), dim3(c.nb), dim3(kThreads), 0, stream,
                           c.V, c.U, static_cast<Elem*>(c.y), c.tab, c.g, c.kw, c.n_kb, c.rb, c.n_slices, c.xp,
                           static_cast<const Elem*>(c.x), c.itab);
        return hipGetLastError();
    } else {
        return hipErrorInvalidValue;
    }
}

template <int D, int TT, int A, class CO>
hipError_t launch_unrolled_instance(const CoArgs& c, hipStream_t stream) {
    using Elem = typename DTypeOf<D>::type;
#define WG_UNR_LAUNCH(NSL, XP, CH, NCK)                                                                         \
    hipLaunchKernelGGL((contract_output_unrolled_kernel<D, TT - 2, A, CO, NSL, XP, CH, NCK>), dim3(c.nb),        \
                       dim3(kThreads), 0, stream, c.V, c.U, static_cast<Elem*>(c.y), c.tab, c.g, c.n_kb, c.rb,   \
                       (c.n_slices + 1) / 2)
    if (c.xp == 8) WG_UNR_LAUNCH(1, 8, false, 1);
    else if (c.xp == 4) WG_UNR_LAUNCH(1, 4, false, 1);
    else if (c.xp == 2) WG_UNR_LAUNCH(1, 2, false, 1);
    else if (c.n_slices == 1) WG_UNR_LAUNCH(1, 1, false, 1);
    else if (c.n_slices == 2) WG_UNR_LAUNCH(2, 1, false, 1);
    else if (c.n_slices <= 4) WG_UNR_LAUNCH(2, 1, false, 2);
    else WG_UNR_LAUNCH(2, 1, true, 1);
#undef WG_UNR_LAUNCH
    return hipGetLastError();
}

// x == nullptr: V from memory; else the input transform in the prologue.
// builtin: id of the built-in plan with the same tables, or -1.
template <int D>
hipError_t launch_co(const Geometry& g, const OutputTable& tab, const void* V, const void* U, void* y,
                     const void* x, const InputTable* itab, int builtin, hipStream_t stream) {
    const int rb = static_cast<int>(g.Cp * (D == 0 ? 4 : 2));
    const int kw0 = g.K <= 16 ? 1 : g.K <= 32 ? 2 : 4;
    const int wt = pick_wt(g, std::max(kw0, 2));
    const int kw = wt == 2 ? std::max(kw0, 2) : kw0;   // a stage holds at most 96 rows
    const int n_kb = static_cast<int>((g.K + 16 * kw - 1) / (16 * kw));
    const int64_t n_tb = (g.T + 16 * wt * (4 / kw) - 1) / (16 * wt * (4 / kw));
    const int64_t grid = n_kb * n_tb;
    if (grid > 0x7fffffff) return hipErrorInvalidValue;
    // rows of at most 64 bytes: several domain points per step (all planes
    // addressed with 32-bit offsets); else one 128-byte slice per step
    int xp = 1;
    const int64_t a2 = static_cast<int64_t>(g.alpha) * g.alpha;
    if (x) xp = rb <= 16 ? 8 : 4;   // checked by input_contract_output_supported_t
    else if (rb <= 64 && a2 * g.T * rb < 0xffff0000LL && a2 * g.K * rb < 0xffff0000LL)
        xp = rb <= 16 ? 8 : rb <= 32 ? 4 : 2;
    CoArgs c;
    c.V = static_cast<const unsigned char*>(x ? U : V);   // unused with the input transform fused
    c.U = static_cast<const unsigned char*>(U);
    c.y = y;
    c.tab = tab;
    c.g = g;
    c.kw = kw;
    c.n_kb = n_kb;
    c.rb = rb;
    c.n_slices = xp > 1 ? 1 : (rb + kSlice - 1) / kSlice;
    c.xp = xp;
    c.x = x;
    if (itab) c.itab = *itab;
    else std::memset(&c.itab, 0, sizeof(c.itab));
    c.nb = static_cast<unsigned>(grid);
    if (!x && wt == 2 && kw == 4) {
        // whole rows per step, blocks of 64 output channels x 32 tiles
        switch (builtin) {
#define WG_UNR_BUILTIN(ID, TT, A)                                                                          \
    case ID:                                                                                               \
        if constexpr (TT <= 6)                                                                             \
            if (g.t == TT && g.alpha == A) return launch_unrolled_instance<D, TT, A, ConstCoefs<BuiltinPlan##ID>>(c, stream); \
        break;
            WG_BUILTIN_PLANS(WG_UNR_BUILTIN)
#undef WG_UNR_BUILTIN
            default:
                break;
        }
#define WG_UNR_CASE(TT, A) \
        if (g.t == TT && g.alpha == A) return launch_unrolled_instance<D, TT, A, RuntimeCoefs>(c, stream);
        WG_UNR_CASE(4, 4) WG_UNR_CASE(4, 5) WG_UNR_CASE(4, 6) WG_UNR_CASE(4, 7)
        WG_UNR_CASE(6, 6) WG_UNR_CASE(6, 7) WG_UNR_CASE(6, 8) WG_UNR_CASE(6, 9)
#undef WG_UNR_CASE
    }
#define WG_CO_CASE(TT, A, W)                                                                              \
    if (g.t == TT && g.alpha == A && wt == W) {                                                           \
        if (x && xp == 8) return launch_co_instance<D, TT, A, W, true, 8, true>(c, stream);               \
        if (x) return launch_co_instance<D, TT, A, W, true, 4, true>(c, stream);                          \
        if (xp > 1) return launch_co_instance<D, TT, A, W, true, 0, true>(c, stream);                     \
        if (c.n_slices == 1) return launch_co_instance<D, TT, A, W, false, 0, true>(c, stream);           \
        return launch_co_instance<D, TT, A, W, false, 0, false>(c, stream);                               \
    }
    WG_CO_CASE(4, 4, 1) WG_CO_CASE(4, 5, 1) WG_CO_CASE(4, 6, 1) WG_CO_CASE(4, 7, 1)
    WG_CO_CASE(4, 4, 2) WG_CO_CASE(4, 5, 2) WG_CO_CASE(4, 6, 2) WG_CO_CASE(4, 7, 2)
    WG_CO_CASE(6, 6, 1) WG_CO_CASE(6, 7, 1) WG_CO_CASE(6, 8, 1) WG_CO_CASE(6, 9, 1)
    WG_CO_CASE(6, 6, 2) WG_CO_CASE(6, 7, 2) WG_CO_CASE(6, 8, 2) WG_CO_CASE(6, 9, 2)
    WG_CO_CASE(8, 8, 1) WG_CO_CASE(8, 9, 1) WG_CO_CASE(8, 10, 1) WG_CO_CASE(8, 11, 1) WG_CO_CASE(8, 12, 1)
#undef WG_CO_CASE
    return hipErrorInvalidValue;
}

}  // namespace

template <>
hipError_t launch_contract_output_t<WG_DTYPE>(const Geometry& g, const OutputTable& tab, const void* V,
                                              const void* U, void* y, int builtin, hipStream_t stream) {
    if (!contract_output_supported_t<WG_DTYPE>(g)) return hipErrorInvalidValue;
    return launch_co<WG_DTYPE>(g, tab, V, U, y, nullptr, nullptr, builtin, stream);
}

template <>
hipError_t launch_input_contract_output_t<WG_DTYPE>(const Geometry& g, const InputTable& itab,
                                                    const OutputTable& otab, const void* x, const void* U, void* y,
                                                    hipStream_t stream) {
    if (!input_contract_output_supported_t<WG_DTYPE>(g) || !x) return hipErrorInvalidValue;
    return launch_co<WG_DTYPE>(g, otab, nullptr, U, y, x, &itab, -1, stream);
}

}  // namespace wg
