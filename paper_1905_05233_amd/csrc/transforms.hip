// Winograd transforms of eq. (2) (Barabasz & Gregg, arXiv 1905.05233) for
// gfx950: the kernel transform U = G g G^T, the input transform V = B^T d B
// and the output transform Y = A^T M A fused with the NHWC store.
//
// All three stream channel-last data: a wavefront's loads and stores sweep 64
// consecutive channels of NHWC / channel-last buffers (coalesced).  The kernel
// transform runs one thread per (domain row, kernel, channel), the input
// transform one workgroup per (tile, 64 channels) with its window staged in
// LDS and its domain rows split over the waves, the output transform one
// workgroup per (tile, 64 output channels) with its output rows split over
// the waves.  The transform matrices arrive by value
// in the kernel-argument segment (uniform across the grid, so they live in
// scalar registers); the small matrices are applied as two separable 1D passes
// in fp32 registers with ascending-index fused multiply-adds, and results are
// rounded to the storage dtype once, at the store.
//
// This file is compiled once per storage dtype (WG_DTYPE = 0 fp32, 1 fp16,
// 2 bf16); each (input tile, alpha') shape is a template instance so that the
// register arrays have compile-time sizes.
#include <utility>

#include "coefs.hpp"
#include "device_common.hpp"
#include "kernels.hpp"

#ifndef WG_DTYPE
#error "compile with -DWG_DTYPE=0|1|2"
#endif

namespace wg {

namespace {

constexpr int kBlock = 256;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// ----------------------------------------------------------------- kernel
// U[xi = a*alpha + b][k][c] = sum_j (sum_i G[a][i] g[i][j]) G[b][j]; one thread
// per (row a, k, run of kRun channels), runs fastest, so loads and stores are
// kRun elements per lane (16 bytes in the stand-alone kernel; 4 channels when
// it shares a launch with the input transform, to keep that kernel's register
// count low).  kWhole: C is a multiple of the run, so the runs of w are
// aligned; otherwise w is read element by element.
template <int BYTES> struct RunBits;
template <> struct RunBits<16> { using type = uint4; };
template <> struct RunBits<8> { using type = uint2; };

template <typename Elem, int ALPHA, int kRun, bool kWhole>
__device__ __forceinline__ void kernel_transform_run(const KernelTable& tab, const Elem* __restrict__ w,
                                                     Elem* __restrict__ U, int64_t K, int64_t C, int64_t Cp,
                                                     int64_t gid) {
    using S = Storage<Elem>;
    using Bits = typename RunBits<kRun * sizeof(Elem)>::type;
    const int64_t runs = Cp / kRun;                              // Cp is a multiple of 8
    if (gid >= ALPHA * K * runs) return;
    const int64_t c = (gid % runs) * kRun;
    const int64_t k = (gid / runs) % K;
    const int a = static_cast<int>(gid / (runs * K));
    const int64_t plane = K * Cp;
    float g[3][3][kRun];
#pragma unroll
    for (int i = 0; i < 3; ++i)
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            const Elem* src = w + ((k * 3 + i) * 3 + j) * C + c;
            Elem e[kRun];
            if constexpr (kWhole) {
                // a run starts inside C only if it ends inside it (for fp32, Cp may exceed C by a run)
                *reinterpret_cast<Bits*>(e) = c < C ? *reinterpret_cast<const Bits*>(src) : Bits{};
            } else {
#pragma unroll
                for (int q = 0; q < kRun; ++q) e[q] = c + q < C ? src[q] : S::from_f32(0.0f);
            }
#pragma unroll
            for (int q = 0; q < kRun; ++q) g[i][j][q] = S::to_f32(e[q]);
        }
    float Gg[3][kRun];
#pragma unroll
    for (int j = 0; j < 3; ++j)
#pragma unroll
        for (int q = 0; q < kRun; ++q) {
            float acc = 0.0f;
#pragma unroll
            for (int i = 0; i < 3; ++i) acc = __builtin_fmaf(tab.g[a * 3 + i], g[i][j][q], acc);
            Gg[j][q] = acc;
        }
    Elem* out = U + static_cast<int64_t>(a) * ALPHA * plane + k * Cp + c;
#pragma unroll
    for (int b = 0; b < ALPHA; ++b) {
        Elem e[kRun];
#pragma unroll
        for (int q = 0; q < kRun; ++q) {
            float acc = 0.0f;
#pragma unroll
            for (int j = 0; j < 3; ++j) acc = __builtin_fmaf(Gg[j][q], tab.g[b * 3 + j], acc);
            e[q] = S::from_f32(acc);   // channels past C: g = 0, so zeros
        }
        *reinterpret_cast<Bits*>(out + b * plane) = *reinterpret_cast<const Bits*>(e);
    }
}

// The same, one thread per (k, run of kRun channels) computing every row a:
// the 3x3 taps are loaded once instead of once per row, and a launch needs
// alpha' times fewer threads (the form the combined kernel/input launch uses,
// so that fewer kernel-transform workgroups precede the input-transform ones).
// Each output is computed in the same order as above.
template <typename Elem, int ALPHA, int kRun, bool kWhole>
__device__ __forceinline__ void kernel_transform_rows(const KernelTable& tab, const Elem* __restrict__ w,
                                                      Elem* __restrict__ U, int64_t K, int64_t C, int64_t Cp,
                                                      int64_t gid) {
    using S = Storage<Elem>;
    using Bits = typename RunBits<kRun * sizeof(Elem)>::type;
    const int64_t runs = Cp / kRun;
    if (gid >= K * runs) return;
    const int64_t c = (gid % runs) * kRun;
    const int64_t k = gid / runs;
    const int64_t plane = K * Cp;
    float g[3][3][kRun];
#pragma unroll
    for (int i = 0; i < 3; ++i)
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            const Elem* src = w + ((k * 3 + i) * 3 + j) * C + c;
            Elem e[kRun];
            if constexpr (kWhole) {
                *reinterpret_cast<Bits*>(e) = c < C ? *reinterpret_cast<const Bits*>(src) : Bits{};
            } else {
#pragma unroll
                for (int q = 0; q < kRun; ++q) e[q] = c + q < C ? src[q] : S::from_f32(0.0f);
            }
#pragma unroll
            for (int q = 0; q < kRun; ++q) g[i][j][q] = S::to_f32(e[q]);
        }
    Elem* out = U + k * Cp + c;
#pragma unroll
    for (int a = 0; a < ALPHA; ++a) {
        float Gg[3][kRun];
#pragma unroll
        for (int j = 0; j < 3; ++j)
#pragma unroll
            for (int q = 0; q < kRun; ++q) {
                float acc = 0.0f;
#pragma unroll
                for (int i = 0; i < 3; ++i) acc = __builtin_fmaf(tab.g[a * 3 + i], g[i][j][q], acc);
                Gg[j][q] = acc;
            }
#pragma unroll
        for (int b = 0; b < ALPHA; ++b) {
            Elem e[kRun];
#pragma unroll
            for (int q = 0; q < kRun; ++q) {
                float acc = 0.0f;
#pragma unroll
                for (int j = 0; j < 3; ++j) acc = __builtin_fmaf(Gg[j][q], tab.g[b * 3 + j], acc);
                e[q] = S::from_f32(acc);
            }
            *reinterpret_cast<Bits*>(out + (a * ALPHA + b) * plane) = *reinterpret_cast<const Bits*>(e);
        }
    }
}

template <typename Elem, int ALPHA, bool kWhole>
__global__ __launch_bounds__(kBlock) void kernel_transform(KernelTable tab, const Elem* __restrict__ w,
                                                           Elem* __restrict__ U, int64_t K, int64_t C,
                                                           int64_t Cp) {
    kernel_transform_run<Elem, ALPHA, 16 / sizeof(Elem), kWhole>(tab, w, U, K, C, Cp,
                                                                 static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x);
}

// ------------------------------------------------------------------ input
// V[xi = a*alpha + b][tile][c] = sum_v (sum_u B^T[a][u] d[u][v]) B^T[b][v],
// d = the (m+2)^2 window whose top-left pixel is (ty*m - 1, tx*m - 1).
//
// One workgroup per (tile, 64 channels).  The t x t x 64 window (neighbouring
// tiles overlap by two pixels) is fetched with coalesced 16-byte NHWC loads,
// zero outside the image and past C, converted to fp32 once and staged in
// LDS.  The alpha' output rows are split over the waves: wave g computes rows
// [g*R, g*R + R) for its 64 channels, so each wave runs both passes for few
// rows and the workgroup's VALU work is spread over several waves.  Row
// indices are compile-time constants in every wave (one template instance per
// row group), which keeps the coefficients in scalar registers.
constexpr int kInCh = 64;   // LDS columns per workgroup, one per lane

// channels per tile in a workgroup: 64, or fewer for narrow layers so that the
// lanes still find work (Cp is a multiple of 8: 8, 16, 32 or 64)
__host__ __device__ inline int input_column_width(int64_t Cp) {
    return Cp >= 64 ? 64 : Cp > 16 ? 32 : Cp > 8 ? 16 : 8;
}
// Tiles a wide-layer workgroup walks in turn (PT, a template parameter of
// the kernel: the next two windows are fetched while the current one is
// transformed).  PT = kInTiles for layers with many units (fewer,
// longer-lived workgroups); PT = 1 for small ones, which spreads them over
// more CUs and keeps the leaner single-tile instance (fewer registers).
constexpr int kInTiles = 4;
constexpr int64_t kInManyUnits = 8192;
// tiles per unit: PT in turn for wide layers, 64 / cw side by side for narrow ones
__host__ __device__ inline int input_tiles_per_unit(int64_t Cp, int pt) {
    const int cw = input_column_width(Cp);
    return cw == kInCh ? pt : kInCh / cw;
}
// the PT instance a layer runs (whole: C is a multiple of the 16-byte chunk)
inline int input_pt(const Geometry& g, bool whole) {
    const int cw = input_column_width(g.Cp);
    if (!whole || cw != kInCh) return 1;
    return g.T * ((g.Cp + cw - 1) / cw) >= kInManyUnits ? kInTiles : 1;
}
// workgroups (units) of the input transform
inline int64_t input_units(const Geometry& g, int pt) {
    const int cw = input_column_width(g.Cp);
    const int nt = input_tiles_per_unit(g.Cp, pt);
    return (g.T + nt - 1) / nt * ((g.Cp + cw - 1) / cw);
}

// rows per wave: the split that measured fastest for each alpha'
constexpr int input_rows_per_wave(int alpha) { return alpha == 7 || alpha == 8 ? 2 : 3; }

template <typename Elem, int TT, int ALPHA>
struct InputShape {
    static constexpr int kR = input_rows_per_wave(ALPHA);
    static constexpr int kG = (ALPHA + kR - 1) / kR;                  // waves (row groups)
    static constexpr int kThreads = 64 * kG;
    static constexpr int kChunkElems = 16 / static_cast<int>(sizeof(Elem));
    static constexpr int kChunksPerPix = kInCh / kChunkElems;
    static constexpr int kChunks = TT * TT * kChunksPerPix;            // 16-byte chunks per window
    static constexpr int kPer = (kChunks + kThreads - 1) / kThreads;
};

// Both passes for rows A0 .. A0+R-1 of one (tile, channel): pass 1 in ascending
// u, pass 2 in ascending v, rounded to the storage type at the store.
template <typename Elem, int TT, int ALPHA, int R, int A0, class CO>
__device__ __forceinline__ void input_rows(const InputTable& tab, const float* wb, Elem* __restrict__ out,
                                           int64_t plane) {
    using S = Storage<Elem>;
    float W1[R][TT];
#pragma unroll
    for (int v = 0; v < TT; ++v) {
        float col[TT];
#pragma unroll
        for (int u = 0; u < TT; ++u) col[u] = wb[(u * TT + v) * kInCh];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            float acc = 0.0f;
            if (A0 + r < ALPHA) {
#pragma unroll
                for (int u = 0; u < TT; ++u) acc = term<CO>(CO::bt(tab, (A0 + r) * TT + u), col[u], acc);
            }
            W1[r][v] = acc;
        }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (A0 + r >= ALPHA) break;
#pragma unroll
        for (int b = 0; b < ALPHA; ++b) {
            float acc = 0.0f;
#pragma unroll
            for (int v = 0; v < TT; ++v) acc = term<CO>(CO::bt(tab, b * TT + v), W1[r][v], acc);
            out[((A0 + r) * ALPHA + b) * plane] = S::from_f32(acc);
        }
    }
}

template <typename Elem, int TT, int ALPHA, int R, class CO, int... Gs>
__device__ __forceinline__ void input_row_groups(int g, const InputTable& tab, const float* wb, Elem* out,
                                                 int64_t plane, std::integer_sequence<int, Gs...>) {
    ((g == Gs ? (input_rows<Elem, TT, ALPHA, R, Gs * R, CO>(tab, wb, out, plane), 0) : 0), ...);
}

// kWhole: C is a multiple of the 16-byte chunk width, so a chunk lies wholly
// inside or wholly past C; otherwise the window is fetched element by element.
template <typename Elem, int TT, int ALPHA, bool kWhole, class CO, int PT>
__device__ __forceinline__ void input_transform_unit(const InputTable& tab, const Elem* __restrict__ x,
                                                     Elem* __restrict__ V, const Geometry& geo, int64_t bid,
                                                     int64_t G) {
    using S = Storage<Elem>;
    using P = InputShape<Elem, TT, ALPHA>;
    __shared__ __attribute__((aligned(16))) float win[TT * TT * kInCh];   // [u][v][64] fp32

    // the 64 LDS columns (one per lane) hold cw channels of 64 / cw tiles:
    // cw = 64 for wide layers, the channel count rounded up to a power of two
    // for narrow ones (C = 3: 8 tiles of 8 channels per workgroup)
    const int cw = input_column_width(geo.Cp);
    const int cwl = __builtin_ctz(cw);   // cw is a power of two
    const int64_t nch = (geo.Cp + cw - 1) / cw;
    // XCD-aware numbering: the hardware deals workgroup ids round-robin to the
    // 8 XCDs; giving each XCD a contiguous run of units keeps neighbouring
    // tiles, whose windows overlap, in the same L2
    const int64_t unit = (G % 8 == 0) ? (bid % 8) * (G / 8) + bid / 8 : bid;
    const int per = input_tiles_per_unit(geo.Cp, PT);
    const int64_t tile0 = (unit / nch) * per;
    const int64_t c0 = (unit % nch) * cw;
    const int tw = static_cast<int>(geo.tw), th = static_cast<int>(geo.th);
    const int tid = threadIdx.x;
    // coordinates of the unit's first tile (the walking loop carries them on)
    int tx0 = static_cast<int>(tile0 % geo.tw);
    int ty0 = static_cast<int>((tile0 / geo.tw) % geo.th);
    int n0 = static_cast<int>(tile0 / (geo.tw * geo.th));

    uint4 regs[2][P::kPer];   // two register sets: windows in flight
    // the window of tile t at (tx0, ty0, n0) (wide: 64 channels of one tile;
    // narrow: cw channels of tiles t .. t + 64 / cw - 1, one per group of cw
    // LDS columns)
    auto fetch = [&](int64_t t, bool wide, int set = 0) __attribute__((always_inline)) {
#pragma unroll
    for (int p = 0; p < P::kPer; ++p) {
        const int ci = tid + p * P::kThreads;
        const int pix = ci / P::kChunksPerPix;
        const int col = (ci % P::kChunksPerPix) * P::kChunkElems;   // first LDS column of the chunk
        const int d = wide ? 0 : col >> cwl;   // tile of the workgroup, 0 .. 7
        const int64_t tile = t + d;
        // coordinates of t + d by carrying (no per-lane division); one
        // carry at most unless a row has fewer than 8 tiles
        int tx = tx0 + d, ty = ty0, n = n0;
        if (!wide && tx >= tw) {
            do {
                tx -= tw;
                if (++ty == th) {
                    ty = 0;
                    ++n;
                }
            } while (tx >= tw);
        }
        const int64_t hr = static_cast<int64_t>(ty) * geo.m - 1 + pix / TT;
        const int64_t wc = static_cast<int64_t>(tx) * geo.m - 1 + pix % TT;
        const int64_t cc = c0 + (wide ? col : col & (cw - 1));
        const bool in = ci < P::kChunks && tile < geo.T && hr >= 0 && hr < geo.H && wc >= 0 && wc < geo.W;
        const Elem* src = x + ((static_cast<int64_t>(n) * geo.H + hr) * geo.W + wc) * geo.C + cc;
        if constexpr (kWhole) {
            // large layers (the walking instance) stream their input: it is
            // read here and by no later kernel of the layer, so it is kept out
            // of the last-level cache, which holds V for the contraction; a
            // small layer's input stays cached, which pays when the same layer
            // runs again (a 28x28 or 56x56 layer repeated back to back: 10.2
            // against 12.5 us)
            u32x4 t = u32x4{0u, 0u, 0u, 0u};
            if (in && cc < geo.C) {
                if constexpr (PT > 1) t = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src));
                else t = *reinterpret_cast<const u32x4*>(src);
            }
            regs[set][p] = uint4{t[0], t[1], t[2], t[3]};
        } else {
            Elem e[P::kChunkElems];
#pragma unroll
            for (int k = 0; k < P::kChunkElems; ++k) e[k] = (in && cc + k < geo.C) ? src[k] : S::from_f32(0.0f);
            regs[set][p] = __builtin_bit_cast(uint4, e);
        }
    }
    };
    auto park = [&](int set = 0) __attribute__((always_inline)) {
#pragma unroll
        for (int p = 0; p < P::kPer; ++p) {
            const int ci = tid + p * P::kThreads;
            if (ci < P::kChunks) {
                const Elem* e = reinterpret_cast<const Elem*>(&regs[set][p]);
#pragma unroll
                for (int k = 0; k < P::kChunkElems; ++k) win[ci * P::kChunkElems + k] = S::to_f32(e[k]);
            }
        }
    };

    const int c = tid % kInCh;
    const int g = __builtin_amdgcn_readfirstlane(tid / kInCh);
    // channels C..Cp-1 read as zero and so store zeros
    if (PT > 1 && cw == kInCh) {
        // wide, PT > 1: PT consecutive tiles in turn; the next two windows
        // are in flight while the current one is transformed, in alternating
        // register sets (the loop is unrolled, so the set indices are
        // constants and the compiler's waits for the window loads are exact;
        // a VGG-16 pass measured 1.76 against 1.78 ms with one window ahead,
        // the layer input being read from HBM)
        const int64_t cg = c0 + c;
        auto advance = [&]() __attribute__((always_inline)) {
            if (++tx0 == tw) {
                tx0 = 0;
                if (++ty0 == th) {
                    ty0 = 0;
                    ++n0;
                }
            }
        };
        fetch(tile0, true, 0);
        advance();
        fetch(tile0 + 1, true, 1);
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            const int64_t tile = tile0 + i;
            if (i > 0) __syncthreads();   // the last tile's rows have read the window
            park(i % 2);
            __syncthreads();
            if (i + 2 < PT) {
                advance();
                fetch(tile + 2, true, i % 2);
            }
            if (tile < geo.T && cg < geo.Cp)
                input_row_groups<Elem, TT, ALPHA, P::kR, CO>(g, tab, win + c, V + tile * geo.Cp + cg,
                                                             geo.T * geo.Cp,
                                                             std::make_integer_sequence<int, P::kG>{});
        }
        return;
    }
    // one window: a wide layer's single tile (coordinates uniform) or a
    // narrow layer's tiles side by side
    if (cw == kInCh) fetch(tile0, true);
    else fetch(tile0, false);
    park();
    __syncthreads();
    const int64_t tile = tile0 + (c >> cwl);
    const int64_t cg = c0 + (c & (cw - 1));
    if (tile >= geo.T || cg >= geo.Cp) return;
    input_row_groups<Elem, TT, ALPHA, P::kR, CO>(g, tab, win + c, V + tile * geo.Cp + cg, geo.T * geo.Cp,
                                                 std::make_integer_sequence<int, P::kG>{});
}

template <typename Elem, int TT, int ALPHA, bool kWhole, class CO, int PT>
__global__ __launch_bounds__((InputShape<Elem, TT, ALPHA>::kThreads)) void input_transform(
    InputTable tab, const Elem* __restrict__ x, Elem* __restrict__ V, Geometry geo) {
    input_transform_unit<Elem, TT, ALPHA, kWhole, CO, PT>(tab, x, V, geo, blockIdx.x, gridDim.x);
}

// The kernel and input transforms are independent: conv2d runs them as one
// launch.  The first n_kt workgroups each take P::kThreads (k, 4-channel run)
// pairs of the kernel transform, every row a of each, the rest are
// input-transform units (one launch instead of two, and the short kernel
// transform overlaps the input transform).
template <typename Elem, int TT, int ALPHA, bool kWhole, class CO, int PT>
__global__ __launch_bounds__((InputShape<Elem, TT, ALPHA>::kThreads)) void kernel_input_transform(
    KernelTable ktab, InputTable itab, const Elem* __restrict__ w, const Elem* __restrict__ x,
    Elem* __restrict__ U, Elem* __restrict__ V, Geometry geo, int64_t n_kt) {
    using P = InputShape<Elem, TT, ALPHA>;
    const int64_t bid = blockIdx.x;
    if (bid < n_kt) {
        kernel_transform_rows<Elem, ALPHA, 4, kWhole>(ktab, w, U, geo.K, geo.C, geo.Cp, bid * P::kThreads + threadIdx.x);
        return;
    }
    input_transform_unit<Elem, TT, ALPHA, kWhole, CO, PT>(itab, x, V, geo, bid - n_kt, gridDim.x - n_kt);
}

// ----------------------------------------------------------------- output
// y[n][ty*m+o][tx*m+p][k] = sum_b (sum_a A^T[o][a] M[a][b]) A^T[p][b]
//
// One workgroup per (tile, 64 output channels); the m output rows are split
// over its waves (wave g computes rows [g*R, g*R + R) for its 64 channels).
// Every wave loads the tile's alpha'^2 values of M for its channels, all
// before any arithmetic (coalesced 256-byte rows; the repeats across the
// workgroup's waves are served by the caches), then runs pass 1 in ascending
// a and pass 2 in ascending b and stores its rows, masked at the right and
// bottom edges of the image.
constexpr int kOutCh = 64;   // output channels per workgroup, one per lane

// rows per wave: the split that measured fastest
constexpr int output_rows_per_wave(int alpha) { return alpha >= 9 ? 3 : 2; }

template <int MM, int ALPHA>
struct OutputShape {
    static constexpr int kR = output_rows_per_wave(ALPHA);
    static constexpr int kG = (MM + kR - 1) / kR;   // waves (row groups)
    static constexpr int kThreads = 64 * kG;
};

template <typename Elem, int MM, int ALPHA, int O0, class CO>
__device__ __forceinline__ void output_rows(const OutputTable& tab, const float* __restrict__ in, int64_t plane,
                                            Elem* __restrict__ yk, int64_t hr0, int64_t wc0, const Geometry& geo) {
    using S = Storage<Elem>;
    constexpr int R = OutputShape<MM, ALPHA>::kR;
    float Mv[ALPHA][ALPHA];
#pragma unroll
    for (int a = 0; a < ALPHA; ++a)
#pragma unroll
        for (int b = 0; b < ALPHA; ++b) Mv[a][b] = in[(a * ALPHA + b) * plane];
    // pass 1, one domain column at a time: Z[r][b] = sum_a A^T[O0+r][a] M[a][b]
    float Z[R][ALPHA];
#pragma unroll
    for (int b = 0; b < ALPHA; ++b)
#pragma unroll
        for (int r = 0; r < R; ++r) {
            float acc = 0.0f;
            if (O0 + r < MM) {
#pragma unroll
                for (int a = 0; a < ALPHA; ++a) acc = term<CO>(CO::at(tab, (O0 + r) * ALPHA + a), Mv[a][b], acc);
            }
            Z[r][b] = acc;
        }
    // pass 2 and the masked NHWC store
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t hr = hr0 + O0 + r;
        if (O0 + r >= MM || hr >= geo.H) break;
#pragma unroll
        for (int p = 0; p < MM; ++p) {
            const int64_t wc = wc0 + p;
            float acc = 0.0f;
#pragma unroll
            for (int b = 0; b < ALPHA; ++b) acc = term<CO>(CO::at(tab, p * ALPHA + b), Z[r][b], acc);
            if (wc < geo.W) yk[(hr * geo.W + wc) * geo.K] = S::from_f32(acc);
        }
    }
}

template <typename Elem, int MM, int ALPHA, class CO, int... Gs>
__device__ __forceinline__ void output_row_groups(int g, const OutputTable& tab, const float* in, int64_t plane,
                                                  Elem* yk, int64_t hr0, int64_t wc0, const Geometry& geo,
                                                  std::integer_sequence<int, Gs...>) {
    ((g == Gs ? (output_rows<Elem, MM, ALPHA, Gs * OutputShape<MM, ALPHA>::kR, CO>(tab, in, plane, yk, hr0, wc0, geo),
                 0)
              : 0),
     ...);
}

template <typename Elem, int MM, int ALPHA, class CO>
__global__ __launch_bounds__((OutputShape<MM, ALPHA>::kThreads)) void output_transform(
    OutputTable tab, const float* __restrict__ Mx, Elem* __restrict__ y, Geometry geo) {
    const int64_t nkc = (geo.K + kOutCh - 1) / kOutCh;
    const int64_t unit = blockIdx.x;
    const int64_t tile = unit / nkc;
    const int64_t k = (unit % nkc) * kOutCh + threadIdx.x % kOutCh;
    const int g = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kOutCh);
    if (k >= geo.K) return;
    const int64_t tx = tile % geo.tw;
    const int64_t ty = (tile / geo.tw) % geo.th;
    const int64_t n = tile / (geo.tw * geo.th);
    output_row_groups<Elem, MM, ALPHA, CO>(g, tab, Mx + tile * geo.Kp + k, geo.T * geo.Kp,
                                       y + n * geo.H * geo.W * geo.K + k, ty * MM, tx * MM, geo,
                                       std::make_integer_sequence<int, OutputShape<MM, ALPHA>::kG>{});
}

inline unsigned blocks_for(int64_t n) { return static_cast<unsigned>((n + kBlock - 1) / kBlock); }

}  // namespace

// ------------------------------------------------------------- launchers

template <int D>
hipError_t launch_kernel_transform_t(const Geometry& g, const KernelTable& tab, const void* w, void* U,
                                     hipStream_t stream) {
    using Elem = typename DTypeOf<D>::type;
    const auto* wp = static_cast<const Elem*>(w);
    auto* up = static_cast<Elem*>(U);
    constexpr int kRun = 16 / static_cast<int>(sizeof(Elem));
    const unsigned nb = blocks_for(static_cast<int64_t>(g.alpha) * g.K * (g.Cp / kRun));
    const bool whole = g.C % kRun == 0;
    switch (g.alpha) {
#define WG_KT_CASE(A)                                                                                   \
    case A:                                                                                             \
        if (whole)                                                                                      \
            hipLaunchKernelGGL((kernel_transform<Elem, A, true>), dim3(nb), dim3(kBlock), 0, stream, tab, wp, up, \
                               g.K, g.C, g.Cp);                                                         \
        else                                                                                            \
            hipLaunchKernelGGL((kernel_transform<Elem, A, false>), dim3(nb), dim3(kBlock), 0, stream, tab, wp, up, \
                               g.K, g.C, g.Cp);                                                         \
        break;
        WG_KT_CASE(4) WG_KT_CASE(5) WG_KT_CASE(6) WG_KT_CASE(7) WG_KT_CASE(8) WG_KT_CASE(9)
        WG_KT_CASE(10) WG_KT_CASE(11) WG_KT_CASE(12) WG_KT_CASE(13) WG_KT_CASE(14) WG_KT_CASE(15)
        WG_KT_CASE(16)
#undef WG_KT_CASE
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// One launch of each kernel shape, with the coefficient source CO.
template <typename Elem, int TT, int A, class CO>
hipError_t launch_it(const Geometry& g, const InputTable& tab, const Elem* xp, Elem* vp, hipStream_t stream) {
    constexpr int kChunkElems = 16 / static_cast<int>(sizeof(Elem));
    const bool whole = g.C % kChunkElems == 0;
    // the walking instance only with compile-time coefficients (with tables
    // read at run time its loop would hoist them all into registers)
    constexpr bool kWalk = !__is_same(CO, RuntimeCoefs);
    const int pt = kWalk ? input_pt(g, whole) : 1;
    const int64_t units = input_units(g, pt);
    if (units > 0x7fffffff) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(units)), block(InputShape<Elem, TT, A>::kThreads);
    if constexpr (kWalk)
        if (whole && pt == kInTiles) {
            hipLaunchKernelGGL((input_transform<Elem, TT, A, true, CO, kInTiles>), grid, block, 0, stream, tab, xp, vp,
                               g);
            return hipGetLastError();
        }
    if (whole)
        hipLaunchKernelGGL((input_transform<Elem, TT, A, true, CO, 1>), grid, block, 0, stream, tab, xp, vp, g);
    else
        hipLaunchKernelGGL((input_transform<Elem, TT, A, false, CO, 1>), grid, block, 0, stream, tab, xp, vp, g);
    return hipGetLastError();
}

template <typename Elem, int TT, int A, class CO>
hipError_t launch_kit(const Geometry& g, const KernelTable& ktab, const InputTable& itab, const Elem* wp,
                      const Elem* xp, Elem* up, Elem* vp, hipStream_t stream) {
    constexpr int kChunkElems = 16 / static_cast<int>(sizeof(Elem));
    constexpr int kThr = InputShape<Elem, TT, A>::kThreads;
    const bool whole = g.C % kChunkElems == 0;   // then C is also a multiple of the 4-channel runs
    constexpr bool kWalk = !__is_same(CO, RuntimeCoefs);   // as in launch_it
    const int pt = kWalk ? input_pt(g, whole) : 1;
    const int64_t units = input_units(g, pt);
    const int64_t kt_runs = g.K * (g.Cp / 4);   // one thread per (k, 4-channel run), every row a
    // a multiple of 8, so the input transform's ids keep their XCD (id mod 8)
    const int64_t n_kt = (kt_runs + 8 * kThr - 1) / (8 * kThr) * 8;
    if (n_kt + units > 0x7fffffff) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(n_kt + units));
    if constexpr (kWalk)
        if (whole && pt == kInTiles) {
            hipLaunchKernelGGL((kernel_input_transform<Elem, TT, A, true, CO, kInTiles>), grid, dim3(kThr), 0, stream,
                               ktab, itab, wp, xp, up, vp, g, n_kt);
            return hipGetLastError();
        }
    if (whole)
        hipLaunchKernelGGL((kernel_input_transform<Elem, TT, A, true, CO, 1>), grid, dim3(kThr), 0, stream, ktab,
                           itab, wp, xp, up, vp, g, n_kt);
    else
        hipLaunchKernelGGL((kernel_input_transform<Elem, TT, A, false, CO, 1>), grid, dim3(kThr), 0, stream, ktab,
                           itab, wp, xp, up, vp, g, n_kt);
    return hipGetLastError();
}

template <typename Elem, int TT, int A, class CO>
hipError_t launch_ot(const Geometry& g, const OutputTable& tab, const float* M, Elem* yp, hipStream_t stream) {
    const int64_t units = g.T * ((g.K + kOutCh - 1) / kOutCh);
    if (units > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((output_transform<Elem, TT - 2, A, CO>), dim3(static_cast<unsigned>(units)),
                       dim3(OutputShape<TT - 2, A>::kThreads), 0, stream, tab, M, yp, g);
    return hipGetLastError();
}

// Dispatch: the constant-coefficient instance of a built-in plan (builtin =
// its id, when the shape matches), else the kernel-argument tables.
template <int D>
hipError_t launch_input_transform_t(const Geometry& g, const InputTable& tab, const void* x, void* V,
                                    int builtin, hipStream_t stream) {
    using Elem = typename DTypeOf<D>::type;
    const auto* xp = static_cast<const Elem*>(x);
    auto* vp = static_cast<Elem*>(V);
    switch (builtin) {
#define WG_IT_BUILTIN(ID, TT, A)                                                                           \
    case ID:                                                                                               \
        if (g.t == TT && g.alpha == A) return launch_it<Elem, TT, A, ConstCoefs<BuiltinPlan##ID>>(g, tab, xp, vp, stream); \
        break;
        WG_BUILTIN_PLANS(WG_IT_BUILTIN)
#undef WG_IT_BUILTIN
        default:
            break;
    }
#define WG_IT_CASE(TT, A) \
    if (g.t == TT && g.alpha == A) return launch_it<Elem, TT, A, RuntimeCoefs>(g, tab, xp, vp, stream);
    WG_TRANSFORM_SHAPES(WG_IT_CASE)
    WG_TRANSFORM_SHAPES_ODD(WG_IT_CASE)
#undef WG_IT_CASE
    return hipErrorInvalidValue;
}

template <int D>
hipError_t launch_kernel_input_transform_t(const Geometry& g, const KernelTable& ktab, const InputTable& itab,
                                           const void* w, const void* x, void* U, void* V, int builtin,
                                           hipStream_t stream) {
    using Elem = typename DTypeOf<D>::type;
    const auto* wp = static_cast<const Elem*>(w);
    const auto* xp = static_cast<const Elem*>(x);
    auto* up = static_cast<Elem*>(U);
    auto* vp = static_cast<Elem*>(V);
    if (g.t > 8) {   // larger tiles: two launches (their input transform has no registers to spare)
        const hipError_t e = launch_kernel_transform_t<D>(g, ktab, w, U, stream);
        return e != hipSuccess ? e : launch_input_transform_t<D>(g, itab, x, V, builtin, stream);
    }
    switch (builtin) {
#define WG_KIT_BUILTIN(ID, TT, A)                                                                          \
    case ID:                                                                                               \
        if (g.t == TT && g.alpha == A)                                                                     \
            return launch_kit<Elem, TT, A, ConstCoefs<BuiltinPlan##ID>>(g, ktab, itab, wp, xp, up, vp, stream); \
        break;
        WG_BUILTIN_PLANS(WG_KIT_BUILTIN)
#undef WG_KIT_BUILTIN
        default:
            break;
    }
#define WG_KIT_CASE(TT, A)                                                                                 \
    if constexpr (TT <= 8)                                                                                 \
        if (g.t == TT && g.alpha == A) return launch_kit<Elem, TT, A, RuntimeCoefs>(g, ktab, itab, wp, xp, up, vp, stream);
    WG_TRANSFORM_SHAPES(WG_KIT_CASE)
    WG_TRANSFORM_SHAPES_ODD(WG_KIT_CASE)
#undef WG_KIT_CASE
    return hipErrorInvalidValue;
}

template <int D>
hipError_t launch_output_transform_t(const Geometry& g, const OutputTable& tab, const float* M, void* y,
                                     int builtin, hipStream_t stream) {
    using Elem = typename DTypeOf<D>::type;
    auto* yp = static_cast<Elem*>(y);
    switch (builtin) {
#define WG_OT_BUILTIN(ID, TT, A)                                                                           \
    case ID:                                                                                               \
        if (g.t == TT && g.alpha == A) return launch_ot<Elem, TT, A, ConstCoefs<BuiltinPlan##ID>>(g, tab, M, yp, stream); \
        break;
        WG_BUILTIN_PLANS(WG_OT_BUILTIN)
#undef WG_OT_BUILTIN
        default:
            break;
    }
#define WG_OT_CASE(TT, A) \
    if (g.t == TT && g.alpha == A) return launch_ot<Elem, TT, A, RuntimeCoefs>(g, tab, M, yp, stream);
    WG_TRANSFORM_SHAPES(WG_OT_CASE)
    WG_TRANSFORM_SHAPES_ODD(WG_OT_CASE)
#undef WG_OT_CASE
    return hipErrorInvalidValue;
}

template hipError_t launch_kernel_transform_t<WG_DTYPE>(const Geometry&, const KernelTable&, const void*, void*,
                                                        hipStream_t);
template hipError_t launch_input_transform_t<WG_DTYPE>(const Geometry&, const InputTable&, const void*, void*, int,
                                                       hipStream_t);
template hipError_t launch_kernel_input_transform_t<WG_DTYPE>(const Geometry&, const KernelTable&,
                                                              const InputTable&, const void*, const void*, void*,
                                                              void*, int, hipStream_t);
template hipError_t launch_output_transform_t<WG_DTYPE>(const Geometry&, const OutputTable&, const float*, void*,
                                                        int, hipStream_t);

}  // namespace wg
