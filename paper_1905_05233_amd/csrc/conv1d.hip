// 1D Winograd convolution F(m, 3) on gfx950: the one-dimensional form of the
// algorithm of Section 2 of Barabasz & Gregg (arXiv 1905.05233),
//     y = A^T [ (G g) (.) (B^T d) ],
// on input tiles d of m + 2 values overlapping by two, summed over input
// channels; Section 3.1 studies its error next to the 2D form.
//
// Layouts (channels last): x [N][1][L][C], w [K][1][3][C], y [N][1][L][K];
// U [alpha'][K][Cp], V [alpha'][T][Cp] (T = N * ceil(L / m), tile index
// t = n * ceil(L / m) + tx), M [alpha'][T][Kp] fp32.  The contraction is the
// 2D library's (alpha' planes instead of alpha'^2).
//
// Each transform is one 1D pass with the operation order of the 2D kernels:
// from zero, ascending index, one fused multiply-add per term in fp32, one
// rounding to the storage dtype at the store.  One thread per (tile or
// kernel, channel), channels fastest, so a wave's loads and stores sweep 64
// consecutive channels.  Loops run to the largest tile (16) and stop at the
// layer's t and alpha' by uniform conditions, so the register arrays keep
// compile-time indices and one instance serves every plan.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "device_common.hpp"
#include "kernels.hpp"

namespace wg {

namespace {

constexpr int kBlock1d = 256;

// U[a][k][c] = sum_i G[a][i] g[k][i][c]
template <typename Elem>
__global__ __launch_bounds__(kBlock1d) void kernel_transform_1d(KernelTable tab, const Elem* __restrict__ w,
                                                                Elem* __restrict__ U, int64_t K, int64_t C,
                                                                int64_t Cp, int alpha) {
    using S = Storage<Elem>;
    const int64_t gid = static_cast<int64_t>(blockIdx.x) * kBlock1d + threadIdx.x;
    if (gid >= K * Cp) return;
    const int64_t c = gid % Cp, k = gid / Cp;
    float g[3];
#pragma unroll
    for (int i = 0; i < 3; ++i) g[i] = c < C ? S::to_f32(w[(k * 3 + i) * C + c]) : 0.0f;
#pragma unroll
    for (int a = 0; a < kMaxAlpha; ++a) {
        if (a >= alpha) break;
        float acc = 0.0f;
#pragma unroll
        for (int i = 0; i < 3; ++i) acc = __builtin_fmaf(tab.g[a * 3 + i], g[i], acc);
        U[(a * K + k) * Cp + c] = S::from_f32(acc);
    }
}

// V[a][t][c] = sum_u B^T[a][u] d[u], d the window of t values at tx*m - 1
template <typename Elem>
__global__ __launch_bounds__(kBlock1d) void input_transform_1d(InputTable tab, const Elem* __restrict__ x,
                                                               Elem* __restrict__ V, int64_t L, int64_t C, int64_t Cp,
                                                               int64_t tl, int64_t T, int m, int tt, int alpha) {
    using S = Storage<Elem>;
    const int64_t gid = static_cast<int64_t>(blockIdx.x) * kBlock1d + threadIdx.x;
    if (gid >= T * Cp) return;
    const int64_t c = gid % Cp, t = gid / Cp;
    const int64_t tx = t % tl, n = t / tl;
    const int64_t l0 = tx * m - 1;
    float d[kMaxTile];
#pragma unroll
    for (int u = 0; u < kMaxTile; ++u) {
        const int64_t l = l0 + u;
        d[u] = (u < tt && c < C && l >= 0 && l < L) ? S::to_f32(x[(n * L + l) * C + c]) : 0.0f;
    }
#pragma unroll
    for (int a = 0; a < kMaxAlpha; ++a) {
        if (a >= alpha) break;
        float acc = 0.0f;
#pragma unroll
        for (int u = 0; u < kMaxTile; ++u) {
            if (u >= tt) break;
            acc = __builtin_fmaf(tab.bt[a * tt + u], d[u], acc);
        }
        V[(a * T + t) * Cp + c] = S::from_f32(acc);
    }
}

// y[n][tx*m + o][k] = sum_a A^T[o][a] M[a][t][k], stored inside L only
template <typename Elem>
__global__ __launch_bounds__(kBlock1d) void output_transform_1d(OutputTable tab, const float* __restrict__ M,
                                                                Elem* __restrict__ y, int64_t L, int64_t K, int64_t Kp,
                                                                int64_t tl, int64_t T, int m, int alpha) {
    using S = Storage<Elem>;
    const int64_t gid = static_cast<int64_t>(blockIdx.x) * kBlock1d + threadIdx.x;
    if (gid >= T * K) return;
    const int64_t k = gid % K, t = gid / K;
    const int64_t tx = t % tl, n = t / tl;
    float mv[kMaxAlpha];
#pragma unroll
    for (int a = 0; a < kMaxAlpha; ++a) mv[a] = a < alpha ? M[(a * T + t) * Kp + k] : 0.0f;
#pragma unroll
    for (int o = 0; o < kMaxTile; ++o) {
        const int64_t l = tx * m + o;
        if (o >= m || l >= L) break;
        float acc = 0.0f;
#pragma unroll
        for (int a = 0; a < kMaxAlpha; ++a) {
            if (a >= alpha) break;
            acc = __builtin_fmaf(tab.at[o * alpha + a], mv[a], acc);
        }
        y[(n * L + l) * K + k] = S::from_f32(acc);
    }
}

inline unsigned blocks_1d(int64_t n) { return static_cast<unsigned>((n + kBlock1d - 1) / kBlock1d); }
inline bool grid_ok(int64_t n) { return (n + kBlock1d - 1) / kBlock1d <= 0x7fffffff; }

}  // namespace

template <int D>
hipError_t launch_kernel_transform_1d_t(const Geometry& g, const KernelTable& tab, const void* w, void* U,
                                        hipStream_t stream) {
    using Elem = typename DTypeOf<D>::type;
    if (g.alpha > kMaxAlpha || !grid_ok(g.K * g.Cp)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(kernel_transform_1d<Elem>, dim3(blocks_1d(g.K * g.Cp)), dim3(kBlock1d), 0, stream, tab,
                       static_cast<const Elem*>(w), static_cast<Elem*>(U), g.K, g.C, g.Cp, g.alpha);
    return hipGetLastError();
}

template <int D>
hipError_t launch_input_transform_1d_t(const Geometry& g, const InputTable& tab, const void* x, void* V,
                                       hipStream_t stream) {
    using Elem = typename DTypeOf<D>::type;
    if (g.alpha > kMaxAlpha || g.t > kMaxTile || !grid_ok(g.T * g.Cp)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(input_transform_1d<Elem>, dim3(blocks_1d(g.T * g.Cp)), dim3(kBlock1d), 0, stream, tab,
                       static_cast<const Elem*>(x), static_cast<Elem*>(V), g.W, g.C, g.Cp, g.tw, g.T, g.m, g.t,
                       g.alpha);
    return hipGetLastError();
}

template <int D>
hipError_t launch_output_transform_1d_t(const Geometry& g, const OutputTable& tab, const float* M, void* y,
                                        hipStream_t stream) {
    using Elem = typename DTypeOf<D>::type;
    if (g.alpha > kMaxAlpha || g.m > kMaxTile || !grid_ok(g.T * g.K)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(output_transform_1d<Elem>, dim3(blocks_1d(g.T * g.K)), dim3(kBlock1d), 0, stream, tab, M,
                       static_cast<Elem*>(y), g.W, g.K, g.Kp, g.tw, g.T, g.m, g.alpha);
    return hipGetLastError();
}

#define WG_1D_INSTANCES(D)                                                                                       \
    template hipError_t launch_kernel_transform_1d_t<D>(const Geometry&, const KernelTable&, const void*, void*, \
                                                        hipStream_t);                                            \
    template hipError_t launch_input_transform_1d_t<D>(const Geometry&, const InputTable&, const void*, void*,   \
                                                       hipStream_t);                                             \
    template hipError_t launch_output_transform_1d_t<D>(const Geometry&, const OutputTable&, const float*,       \
                                                        void*, hipStream_t);
WG_1D_INSTANCES(0)
WG_1D_INSTANCES(1)
WG_1D_INSTANCES(2)
#undef WG_1D_INSTANCES

}  // namespace wg
