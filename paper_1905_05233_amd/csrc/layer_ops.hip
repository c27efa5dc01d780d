// Operations around the Winograd layer on gfx950:
//   * ReLU and 2x2 stride-2 max-pooling between the convolutions of a CNN
//     (the VGG-16 stack of the experiments of Section 3.2 of Barabasz &
//     Gregg, arXiv 1905.05233);
//   * a float64 direct convolution, the reference against which Section 3.1
//     measures the error of a Winograd convolution computed in lower
//     precision;
//   * the two sums of squares that the relative L2 error of a result against
//     such a reference needs, reduced in float64 in a fixed order.
// None of these is on the Winograd path itself; they keep the stack and the
// error studies on the device.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "device_common.hpp"
#include "kernels.hpp"

namespace wg {

namespace {

constexpr int kOpBlock = 256;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// 16 bytes as non-temporal (streaming) accesses: the input is read once and
// the output is read once, by the next layer's transforms; kept out of the
// caches, they leave the last-level cache to the next layer's V and U (a
// VGG-16 pass at N = 32: 1.78 against 1.82 ms of convolution time for the
// stores, 1.73 against 1.74 ms for the loads)
__device__ __forceinline__ void store16_nt(void* dst, const void* src) {
    __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(src), reinterpret_cast<u32x4*>(dst));
}
__device__ __forceinline__ u32x4 load16_nt(const void* src) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src));
}

template <typename Elem>
__device__ __forceinline__ float relu(Elem v) {
    const float f = Storage<Elem>::to_f32(v);
    return f > 0.0f ? f : 0.0f;   // NaN and -0 give +0
}

// y = ReLU(x), elementwise over n values; vec values per thread (a 16-byte
// run when the whole tensor is made of such runs, else one value).
template <typename Elem, int VEC>
__global__ __launch_bounds__(kOpBlock) void relu_kernel(const Elem* __restrict__ x, Elem* __restrict__ y,
                                                        int64_t n) {
    using S = Storage<Elem>;
    const int64_t i = (static_cast<int64_t>(blockIdx.x) * kOpBlock + threadIdx.x) * VEC;
    if (i >= n) return;
    Elem e[VEC];
    if constexpr (VEC * sizeof(Elem) == 16) {
        *reinterpret_cast<u32x4*>(e) = load16_nt(x + i);
    } else {
#pragma unroll
        for (int q = 0; q < VEC; ++q) e[q] = x[i + q];
    }
#pragma unroll
    for (int q = 0; q < VEC; ++q) e[q] = S::from_f32(relu(e[q]));
    if constexpr (VEC * sizeof(Elem) == 16) {
        store16_nt(y + i, e);
    } else {
#pragma unroll
        for (int q = 0; q < VEC; ++q) y[i + q] = e[q];
    }
}

// y[n][i][j][c] = max over the 2x2 window at (2i, 2j) of ReLU(x); one thread
// per (output pixel, run of VEC channels), channels fastest (coalesced).
template <typename Elem, int VEC>
__global__ __launch_bounds__(kOpBlock) void relu_pool_kernel(const Elem* __restrict__ x, Elem* __restrict__ y,
                                                             int64_t N, int64_t H, int64_t W, int64_t C) {
    using S = Storage<Elem>;
    const int64_t Ho = H / 2, Wo = W / 2, runs = C / VEC;
    const int64_t gid = static_cast<int64_t>(blockIdx.x) * kOpBlock + threadIdx.x;
    if (gid >= N * Ho * Wo * runs) return;
    const int64_t c = (gid % runs) * VEC;
    const int64_t pix = gid / runs;
    const int64_t j = pix % Wo, i = (pix / Wo) % Ho, n = pix / (Wo * Ho);
    float best[VEC];
#pragma unroll
    for (int q = 0; q < VEC; ++q) best[q] = 0.0f;
#pragma unroll
    for (int di = 0; di < 2; ++di)
#pragma unroll
        for (int dj = 0; dj < 2; ++dj) {
            const Elem* src = x + ((n * H + 2 * i + di) * W + 2 * j + dj) * C + c;
            Elem e[VEC];
            if constexpr (VEC * sizeof(Elem) == 16) {
                *reinterpret_cast<u32x4*>(e) = load16_nt(src);
            } else {
#pragma unroll
                for (int q = 0; q < VEC; ++q) e[q] = src[q];
            }
#pragma unroll
            for (int q = 0; q < VEC; ++q) best[q] = fmaxf(best[q], relu(e[q]));
        }
    Elem o[VEC];
#pragma unroll
    for (int q = 0; q < VEC; ++q) o[q] = S::from_f32(best[q]);
    Elem* dst = y + pix * C + c;
    if constexpr (VEC * sizeof(Elem) == 16) {
        store16_nt(dst, o);
    } else {
#pragma unroll
        for (int q = 0; q < VEC; ++q) dst[q] = o[q];
    }
}

// yd[n][h][v][k] = sum_{i<KH, j<3, c} w[k][i][j][c] x[n][h + i - KH/2][v + j - 1][c]
// in float64 (zero outside the image).  One thread per output, output
// channels fastest: the 64 lanes of a wave share their input pixel.
template <typename Elem, int KH>
__global__ __launch_bounds__(kOpBlock) void direct_f64_kernel(const Elem* __restrict__ x, const Elem* __restrict__ w,
                                                              double* __restrict__ yd, int64_t N, int64_t H, int64_t W,
                                                              int64_t C, int64_t K) {
    using S = Storage<Elem>;
    const int64_t gid = static_cast<int64_t>(blockIdx.x) * kOpBlock + threadIdx.x;
    if (gid >= N * H * W * K) return;
    const int64_t k = gid % K;
    const int64_t pix = gid / K;
    const int64_t v = pix % W, h = (pix / W) % H, n = pix / (W * H);
    double acc = 0.0;
    for (int i = 0; i < KH; ++i) {
        const int64_t hh = h + i - KH / 2;
        if (hh < 0 || hh >= H) continue;
        for (int j = 0; j < 3; ++j) {
            const int64_t vv = v + j - 1;
            if (vv < 0 || vv >= W) continue;
            const Elem* xs = x + ((n * H + hh) * W + vv) * C;
            const Elem* ws = w + ((k * KH + i) * 3 + j) * C;
            for (int64_t c = 0; c < C; ++c)
                acc = fma(static_cast<double>(S::to_f32(ws[c])), static_cast<double>(S::to_f32(xs[c])), acc);
        }
    }
    yd[gid] = acc;
}

// Sums of (y - ref)^2 and ref^2 over n values in float64: each of the
// kSumBlocks blocks strides over the values and reduces its part in LDS in a
// fixed order into sums[2 + 2 b], sums[3 + 2 b]; one block then adds the
// partials in block order into sums[0], sums[1].  Deterministic.
constexpr int kSumBlocks = 256;

template <typename Elem>
__global__ __launch_bounds__(kOpBlock) void sq_sums_partial(const Elem* __restrict__ y, const double* __restrict__ ref,
                                                            int64_t n, double* __restrict__ sums) {
    using S = Storage<Elem>;
    __shared__ double se[kOpBlock], sr[kOpBlock];
    double e2 = 0.0, r2 = 0.0;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kOpBlock + threadIdx.x; i < n;
         i += static_cast<int64_t>(kSumBlocks) * kOpBlock) {
        const double r = ref[i];
        const double d = static_cast<double>(S::to_f32(y[i])) - r;
        e2 = fma(d, d, e2);
        r2 = fma(r, r, r2);
    }
    se[threadIdx.x] = e2;
    sr[threadIdx.x] = r2;
    __syncthreads();
    for (int s = kOpBlock / 2; s > 0; s >>= 1) {
        if (static_cast<int>(threadIdx.x) < s) {
            se[threadIdx.x] += se[threadIdx.x + s];
            sr[threadIdx.x] += sr[threadIdx.x + s];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        sums[2 + 2 * blockIdx.x] = se[0];
        sums[3 + 2 * blockIdx.x] = sr[0];
    }
}

__global__ __launch_bounds__(64) void sq_sums_final(double* __restrict__ sums) {
    if (threadIdx.x != 0) return;
    double e2 = 0.0, r2 = 0.0;
    for (int b = 0; b < kSumBlocks; ++b) {
        e2 += sums[2 + 2 * b];
        r2 += sums[3 + 2 * b];
    }
    sums[0] = e2;
    sums[1] = r2;
}

inline unsigned op_blocks(int64_t n) { return static_cast<unsigned>((n + kOpBlock - 1) / kOpBlock); }

}  // namespace

template <int D>
hipError_t launch_relu_pool_t(const void* x, void* y, int64_t N, int64_t H, int64_t W, int64_t C, bool pool,
                              hipStream_t stream) {
    using Elem = typename DTypeOf<D>::type;
    constexpr int kVec = 16 / static_cast<int>(sizeof(Elem));
    const auto* xp = static_cast<const Elem*>(x);
    auto* yp = static_cast<Elem*>(y);
    const bool vec = C % kVec == 0;
    if (!pool) {
        const int64_t n = N * H * W * C;
        const int64_t threads = vec ? n / kVec : n;
        if ((threads + kOpBlock - 1) / kOpBlock > 0x7fffffff) return hipErrorInvalidValue;
        if (vec)
            hipLaunchKernelGGL((relu_kernel<Elem, kVec>), dim3(op_blocks(threads)), dim3(kOpBlock), 0, stream, xp, yp, n);
        else
            hipLaunchKernelGGL((relu_kernel<Elem, 1>), dim3(op_blocks(threads)), dim3(kOpBlock), 0, stream, xp, yp, n);
        return hipGetLastError();
    }
    const int64_t threads = N * (H / 2) * (W / 2) * (vec ? C / kVec : C);
    if (threads == 0) return hipSuccess;
    if ((threads + kOpBlock - 1) / kOpBlock > 0x7fffffff) return hipErrorInvalidValue;
    if (vec)
        hipLaunchKernelGGL((relu_pool_kernel<Elem, kVec>), dim3(op_blocks(threads)), dim3(kOpBlock), 0, stream, xp, yp,
                           N, H, W, C);
    else
        hipLaunchKernelGGL((relu_pool_kernel<Elem, 1>), dim3(op_blocks(threads)), dim3(kOpBlock), 0, stream, xp, yp, N,
                           H, W, C);
    return hipGetLastError();
}

template <int D>
hipError_t launch_direct_f64_t(const void* x, const void* w, double* y, int64_t N, int64_t H, int64_t W, int64_t C,
                               int64_t K, int kh, hipStream_t stream) {
    using Elem = typename DTypeOf<D>::type;
    const int64_t n = N * H * W * K;
    if ((n + kOpBlock - 1) / kOpBlock > 0x7fffffff) return hipErrorInvalidValue;
    const auto* xp = static_cast<const Elem*>(x);
    const auto* wp = static_cast<const Elem*>(w);
    if (kh == 3)
        hipLaunchKernelGGL((direct_f64_kernel<Elem, 3>), dim3(op_blocks(n)), dim3(kOpBlock), 0, stream, xp, wp, y, N, H,
                           W, C, K);
    else
        hipLaunchKernelGGL((direct_f64_kernel<Elem, 1>), dim3(op_blocks(n)), dim3(kOpBlock), 0, stream, xp, wp, y, N, H,
                           W, C, K);
    return hipGetLastError();
}

template <int D>
hipError_t launch_sq_sums_t(const void* y, const double* ref, int64_t n, double* sums, hipStream_t stream) {
    using Elem = typename DTypeOf<D>::type;
    hipLaunchKernelGGL((sq_sums_partial<Elem>), dim3(kSumBlocks), dim3(kOpBlock), 0, stream,
                       static_cast<const Elem*>(y), ref, n, sums);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sq_sums_final, dim3(1), dim3(64), 0, stream, sums);
    return hipGetLastError();
}

template hipError_t launch_relu_pool_t<0>(const void*, void*, int64_t, int64_t, int64_t, int64_t, bool, hipStream_t);
template hipError_t launch_relu_pool_t<1>(const void*, void*, int64_t, int64_t, int64_t, int64_t, bool, hipStream_t);
template hipError_t launch_relu_pool_t<2>(const void*, void*, int64_t, int64_t, int64_t, int64_t, bool, hipStream_t);
template hipError_t launch_direct_f64_t<0>(const void*, const void*, double*, int64_t, int64_t, int64_t, int64_t,
                                           int64_t, int, hipStream_t);
template hipError_t launch_direct_f64_t<1>(const void*, const void*, double*, int64_t, int64_t, int64_t, int64_t,
                                           int64_t, int, hipStream_t);
template hipError_t launch_direct_f64_t<2>(const void*, const void*, double*, int64_t, int64_t, int64_t, int64_t,
                                           int64_t, int, hipStream_t);
template hipError_t launch_sq_sums_t<0>(const void*, const double*, int64_t, double*, hipStream_t);
template hipError_t launch_sq_sums_t<1>(const void*, const double*, int64_t, double*, hipStream_t);
template hipError_t launch_sq_sums_t<2>(const void*, const double*, int64_t, double*, hipStream_t);

}  // namespace wg
