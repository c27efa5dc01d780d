// Internal interface between the C ABI (api.hip) and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace wg {

constexpr int kMaxAlpha = 16;  // largest Winograd-domain size alpha'
constexpr int kMaxTile = 16;   // largest input tile m + 2

enum DType : int { kF32 = 0, kF16 = 1, kBF16 = 2 };

inline int dtype_bytes(int dt) { return dt == kF32 ? 4 : 2; }

// fp32 transform tables, passed by value in the kernel-argument segment.
struct InputTable { float bt[kMaxAlpha * kMaxTile]; };    // B^T, alpha x t, row-major
struct KernelTable { float g[kMaxAlpha * 3]; };           // G, alpha x 3
struct OutputTable { float at[kMaxTile * kMaxAlpha]; };   // A^T, m x alpha

// Geometry of one layer: T tiles of m x m outputs, (m+2) x (m+2) inputs.
struct Geometry {
    int64_t N, H, W, C, K;
    int m, t, alpha;
    int64_t th, tw, T;  // tiles along H, along W, total
    int64_t Cp, Kp;     // channel strides of U / V and of M
    int64_t planes;     // Winograd-domain points: alpha'^2 (2D) or alpha' (1D)
};

inline int64_t round_up(int64_t v, int64_t q) { return (v + q - 1) / q * q; }

inline Geometry make_geometry(int64_t N, int64_t H, int64_t W, int64_t C, int64_t K, int m, int alpha) {
    Geometry g;
    g.N = N; g.H = H; g.W = W; g.C = C; g.K = K;
    g.m = m; g.t = m + 2; g.alpha = alpha;
    g.th = (H + m - 1) / m;
    g.tw = (W + m - 1) / m;
    g.T = N * g.th * g.tw;
    g.Cp = round_up(C, 8);
    g.Kp = round_up(K, 8);
    g.planes = static_cast<int64_t>(alpha) * alpha;
    return g;
}

// A 1D layer (rows of length W = L, H = 1, a 1 x 3 kernel): tiles of m
// outputs along W only, alpha' domain points.
inline Geometry make_geometry_1d(int64_t N, int64_t L, int64_t C, int64_t K, int m, int alpha) {
    Geometry g = make_geometry(N, 1, L, C, K, m, alpha);
    g.th = 1;
    g.T = N * g.tw;
    g.planes = alpha;
    return g;
}

// (input tile m + 2, alpha') shapes with compiled 2D input/output transforms:
// even m from 2 to 12 and alpha' = m + 2 + q, where q = 0..3 counts the extra
// multiplications per dimension that degree-2 moduli add (q = 0..4 for m = 6,
// the all-quadratic F(6x6) column of Table 1), capped at alpha' = 16.
#define WG_TRANSFORM_SHAPES(X)                                   \
    X(4, 4) X(4, 5) X(4, 6) X(4, 7)                              \
    X(6, 6) X(6, 7) X(6, 8) X(6, 9)                              \
    X(8, 8) X(8, 9) X(8, 10) X(8, 11) X(8, 12)                   \
    X(10, 10) X(10, 11) X(10, 12) X(10, 13)                      \
    X(12, 12) X(12, 13) X(12, 14) X(12, 15)                      \
    X(14, 14) X(14, 15) X(14, 16)

// Odd output tiles m = 3, 5, 7 (input tiles 5, 7, 9) with all-linear sets or
// one degree-2 modulus: the tile sizes of the random-data study of Section
// 3.1.  Separate path only (the fused kernel takes even tiles).
#define WG_TRANSFORM_SHAPES_ODD(X) X(5, 5) X(5, 6) X(7, 7) X(7, 8) X(9, 9) X(9, 10)

inline bool transform_shape_supported(int t, int alpha) {
#define WG_SHAPE_TEST(TT, A) if (t == TT && alpha == A) return true;
    WG_TRANSFORM_SHAPES(WG_SHAPE_TEST)
    WG_TRANSFORM_SHAPES_ODD(WG_SHAPE_TEST)
#undef WG_SHAPE_TEST
    return false;
}

// Launchers, one instance per storage dtype D (0 fp32, 1 fp16, 2 bf16).  Each
// returns hipSuccess or the launch error and never synchronises.
template <int D>
hipError_t launch_kernel_transform_t(const Geometry& g, const KernelTable& tab, const void* w, void* U,
                                     hipStream_t stream);
// builtin: the id of a built-in plan whose tables the plan has (its
// constant-coefficient kernels are used), or -1.
template <int D>
hipError_t launch_input_transform_t(const Geometry& g, const InputTable& tab, const void* x, void* V, int builtin,
                                    hipStream_t stream);
// Both transforms in one launch (they are independent): U from w and V from x.
template <int D>
hipError_t launch_kernel_input_transform_t(const Geometry& g, const KernelTable& ktab, const InputTable& itab,
                                           const void* w, const void* x, void* U, void* V, int builtin,
                                           hipStream_t stream);
template <int D>
hipError_t launch_output_transform_t(const Geometry& g, const OutputTable& tab, const float* M, void* y,
                                     int builtin, hipStream_t stream);
template <int D>
hipError_t launch_contract_t(const Geometry& g, const void* V, const void* U, float* M, hipStream_t stream);

// The same contraction with the channels summed pairwise (contract_pairwise.hip):
// leaves of 64 bytes of each channel row, added in a binary tree.
template <int D>
hipError_t launch_contract_pairwise_t(const Geometry& g, const void* V, const void* U, float* M, hipStream_t stream);

// Contraction fused with the output transform: V, U -> y with no M in memory.
// Supported for input tiles up to 8 (m <= 6) and planes addressable with
// 32-bit offsets; the launcher returns hipErrorInvalidValue otherwise.
template <int D> bool contract_output_supported_t(const Geometry& g);
template <int D>
hipError_t launch_contract_output_t(const Geometry& g, const OutputTable& tab, const void* V, const void* U,
                                    void* y, int builtin, hipStream_t stream);
// The same kernel with the input transform in its prologue: x, U -> y, no V
// in memory.  Supported for channel rows of at most 32 bytes and K > 32.
template <int D> bool input_contract_output_supported_t(const Geometry& g);
template <int D>
hipError_t launch_input_contract_output_t(const Geometry& g, const InputTable& itab, const OutputTable& otab,
                                          const void* x, const void* U, void* y, hipStream_t stream);

// Around the layer (layer_ops.hip): ReLU, optionally followed by 2x2 stride-2
// max-pooling (NHWC, storage dtype D); a float64 direct convolution with a
// kernel of kh x 3 taps (kh = 3: pad 1 in both directions; kh = 1: a 1D
// convolution along W, pad 1); the float64 sums of (y - ref)^2 and ref^2
// over n values into sums[0], sums[1] (sums[2 ..] holds the kSqSumPartials
// per-block partial pairs).
constexpr int kSqSumDoubles = 2 + 2 * 256;
template <int D>
hipError_t launch_relu_pool_t(const void* x, void* y, int64_t N, int64_t H, int64_t W, int64_t C, bool pool,
                              hipStream_t stream);
template <int D>
hipError_t launch_direct_f64_t(const void* x, const void* w, double* y, int64_t N, int64_t H, int64_t W, int64_t C,
                               int64_t K, int kh, hipStream_t stream);
template <int D>
hipError_t launch_sq_sums_t(const void* y, const double* ref, int64_t n, double* sums, hipStream_t stream);

// 1D F(m, 3) (conv1d.hip): kernel transform U [alpha'][K][Cp] from w
// [K][1][3][C], input transform V [alpha'][T][Cp] from x [N][1][L][C], output
// transform y [N][1][L][K] from M [alpha'][T][Kp] (the contraction is
// launch_contract_t with g.planes = alpha').
template <int D>
hipError_t launch_kernel_transform_1d_t(const Geometry& g, const KernelTable& tab, const void* w, void* U,
                                        hipStream_t stream);
template <int D>
hipError_t launch_input_transform_1d_t(const Geometry& g, const InputTable& tab, const void* x, void* V,
                                       hipStream_t stream);
template <int D>
hipError_t launch_output_transform_1d_t(const Geometry& g, const OutputTable& tab, const float* M, void* y,
                                        hipStream_t stream);

// Compute units of the current device (cached per device).
int device_cu_count();

}  // namespace wg
