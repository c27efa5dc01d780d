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
    return g;
}

// (input tile m + 2, alpha') shapes with compiled input/output transforms:
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

inline bool transform_shape_supported(int t, int alpha) {
#define WG_SHAPE_TEST(TT, A) if (t == TT && alpha == A) return true;
    WG_TRANSFORM_SHAPES(WG_SHAPE_TEST)
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

// Contraction fused with the output transform: V, U -> y with no M in memory.
// Supported for input tiles up to 8 (m <= 6) and planes addressable with
// 32-bit offsets; the launcher returns hipErrorInvalidValue otherwise.
template <int D> bool contract_output_supported_t(const Geometry& g);
template <int D>
hipError_t launch_contract_output_t(const Geometry& g, const OutputTable& tab, const void* V, const void* U,
                                    void* y, hipStream_t stream);
// The same kernel with the input transform in its prologue: x, U -> y, no V
// in memory.  Supported for channel rows of at most 32 bytes and K > 32.
template <int D> bool input_contract_output_supported_t(const Geometry& g);
template <int D>
hipError_t launch_input_contract_output_t(const Geometry& g, const InputTable& itab, const OutputTable& otab,
                                          const void* x, const void* U, void* y, hipStream_t stream);

// Compute units of the current device (cached per device).
int device_cu_count();

}  // namespace wg
