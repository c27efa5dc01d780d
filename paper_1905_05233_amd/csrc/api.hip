// C ABI of the Winograd convolution library (declared in winograd_crt.h).
//
// Host side: plan creation (exact transforms from plan.cpp), argument and
// workspace validation, and the four kernel launches of eq. (2)
// (Barabasz & Gregg, arXiv 1905.05233).  No C++ exception leaves this file;
// every failure becomes a wg_status plus a thread-local message.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "builtin_plans.hpp"

#include "kernels.hpp"
#include "plan.hpp"
#include "winograd_crt.h"

// Workspace of winograd_conv2d_static (U, V and M of one layer), one copy per
// GPU, held until the process ends.  Host code never passes `scratch` itself
// to a kernel (in host code the name is only a stand-in); it uses the device
// address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[WG_STATIC_SCRATCH_BYTES];

struct wg_plan_s {
    wg::Transforms tr;
    int dtype = 0;
    int path = WG_PATH_AUTO;
    int builtin = -1;   // id of the built-in plan with the same fp32 tables, or -1
    int channel_sum = WG_SUM_MFMA;
    void* ws = nullptr;
    size_t ws_bytes = 0;
    wg::InputTable itab{};
    wg::KernelTable ktab{};
    wg::OutputTable otab{};
};

namespace {

thread_local std::string g_last_error;

wg_status fail(wg_status s, const std::string& msg) {
    g_last_error = msg;
    return s;
}

wg_status from_hip(hipError_t e, const char* what) {
    if (e == hipSuccess) return WG_OK;
    return fail(WG_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

template <typename F>
wg_status guarded(F&& f) {
    try {
        return f();
    } catch (const wg::PlanError& e) {
        return fail(static_cast<wg_status>(e.status), e.what());
    } catch (const wg::OverflowError& e) {
        return fail(WG_ERR_OVERFLOW, e.what());
    } catch (const std::bad_alloc&) {
        return fail(WG_ERR_INTERNAL, "host out of memory");
    } catch (const std::exception& e) {
        return fail(WG_ERR_INTERNAL, e.what());
    } catch (...) {
        return fail(WG_ERR_INTERNAL, "unknown error");
    }
}

// The built-in plan whose fp32 tables (and shape) equal the plan's, or -1.
template <class P>
bool same_tables(const wg_plan_s* p) {
    const int al = p->tr.alpha, t = p->tr.tile_in, m = p->tr.m;
    if (m != P::kM || t != P::kT || al != P::kAlpha) return false;
    for (int i = 0; i < al * t; ++i)
        if (std::memcmp(&p->itab.bt[i], &P::bt[i], sizeof(float)) != 0) return false;
    for (int i = 0; i < al * 3; ++i)
        if (std::memcmp(&p->ktab.g[i], &P::g[i], sizeof(float)) != 0) return false;
    for (int i = 0; i < m * al; ++i)
        if (std::memcmp(&p->otab.at[i], &P::at[i], sizeof(float)) != 0) return false;
    return true;
}

int identify_builtin(const wg_plan_s* p) {
#define WG_SAME(ID, TT, A) \
    if (same_tables<wg::BuiltinPlan##ID>(p)) return ID;
    WG_BUILTIN_PLANS(WG_SAME)
#undef WG_SAME
    return -1;
}

wg_status finish_plan(wg::Transforms&& tr, wg_dtype dtype, wg_plan* out) {
    if (tr.alpha > wg::kMaxAlpha || tr.tile_in > wg::kMaxTile)
        return fail(WG_ERR_UNSUPPORTED, "alpha' and the input tile must be at most 16");
    auto* p = new wg_plan_s();
    p->tr = std::move(tr);
    p->dtype = static_cast<int>(dtype);
    const int al = p->tr.alpha, t = p->tr.tile_in, m = p->tr.m;
    // B^T (alpha x t), G (alpha x 3), A^T (m x alpha), densely packed
    for (int a = 0; a < al; ++a)
        for (int u = 0; u < t; ++u) p->itab.bt[a * t + u] = p->tr.Bf[static_cast<size_t>(u * al + a)];
    for (int a = 0; a < al; ++a)
        for (int i = 0; i < 3; ++i) p->ktab.g[a * 3 + i] = p->tr.Gf[static_cast<size_t>(a * 3 + i)];
    for (int o = 0; o < m; ++o)
        for (int a = 0; a < al; ++a) p->otab.at[o * al + a] = p->tr.Af[static_cast<size_t>(a * m + o)];
    p->builtin = identify_builtin(p);
    *out = p;
    return WG_OK;
}

wg_status check_create_args(int m, int r, wg_dtype dtype, wg_plan* out) {
    if (!out) return fail(WG_ERR_ARG, "null output pointer");
    if (r != 3) return fail(WG_ERR_UNSUPPORTED, "only 3x3 kernels (r = 3) are supported");
    if (m < 1 || m + r - 1 > wg::kMaxTile) return fail(WG_ERR_UNSUPPORTED, "output tile m out of range");
    if (dtype != WG_F32 && dtype != WG_F16 && dtype != WG_BF16) return fail(WG_ERR_UNSUPPORTED, "unknown dtype");
    return WG_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool fused_supported(int dt, const wg::Geometry& g) {
    switch (dt) {
        case 0: return wg::contract_output_supported_t<0>(g);
        case 1: return wg::contract_output_supported_t<1>(g);
        default: return wg::contract_output_supported_t<2>(g);
    }
}
bool input_fused_supported(int dt, const wg::Geometry& g) {
    switch (dt) {
        case 0: return wg::input_contract_output_supported_t<0>(g);
        case 1: return wg::input_contract_output_supported_t<1>(g);
        default: return wg::input_contract_output_supported_t<2>(g);
    }
}

// The path winograd_conv2d takes; -1 if the plan asks for the fused path and
// the shape does not allow it.
//
// The automatic choice follows where each path spends its time.  The separate
// path moves 8 bytes of M per (tile, output channel, domain point) through
// HBM; the fused kernel instead streams one 128-byte slice of every channel
// row per domain point through LDS for each block of 2048 (tile, channel)
// pairs, and each such step costs about as much as 8 bytes of M per pair when
// rows are longer than two slices (measured on VGG-16 layer shapes).  It also
// needs enough pair blocks to occupy every CU twice.  Hence: fused when a
// channel row fits two slices (C <= 64 fp32, C <= 128 fp16/bf16) and there
// are at least 2^20 pairs.  The rule uses no device query, so the workspace
// size it implies is the same on every machine.
//
// WG_PATH_FUSED_INPUT is taken only when asked for: on the RGB layer of the
// VGG-16 stack it measured slower than the input-transform kernel followed by
// the fused kernel (its prologue runs the transform with run-time
// coefficients, serialised ahead of each block's contraction).
int resolve_path(const wg_plan_s* p, const wg::Geometry& g) {
    if (p->channel_sum == WG_SUM_PAIRWISE) return WG_PATH_SEPARATE;   // the fused kernels chain on MFMA
    const bool ok = fused_supported(p->dtype, g);
    if (p->path == WG_PATH_FUSED_INPUT) return ok && input_fused_supported(p->dtype, g) ? WG_PATH_FUSED_INPUT : -1;
    if (p->path == WG_PATH_FUSED) return ok ? WG_PATH_FUSED : -1;
    if (p->path == WG_PATH_SEPARATE || !ok) return WG_PATH_SEPARATE;
    // fused for layers with many (tile, output channel) pairs and short rows;
    // with the fused kernel's unrolled instance (output tile at most 4 x 4, 64
    // or more output channels) rows of up to 512 bytes, from half as many pairs
    const int64_t row_bytes = g.Cp * wg::dtype_bytes(p->dtype);
    const int64_t pairs = g.T * g.K;
    const bool unrolled = g.m <= 4 && g.K >= 64;
    const bool fused = (row_bytes <= 256 && pairs >= (int64_t(1) << 20)) ||
                       (unrolled && row_bytes <= 512 && pairs >= (int64_t(1) << 19));
    return fused ? WG_PATH_FUSED : WG_PATH_SEPARATE;
}

struct Layout {
    wg::Geometry g;
    int path;
    int64_t n_chunks;   // launch pairs of the fused path: chunks of the batch, sizes differing by at most one
    int64_t chunk;      // images of the largest chunk
    size_t u_off, v_off, m_off, total;
};

// On the fused path a large batch goes through in chunks of whole images
// whose V is at most this size, one V buffer reused by every chunk: the input
// transform writes a chunk's V and the fused kernel reads it back while it is
// still in the GPU's 256 MB last-level cache, instead of from HBM.
constexpr int64_t kChunkVBytes = int64_t(160) << 20;

size_t align256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

Layout layout_for(const wg_plan_s* p, int64_t N, int64_t H, int64_t W, int64_t C, int64_t K) {
    Layout L;
    L.g = wg::make_geometry(N, H, W, C, K, p->tr.m, p->tr.alpha);
    L.path = resolve_path(p, L.g);
    const size_t es = static_cast<size_t>(wg::dtype_bytes(p->dtype));
    const size_t a2 = static_cast<size_t>(p->tr.alpha) * static_cast<size_t>(p->tr.alpha);
    L.n_chunks = 1;
    L.chunk = N;
    if (L.path == WG_PATH_FUSED) {
        // the fewest chunks within the budget, their sizes balanced
        const int64_t v_img = static_cast<int64_t>(a2) * L.g.th * L.g.tw * L.g.Cp * static_cast<int64_t>(es);
        if (v_img * N > kChunkVBytes) {
            const int64_t per = std::max<int64_t>(1, kChunkVBytes / v_img);
            L.n_chunks = (N + per - 1) / per;
            L.chunk = (N + L.n_chunks - 1) / L.n_chunks;
        }
    }
    const size_t ub = a2 * static_cast<size_t>(K) * static_cast<size_t>(L.g.Cp) * es;
    const size_t vb = a2 * static_cast<size_t>(L.chunk * L.g.th * L.g.tw) * static_cast<size_t>(L.g.Cp) * es;
    const size_t mb = a2 * static_cast<size_t>(L.g.T) * static_cast<size_t>(L.g.Kp) * sizeof(float);
    // no M on the fused paths, no V either when the input transform is fused
    L.u_off = 0;
    L.v_off = align256(ub);
    L.m_off = L.v_off + (L.path == WG_PATH_FUSED_INPUT ? 0 : align256(vb));
    L.total = L.m_off + (L.path == WG_PATH_SEPARATE ? align256(mb) : 0);
    return L;
}

// Device address of `scratch` on the current device, looked up on the first
// call made with that device current and kept per device.
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

wg_status static_scratch(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return from_hip(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxScratchDevices) return fail(WG_ERR_UNSUPPORTED, "device index beyond 63");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return from_hip(e, "hipGetSymbolAddress(scratch)");
        if (!p) return fail(WG_ERR_HIP, "hipGetSymbolAddress(scratch) returned a null address");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return WG_OK;
}

bool dims_ok(int64_t N, int64_t H, int64_t W, int64_t C, int64_t K) {
    const int64_t lim = int64_t(1) << 31;
    return N >= 1 && H >= 1 && W >= 1 && C >= 1 && K >= 1 && N < lim && H < lim && W < lim && C < lim && K < lim;
}

wg_status check_plan(wg_plan plan) {
    if (!plan) return fail(WG_ERR_ARG, "null plan");
    if (!wg::transform_shape_supported(plan->tr.tile_in, plan->tr.alpha))
        return fail(WG_ERR_UNSUPPORTED, "no compiled transform kernel for input tile " +
                                            std::to_string(plan->tr.tile_in) + " and alpha' " +
                                            std::to_string(plan->tr.alpha));
    return WG_OK;
}

wg_status check_tensor(const wg_tensor* t, const char* name) {
    if (!t || !t->data) return fail(WG_ERR_ARG, std::string("null tensor ") + name);
    if (!aligned16(t->data)) return fail(WG_ERR_ARG, std::string("tensor ") + name + " is not 16-byte aligned");
    return WG_OK;
}

hipError_t launch_kt(int dt, const wg::Geometry& g, const wg::KernelTable& t, const void* w, void* U,
                     hipStream_t s) {
    switch (dt) {
        case 0: return wg::launch_kernel_transform_t<0>(g, t, w, U, s);
        case 1: return wg::launch_kernel_transform_t<1>(g, t, w, U, s);
        default: return wg::launch_kernel_transform_t<2>(g, t, w, U, s);
    }
}
hipError_t launch_kit(int dt, const wg::Geometry& g, const wg::KernelTable& kt, const wg::InputTable& it,
                      const void* w, const void* x, void* U, void* V, int bi, hipStream_t s) {
    switch (dt) {
        case 0: return wg::launch_kernel_input_transform_t<0>(g, kt, it, w, x, U, V, bi, s);
        case 1: return wg::launch_kernel_input_transform_t<1>(g, kt, it, w, x, U, V, bi, s);
        default: return wg::launch_kernel_input_transform_t<2>(g, kt, it, w, x, U, V, bi, s);
    }
}
hipError_t launch_it(int dt, const wg::Geometry& g, const wg::InputTable& t, const void* x, void* V, int bi,
                     hipStream_t s) {
    switch (dt) {
        case 0: return wg::launch_input_transform_t<0>(g, t, x, V, bi, s);
        case 1: return wg::launch_input_transform_t<1>(g, t, x, V, bi, s);
        default: return wg::launch_input_transform_t<2>(g, t, x, V, bi, s);
    }
}
hipError_t launch_ct(int dt, const wg::Geometry& g, const void* V, const void* U, float* M, hipStream_t s,
                     int channel_sum = WG_SUM_MFMA) {
    if (channel_sum == WG_SUM_PAIRWISE) {
        switch (dt) {
            case 0: return wg::launch_contract_pairwise_t<0>(g, V, U, M, s);
            case 1: return wg::launch_contract_pairwise_t<1>(g, V, U, M, s);
            default: return wg::launch_contract_pairwise_t<2>(g, V, U, M, s);
        }
    }
    switch (dt) {
        case 0: return wg::launch_contract_t<0>(g, V, U, M, s);
        case 1: return wg::launch_contract_t<1>(g, V, U, M, s);
        default: return wg::launch_contract_t<2>(g, V, U, M, s);
    }
}
hipError_t launch_ot(int dt, const wg::Geometry& g, const wg::OutputTable& t, const float* M, void* y, int bi,
                     hipStream_t s) {
    switch (dt) {
        case 0: return wg::launch_output_transform_t<0>(g, t, M, y, bi, s);
        case 1: return wg::launch_output_transform_t<1>(g, t, M, y, bi, s);
        default: return wg::launch_output_transform_t<2>(g, t, M, y, bi, s);
    }
}
hipError_t launch_co(int dt, const wg::Geometry& g, const wg::OutputTable& t, const void* V, const void* U,
                     void* y, int bi, hipStream_t s) {
    switch (dt) {
        case 0: return wg::launch_contract_output_t<0>(g, t, V, U, y, bi, s);
        case 1: return wg::launch_contract_output_t<1>(g, t, V, U, y, bi, s);
        default: return wg::launch_contract_output_t<2>(g, t, V, U, y, bi, s);
    }
}
hipError_t launch_ico(int dt, const wg::Geometry& g, const wg::InputTable& it, const wg::OutputTable& ot,
                      const void* x, const void* U, void* y, hipStream_t s) {
    switch (dt) {
        case 0: return wg::launch_input_contract_output_t<0>(g, it, ot, x, U, y, s);
        case 1: return wg::launch_input_contract_output_t<1>(g, it, ot, x, U, y, s);
        default: return wg::launch_input_contract_output_t<2>(g, it, ot, x, U, y, s);
    }
}

}  // namespace

extern "C" {

wg_status winograd_plan_create(const wg_poly_set* set, int m, int r, wg_dtype dtype, wg_plan* out) {
    return guarded([&]() -> wg_status {
        wg_status s = check_create_args(m, r, dtype, out);
        if (s != WG_OK) return s;
        if (!set || set->n_mod <= 0 || !set->mods) return fail(WG_ERR_ARG, "empty modulus set");
        std::vector<wg::Modulus> mods;
        for (int i = 0; i < set->n_mod; ++i) {
            const wg_modulus& md = set->mods[i];
            wg::Modulus x;
            if (md.degree == 0) {
                x.inf = true;
            } else {
                if (md.degree < 0 || md.degree > 3) return fail(WG_ERR_UNSUPPORTED, "modulus degree must be 1..3");
                std::vector<wg::Rat> c;
                for (int k = 0; k <= md.degree; ++k) {
                    if (md.coef[k].den == 0) return fail(WG_ERR_ARG, "zero denominator in a modulus");
                    c.emplace_back(md.coef[k].num, md.coef[k].den);
                }
                x.p = wg::Poly(c);
                if (x.p.deg() != md.degree) return fail(WG_ERR_ARG, "leading coefficient of a modulus is zero");
            }
            mods.push_back(x);
        }
        std::vector<wg::Rat> inner;
        bool inner_inf = true;
        if (set->n_inner > 0) {
            if (!set->inner_pts) return fail(WG_ERR_ARG, "null inner points");
            for (int i = 0; i < set->n_inner; ++i) {
                if (set->inner_pts[i].den == 0) return fail(WG_ERR_ARG, "zero denominator in an inner point");
                inner.emplace_back(set->inner_pts[i].num, set->inner_pts[i].den);
            }
            inner_inf = set->inner_inf != 0;
        } else {
            inner = {wg::Rat(0), wg::Rat(-1)};
        }
        return finish_plan(wg::build_transforms(mods, inner, inner_inf, m, r), dtype, out);
    });
}

wg_status winograd_plan_create_str(const char* moduli, const char* inner, int m, int r, wg_dtype dtype,
                                   wg_plan* out) {
    return guarded([&]() -> wg_status {
        wg_status s = check_create_args(m, r, dtype, out);
        if (s != WG_OK) return s;
        if (!moduli) return fail(WG_ERR_ARG, "null modulus string");
        const std::vector<wg::Modulus> mods = wg::parse_moduli(moduli);
        std::vector<wg::Rat> pts;
        bool inf = true;
        if (inner && inner[0] != '\0') wg::parse_points(inner, &pts, &inf);
        else pts = {wg::Rat(0), wg::Rat(-1)};
        return finish_plan(wg::build_transforms(mods, pts, inf, m, r), dtype, out);
    });
}

wg_status winograd_plan_create_ex(const char* moduli, const char* inner, int m, int r, wg_dtype dtype,
                                  const wg_plan_options* opts, wg_plan* out) {
    return guarded([&]() -> wg_status {
        wg_status s = check_create_args(m, r, dtype, out);
        if (s != WG_OK) return s;
        if (!moduli) return fail(WG_ERR_ARG, "null modulus string");
        const int factors = opts ? static_cast<int>(opts->factors) : WG_FACTORS_IN_B;
        if (factors != WG_FACTORS_IN_B && factors != WG_FACTORS_IN_G)
            return fail(WG_ERR_ARG, "unknown CRT factor placement");
        const int path = opts ? static_cast<int>(opts->path) : WG_PATH_AUTO;
        if (path != WG_PATH_AUTO && path != WG_PATH_SEPARATE && path != WG_PATH_FUSED && path != WG_PATH_FUSED_INPUT)
            return fail(WG_ERR_ARG, "unknown convolution path");
        const int generic = opts ? opts->generic_transforms : 0;
        if (generic != 0 && generic != 1) return fail(WG_ERR_ARG, "generic_transforms must be 0 or 1");
        const int scaling = opts ? static_cast<int>(opts->scaling) : WG_SCALE_NONE;
        if (scaling != WG_SCALE_NONE && scaling != WG_SCALE_ROWS_L1) return fail(WG_ERR_ARG, "unknown scaling");
        const int csum = opts ? static_cast<int>(opts->channel_sum) : WG_SUM_MFMA;
        if (csum != WG_SUM_MFMA && csum != WG_SUM_PAIRWISE) return fail(WG_ERR_ARG, "unknown channel sum");
        if (csum == WG_SUM_PAIRWISE && (path == WG_PATH_FUSED || path == WG_PATH_FUSED_INPUT))
            return fail(WG_ERR_ARG, "pairwise channel sums run on the separate path only");
        const std::vector<wg::Modulus> mods = wg::parse_moduli(moduli);
        std::vector<wg::Rat> pts;
        bool inf = true;
        if (inner && inner[0] != '\0') wg::parse_points(inner, &pts, &inf);
        else pts = {wg::Rat(0), wg::Rat(-1)};
        s = finish_plan(wg::build_transforms(mods, pts, inf, m, r, factors == WG_FACTORS_IN_G,
                                             scaling == WG_SCALE_ROWS_L1),
                        dtype, out);
        if (s == WG_OK) {
            (*out)->path = path;
            (*out)->channel_sum = csum;
            if (generic) (*out)->builtin = -1;
        }
        return s;
    });
}

void winograd_plan_destroy(wg_plan plan) { delete plan; }

int winograd_plan_alpha(wg_plan plan) { return plan ? plan->tr.alpha : 0; }

wg_status winograd_plan_builtin(wg_plan plan, int* id) {
    if (!plan || !id) return fail(WG_ERR_ARG, "null argument");
    *id = plan->builtin;
    return WG_OK;
}

wg_status winograd_plan_info(wg_plan plan, int* m, int* r, int* alpha, int* tile_in, int* dtype) {
    if (!plan) return fail(WG_ERR_ARG, "null plan");
    if (m) *m = plan->tr.m;
    if (r) *r = plan->tr.r;
    if (alpha) *alpha = plan->tr.alpha;
    if (tile_in) *tile_in = plan->tr.tile_in;
    if (dtype) *dtype = plan->dtype;
    return WG_OK;
}

wg_status winograd_plan_matrix(wg_plan plan, char which, wg_rational* out, size_t cap) {
    if (!plan || !out) return fail(WG_ERR_ARG, "null argument");
    const std::vector<wg::Rat>* src = which == 'G' ? &plan->tr.G : which == 'A' ? &plan->tr.A
                                    : which == 'B' ? &plan->tr.B : nullptr;
    if (!src) return fail(WG_ERR_ARG, "matrix must be 'G', 'A' or 'B'");
    if (cap < src->size()) return fail(WG_ERR_ARG, "output capacity too small");
    for (size_t i = 0; i < src->size(); ++i) out[i] = wg_rational{(*src)[i].num(), (*src)[i].den()};
    return WG_OK;
}

wg_status winograd_plan_matrix_f32(wg_plan plan, char which, float* out, size_t cap) {
    if (!plan || !out) return fail(WG_ERR_ARG, "null argument");
    const std::vector<float>* src = which == 'G' ? &plan->tr.Gf : which == 'A' ? &plan->tr.Af
                                  : which == 'B' ? &plan->tr.Bf : nullptr;
    if (!src) return fail(WG_ERR_ARG, "matrix must be 'G', 'A' or 'B'");
    if (cap < src->size()) return fail(WG_ERR_ARG, "output capacity too small");
    std::memcpy(out, src->data(), src->size() * sizeof(float));
    return WG_OK;
}

wg_status winograd_plan_ratio(wg_plan plan, int64_t* num, int64_t* den) {
    if (!plan || !num || !den) return fail(WG_ERR_ARG, "null argument");
    return guarded([&]() -> wg_status {
        const wg::Rat q = wg::Rat(int64_t(plan->tr.alpha) * plan->tr.alpha, int64_t(plan->tr.m) * plan->tr.m);
        *num = q.num();
        *den = q.den();
        return WG_OK;
    });
}

wg_status winograd_workspace_bytes(wg_plan plan, int64_t N, int64_t H, int64_t W, int64_t C, int64_t K,
                                   size_t* bytes) {
    if (!plan || !bytes) return fail(WG_ERR_ARG, "null argument");
    if (!dims_ok(N, H, W, C, K)) return fail(WG_ERR_ARG, "layer sizes must be in [1, 2^31)");
    const Layout L = layout_for(plan, N, H, W, C, K);
    if (L.path < 0) return fail(WG_ERR_UNSUPPORTED, "the fused path does not support this layer shape");
    *bytes = L.total;
    return WG_OK;
}

wg_status winograd_conv_path(wg_plan plan, int64_t N, int64_t H, int64_t W, int64_t C, int64_t K,
                             wg_conv_path* path) {
    if (!plan || !path) return fail(WG_ERR_ARG, "null argument");
    if (!dims_ok(N, H, W, C, K)) return fail(WG_ERR_ARG, "layer sizes must be in [1, 2^31)");
    const int p = resolve_path(plan, wg::make_geometry(N, H, W, C, K, plan->tr.m, plan->tr.alpha));
    if (p < 0) return fail(WG_ERR_UNSUPPORTED, "the fused path does not support this layer shape");
    *path = static_cast<wg_conv_path>(p);
    return WG_OK;
}

wg_status winograd_conv_chunks(wg_plan plan, int64_t N, int64_t H, int64_t W, int64_t C, int64_t K,
                               int64_t* n_chunks, int64_t* chunk) {
    if (!plan || !n_chunks || !chunk) return fail(WG_ERR_ARG, "null argument");
    if (!dims_ok(N, H, W, C, K)) return fail(WG_ERR_ARG, "layer sizes must be in [1, 2^31)");
    const Layout L = layout_for(plan, N, H, W, C, K);
    if (L.path < 0) return fail(WG_ERR_UNSUPPORTED, "the fused path does not support this layer shape");
    *n_chunks = L.n_chunks;
    *chunk = L.chunk;
    return WG_OK;
}

wg_status winograd_plan_set_workspace(wg_plan plan, void* dev_ptr, size_t bytes) {
    if (!plan) return fail(WG_ERR_ARG, "null plan");
    if (dev_ptr && (reinterpret_cast<uintptr_t>(dev_ptr) & 255u) != 0)
        return fail(WG_ERR_ARG, "workspace must be 256-byte aligned");
    plan->ws = dev_ptr;
    plan->ws_bytes = dev_ptr ? bytes : 0;
    return WG_OK;
}

}  // extern "C"

namespace {

// The launches of winograd_conv2d with the workspace at ws (ws_bytes long,
// 256-byte aligned; nullptr: none) after the argument checks.
wg_status conv2d_with(wg_plan plan, const wg_tensor* x, const wg_tensor* w, wg_tensor* y, void* ws,
                      size_t ws_bytes, bool static_ws, hipStream_t stream) {
    wg_status s = check_plan(plan);
    if (s != WG_OK) return s;
    if ((s = check_tensor(x, "x")) != WG_OK || (s = check_tensor(w, "w")) != WG_OK ||
        (s = check_tensor(y, "y")) != WG_OK)
        return s;
    if (w->h != 3 || w->w != 3 || w->c != x->c)
        return fail(WG_ERR_ARG, "w must be [K][3][3][C] with the input's C");
    if (y->n != x->n || y->h != x->h || y->w != x->w || y->c != w->n)
        return fail(WG_ERR_ARG, "y must be [N][H][W][K]");
    if (!dims_ok(x->n, x->h, x->w, x->c, w->n)) return fail(WG_ERR_ARG, "layer sizes must be in [1, 2^31)");
    const Layout L = layout_for(plan, x->n, x->h, x->w, x->c, w->n);
    if (L.path < 0) return fail(WG_ERR_UNSUPPORTED, "the fused path does not support this layer shape");
    if (static_ws) {
        if (L.total > ws_bytes)
            return fail(WG_ERR_WORKSPACE, "layer needs " + std::to_string(L.total) +
                                              " bytes of workspace, more than the " + std::to_string(ws_bytes) +
                                              " bytes of the allocation-free entry point");
    } else {
        if (!ws) return fail(WG_ERR_WORKSPACE, "no workspace bound to the plan");
        if (ws_bytes < L.total)
            return fail(WG_ERR_WORKSPACE, "workspace too small: need " + std::to_string(L.total) + " bytes");
    }
    auto* base = static_cast<unsigned char*>(ws);
    void* U = base + L.u_off;
    void* V = base + L.v_off;
    auto* M = reinterpret_cast<float*>(base + L.m_off);
    const int dt = plan->dtype;
    if (L.path == WG_PATH_FUSED_INPUT) {
        // kernel transform, then the fused kernel computes V itself
        if ((s = from_hip(launch_kt(dt, L.g, plan->ktab, w->data, U, stream), "kernel transform")) != WG_OK) return s;
        return from_hip(launch_ico(dt, L.g, plan->itab, plan->otab, x->data, U, y->data, stream),
                        "fused input transform and contraction");
    }
    if (L.path == WG_PATH_FUSED && L.n_chunks > 1) {
        // chunks of images: the transforms of the first chunk compute U as well
        const int64_t es = wg::dtype_bytes(dt);
        const int64_t base = x->n / L.n_chunks, rem = x->n % L.n_chunks;
        for (int64_t i = 0, n0 = 0; i < L.n_chunks; ++i) {
            const int64_t nc = base + (i < rem ? 1 : 0);
            const wg::Geometry g = wg::make_geometry(nc, x->h, x->w, x->c, w->n, plan->tr.m, plan->tr.alpha);
            const void* xc = static_cast<const unsigned char*>(x->data) + n0 * x->h * x->w * x->c * es;
            void* yc = static_cast<unsigned char*>(y->data) + n0 * y->h * y->w * y->c * es;
            s = n0 == 0 ? from_hip(launch_kit(dt, g, plan->ktab, plan->itab, w->data, xc, U, V, plan->builtin, stream),
                                   "kernel and input transforms")
                        : from_hip(launch_it(dt, g, plan->itab, xc, V, plan->builtin, stream), "input transform");
            if (s != WG_OK) return s;
            if ((s = from_hip(launch_co(dt, g, plan->otab, V, U, yc, plan->builtin, stream), "fused contraction")) !=
                WG_OK)
                return s;
            n0 += nc;
        }
        return WG_OK;
    }
    s = from_hip(launch_kit(dt, L.g, plan->ktab, plan->itab, w->data, x->data, U, V, plan->builtin, stream),
                 "kernel and input transforms");
    if (s != WG_OK) return s;
    if (L.path == WG_PATH_FUSED)
        return from_hip(launch_co(dt, L.g, plan->otab, V, U, y->data, plan->builtin, stream), "fused contraction");
    if ((s = from_hip(launch_ct(dt, L.g, V, U, M, stream, plan->channel_sum), "contraction")) != WG_OK) return s;
    return from_hip(launch_ot(dt, L.g, plan->otab, M, y->data, plan->builtin, stream), "output transform");
}

// Workspace of the 1D path: U [alpha'][K][Cp], V [alpha'][T][Cp], M [alpha'][T][Kp].
struct Layout1d {
    wg::Geometry g;
    size_t u_off, v_off, m_off, total;
};

Layout1d layout_1d(const wg_plan_s* p, int64_t N, int64_t L, int64_t C, int64_t K) {
    Layout1d o;
    o.g = wg::make_geometry_1d(N, L, C, K, p->tr.m, p->tr.alpha);
    const size_t es = static_cast<size_t>(wg::dtype_bytes(p->dtype));
    const size_t al = static_cast<size_t>(p->tr.alpha);
    o.u_off = 0;
    o.v_off = align256(al * static_cast<size_t>(K) * static_cast<size_t>(o.g.Cp) * es);
    o.m_off = o.v_off + align256(al * static_cast<size_t>(o.g.T) * static_cast<size_t>(o.g.Cp) * es);
    o.total = o.m_off + align256(al * static_cast<size_t>(o.g.T) * static_cast<size_t>(o.g.Kp) * sizeof(float));
    return o;
}

}  // namespace

extern "C" {

wg_status winograd_workspace_bytes_1d(wg_plan plan, int64_t N, int64_t L, int64_t C, int64_t K, size_t* bytes) {
    if (!plan || !bytes) return fail(WG_ERR_ARG, "null argument");
    if (!dims_ok(N, 1, L, C, K)) return fail(WG_ERR_ARG, "layer sizes must be in [1, 2^31)");
    *bytes = layout_1d(plan, N, L, C, K).total;
    return WG_OK;
}

wg_status winograd_conv1d(wg_plan plan, const wg_tensor* x, const wg_tensor* w, wg_tensor* y, hipStream_t stream) {
    if (!plan) return fail(WG_ERR_ARG, "null plan");
    wg_status s;
    if ((s = check_tensor(x, "x")) != WG_OK || (s = check_tensor(w, "w")) != WG_OK ||
        (s = check_tensor(y, "y")) != WG_OK)
        return s;
    if (x->h != 1 || w->h != 1 || w->w != 3 || w->c != x->c)
        return fail(WG_ERR_ARG, "x must be [N][1][L][C] and w [K][1][3][C] with the input's C");
    if (y->n != x->n || y->h != 1 || y->w != x->w || y->c != w->n) return fail(WG_ERR_ARG, "y must be [N][1][L][K]");
    if (!dims_ok(x->n, 1, x->w, x->c, w->n)) return fail(WG_ERR_ARG, "layer sizes must be in [1, 2^31)");
    if (plan->tr.r != 3) return fail(WG_ERR_UNSUPPORTED, "only 3-tap kernels");
    const Layout1d L = layout_1d(plan, x->n, x->w, x->c, w->n);
    if (!plan->ws) return fail(WG_ERR_WORKSPACE, "no workspace bound to the plan");
    if (plan->ws_bytes < L.total)
        return fail(WG_ERR_WORKSPACE, "workspace too small: need " + std::to_string(L.total) + " bytes");
    auto* base = static_cast<unsigned char*>(plan->ws);
    void* U = base + L.u_off;
    void* V = base + L.v_off;
    auto* M = reinterpret_cast<float*>(base + L.m_off);
    hipError_t e;
    switch (plan->dtype) {
        case 0: e = wg::launch_kernel_transform_1d_t<0>(L.g, plan->ktab, w->data, U, stream); break;
        case 1: e = wg::launch_kernel_transform_1d_t<1>(L.g, plan->ktab, w->data, U, stream); break;
        default: e = wg::launch_kernel_transform_1d_t<2>(L.g, plan->ktab, w->data, U, stream); break;
    }
    if ((s = from_hip(e, "1D kernel transform")) != WG_OK) return s;
    switch (plan->dtype) {
        case 0: e = wg::launch_input_transform_1d_t<0>(L.g, plan->itab, x->data, V, stream); break;
        case 1: e = wg::launch_input_transform_1d_t<1>(L.g, plan->itab, x->data, V, stream); break;
        default: e = wg::launch_input_transform_1d_t<2>(L.g, plan->itab, x->data, V, stream); break;
    }
    if ((s = from_hip(e, "1D input transform")) != WG_OK) return s;
    if ((s = from_hip(launch_ct(plan->dtype, L.g, V, U, M, stream, plan->channel_sum), "contraction")) != WG_OK)
        return s;
    switch (plan->dtype) {
        case 0: e = wg::launch_output_transform_1d_t<0>(L.g, plan->otab, M, y->data, stream); break;
        case 1: e = wg::launch_output_transform_1d_t<1>(L.g, plan->otab, M, y->data, stream); break;
        default: e = wg::launch_output_transform_1d_t<2>(L.g, plan->otab, M, y->data, stream); break;
    }
    return from_hip(e, "1D output transform");
}

wg_status winograd_conv2d(wg_plan plan, const wg_tensor* x, const wg_tensor* w, wg_tensor* y,
                          hipStream_t stream) {
    if (!plan) return fail(WG_ERR_ARG, "null plan");
    return conv2d_with(plan, x, w, y, plan->ws, plan->ws_bytes, false, stream);
}

wg_status winograd_conv2d_static(wg_plan plan, const wg_tensor* x, const wg_tensor* w, wg_tensor* y,
                                 hipStream_t stream) {
    if (!plan) return fail(WG_ERR_ARG, "null plan");
    void* ws = nullptr;
    const wg_status s = static_scratch(&ws);
    if (s != WG_OK) return s;
    return conv2d_with(plan, x, w, y, ws, WG_STATIC_SCRATCH_BYTES, true, stream);
}

wg_status winograd_kernel_transform(wg_plan plan, const wg_tensor* w, void* U, hipStream_t stream) {
    wg_status s = check_plan(plan);
    if (s != WG_OK) return s;
    if ((s = check_tensor(w, "w")) != WG_OK) return s;
    if (!U || !aligned16(U)) return fail(WG_ERR_ARG, "U must be a 16-byte aligned device pointer");
    if (w->h != 3 || w->w != 3) return fail(WG_ERR_ARG, "w must be [K][3][3][C]");
    if (!dims_ok(1, 1, 1, w->c, w->n)) return fail(WG_ERR_ARG, "sizes must be in [1, 2^31)");
    const wg::Geometry g = wg::make_geometry(1, 1, 1, w->c, w->n, plan->tr.m, plan->tr.alpha);
    return from_hip(launch_kt(plan->dtype, g, plan->ktab, w->data, U, stream), "kernel transform");
}

wg_status winograd_input_transform(wg_plan plan, const wg_tensor* x, void* V, hipStream_t stream) {
    wg_status s = check_plan(plan);
    if (s != WG_OK) return s;
    if ((s = check_tensor(x, "x")) != WG_OK) return s;
    if (!V || !aligned16(V)) return fail(WG_ERR_ARG, "V must be a 16-byte aligned device pointer");
    if (!dims_ok(x->n, x->h, x->w, x->c, 1)) return fail(WG_ERR_ARG, "sizes must be in [1, 2^31)");
    const wg::Geometry g = wg::make_geometry(x->n, x->h, x->w, x->c, 1, plan->tr.m, plan->tr.alpha);
    return from_hip(launch_it(plan->dtype, g, plan->itab, x->data, V, plan->builtin, stream), "input transform");
}

wg_status winograd_kernel_input_transform(wg_plan plan, const wg_tensor* w, const wg_tensor* x, void* U, void* V,
                                          hipStream_t stream) {
    wg_status s = check_plan(plan);
    if (s != WG_OK) return s;
    if ((s = check_tensor(w, "w")) != WG_OK || (s = check_tensor(x, "x")) != WG_OK) return s;
    if (!U || !V || !aligned16(U) || !aligned16(V))
        return fail(WG_ERR_ARG, "U and V must be 16-byte aligned device pointers");
    if (w->h != 3 || w->w != 3 || w->c != x->c) return fail(WG_ERR_ARG, "w must be [K][3][3][C] with the input's C");
    if (!dims_ok(x->n, x->h, x->w, x->c, w->n)) return fail(WG_ERR_ARG, "sizes must be in [1, 2^31)");
    const wg::Geometry g = wg::make_geometry(x->n, x->h, x->w, x->c, w->n, plan->tr.m, plan->tr.alpha);
    return from_hip(launch_kit(plan->dtype, g, plan->ktab, plan->itab, w->data, x->data, U, V, plan->builtin, stream),
                    "kernel and input transforms");
}

wg_status winograd_contract(wg_plan plan, const void* V, const void* U, float* M, int64_t T, int64_t C,
                            int64_t K, hipStream_t stream) {
    wg_status s = check_plan(plan);
    if (s != WG_OK) return s;
    if (!V || !U || !M || !aligned16(V) || !aligned16(U) || !aligned16(M))
        return fail(WG_ERR_ARG, "V, U and M must be 16-byte aligned device pointers");
    if (!dims_ok(T, 1, 1, C, K)) return fail(WG_ERR_ARG, "sizes must be in [1, 2^31)");
    wg::Geometry g = wg::make_geometry(1, 1, 1, C, K, plan->tr.m, plan->tr.alpha);
    g.T = T;
    return from_hip(launch_ct(plan->dtype, g, V, U, M, stream, plan->channel_sum), "contraction");
}

wg_status winograd_output_transform(wg_plan plan, const float* M, wg_tensor* y, hipStream_t stream) {
    wg_status s = check_plan(plan);
    if (s != WG_OK) return s;
    if ((s = check_tensor(y, "y")) != WG_OK) return s;
    if (!M || !aligned16(M)) return fail(WG_ERR_ARG, "M must be a 16-byte aligned device pointer");
    if (!dims_ok(y->n, y->h, y->w, 1, y->c)) return fail(WG_ERR_ARG, "sizes must be in [1, 2^31)");
    const wg::Geometry g = wg::make_geometry(y->n, y->h, y->w, 1, y->c, plan->tr.m, plan->tr.alpha);
    return from_hip(launch_ot(plan->dtype, g, plan->otab, M, y->data, plan->builtin, stream), "output transform");
}

wg_status winograd_contract_output(wg_plan plan, const void* V, const void* U, int64_t C, wg_tensor* y,
                                   hipStream_t stream) {
    wg_status s = check_plan(plan);
    if (s != WG_OK) return s;
    if ((s = check_tensor(y, "y")) != WG_OK) return s;
    if (!V || !U || !aligned16(V) || !aligned16(U))
        return fail(WG_ERR_ARG, "V and U must be 16-byte aligned device pointers");
    if (!dims_ok(y->n, y->h, y->w, C, y->c)) return fail(WG_ERR_ARG, "sizes must be in [1, 2^31)");
    const wg::Geometry g = wg::make_geometry(y->n, y->h, y->w, C, y->c, plan->tr.m, plan->tr.alpha);
    if (!fused_supported(plan->dtype, g))
        return fail(WG_ERR_UNSUPPORTED, "the fused kernel does not support this layer shape");
    return from_hip(launch_co(plan->dtype, g, plan->otab, V, U, y->data, plan->builtin, stream), "fused contraction");
}

wg_status winograd_input_contract_output(wg_plan plan, const wg_tensor* x, const void* U, wg_tensor* y,
                                         hipStream_t stream) {
    wg_status s = check_plan(plan);
    if (s != WG_OK) return s;
    if ((s = check_tensor(x, "x")) != WG_OK || (s = check_tensor(y, "y")) != WG_OK) return s;
    if (!U || !aligned16(U)) return fail(WG_ERR_ARG, "U must be a 16-byte aligned device pointer");
    if (y->n != x->n || y->h != x->h || y->w != x->w) return fail(WG_ERR_ARG, "y must be [N][H][W][K] for x's N, H, W");
    if (!dims_ok(x->n, x->h, x->w, x->c, y->c)) return fail(WG_ERR_ARG, "sizes must be in [1, 2^31)");
    const wg::Geometry g = wg::make_geometry(x->n, x->h, x->w, x->c, y->c, plan->tr.m, plan->tr.alpha);
    if (!input_fused_supported(plan->dtype, g))
        return fail(WG_ERR_UNSUPPORTED, "the input transform is not fused for this layer shape");
    return from_hip(launch_ico(plan->dtype, g, plan->itab, plan->otab, x->data, U, y->data, stream),
                    "fused input transform and contraction");
}

wg_status winograd_relu_pool(wg_dtype dtype, const wg_tensor* x, wg_tensor* y, int pool, hipStream_t stream) {
    wg_status s;
    if ((s = check_tensor(x, "x")) != WG_OK) return s;
    if (!y) return fail(WG_ERR_ARG, "null tensor y");
    if (dtype != WG_F32 && dtype != WG_F16 && dtype != WG_BF16) return fail(WG_ERR_UNSUPPORTED, "unknown dtype");
    if (pool != 0 && pool != 1) return fail(WG_ERR_ARG, "pool must be 0 or 1");
    if (!dims_ok(x->n, x->h, x->w, x->c, 1)) return fail(WG_ERR_ARG, "sizes must be in [1, 2^31)");
    const int64_t ho = pool ? x->h / 2 : x->h, wo = pool ? x->w / 2 : x->w;
    if (y->n != x->n || y->h != ho || y->w != wo || y->c != x->c)
        return fail(WG_ERR_ARG, pool ? "y must be [N][H/2][W/2][C]" : "y must be shaped like x");
    if (ho == 0 || wo == 0) return WG_OK;   // pooling a single row or column: nothing to store
    if ((s = check_tensor(y, "y")) != WG_OK) return s;
    const int64_t es = wg::dtype_bytes(dtype);
    const auto* xb = static_cast<const unsigned char*>(x->data);
    const auto* yb = static_cast<const unsigned char*>(y->data);
    const int64_t xbytes = x->n * x->h * x->w * x->c * es, ybytes = y->n * y->h * y->w * y->c * es;
    if (xb < yb + ybytes && yb < xb + xbytes) return fail(WG_ERR_ARG, "x and y overlap");
    hipError_t e;
    switch (dtype) {
        case WG_F32: e = wg::launch_relu_pool_t<0>(x->data, y->data, x->n, x->h, x->w, x->c, pool, stream); break;
        case WG_F16: e = wg::launch_relu_pool_t<1>(x->data, y->data, x->n, x->h, x->w, x->c, pool, stream); break;
        default: e = wg::launch_relu_pool_t<2>(x->data, y->data, x->n, x->h, x->w, x->c, pool, stream); break;
    }
    return from_hip(e, "relu/max-pool");
}

wg_status winograd_direct_conv_f64(wg_dtype dtype, const wg_tensor* x, const wg_tensor* w, double* y,
                                   hipStream_t stream) {
    wg_status s;
    if ((s = check_tensor(x, "x")) != WG_OK || (s = check_tensor(w, "w")) != WG_OK) return s;
    if (!y || (reinterpret_cast<uintptr_t>(y) & 7u) != 0) return fail(WG_ERR_ARG, "y must be an 8-byte aligned device pointer");
    if (dtype != WG_F32 && dtype != WG_F16 && dtype != WG_BF16) return fail(WG_ERR_UNSUPPORTED, "unknown dtype");
    if ((w->h != 3 && w->h != 1) || w->w != 3 || w->c != x->c)
        return fail(WG_ERR_ARG, "w must be [K][3][3][C] or [K][1][3][C] with the input's C");
    if (!dims_ok(x->n, x->h, x->w, x->c, w->n)) return fail(WG_ERR_ARG, "sizes must be in [1, 2^31)");
    const int kh = static_cast<int>(w->h);
    hipError_t e;
    switch (dtype) {
        case WG_F32: e = wg::launch_direct_f64_t<0>(x->data, w->data, y, x->n, x->h, x->w, x->c, w->n, kh, stream); break;
        case WG_F16: e = wg::launch_direct_f64_t<1>(x->data, w->data, y, x->n, x->h, x->w, x->c, w->n, kh, stream); break;
        default: e = wg::launch_direct_f64_t<2>(x->data, w->data, y, x->n, x->h, x->w, x->c, w->n, kh, stream); break;
    }
    return from_hip(e, "float64 direct convolution");
}

wg_status winograd_sq_error_sums(wg_dtype dtype, const void* y, const double* ref, int64_t n, double* sums,
                                 hipStream_t stream) {
    static_assert(WG_SQ_SUMS_DOUBLES == wg::kSqSumDoubles, "sums buffer size");
    if (!y || !ref || !sums) return fail(WG_ERR_ARG, "null pointer");
    if ((reinterpret_cast<uintptr_t>(ref) & 7u) != 0 || (reinterpret_cast<uintptr_t>(sums) & 7u) != 0)
        return fail(WG_ERR_ARG, "ref and sums must be 8-byte aligned");
    if (n < 0) return fail(WG_ERR_ARG, "n must be non-negative");
    if (dtype != WG_F32 && dtype != WG_F16 && dtype != WG_BF16) return fail(WG_ERR_UNSUPPORTED, "unknown dtype");
    hipError_t e;
    switch (dtype) {
        case WG_F32: e = wg::launch_sq_sums_t<0>(y, ref, n, sums, stream); break;
        case WG_F16: e = wg::launch_sq_sums_t<1>(y, ref, n, sums, stream); break;
        default: e = wg::launch_sq_sums_t<2>(y, ref, n, sums, stream); break;
    }
    return from_hip(e, "error sums");
}

const char* winograd_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
