/*
 * winograd_crt.h -- C ABI of the MI355X (gfx950) Winograd convolution library.
 *
 * The library computes a DNN convolution layer with 3x3 kernels (stride 1,
 * zero padding 1, cross-correlation as in DNN frameworks) by the 2D Winograd
 * algorithm in the matrix-exchange form of Barabasz & Gregg, "Winograd
 * Convolution for DNNs: Beyond linear polynomials" (arXiv 1905.05233),
 * eq. (2):
 *
 *     Y = A^T [ (G g G^T) (.) (B^T d B) ] A
 *
 * on every (m+2)x(m+2) input tile d and 3x3 kernel g, summed over input
 * channels.  The transforms G (alpha' x 3), A (alpha' x m) and B
 * ((m+2) x alpha') are built by the polynomial Chinese Remainder Theorem
 * (Section 2.1, eq. (1)) from a set of moduli that may contain degree-2
 * ("superlinear") polynomials as well as linear ones (points), following
 * Algorithm 1 (G, A) and Algorithm 2 (B) of Section 2.2, in exact rational
 * arithmetic on the host.
 *
 * Conventions shared by every entry point
 *   - Tensors are dense, row-major, in device memory:
 *       x  [N][H][W][C]   (NHWC input)
 *       w  [K][3][3][C]   (weights)
 *       y  [N][H][W][K]   (NHWC output)
 *     all in the plan's storage dtype (fp32, fp16 or bf16).  Every transform
 *     runs in fp32 registers; the channel contraction accumulates in fp32 for
 *     every dtype; results are rounded to the dtype once, when stored.
 *   - Device pointers must be 16-byte aligned.
 *   - Every function returns a wg_status; on error the out-parameters are left
 *     untouched and winograd_last_error() describes the failure.  No C++
 *     exception crosses this interface.
 *   - Launching functions are asynchronous on the given HIP stream and never
 *     synchronise.  A plan is immutable after creation except for its bound
 *     workspace: do not use one plan on two streams at the same time.
 *   - The caller owns every buffer and the stream; a plan owns only its host
 *     tables and is released by winograd_plan_destroy().
 */
#ifndef WINOGRAD_CRT_H
#define WINOGRAD_CRT_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { WG_F32 = 0, WG_F16 = 1, WG_BF16 = 2 } wg_dtype;

typedef enum {
    WG_OK = 0,
    WG_ERR_ARG = 1,          /* null pointer, bad size, misaligned pointer, parse error */
    WG_ERR_DEGREE_SUM = 2,   /* sum of modulus degrees does not match m + r - 1 */
    WG_ERR_NOT_COPRIME = 3,  /* two moduli share a factor (Section 2.1) */
    WG_ERR_REDUCIBLE = 4,    /* a modulus is reducible over Q (Section 2.1) */
    WG_ERR_UNSUPPORTED = 5,  /* r != 3, alpha' or tile beyond the kernels' range, dtype */
    WG_ERR_OVERFLOW = 6,     /* exact rational arithmetic left the int64 range */
    WG_ERR_WORKSPACE = 7,    /* no workspace bound, or too small */
    WG_ERR_HIP = 8,          /* a HIP runtime call or kernel launch failed */
    WG_ERR_INTERNAL = 9      /* the exact self-check of a built plan failed */
} wg_status;

/* An exact rational num/den (den > 0 after normalisation). */
typedef struct { int64_t num, den; } wg_rational;

/* One modulus m_i(a) of the CRT (Section 2.1).  degree 0 denotes the
 * pseudo-point infinity of the "modified" algorithm (Section 2.1, Algorithm 1
 * last rows); otherwise coef[0..degree] are the coefficients, lowest power
 * first (the paper's vec() order).  Moduli are made monic by the library. */
typedef struct { int degree; wg_rational coef[4]; } wg_modulus;

/* The modulus set and the evaluation points of the inner Toom-Cook
 * algorithm F_T-C(d x d, d x d) used for every degree-d modulus
 * (Section 2.1, Algorithm 1 and 2).  Row order of the Winograd domain:
 * modulus list order, 2d-1 rows per degree-d modulus in inner-point order,
 * the pseudo-point last.  A degree-d modulus uses the first 2d-2 inner points
 * plus infinity when inner_inf != 0, else the first 2d-1 points.  With
 * n_inner == 0 the points 0, -1 and infinity are used (Section 3.1). */
typedef struct {
    int n_mod;
    const wg_modulus* mods;
    int n_inner;
    const wg_rational* inner_pts;
    int inner_inf;
} wg_poly_set;

/* A dense NHWC tensor (weights: n = K, h = w = 3, c = C). */
typedef struct { void* data; int64_t n, h, w, c; } wg_tensor;

typedef struct wg_plan_s* wg_plan;

/* Build the transforms of F(m x m, r x r) from a modulus set (Algorithms 1
 * and 2) in exact rational arithmetic, check them with the exact CRT
 * reconstruction identity sum_xi B[k,xi] G[xi,i] A[xi,j] = [k == i+j], and
 * round them once to fp32 (nearest, ties to even) for the kernels.
 * Requirements: r == 3; the moduli are irreducible and pairwise coprime;
 * sum of finite degrees == m + r - 2 with the pseudo-point, m + r - 1
 * without; 3 <= m + 2 <= 16 and alpha' <= 16.  *out receives a new plan. */
wg_status winograd_plan_create(const wg_poly_set* set, int m, int r, wg_dtype dtype, wg_plan* out);

/* Same as winograd_plan_create with the set written as text: a comma list
 * of points ("0", "-1/2"), polynomials in a ("a^2+1", "a^2-a+1") and "inf";
 * inner is the inner point list, e.g. "0,-1,inf" (NULL or "" = default). */
wg_status winograd_plan_create_str(const char* moduli, const char* inner, int m, int r,
                                   wg_dtype dtype, wg_plan* out);

/* Where the CRT factors N_i of eq. (1) go.  WG_FACTORS_IN_B is the paper's
 * construction (Section 2.2: the matrices G and A are not scaled by N_i, the
 * factors sit in B through E).  WG_FACTORS_IN_G multiplies the kernel
 * residues by N_i instead: G' = [vec(R_m[N_i a^k])] (for a linear modulus
 * a - p the row [p^0 .. p^(r-1)] times the constant N_i = 1 / M_i(p)) and
 * E_i = [vec(R_M[a^k M_i])].  Both are exact; they round differently.  For
 * linear points the second gives the matrices of Lavin & Gray's F(4,3). */
typedef enum { WG_FACTORS_IN_B = 0, WG_FACTORS_IN_G = 1 } wg_crt_factors;

/* How winograd_conv2d evaluates eq. (2) after the two transforms.
 * WG_PATH_SEPARATE: the alpha'^2 channel contractions write M to the
 * workspace and the output transform reads it back (four kernels).
 * WG_PATH_FUSED: one kernel contracts and applies the output transform while
 * M of each domain point is still in registers, so M never reaches memory
 * (input tiles up to 8, i.e. m <= 6, and per-plane sizes of V and U under
 * 4 GiB).  WG_PATH_FUSED_INPUT: the fused kernel also computes the input
 * transform, per block into LDS, so V never reaches memory either (channel
 * rows of at most 32 bytes, i.e. C <= 16 fp16/bf16 or C <= 8 fp32, more than
 * 32 output channels and the block's alpha'^2 x 32 V rows within 48 KB; the
 * same values as WG_PATH_FUSED bit for bit).  WG_PATH_AUTO picks per layer
 * shape between the first two (winograd_conv_path reports the choice).  All
 * paths give results within the same error bound; the separate and fused
 * ones may differ in the last bits because the channel sums run in another
 * order. */
typedef enum { WG_PATH_AUTO = 0, WG_PATH_SEPARATE = 1, WG_PATH_FUSED = 2, WG_PATH_FUSED_INPUT = 3 } wg_conv_path;

/* Diagonal scaling of the transforms (the scaling of G and A^T that the
 * related work of Section 4 cites from Vincent et al.).  WG_SCALE_NONE keeps
 * the matrices of Algorithms 1 and 2.  WG_SCALE_ROWS_L1 divides every domain
 * row of G and of A by its 1-norm (sum of absolute values; a zero row stays
 * as it is) and multiplies the matching column of B by both norms: each
 * domain point's rank-1 term
 * B[:, xi] G[xi] A[xi] is unchanged, so the algorithm stays exact and only
 * its roundings change. */
typedef enum { WG_SCALE_NONE = 0, WG_SCALE_ROWS_L1 = 1 } wg_scaling;

/* generic_transforms = 1 keeps a plan on the transform kernels that read its
 * coefficients at run time even when its tables equal a built-in plan's (see
 * winograd_plan_builtin); 0 (the default) lets it use the built-in kernels. */
/* How the contraction sums over the input channels.  WG_SUM_MFMA: the
 * matrix cores' accumulation chains (the fast kernels).  WG_SUM_PAIRWISE: the
 * pairwise summation over channels that the related work of Section 4 names
 * (after Barabasz et al. 2018): each 64-byte piece of a channel row (16 fp32
 * or 32 fp16/bf16 channels) is summed into its own fp32 partial, and the
 * partials are added in a binary tree in channel order, so the rounding
 * error of the sum grows with log2 C rather than C.  It runs on the separate
 * path with a slower kernel (fragments from memory, nothing staged). */
typedef enum { WG_SUM_MFMA = 0, WG_SUM_PAIRWISE = 1 } wg_channel_sum;

typedef struct {
    wg_crt_factors factors;
    wg_conv_path path;
    int generic_transforms;
    wg_scaling scaling;
    wg_channel_sum channel_sum;
} wg_plan_options;

/* winograd_plan_create_str with options (opts == NULL means all defaults:
 * WG_FACTORS_IN_B, WG_PATH_AUTO, generic_transforms 0, WG_SCALE_NONE,
 * WG_SUM_MFMA).  An unknown option value is WG_ERR_ARG, and so is
 * WG_SUM_PAIRWISE with a fused path. */
wg_status winograd_plan_create_ex(const char* moduli, const char* inner, int m, int r, wg_dtype dtype,
                                  const wg_plan_options* opts, wg_plan* out);

/* Release a plan (NULL is ignored).  Does not free a bound workspace. */
void winograd_plan_destroy(wg_plan plan);

/* alpha' = sum over finite moduli of (2 deg - 1), plus 1 for infinity: the
 * number of Winograd-domain points per dimension, i.e. the rows of G and A
 * that Algorithm 1 stacks (a degree-d modulus contributes the 2d - 1 rows of
 * its inner Toom-Cook algorithm); alpha'^2 / m^2 is the ratio of Section 2.3,
 * Table 1.  0 for a NULL plan. */
int winograd_plan_alpha(wg_plan plan);

/* The library carries input and output transform kernels with the
 * coefficients of a few plans compiled in (the F(2x2), F(4x4) and F(6x6) sets
 * of its workloads; the compiler drops the zero terms).  *id is the index of
 * the built-in plan whose fp32 tables are bit-identical to this plan's, which
 * the plan then uses, or -1.  Results equal the generic kernels' for finite
 * data (up to the sign of zero). */
wg_status winograd_plan_builtin(wg_plan plan, int* id);

/* m, r, alpha', input tile m + r - 1 and dtype of a plan. */
wg_status winograd_plan_info(wg_plan plan, int* m, int* r, int* alpha, int* tile_in, int* dtype);

/* Exact matrix 'G' (alpha' x r) or 'A' (alpha' x m) of Algorithm 1, or 'B'
 * ((m+r-1) x alpha') of Algorithm 2 (B^W = [E C | vec(M)]), row-major, into
 * out[cap] (cap >= rows * cols), each entry num/den in lowest terms with
 * den > 0.  WG_ERR_ARG for another letter, a NULL pointer or a short cap. */
wg_status winograd_plan_matrix(wg_plan plan, char which, wg_rational* out, size_t cap);

/* The same matrix as the fp32 values the kernels use. */
wg_status winograd_plan_matrix_f32(wg_plan plan, char which, float* out, size_t cap);

/* Elementwise multiplications per output point, alpha'^2 / m^2 (Section 2.3,
 * Table 1), as an exact fraction. */
wg_status winograd_plan_ratio(wg_plan plan, int64_t* num, int64_t* den);

/* Device workspace needed by winograd_conv2d for this layer shape (U and V,
 * plus M on the separate path; on the fused path V of one chunk of the batch
 * when winograd_conv2d runs the batch in chunks, see there). */
wg_status winograd_workspace_bytes(wg_plan plan, int64_t N, int64_t H, int64_t W, int64_t C,
                                   int64_t K, size_t* bytes);

/* The path winograd_conv2d takes for this layer shape: WG_PATH_SEPARATE,
 * WG_PATH_FUSED or WG_PATH_FUSED_INPUT.  WG_ERR_UNSUPPORTED if the plan asks
 * for a fused path and the shape does not allow it. */
wg_status winograd_conv_path(wg_plan plan, int64_t N, int64_t H, int64_t W, int64_t C, int64_t K,
                             wg_conv_path* path);

/* How winograd_conv2d splits the batch for this layer shape: n_chunks launch
 * pairs (1 unless the fused path chunks the batch), the largest chunk having
 * `chunk` images (the others one fewer at most).  WG_ERR_UNSUPPORTED as
 * winograd_conv_path. */
wg_status winograd_conv_chunks(wg_plan plan, int64_t N, int64_t H, int64_t W, int64_t C, int64_t K,
                               int64_t* n_chunks, int64_t* chunk);

/* Bind a caller-owned device workspace (256-byte aligned) to the plan; a
 * NULL pointer unbinds.  The plan keeps the pointer, not the memory. */
wg_status winograd_plan_set_workspace(wg_plan plan, void* dev_ptr, size_t bytes);

/* y = conv3x3(x, w) by eq. (2): launches the kernel transform, the input
 * transform, then the alpha'^2 batched channel contraction and the output
 * transform (separate path) or the fused kernel that does both (fused path)
 * on `stream`, using the bound workspace; on WG_PATH_FUSED_INPUT the kernel
 * transform and the fused kernel that also computes V.  On WG_PATH_FUSED a
 * batch whose V would exceed 160 MiB goes through in chunks of whole images
 * (sizes differing by at most one), the input transform and the fused kernel
 * launched per chunk with one V buffer, so that V is read back from the
 * GPU's last-level cache; the results are the same bits as one launch pair
 * over the whole batch.  x is [N][H][W][C], w is [K][3][3][C], y is
 * [N][H][W][K]; N, H, W, C, K >= 1 (y->c = K). */
wg_status winograd_conv2d(wg_plan plan, const wg_tensor* x, const wg_tensor* w, wg_tensor* y,
                          hipStream_t stream);

/* Bytes of device workspace that winograd_conv2d_static has on each GPU. */
#define WG_STATIC_SCRATCH_BYTES ((size_t)64 << 20)

/* winograd_conv2d without a bound workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc).  The workspace (U, V and, on the
 * separate path, M) is a 64 MiB array in the library's device memory, one
 * copy per GPU, kept until the process ends; its address on a device is
 * looked up on the first call with that device current.  The call itself
 * allocates nothing: no hipMalloc, no hipFree.  Arguments, layouts, path
 * choice and results are those of winograd_conv2d with the same plan (the
 * plan's bound workspace is neither used nor needed).  A layer whose
 * workspace (winograd_workspace_bytes) exceeds WG_STATIC_SCRATCH_BYTES is
 * rejected with WG_ERR_WORKSPACE before anything is launched.  Every call on
 * a GPU uses that GPU's one array: calls that overlap in time on one GPU
 * (other streams, other threads) race and give wrong results; calls in
 * order on one stream are safe.  Nothing in the array needs to start at zero
 * (every kernel writes what a later one reads). */
wg_status winograd_conv2d_static(wg_plan plan, const wg_tensor* x, const wg_tensor* w, wg_tensor* y,
                                 hipStream_t stream);

/* ---- 1D convolution F(m, 3) ------------------------------------------------
 * The same plan applied in one dimension (Section 2.1's polynomial product,
 * y = A^T [(G g) (.) (B^T d)] on tiles of m outputs; Section 3.1 measures its
 * error beside the 2D form): y[n][0][l][k] = sum_{j<3,c} w[k][0][j][c]
 * x[n][0][l+j-1][c], zero padding 1, cross-correlation.  Tensors use the 4-D
 * descriptor with height 1: x [N][1][L][C], w [K][1][3][C], y [N][1][L][K],
 * storage dtype of the plan.  Rounding points as in 2D: fp32 transforms (one
 * pass each), U and V rounded to the dtype, fp32 channel sums, y rounded once.
 * The workspace (winograd_workspace_bytes_1d: U [alpha'][K][Cp],
 * V [alpha'][T][Cp], M [alpha'][T][Kp] fp32, T = N ceil(L/m)) is the plan's
 * bound one.  Asynchronous on stream; errors as winograd_conv2d. */
wg_status winograd_workspace_bytes_1d(wg_plan plan, int64_t N, int64_t L, int64_t C, int64_t K, size_t* bytes);
wg_status winograd_conv1d(wg_plan plan, const wg_tensor* x, const wg_tensor* w, wg_tensor* y, hipStream_t stream);

/* ---- Stage entry points (each launches one kernel of winograd_conv2d) ----
 * Intermediate layouts, with Cp = C rounded up to a multiple of 8,
 * Kp = K rounded up to a multiple of 8, T = N * ceil(H/m) * ceil(W/m) tiles,
 * tile index t = (n * ceil(H/m) + ty) * ceil(W/m) + tx and Winograd-domain
 * index xi = i * alpha' + j:
 *   U [alpha'^2][K][Cp]  dtype, channels Cp > C are zero
 *   V [alpha'^2][T][Cp]  dtype, channels Cp > C are zero
 *   M [alpha'^2][T][Kp]  fp32 (columns K..Kp-1 hold unspecified values)   */

/* U[xi][k][c] = (G g_kc G^T)[i][j]: eq. (2)'s kernel transform. */
wg_status winograd_kernel_transform(wg_plan plan, const wg_tensor* w, void* U, hipStream_t stream);

/* V[xi][t][c] = (B^T d_tc B)[i][j]: eq. (2)'s input transform, on the
 * overlapping tiles of Section 2.3; d_tc is the (m+2)^2 window of channel c
 * whose top-left input pixel is (ty*m - 1, tx*m - 1); pixels outside x read 0.
 * x is [N][H][W][C] in the plan's dtype; V (caller-owned, 16-byte aligned)
 * is written in the layout above, its pad channels C..Cp-1 as zeros. */
wg_status winograd_input_transform(wg_plan plan, const wg_tensor* x, void* V, hipStream_t stream);

/* Both transforms above in one launch (the first kernel of winograd_conv2d):
 * U from w ([K][3][3][C]) and V from x ([N][H][W][C], same C), with the same
 * values as the two separate calls. */
wg_status winograd_kernel_input_transform(wg_plan plan, const wg_tensor* w, const wg_tensor* x, void* U, void* V,
                                          hipStream_t stream);

/* M[xi][t][k] = sum_c V[xi][t][c] U[xi][k][c]: alpha'^2 GEMMs [T x C][C x K]
 * on the matrix cores with fp32 accumulation (the Hadamard product of eq. (2)
 * summed over input channels), in the plan's channel-sum order.  The kernels address 128 rows of V or U with
 * 32-bit offsets: a channel row (Cp storage elements) of 33,553,920 bytes
 * (just under 32 MiB) or more, or
 * more than 2^31 - 1 blocks of 128 x 128, fails with WG_ERR_HIP ("invalid
 * argument") before anything is launched. */
wg_status winograd_contract(wg_plan plan, const void* V, const void* U, float* M, int64_t T,
                            int64_t C, int64_t K, hipStream_t stream);

/* y[n][ty*m+o][tx*m+p][k] = (A^T M_tk A)[o][p]: eq. (2)'s output transform
 * of the fp32 M above, rounded once to the plan's dtype and stored only
 * inside H x W (y gives N, H, W and K).  M and y are caller-owned. */
wg_status winograd_output_transform(wg_plan plan, const float* M, wg_tensor* y, hipStream_t stream);

/* The fused path's kernel: y = output transform of the contraction of V and U
 * (the two calls above) without M in memory; C is the input channel count
 * (V and U rows hold Cp channels), y gives N, H, W and K.  WG_ERR_UNSUPPORTED
 * for input tiles over 8 or per-plane sizes of V or U of 4 GiB or more. */
wg_status winograd_contract_output(wg_plan plan, const void* V, const void* U, int64_t C, wg_tensor* y,
                                   hipStream_t stream);

/* The fused kernel with the input transform in its prologue: y from x
 * ([N][H][W][C]) and U, with V computed per block in LDS (the same values as
 * winograd_input_transform) and never written to memory: the second kernel
 * of winograd_conv2d on WG_PATH_FUSED_INPUT.  WG_ERR_UNSUPPORTED where that
 * path is not available. */
wg_status winograd_input_contract_output(wg_plan plan, const wg_tensor* x, const void* U, wg_tensor* y,
                                         hipStream_t stream);

/* ---- Around the layer (not part of eq. (2)) ------------------------------ */

/* y = ReLU(x) (pool == 0, y shaped like x) or y = 2x2 stride-2 max-pooling
 * of ReLU(x) (pool == 1, y [N][H/2][W/2][C], odd last rows and columns
 * dropped): the operations between the convolutions of the VGG-16 network of
 * Section 3.2.  x and y are NHWC in dtype, 16-byte aligned, and must not
 * overlap (an empty pooled y, from H or W equal to 1, may have a null data
 * pointer: nothing is launched); ReLU maps NaN and -0 to +0.  Asynchronous
 * on stream. */
wg_status winograd_relu_pool(wg_dtype dtype, const wg_tensor* x, wg_tensor* y, int pool, hipStream_t stream);

/* Direct convolution in float64, the reference of the error studies of
 * Section 3.1: y[n][h][v][k] = sum w[k][i][j][c] x[n][h+i-1][v+j-1][c] over the
 * 3x3 taps (w->h == 3, zero padding 1), or, with w->h == 1, the 1D
 * convolution y[n][h][v][k] = sum_j,c w[k][0][j][c] x[n][h][v+j-1][c] of each
 * row (zero padding 1 along W).  x [N][H][W][C] and w [K][w->h][3][C] are in
 * dtype (each value is widened exactly); y [N][H][W][K] is float64, 8-byte
 * aligned, caller-owned.  Asynchronous on stream. */
wg_status winograd_direct_conv_f64(wg_dtype dtype, const wg_tensor* x, const wg_tensor* w, double* y,
                                   hipStream_t stream);

/* Doubles of the sums buffer of winograd_sq_error_sums. */
#define WG_SQ_SUMS_DOUBLES 514

/* sums[0] = sum_i (y[i] - ref[i])^2 and sums[1] = sum_i ref[i]^2 over n
 * values, in float64, in a fixed order (the same bits on every run), so that
 * sqrt(sums[0] / sums[1]) is the relative L2 error of y (dtype) against the
 * float64 reference.  sums (device, WG_SQ_SUMS_DOUBLES doubles, 8-byte
 * aligned) also holds the per-block partial sums.  Asynchronous on stream. */
wg_status winograd_sq_error_sums(wg_dtype dtype, const void* y, const double* ref, int64_t n, double* sums,
                                 hipStream_t stream);

/* Message describing the last error of the calling thread ("" if none). */
const char* winograd_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* WINOGRAD_CRT_H */
