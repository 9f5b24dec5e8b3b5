/*
 * wino.h -- C ABI of libwino, an N-dimensional Winograd correlation forward
 * F(m^N, r^N) for 2-D and 3-D ConvNet layers on AMD MI355X (gfx950), with
 * the layer's data and weight gradients on the same transforms.
 *
 * Method: Budden et al., "Deep Tensor Convolution on Multicores" (arXiv
 * 1611.06565).  The layer is eq. (2) of §3.1: for every sample n, kernel k and
 * output position o,
 *
 *     y[n][k][o] = f( b[k] + sum_c sum_{p in [0,r)^N} w[k][c][p] * x~[n][c][o + p - pad] )
 *
 * a cross-correlation (no kernel flip) with f = identity, ReLU or leaky ReLU, b = 0 unless
 * given (wino_forward_ex) and x~ equal to x zero-extended outside [0, X).
 * Sizes (N, m, r): F(2,3) and F(4,3) in 2-D and 3-D; F(3,2), F(5,4), F(4,5)
 * and F(3,6) (Table 1) in 2-D.  It is computed by eq. (4),
 *
 *     S = [ (g x_n G) (.) (d x_n B^T) ] x_n A^T      over each axis n,
 *
 * on overlapping alpha^N input tiles stepping by m (§3.3, alpha = m + r - 1),
 * with the element-wise product and the channel sum fused into one matrix
 * product per transformed element xi (eq. 5 of §4.1):
 *
 *     M_xi [T x K] = V_xi [T x C] . U_xi [C x K],   xi in [0, alpha^N).
 *
 * Conventions for every entry point
 * ---------------------------------
 * - Tensors are dense, C-order, float32, with the shapes given below.  Device
 *   pointers are allocated and owned by the caller and must be 16-byte
 *   aligned.  The library never allocates device memory.
 * - "stream" is a hipStream_t passed as void*; NULL means the null stream.
 *   Device work is enqueued asynchronously on it; the call returns once the
 *   launches are enqueued and the caller synchronises.
 * - Argument and shape errors are reported synchronously with a negative
 *   wino_status and leave every buffer untouched.  Launch failures return
 *   WINO_EDEVICE.  Nothing aborts or throws across the ABI.
 * - A plan is immutable after wino_plan returns; it may be used from several
 *   host threads and streams at once provided each call gets its own
 *   workspace and output buffers.
 */
#ifndef WINO_H_
#define WINO_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WINO_OK = 0,
  WINO_EINVAL = -1,        /* bad argument, shape, pointer or alignment           */
  WINO_EUNSUPPORTED = -2,  /* (N, m, r) has no kernel instantiation                */
  WINO_EWORKSPACE = -3,    /* workspace smaller than wino_workspace_bytes          */
  WINO_EDEVICE = -4        /* a HIP launch or query failed                         */
} wino_status;

typedef struct wino_plan_s wino_plan_t; /* opaque, immutable after creation */

/* The activation f of eq. (2) (§3.1: a ReLU or another non-linear
 * activation), applied to every output in the output-transform epilogue,
 * after the bias.  At most one of the two may be set.
 *   WINO_RELU        f(v) = max(0, v)
 *   WINO_LEAKY_RELU  f(v) = v for v > 0, slope * v otherwise
 *                    (slope = wino_opts.slope, finite) */
#define WINO_RELU 1u
#define WINO_LEAKY_RELU 4u
/* Never split the channel-element passes of a product block over several
 * work-groups (no partials scratch in the workspace; see
 * wino_workspace_bytes). */
#define WINO_NO_SPLIT 2u
/* Keep the forward of an F(4^3, 3^3) layer with at most 64 kernels in two
 * stages (input transform to the workspace, then the product) instead of
 * fusing the input transform into the product (see wino_forward). */
#define WINO_NO_FUSE 8u

typedef struct {
  /* Symmetric zero padding per spatial axis, outer to inner.  0 is the
   * paper's unpadded correlation with S = D - G + 1 outputs per axis (§2.2). */
  int32_t pad[3];
  /* alpha-1 distinct finite interpolation points (the point at infinity is
   * implied), or NULL for the default set of (m, r).  Each point must be a
   * rational with denominator below 2^20 whose nearest double is the value
   * passed (1/3 may be passed as 1.0/3.0).  §2.2: the polynomial m(x) built
   * from these points is the only input of transform synthesis. */
  const double* points;
  int32_t n_points;
  uint32_t flags; /* WINO_RELU or WINO_LEAKY_RELU, | WINO_NO_SPLIT | WINO_NO_FUSE; or 0 */
  float slope;    /* WINO_LEAKY_RELU: the slope below zero; ignored otherwise */
  /* Per-axis output tiles: eq. (4) lets every axis n carry its own transform
   * triple (C_n, B_n, A_n).  tile[i] = 0 keeps m; a non-zero entry sets axis
   * i's tile extent m_i, with F(m_i, r)'s matrices on that axis (equal
   * extents on every axis make an ordinary plan of that m).  Compiled
   * mixed tiles: N = 3, r = 3, m_0 != m_1 = m_2 with {m_0, m_1} = {2, 4}
   * (e.g. {2, 4, 4}: 2 on a short first axis, 4 on the others); each axis
   * uses its F(m, r)'s default points (points must be NULL).  Entries past N
   * must be 0. */
  int32_t tile[3];
} wino_opts;

/* Plan summary (host-side numbers only). */
typedef struct {
  int32_t N, m, r, alpha; /* alpha = m + r - 1; 0 when the axes' tiles differ    */
  int32_t n_xi;          /* transformed elements per tile: prod of alpha_axis     */
  int32_t C, K;
  int32_t C_pad, K_pad;  /* C and K rounded up to the GEMM step / block           */
  int64_t batch;
  int64_t X[3], Y[3];    /* input and output extents per axis (unused axes 1)     */
  int64_t tiles[3];      /* ceil(Y_i / m) tiles per axis                          */
  int64_t T, T_pad;      /* tiles over the whole batch, and rounded to the block  */
  int32_t block_tiles;   /* GEMM rows per work-group                             */
  int32_t block_kernels; /* GEMM columns per work-group                          */
  int32_t default_points;/* 1 when the transform constants are compiled in        */
  int32_t channel_group; /* CG: channels interleaved innermost in V                 */
  int32_t filter_channel_group; /* CGU: channels interleaved innermost in U        */
  int32_t gemm_parts;    /* parts each tail block of the product is split into   */
  int64_t gemm_tail_blocks; /* product blocks split into gemm_parts parts         */
  int32_t fused;         /* 1: wino_forward fuses the input transform into the product */
  int32_t tile[3];       /* output-tile extent per axis (1 past N)                */
  int32_t alpha_axis[3]; /* input-tile extent per axis, tile + r - 1 (1 past N)   */
} wino_plan_desc;

/* Build a plan for one layer.  §3.1-§3.3 and §4.1.
 *   N      number of spatial axes: 2 or 3
 *   m, r   output-tile and kernel extent per axis; supported (m, r) pairs are
 *          (2, 3) and (4, 3) for N = 2 and 3 (alpha = 4 or 6), and (3, 2),
 *          (5, 4), (4, 5), (3, 6) for N = 2 (alpha = 4 or 8); others give
 *          WINO_EUNSUPPORTED
 *   C, K   input channels and kernels, each in [1, 2^20]
 *   dims   [batch, X_1 .. X_N], each in [1, 2^31 - 1]; the output extent per
 *          axis Y_i = X_i + 2 pad_i - r + 1 must be >= 1
 *   opts   may be NULL (no padding, default points, no activation); pads in
 *          [0, 2^20]
 *   out    receives the plan; unchanged on error
 * Returns WINO_EINVAL for bad arguments and for layers whose tile count
 * (batch x tiles over every axis), padded sizes, byte counts or launch grids
 * do not fit the library's integer ranges (all computed in 64 bits with
 * overflow checks before any narrowing).
 * Generates A^T (m x alpha), B^T (alpha x alpha) and G (alpha x r) in exact
 * rational arithmetic and rounds each entry once to float32.  No device work;
 * the compute-unit count of the current device is read to size the product's
 * tail split (see wino_workspace_bytes). */
wino_status wino_plan(int N, int m, int r, int C, int K, const int64_t* dims,
                      const wino_opts* opts, wino_plan_t** out);

/* Free a plan's host memory (NULL is a no-op).  The plan must not be in use
 * by a call in progress; device buffers stay the caller's. */
void wino_destroy(wino_plan_t* plan);

/* Fill *desc from the plan (the numbers of §3.3's tiling and §4.1's products).
 * Returns WINO_EINVAL for NULL arguments. */
wino_status wino_plan_describe(const wino_plan_t* plan, wino_plan_desc* desc);

/* Bytes of the transformed-filter buffer U (float32): the alpha^N transformed
 * elements of every (kernel, channel) pair, the kernel side of eq. (4)
 * (§3.3 caches it across forwards), laid out as
 * U[alpha^N][C_pad/CGU][K_pad][CGU] with CGU = filter_channel_group: element
 * (xi, c, k) sits at ((xi*C_pad/CGU + c/CGU)*K_pad + k)*CGU + c%CGU.
 * Padding channels and kernels are zero. */
size_t wino_filter_bytes(const wino_plan_t* plan);

/* Bytes of workspace wino_forward needs.  It starts with the transformed
 * input V (float32): the data side of eq. (4), one alpha^N tile per (tile,
 * channel) with tiles of alpha values stepping by m along each axis (§3.3),
 * stored as the [T x C] operands of eq. (5) (§4.1), tile-block major as
 * V[T_pad/B][C_pad/CG][alpha^N][B][CG] with B = block_tiles: element
 * (xi, c, t) sits at (((t/B)*C_pad/CG + c/CG)*alpha^N + xi)*B*CG + (t%B)*CG
 * + c%CG.  For F(2^N, 3^N) and F(4^2, 3^2) the product's blocks (64 tiles x 64
 * or 32 kernels) that would run in a last, partly filled round of resident
 * work-groups on the device current at wino_plan (gemm_tail_blocks) are split
 * by element passes into gemm_parts work-groups each, and a scratch area for
 * their partial outputs follows V (at V's size rounded up to 256 bytes);
 * wino_gemm_inverse overwrites it.
 * The split is fixed when the plan is made and the partials are summed in a
 * fixed order, so a plan's results are bitwise reproducible. */
size_t wino_workspace_bytes(const wino_plan_t* plan);

/* Bytes of workspace wino_forward (and wino_forward_ex) needs: 0 when the
 * plan fuses the input transform into the product (desc.fused: F(4^3, 3^3)
 * with at most 64 kernels, unless WINO_NO_FUSE), wino_workspace_bytes
 * otherwise.  The two-stage calls (wino_transform_input, wino_gemm_inverse)
 * always need wino_workspace_bytes. */
size_t wino_forward_workspace_bytes(const wino_plan_t* plan);

/* out[0..N+1] = [batch, K, Y_1 .. Y_N]: the output extent of the valid
 * correlation S = D - G + 1 per axis (§2.2), on the zero-padded input,
 * Y_i = X_i + 2 pad_i - r + 1.  WINO_EINVAL for NULL arguments. */
wino_status wino_output_dims(const wino_plan_t* plan, int64_t* out);

/* Test hook: copy the transform matrices of Theorem 1 / Algorithm 1 (§2.1-§2.2;
 * the paper's A, B and C of eq. (1)), each entry the exact rational rounded
 * once to the nearest double, row-major: AT [m][alpha], BT [alpha][alpha],
 * G [alpha][r].  Any pointer may be NULL; WINO_EINVAL for a NULL plan,
 * WINO_EUNSUPPORTED for a plan with per-axis tiles (one triple per axis). */
wino_status wino_get_matrices(const wino_plan_t* plan, double* AT, double* BT, double* G);

/* Kernel transform U = g x_1 G ... x_N G for every (k, c) (eq. 4; §3.3 caches
 * it across forwards).
 *   w  device, [K][C][r^N] float32
 *   U  device, wino_filter_bytes(plan) bytes, fully overwritten */
wino_status wino_transform_filter(const wino_plan_t* plan, const float* w, float* U, void* stream);

/* Data gradient (the adjoint of eq. 2's correlation; the backward pass of a
 * layer, which the paper leaves out).  For a forward plan with C channels, K
 * kernels, input extents X and padding pad <= r - 1 on every axis,
 *
 *     dx[n][c][q] = sum_k sum_{p in [0,r)^N} w[k][c][p] * dy~[n][k][q - p + pad]
 *
 * (dy~ = dy zero-extended outside [0, Y)) is itself a correlation: of dy with
 * the kernel w'[c][k][p] = w[k][c][r-1-p] (every axis reversed) and padding
 * r - 1 - pad, with output extent X.  So it runs on the forward path:
 *
 *   wino_plan_adjoint(fwd, &adj)              adjoint plan: C and K swapped,
 *                                             dims [batch, Y_1..Y_N], pads
 *                                             r - 1 - pad, the same points and
 *                                             WINO_NO_SPLIT, no ReLU
 *   wino_transform_filter_adjoint(adj, w, U)  U of w' from the forward kernels
 *                                             w [K][C][r^N] (the plan's
 *                                             [C_adj][K_adj][r^N])
 *   wino_forward(adj, dy, U, dx, ...)         dy [batch][K][Y..] -> dx
 *                                             [batch][C][X..]
 *
 * A ReLU of the forward layer is not part of the adjoint: mask dy first.
 * wino_plan_adjoint returns WINO_EINVAL when a pad exceeds r - 1 and the
 * errors of wino_plan otherwise; wino_transform_filter_adjoint behaves as
 * wino_transform_filter (U fully overwritten). */
wino_status wino_plan_adjoint(const wino_plan_t* forward_plan, wino_plan_t** out);
wino_status wino_transform_filter_adjoint(const wino_plan_t* plan, const float* w, float* U, void* stream);

/* Weight gradient (the backward pass on the kernel side, which the paper also
 * leaves out) of the layer of a forward plan:
 *
 *     dw[k][c][p] = sum_n sum_o dy[n][k][o] * x~[n][c][o + p - pad]
 *
 * Per axis the r taps' gradient over one output tile is the minimal filtering
 * algorithm F(r, m) (§2.2) with the tile's m output gradients as its kernel
 * and the tile's alpha-value input window as its data; its data transform is
 * the forward's B^T (same points), so the forward's V is reused, the
 * output gradients are transformed with F(r, m)'s G, one product per element
 * xi sums over every tile of the batch (M_xi[K x C] = sum_t D_xi V_xi^T,
 * eq. 5 read the other way) and F(r, m)'s A^T maps M back to r^N taps.
 * Supported for every size (WINO_EUNSUPPORTED and a workspace size of 0 only
 * if F(r, m)'s data transform differed from the forward's, or for grids past
 * 32-bit counts).  Bias, ReLU and the plan's flags play no part (mask dy for
 * a ReLU layer first).
 *   x          device, [batch][C][X_1..X_N] float32 (the layer's input)
 *   dy         device, [batch][K][Y_1..Y_N] float32 (the output gradient)
 *   dw         device, [K][C][r^N] float32, fully overwritten
 *   workspace  device, wino_weight_gradient_workspace_bytes(plan) bytes: V,
 *              then the transformed dy and the partial products of the
 *              tile ranges (all overwritten)
 * The partial products are summed in a fixed order: results are bitwise
 * reproducible for a plan. */
size_t wino_weight_gradient_workspace_bytes(const wino_plan_t* plan);
wino_status wino_weight_gradient(const wino_plan_t* plan, const float* x, const float* dy, float* dw,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* Data transform V = d x_1 B^T ... x_N B^T of every tile and channel (eq. 4),
 * written straight into the GEMM operand layout above (§4.1's reshuffle).
 *   x          device, [batch][C][X_1..X_N] float32
 *   workspace  device, at least wino_workspace_bytes(plan) bytes */
wino_status wino_transform_input(const wino_plan_t* plan, const float* x, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* Batched product M_xi = V_xi . U_xi over all xi (eq. 5) with the inverse
 * transform S = M x_n A^T, tile stitching, cropping and the optional ReLU
 * fused into its epilogue (eq. 4).  Reads the V part of the workspace written
 * by wino_transform_input (and may overwrite the scratch area after it).
 *   y  device, [batch][K][Y_1..Y_N] float32, fully overwritten */
wino_status wino_gemm_inverse(const wino_plan_t* plan, void* workspace, size_t workspace_bytes,
                              const float* U, float* y, void* stream);

/* The whole forward (eq. 4 with eq. 5) on one stream, with
 * wino_forward_workspace_bytes(plan) bytes of workspace (workspace may be
 * NULL when that is 0).  Two-stage plans run wino_transform_input and then
 * wino_gemm_inverse; fused plans (F(4^3, 3^3), at most 64 kernels) form
 * each tile block's transformed input in LDS inside the product, 8 channels
 * at a time, so V never reaches memory (§4.1's reshuffle and §4.3's
 * cache-sized tile blocks, on the GPU). */
wino_status wino_forward(const wino_plan_t* plan, const float* x, const float* U, float* y,
                         void* workspace, size_t workspace_bytes, void* stream);

/* wino_gemm_inverse and wino_forward with the per-kernel bias b of eq. (2)
 * (§3.1): y[n][k][...] = f(sum + bias[k]), f the plan's activation.
 *   bias  device, [K] float32, 4-byte aligned, read only; NULL = no bias
 *         (then identical to the calls above).
 * Errors as for the calls above; a misaligned bias is WINO_EINVAL. */
wino_status wino_gemm_inverse_ex(const wino_plan_t* plan, void* workspace, size_t workspace_bytes,
                                 const float* U, const float* bias, float* y, void* stream);
wino_status wino_forward_ex(const wino_plan_t* plan, const float* x, const float* U, const float* bias,
                            float* y, void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * wino_forward_ex without a workspace argument.  The workspace is a static
 * device array of WINO_NOALLOC_SCRATCH_BYTES inside the library, one per GPU
 * the library runs on, held until the process ends; its device address is
 * looked up once per device on the first call with that device current.
 * The call allocates nothing.  Plans whose wino_forward_workspace_bytes
 * exceeds WINO_NOALLOC_SCRATCH_BYTES get WINO_EWORKSPACE.  Every call on a GPU
 * shares that GPU's array: calls that overlap in time on one GPU (different
 * streams, or host threads without ordering) race and give wrong results;
 * calls on one stream are ordered and safe.  Other arguments and errors as
 * wino_forward_ex. */
#define WINO_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
wino_status wino_forward_noalloc(const wino_plan_t* plan, const float* x, const float* U, const float* bias,
                                 float* y, void* stream);

/* Max-pool with window = stride and floor rounding over the trailing 3 axes
 * of x [lead][X_1][X_2][X_3] -> y [lead][X_1/p_1][X_2/p_2][X_3/p_3]
 * (the C3D stack's pooling layers; not part of the Winograd method).
 *   dims    [lead, X_1, X_2, X_3], window [p_1, p_2, p_3], each >= 1 */
wino_status wino_maxpool3d(const int64_t* dims, const int32_t* window, const float* x, float* y,
                           void* stream);

/* wino_forward_ex followed by wino_maxpool3d, with the pooling inside the
 * product's epilogue, so only the pooled outputs reach memory: F(4^3)
 * plans, fused (wino_plan_info.fused = 1, no workspace) or in two stages
 * (the input transform to the workspace, then the product), and F(2^3)
 * plans with window (2, 2, 2) (a window is one tile).  eq. (2)'s f
 * (the plan's activation) is applied before the maximum, as a pooling layer
 * after the convolution does; the result has the same bits as
 * wino_forward_ex then wino_maxpool3d.
 *   window     host, [3] int32: (1, 2, 2) or (2, 2, 2) (F(2^3): (2, 2, 2)),
 *              window = stride, floor rounding
 *   y          device, [batch][K][Y_1/w_1][Y_2/w_2][Y_3/w_3] float32,
 *              16-byte aligned (Y of wino_output_dims)
 *   bias       as for wino_forward_ex
 *   workspace  as for wino_forward_ex: wino_forward_workspace_bytes(plan)
 *              bytes (0 and NULL for a fused plan)
 * Errors: WINO_EINVAL for null or misaligned pointers, a window entry below
 * 1 or a pooled extent of 0; WINO_EWORKSPACE for a short workspace;
 * WINO_EUNSUPPORTED for other windows and for other sizes (pool those with
 * wino_maxpool3d). */
wino_status wino_forward_pool(const wino_plan_t* plan, const float* x, const float* U, const float* bias,
                              const int32_t* window, float* y, void* workspace, size_t workspace_bytes,
                              void* stream);

/* Accuracy of a point set (§2.2, §3.3: the points trade fp32 accuracy).
 * wino_points_error_growth: kappa = kappa_1^N, where kappa_1 is the largest
 * over outputs i of sum_xi |A^T[i][xi]| |G[xi,:]|_1 |B^T[xi,:]|_1 / r, the
 * first-order bound on the rounding error of the 1-D algorithm relative to the
 * direct sum's magnitude for inputs of magnitude <= 1 (the N-D transforms are
 * products over the axes).  Computed on the host from the exact rational
 * matrices of Theorem 1 / Algorithm 1.
 *   points  the alpha - 1 finite points (infinity implied), or NULL for the
 *           default set; n_points = m + r - 2 when given
 *   growth  out: kappa
 * wino_search_points: the symmetric set {0 (if m + r - 2 is odd), +-p_1,
 * +-p_2, ...} with p_i from {1, 2, 1/2, 3, 1/3, 3/2, 2/3, 4, 1/4} that
 * minimises kappa (ties: earlier in that order); points[m + r - 2] and growth
 * are written.  Host only, no device work; WINO_EINVAL for bad sizes or
 * points (coincident, or not small rationals). */
wino_status wino_points_error_growth(int N, int m, int r, const double* points, int n_points,
                                     double* growth);
wino_status wino_search_points(int N, int m, int r, double* points, double* growth);

/* A static, NUL-terminated description of a status code ("unknown status"
 * for values outside wino_status); never NULL. */
const char* wino_status_string(wino_status s);

#ifdef __cplusplus
}
#endif

#endif /* WINO_H_ */
