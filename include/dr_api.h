/*
 * dr_api.h -- C ABI of the MI355X (gfx950) library for the data-parallel hot
 * path of Dr. Post-Training (arXiv 2605.07063): per-example gradient
 * sketches of linear layers, their Gram matrix and target scores, and the
 * projection of the mean target direction onto a feasible set induced by
 * the general-data gradients (span, cone, or top-k subset).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pointers are DEVICE pointers unless marked (host).  Matrices are
 *   row-major; a leading dimension is counted in elements.
 * - The caller owns every buffer, including the workspace whose size the
 *   matching *_workspace_size query returns.  The library allocates no
 *   device memory and keeps no data between calls.  The one runtime object
 *   it keeps: dr_project_span with n > 256 runs its look-ahead on two
 *   auxiliary streams (default priority) and five events per device,
 *   created by the first such call on that device and kept until the
 *   process ends.
 * - `stream` is a hipStream_t (NULL = the default stream).  Calls only
 *   enqueue work.  The returned dr_status covers argument validation and
 *   launch errors; every argument is validated before the first HIP call,
 *   so validation errors are reported even on a host without a GPU.
 * - Numerical outcomes are written to a device int32 array `info[P]`
 *   (one entry per group), LAPACK style: 0 = ok, j > 0 = the j-th pivot
 *   (1-based) of a Cholesky factorisation was not positive,
 *   DR_INFO_NOT_CONVERGED (-2) = iteration budget exhausted before the
 *   requested tolerance, DR_INFO_NONFINITE (-3) = NaN in the input.
 *   Read it after synchronising the stream.
 * - Outputs must not alias inputs.  Results are deterministic: identical
 *   inputs on the same device give bitwise identical outputs (no
 *   floating-point atomics anywhere).
 * - Two calls that share a workspace buffer must be ordered (same stream
 *   or synchronised); calls on different streams with separate workspaces
 *   may overlap.
 *
 * Notation: N = n + m rows of a merged batch (n general examples followed
 * by m target examples, one forward/backward pass over both -- Sec. 4.2,
 * "merging training and target batch"); T = padded sequence length;
 * len[i] = valid tokens of example i; a linear layer has weight
 * W in R^{d_out x d_in}, input activations x (= a) and output gradients
 * dy = dL/de (Sec. 4.1).
 */
#ifndef DR_API_H
#define DR_API_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DR_ABI_VERSION 1

typedef enum {
  DR_OK = 0,
  DR_ERR_ARG = 1,           /* invalid size, pointer, stride or alignment */
  DR_ERR_DTYPE = 2,         /* unsupported dtype */
  DR_ERR_NOT_SPD = 3,       /* reserved for callers that map info > 0 */
  DR_ERR_NOT_CONVERGED = 4, /* reserved for callers that map info == -2 */
  DR_ERR_NONFINITE = 5,     /* reserved for callers that map info == -3 */
  DR_ERR_WORKSPACE = 6,     /* workspace pointer NULL or smaller than the query */
  DR_ERR_HIP = 7,           /* a HIP launch failed */
  DR_ERR_UNSUPPORTED = 8,   /* valid but not implemented (e.g. projection size) */
  DR_ERR_TOO_LARGE = 9      /* needs more scratch than a no-allocation entry point holds */
} dr_status;

#define DR_INFO_NOT_CONVERGED (-2)
#define DR_INFO_NONFINITE (-3)

typedef enum { DR_F32 = 0, DR_BF16 = 1 } dr_dtype;

typedef enum { DR_SCORE_DIRECT = 0, DR_SCORE_GIP = 1, DR_SCORE_PIP = 2 } dr_score_method;

typedef enum {
  DR_RIDGE_ABS = 0,       /* lam_eff = lambda */
  DR_RIDGE_REL_TRACE = 1  /* lam_eff = lambda * trace(K_p) / n */
} dr_ridge_mode;

/* One linear layer's retained pair (x, dy) and its two Gaussian
 * projectors (host struct; the pointers inside are device pointers).
 *   x     [N][T][ldx]   layer inputs, ldx >= d_in; example stride T*ldx
 *   dy    [N][T][lddy]  output gradients, lddy >= d_out
 *   p_in  [k_in][d_in]  dense, same dtype as x
 *   p_out [k_out][d_out]
 *   col_offset: first column of this layer's k_out*k_in block in S. */
typedef struct {
  const void* x;
  int64_t ldx;
  const void* dy;
  int64_t lddy;
  const void* p_in;
  const void* p_out;
  int64_t d_in, d_out, k_in, k_out;
  int64_t col_offset;
} dr_layer;

int dr_abi_version(void);
const char* dr_status_string(dr_status s);

/* ---------------------------------------------------------------------------
 * dr_sketch_grads -- factorised per-example gradient sketches.
 *
 * Computes, for every example i < N and layer l,
 *   S[i][col_offset_l + a*k_in + b] =
 *       sum_{t < len[i]} (P_out dy_{i,t})[a] * (P_in x_{i,t})[b],
 * i.e. P_out G_i P_in^T with G_i = sum_t dy_{i,t} x_{i,t}^T the per-sample
 * weight gradient (Sec. 4.1 "Backward pass"; compressed as in App. C.3,
 * "Factorized Projection" forward form and "Per-Sample Gradient
 * Compression", with the second-stage projector taken as the identity).
 * G_i is never formed.  Tokens t >= len[i] are padding: they are never
 * read, so padding may hold any bits (NaN included).
 *
 * Arithmetic: DR_BF16 inputs are contracted on bf16 MFMA with fp32
 * accumulation; the second (token) contraction splits each fp32 stage-1
 * value into bf16 hi + lo parts and sums Dh Yh + Dh Yl + Dl Yh on bf16
 * MFMA with fp32 accumulation (about 3 * 2^-16 relative error per
 * product, far inside the bf16 inputs' own rounding).  DR_F32 inputs use
 * fp32 MFMA throughout.
 *
 * Arguments
 *   layers      (host) array of num_layers descriptors, 1 <= num_layers.
 *   N, T        examples and padded length, N >= 0, T >= 0.
 *   len         device int32 [N] with 0 <= len[i] <= T, or NULL (= all T).
 *               Values outside [0, T] are clamped.
 *   dtype       DR_BF16 or DR_F32 (x, dy, p_in, p_out all share it).
 *   S, ldS      fp32 output [N][ldS]; every block of every row is written
 *               (zeros for len[i] = 0).  Columns outside the layers'
 *               blocks are not touched.
 *   workspace   device buffer of at least dr_sketch_workspace_size() bytes
 *               (may be NULL when that size is 0).
 * Requirements (else DR_ERR_ARG): k_in, k_out in {16, 32, 64};
 *   d_in, d_out >= 1 and multiples of 8 (bf16) or 4 (f32); ldx, lddy
 *   multiples of the same; x, dy, p_in, p_out 16-byte aligned; blocks
 *   within ldS.
 * ------------------------------------------------------------------------- */
dr_status dr_sketch_grads(const dr_layer* layers, int num_layers, int64_t N, int64_t T,
                          const int32_t* len, dr_dtype dtype, float* S, int64_t ldS,
                          void* workspace, size_t ws_bytes, void* stream);
size_t dr_sketch_workspace_size(const dr_layer* layers, int num_layers, int64_t N, int64_t T,
                                dr_dtype dtype);

/* ---------------------------------------------------------------------------
 * dr_gram -- target mean, Gram matrix and scores per parameter group.
 *
 * For each group p (columns [goff[p], goff[p+1]) of the sketch matrix):
 *   gbar_p = (1/m) sum_j Gt[j][cols_p]       mean target gradient (Sec. 3.2)
 *   K_p    = G_p G_p^T                        all <g_i, g_i'> (the
 *                                             redundancy term, Sec. 3.3.2)
 *   s_p    = G_p gbar_p                       alignment scores (Sec. 3.3.2;
 *                                             group-wise form, Sec. 3.3.3)
 *   t2_p   = ||gbar_p||^2
 * Arguments
 *   G [n][ldG], Gt [m][ldGt]  general and target sketches (dtype DR_F32 or
 *                             DR_BF16), n >= 0, m >= 1, ld >= goff[P].
 *   goff  (host) int64 [P+1], 0 <= goff[0] <= ... <= goff[P], P >= 1.
 *   K     fp32 [P][n][n], both triangles written.  s fp32 [P][n].  t2 fp32 [P].
 * Arithmetic: fp32 inputs -> fp32 MFMA products with fp32 accumulation;
 * bf16 inputs -> bf16 MFMA with fp32 accumulation.
 * Requirements: ldG, ldGt and every goff[p] multiples of 4 (f32) or 8 (bf16);
 * G and Gt 16-byte aligned.
 * ------------------------------------------------------------------------- */
dr_status dr_gram(const void* G, int64_t n, int64_t ldG, const void* Gt, int64_t m, int64_t ldGt,
                  dr_dtype dtype, const int64_t* goff, int P, float* K, float* s, float* t2,
                  void* workspace, size_t ws_bytes, void* stream);
size_t dr_gram_workspace_size(int64_t n, int64_t m, const int64_t* goff, int P, dr_dtype dtype);

/* ---------------------------------------------------------------------------
 * dr_gram_noalloc -- dr_gram for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same computation, arguments and results as dr_gram, minus
 * the workspace.  Its workspace is a fixed array of DR_GRAM_NOALLOC_MAX_BYTES
 * in the library's device code, one per GPU, held until the process ends.
 * The call allocates nothing (no hipMalloc / hipFree, no allocating library
 * routine); its first call on a device looks up that device's array.
 *   Returns DR_ERR_TOO_LARGE, before any HIP call, when
 *   dr_gram_workspace_size(n, m, goff, P, dtype) > DR_GRAM_NOALLOC_MAX_BYTES
 *   (the largest workload shape here needs 36 MiB: 256 fp32 rows over
 *   229376 columns in 224 groups; 24 MiB as one group).
 * All calls on one GPU share its array (and it keeps the last call's
 * contents; nothing in it needs to start at zero): calls that overlap on one
 * GPU -- on different streams, or from different host threads without
 * ordering -- race.  Order them on one stream, or synchronise.
 * ------------------------------------------------------------------------- */
#define DR_GRAM_NOALLOC_MAX_BYTES ((size_t)64 << 20)
dr_status dr_gram_noalloc(const void* G, int64_t n, int64_t ldG, const void* Gt, int64_t m, int64_t ldGt,
                          dr_dtype dtype, const int64_t* goff, int P, float* K, float* s, float* t2,
                          void* stream);

/* ---------------------------------------------------------------------------
 * dr_project_span -- Eq. (proj) onto the span of the general gradients,
 * as ridge least squares:  (K_p + lam_eff_p I) w_p = s_p.
 *
 * u_p = G_p^T w_p (see dr_combine) minimises ||u - gbar_p||^2 +
 * lam_eff ||w||^2 over the span; lam_eff -> 0 recovers Eq. (proj).
 * lam_eff = lambda (DR_RIDGE_ABS) or lambda*trace(K_p)/n (DR_RIDGE_REL_TRACE).
 *   K [P][n][n] fp32 symmetric (lower triangle is read), s [P][n], t2 [P].
 *   w [P][n] out; lam_eff [P] out; resid2 [P] out = ||gbar_p - u_p||^2
 *   computed as t2 - 2 s.w + w.K.w; info [P] out.
 * Empty feasible set: n = 0 is a valid no-op beyond lam_eff = resid2 = t2,
 * info = 0; a group with trace(K) = 0 under REL_TRACE returns w = 0.
 * A factor pivot that is not positive sets info = its 1-based index and
 * w = 0.  Arithmetic: n <= 64 entirely in fp64 on the exact fp32 K; n > 64
 * an fp32 Cholesky factor and at most two steps of iterative refinement
 * with fp64 residuals of the fp32 K.  Refinement stops once the last two
 * corrections (the first solution counting as the first) estimate the
 * error left at about 1e-6 relative or less, so a well-conditioned group
 * takes one step.  When two steps do not get there (the corrections do not
 * shrink fast enough, which happens when cond(K + lam_eff I) * 2^-24 is not
 * small), info = DR_INFO_NOT_CONVERGED and w holds the last iterate.
 * ------------------------------------------------------------------------- */
dr_status dr_project_span(const float* K, const float* s, const float* t2, int64_t n, int P,
                          float lambda, dr_ridge_mode mode, float* w, float* lam_eff,
                          float* resid2, int32_t* info, void* workspace, size_t ws_bytes,
                          void* stream);
size_t dr_span_workspace_size(int64_t n, int P);

/* ---------------------------------------------------------------------------
 * dr_project_cone -- Eq. (proj) onto the convex cone of the general
 * gradients:  w_p = argmin_{w >= 0} 1/2 w^T K_p w - s_p^T w.
 *
 * Projected gradient on the Jacobi-scaled problem (K~ = D^-1/2 K D^-1/2,
 * D = diag K, start at 0, step 1/L with L the largest absolute row sum of
 * K~), iterated in fp64 on the fp32 K.  Stops after max_iter steps, or as
 * soon as the scaled KKT residual
 *   rho = max_i |min(w~_i, (K~ w~ - s~)_i)| / max_i |s~_i|
 * is <= kkt_tol (kkt_tol <= 0: run exactly max_iter steps).
 *   w [P][n] out; resid2 [P] out (as for the span); iters [P] out (steps
 *   taken); kkt [P] out (rho of the returned w); info [P] out
 *   (DR_INFO_NOT_CONVERGED if kkt_tol > 0 and rho > kkt_tol at the end).
 * Coordinates with K_ii = 0 get w_i = 0.  Supports n <= 256 (larger n:
 * DR_ERR_UNSUPPORTED); the whole problem runs in one workgroup per group.
 * ------------------------------------------------------------------------- */
dr_status dr_project_cone(const float* K, const float* s, const float* t2, int64_t n, int P,
                          int max_iter, float kkt_tol, float* w, float* resid2, int32_t* iters,
                          float* kkt, int32_t* info, void* workspace, size_t ws_bytes,
                          void* stream);
size_t dr_cone_workspace_size(int64_t n, int P);

/* ---------------------------------------------------------------------------
 * dr_project_simplex -- soft weighting (Sec. 6, "Designing New Feasible
 * Sets"): Eq. (proj) onto U_soft = { G^T w : w in the probability simplex },
 * i.e. w_p = argmin { w^T K_p w - 2 s_p^T w : w >= 0, sum_i w_i = 1 }.
 * Accelerated projected gradient (FISTA, step 1/L with L = 2 max_i
 * sum_j |K_ij|) from the best single vertex, each step projected exactly onto
 * the simplex; fp64 iterates on the fp32 K.  Stops after max_iter steps or
 * when the step residual max_i |w_i - y_i| (projected point minus the point
 * the gradient was taken at) is <= tol (tol <= 0: exactly max_iter steps).
 *   w [P][n] out (on the simplex); resid2 [P] out = t2 + w.K.w - 2 s.w;
 *   iters [P] out; res [P] out (the last step residual); info [P] out
 *   (DR_INFO_NOT_CONVERGED if tol > 0 was not reached, DR_INFO_NONFINITE on
 *   NaN / inf input).  n = 0: nothing to project onto (resid2 = t2).
 *   Supports n <= 256.
 * ------------------------------------------------------------------------- */
dr_status dr_project_simplex(const float* K, const float* s, const float* t2, int64_t n, int P, int max_iter,
                             float tol, float* w, float* resid2, int32_t* iters, float* res, int32_t* info,
                             void* stream);

/* ---------------------------------------------------------------------------
 * dr_back_project -- the transpose of the factorised compressor (App. C.3,
 * "Backward projection"), layer by layer: U + u_offset[l] (row-major
 * [d_out][d_in], fp32) = P_out^T X' P_in with X' the layer's block of the
 * sketch-space vector u (columns col_offset .. + k_out*k_in, read as
 * [k_out][k_in], the layout of dr_sketch_grads).  With u = dr_combine's
 * sketch-space update this is the parameter-space update of the MeSO
 * variant.  p_in / p_out have dtype `dtype`; x, dy are not used.
 * Requirements: 1 <= k_in, k_out <= 64; d_in a multiple of 4; U + u_offset[l]
 * 16-byte aligned; workspace of at least
 * dr_backproject_workspace_size() bytes (X' P_in of up to 16 layers, as
 * fp32 or as three bf16 planes).  bf16 projectors with d_in, d_out
 * multiples of 8 run P_out^T on bf16 MFMA over the three planes (exact to
 * fp32 rounding); otherwise fp32 FMA.
 * ------------------------------------------------------------------------- */
dr_status dr_back_project(const dr_layer* layers, int num_layers, dr_dtype dtype, const float* u, float* U,
                          const int64_t* u_offset, void* workspace, size_t ws_bytes, void* stream);
size_t dr_backproject_workspace_size(const dr_layer* layers, int num_layers);

/* ---------------------------------------------------------------------------
 * dr_select_topk -- the top-k rule of Sec. 3.3.2 (Select-S in the one-pass
 * algorithms of Sec. 4.2), per group.
 *
 * idx[p][0..k) = the k indices with the largest s[p][i], ties broken
 * toward the lowest index, written in ascending index order.  -0.0 equals
 * +0.0; +-inf order normally.  A NaN anywhere in s[p] sets info[p] = -3
 * and fills idx[p] with -1.  If w is not NULL, w[p][i] = 1/k on the
 * selected set and 0 elsewhere (u = G^T w is then the subset mean g_S).
 *   s [P][n] fp32, 0 <= k <= n, n <= 2^30 (else DR_ERR_UNSUPPORTED).
 *   idx int32 [P][k]; w fp32 [P][n] or NULL; info int32 [P].
 * ------------------------------------------------------------------------- */
dr_status dr_select_topk(const float* s, int64_t n, int P, int64_t k, int32_t* idx, float* w,
                         int32_t* info, void* stream);

/* ---------------------------------------------------------------------------
 * dr_select_threshold -- the thresholding rule of Sec. 3.3.2 (keep every
 * example whose score exceeds a fixed threshold: a subset of variable
 * size), per group.  inclusive = 0 keeps s[p][i] > tau; inclusive = 1 keeps
 * s[p][i] >= tau, so (tau = 0, inclusive = 1) is the negative score
 * filtering of the RL experiments of Sec. 5 (drop the negative scores).
 *   s [P][n] fp32; tau finite (else DR_ERR_ARG); n <= 2^30.
 *   idx   int32 [P][n] or NULL: the kept indices in ascending order, then -1.
 *   count int32 [P] (required): |S_p|.
 *   w     fp32 [P][n] or NULL: 1/|S_p| on the kept set, 0 elsewhere (u =
 *         G^T w is the subset mean g_S; all zero when nothing is kept).
 *   info  int32 [P]: 0, or DR_INFO_NONFINITE if s[p] holds a NaN (then
 *         count = 0, idx = -1, w = 0).
 * ------------------------------------------------------------------------- */
dr_status dr_select_threshold(const float* s, int64_t n, int P, float tau, int inclusive, int32_t* idx,
                              int32_t* count, float* w, int32_t* info, void* stream);

/* ---------------------------------------------------------------------------
 * dr_select_greedy -- the greedy construction of Sec. 3.3.2, per group:
 * starting from the empty set, k times add the example c whose addition
 * minimises the full subset objective
 *   f(S) = ||g_S||^2 - 2 <g_S, gbar> = (1/|S|^2) sum_{S x S} K - (2/|S|) sum_S s
 * (alignment and redundancy, the latter ignored by top-k), ties to the
 * lowest index.  f is evaluated in fp64 from the fp32 K and s.
 *   K [P][n][n] fp32 symmetric, s [P][n]; 0 <= k <= n <= 16384 (larger n:
 *   DR_ERR_UNSUPPORTED).
 *   idx int32 [P][k]: the chosen set in ascending index order.
 *   w   fp32 [P][n] or NULL: 1/k on the set, 0 elsewhere.
 *   info int32 [P]: 0, or DR_INFO_NONFINITE if K_p or s_p holds a NaN
 *   (then idx = -1, w = 0).
 *   workspace: at least dr_greedy_workspace_size(n, P) bytes.
 * ------------------------------------------------------------------------- */
dr_status dr_select_greedy(const float* K, const float* s, int64_t n, int P, int64_t k, int32_t* idx, float* w,
                           int32_t* info, void* workspace, size_t ws_bytes, void* stream);
size_t dr_greedy_workspace_size(int64_t n, int P);

/* ---------------------------------------------------------------------------
 * dr_combine -- the update direction in sketch space, u = G_p^T w_p per
 * group (the assembled update of Eq. (proj) for span and cone weights, or
 * the subset mean g_S for top-k weights).
 *   G [n][ldG] (DR_F32 or DR_BF16), w fp32 [P][n], u fp32 [goff[P]]
 *   (columns outside [goff[0], goff[P]) untouched).  fp64 accumulation.
 *   workspace: at least dr_combine_workspace_size() bytes (row-chunk
 *   partials in fp64; none for n <= 256, which runs in one pass).
 * ------------------------------------------------------------------------- */
dr_status dr_combine(const void* G, int64_t n, int64_t ldG, dr_dtype dtype, const int64_t* goff,
                     int P, const float* w, float* u, void* workspace, size_t ws_bytes,
                     void* stream);
size_t dr_combine_workspace_size(int64_t n, const int64_t* goff, int P);

/* ---------------------------------------------------------------------------
 * dr_assemble_update -- the update in full parameter space, assembled from
 * the retained pairs once the weights are known (Sec. 4.2: the post-hoc
 * assembly step of the Global Subset Update algorithm and the per-layer
 * assembly of the Layer-Wise Subset Update algorithm).  For every layer l
 *   U_l = sum_{i < n, w[g_l][i] != 0} w[g_l][i] * sum_{t < len[i]} dy_{i,t} x_{i,t}^T
 * a d_out x d_in matrix.  Top-k weights (1/k on S, dr_select_topk) give the
 * subset mean g_S of Sec. 3.3.2; span or cone weights give u = G^T w of
 * Eq. (proj) in parameter space.  Examples with weight 0 and padded tokens
 * t >= len[i] are never read (they may hold any bits, NaN included).
 *
 * Arithmetic: DR_BF16 inputs on bf16 MFMA with fp32 accumulation.  The
 * weighted examples of a layer are taken in |w|-ascending order into one
 * fp32 accumulator holding sum_e (w_e / w_cur) G_e, multiplied by
 * w_cur / w_next when the weight changes and by the last weight at the end
 * (every factor lies in [-1, 1]; equal weights cost nothing).  DR_F32
 * inputs on fp32 MFMA.
 *
 * Arguments
 *   layers      (host) num_layers descriptors; x, ldx, dy, lddy, d_in, d_out
 *               are used (p_in, p_out, k_*, col_offset are ignored).  The
 *               first n examples of x / dy are the weighted ones (target rows
 *               after them never enter).
 *   n, T        weighted examples and padded length, n >= 0, T >= 0.
 *   len         device int32 [n] (clamped to [0, T]) or NULL (= all T).
 *   dtype       DR_BF16 or DR_F32 (x and dy share it).
 *   w, P, ldw   device fp32 weights [P][ldw], P >= 1, ldw >= n.
 *   group_of_layer  (host) int32 [num_layers] in [0, P): the weight row of
 *               each layer (group-wise mode, Sec. 3.3.3), or NULL (= row 0).
 *   U, u_offset fp32 output; layer l's block is U + u_offset[l] (host int64),
 *               row-major [d_out][d_in].  Blocks must not overlap.  Every
 *               element of every block is written (zeros if no example has a
 *               non-zero weight).
 *   workspace   at least dr_update_workspace_size() bytes.
 * Requirements (else DR_ERR_ARG): d_in, d_out, ldx, lddy multiples of 8
 *   (bf16) or 4 (f32); x, dy 16-byte aligned.  One example's rows must span
 *   less than 4 GiB (T * ld * element size), else DR_ERR_UNSUPPORTED.
 * ------------------------------------------------------------------------- */
dr_status dr_assemble_update(const dr_layer* layers, int num_layers, int64_t n, int64_t T,
                             const int32_t* len, dr_dtype dtype, const float* w, int P, int64_t ldw,
                             const int32_t* group_of_layer, float* U, const int64_t* u_offset,
                             void* workspace, size_t ws_bytes, void* stream);
size_t dr_update_workspace_size(const dr_layer* layers, int num_layers, int64_t n, int64_t T,
                                dr_dtype dtype);

/* ---------------------------------------------------------------------------
 * dr_score_exact -- exact per-sample scores of every layer (Sec. 4.3),
 *   s[l][i] = <gbar*_l, G_i^(l)>,   gbar*_l = (1/m) sum_j G*_j^(l),
 * the alignment score of Sec. 3.3.2 restricted to one layer, without any
 * sketch.  `method` picks the contraction order of Sec. 4.3:
 *   DR_SCORE_DIRECT  form G_i (tile by tile, never stored) and take its
 *                    inner product with gbar* ("Direct");
 *   DR_SCORE_GIP     (1/m) sum_j <D_i D*_j^T, X_i X*_j^T>, two T x T token
 *                    cross-correlations per pair ("Ghost Inner Product");
 *   DR_SCORE_PIP     sum_t dy_{i,t}^T gbar* x_{i,t} ("Per-Token Inner
 *                    Product").
 * All three give the same scores up to rounding; their costs differ with T,
 * m and the layer size (the crossover the section analyses).
 * Arguments
 *   layers   (host) num_layers descriptors (x, ldx, dy, lddy, d_in, d_out
 *            used); rows 0..n-1 of x / dy are the general examples, rows
 *            n..n+m-1 the targets.
 *   n >= 0, m >= 1, T >= 0; len device int32 [n + m] or NULL (all T).
 *   dtype    DR_BF16 (DR_F32: DR_ERR_UNSUPPORTED).
 *   s        fp32 [num_layers][n] out (a group's score is the sum over its
 *            layers).
 *   workspace at least dr_score_workspace_size() bytes.
 * Arithmetic: bf16 MFMA with fp32 accumulation, partial sums in fp64; PIP
 * multiplies by gbar* as a bf16 hi + lo pair.  Layers are processed one at a
 * time (the workspace holds one layer's gbar*).
 * Requirements as for dr_assemble_update; one layer's gbar* rows and one
 * example's rows must span less than 4 GiB (else DR_ERR_UNSUPPORTED).
 * ------------------------------------------------------------------------- */
dr_status dr_score_exact(const dr_layer* layers, int num_layers, int64_t n, int64_t m, int64_t T,
                         const int32_t* len, dr_dtype dtype, dr_score_method method, float* s,
                         void* workspace, size_t ws_bytes, void* stream);
size_t dr_score_workspace_size(const dr_layer* layers, int num_layers, int64_t n, int64_t m, int64_t T,
                               dr_dtype dtype, dr_score_method method);

#ifdef __cplusplus
}
#endif

#endif /* DR_API_H */
