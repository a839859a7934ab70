/*
 * mesorasi.h -- C ABI of the MI355X (gfx950) delayed-aggregation library
 * libmesorasi.so.
 *
 * Method: Feng et al., "Mesorasi: Architecture Support for Point Cloud
 * Analytics via Delayed-Aggregation" (arXiv 2008.06967).  A point-cloud
 * module computes p_o = F(A(N(p_i), p_i)) (Sec. 3.1, Eq. (1)).  Delayed
 * aggregation (Sec. 4.1, Eq. (2)-(3)) instead runs the shared MLP F once on
 * the N input points (the point feature table, PFT), runs the neighbor
 * search N concurrently into the neighbor index table (NIT), and finally
 * aggregates PFT rows by the NIT: max over the K neighbors, then subtract
 * the centroid's own PFT row (max(f_j - f_c) = max(f_j) - f_c, end of the
 * Sec. 4.1 walk-through).
 *
 * General rules for every entry point
 *  - Pointers are DEVICE pointers unless marked "host".  The caller owns
 *    every buffer; the library never allocates, frees or synchronises, so
 *    every call may be captured into a HIP graph.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Work is enqueued asynchronously on it; ordering across streams is the
 *    caller's job (events).
 *  - Arrays are row-major and contiguous unless a leading dimension `ld_*`
 *    (in elements) is given.  Index arrays are int32 and local to their
 *    cloud: 0 <= index < N.  Point coordinates are float32 [B, N, 3].
 *  - Inputs are const; outputs must not alias inputs.  Every output element
 *    is written, padding included.
 *  - Return value: MESORASI_OK or a negative status.  All argument checks
 *    run on the host BEFORE any HIP call, so a rejected call touches no
 *    device state.  MESORASI_EHIP reports a failed launch; device faults
 *    surface at the caller's next synchronisation.  Out-of-range indices
 *    in a caller-supplied NIT/index array are undefined behaviour.
 *  - mesorasi_last_error() returns a thread-local text describing the last
 *    failure on the calling thread.
 *  - Zero-sized batches (B == 0, M == 0 or rows == 0) are valid no-ops.
 */
#ifndef MESORASI_H
#define MESORASI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MESORASI_VERSION 1

enum {
    MESORASI_OK = 0,
    MESORASI_EINVAL = -1,        /* invalid argument (NULL, negative size, inconsistent shape) */
    MESORASI_EUNSUPPORTED = -2,  /* valid but outside the implemented limits */
    MESORASI_EHIP = -3,          /* the HIP runtime reported an error at launch */
    MESORASI_EWORKSPACE = -4     /* workspace NULL or smaller than the matching *_workspace() size */
};

enum { MESORASI_F32 = 0, MESORASI_BF16 = 1 };

/* Limits (MESORASI_EUNSUPPORTED beyond them). */
#define MESORASI_MAX_N_FPS 65536     /* points per cloud for FPS */
#define MESORASI_MAX_K_BALL 1024     /* neighbors per ball query */
#define MESORASI_MAX_K_KNN 64        /* neighbors per kNN query */
#define MESORASI_MAX_C_KNN 128       /* kNN feature width */
#define MESORASI_MAX_LAYERS 8        /* MLP depth */
#define MESORASI_MAX_WIDTH 4096      /* MLP layer width */

int mesorasi_version(void);
const char* mesorasi_strerror(int status);
const char* mesorasi_last_error(void);

/*
 * Farthest-point sampling (the centroid sampling of the PointNet++ modules,
 * Sec. 6 "Software Setup"; the paper names it without defining it).
 * Greedy: start at point 0; keep for each point its squared distance to the
 * nearest selected point; select the point where it is largest, the lowest
 * index on ties.  Squared distance: t_c = x_c - y_c, d = fma(t_c, t_c, d)
 * for c = x, y, z from d = 0, each step rounded to fp32 -- bit-exact and
 * deterministic.
 *   xyz   [B, N, 3] float32
 *   idx   [B, M] int32 out: selected indices in selection order
 *   cxyz  [B, M, 3] float32 out, nullable: copies of the selected points
 *   ws    device workspace of at least mesorasi_fps_workspace(B, N, M)
 *         bytes, 8-byte aligned (NULL allowed when that size is 0).  Large
 *         clouds spread each cloud over several workgroups that exchange
 *         their per-iteration winners through it; it is cleared by the call
 *         itself (any contents on entry), and its first 4 bytes hold 0 after
 *         the call, or 1 if a workgroup gave up waiting on the others (it
 *         then finishes on its own and the indices, though in [0, N), are
 *         not the sampling's; this needs the call's workgroups to be kept
 *         from running together, which a working GPU does not do).  Calls
 *         that overlap in time need separate workspaces.
 * Errors: EINVAL for NULL xyz/idx, B/N/M < 0, M > N, N == 0 < M, a
 *         misaligned ws;  EUNSUPPORTED for N > MESORASI_MAX_N_FPS;
 *         EWORKSPACE when ws is too small.
 * The M iterations are sequential: one workgroup per cloud for small
 * clouds, several single-wave workgroups per cloud for large ones.
 */
int mesorasi_fps(const float* xyz, int64_t B, int64_t N, int64_t M, int32_t* idx, float* cxyz, void* ws,
                 size_t ws_bytes, void* stream);

/* Workspace bytes for mesorasi_fps with these sizes (0 when none is
 * needed).  Returns 0 for invalid sizes as well. */
size_t mesorasi_fps_workspace(int64_t B, int64_t N, int64_t M);

/*
 * Farthest-point sampling of a sampled set: the nested sampling of stacked
 * set-abstraction modules, where each module samples its centroids from the
 * previous module's centroids (Sec. 6 "Software Setup"; Sec. 3.1, each
 * module's output points are the next module's input points).
 * The greedy sampling above is a greedy permutation: run from index 0 on
 * the ordered output of an earlier run (M_prev points), it selects exactly
 * the first M of them.  (At step k the earlier run chose the point of
 * largest min-distance to the points chosen so far among all points; that
 * point is in the subset, with the same fp32 min-distance, and every other
 * subset point of that value comes later in the subset.  A step whose
 * largest min-distance is 0 -- the cloud's distinct points used up -- chose
 * point 0 in the earlier run and chooses subset point 0 here.)  So no
 * distance is computed:
 *   idx[b][k]  = k, or 0 where k > 0 and idx_prev[b][k] == 0
 *   cxyz[b][k] = cxyz_prev[b][k]
 * which equals mesorasi_fps(cxyz_prev, B, M_prev, M) bit for bit when
 * (idx_prev, cxyz_prev) is an output of mesorasi_fps or of this call; for
 * any other input the result is not a sampling of it.
 *   idx_prev  [B, M_prev] int32, cxyz_prev [B, M_prev, 3] float32 (nullable
 *             when cxyz is NULL)
 *   idx       [B, M] int32 out; cxyz [B, M, 3] float32 out, nullable
 * Errors: EINVAL for sizes < 0, M > M_prev, NULL idx_prev/idx, cxyz
 *         without cxyz_prev; EUNSUPPORTED for M_prev > MESORASI_MAX_N_FPS.
 */
int mesorasi_fps_prefix(const int32_t* idx_prev, const float* cxyz_prev, int64_t B, int64_t M_prev, int64_t M,
                        int32_t* idx, float* cxyz, void* stream);

/*
 * Several nested levels at once: level v (v < n_levels) is the sampling of
 * M[v] points from the previous level, level 0's sampling being
 * (idx0, cxyz0) with M0 points.  By the property above every level is a
 * prefix of level 0 and its indices follow from idx0 alone:
 *   idx[v][b][k]  = k, or 0 where k > 0 and idx0[b][k] == 0
 *   cxyz[v][b][k] = cxyz0[b][k]
 * (for M[0] >= M[1] >= ..., each level equals mesorasi_fps_prefix on the
 * previous one).  One launch for all levels.
 *   idx0 [B, M0] int32, cxyz0 [B, M0, 3] float32 (nullable when no cxyz
 *        output is requested)
 *   M    host array [n_levels], 0 <= M[v] <= M0
 *   idx  host array [n_levels] of device [B, M[v]] int32 outputs
 *   cxyz host array [n_levels] of device [B, M[v], 3] float32 outputs, or
 *        NULL; an entry may be NULL
 * Errors: EINVAL for sizes < 0, n_levels outside [0, MESORASI_MAX_LAYERS],
 *         M[v] outside [0, M0], NULL M/idx/idx[v]/idx0, cxyz without cxyz0;
 *         EUNSUPPORTED for M0 > MESORASI_MAX_N_FPS.
 */
int mesorasi_fps_prefix_levels(const int32_t* idx0, const float* cxyz0, int64_t B, int64_t M0, int32_t n_levels,
                               const int64_t* M, int32_t* const* idx, float* const* cxyz, void* stream);

/*
 * Ball query: neighbor search N (Sec. 3.1 "Neighbor Search") producing the
 * NIT (Sec. 4.1 walk-through).  For each query q, the first K point indices
 * in ascending order with squared distance (same rule as FPS) strictly
 * below fl32(radius * radius); remaining slots repeat the first hit, or
 * hold 0 when there is none.
 *   xyz   [B, N, 3] float32 points;  qxyz [B, M, 3] float32 queries
 *   nit   [B, M, K] int32 out
 *   cnt   [B, M] int32 out, nullable: number of real hits (<= K)
 *   ws    device workspace of at least mesorasi_ball_query_workspace(B, N,
 *         M) bytes, 256-byte aligned (NULL allowed when that size is 0).
 *         Clouds of 8192 points or more are binned into a grid of cells of
 *         edge >= radius in it (rebuilt by every call; any contents on
 *         entry); calls that overlap in time need separate workspaces.
 * Errors: EINVAL for NULL xyz/qxyz/nit, B/N/M < 0, N == 0 < M, K < 1,
 *         radius not finite or <= 0, a misaligned ws;  EUNSUPPORTED for
 *         K > MESORASI_MAX_K_BALL, N > 2^31 - 321 (N > MESORASI_MAX_N_FPS
 *         with a workspace), M > 2^31 - 1;  EWORKSPACE when ws is too small.
 */
int mesorasi_ball_query(const float* xyz, const float* qxyz, int64_t B, int64_t N, int64_t M, float radius,
                        int32_t K, int32_t* nit, int32_t* cnt, void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes for mesorasi_ball_query with these sizes (0 when none is
 * needed, and for invalid sizes). */
size_t mesorasi_ball_query_workspace(int64_t B, int64_t N, int64_t M);

/*
 * The ball query above in two steps, so the cloud can be binned before its
 * query centroids exist (the input points of a network are known while its
 * first sampling still runs):
 *   mesorasi_ball_query_grid_build bins each cloud of xyz [B, N, 3] into
 *   cubic cells of edge at least radius (1 + 2^-12) in ws;
 *   mesorasi_ball_query_grid answers the queries against those cells, with
 *   exactly the result of mesorasi_ball_query (same rule, same order, same
 *   padding and counts).
 * xyz must be the cloud the grid was built from, unchanged since; a query
 * radius above the build's walks the cloud instead (same result).  The
 * workspace ws (at least mesorasi_ball_query_grid_workspace(B, N) bytes,
 * 256-byte aligned) holds the grid between the calls; a query only reads
 * it, so several queries may share one grid.
 * Errors: as mesorasi_ball_query; EWORKSPACE when ws is NULL or too small;
 *         EUNSUPPORTED for N > MESORASI_MAX_N_FPS.
 */
size_t mesorasi_ball_query_grid_workspace(int64_t B, int64_t N);
int mesorasi_ball_query_grid_build(const float* xyz, int64_t B, int64_t N, float radius, void* ws, size_t ws_bytes,
                                   void* stream);
int mesorasi_ball_query_grid(const float* xyz, const float* qxyz, int64_t B, int64_t N, int64_t M, float radius,
                             int32_t K, int32_t* nit, int32_t* cnt, const void* ws, size_t ws_bytes, void* stream);

/*
 * k nearest neighbours in C-dimensional feature space (the DGCNN search in
 * the previous module's output space, Sec. 5.1 "Work Flow").  Squared
 * distance t_c = r_c - q_c, d = fma(t_c, t_c, d) for c ascending from 0;
 * the K smallest by (distance, index), sorted; self is included when the
 * query is one of the reference points.
 *   ref   [B, N, ld_ref] float32 (first C columns used)
 *   query [B, M, ld_query] float32
 *   nit   [B, M, K] int32 out;  dist [B, M, K] float32 out, nullable
 * Errors: EINVAL for NULL ref/query/nit, sizes < 0, K < 1, K > N, C < 1,
 *         ld < C;  EUNSUPPORTED for K > MESORASI_MAX_K_KNN,
 *         C > MESORASI_MAX_C_KNN, or more query blocks than one launch
 *         holds (B x ceil(M / 16) above 2^31 - 1).
 */
int mesorasi_knn(const float* ref, int64_t ld_ref, const float* query, int64_t ld_query, int64_t B, int64_t N,
                 int64_t M, int32_t C, int32_t K, int32_t* nit, float* dist, void* stream);

/*
 * Shared per-point MLP: feature computation F (Sec. 3.1 "Feature
 * Computation"; Eq. (3) with phi = ReLU), run on any set of rows -- in the
 * delayed module on the N input points, producing the PFT.
 *   layer l: h_{l+1} = phi_l(h_l W_l^T + b_l), phi_l = ReLU iff bit l of
 *   relu_mask is set.
 * Input rows are the column concatenation [x0 | x1]:
 *   x0 [rows, ld0] float32 (first c0 columns), x1 [rows, ld1] float32 (first
 *   c1 columns; NULL iff c1 == 0).  dims (host) has n_layers + 1 entries,
 *   dims[0] == c0 + c1.
 *   W    host array of n_layers device pointers; W[l] is [dims[l+1], dims[l]]
 *        row-major (torch Linear layout), float32 when dtype == F32, bf16
 *        bits (uint16, round-to-nearest-even) when dtype == BF16.
 *   bias host array of n_layers float32 device pointers (entries nullable).
 *   dtype F32: fp32 inputs/weights on fp32 MFMA, fp32 activations.
 *         BF16: inputs rounded to bf16, bf16 weights, bf16 MFMA with fp32
 *         accumulation; bias and ReLU in fp32; every stored activation
 *         (intermediate and output) rounded to bf16.
 *   out_dtype F32 or BF16: storage type of y (a BF16-path result stored as
 *         F32 holds bf16-representable values).
 *   pool_group 0: y is [rows, ld_y].  G > 0: rows % G == 0 and y is
 *         [rows / G, ld_y] holding the column max over each group of G
 *         consecutive rows (the reduction after F, Sec. 3.1; group-all
 *         modules).  Pooling needs ReLU on the last layer and out_dtype F32.
 *   ws   device workspace of at least mesorasi_pointwise_mlp_workspace()
 *        bytes (NULL allowed when that size is 0).
 * Errors: EINVAL for NULL x0/y/W/dims, c0 < 1, c1 < 0, ld < c, dims[0] !=
 *         c0 + c1, a width < 1, ld_y < dims[n], rows % G != 0;
 *         EUNSUPPORTED for n_layers outside [1, MESORASI_MAX_LAYERS], a width
 *         above MESORASI_MAX_WIDTH, pooling without a final ReLU or with
 *         out_dtype BF16, G > 2^31 - 1;  EWORKSPACE when ws is too small.
 */
int mesorasi_pointwise_mlp(const float* x0, int32_t c0, int64_t ld0, const float* x1, int32_t c1, int64_t ld1,
                           int64_t rows, int32_t n_layers, const int32_t* dims, const void* const* W,
                           const float* const* bias, uint32_t relu_mask, int32_t dtype, int32_t out_dtype, void* y,
                           int64_t ld_y, int64_t pool_group, void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes for mesorasi_pointwise_mlp with these arguments (0 when
 * none is needed).  Returns 0 for invalid arguments as well. */
size_t mesorasi_pointwise_mlp_workspace(int64_t rows, int32_t n_layers, const int32_t* dims, int32_t dtype,
                                        int64_t pool_group);

/*
 * mesorasi_pointwise_mlp without a workspace argument and without any
 * allocation, for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * Same arguments, results and errors as mesorasi_pointwise_mlp, except:
 *  - the intermediate activations and split-K partials live in a fixed
 *    device array of MESORASI_NOALLOC_WS_BYTES inside the library, one per
 *    GPU, held until the process ends;
 *  - a call whose mesorasi_pointwise_mlp_workspace() exceeds that size is
 *    rejected with EUNSUPPORTED before any HIP call;
 *  - EHIP if the array's device address cannot be obtained (looked up once
 *    per device, with that device current, on the first call that needs it).
 * Every call on one GPU shares that GPU's array and leaves its last
 * contents there: calls that overlap on one GPU (different streams or host
 * threads without ordering between them) race and give wrong results.
 * Nothing in the array needs to start at zero.
 */
#define MESORASI_NOALLOC_WS_BYTES (32u << 20)
int mesorasi_pointwise_mlp_noalloc(const float* x0, int32_t c0, int64_t ld0, const float* x1, int32_t c1,
                                   int64_t ld1, int64_t rows, int32_t n_layers, const int32_t* dims,
                                   const void* const* W, const float* const* bias, uint32_t relu_mask, int32_t dtype,
                                   int32_t out_dtype, void* y, int64_t ld_y, int64_t pool_group, void* stream);

/*
 * Aggregation A on the PFT (Sec. 5.2 first paragraph; Sec. 4.1 max/subtract
 * distributivity): for each NIT entry, gather the K PFT rows, take the
 * column-wise max (exact), then combine with the centroid row in one fp32
 * operation: out = max + sign * centroid, then ReLU when relu != 0.
 *   pft   [B, N, ld_pft] of pft_dtype (F32 or BF16), first C columns used
 *   nit   [B, M, K] int32
 *   centroid row: cidx [B, M] int32 (a PFT row: pft[b, cidx]) or cfeat
 *         [B, M, ld_c] of pft_dtype (explicit table); both NULL = no
 *         centroid term.  At most one may be non-NULL.
 *   sign  -1 (PointNet++: subtract the centroid feature) or +1 (DGCNN: add
 *         the (W1 - W2) x_i term).
 *   out   [B, M, ld_out] float32
 * Errors: EINVAL for NULL pft/nit/out, sizes < 0, K < 1, C < 1, ld < C,
 *         both cidx and cfeat set, sign not +-1, N == 0 < M;
 *         EUNSUPPORTED for an unknown dtype or C > 65536.
 */
int mesorasi_aggregate_max(const void* pft, int64_t ld_pft, int32_t pft_dtype, const int32_t* nit, int64_t B,
                           int64_t N, int64_t M, int32_t K, int32_t C, const int32_t* cidx, const void* cfeat,
                           int64_t ld_c, int32_t sign, int32_t relu, float* out, int64_t ld_out, void* stream);

/*
 * Aggregation fused into the next module's MLP (the GPU analogue of the
 * aggregation unit writing into the NPU's global buffer, Sec. 5.2): for the
 * B * M centroids of module i (delayed order), the first-layer input rows
 * of module i + 1 are [cxyz_c | max_k pft[b, nit[c, k]] - pft[b, cidx[c]]]
 * -- mesorasi_aggregate_max's result with sign -1, bit for bit -- built in
 * the MLP kernel's loader instead of going through HBM; then the MLP of
 * mesorasi_pointwise_mlp on them.
 *   cxyz [B, M, 3] float32 (module i's centroids = module i + 1's points)
 *   pft  [B, N, ld_pft] float32 (module i's PFT), nit [B, M, K] int32,
 *   cidx [B, M] int32 (module i's FPS indices)
 *   MLP arguments as in mesorasi_pointwise_mlp with dtype F32 and
 *   dims[0] == 3 + C;  y [B * M, ld_y] float32 out
 *   agg_out [B, M, ld_agg] float32 out, nullable: the aggregated rows as
 *   well (module i's output, e.g. a skip connection)
 * Errors: EINVAL for NULL pointers, sizes < 0, K < 1, C < 1, ld < width,
 *         dims[0] != 3 + C;  EUNSUPPORTED unless the MLP has at least two
 *         layers with inputs <= 160 and outputs <= 128 channels, C and the
 *         leading dimensions are multiples of 4 and pft / agg_out are
 *         16-byte aligned.
 */
int mesorasi_aggregate_mlp(const float* cxyz, const float* pft, int64_t ld_pft, const int32_t* nit,
                           const int32_t* cidx, int64_t B, int64_t N, int64_t M, int32_t K, int32_t C, int32_t n_layers,
                           const int32_t* dims, const void* const* W, const float* const* bias, uint32_t relu_mask,
                           float* y, int64_t ld_y, float* agg_out, int64_t ld_agg, void* stream);

/*
 * Conventional module, kept as the comparison path (Eq. (1); Sec. 3.1
 * "Aggregation" and "Feature Computation"): the neighbor feature matrix
 * (NFM), the MLP on every (centroid, neighbor) row, and the max over the
 * K rows of each centroid.  fp32 PointNet++ grouping reads the NFM rows
 * straight from xyz / feat through nit (inside the fused MLP kernel, or in
 * the first layer's GEMM when cf and ld_f are multiples of 4 and feat is
 * 16-byte aligned); otherwise (bf16, DGCNN edge grouping, other widths)
 * the NFM is built in the workspace first.  Results agree to fp32
 * rounding either way.
 *   grouping 0 (PointNet++): NFM row = [xyz_j - cxyz_c | feat_j], dims[0] =
 *            3 + cf; needs xyz and cxyz [B, M, 3].
 *   grouping 1 (DGCNN edge): NFM row = [f_i | f_j - f_i] with f = feat
 *            [B, N, ld_f] (cf columns), centroid i = point i (M == N);
 *            dims[0] = 2 cf; xyz/cxyz unused (nullable).
 *   nit [B, M, K] int32; out [B, M, ld_out] float32.
 *   MLP arguments as in mesorasi_pointwise_mlp (last layer must have ReLU).
 *   ws  at least mesorasi_conventional_workspace() bytes.
 * Errors: as mesorasi_pointwise_mlp plus EINVAL for an unknown grouping,
 *         NULL nit, M != N for grouping 1, dims[0] inconsistent with cf.
 */
int mesorasi_conventional_module(const float* xyz, const float* feat, int32_t cf, int64_t ld_f, const float* cxyz,
                                 const int32_t* nit, int64_t B, int64_t N, int64_t M, int32_t K, int32_t grouping,
                                 int32_t n_layers, const int32_t* dims, const void* const* W,
                                 const float* const* bias, uint32_t relu_mask, int32_t dtype, float* out,
                                 int64_t ld_out, void* ws, size_t ws_bytes, void* stream);

size_t mesorasi_conventional_workspace(int64_t B, int64_t M, int32_t K, int32_t n_layers, const int32_t* dims,
                                       int32_t dtype);

/*
 * Limited delayed aggregation (Sec. 7.3, "Ltd"): only the first MLP
 * layer's matrix product is hoisted before aggregation, which keeps the
 * module exact because that product is linear.  The caller computes
 *   p1 = [xyz | feat] W1^T on the N input points  (mesorasi_pointwise_mlp,
 *        one layer, no bias, no ReLU)            -> [B, N, ld_p], C1 columns
 *   q  = cxyz W1[:, :3]^T on the M centroids      -> [B, M, ld_q], C1 columns
 * and this call forms, for every (centroid c, neighbor k) row,
 *   h1 = ReLU(p1[b, nit[b, c, k], :] - q[b, c, :] + b1)
 * (fp32: the subtraction, then the bias), runs the remaining layers
 * (n_layers >= 1, dims[0] == C1) on those B*M*K rows and max-reduces over
 * the K rows of each centroid into out [B, M, ld_out].  In fp32 the h1
 * rows are formed in the next layer's loader (fused MLP kernel, or a GEMM
 * when C1, ld_p, ld_q are multiples of 4 and p1, q, b1, W[0] are 16-byte
 * aligned); otherwise they are written to the workspace first.
 *   b1  [C1] float32 or NULL (no first-layer bias).
 *   nit [B, M, K] int32, per-cloud indices in [0, N).
 *   MLP arguments as in mesorasi_pointwise_mlp (last layer must have ReLU).
 *   ws  at least mesorasi_ltd_workspace() bytes.
 * Errors: as mesorasi_pointwise_mlp plus EINVAL for NULL p1, q or nit,
 *         ld_p or ld_q < C1, dims[0] != C1; EUNSUPPORTED for n_layers < 1
 *         (a one-layer module's limited order is its delayed order:
 *         mesorasi_aggregate_max).
 */
int mesorasi_ltd_module(const float* p1, int64_t ld_p, const float* q, int64_t ld_q, const float* b1,
                        const int32_t* nit, int64_t B, int64_t N, int64_t M, int32_t K, int32_t C1, int32_t n_layers,
                        const int32_t* dims, const void* const* W, const float* const* bias, uint32_t relu_mask,
                        int32_t dtype, float* out, int64_t ld_out, void* ws, size_t ws_bytes, void* stream);

size_t mesorasi_ltd_workspace(int64_t B, int64_t M, int32_t K, int32_t n_layers, const int32_t* dims, int32_t dtype);

/*
 * Feature propagation by 3-NN inverse-distance interpolation (the
 * three_interpolate kernel of the PointNet++ segmentation baseline, Sec. 6
 * "Software Setup").  For every destination point: its 3 nearest source
 * points by the kNN rule above (C = 3), weights w = 1 / max(d2, 1e-10),
 * f_dst = sum_k w_k f_k / sum_k w_k (fp32).
 *   xyz_dst [B, Nd, 3], xyz_src [B, Ns, 3], f_src [B, Ns, ld_src] float32
 *   f_dst   [B, Nd, ld_dst] float32 out (first C columns written)
 * Errors: EINVAL for NULL pointers, sizes < 0, Ns < 3, C < 1, ld < C.
 */
int mesorasi_interpolate3(const float* xyz_dst, const float* xyz_src, const float* f_src, int64_t ld_src,
                          int64_t B, int64_t Nd, int64_t Ns, int32_t C, float* f_dst, int64_t ld_dst, void* stream);

/*
 * The two halves of mesorasi_interpolate3 (three_nn and three_interpolate
 * of the same baseline, Sec. 6), so that the search, which needs only
 * coordinates, can run as soon as both levels are sampled, apart from the
 * interpolation, which waits for the coarse features.
 * mesorasi_three_nn: for every destination, its 3 nearest sources in
 * (distance, index) order (the kNN rule, C = 3) and their squared
 * distances -- the same values mesorasi_knn returns with K = 3.
 *   xyz_dst [B, Nd, 3], xyz_src [B, Ns, 3] float32
 *   nit [B, Nd, 3] int32 out, dist [B, Nd, 3] float32 out
 * Errors: EINVAL for NULL pointers, sizes < 0, Ns < 3.
 * mesorasi_interpolate3_apply: f_dst = sum_k w_k f_src[nit_k] / sum_k w_k
 * with w_k = 1 / max(dist_k, 1e-10), in the fp32 operations of
 * mesorasi_interpolate3 (so the two give identical results).
 *   nit [B, Nd, 3] int32 (0 <= index < Ns), dist [B, Nd, 3] float32
 *   f_src [B, Ns, ld_src], f_dst [B, Nd, ld_dst] float32 (first C columns)
 * Errors: EINVAL for NULL pointers, sizes < 0, Ns < 1, C < 1, ld < C.
 */
int mesorasi_three_nn(const float* xyz_dst, const float* xyz_src, int64_t B, int64_t Nd, int64_t Ns, int32_t* nit,
                      float* dist, void* stream);
int mesorasi_interpolate3_apply(const int32_t* nit, const float* dist, const float* f_src, int64_t ld_src, int64_t B,
                                int64_t Nd, int64_t Ns, int32_t C, float* f_dst, int64_t ld_dst, void* stream);

/*
 * A feature-propagation layer's first product taken on the coarse points.
 * The 3-NN interpolation is a convex combination, so for the first layer
 * of the feature-propagation MLP on [interpolated | skip] rows,
 *   W1 [interp(f) | s] + b1 = interp(W1a f) + (W1b s + b1),
 * with W1a the columns of W1 that read the interpolated features: W1a f is
 * then computed on the coarse points (4x fewer rows here) and W1b s + b1
 * ahead of time, and this call forms the layer's output:
 *   f_dst = phi(sum_k w_k f_src[nit_k] / sum_k w_k + add),
 * the interpolation in the fp32 operations of mesorasi_interpolate3_apply
 * followed by one fp32 addition; phi = ReLU when relu != 0, else identity.
 *   nit, dist as for mesorasi_interpolate3_apply
 *   f_src [B, Ns, ld_src] float32 (W1a f on the coarse points)
 *   add   [B, Nd, ld_add] float32 (W1b s + b1 on the fine points); may be
 *         f_dst itself when ld_add == ld_dst (in-place update)
 *   f_dst [B, Nd, ld_dst] float32 out (first C columns written)
 * Errors: EINVAL for NULL pointers, sizes < 0, Ns < 1, C < 1, ld < C, or
 * add aliasing f_dst with another leading dimension.
 */
int mesorasi_interpolate3_add(const int32_t* nit, const float* dist, const float* f_src, int64_t ld_src, int64_t B,
                              int64_t Nd, int64_t Ns, int32_t C, const float* add, int64_t ld_add, int32_t relu,
                              float* f_dst, int64_t ld_dst, void* stream);

/*
 * mesorasi_interpolate3_add followed by an MLP on its rows, in one kernel:
 * the interpolation, the addition and phi are done in the register-resident
 * MLP's row loader, so the layer's output never goes to memory (the
 * feature-propagation level of mesorasi_interpolate3_add, its remaining
 * layers included).
 *   y = MLP(phi(sum_k w_k f_src[nit_k] / sum_k w_k + add))
 * with the interpolation, addition and phi in the fp32 operations of
 * mesorasi_interpolate3_add and the MLP as in mesorasi_pointwise_mlp (fp32).
 *   nit, dist, f_src, add as for mesorasi_interpolate3_add, over C = dims[0]
 *         channels; f_src and add 16-byte aligned
 *   W, bias, relu_mask: the MLP as in mesorasi_pointwise_mlp (dims[0] = C)
 *   y [B, Nd, ld_y] float32 out; must not overlap add
 * No workspace.  The layers' permuted weights live in LDS; when they do not
 * all fit its 160 KB at once (e.g. the level's layers followed by the
 * per-point head) they are staged in phases, which needs every wave of the
 * device to hold at most one 32-row tile: B * Nd <= 32 x 8 x (compute
 * units), 65536 rows on MI355X.
 * Errors: EINVAL for NULL pointers, sizes < 0, Ns = 0 with points, ld < C
 * or ld_y < dims[n_layers]; EUNSUPPORTED unless every layer is at most 128
 * wide (its own permuted weights fitting 160 KB), the row bound above holds
 * when phases are needed, dims[0], ld_src and ld_add are multiples of 4 and
 * f_src and add are 16-byte aligned -- callers fall back to
 * mesorasi_interpolate3_add + mesorasi_pointwise_mlp.
 */
int mesorasi_interpolate3_mlp(const int32_t* nit, const float* dist, const float* f_src, int64_t ld_src, int64_t B,
                              int64_t Nd, int64_t Ns, const float* add, int64_t ld_add, int32_t relu,
                              int32_t n_layers, const int32_t* dims, const void* const* W, const float* const* bias,
                              uint32_t relu_mask, float* y, int64_t ld_y, void* stream);

/*
 * float32 -> bf16 bits, round to nearest even (weights and inputs of the
 * bf16 MLP variant).  x [n] float32, y [n] uint16 out.
 * Errors: EINVAL for NULL pointers or n < 0.
 */
int mesorasi_cast_bf16(const float* x, int64_t n, uint16_t* y, void* stream);

/*
 * EdgeConv weight fold for the delayed DGCNN module.  The edge function
 * W [x_i | x_j - x_i] + b equals (W1 - W2) x_i + W2 x_j + b, so the PFT of
 * the delayed module is X [W1 - W2 ; W2]^T with bias [b ; 0].
 *   W [C_out, 2 C] float32 (W1 = first C columns, W2 = last C)
 *   b [C_out] float32 (nullable: treated as 0)
 *   W_out [2 C_out, C] float32 out: rows 0..C_out-1 = fl32(W1 - W2),
 *         rows C_out.. = W2;  b_out [2 C_out] float32 out = [b ; 0]
 * Errors: EINVAL for NULL W/W_out/b_out, C < 1, C_out < 1.
 */
int mesorasi_edgeconv_fold(const float* W, const float* b, int32_t C, int32_t C_out, float* W_out, float* b_out,
                           void* stream);

/*
 * Debug check of an index array (the NIT, FPS or 3-NN indices before they
 * are used to read rows): *count = the number of entries of idx outside
 * [0, bound).  The library's gathers trust their index arrays (an index out
 * of range there is undefined behaviour); this check reads only idx and
 * writes only *count, so it is safe on any input.
 *   idx [n] int32, count: one device int32 out (overwritten)
 * Errors: EINVAL for NULL count, NULL idx with n > 0, n < 0.
 */
int mesorasi_count_out_of_range(const int32_t* idx, int64_t n, int32_t bound, int32_t* count, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MESORASI_H */
