/*
 * vkv.h -- C ABI of libvkv: the decode-time hot path of VestigeKV
 * (arXiv 2609.03949) on AMD Instinct MI355X (gfx950).
 *
 * One decode step over a multi-head-latent-attention KV cache whose rows are
 * 576 bf16 wide (512 content latent + 64 decoupled branch; Sec. 3, Eq. (setup)):
 *
 *   vkv_digest_build  index of every cache row: [branch ; RNE_bf16(P c_u)] and
 *                     the row certificate scalars (Sec. 4.2, index entry; run
 *                     once per context, the paper's compression event)
 *   vkv_query_prep    query side of the scan: the query digest and head scalars
 *   vkv_score         index score of every archived row from the narrow slice:
 *                     the exact-branch and sketch terms of Eq. (trigger),
 *                     maximised over heads (fp32 MFMA, with a certified error)
 *   vkv_select        exact per-sequence top-k by (score desc, index asc)
 *   vkv_admit         optional two-tier admission: rows outside the top-k whose
 *                     certified upper bound (Lemma (Index certificate)) exceeds
 *                     the k-th selected score
 *   vkv_attend        exact softmax attention over the selected rows, the
 *                     recent window and the admitted rows, on full 576-wide
 *                     rows (Lemma (Exchangeability): fetched rows join the
 *                     softmax as exact copies)
 *   vkv_step_run      query_prep -> score -> select -> [admit] -> attend in one call
 *
 * Conventions (all entry points):
 *   - Pointers are DEVICE pointers unless stated.  The caller owns every
 *     buffer; the library never allocates or frees caller memory.  Per-step
 *     scratch lives in a caller-provided workspace (vkv_workspace_size).
 *   - bf16 values are passed as uint16_t bit patterns.  Index lists are
 *     int32, sorted ascending.
 *   - Every call is asynchronous on `stream` (a hipStream_t, NULL = default
 *     stream) and does no device synchronisation, except vkv_digest_build in
 *     certificate mode (it reads back the contractivity check of P once).
 *   - Arguments are validated before anything is launched; on error the
 *     return code is negative, outputs are untouched and vkv_last_error()
 *     describes the failure.  No C++ exception or abort crosses the ABI.
 *   - A context is bound to one device and may be used from one host thread
 *     at a time.
 */
#ifndef VKV_H
#define VKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------ status codes */
#define VKV_OK 0
#define VKV_E_ARG (-1)            /* null pointer, bad enum, k or cap out of range */
#define VKV_E_SHAPE (-2)          /* sizes out of the supported range */
#define VKV_E_ALIGN (-3)          /* pointer or stride not 16-byte aligned */
#define VKV_E_UNSUPPORTED (-4)    /* valid request the library does not implement */
#define VKV_E_NOT_CONTRACTIVE (-5)/* certificate requested with ||P||_2 not certified <= 1 */
#define VKV_E_HIP (-6)            /* a HIP runtime call failed */
#define VKV_E_WORKSPACE (-7)      /* workspace null or smaller than vkv_workspace_size */
#define VKV_E_DEBUG_ROWS (-8)     /* VKV_DEBUG_ROWS row-set assertion failed */

/* ---------------------------------------------------------- scoring modes */
#define VKV_MODE_ROPE 1           /* 64 branch dims only (read in place or from the index) */
#define VKV_MODE_DIGEST 2         /* r sketch dims only */
#define VKV_MODE_ROPE_DIGEST 3    /* 64 branch dims + r sketch dims (the paper's index) */

#define VKV_D_LAT 512
#define VKV_D_ROPE 64
#define VKV_D_ROW 576

typedef struct vkv_ctx vkv_ctx;

/*
 * One decode step's inputs.  Shapes: B sequences, H heads, T cache rows per
 * sequence, W recent rows.  Rows [0, A) with A = T - W are archived (scored);
 * rows [A, T) are the recent window (always attended, never scored).
 *
 *   q_lat   [B, H, 512] bf16, contiguous: absorbed content query W_UK^T q^c
 *   q_rope  [B, H, 64]  bf16, contiguous: branch query q^r
 *   cache   row u of sequence b at cache + b*cache_batch_stride + u*cache_row_stride
 *           (elements); 576 bf16 = [c_u (512) ; r_u (64)]
 *   index   packed index rows from vkv_digest_build, same addressing with
 *           index_row_stride / index_batch_stride; columns are
 *           [r_u (64, iff index_has_rope) ; digest (r)].  May be NULL in
 *           VKV_MODE_ROPE, which then reads cache[..., 512:576] in place.
 *   P       [r, 512] bf16 digest basis (modes with a digest)
 *   eta, eps, gam  [B, T] fp32 row certificate scalars from vkv_digest_build
 *           (needed by vkv_admit only), built with the same P and r
 *   mode    VKV_MODE_*; r in {0} for ROPE, else a multiple of 32 in [32, 512]
 *
 * Supported: 1 <= B <= 65535, 1 <= H <= 128, 1 <= T < 2^31, 0 <= W <= T.
 * The index width n = (64 if mode has rope) + (r if mode has digest) must be
 * a multiple of 32 and at most 576; row strides and base pointers must be
 * 16-byte aligned.
 */
typedef struct vkv_step {
    int64_t B, H, T, W;
    int32_t mode, r;
    const uint16_t* q_lat;
    const uint16_t* q_rope;
    const uint16_t* cache;
    int64_t cache_row_stride, cache_batch_stride;
    const uint16_t* index;
    int64_t index_row_stride, index_batch_stride;
    int32_t index_has_rope;
    int32_t reserved0;
    const uint16_t* P;
    const float* eta;
    const float* eps;
    const float* gam;
} vkv_step;

/* Context on HIP device `device`.  Owns a few KB of device scratch for the
 * contractivity check and the last error string.  Reads VKV_DEBUG_ROWS from
 * the environment: if set to a non-zero value, vkv_select / vkv_admit
 * synchronise and assert the row-set invariants (in range, strictly
 * ascending, |S| = k, S outside the recent window, admitted rows outside S,
 * count <= cap), returning VKV_E_DEBUG_ROWS on violation. */
int vkv_create(vkv_ctx** out, int device);
int vkv_destroy(vkv_ctx* ctx);
const char* vkv_status_string(int status);
const char* vkv_last_error(const vkv_ctx* ctx);
/* Library version as major*10000 + minor*100 + patch. */
int vkv_version(void);

/*
 * Index build (Sec. 4.2: archived row u keeps (r_u, V_r^T c_u, eta_u); the
 * paper draws the basis from the context's own queries, here P is given).
 * For every row u < T of every sequence:
 *   index[b,u,:] = [ r_u (bit copy, iff with_rope) ; d_u ],
 *   d_u[j] = RNE_bf16( sum_{i<512} P[j,i] c_u[i] )   (fp64, i ascending, one rounding)
 * If eta != NULL (certificate mode; eps and gam must then be non-NULL too),
 * also the row scalars, each an fp32 upper bound rounded toward +inf:
 *   eta_u >= sqrt(c_u^T (I - P^T P) c_u),  eps_u >= ||d_u - P c_u||,  gam_u >= ||P c_u||
 * Certificate mode first checks on the device that ||P||_2 <= 1 (Gershgorin on
 * P P^T with margin) and synchronises the stream to read the verdict; it
 * returns VKV_E_NOT_CONTRACTIVE, writing nothing, if the check fails.
 * r = 0 is allowed (no digest; eta_u >= ||c_u||, eps = gam = 0).  index may be
 * NULL when only the scalars are wanted.
 */
int vkv_digest_build(vkv_ctx* ctx, const uint16_t* cache, int64_t B, int64_t T,
                     int64_t cache_row_stride, int64_t cache_batch_stride, const uint16_t* P,
                     int32_t r, int32_t with_rope, uint16_t* index, int64_t index_row_stride,
                     int64_t index_batch_stride, float* eta, float* eps, float* gam,
                     void* stream);

/*
 * The data-driven sketch basis (Sec. 4.2, the index entry: V_r is drawn from
 * the context's own prefix queries).  q [m, 512] bf16 holds the prefix content
 * queries (one row per query and head).  V_r spans the dominant r-dimensional
 * eigenspace of their second moment C = sum_i q_i q_i^T (fp64; the products of
 * bf16 values are exact), found by subspace iteration: a fixed +-1 start
 * pattern, then `iters` rounds of V <- orth(C V), orth = Cholesky QR twice.  The
 * subspace error shrinks as (lambda_{r+1}/lambda_r)^iters; the index scores
 * depend on the subspace only, not on the basis within it.  Writes
 * P [r, 512] bf16 = RNE_bf16((1 - 2^-6) V_r^T), the basis vkv_digest_build
 * takes (the factor keeps the rounded basis contractive), and, if
 * energy != NULL, energy [2] fp64 (device) = { trace(V_r^T C V_r), trace(C) }:
 * the queries' second moment the sketch captures and the total (both
 * basis-independent; their ratio is the captured fraction).  r: a multiple of
 * 32 in [32, 512]; iters in [0, 64]; ws: vkv_sketch_workspace_size bytes,
 * 256-byte aligned, fully overwritten.  Synchronises `stream` to read the
 * factorisation's verdict and returns VKV_E_UNSUPPORTED if the queries span
 * fewer than r dimensions (a non-positive pivot); P is then not usable.
 */
int vkv_sketch_workspace_size(int32_t r, size_t* bytes);
int vkv_sketch_basis(vkv_ctx* ctx, const uint16_t* q, int64_t m, int32_t r, int32_t iters, void* ws,
                     size_t ws_bytes, uint16_t* P, double* energy, void* stream);

/*
 * The query-independent tier-1 selector (Sec. 4.1, the sigma equation; the
 * block close of the deployment specification's request lifecycle).  Rows are
 * closed in fixed blocks of VKV_SIGMA_BLOCK rows; for every closed block and
 * each of the 64 channels of the branch r_u as the cache row stores it
 * (elements 512..575) the sequence-axis DFT keeps bins [0, kappa) and their
 * mirrors, the rest is zeroed and the transform inverted; sigma_u is the norm
 * over the channels of what this low-pass reconstruction misses at row u.
 *
 * vkv_sigma_close: sigma for rows [t0, t0 + nblk * VKV_SIGMA_BLOCK) of every
 * sequence, t0 a multiple of VKV_SIGMA_BLOCK and the range within T; cache as
 * in vkv_digest_build; kappa in [1, VKV_SIGMA_BLOCK / 2].  sigma [B,
 * sigma_stride] fp64 (device), only the closed range is written.  Each block
 * is transformed on its own, so closing blocks one call at a time or all at
 * once gives the same bits.  fp64 FFT (error about 1e-15 of the block's
 * norm).  ws: vkv_sigma_workspace_size(B, nblk) bytes, 256-byte aligned.
 *
 * vkv_sigma_select: the sigma tier of the first n_closed rows: rows
 * [0, min(nsink, n_closed)) (the sinks) plus the m rows of largest sigma among
 * the other closed rows (ties: the lower row), written ascending to kept
 * [B, K] int32, K = min(nsink, n) + min(m, n - min(nsink, n)), n = n_closed.
 * The tier of the rows closed so far equals the one kept incrementally as
 * blocks close (Corollary (Ranking stationarity)), so one call after each
 * close rebalances it.
 */
#define VKV_SIGMA_BLOCK 4096
int vkv_sigma_workspace_size(int64_t B, int64_t nblk, size_t* bytes);
int vkv_sigma_close(vkv_ctx* ctx, const uint16_t* cache, int64_t B, int64_t T, int64_t cache_row_stride,
                    int64_t cache_batch_stride, int64_t t0, int64_t nblk, int32_t kappa, void* ws,
                    size_t ws_bytes, double* sigma, int64_t sigma_stride, void* stream);
int vkv_sigma_select(vkv_ctx* ctx, const double* sigma, int64_t B, int64_t n_closed, int64_t sigma_stride,
                     int64_t m, int32_t nsink, int32_t* kept, void* stream);

/*
 * One decode step on a given tier-1 set (the per-decode-step line of the
 * deployment specification's request lifecycle): the k rows kept[b] of the
 * archive [0, A) (ascending, for instance the sigma tier) and the recent
 * window are attended; query_prep -> score (ub at cert_mult) -> the exact
 * maximum logit s*_h over kept and window (as vkv_row_max) -> the calibrated
 * trigger against s*_h with the optional top-j cap (as vkv_trigger, kept in
 * place of S) -> attention over kept, window and fired rows (as vkv_attend).
 * kept must be ascending and inside [0, A) (VKV_DEBUG_ROWS checks it after
 * the step); the other arguments and results are those of the calls named.
 * key may be NULL: the step reads only ub (here the trigger margins), and
 * without a key buffer the scan writes no keys at all (faster: each wave of
 * the scan then takes twice the rows).  ws: vkv_workspace_size(st, k, cap)
 * bytes.
 */
int vkv_step_run_kept(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k,
                      const int32_t* kept, float* key, float* ub, float cert_mult, double* smax,
                      int32_t* argmax, int64_t topj, int32_t* fired, int32_t* fired_count, int64_t cap,
                      float scale, uint16_t* out, float* lse, void* stream);

/*
 * The all-layer CSR pack of row lists (Sec. 4.3, the decode step's all-layer
 * CSR pack): n lists of capacity cap, lists [n, cap] int32 (for instance the
 * fired rows of every layer and sequence of a step, each list from
 * vkv_trigger / vkv_step_run_kept), counts [n] (the lists' true counts; a
 * count above cap packs cap rows, a negative one none) ->
 * offsets [n + 1] = the exclusive prefix sums of the packed lengths and
 * packed [offsets[n]] = the lists' rows back to back.  Worst-case buffers
 * (packed of n * cap) make it fit for graph capture: it launches two kernels,
 * never synchronises and allocates nothing.  n <= 65535.
 */
int vkv_pack_rows(vkv_ctx* ctx, const int32_t* lists, const int32_t* counts, int64_t n, int64_t cap,
                  int32_t* offsets, int32_t* packed, void* stream);

/* Page-box bound (the page-bound pruning paragraph of the appendix "The
 * dividend inside prior algorithms", and its equation).  The archived rows
 * [0, A) of each sequence, A = T - W, are cut into npages = ceil(A / page)
 * pages of `page` consecutive rows (the last one ragged).
 *
 * vkv_page_box: box [B][npages][2][n] (device, bf16 bits, n = the index
 * width of the step) receives, per page and index column d, the smallest
 * (box[b][j][0][d]) and the largest (box[b][j][1][d]) value of x_u[d] over
 * the page's rows, x_u the index row as vkv_score reads it; a zero is written
 * as +0.  It reads the index (the cache's branch columns in mode ROPE without
 * an index) once; the boxes change only when rows are appended.
 *
 * vkv_page_bound: after vkv_query_prep on ws, bound [B][npages] (device, fp64)
 * receives
 *     bound[b][j] = max_h sum_d max(qt_hd lo_d, qt_hd hi_d)
 * with each term one exact product (qt_hd hi_d for qt_hd >= 0, else
 * qt_hd lo_d) and the terms summed d ascending with one fp64 rounding each,
 * the order of the fp64 index key.  bound[b][j] >= the fp64 index key of
 * every row of page j, bit for bit, so a page with bound < theta_b (the
 * tier-1 threshold of vkv_select) holds no tier-1 row and a scan may skip it.
 * box is what vkv_page_box wrote for the same page size.
 *
 * Both are asynchronous on `stream` and allocate nothing.  They return
 * VKV_E_ARG for page < 1 or a NULL box or bound, and the step's validation
 * errors; with A = 0 they launch nothing and accept NULL buffers. */
int vkv_page_box(vkv_ctx* ctx, const vkv_step* st, int64_t page, uint16_t* box, void* stream);
int vkv_page_bound(vkv_ctx* ctx, const vkv_step* st, const void* ws, size_t ws_bytes, int64_t page,
                   const uint16_t* box, double* bound, void* stream);

/* Bytes of device workspace a step with budget k and admission capacity cap
 * (0 without admission) needs; the workspace must be 256-byte aligned. */
int vkv_workspace_size(const vkv_step* st, int64_t k, int64_t cap, size_t* bytes);

/*
 * Query side of the index scan, once per step (Eq. (trigger): V_r^T q^c' and
 * the residual scale of the certificate):
 *   qt[b,h,:] = [ q_rope (mode has the branch) ; RNE_bf16(P q_lat) (mode has a digest) ]
 * (fp64, i ascending, one rounding) and the head certificate scalars, fp32
 * rounded toward +inf:  a_h >= sqrt(q^T (I - P^T P) q),  n_h >= ||qd_h||,
 * e_h >= ||qd_h - P q||, all into the workspace.  Must precede vkv_score.
 */
int vkv_query_prep(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, void* stream);

/*
 * Index scores (Eq. (trigger), first two terms; lambda > 0 dropped as it does
 * not change the ranking):
 *   key~[b,u] ~= max_h  sum_d qt[b,h,d] x_u[d],   u in [0, A)
 * with x_u the mode's index row and qt from vkv_query_prep.  bf16 MFMA with
 * fp32 accumulation.  The workspace receives key~ for every row and the
 * per-sequence maxima of ||qt_h|| and ||x_u||, from which vkv_select takes
 * the certified interval [key~ - E, key~ + E] of every fp64 index score,
 *   E = 2 (n + n/32) 2^-23 max_h ||qt_h|| max_u ||x_u||
 * (the fp32 accumulation error, by Cauchy-Schwarz on sum |q_d x_d|).  key
 * (may be NULL) receives key~ as well, for diagnostics.  If ub != NULL
 * (two-tier mode; needs st->eta/eps/gam), also
 *   ub[b,u] ~= max_h ( s^_h(u) + a'_h eta_u + n_h eps_u + e_h gam_u ),
 *   a'_h = the smallest float >= cert_mult * a_h,
 * the Cauchy-Schwarz upper bound of the full score (Lemma (Index certificate))
 * with the certificate term scaled as in Eq. (trigger): cert_mult =
 * z / sqrt(d_c - r), 1 = the sound bound, smaller = a calibrated trigger (then
 * the bound is no longer a certificate; the bf16 rounding terms stay).
 * cert_mult must be finite and >= 0 (ignored when ub is NULL).
 * key, ub: [B, A] fp32, contiguous.  ws is the workspace vkv_query_prep filled
 * for this step; it must then be passed unchanged to the vkv_select /
 * vkv_admit / vkv_attend calls of the same step.
 */
int vkv_score(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, float* key,
              float* ub, float cert_mult, void* stream);

/*
 * Exact top-k of the index scores: the tier-1 set of the recall tier (Sec. 4.2,
 * the rows whose index score competes for this query; in the task's reading one
 * set per sequence, keyed by the maximum over heads of the first two terms of
 * Eq. (trigger), ties to the lower row index).
 * S_b = the first k rows of [0, A) ordered by (exact index score desc, row
 * index asc), written ascending to sel[b*k .. b*k+k).  The exact score is the
 * fp64 dot product with d ascending; rows whose certified interval (from
 * vkv_score) decides the question are classified from it, the others are
 * re-scored in fp64, so the set equals the fp64 definition bit for bit.
 * theta[b] (fp64) = min over S_b of the exact score (-inf if k = 0).
 * 0 <= k <= A.  Reads the keys vkv_score left in ws and overwrites only its
 * own parts of ws, so it may be called again (another k) after one vkv_score.
 * sel [B, k] int32, theta [B] fp64; errors: VKV_E_ARG (k out of range, NULL
 * output), VKV_E_WORKSPACE.
 */
int vkv_select(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k,
               int32_t* sel, double* theta, void* stream);

/*
 * Two-tier admission (Lemma (Index certificate) with the bf16 rounding of the
 * stored sketch; the fired set of Eq. (trigger) against the k-th selected
 * score): admitted_b = { u in [0, A) \ S_b : UB_u > theta_b } ascending,
 *   UB_u = max_h fl64( s^_h(u) + fma(a'_h, eta_u, fma(n_h, eps_u, e_h gam_u)) ),
 *   a'_h = the smallest float >= cert_mult * a_h.
 * Undecided rows are decided in fp64 as above.  adm [B, cap] int32; adm_count[b]
 * = the true count (may exceed cap; then only the first cap rows are written).
 * Needs mode ROPE or ROPE_DIGEST (the key must contain the exact branch
 * summand), ub from vkv_score, and sel/theta from vkv_select with the same ws.
 * The band shortcut uses ub only if vkv_score was given the same cert_mult;
 * otherwise every row outside S is decided by its exact bound (slower, same
 * result).  May be called again on the same ws.  Soundness (cert_mult = 1)
 * needs ||P||_2 <= 1, which vkv_digest_build certifies.
 */
int vkv_admit(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k,
              const int32_t* sel, const double* theta, const float* ub, float cert_mult,
              int32_t* adm, int32_t* adm_count, int64_t cap, void* stream);

/*
 * Exact attention of every head over the attended multiset of sequence b:
 *   sel[b, 0..k)  ++  [A, T)  ++  adm[b, 0..min(adm_count[b], cap))
 *   s_h(u) = scale * ( q_lat[b,h] . c_u + q_rope[b,h] . r_u )        (576 dims)
 *   out[b,h,:] = RNE_bf16( sum_u softmax_u(s_h) c_u[0:512] )           [B, H, 512]
 *   lse[b,h]   = log sum_u exp(s_h(u))   (natural log)                  [B, H] fp32
 * bf16 MFMA, fp32 accumulation, online softmax, split-KV with an LSE merge
 * (the appendix's kernel mapping: fetched rows are one more split-KV
 * partition).  adm/adm_count may be NULL (cap must then be 0).  An empty set
 * gives out = 0 and lse = -inf.  cap must not exceed the workspace's cap.
 */
int vkv_attend(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k,
               const int32_t* sel, const int32_t* adm, const int32_t* adm_count, int64_t cap,
               float scale, uint16_t* out, float* lse, void* stream);

/* query_prep -> score -> select -> [admit iff adm_count != NULL] -> attend,
 * same arguments as the individual calls (key and ub are the caller's
 * intermediates; cert_mult is used by the two-tier stages only), all queued on
 * `stream`; validates every stage's arguments before it launches anything. */
int vkv_step_run(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k,
                 float* key, float* ub, int32_t* sel, double* theta, int32_t* adm,
                 int32_t* adm_count, int64_t cap, float cert_mult, float scale, uint16_t* out,
                 float* lse, void* stream);

/* ------------------------------------------------- the calibrated trigger */

/*
 * Per head, the maximum over a row list of the exact full score (Sec. 3,
 * Eq. (setup), unscaled; fp64 over the 576 dims, latent then branch) and the
 * row attaining it, ties to the lower row index.  Over the attended tier-1
 * rows (sel[b] and the recent window) it is the trigger threshold s*_h, the
 * tier-1 maximum logit of Sec. 4.2 (its figure: attention max logit s*); over
 * every row of the context it is the causal argmax row of a calibration query.
 *   rows    [B, nrows] int32 (each list in [0, A)), or NULL for the whole archive [0, A)
 *   add_recent != 0: the recent window [A, T) is part of the list
 *   smax    [B, H] fp64 (-inf for an empty list), argmax [B, H] int32 (-1 then)
 * bf16 MFMA screening with a certified band, fp64 for the rows that can hold
 * the maximum: bit for bit the fp64 definition.
 */
int vkv_row_max(vkv_ctx* ctx, const vkv_step* st, const int32_t* rows, int64_t nrows,
                int32_t add_recent, double* smax, int32_t* argmax, void* stream);

/*
 * The calibrated trigger (Sec. 4.2, Eq. (trigger): fetch the archived rows
 * whose trigger score exceeds the tier-1 maximum; the optional top-j cap of
 * Sec. 4.3 and the deployment specification's request lifecycle):
 *   fired_b = { u in [0, A) \ S_b : UB_h(u) > s*_h for some h },
 *   UB_h(u) = fl64( s^_h(u) + fma(a'_h, eta_u, fma(n_h, eps_u, e_h gam_u)) ),
 *   a'_h = the smallest float >= cert_mult * a_h,  cert_mult = z / sqrt(d_c - r),
 * with smax = s*_h [B, H] fp64 (vkv_row_max over S and the recent window).
 * With topj > 0 only the topj fired rows of largest margin max_h (UB_h - s*_h)
 * are kept (ties: the lower row).  fired [B, cap] int32 ascending, fired_count
 * [B] = the number kept (may exceed cap; then cap rows are written).  Needs
 * the step's vkv_query_prep / vkv_score (with ub, the same cert_mult for the
 * band shortcut) / vkv_select on ws.  Decisions are exact: rows the fp32
 * bound cannot decide get fp64 margins.  The fired rows attend as the
 * admitted rows of vkv_attend.  May be repeated on the same ws.
 */
int vkv_trigger(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k,
                const int32_t* sel, const float* ub, float cert_mult, const double* smax,
                int64_t topj, int32_t* fired, int32_t* fired_count, int64_t cap, void* stream);

/*
 * Calibration statistic of the trigger (Sec. 4.2, the z paragraph): for each
 * calibration query b (a sequence of the step: one query of the request
 * against its context) and head h, with u* = argmax[b, h] the causal argmax
 * row (vkv_row_max over the whole context) and s*_h = tier1_max[b, h]:
 *   hard[b, h] = u* is archived and not in sel[b]
 *   zq[b, h]   = (s*_h - idx_h(u*)) / cert_h(u*)  for hard pairs, else 0, with
 *   idx_h(u) = fl64(s^_h(u) + fma(n_h, eps_u, e_h gam_u)),  cert_h(u) = a_h eta_u / sqrt(d_c - r)
 * the inflation at which the trigger score of u* reaches s*_h.  Needs the
 * step's vkv_query_prep on ws.  hard [B, H] int32, zq [B, H] fp64.
 */
int vkv_required_inflation(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k,
                           const int32_t* sel, const double* tier1_max, const int32_t* argmax,
                           int32_t* hard, double* zq, void* stream);

/*
 * The conformal quantile (Sec. 4.2, the z paragraph; Sec. 5.2, the closed-form
 * chain from the recall target tau = tau_num / tau_den, e.g. 9 / 10):
 *   alpha = (1 - tau) / 2,  tau_s = tau / (1 - alpha),
 *   min_hard = ceil(tau_s / (1 - tau_s)),  k = ceil((n + 1) tau_s),
 *   z = the k-th smallest of zq[0 .. n), clamped to [0, zmax]; z = zmax when
 *   n < min_hard or k > n (the quantile does not exist).
 * HOST pointers: zq (the z_q of the hard pairs), z, min_hard, rank (= k, or 0
 * when z is the clamp).  A host-side order statistic; no device work.
 */
int vkv_conformal_z(const double* zq, int64_t n, int64_t tau_num, int64_t tau_den, double zmax,
                    double* z, int64_t* min_hard, int64_t* rank);

/*
 * One step with the calibrated trigger in place of the admission:
 * query_prep -> score (with ub at cert_mult) -> select -> vkv_row_max over
 * S and the recent window (smax, argmax [B, H]: caller buffers, written) ->
 * vkv_trigger -> attend over S, the recent window and the fired rows (the
 * fetched rows join the softmax as exact copies, Lemma (Exchangeability)).
 */
int vkv_step_run_trigger(vkv_ctx* ctx, const vkv_step* st, void* ws, size_t ws_bytes, int64_t k,
                         float* key, float* ub, int32_t* sel, double* theta, float cert_mult,
                         double* smax, int32_t* argmax, int64_t topj, int32_t* fired,
                         int32_t* fired_count, int64_t cap, float scale, uint16_t* out, float* lse,
                         void* stream);

/*
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same step
 * as vkv_step_run (same arguments and results, the same kernels) on a
 * workspace the library owns: a static device array of VKV_STATIC_WS_BYTES per
 * device, held until the process ends.  The call allocates nothing.  Steps
 * whose workspace (vkv_workspace_size) exceeds it are refused with
 * VKV_E_WORKSPACE before anything is launched.  Every call on one device
 * shares that device's array, which keeps the last call's contents (each step
 * initialises what it reads); calls that overlap on one device -- on two
 * streams, or from two host threads -- race and must be serialised by the
 * caller.  The context must belong to the device the buffers live on.
 */
#define VKV_STATIC_WS_BYTES (64u << 20)
int vkv_step_run_static(vkv_ctx* ctx, const vkv_step* st, int64_t k, float* key, float* ub,
                        int32_t* sel, double* theta, int32_t* adm, int32_t* adm_count, int64_t cap,
                        float cert_mult, float scale, uint16_t* out, float* lse, void* stream);

/*
 * The executable row-set invariant (the deployment's per-step row-set
 * assertion, appendix "Measurement integrity: full protocol"), on caller
 * buffers: every sel[b] row lies in the archive [0, A) and the list is strictly
 * ascending; if adm_count != NULL, 0 <= adm_count[b] <= A - k and the first
 * min(adm_count[b], cap) adm[b] rows lie in the archive, strictly ascending
 * and outside sel[b].  Copies the lists to the host and synchronises `stream`.
 * Returns VKV_OK, VKV_E_DEBUG_ROWS naming the first violation, or an argument
 * error.  The same checks run inside vkv_select / vkv_admit / vkv_step_run when
 * VKV_DEBUG_ROWS is set.
 */
int vkv_check_rows(vkv_ctx* ctx, const vkv_step* st, int64_t k, const int32_t* sel,
                   const int32_t* adm, const int32_t* adm_count, int64_t cap, void* stream);

/* enable != 0: vkv_step_run records a pair of HIP events around its score
 * scan, on the call's stream, for up to 512 calls; vkv_score_timing reads
 * them.  Either call clears what was recorded. */
int vkv_set_timing(vkv_ctx* ctx, int enable);

/* Durations in ms of the score scans recorded since timing was enabled or last
 * read, in launch order, into ms[0..max); waits for those events and forgets
 * them.  Returns the number written (>= 0) or a negative VKV_E_* status. */
int vkv_score_timing(vkv_ctx* ctx, float* ms, int max);

#ifdef __cplusplus
}
#endif
#endif /* VKV_H */
