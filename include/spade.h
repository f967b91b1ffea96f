/*
 * spade.h — C ABI of the MI355X (gfx950) block-sparse attention hot path of
 * SPADE (arXiv 2608.03335, "An Input-Adaptive Sparse Attention Engine for Fast
 * Video Diffusion Models Inference").
 *
 * The path (paper §3.3, Head-wise Sparse Attention), one call per step:
 *   spade_block_reorder      blocking / layout transform and its inverse
 *                            (optionally for a group of heads, §3.3 (2))
 *   spade_summarize          Summarizer (block means) + optional SICS (§3.2)
 *   spade_block_summarize    the two above fused into one pass over the raster
 *                            tensors (§3.3 (1)), optionally for a group of heads
 *   spade_estimate_select    inter-block Estimator + Top-K / Top-P index search
 *   spade_block_minmax       max/min Summarizer + optional SICS, from the raster
 *                            tensors (the summaries of the DSA estimators)
 *   spade_compose_select     the full mask: an estimator (mean, DSA, DSA2), the
 *                            Top-K/Top-P rule with optional per-head budgets, the
 *                            intra-block filter, local window and attention sink
 *   spade_policy_budgets     per-head dynamic budgets from the Selected
 *                            Aggregation Score (the policy function, §3.1)
 *   spade_policy_tau         the same for Top-P schemes (per-head mass)
 *   spade_policy_dense       the policy's dense warm-up schedule (host)
 *   spade_policy_split       the policy's static/dynamic budget split (host)
 *   spade_block_sparse_attn  flash block-sparse attention, Eq. (2)
 *   spade_validate_lists     check of block lists (debug aid)
 *   spade_sparse_attn_raster the same on raster tensors (blocking applied on read)
 *   spade_sparse_attn_raster_multi  the same over heads with different blockings
 * and the head-wise blocking-scheme choice (§3.2, Eq. (3)):
 *   spade_candidate_sics     SICS of every candidate blocking in one pass
 *   spade_aggregation_score  per-head Aggregation Score of one candidate scheme
 *   spade_choose_scheme      per-head argmax over the candidates
 *
 * Conventions shared by every call
 *   - All tensor pointers are DEVICE pointers, owned by the caller, contiguous,
 *     16-byte aligned (the one host pointer, a reorder call's head list, is
 *     read before the call returns). The library never allocates, frees or
 *     synchronises, and keeps no state; calls are reentrant and asynchronous on
 *     `stream`.
 *   - Shapes follow the paper's problem statement: B batches, H heads, N tokens
 *     of head dimension d, where the N tokens form a (T, Hs, Ws) latent grid
 *     flattened T-major: token n = (t*Hs + y)*Ws + x (§2.1).
 *   - A blocking scheme (bt, bh, bw) tiles the grid (§3.1, Fig. 3). The block
 *     grid is ceil(T/bt) x ceil(Hs/bh) x ceil(Ws/bw), NB blocks numbered
 *     T-major; BS = bt*bh*bw slots per block. Inside a block the n_b real tokens
 *     occupy slots 0..n_b-1 in raster order of (dt, dy, dx); slots n_b..BS-1 are
 *     padding (only blocks at the grid's far edges have them).
 *   - "Blocked" tensors are [B, H, NB*BS, d]; raster tensors [B, H, N, d].
 *   - Errors: argument checks run on the host before any launch and return a
 *     status (no partial work). A launch failure returns SPADE_ERR_HIP. Device
 *     faults surface at the caller's next synchronisation. spade_last_error()
 *     gives a message for the calling thread's most recent failure.
 *   - Limits: d in {64, 128}; BS <= 256; NB <= 1024 for the selection call and
 *     NB <= 16384 for the attention call.
 *     B, H, T, Hs or Ws equal to 0 is an empty problem: the call returns
 *     SPADE_OK without launching anything (pointers are then not read), except
 *     spade_validate_lists, which still clears its report.
 */
#ifndef SPADE_H
#define SPADE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPADE_OK = 0,
  SPADE_ERR_INVALID_ARG = 1, /* null pointer, bad shape, bad mode/parameter  */
  SPADE_ERR_UNSUPPORTED = 2, /* valid but outside the limits above           */
  SPADE_ERR_WORKSPACE = 3,   /* workspace missing or too small               */
  SPADE_ERR_HIP = 4          /* a HIP launch or query failed                 */
} spade_status;

enum { SPADE_BF16 = 0, SPADE_FP32 = 1 };  /* element type of spade_block_reorder */
enum { SPADE_TOPK = 0, SPADE_TOPP = 1 };  /* row rule of spade_estimate_select   */
enum { SPADE_EST_MEAN = 0, SPADE_EST_DSA = 1, SPADE_EST_DSA2 = 2 };  /* inter-block estimator */
enum { SPADE_INTRA_NONE = 0, SPADE_INTRA_THRESHOLD = 1, SPADE_INTRA_TOPK = 2 };  /* intra filter */

/* Problem geometry: batch, heads, head dim; latent grid; blocking scheme. */
typedef struct {
  int32_t B, H, d;
  int32_t T, Hs, Ws;
  int32_t bt, bh, bw;
} spade_geom;

/*
 * Blocking (layout transform) and its inverse — paper §3.3: Q, K, V are
 * rearranged into the blocked layout of the selected scheme for intra-block
 * contiguity, and output blocks are restored to the original layout. With a
 * head list this is §3.3 optimisation (2), head grouping: the heads that share
 * one blocking scheme are gathered from (scattered back to) the full raster
 * tensor in the same pass, so each group runs as one [B, n_heads, ...] problem.
 *
 *   heads, n_heads: HOST array of n_heads distinct head indices in [0, H),
 *                 1 <= n_heads <= 64, read before the call returns; or
 *                 heads == NULL with n_heads == 0 for all H heads in order.
 *                 A non-null list with n_heads == 0 moves nothing. Let
 *                 n = n_heads (H when heads is NULL) and h_k = heads[k] (k).
 *   inverse == 0: x is raster [B,H,N,d], y is blocked [B,n,NB*BS,d];
 *                 y[b, k, p*BS+s, :] = x[b, h_k, token(p,s), :] for real slots,
 *                 0 for padding slots (every element of y is written).
 *   inverse == 1: x is blocked [B,n,NB*BS,d], y is raster [B,H,N,d]; only the
 *                 rows of the listed heads are written; padding slots of x are
 *                 not read.
 *   dtype: SPADE_BF16 (2-byte elements) or SPADE_FP32 (4-byte). Bit-exact copy.
 *   x and y must not overlap.
 */
spade_status spade_block_reorder(const spade_geom* g, const void* x, void* y,
                                 int32_t dtype, int32_t inverse, const int32_t* heads,
                                 int32_t n_heads, hipStream_t stream);

/*
 * Summarizer and intra-block estimator — paper §3.1 (Summarizer = mean,
 * MEAN-SPADE) and §3.2, Eq. (4)/(5), Alg. 1 (SICS).
 *
 *   qb, kb:       blocked bf16 [B,H,NB*BS,d] (output of spade_block_reorder).
 *   qbar, kbar:   out, fp64 [B,H,NB,d]: mean over each block's real tokens
 *                 (accumulated in fp64).
 *   sics_q, sics_k: out, nullable, fp64 [B,H,NB]: SICS of each block's real
 *                 rows, computed as |sum_k q_k/|q_k||^2 (equal to Eq. (4); a
 *                 zero row contributes nothing). Pass both or neither.
 */
spade_status spade_summarize(const spade_geom* g, const void* qb, const void* kb,
                             double* qbar, double* kbar, double* sics_q, double* sics_k,
                             hipStream_t stream);

/*
 * Blocking, Summarizer and intra-block estimator fused — paper §3.3 optimisation
 * (1): one pass reads each block's rows of Q and K from the raster layout and
 * produces what spade_block_reorder (inverse == 0) and spade_summarize produce,
 * bit for bit for the blocked copies and the same fp64 reductions for the
 * summaries. With qb/kb NULL nothing is written to the blocked layout: the call
 * then evaluates a blocking scheme (summaries, SICS) straight from the raster
 * tensors, as the head-wise scheme choice of §3.2 needs for every candidate.
 *
 *   q, k:         raster bf16 [B,H,N,d].
 *   qb, kb:       out, nullable (both or neither), blocked bf16 [B,n,NB*BS,d].
 *   qbar, kbar:   out, nullable (both or neither), fp64 [B,n,NB,d].
 *   sics_q, sics_k: out, nullable (both or neither), fp64 [B,n,NB].
 *   heads, n_heads: head list as in spade_block_reorder; n = n_heads (H if NULL).
 *   At least one output pair must be given. Outputs must not alias the inputs.
 */
spade_status spade_block_summarize(const spade_geom* g, const void* q, const void* k, void* qb,
                                   void* kb, double* qbar, double* kbar, double* sics_q,
                                   double* sics_k, const int32_t* heads, int32_t n_heads,
                                   hipStream_t stream);

/*
 * SICS of every candidate blocking in one pass — paper §3.2: the head-wise scheme
 * choice scores each candidate by Eq. (3), the sum of its blocks' SICS (Eq. (4)/(5)),
 * for Q and for K. Reading Q and K once for all candidates: each token's unit vector
 * is added into a cell of the candidates' common refinement, and every candidate
 * block's sum of unit vectors is the sum of its cells.
 *
 *   geoms, n_geoms: the candidate blockings (1 <= n_geoms <= 8); all share B, H, d
 *            and the grid (T, Hs, Ws).
 *   q, k:    raster bf16 [B,H,N,d].
 *   sics_q, sics_k: HOST arrays of n_geoms DEVICE pointers; entry c receives fp64
 *            [B,H,NB_c], the SICS spade_block_summarize computes under geoms[c] (up
 *            to rounding: same fp64 unit rows, summed cell by cell).
 *   Summation orders are fixed (tokens in raster order inside a cell, cells in
 *   (t, y, x) order inside a block): deterministic.
 *   Returns SPADE_ERR_UNSUPPORTED when the candidates' block boundaries cut an axis
 *   of their common region (per axis the least common multiple of the extents) into
 *   more than 48 cells, or a region's cells need more than 144 KiB of fp64 sums
 *   (cells x d x 8 bytes); the caller then scores the candidates one at a time.
 */
spade_status spade_candidate_sics(const spade_geom* geoms, int32_t n_geoms, const void* q,
                                  const void* k, double* const* sics_q, double* const* sics_k,
                                  hipStream_t stream);

/*
 * Aggregation Score of one blocking-scheme candidate — paper §3.2, Eq. (3):
 * a head's AS under a scheme is the sum over its blocks of SICS, for Q and for K.
 *
 *   sics_q, sics_k: fp64 [B,H,NB], as written by spade_summarize under g's scheme.
 *   as_q, as_k:   out, nullable, fp64 [B,H]: sum_p SICS_p / sum_p n_p^2, where n_p
 *                 is block p's real-token count. The divisor is the score of a
 *                 block whose vectors are all parallel, so candidates with
 *                 different block sizes or padding compare on one scale (for
 *                 equal unpadded blocks it is a constant factor). The raw Eq. (3)
 *                 sum is as_q * sum_p n_p^2.
 *   as_qk:        out, fp64 [B,H]: as_q + as_k, the score spade_choose_scheme ranks.
 *   Each output is a fixed-order reduction (deterministic).
 */
spade_status spade_aggregation_score(const spade_geom* g, const double* sics_q,
                                     const double* sics_k, double* as_q, double* as_k,
                                     double* as_qk, hipStream_t stream);

/*
 * Selected Blocking Scheme per head — paper §3.2: each head takes the candidate
 * with the highest Aggregation Score.
 *
 *   as_qk:  fp64 [C,B,H]: row c is spade_aggregation_score's as_qk for candidate c.
 *   choice: out, int32 [H]: per head, the candidate c with the largest batch mean
 *           (1/B) sum_b as_qk[c,b,h]; ties go to the lower c (a NaN never wins
 *           over candidate 0's value).
 *   best:   out, nullable, fp64 [H]: that mean (the Selected Aggregation Score).
 *   1 <= C <= 1024. B or H equal to 0 is a no-op.
 */
spade_status spade_choose_scheme(const double* as_qk, int32_t C, int32_t B, int32_t H,
                                 int32_t* choice, double* best, hipStream_t stream);

/*
 * Inter-block Estimator + Top-K / Top-P index search — paper §3.3 (inter-block
 * importance matrix of size NB x NB from the Q/K summaries, filtered by Top-K
 * or Top-P) with §3.1's Top-K/Top-P mode parameter.
 *
 *   score(i, j) = <qbar_i, kbar_j> * scale, in fp64 (scale is normally 1/sqrt(d)).
 *   Each row (b, h, i) ranks blocks j by (score descending, j ascending) and keeps
 *     SPADE_TOPK: the first min(topk, NB) blocks (topk >= 1; tau ignored);
 *     SPADE_TOPP: the shortest prefix whose softmax mass over the row's scores
 *                 reaches tau, at least one block; tau in (0, 1], tau == 1 keeps
 *                 every block (topk ignored).
 *   counts:  out, int32 [B,H,NB]: number of kept blocks per row.
 *   indices: out, int32 [B,H,NB,NB]: row (b,h,i) holds its kept block indices in
 *            ascending order in entries 0..counts-1; later entries are not written.
 *   scores:  out, nullable, fp64 [B,H,NB,NB]: the score matrix (for checking).
 *   Requires NB <= 1024.
 */
spade_status spade_estimate_select(const spade_geom* g, const double* qbar, const double* kbar,
                                   int32_t mode, int32_t topk, double tau, double scale,
                                   int32_t* counts, int32_t* indices, double* scores,
                                   hipStream_t stream);

/*
 * Max/min Summarizer and intra-block estimator from the raster tensors — paper
 * §3.1 (the Summarizer Expression reduces over a block's positions with max, min
 * or mean; the DSA-SPADE and DSA2-SPADE estimators take the max and min
 * summaries) and §3.2 (SICS), in one pass over each block's rows (§3.3 (1)).
 *
 *   q, k:         raster bf16 [B,H,N,d].
 *   qmax, qmin, kmax, kmin: out, fp64 [B,n,NB,d]: elementwise max / min over each
 *                 block's real tokens (exact).
 *   sics_q, sics_k: out, nullable (both or neither), fp64 [B,n,NB]: SICS, bit-equal
 *                 to spade_block_summarize's.
 *   heads, n_heads: head list as in spade_block_reorder; n = n_heads (H if NULL).
 */
spade_status spade_block_minmax(const spade_geom* g, const void* q, const void* k, double* qmax,
                                double* qmin, double* kmax, double* kmin, double* sics_q,
                                double* sics_k, const int32_t* heads, int32_t n_heads,
                                hipStream_t stream);

/* Block summaries a selection call reads (device pointers, fp64, [B,H,NB,d] or
 * [B,H,NB] for SICS); each estimator and filter names the fields it needs. */
typedef struct {
  const double* qbar;   /* SPADE_EST_MEAN: block means of Q and K */
  const double* kbar;
  const double* qmax;   /* SPADE_EST_DSA, SPADE_EST_DSA2: block max / min */
  const double* qmin;
  const double* kmax;
  const double* kmin;
  const double* sics_q; /* intra-block filter: SICS of the Q and K blocks */
  const double* sics_k;
} spade_summaries;

/* One head-wise sparsity scheme (paper §3.1: estimator expression, Top-K/Top-P
 * inter value, intra value, local-window length, attention-sink length). Host
 * struct, read before the call returns; the per-head arrays are device memory. */
typedef struct {
  int32_t estimator;     /* SPADE_EST_MEAN | SPADE_EST_DSA | SPADE_EST_DSA2 */
  int32_t mode;          /* inter rule: SPADE_TOPK | SPADE_TOPP */
  int32_t topk;          /* SPADE_TOPK: blocks per row (>= 1 unless topk_per_head) */
  double tau;            /* SPADE_TOPP: mass in (0, 1] (unless tau_per_head) */
  double scale;          /* logit scale of the estimate, normally 1/sqrt(d) */
  const int32_t* topk_per_head; /* nullable DEVICE int32 [H]: replaces topk, each
                                   value clamped to [1, NB] */
  const double* tau_per_head;   /* nullable DEVICE fp64 [H]: replaces tau; >= 1 keeps
                                   every block, <= 0 or NaN keeps the top block */
  int32_t intra;         /* SPADE_INTRA_NONE | _THRESHOLD | _TOPK */
  int32_t intra_topk;    /* _TOPK: how many least coherent blocks per head (>= 0) */
  double intra_theta;    /* _THRESHOLD: coherence bound */
  int32_t window[3];     /* local window radii in blocks along (t, y, x); any
                            negative radius: no window */
  int64_t sink_tokens;   /* attention-sink length in raster tokens (>= 0) */
} spade_mask_spec;

/*
 * Full mask composition — paper §3.3: the inter-block importance matrix from the
 * Estimator Expression, filtered by Top-K or Top-P; intra-block scores
 * broadcast and OR-combined with it; the result united with the local-window
 * and attention-sink masks; §3.1: the sparsity-ratio scheme's parts, and
 * head-wise budgets (the policy function's output per head).
 *
 *   Estimate, fp64, times scale:
 *     MEAN: <qbar_i, kbar_j>;
 *     DSA:  sum_c max(m_c kmax_jc, m_c kmin_jc) with m = (qmax_i + qmin_i)/2, the
 *           largest <m, k> over the box spanned by block j's keys;
 *     DSA2: sum_c of the largest product of {qmax_ic, qmin_ic} and
 *           {kmax_jc, kmin_jc}: an upper bound of every logit of the block pair.
 *   Inter rule per row as in spade_estimate_select (the head's per-head k or tau
 *   when given).
 *   Block j is kept in row i when the inter rule keeps it, or
 *     - the intra filter marks query block i (its whole row is kept) or key
 *       block j (its whole column). A block's coherence is SICS / n_b^2; the
 *       filter marks coherence < intra_theta (_THRESHOLD) or the intra_topk least
 *       coherent blocks of the head, ties to the lower index (_TOPK);
 *     - the block-grid coordinates of i and j differ by at most window[] on
 *       every axis;
 *     - block j holds one of the first sink_tokens raster tokens.
 *   counts, indices, scores: as in spade_estimate_select (scores = the estimate).
 *   Requires NB <= 1024. With everything but the inter rule off and the MEAN
 *   estimator the result equals spade_estimate_select's.
 */
spade_status spade_compose_select(const spade_geom* g, const spade_mask_spec* spec,
                                  const spade_summaries* sum, int32_t* counts, int32_t* indices,
                                  double* scores, hipStream_t stream);

/*
 * Head-wise budgets of the policy function — paper §3.1 (the policy function maps
 * each head's Selected Aggregation Score and the inference state to its
 * sparsity-ratio scheme) and §4 (the policy study: budgets negatively correlated
 * with the score). The output feeds spade_mask_spec.topk_per_head.
 *
 *   as_best: fp64 [H] device: the Selected Aggregation Score per head (the `best`
 *            output of spade_choose_scheme).
 *   heads, n_heads: HOST list of heads as in spade_block_reorder (NULL: all H in
 *            order); n = n_heads (H if NULL). Read before the call returns.
 *   k_dyn:   mean dynamic blocks per row (>= 1); NB: upper clamp (>= 1).
 *   k_out:   out, int32 [n] device, in list order:
 *            k = clamp(floor(n * k_dyn * w / W + 1/2), 1, NB) with w = 1 / AS of the
 *            head (0 when AS <= 0) and W the sum of the listed heads' w in list
 *            order (W = 0: every head gets clamp(k_dyn, 1, NB)). fp64, correctly
 *            rounded operations in a fixed order: the result is deterministic.
 *   0 <= H <= 65535; H == 0 or an empty list is a no-op.
 */
spade_status spade_policy_budgets(const double* as_best, int32_t H, const int32_t* heads,
                                  int32_t n_heads, int32_t k_dyn, int32_t NB, int32_t* k_out,
                                  hipStream_t stream);

/*
 * Head-wise Top-P mass of the policy function — paper §3.1 and §4 (as for
 * spade_policy_budgets) for a Top-P scheme. The output feeds
 * spade_mask_spec.tau_per_head.
 *
 *   as_best, H, heads, n_heads: as for spade_policy_budgets.
 *   tau:     the scheme's mass, in (0, 1].
 *   tau_out: out, fp64 [n] device, in list order: tau_k = 1 - n (1 - tau) a_k / S with
 *            a_k = max(AS of the head, 0) and S the sum of the listed heads' a in list
 *            order (S = 0: every head gets tau). The dropped mass is spread over the
 *            heads in proportion to their score, so it averages 1 - tau; a value
 *            <= 0 keeps only each row's top block. fp64, correctly rounded
 *            operations in a fixed order: deterministic.
 *   H == 0 or an empty list is a no-op.
 */
spade_status spade_policy_tau(const double* as_best, int32_t H, const int32_t* heads,
                              int32_t n_heads, double tau, double* tau_out, hipStream_t stream);

enum { SPADE_TASK_T2V = 0, SPADE_TASK_I2V = 1 };  /* denoising task of spade_policy_dense */

/*
 * Warm-up schedule of the policy function — paper §4.1 (configurations): full
 * attention for the first 30% of the denoising steps in text-to-video and 25% in
 * image-to-video; SPADE-Turbo only for the first step. Host function (no GPU).
 *
 *   step:   0-based denoising step, 0 <= step < n_steps.
 *   task:   SPADE_TASK_T2V or SPADE_TASK_I2V; turbo: nonzero for SPADE-Turbo.
 *   dense:  out (host): 1 when the step runs full attention: step < ceil(0.3 n_steps)
 *           (t2v) or step < ceil(0.25 n_steps) (i2v); Turbo: step < 1. Else 0.
 */
spade_status spade_policy_dense(int32_t step, int32_t n_steps, int32_t task, int32_t turbo,
                                int32_t* dense);

/*
 * Static/dynamic budget split of a head-wise scheme — paper §4.1: Func 0 gives
 * the dynamic and static parts a 30:1 budget, Func 1 about 80% dynamic. Host
 * function (no GPU).
 *
 *   k_total: blocks per row (>= 1); func: 0 or 1.
 *   The static share, round(k_total / 31) (Func 0) or round(k_total / 5) (Func 1),
 *   halves rounded up, buys the largest window of the radius ladder
 *   (t, y, x) = (0,0,0), (0,0,1), (0,1,1), (1,1,1), (1,1,2), (1,2,2), (2,2,2)
 *   (1, 3, 9, 27, 45, 75, 125 blocks) that fits; the dynamic Top-K keeps the rest.
 *   window:  out (host) int32 [3]: the radii, or -1, -1, -1 when no window fits.
 *   window_blocks: out (host): the window's block count (0 without a window).
 *   k_dyn:   out (host): k_total - window_blocks.
 */
spade_status spade_policy_split(int32_t k_total, int32_t func, int32_t* window,
                                int32_t* window_blocks, int32_t* k_dyn);

/*
 * Check of block lists (a debug aid; the attention calls accept any lists and skip
 * what is malformed). The lists are the block mask in the row-wise sparse form the
 * attention walks (§3.3 optimisation (3)): per query block, the kept key blocks in
 * ascending order. Each row (b, h, i) passes when 0 <= counts <= NB and its listed
 * indices lie in [0, NB) and strictly ascend.
 *
 *   counts, indices: int32 [B,H,NB] and [B,H,NB,NB], as spade_estimate_select writes.
 *   report:  out, device int32[4]: [0] the number of failing rows; [1] the lowest
 *            failing row, numbered (b*H + h)*NB + i (INT32_MAX when none); [2] the
 *            OR of the failure bits of every failing row (SPADE_LIST_*); [3] 0.
 *            Written on `stream` by two launches (a clear, then the check).
 *   Errors: as for every call, the geometry's (SPADE_ERR_INVALID_ARG,
 *           SPADE_ERR_UNSUPPORTED); SPADE_ERR_INVALID_ARG for a null pointer (counts
 *           and indices may be null for an empty problem, report may not);
 *           SPADE_ERR_UNSUPPORTED when B*H*NB exceeds 2^31 - 1. For an empty problem
 *           the report is still written (no failing rows).
 */
enum { SPADE_LIST_BAD_COUNT = 1, SPADE_LIST_BAD_INDEX = 2, SPADE_LIST_NOT_ASCENDING = 4 };
spade_status spade_validate_lists(const spade_geom* g, const int32_t* counts,
                                  const int32_t* indices, int32_t* report, hipStream_t stream);

/*
 * Scratch bytes spade_block_sparse_attn and spade_sparse_attn_raster need for
 * their work schedule (§3.3 optimisation (3): the mask preprocessed into a ranked
 * layout, heads of similar density co-scheduled), and spade_sparse_attn_raster_multi
 * for the same: 16 bytes per (batch, head) pair, 0 for an empty problem or more
 * than 4096 pairs (grid order then).
 */
size_t spade_attn_workspace_bytes(const spade_geom* g);

/*
 * Flash block-sparse attention — paper Eq. (2) with block mask M (0 on kept
 * block pairs, -inf elsewhere) and §3.3 optimisation (3): online softmax over the
 * kept K/V blocks of each query block, never materialising the score matrix.
 *
 *   qb, kb, vb: blocked bf16 [B,H,NB*BS,d].
 *   counts, indices: the block lists, in the layout spade_estimate_select writes.
 *            Any lists are accepted; entries outside [0, NB) are skipped and
 *            counts above NB are clamped, so malformed lists cannot fault.
 *            Each kept block contributes its real key slots only.
 *   scale:   logit scale (normally 1/sqrt(d)).
 *   ob:      out, bf16 [B,H,NB*BS,d]: real query slots hold the attention output,
 *            padding slots are written 0. A row with no kept block gets 0.
 *   lse:     out, nullable, fp32 [B,H,NB*BS]: natural-log softmax denominator
 *            (max included) per real query slot; padding slots are not written.
 *   workspace: device scratch of at least spade_attn_workspace_bytes(g) bytes,
 *            16-byte aligned (contents on entry do not matter). The call ranks the
 *            (batch, head) pairs there by their heaviest row, then their total kept
 *            blocks, and dispatches the heaviest first, so long rows do not form
 *            the launch's tail; results do not depend on the order. A workspace
 *            serves one call at a time (calls that share one must be ordered).
 *   bf16 MFMA with fp32 accumulation; softmax in fp32; P rounded to bf16 for
 *   the P*V product; output rounded to bf16 (round to nearest even).
 */
spade_status spade_block_sparse_attn(const spade_geom* g, const void* qb, const void* kb,
                                     const void* vb, const int32_t* counts,
                                     const int32_t* indices, double scale, void* ob, float* lse,
                                     void* workspace, size_t workspace_bytes,
                                     hipStream_t stream);

/*
 * Flash block-sparse attention on raster tensors — the same computation as
 * spade_block_sparse_attn, with the blocking applied while reading (each key or
 * query slot is fetched from its raster token) and the output written back in
 * raster order: §3.3's rearrangement and restoration without blocked copies.
 *
 *   q, k, v: raster bf16 [B,H,N,d].
 *   counts, indices, scale, workspace: as for spade_block_sparse_attn.
 *   o:       out, raster bf16 [B,H,N,d]; every token row is written.
 *   lse:     out, nullable, fp32 [B,H,N].
 *   Requires N*d*2 < 2^31 (one head's rows addressable with 32-bit offsets).
 *   Results equal spade_block_sparse_attn's on the blocked copies, bit for bit.
 */
spade_status spade_sparse_attn_raster(const spade_geom* g, const void* q, const void* k,
                                      const void* v, const int32_t* counts,
                                      const int32_t* indices, double scale, void* o, float* lse,
                                      void* workspace, size_t workspace_bytes,
                                      hipStream_t stream);

/*
 * spade_sparse_attn_raster without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Arguments, results and errors are those of
 * spade_sparse_attn_raster, bit for bit; the schedule's scratch (the head ranking,
 * 16 bytes per (batch, head) pair) lives in a 64 KiB array the library holds in
 * each GPU's memory until the process ends, so the call allocates nothing. Its
 * address is looked up once per device, on the first call there (a failed lookup
 * returns SPADE_ERR_HIP). The ranking rewrites every scratch byte it reads, so no
 * clearing is needed; a problem whose schedule needs more scratch than the array
 * holds returns SPADE_ERR_UNSUPPORTED (with at most 4096 pairs none does).
 * All calls on one GPU share the array: calls that may overlap on that GPU (other
 * streams, other threads) race and must be ordered by the caller.
 */
spade_status spade_sparse_attn_raster_noalloc(const spade_geom* g, const void* q, const void* k,
                                              const void* v, const int32_t* counts,
                                              const int32_t* indices, double scale, void* o,
                                              float* lse, hipStream_t stream);

/* Block lists of one head for spade_sparse_attn_raster_multi (device pointers). */
typedef struct {
  int32_t scheme;           /* index of the head's blocking among the call's geometries */
  const int32_t* counts;    /* counts of (batch 0, this head): [NB] of its blocking */
  const int32_t* indices;   /* kept lists of (batch 0, this head): [NB, NB] */
  int64_t counts_bstride;   /* elements from one batch element's counts to the next */
  int64_t indices_bstride;  /* elements from one batch element's lists to the next */
} spade_head_lists;

/*
 * Head-wise sparse attention over heads with different blockings — paper §3.2
 * (each head runs under its own Selected Blocking Scheme) and §3.3 (2) (heads
 * sharing work are launched together): the raster attention of
 * spade_sparse_attn_raster for every head in one pass over the shared raster
 * Q, K, V, each head addressed through its own blocking.
 *
 *   geoms, n_geoms: the candidate blockings (1 <= n_geoms <= 8); all must share B,
 *            H, d and the grid (T, Hs, Ws). H <= 64.
 *   heads:   HOST array [H]: per head its blocking and block lists (any layout, e.g.
 *            per-group buffers written by spade_compose_select with a head list).
 *   q, k, v, scale, o, lse: as for spade_sparse_attn_raster.
 *   workspace: spade_attn_workspace_bytes(&geoms[0]) bytes, 16-byte aligned
 *            (contents on entry do not matter); each launch ranks its heads there
 *            per batch element, heaviest first, as spade_block_sparse_attn does.
 *   Each head's output equals spade_sparse_attn_raster's under its own blocking,
 *   bit for bit. Heads whose blocks need the same number of 32-row waves
 *   (ceil(BS/32)) run in one launch: one launch in total when all blockings
 *   share it.
 */
spade_status spade_sparse_attn_raster_multi(const spade_geom* geoms, int32_t n_geoms,
                                            const spade_head_lists* heads, const void* q,
                                            const void* k, const void* v, double scale, void* o,
                                            float* lse, void* workspace, size_t workspace_bytes,
                                            hipStream_t stream);

/* Static, human-readable name of a status code. */
const char* spade_status_string(spade_status s);

/* Message describing the calling thread's most recent non-OK status ("" if none). */
const char* spade_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SPADE_H */
