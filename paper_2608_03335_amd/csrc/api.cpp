// C-ABI entry points: host-side argument validation, then the kernel launchers.
// Validation never touches the HIP runtime, so every error path runs without a GPU.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <set>
#include <utility>

#include "spade.h"
#include "spade_internal.h"

namespace spade {

hipError_t ensure_dynamic_lds(const void* fn, int bytes) {
  static std::mutex mu;
  static std::set<std::pair<const void*, int>> done;  // (kernel, device) already raised
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  if (done.count({fn, dev})) return hipSuccess;
  e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess) done.insert({fn, dev});
  return e;
}

}  // namespace spade

namespace {

thread_local char g_last_error[512] = "";

spade_status fail(spade_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Checks the geometry and fills `dg`. Sets *empty when there is nothing to do.
spade_status check_geom(const spade_geom* g, spade::DevGeom* dg, bool* empty) {
  if (!g) return fail(SPADE_ERR_INVALID_ARG, "geometry pointer is null");
  if (g->B < 0 || g->H < 0 || g->T < 0 || g->Hs < 0 || g->Ws < 0)
    return fail(SPADE_ERR_INVALID_ARG, "negative size (B=%d H=%d T=%d Hs=%d Ws=%d)", g->B, g->H,
                g->T, g->Hs, g->Ws);
  if (g->bt < 1 || g->bh < 1 || g->bw < 1)
    return fail(SPADE_ERR_INVALID_ARG, "block dims must be >= 1 (got %d,%d,%d)", g->bt, g->bh,
                g->bw);
  if (g->d != 64 && g->d != 128)
    return fail(SPADE_ERR_UNSUPPORTED, "head dim d=%d not supported (64 or 128)", g->d);
  const int64_t BS = int64_t(g->bt) * g->bh * g->bw;
  if (BS > spade::kMaxBS)
    return fail(SPADE_ERR_UNSUPPORTED, "block size bt*bh*bw=%lld exceeds %d", (long long)BS,
                spade::kMaxBS);
  *empty = (g->B == 0 || g->H == 0 || g->T == 0 || g->Hs == 0 || g->Ws == 0);
  dg->B = g->B; dg->H = g->H; dg->d = g->d;
  dg->T = g->T; dg->Hs = g->Hs; dg->Ws = g->Ws;
  dg->bt = g->bt; dg->bh = g->bh; dg->bw = g->bw;
  dg->nT = (g->T + g->bt - 1) / g->bt;
  dg->nH = (g->Hs + g->bh - 1) / g->bh;
  dg->nW = (g->Ws + g->bw - 1) / g->bw;
  const int64_t NB = int64_t(dg->nT) * dg->nH * dg->nW;
  const int64_t N = int64_t(g->T) * g->Hs * g->Ws;
  dg->N = N;
  dg->BS = int(BS);
  // Offsets are 64-bit in the kernels; keep per-head block counts and grid
  // dimensions inside int32 and the largest tensor inside 2^40 elements.
  if (NB > (int64_t(1) << 30) || N > (int64_t(1) << 31))
    return fail(SPADE_ERR_UNSUPPORTED, "grid too large (N=%lld NB=%lld)", (long long)N,
                (long long)NB);
  const int64_t rows = int64_t(g->B) * g->H * NB * BS;
  if (rows * g->d > (int64_t(1) << 40) || int64_t(g->B) * g->H > 65535)
    return fail(SPADE_ERR_UNSUPPORTED, "tensor too large (B*H*NB*BS*d)");
  dg->NB = int(NB);
  return SPADE_OK;
}

// Reads a host head list (NULL = all heads) into the by-value map the kernels take.
spade_status parse_heads(const spade::DevGeom& dg, const int32_t* heads, int32_t n_heads,
                         spade::HeadMap* hm) {
  hm->n = dg.H;
  hm->ident = 1;
  if (heads == nullptr) {
    if (n_heads != 0)
      return fail(SPADE_ERR_INVALID_ARG, "n_heads must be 0 when heads is null (got %d)", n_heads);
    return SPADE_OK;
  }
  if (n_heads < 0 || n_heads > spade::kMaxHeadList)
    return fail(SPADE_ERR_INVALID_ARG, "n_heads must lie in [0, %d] (got %d)", spade::kMaxHeadList,
                n_heads);
  hm->n = n_heads;
  hm->ident = 0;
  for (int k = 0; k < n_heads; ++k) {
    if (heads[k] < 0 || heads[k] >= dg.H)
      return fail(SPADE_ERR_INVALID_ARG, "heads[%d]=%d outside [0, H=%d)", k, heads[k], dg.H);
    for (int j = 0; j < k; ++j)
      if (heads[j] == heads[k]) return fail(SPADE_ERR_INVALID_ARG, "head %d listed twice", heads[k]);
    hm->h[k] = heads[k];
  }
  return SPADE_OK;
}

spade_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return SPADE_OK;
  return fail(SPADE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

spade_status sparse_attn(const spade_geom* g, const void* q, const void* k, const void* v,
                         const int32_t* counts, const int32_t* indices, double scale, void* o,
                         float* lse, void* workspace, size_t workspace_bytes, bool raster,
                         hipStream_t stream) {
  spade::DevGeom dg;
  bool empty = false;
  spade_status st = check_geom(g, &dg, &empty);
  if (st != SPADE_OK) return st;
  if (!(isfinite(scale) && scale > 0.0))
    return fail(SPADE_ERR_INVALID_ARG, "scale must be finite and > 0 (got %g)", scale);
  if (!empty && dg.NB > spade::kMaxAttnNB)
    return fail(SPADE_ERR_UNSUPPORTED, "NB=%d exceeds the attention limit %d", dg.NB,
                spade::kMaxAttnNB);
  if (!empty && raster && dg.N * int64_t(dg.d) * 2 >= (int64_t(1) << 31))
    return fail(SPADE_ERR_UNSUPPORTED, "raster attention needs N*d*2 < 2^31 bytes per head");
  if (empty) return SPADE_OK;
  if (!q || !k || !v || !counts || !indices || !o)
    return fail(SPADE_ERR_INVALID_ARG, "q, k, v, counts, indices and o must be non-null");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
    return fail(SPADE_ERR_INVALID_ARG, "q, k, v and o must be 16-byte aligned");
  const size_t need = spade::attn_workspace_bytes(dg);
  if (workspace_bytes < need || (need > 0 && (workspace == nullptr || !aligned16(workspace))))
    return fail(SPADE_ERR_WORKSPACE, "16-byte aligned workspace of %zu bytes needed, %zu given",
                need, workspace_bytes);
  return hip_status(spade::launch_block_sparse_attn(dg, q, k, v, counts, indices, float(scale), o,
                                                    lse, workspace, raster, stream),
                    "sparse attention launch");
}
}  // namespace

extern "C" {

const char* spade_status_string(spade_status s) {
  switch (s) {
    case SPADE_OK: return "SPADE_OK";
    case SPADE_ERR_INVALID_ARG: return "SPADE_ERR_INVALID_ARG";
    case SPADE_ERR_UNSUPPORTED: return "SPADE_ERR_UNSUPPORTED";
    case SPADE_ERR_WORKSPACE: return "SPADE_ERR_WORKSPACE";
    case SPADE_ERR_HIP: return "SPADE_ERR_HIP";
  }
  return "SPADE_ERR_UNKNOWN";
}

const char* spade_last_error(void) { return g_last_error; }

spade_status spade_block_reorder(const spade_geom* g, const void* x, void* y, int32_t dtype,
                                 int32_t inverse, const int32_t* heads, int32_t n_heads,
                                 hipStream_t stream) {
  spade::DevGeom dg;
  bool empty = false;
  spade_status st = check_geom(g, &dg, &empty);
  if (st != SPADE_OK) return st;
  if (dtype != SPADE_BF16 && dtype != SPADE_FP32)
    return fail(SPADE_ERR_INVALID_ARG, "dtype must be SPADE_BF16 or SPADE_FP32 (got %d)", dtype);
  if (inverse != 0 && inverse != 1)
    return fail(SPADE_ERR_INVALID_ARG, "inverse must be 0 or 1 (got %d)", inverse);
  spade::HeadMap hm;
  st = parse_heads(dg, heads, n_heads, &hm);
  if (st != SPADE_OK) return st;
  if (empty || hm.n == 0) return SPADE_OK;
  if (!x || !y) return fail(SPADE_ERR_INVALID_ARG, "x and y must be non-null");
  if (!aligned16(x) || !aligned16(y))
    return fail(SPADE_ERR_INVALID_ARG, "x and y must be 16-byte aligned");
  if (x == y) return fail(SPADE_ERR_INVALID_ARG, "x and y must not alias");
  const int esize = dtype == SPADE_BF16 ? 2 : 4;
  return hip_status(spade::launch_reorder(dg, x, y, esize, inverse, hm, stream), "reorder launch");
}

spade_status spade_summarize(const spade_geom* g, const void* qb, const void* kb, double* qbar,
                             double* kbar, double* sics_q, double* sics_k, hipStream_t stream) {
  spade::DevGeom dg;
  bool empty = false;
  spade_status st = check_geom(g, &dg, &empty);
  if (st != SPADE_OK) return st;
  if ((sics_q == nullptr) != (sics_k == nullptr))
    return fail(SPADE_ERR_INVALID_ARG, "sics_q and sics_k must both be given or both be null");
  if (empty) return SPADE_OK;
  if (!qb || !kb || !qbar || !kbar)
    return fail(SPADE_ERR_INVALID_ARG, "qb, kb, qbar and kbar must be non-null");
  if (!aligned16(qb) || !aligned16(kb) || !aligned16(qbar) || !aligned16(kbar))
    return fail(SPADE_ERR_INVALID_ARG, "qb, kb, qbar and kbar must be 16-byte aligned");
  return hip_status(spade::launch_summarize(dg, qb, kb, qbar, kbar, sics_q, sics_k, stream),
                    "summarize launch");
}

spade_status spade_block_summarize(const spade_geom* g, const void* q, const void* k, void* qb,
                                   void* kb, double* qbar, double* kbar, double* sics_q,
                                   double* sics_k, const int32_t* heads, int32_t n_heads,
                                   hipStream_t stream) {
  spade::DevGeom dg;
  bool empty = false;
  spade_status st = check_geom(g, &dg, &empty);
  if (st != SPADE_OK) return st;
  if ((qb == nullptr) != (kb == nullptr))
    return fail(SPADE_ERR_INVALID_ARG, "qb and kb must both be given or both be null");
  if ((qbar == nullptr) != (kbar == nullptr))
    return fail(SPADE_ERR_INVALID_ARG, "qbar and kbar must both be given or both be null");
  if ((sics_q == nullptr) != (sics_k == nullptr))
    return fail(SPADE_ERR_INVALID_ARG, "sics_q and sics_k must both be given or both be null");
  if (!qb && !qbar && !sics_q)
    return fail(SPADE_ERR_INVALID_ARG, "nothing requested: give qb/kb, qbar/kbar or sics_q/sics_k");
  spade::HeadMap hm;
  st = parse_heads(dg, heads, n_heads, &hm);
  if (st != SPADE_OK) return st;
  if (empty || hm.n == 0) return SPADE_OK;
  if (!q || !k) return fail(SPADE_ERR_INVALID_ARG, "q and k must be non-null");
  if (!aligned16(q) || !aligned16(k) || (qb && (!aligned16(qb) || !aligned16(kb))))
    return fail(SPADE_ERR_INVALID_ARG, "q, k, qb and kb must be 16-byte aligned");
  if (qb && (qb == q || qb == k || kb == q || kb == k || qb == kb))
    return fail(SPADE_ERR_INVALID_ARG, "blocked outputs must not alias the inputs or each other");
  return hip_status(spade::launch_block_summarize(dg, hm, q, k, qb, kb, qbar, kbar, sics_q, sics_k,
                                                  stream),
                    "block_summarize launch");
}

spade_status spade_aggregation_score(const spade_geom* g, const double* sics_q,
                                     const double* sics_k, double* as_q, double* as_k,
                                     double* as_qk, hipStream_t stream) {
  spade::DevGeom dg;
  bool empty = false;
  spade_status st = check_geom(g, &dg, &empty);
  if (st != SPADE_OK) return st;
  if (empty) return SPADE_OK;
  if (!sics_q || !sics_k || !as_qk)
    return fail(SPADE_ERR_INVALID_ARG, "sics_q, sics_k and as_qk must be non-null");
  return hip_status(spade::launch_aggregation_score(dg, sics_q, sics_k, as_q, as_k, as_qk, stream),
                    "aggregation_score launch");
}

spade_status spade_choose_scheme(const double* as_qk, int32_t C, int32_t B, int32_t H,
                                 int32_t* choice, double* best, hipStream_t stream) {
  if (C < 1 || C > spade::kMaxCandidates)
    return fail(SPADE_ERR_INVALID_ARG, "candidate count C must lie in [1, %d] (got %d)",
                spade::kMaxCandidates, C);
  if (B < 0 || H < 0) return fail(SPADE_ERR_INVALID_ARG, "negative B or H (B=%d H=%d)", B, H);
  if (int64_t(C) * B * H > (int64_t(1) << 40) || H > (1 << 24))
    return fail(SPADE_ERR_UNSUPPORTED, "score table too large (C=%d B=%d H=%d)", C, B, H);
  if (B == 0 || H == 0) return SPADE_OK;
  if (!as_qk || !choice) return fail(SPADE_ERR_INVALID_ARG, "as_qk and choice must be non-null");
  return hip_status(spade::launch_choose_scheme(as_qk, C, B, H, choice, best, stream),
                    "choose_scheme launch");
}

spade_status spade_estimate_select(const spade_geom* g, const double* qbar, const double* kbar,
                                   int32_t mode, int32_t topk, double tau, double scale,
                                   int32_t* counts, int32_t* indices, double* scores,
                                   hipStream_t stream) {
  spade::DevGeom dg;
  bool empty = false;
  spade_status st = check_geom(g, &dg, &empty);
  if (st != SPADE_OK) return st;
  if (mode != SPADE_TOPK && mode != SPADE_TOPP)
    return fail(SPADE_ERR_INVALID_ARG, "mode must be SPADE_TOPK or SPADE_TOPP (got %d)", mode);
  if (mode == SPADE_TOPK && topk < 1)
    return fail(SPADE_ERR_INVALID_ARG, "topk must be >= 1 (got %d)", topk);
  if (mode == SPADE_TOPP && !(tau > 0.0 && tau <= 1.0))
    return fail(SPADE_ERR_INVALID_ARG, "tau must lie in (0, 1] (got %g)", tau);
  if (!(isfinite(scale) && scale > 0.0))
    return fail(SPADE_ERR_INVALID_ARG, "scale must be finite and > 0 (got %g)", scale);
  if (!empty && dg.NB > spade::kMaxSelectNB)
    return fail(SPADE_ERR_UNSUPPORTED, "NB=%d exceeds the selection limit %d", dg.NB,
                spade::kMaxSelectNB);
  if (empty) return SPADE_OK;
  if (!qbar || !kbar || !counts || !indices)
    return fail(SPADE_ERR_INVALID_ARG, "qbar, kbar, counts and indices must be non-null");
  if (!aligned16(qbar) || !aligned16(kbar))
    return fail(SPADE_ERR_INVALID_ARG, "qbar and kbar must be 16-byte aligned");
  spade::SelectSpec p = {};
  p.q0 = qbar;
  p.k0 = kbar;
  p.estimator = spade::kEstMean;
  p.mode = mode;
  p.topk = topk;
  p.tau = tau;
  p.scale = scale;
  p.intra = spade::kIntraNone;
  p.wt = p.wh = p.ww = -1;
  p.counts = counts;
  p.indices = indices;
  p.scores = scores;
  return hip_status(spade::launch_select(dg, p, stream), "estimate_select launch");
}

spade_status spade_block_minmax(const spade_geom* g, const void* q, const void* k, double* qmax,
                                double* qmin, double* kmax, double* kmin, double* sics_q,
                                double* sics_k, const int32_t* heads, int32_t n_heads,
                                hipStream_t stream) {
  spade::DevGeom dg;
  bool empty = false;
  spade_status st = check_geom(g, &dg, &empty);
  if (st != SPADE_OK) return st;
  if ((sics_q == nullptr) != (sics_k == nullptr))
    return fail(SPADE_ERR_INVALID_ARG, "sics_q and sics_k must both be given or both be null");
  spade::HeadMap hm;
  st = parse_heads(dg, heads, n_heads, &hm);
  if (st != SPADE_OK) return st;
  if (empty || hm.n == 0) return SPADE_OK;
  if (!q || !k || !qmax || !qmin || !kmax || !kmin)
    return fail(SPADE_ERR_INVALID_ARG, "q, k, qmax, qmin, kmax and kmin must be non-null");
  if (!aligned16(q) || !aligned16(k))
    return fail(SPADE_ERR_INVALID_ARG, "q and k must be 16-byte aligned");
  return hip_status(spade::launch_block_minmax(dg, hm, q, k, qmax, qmin, kmax, kmin, sics_q,
                                               sics_k, stream),
                    "block_minmax launch");
}

spade_status spade_sparse_attn_raster_multi(const spade_geom* geoms, int32_t n_geoms,
                                            const spade_head_lists* heads, const void* q,
                                            const void* k, const void* v, double scale, void* o,
                                            float* lse, void* workspace, size_t workspace_bytes,
                                            hipStream_t stream) {
  if (!geoms || n_geoms < 1 || n_geoms > spade::kMaxMultiGeoms)
    return fail(SPADE_ERR_INVALID_ARG, "need 1..%d geometries (got %d)", spade::kMaxMultiGeoms,
                n_geoms);
  spade::DevGeom dg[spade::kMaxMultiGeoms];
  bool empty = false;
  for (int c = 0; c < n_geoms; ++c) {
    bool e = false;
    spade_status st = check_geom(&geoms[c], &dg[c], &e);
    if (st != SPADE_OK) return st;
    const spade_geom& a = geoms[0];
    const spade_geom& b = geoms[c];
    if (b.B != a.B || b.H != a.H || b.d != a.d || b.T != a.T || b.Hs != a.Hs || b.Ws != a.Ws)
      return fail(SPADE_ERR_INVALID_ARG, "geometry %d differs from geometry 0 outside the blocking",
                  c);
    empty = e;
    if (!e && dg[c].NB > spade::kMaxAttnNB)
      return fail(SPADE_ERR_UNSUPPORTED, "NB=%d exceeds the attention limit %d", dg[c].NB,
                  spade::kMaxAttnNB);
  }
  if (!(isfinite(scale) && scale > 0.0))
    return fail(SPADE_ERR_INVALID_ARG, "scale must be finite and > 0 (got %g)", scale);
  if (dg[0].H > spade::kMaxMultiHeads)
    return fail(SPADE_ERR_UNSUPPORTED, "H=%d exceeds %d heads per call", dg[0].H,
                spade::kMaxMultiHeads);
  if (!empty && dg[0].N * int64_t(dg[0].d) * 2 >= (int64_t(1) << 31))
    return fail(SPADE_ERR_UNSUPPORTED, "raster attention needs N*d*2 < 2^31 bytes per head");
  if (empty) return SPADE_OK;
  if (!heads) return fail(SPADE_ERR_INVALID_ARG, "heads must be non-null");
  if (!q || !k || !v || !o) return fail(SPADE_ERR_INVALID_ARG, "q, k, v and o must be non-null");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
    return fail(SPADE_ERR_INVALID_ARG, "q, k, v and o must be 16-byte aligned");
  spade::MultiHead mh[spade::kMaxMultiHeads];
  for (int h = 0; h < dg[0].H; ++h) {
    const spade_head_lists& x = heads[h];
    if (x.scheme < 0 || x.scheme >= n_geoms)
      return fail(SPADE_ERR_INVALID_ARG, "heads[%d].scheme=%d outside [0, %d)", h, x.scheme,
                  n_geoms);
    if (!x.counts || !x.indices)
      return fail(SPADE_ERR_INVALID_ARG, "heads[%d]: counts and indices must be non-null", h);
    if (x.counts_bstride < 0 || x.counts_bstride >= (int64_t(1) << 31) || x.indices_bstride < 0)
      return fail(SPADE_ERR_INVALID_ARG, "heads[%d]: batch strides out of range", h);
    mh[h] = {x.counts, x.indices, x.indices_bstride, int(x.counts_bstride), x.scheme, h, 0};
  }
  const size_t need = spade::attn_workspace_bytes(dg[0]);
  if (workspace_bytes < need || (need > 0 && (workspace == nullptr || !aligned16(workspace))))
    return fail(SPADE_ERR_WORKSPACE, "16-byte aligned workspace of %zu bytes needed, %zu given",
                need, workspace_bytes);
  return hip_status(spade::launch_sparse_attn_multi(dg, n_geoms, mh, dg[0].H, q, k, v,
                                                    float(scale), o, lse, workspace, stream),
                    "multi-scheme attention launch");
}

spade_status spade_policy_budgets(const double* as_best, int32_t H, const int32_t* heads,
                                  int32_t n_heads, int32_t k_dyn, int32_t NB, int32_t* k_out,
                                  hipStream_t stream) {
  if (H < 0 || H > 65535) return fail(SPADE_ERR_INVALID_ARG, "H must lie in [0, 65535] (got %d)", H);
  if (k_dyn < 1) return fail(SPADE_ERR_INVALID_ARG, "k_dyn must be >= 1 (got %d)", k_dyn);
  if (NB < 1) return fail(SPADE_ERR_INVALID_ARG, "NB must be >= 1 (got %d)", NB);
  spade::DevGeom dg = {};
  dg.H = H;
  spade::HeadMap hm;
  spade_status st = parse_heads(dg, heads, n_heads, &hm);
  if (st != SPADE_OK) return st;
  if (hm.n == 0) return SPADE_OK;
  if (!as_best || !k_out) return fail(SPADE_ERR_INVALID_ARG, "as_best and k_out must be non-null");
  return hip_status(spade::launch_policy_budgets(as_best, hm, k_dyn, NB, k_out, stream),
                    "policy_budgets launch");
}

spade_status spade_candidate_sics(const spade_geom* geoms, int32_t n_geoms, const void* q,
                                  const void* k, double* const* sics_q, double* const* sics_k,
                                  hipStream_t stream) {
  if (!geoms || n_geoms < 1 || n_geoms > spade::kMaxCandGeoms)
    return fail(SPADE_ERR_INVALID_ARG, "need 1..%d geometries (got %d)", spade::kMaxCandGeoms,
                n_geoms);
  spade::DevGeom dg[spade::kMaxCandGeoms];
  bool empty = false;
  for (int c = 0; c < n_geoms; ++c) {
    bool e = false;
    spade_status st = check_geom(&geoms[c], &dg[c], &e);
    if (st != SPADE_OK) return st;
    const spade_geom& a = geoms[0];
    const spade_geom& b = geoms[c];
    if (b.B != a.B || b.H != a.H || b.d != a.d || b.T != a.T || b.Hs != a.Hs || b.Ws != a.Ws)
      return fail(SPADE_ERR_INVALID_ARG, "geometry %d differs from geometry 0 outside the blocking",
                  c);
    empty = e;
  }
  if (empty) return SPADE_OK;
  if (dg[0].N * int64_t(dg[0].d) * 2 >= (int64_t(1) << 31))
    return fail(SPADE_ERR_UNSUPPORTED, "one pass over the candidates needs N*d*2 < 2^31 bytes per head");
  if (!q || !k || !sics_q || !sics_k)
    return fail(SPADE_ERR_INVALID_ARG, "q, k, sics_q and sics_k must be non-null");
  if (!aligned16(q) || !aligned16(k))
    return fail(SPADE_ERR_INVALID_ARG, "q and k must be 16-byte aligned");
  spade::CandPlan pl = {};
  pl.C = n_geoms;
  const int G3[3] = {dg[0].T, dg[0].Hs, dg[0].Ws};
  for (int c = 0; c < n_geoms; ++c) {
    if (!sics_q[c] || !sics_k[c])
      return fail(SPADE_ERR_INVALID_ARG, "sics_q[%d] and sics_k[%d] must be non-null", c, c);
    pl.sics_q[c] = sics_q[c];
    pl.sics_k[c] = sics_k[c];
    const int e3[3] = {dg[c].bt, dg[c].bh, dg[c].bw};
    const int n3[3] = {dg[c].nT, dg[c].nH, dg[c].nW};
    for (int a = 0; a < 3; ++a) {
      pl.ext[c][a] = e3[a];
      pl.nblk[c][a] = n3[a];
    }
  }
  int64_t cells = 1;
  for (int a = 0; a < 3; ++a) {
    // region extent: the least common multiple of the candidates' extents on this axis
    int64_t L = 1;
    for (int c = 0; c < n_geoms; ++c) {
      int64_t x = L, y = pl.ext[c][a];
      while (y) { const int64_t t = x % y; x = y; y = t; }
      L = L / x * pl.ext[c][a];
      if (L > (int64_t(1) << 20)) break;
    }
    // cells: the union of the candidates' block boundaries inside [0, L)
    int n = 0;
    for (int64_t p = 0; p < L && n <= spade::kMaxCellsAxis; ++p) {
      bool cut = false;
      for (int c = 0; c < n_geoms; ++c) cut = cut || p % pl.ext[c][a] == 0;
      if (cut) {
        if (n < spade::kMaxCellsAxis) pl.start[a][n] = int(p);
        ++n;
      }
    }
    if (L > (int64_t(1) << 20) || n > spade::kMaxCellsAxis)
      return fail(SPADE_ERR_UNSUPPORTED,
                  "candidate blockings cut axis %d into more than %d cells per region", a,
                  spade::kMaxCellsAxis);
    pl.L[a] = int(L);
    pl.start[a][n] = int(L);
    pl.ncell[a] = n;
    pl.R[a] = int((G3[a] + L - 1) / L);
    cells *= n;
    for (int c = 0; c < n_geoms; ++c)  // cell index of each block boundary j * ext
      for (int j = 0, i = 0; j <= int(L / pl.ext[c][a]); ++j) {
        while (i < n && pl.start[a][i] < j * pl.ext[c][a]) ++i;
        pl.bnd[c][a][j] = static_cast<unsigned char>(i);
      }
  }
  if (cells * dg[0].d * int64_t(sizeof(double)) > spade::kMaxCellLds)
    return fail(SPADE_ERR_UNSUPPORTED, "%lld cells per region exceed the LDS (%d bytes)",
                (long long)cells, spade::kMaxCellLds);
  {  // cells by token count in a full region, largest first (ties: lower index)
    const int nc = int(cells);
    auto size = [&](int c) {
      const int cx = c % pl.ncell[2], cy = (c / pl.ncell[2]) % pl.ncell[1];
      const int ct = c / (pl.ncell[2] * pl.ncell[1]);
      return (pl.start[0][ct + 1] - pl.start[0][ct]) * (pl.start[1][cy + 1] - pl.start[1][cy]) *
             (pl.start[2][cx + 1] - pl.start[2][cx]);
    };
    for (int c = 0; c < nc; ++c) pl.order[c] = static_cast<unsigned short>(c);
    for (int a = 1; a < nc; ++a)  // insertion sort: stable, at most a few hundred cells
      for (int b = a; b > 0 && size(pl.order[b]) > size(pl.order[b - 1]); --b) {
        const unsigned short t = pl.order[b];
        pl.order[b] = pl.order[b - 1];
        pl.order[b - 1] = t;
      }
  }
  if (int64_t(pl.R[0]) * pl.R[1] * pl.R[2] > (int64_t(1) << 31) - 1)
    return fail(SPADE_ERR_UNSUPPORTED, "too many regions");
  return hip_status(spade::launch_candidate_sics(dg[0], pl, q, k, stream),
                    "candidate_sics launch");
}

spade_status spade_policy_tau(const double* as_best, int32_t H, const int32_t* heads,
                              int32_t n_heads, double tau, double* tau_out, hipStream_t stream) {
  if (H < 0 || H > 65535) return fail(SPADE_ERR_INVALID_ARG, "H must lie in [0, 65535] (got %d)", H);
  if (!(tau > 0.0 && tau <= 1.0))
    return fail(SPADE_ERR_INVALID_ARG, "tau must lie in (0, 1] (got %g)", tau);
  spade::DevGeom dg = {};
  dg.H = H;
  spade::HeadMap hm;
  spade_status st = parse_heads(dg, heads, n_heads, &hm);
  if (st != SPADE_OK) return st;
  if (hm.n == 0) return SPADE_OK;
  if (!as_best || !tau_out)
    return fail(SPADE_ERR_INVALID_ARG, "as_best and tau_out must be non-null");
  return hip_status(spade::launch_policy_tau(as_best, hm, tau, tau_out, stream),
                    "policy_tau launch");
}

spade_status spade_policy_dense(int32_t step, int32_t n_steps, int32_t task, int32_t turbo,
                                int32_t* dense) {
  if (!dense) return fail(SPADE_ERR_INVALID_ARG, "dense must be non-null");
  if (n_steps < 1) return fail(SPADE_ERR_INVALID_ARG, "n_steps must be >= 1 (got %d)", n_steps);
  if (step < 0 || step >= n_steps)
    return fail(SPADE_ERR_INVALID_ARG, "step must lie in [0, n_steps) (got %d of %d)", step,
                n_steps);
  if (n_steps > (1 << 27)) return fail(SPADE_ERR_UNSUPPORTED, "n_steps above 2^27");
  if (task != SPADE_TASK_T2V && task != SPADE_TASK_I2V)
    return fail(SPADE_ERR_INVALID_ARG, "task must be SPADE_TASK_T2V or SPADE_TASK_I2V (got %d)",
                task);
  *dense = spade::policy_dense(step, n_steps, task, turbo != 0) ? 1 : 0;
  return SPADE_OK;
}

spade_status spade_policy_split(int32_t k_total, int32_t func, int32_t* window,
                                int32_t* window_blocks, int32_t* k_dyn) {
  if (!window || !window_blocks || !k_dyn)
    return fail(SPADE_ERR_INVALID_ARG, "window, window_blocks and k_dyn must be non-null");
  if (k_total < 1 || k_total > (1 << 27))
    return fail(SPADE_ERR_INVALID_ARG, "k_total must lie in [1, 2^27] (got %d)", k_total);
  if (func != 0 && func != 1) return fail(SPADE_ERR_INVALID_ARG, "func must be 0 or 1 (got %d)", func);
  int w[3], wb = 0, kd = 0;
  spade::policy_split(k_total, func, w, &wb, &kd);
  for (int a = 0; a < 3; ++a) window[a] = w[a];
  *window_blocks = wb;
  *k_dyn = kd;
  return SPADE_OK;
}

spade_status spade_compose_select(const spade_geom* g, const spade_mask_spec* spec,
                                  const spade_summaries* sum, int32_t* counts, int32_t* indices,
                                  double* scores, hipStream_t stream) {
  spade::DevGeom dg;
  bool empty = false;
  spade_status st = check_geom(g, &dg, &empty);
  if (st != SPADE_OK) return st;
  if (!spec || !sum) return fail(SPADE_ERR_INVALID_ARG, "spec and summaries must be non-null");
  const spade_mask_spec& m = *spec;
  if (m.estimator != SPADE_EST_MEAN && m.estimator != SPADE_EST_DSA &&
      m.estimator != SPADE_EST_DSA2)
    return fail(SPADE_ERR_INVALID_ARG, "estimator must be SPADE_EST_MEAN, _DSA or _DSA2 (got %d)",
                m.estimator);
  if (m.mode != SPADE_TOPK && m.mode != SPADE_TOPP)
    return fail(SPADE_ERR_INVALID_ARG, "mode must be SPADE_TOPK or SPADE_TOPP (got %d)", m.mode);
  if (m.mode == SPADE_TOPK && !m.topk_per_head && m.topk < 1)
    return fail(SPADE_ERR_INVALID_ARG, "topk must be >= 1 (got %d)", m.topk);
  if (m.mode == SPADE_TOPP && !m.tau_per_head && !(m.tau > 0.0 && m.tau <= 1.0))
    return fail(SPADE_ERR_INVALID_ARG, "tau must lie in (0, 1] (got %g)", m.tau);
  if (!(isfinite(m.scale) && m.scale > 0.0))
    return fail(SPADE_ERR_INVALID_ARG, "scale must be finite and > 0 (got %g)", m.scale);
  if (m.intra != SPADE_INTRA_NONE && m.intra != SPADE_INTRA_THRESHOLD &&
      m.intra != SPADE_INTRA_TOPK)
    return fail(SPADE_ERR_INVALID_ARG, "intra must be SPADE_INTRA_NONE, _THRESHOLD or _TOPK (got %d)",
                m.intra);
  if (m.intra == SPADE_INTRA_TOPK && m.intra_topk < 0)
    return fail(SPADE_ERR_INVALID_ARG, "intra_topk must be >= 0 (got %d)", m.intra_topk);
  if (m.intra == SPADE_INTRA_THRESHOLD && isnan(m.intra_theta))
    return fail(SPADE_ERR_INVALID_ARG, "intra_theta must not be NaN");
  if (m.sink_tokens < 0)
    return fail(SPADE_ERR_INVALID_ARG, "sink_tokens must be >= 0 (got %lld)",
                (long long)m.sink_tokens);
  if (!empty && dg.NB > spade::kMaxSelectNB)
    return fail(SPADE_ERR_UNSUPPORTED, "NB=%d exceeds the selection limit %d", dg.NB,
                spade::kMaxSelectNB);
  if (empty) return SPADE_OK;
  if (!counts || !indices)
    return fail(SPADE_ERR_INVALID_ARG, "counts and indices must be non-null");
  spade::SelectSpec p = {};
  if (m.estimator == SPADE_EST_MEAN) {
    if (!sum->qbar || !sum->kbar)
      return fail(SPADE_ERR_INVALID_ARG, "the mean estimator needs qbar and kbar");
    p.q0 = sum->qbar;
    p.k0 = sum->kbar;
  } else {
    if (!sum->qmax || !sum->qmin || !sum->kmax || !sum->kmin)
      return fail(SPADE_ERR_INVALID_ARG, "the DSA estimators need qmax, qmin, kmax and kmin");
    p.q0 = sum->qmax;
    p.q1 = sum->qmin;
    p.k0 = sum->kmax;
    p.k1 = sum->kmin;
  }
  if (!aligned16(p.q0) || !aligned16(p.k0) || (p.q1 && (!aligned16(p.q1) || !aligned16(p.k1))))
    return fail(SPADE_ERR_INVALID_ARG, "summaries must be 16-byte aligned");
  if (m.intra != SPADE_INTRA_NONE && (!sum->sics_q || !sum->sics_k))
    return fail(SPADE_ERR_INVALID_ARG, "the intra-block filter needs sics_q and sics_k");
  p.sics_q = sum->sics_q;
  p.sics_k = sum->sics_k;
  p.topk_h = m.topk_per_head;
  p.tau_h = m.tau_per_head;
  p.estimator = m.estimator;
  p.mode = m.mode;
  p.topk = m.topk;
  p.tau = m.tau;
  p.scale = m.scale;
  p.intra = m.intra;
  p.intra_k = m.intra_topk;
  p.intra_theta = m.intra_theta;
  const bool window = m.window[0] >= 0 && m.window[1] >= 0 && m.window[2] >= 0;
  p.wt = window ? m.window[0] : -1;
  p.wh = window ? m.window[1] : -1;
  p.ww = window ? m.window[2] : -1;
  p.sink = m.sink_tokens;
  p.counts = counts;
  p.indices = indices;
  p.scores = scores;
  return hip_status(spade::launch_select(dg, p, stream), "compose_select launch");
}

size_t spade_attn_workspace_bytes(const spade_geom* g) {
  spade::DevGeom dg;
  bool empty = false;
  if (check_geom(g, &dg, &empty) != SPADE_OK || empty) return 0;
  return spade::attn_workspace_bytes(dg);
}

spade_status spade_block_sparse_attn(const spade_geom* g, const void* qb, const void* kb,
                                     const void* vb, const int32_t* counts,
                                     const int32_t* indices, double scale, void* ob, float* lse,
                                     void* workspace, size_t workspace_bytes,
                                     hipStream_t stream) {
  return sparse_attn(g, qb, kb, vb, counts, indices, scale, ob, lse, workspace, workspace_bytes,
                     false, stream);
}

spade_status spade_sparse_attn_raster(const spade_geom* g, const void* q, const void* k,
                                      const void* v, const int32_t* counts,
                                      const int32_t* indices, double scale, void* o, float* lse,
                                      void* workspace, size_t workspace_bytes,
                                      hipStream_t stream) {
  return sparse_attn(g, q, k, v, counts, indices, scale, o, lse, workspace, workspace_bytes, true,
                     stream);
}

spade_status spade_sparse_attn_raster_noalloc(const spade_geom* g, const void* q, const void* k,
                                              const void* v, const int32_t* counts,
                                              const int32_t* indices, double scale, void* o,
                                              float* lse, hipStream_t stream) {
  spade::DevGeom dg;
  bool empty = false;
  spade_status st = check_geom(g, &dg, &empty);
  if (st != SPADE_OK) return st;
  const size_t need = empty ? 0 : spade::attn_workspace_bytes(dg);
  if (need > spade::kNoAllocScratchBytes)
    return fail(SPADE_ERR_UNSUPPORTED, "the schedule needs %zu bytes of scratch, the library holds %zu",
                need, spade::kNoAllocScratchBytes);
  void* ws = nullptr;
  size_t ws_bytes = 0;
  if (need > 0) {
    const hipError_t e = spade::noalloc_scratch(&ws, &ws_bytes);
    if (e != hipSuccess) return hip_status(e, "scratch lookup");
  }
  return sparse_attn(g, q, k, v, counts, indices, scale, o, lse, ws, ws_bytes, true, stream);
}

spade_status spade_validate_lists(const spade_geom* g, const int32_t* counts,
                                  const int32_t* indices, int32_t* report, hipStream_t stream) {
  spade::DevGeom dg;
  bool empty = false;
  spade_status st = check_geom(g, &dg, &empty);
  if (st != SPADE_OK) return st;
  if (!report) return fail(SPADE_ERR_INVALID_ARG, "report must be non-null");
  const int64_t rows = empty ? 0 : int64_t(dg.B) * dg.H * dg.NB;
  if (rows > INT32_MAX)
    return fail(SPADE_ERR_UNSUPPORTED, "B*H*NB = %lld rows exceeds 2^31 - 1", (long long)rows);
  if (rows > 0 && (!counts || !indices))
    return fail(SPADE_ERR_INVALID_ARG, "counts and indices must be non-null");
  return hip_status(spade::launch_validate_lists(empty ? 0 : dg.NB, int(rows), counts, indices,
                                                 report, stream),
                    "validate_lists launch");
}

}  // extern "C"
