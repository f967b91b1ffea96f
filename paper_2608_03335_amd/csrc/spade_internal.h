// Internal declarations shared by the C-ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spade {

// Geometry with the derived block-grid sizes, passed to kernels by value.
struct DevGeom {
  int B, H, d;
  int T, Hs, Ws;
  int bt, bh, bw;
  int nT, nH, nW;
  int NB, BS;
  int64_t N;
};

// Origin, per-axis extent and real-token count of block b (T-major block order).
struct BlockExt {
  int t0, y0, x0;
  int et, eh, ew;
  int n;
};

__device__ __forceinline__ BlockExt block_ext(const DevGeom& g, int b) {
  const int wb = b % g.nW;
  const int r = b / g.nW;
  const int hb = r % g.nH;
  const int tb = r / g.nH;
  BlockExt e;
  e.t0 = tb * g.bt;
  e.y0 = hb * g.bh;
  e.x0 = wb * g.bw;
  e.et = min(g.bt, g.T - e.t0);
  e.eh = min(g.bh, g.Hs - e.y0);
  e.ew = min(g.bw, g.Ws - e.x0);
  e.n = e.et * e.eh * e.ew;
  return e;
}

constexpr int kMaxHeadList = 64;  // head subset of one reorder call (passed by value)

// Which heads a reorder call moves: blocked-side head k <-> raster-side head h[k].
// ident = 1 means all H heads in order (h[] unused).
struct HeadMap {
  int n, ident;
  int h[kMaxHeadList];
};

// Raster token of slot `slot` of block e: slots follow raster order of (dt, dy, dx).
// r_ew and r_eh are 1/e.ew and 1/e.eh to within a few ulp (a division or
// v_rcp_f32): slots and extents stay below 2^8 (see kMaxBS), so (slot + 0.5) / ew
// lies at least 2^-9 from an integer, far beyond the float error, and the
// truncation yields the exact quotient.
__device__ __forceinline__ int64_t block_slot_token(const DevGeom& g, const BlockExt& e,
                                                   float r_ew, float r_eh, int slot) {
  const int q = int((float(slot) + 0.5f) * r_ew);  // slot / ew
  const int dx = slot - q * e.ew;
  const int dt = int((float(q) + 0.5f) * r_eh);    // q / eh
  const int dy = q - dt * e.eh;
  return (int64_t(e.t0 + dt) * g.Hs + (e.y0 + dy)) * g.Ws + (e.x0 + dx);
}

// grid.y enumerates (batch, listed head): index on the blocked side (compact over
// the listed heads) and on the raster side (all H heads).
__device__ __forceinline__ void head_pair(const DevGeom& g, const HeadMap& hm, int64_t* blocked,
                                          int64_t* raster) {
  const int by = blockIdx.y;
  const int b = by / hm.n, k = by - b * hm.n;
  *blocked = by;
  *raster = int64_t(b) * g.H + (hm.ident ? k : hm.h[k]);
}

// Raises kernel `fn`'s dynamic-LDS limit to `bytes` on the current device, once per
// (kernel, device): the attribute is per device, and the first call on each device
// sets it under a lock (thread-safe; later calls only look it up).
hipError_t ensure_dynamic_lds(const void* fn, int bytes);

// Launchers (each returns hipGetLastError() after its launches).
hipError_t launch_reorder(const DevGeom& g, const void* x, void* y, int esize, int inverse,
                          const HeadMap& heads, hipStream_t s);
hipError_t launch_aggregation_score(const DevGeom& g, const double* sics_q, const double* sics_k,
                                    double* as_q, double* as_k, double* as_sum, hipStream_t s);
hipError_t launch_choose_scheme(const double* as_qk, int C, int B, int H, int* choice,
                                double* best, hipStream_t s);
hipError_t launch_block_summarize(const DevGeom& g, const HeadMap& hm, const void* q,
                                  const void* k, void* qb, void* kb, double* qbar, double* kbar,
                                  double* sics_q, double* sics_k, hipStream_t s);
hipError_t launch_block_minmax(const DevGeom& g, const HeadMap& hm, const void* q, const void* k,
                               double* qmax, double* qmin, double* kmax, double* kmin,
                               double* sics_q, double* sics_k, hipStream_t s);
hipError_t launch_summarize(const DevGeom& g, const void* qb, const void* kb, double* qbar,
                            double* kbar, double* sics_q, double* sics_k, hipStream_t s);
// One selection call (estimator, row rule, intra filter, window, sink), as the
// kernel sees it; validated and normalised by the C-ABI layer.
enum { kEstMean = 0, kEstDsa = 1, kEstDsa2 = 2 };
enum { kIntraNone = 0, kIntraThreshold = 1, kIntraTopk = 2 };
struct SelectSpec {
  const double* q0;  // MEAN: qbar; DSA, DSA2: qmax
  const double* q1;  // DSA, DSA2: qmin
  const double* k0;  // MEAN: kbar; DSA, DSA2: kmax
  const double* k1;  // DSA, DSA2: kmin
  const double* sics_q;
  const double* sics_k;
  const int* topk_h;     // per-head k (nullable)
  const double* tau_h;   // per-head tau (nullable)
  int estimator, mode, topk;
  double tau, scale;
  int intra, intra_k;
  double intra_theta;
  int wt, wh, ww;        // window radii in blocks; wt < 0: no window
  int64_t sink;          // attention-sink length in tokens (0: none)
  int* counts;
  int* indices;
  double* scores;
};
hipError_t launch_select(const DevGeom& g, const SelectSpec& p, hipStream_t s);
// Failure bits of a block-list row (the values of SPADE_LIST_* in spade.h).
constexpr int kListBadCount = 1, kListBadIndex = 2, kListNotAscending = 4;
hipError_t launch_validate_lists(int NB, int rows, const int* counts, const int* indices,
                                 int* report, hipStream_t s);

// SICS of every candidate blocking in one pass over the raster Q and K. A region is
// the per-axis least common multiple of the candidates' block extents, so every
// candidate block lies in one region; within a region the union of the candidates'
// block boundaries cuts each axis into cells. The plan (host-built, passed by value)
// gives the cell starts per axis and, per candidate and axis, the cell index of each
// of its block boundaries inside a region.
constexpr int kMaxCandGeoms = 8;
constexpr int kMaxCellsAxis = 48;
constexpr int kMaxCellLds = 144 * 1024;  // fp64 cell sums of one region (d per cell)
struct CandPlan {
  int C;
  int L[3], R[3], ncell[3];         // region extent, regions, cells per axis (t, y, x)
  int start[3][kMaxCellsAxis + 1];  // cell starts inside a region (start[a][ncell] = L)
  int ext[kMaxCandGeoms][3];        // block extents per candidate
  int nblk[kMaxCandGeoms][3];       // blocks per axis of the whole grid
  unsigned char bnd[kMaxCandGeoms][3][kMaxCellsAxis + 1];  // boundary j -> cell index
  unsigned short order[kMaxCellLds / (64 * 8)];  // cells by token count, largest first
  double* sics_q[kMaxCandGeoms];
  double* sics_k[kMaxCandGeoms];
};
hipError_t launch_candidate_sics(const DevGeom& g, const CandPlan& plan, const void* q,
                                 const void* k, hipStream_t s);
hipError_t launch_policy_tau(const double* as_best, const HeadMap& hm, double tau,
                             double* tau_out, hipStream_t s);
bool policy_dense(int step, int n_steps, int task, bool turbo);
void policy_split(int k_total, int func, int window[3], int* window_blocks, int* k_dyn);
hipError_t launch_policy_budgets(const double* as_best, const HeadMap& hm, int k_dyn, int NB,
                                 int* k_out, hipStream_t s);
size_t attn_workspace_bytes(const DevGeom& g);
// One attention launch over heads with different blockings (one grid, one shared
// raster Q/K/V): per head its geometry, its block lists and its first work item.
constexpr int kMaxMultiGeoms = 8;
constexpr int kMaxMultiHeads = 64;
struct MultiHead {
  const int* counts;        // (batch 0, this head): [NB]
  const int* indices;       // (batch 0, this head): [NB, NB]
  int64_t indices_bstride;  // elements between batch elements
  int counts_bstride;
  int geom;                 // index into MultiTable::geo
  int h;                    // raster head index
  int start;                // first work item of the head in each batch element
};
struct MultiTable {
  DevGeom geo[kMaxMultiGeoms];
  MultiHead head[kMaxMultiHeads];
  int n_heads;              // heads of this launch, in ascending `start`
  int items_per_batch;      // work items per batch element (a multiple of 8)
};
// One launch per distinct workgroup shape (compute waves = ceil(BS / 32)); heads
// whose blockings share a shape run in the same launch.
hipError_t launch_sparse_attn_multi(const DevGeom* geo, int n_geo, const MultiHead* heads,
                                    int n_heads, const void* q, const void* k, const void* v,
                                    float scale, void* o, float* lse, void* ws, hipStream_t s);
hipError_t launch_block_sparse_attn(const DevGeom& g, const void* qb, const void* kb,
                                    const void* vb, const int* counts, const int* indices,
                                    float scale, void* ob, float* lse, void* ws, bool raster,
                                    hipStream_t s);

constexpr int kMaxRankedHeads = 4096;  // attention head ranking; beyond: grid order
// scratch of the allocation-free attention call: the ranking of kMaxRankedHeads pairs
constexpr size_t kNoAllocScratchBytes = size_t(kMaxRankedHeads) * 16;
constexpr int kMaxDevices = 64;
// This device's copy of that scratch (looked up once per device, thread-safe).
hipError_t noalloc_scratch(void** ptr, size_t* bytes);
constexpr int kMaxBS = 256;        // attention: one wave per 32 query rows, <= 8 waves
constexpr int kMaxSelectNB = 1024;  // selection: one row of scores per wave in registers
constexpr int kMaxAttnNB = 16384;   // attention: a work item's kept list is staged in LDS
constexpr int kMaxCandidates = 1024;  // blocking-scheme candidates of one choose call

}  // namespace spade
