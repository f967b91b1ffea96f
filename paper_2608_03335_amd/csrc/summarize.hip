// Summarizer (block mean, paper §3.1 MEAN-SPADE; block max/min for the DSA
// estimators) and intra-block estimator SICS (§3.2, Eq. (4)-(5), Alg. 1) over
// the blocked bf16 layout or straight from the raster layout.
//
// One workgroup per (block, head) reads that block's Q rows, then its K rows.
// Lane layout: V = d/8 lanes share one token row (16 bytes = 8 bf16 each), so
// 256/V rows are in flight per pass; every lane accumulates its 8 columns in
// fp64 and the row groups are combined through LDS in a fixed order.
//
// SICS is evaluated in the closed form |sum_k q_k/|q_k||^2, which equals the sum
// of all pairwise cosines of Eq. (4) (expanding the square gives Eq. (5)'s
// diagonal plus twice the off-diagonal sum, the quantity Alg. 1 accumulates).
// It needs one row norm per token (a V-lane DPP reduction) and no sequential
// scan, so all rows of a block proceed in parallel.
#include "spade_internal.h"

namespace spade {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ void bf16x8_to_f32(const uint4 v, float f[8]) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

// One fp64 DPP step: v + (v of the lane that `ctrl` selects within the row).
template <int CTRL>
__device__ __forceinline__ double dpp_add(double v) {
  const uint64_t u = static_cast<uint64_t>(__double_as_longlong(v));
  const int lo = __builtin_amdgcn_update_dpp(0, int(uint32_t(u)), CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, int(uint32_t(u >> 32)), CTRL, 0xf, 0xf, false);
  return v + __longlong_as_double(static_cast<long long>((uint64_t(uint32_t(hi)) << 32) |
                                                         uint32_t(lo)));
}

// Sum over each aligned group of V = 8 or 16 lanes (one token row), left in every
// lane of the group: swap neighbours and pairs inside quads, then mirror the
// half rows (quad 0 <-> 1, 2 <-> 3) and, for 16, the rows. All VALU (DPP), no LDS
// round trips; partners add the same two values, so every lane gets the same bits.
template <int V>
__device__ __forceinline__ double row_group_sum(double v) {
  v = dpp_add<0xB1>(v);   // quad_perm [1,0,3,2]
  v = dpp_add<0x4E>(v);   // quad_perm [2,3,0,1]
  v = dpp_add<0x141>(v);  // row_half_mirror
  if (V == 16) v = dpp_add<0x140>(v);  // row_mirror
  return v;
}

// Row loads in flight per lane: each lane loads its next kRowBatch rows before
// reducing them (the rows a lane reduces, and their order, are those of a plain
// loop over s = grp, grp + G, ...).
constexpr int kRowBatch = 2;

// 1/sqrt(x) for x > 0 in fp64: the hardware estimate (v_rsq_f64) refined by two
// Newton steps y <- y (3 - x y^2) / 2, each of which squares the relative error;
// much cheaper than a correctly rounded fp64 sqrt followed by a division.
__device__ __forceinline__ double inv_sqrt(double x) {
  double y = __builtin_amdgcn_rsq(x);
  const double hx = 0.5 * x;
  y = y * (1.5 - hx * y * y);
  y = y * (1.5 - hx * y * y);
  return y;
}

// SICS accumulation of one token row held by V lanes (8 columns each): adds the
// row's unit vector to uacc. A zero row adds exactly nothing.
template <int V>
__device__ __forceinline__ void add_unit_row(const float (&f)[8], double (&uacc)[8]) {
  double ss = 0.0;
#pragma unroll
  for (int c = 0; c < 8; ++c) ss += double(f[c]) * double(f[c]);
  ss = row_group_sum<V>(ss);
  const double inv = ss > 0.0 ? inv_sqrt(ss) : 0.0;
#pragma unroll
  for (int c = 0; c < 8; ++c) uacc[c] += double(f[c]) * inv;
}

template <int D, bool SICS>
__global__ void __launch_bounds__(kThreads) summarize_kernel(DevGeom g, const uint4* __restrict__ qb,
                                                             const uint4* __restrict__ kb,
                                                             double* __restrict__ qbar,
                                                             double* __restrict__ kbar,
                                                             double* __restrict__ sics_q,
                                                             double* __restrict__ sics_k) {
  constexpr int V = D / 8;          // lanes per token row
  constexpr int G = kThreads / V;   // token rows per pass
  __shared__ double part[G][D];
  __shared__ double upart[SICS ? G : 1][SICS ? D : 1];
  __shared__ double sq[kThreads / 64];

  const int b = blockIdx.x;
  const int64_t bh = blockIdx.y;
  const int n = block_ext(g, b).n;
  const int vec = threadIdx.x % V, grp = threadIdx.x / V;
  const int64_t row0 = (bh * g.NB + b) * int64_t(g.BS);

  for (int which = 0; which < 2; ++which) {
    const uint4* src = (which ? kb : qb) + row0 * V;
    double acc[8], uacc[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = uacc[k] = 0.0;
    for (int s0 = 0; s0 < n; s0 += kRowBatch * G) {  // zero rows past n add nothing
      uint4 v[kRowBatch];
#pragma unroll
      for (int r = 0; r < kRowBatch; ++r) {
        const int s = s0 + r * G + grp;
        v[r] = make_uint4(0, 0, 0, 0);
        if (s < n) v[r] = src[int64_t(s) * V + vec];
      }
#pragma unroll
      for (int r = 0; r < kRowBatch; ++r) {
        float f[8];
        bf16x8_to_f32(v[r], f);
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[k] += double(f[k]);
        if (SICS) add_unit_row<V>(f, uacc);
      }
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      part[grp][vec * 8 + k] = acc[k];
      if (SICS) upart[grp][vec * 8 + k] = uacc[k];
    }
    __syncthreads();
    double u2 = 0.0;
    if (threadIdx.x < D) {
      const int c = threadIdx.x;
      double s = 0.0;
      for (int r = 0; r < G; ++r) s += part[r][c];
      (which ? kbar : qbar)[(bh * g.NB + b) * D + c] = s / double(n);
      if (SICS) {
        double u = 0.0;
        for (int r = 0; r < G; ++r) u += upart[r][c];
        u2 = u * u;
      }
    }
    if (SICS) {
      // sum of u_c^2 over the D columns: wave sums, then a fixed-order total.
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) u2 += __shfl_xor(u2, m, 64);
      if ((threadIdx.x & 63) == 0) sq[threadIdx.x >> 6] = u2;
    }
    __syncthreads();
    if (SICS && threadIdx.x == 0) {
      double t = 0.0;
      for (int w = 0; w < D / 64; ++w) t += sq[w];
      (which ? sics_k : sics_q)[bh * g.NB + b] = t;
    }
    // part/upart/sq are rewritten by the next tensor only after this barrier
    __syncthreads();
  }
}

// Blocking, Summarizer and SICS in one pass over the raster tensors (§3.3
// optimisation (1)): each workgroup gathers its block's rows of Q, then K, from
// the raster layout, optionally writes them to the blocked layout (zeros in the
// padding slots), and reduces them as summarize_kernel does. Grid (block, batch x
// listed head); summaries and blocked rows are indexed by the listed head.
template <int D, bool SICS, bool WRITE>
__global__ void __launch_bounds__(kThreads) block_summarize_kernel(
    DevGeom g, HeadMap hm, const uint4* __restrict__ q, const uint4* __restrict__ k,
    uint4* __restrict__ qb, uint4* __restrict__ kb, double* __restrict__ qbar,
    double* __restrict__ kbar, double* __restrict__ sics_q, double* __restrict__ sics_k) {
  constexpr int V = D / 8;
  constexpr int G = kThreads / V;
  __shared__ double part[G][D];
  __shared__ double upart[SICS ? G : 1][SICS ? D : 1];
  __shared__ double sq[kThreads / 64];

  const int b = blockIdx.x;
  int64_t bh_blk, bh_ras;
  head_pair(g, hm, &bh_blk, &bh_ras);
  const BlockExt e = block_ext(g, b);
  const int n = e.n;
  const float r_ew = 1.0f / float(e.ew), r_eh = 1.0f / float(e.eh);
  const int vec = threadIdx.x % V, grp = threadIdx.x / V;

  for (int which = 0; which < 2; ++which) {
    const uint4* src = (which ? k : q) + bh_ras * g.N * V;
    uint4* dst = WRITE ? (which ? kb : qb) + (bh_blk * g.NB + b) * int64_t(g.BS) * V : nullptr;
    double acc[8], uacc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = uacc[c] = 0.0;
    const int lim = WRITE ? g.BS : n;
    for (int s0 = 0; s0 < lim; s0 += kRowBatch * G) {
      uint4 v[kRowBatch];
#pragma unroll
      for (int r = 0; r < kRowBatch; ++r) {
        const int s = s0 + r * G + grp;
        v[r] = make_uint4(0, 0, 0, 0);
        if (s < n) v[r] = src[block_slot_token(g, e, r_ew, r_eh, s) * V + vec];
      }
#pragma unroll
      for (int r = 0; r < kRowBatch; ++r) {
        const int s = s0 + r * G + grp;
        if (WRITE && s < lim) dst[int64_t(s) * V + vec] = v[r];
        float f[8];
        bf16x8_to_f32(v[r], f);  // padding rows are zero: they add nothing below
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[c] += double(f[c]);
        if (SICS) add_unit_row<V>(f, uacc);
      }
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      part[grp][vec * 8 + c] = acc[c];
      if (SICS) upart[grp][vec * 8 + c] = uacc[c];
    }
    __syncthreads();
    double u2 = 0.0;
    if (threadIdx.x < D) {
      const int c = threadIdx.x;
      double t = 0.0;
      for (int r = 0; r < G; ++r) t += part[r][c];
      double* bar = which ? kbar : qbar;
      if (bar) bar[(bh_blk * g.NB + b) * D + c] = t / double(n);
      if (SICS) {
        double u = 0.0;
        for (int r = 0; r < G; ++r) u += upart[r][c];
        u2 = u * u;
      }
    }
    if (SICS) {
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) u2 += __shfl_xor(u2, m, 64);
      if ((threadIdx.x & 63) == 0) sq[threadIdx.x >> 6] = u2;
    }
    __syncthreads();
    if (SICS && threadIdx.x == 0) {
      double t = 0.0;
      for (int w = 0; w < D / 64; ++w) t += sq[w];
      (which ? sics_k : sics_q)[bh_blk * g.NB + b] = t;
    }
    __syncthreads();
  }
}

// Max/min Summarizer (§3.1: the summaries DSA-SPADE's estimators take) and SICS
// in one pass over the raster tensors: per block, the elementwise max and min
// of its real rows of Q, then K. bf16 values are exact in fp32, so the extremes
// are exact; SICS is accumulated exactly as block_summarize_kernel does (same
// rows, same operations, same order), so the two calls agree bit for bit.
template <int D, bool SICS>
__global__ void __launch_bounds__(kThreads) block_minmax_kernel(
    DevGeom g, HeadMap hm, const uint4* __restrict__ q, const uint4* __restrict__ k,
    double* __restrict__ qmax, double* __restrict__ qmin, double* __restrict__ kmax,
    double* __restrict__ kmin, double* __restrict__ sics_q, double* __restrict__ sics_k) {
  constexpr int V = D / 8;
  constexpr int G = kThreads / V;
  __shared__ float pmax[G][D];
  __shared__ float pmin[G][D];
  __shared__ double upart[SICS ? G : 1][SICS ? D : 1];
  __shared__ double sq[kThreads / 64];

  const int b = blockIdx.x;
  int64_t bh_blk, bh_ras;
  head_pair(g, hm, &bh_blk, &bh_ras);
  const BlockExt e = block_ext(g, b);
  const int n = e.n;
  const float r_ew = 1.0f / float(e.ew), r_eh = 1.0f / float(e.eh);
  const int vec = threadIdx.x % V, grp = threadIdx.x / V;

  for (int which = 0; which < 2; ++which) {
    const uint4* src = (which ? k : q) + bh_ras * g.N * V;
    float mx[8], mn[8];
    double uacc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      mx[c] = -INFINITY;
      mn[c] = INFINITY;
      uacc[c] = 0.0;
    }
    for (int s0 = 0; s0 < n; s0 += kRowBatch * G) {
      uint4 v[kRowBatch];
#pragma unroll
      for (int r = 0; r < kRowBatch; ++r) {
        const int s = s0 + r * G + grp;
        v[r] = make_uint4(0, 0, 0, 0);
        if (s < n) v[r] = src[block_slot_token(g, e, r_ew, r_eh, s) * V + vec];
      }
#pragma unroll
      for (int r = 0; r < kRowBatch; ++r) {
        const bool real = s0 + r * G + grp < n;  // extremes skip the zero rows
        float f[8];
        bf16x8_to_f32(v[r], f);
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          mx[c] = real ? fmaxf(mx[c], f[c]) : mx[c];
          mn[c] = real ? fminf(mn[c], f[c]) : mn[c];
        }
        if (SICS) add_unit_row<V>(f, uacc);
      }
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      pmax[grp][vec * 8 + c] = mx[c];
      pmin[grp][vec * 8 + c] = mn[c];
      if (SICS) upart[grp][vec * 8 + c] = uacc[c];
    }
    __syncthreads();
    double u2 = 0.0;
    if (threadIdx.x < D) {
      const int c = threadIdx.x;
      float a = pmax[0][c], z = pmin[0][c];
      for (int r = 1; r < G; ++r) {
        a = fmaxf(a, pmax[r][c]);
        z = fminf(z, pmin[r][c]);
      }
      const int64_t o = (bh_blk * g.NB + b) * D + c;
      (which ? kmax : qmax)[o] = double(a);
      (which ? kmin : qmin)[o] = double(z);
      if (SICS) {
        double u = 0.0;
        for (int r = 0; r < G; ++r) u += upart[r][c];
        u2 = u * u;
      }
    }
    if (SICS) {
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) u2 += __shfl_xor(u2, m, 64);
      if ((threadIdx.x & 63) == 0) sq[threadIdx.x >> 6] = u2;
    }
    __syncthreads();
    if (SICS && threadIdx.x == 0) {
      double t = 0.0;
      for (int w = 0; w < D / 64; ++w) t += sq[w];
      (which ? sics_k : sics_q)[bh_blk * g.NB + b] = t;
    }
    __syncthreads();
  }
}

template <int D>
hipError_t launch_mm(const DevGeom& g, const HeadMap& hm, const void* q, const void* k,
                     double* qmax, double* qmin, double* kmax, double* kmin, double* sics_q,
                     double* sics_k, hipStream_t s) {
  const dim3 grid(g.NB, g.B * hm.n);
  const uint4* q4 = static_cast<const uint4*>(q);
  const uint4* k4 = static_cast<const uint4*>(k);
  if (sics_q)
    block_minmax_kernel<D, true><<<grid, kThreads, 0, s>>>(g, hm, q4, k4, qmax, qmin, kmax, kmin,
                                                          sics_q, sics_k);
  else
    block_minmax_kernel<D, false><<<grid, kThreads, 0, s>>>(g, hm, q4, k4, qmax, qmin, kmax,
                                                           kmin, nullptr, nullptr);
  return hipGetLastError();
}

template <int D, bool SICS>
hipError_t launch_bs(const DevGeom& g, const HeadMap& hm, const void* q, const void* k, void* qb,
                     void* kb, double* qbar, double* kbar, double* sics_q, double* sics_k,
                     hipStream_t s) {
  const dim3 grid(g.NB, g.B * hm.n);
  const uint4* q4 = static_cast<const uint4*>(q);
  const uint4* k4 = static_cast<const uint4*>(k);
  if (qb)
    block_summarize_kernel<D, SICS, true><<<grid, kThreads, 0, s>>>(
        g, hm, q4, k4, static_cast<uint4*>(qb), static_cast<uint4*>(kb), qbar, kbar, sics_q,
        sics_k);
  else
    block_summarize_kernel<D, SICS, false><<<grid, kThreads, 0, s>>>(
        g, hm, q4, k4, nullptr, nullptr, qbar, kbar, sics_q, sics_k);
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(const DevGeom& g, const void* qb, const void* kb, double* qbar, double* kbar,
                    double* sics_q, double* sics_k, hipStream_t s) {
  const dim3 grid(g.NB, g.B * g.H);
  const uint4* q = static_cast<const uint4*>(qb);
  const uint4* k = static_cast<const uint4*>(kb);
  if (sics_q)
    summarize_kernel<D, true><<<grid, kThreads, 0, s>>>(g, q, k, qbar, kbar, sics_q, sics_k);
  else
    summarize_kernel<D, false><<<grid, kThreads, 0, s>>>(g, q, k, qbar, kbar, nullptr, nullptr);
  return hipGetLastError();
}

// Per head: the batch mean of every candidate's aggregation score, then the
// first candidate with the largest mean (ties go to the lower candidate index).
__global__ void __launch_bounds__(kThreads) choose_scheme_kernel(const double* __restrict__ as_qk,
                                                                 int C, int B, int H,
                                                                 int* __restrict__ choice,
                                                                 double* __restrict__ best) {
  const int h = blockIdx.x * kThreads + threadIdx.x;
  if (h >= H) return;
  int arg = 0;
  double top = 0.0;
  for (int c = 0; c < C; ++c) {
    double s = 0.0;
    for (int b = 0; b < B; ++b) s += as_qk[(int64_t(c) * B + b) * H + h];
    s /= double(B);
    if (c == 0 || s > top) {
      top = s;
      arg = c;
    }
  }
  choice[h] = arg;
  if (best) best[h] = top;
}

// SICS of every candidate blocking in one pass (the head-wise scheme choice of §3.2
// evaluates each candidate's Eq. (3) score; this reads Q and K once for all of them).
// One workgroup per (region, batch x head, tensor). Phase 1: each group of V lanes
// (one token row, 8 columns per lane) walks whole cells in raster order, summing the
// unit rows in fp64, and parks each cell's sum in LDS. Phase 2: each candidate block
// of the region is the sum of its cells in (t, y, x) cell order; its SICS is that
// sum's squared norm. Both orders are fixed, so the result is deterministic.
// The plan's tables are copied to LDS first: indexed per lane group, reads from the
// kernel arguments would be vector-memory round trips on the critical path.
constexpr int kCandThreads = 512;
constexpr int kCandBatch = 8;  // token rows in flight per lane group

template <int D>
__global__ void __launch_bounds__(kCandThreads)
    candidate_sics_kernel(DevGeom g, CandPlan pl, const uint4* __restrict__ q,
                          const uint4* __restrict__ k) {
  constexpr int V = D / 8;
  constexpr int NG = kCandThreads / V;  // lane groups
  extern __shared__ double cell_sum[];  // [cells][8][V]: a lane's 8 columns V apart (no bank conflicts)
  __shared__ int next_cell;
  __shared__ int s_start[3][kMaxCellsAxis + 1];
  __shared__ unsigned short s_order[kMaxCellLds / (64 * 8)];
  __shared__ unsigned char s_bnd[kMaxCandGeoms][3][kMaxCellsAxis + 1];
  __shared__ int s_ext[kMaxCandGeoms][3], s_nblk[kMaxCandGeoms][3];
  __shared__ int s_nb[kMaxCandGeoms], s_b0[kMaxCandGeoms][3];  // blocks per region, first block
  __shared__ double* s_out[kMaxCandGeoms];
  const int vec = threadIdx.x % V, grp = threadIdx.x / V;
  const int reg = blockIdx.x;
  const int rx = reg % pl.R[2], ry = (reg / pl.R[2]) % pl.R[1], rt = reg / (pl.R[2] * pl.R[1]);
  const int o[3] = {rt * pl.L[0], ry * pl.L[1], rx * pl.L[2]};
  const int G3[3] = {g.T, g.Hs, g.Ws};
  const int64_t bh = blockIdx.y;
  const uint4* src = (blockIdx.z ? k : q) + bh * g.N * V;
  const int ncells = pl.ncell[0] * pl.ncell[1] * pl.ncell[2];

  for (int e = threadIdx.x; e < 3 * (kMaxCellsAxis + 1); e += kCandThreads)
    s_start[e / (kMaxCellsAxis + 1)][e % (kMaxCellsAxis + 1)] =
        pl.start[e / (kMaxCellsAxis + 1)][e % (kMaxCellsAxis + 1)];
  for (int e = threadIdx.x; e < ncells; e += kCandThreads) s_order[e] = pl.order[e];
  for (int e = threadIdx.x; e < pl.C * 3 * (kMaxCellsAxis + 1); e += kCandThreads) {
    const int ci = e / (3 * (kMaxCellsAxis + 1)), r = e % (3 * (kMaxCellsAxis + 1));
    s_bnd[ci][r / (kMaxCellsAxis + 1)][r % (kMaxCellsAxis + 1)] =
        pl.bnd[ci][r / (kMaxCellsAxis + 1)][r % (kMaxCellsAxis + 1)];
  }
  if (threadIdx.x < pl.C) {
    const int ci = threadIdx.x;
    int nb = 1;
    for (int a = 0; a < 3; ++a) {
      s_ext[ci][a] = pl.ext[ci][a];
      s_nblk[ci][a] = pl.nblk[ci][a];
      s_b0[ci][a] = o[a] / pl.ext[ci][a];
      nb *= pl.L[a] / pl.ext[ci][a];
    }
    s_nb[ci] = nb;
    s_out[ci] = blockIdx.z ? pl.sics_k[ci] : pl.sics_q[ci];
  }

  // phase 1: cell sums. Groups take cells from a shared counter, largest first, so
  // the groups finish together; a cell is always summed by one group in raster
  // order, so the result does not depend on which group takes it.
  if (threadIdx.x == 0) next_cell = 0;
  __syncthreads();
  const int leader = (threadIdx.x & 63) & ~(V - 1);  // first lane of this group in the wave
  for (;;) {
    int w = 0;
    if (vec == 0) w = atomicAdd(&next_cell, 1);
    w = __shfl(w, leader, 64);
    if (w >= ncells) break;
    const int c = s_order[w];
    const int cx = c % pl.ncell[2], cy = (c / pl.ncell[2]) % pl.ncell[1];
    const int ct = c / (pl.ncell[2] * pl.ncell[1]);
    const int lo[3] = {o[0] + s_start[0][ct], o[1] + s_start[1][cy], o[2] + s_start[2][cx]};
    int ex[3];
    ex[0] = max(0, min(o[0] + s_start[0][ct + 1], G3[0]) - lo[0]);
    ex[1] = max(0, min(o[1] + s_start[1][cy + 1], G3[1]) - lo[1]);
    ex[2] = max(0, min(o[2] + s_start[2][cx + 1], G3[2]) - lo[2]);
    const int n = ex[0] * ex[1] * ex[2];
    double uacc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) uacc[e] = 0.0;
    // walk the cell in raster order with a carry counter (no divisions); rows past the
    // cell re-read its first row and are replaced by zeros, which add nothing
    int pt = 0, py = 0, px = 0;
    const uint32_t base0 = (uint32_t(lo[0]) * g.Hs + lo[1]) * g.Ws + lo[2];
    auto fetch = [&](int s0, uint4 (&v)[kCandBatch]) {
#pragma unroll
      for (int r = 0; r < kCandBatch; ++r) {
        const bool live = s0 + r < n;
        // 32-bit offsets: one head's rows span < 2^31 bytes (checked on the host)
        const uint32_t tok = live ? base0 + (uint32_t(pt) * g.Hs + py) * g.Ws + px : base0;
        const uint4 x = src[tok * V + vec];
        v[r] = live ? x : make_uint4(0, 0, 0, 0);
        if (++px == ex[2]) {
          px = 0;
          if (++py == ex[1]) {
            py = 0;
            ++pt;
          }
        }
      }
    };
    // two batches in flight: the next batch's loads are issued before this one is summed
    uint4 va[kCandBatch], vb[kCandBatch];
    if (n > 0) fetch(0, va);
    for (int s0 = 0; s0 < n; s0 += 2 * kCandBatch) {
      if (s0 + kCandBatch < n) fetch(s0 + kCandBatch, vb);
#pragma unroll
      for (int r = 0; r < kCandBatch; ++r) {
        float f[8];
        bf16x8_to_f32(va[r], f);  // rows past the cell are zero and add nothing
        add_unit_row<V>(f, uacc);
        __builtin_amdgcn_sched_barrier(0);  // one row at a time: few live temporaries
      }
      if (s0 + 2 * kCandBatch < n) fetch(s0 + 2 * kCandBatch, va);
      if (s0 + kCandBatch < n) {
#pragma unroll
        for (int r = 0; r < kCandBatch; ++r) {
          float f[8];
          bf16x8_to_f32(vb[r], f);
          add_unit_row<V>(f, uacc);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) cell_sum[c * D + e * V + vec] = uacc[e];
  }
  __syncthreads();

  // phase 2: candidate blocks of this region
  int total = 0;
  for (int ci = 0; ci < pl.C; ++ci) total += s_nb[ci];
  for (int w = grp; w < total; w += NG) {
    int ci = 0, j = w;
    while (j >= s_nb[ci]) j -= s_nb[ci++];
    const int px = pl.L[2] / s_ext[ci][2], py = pl.L[1] / s_ext[ci][1];
    const int jx = j % px, jy = (j / px) % py, jt = j / (px * py);
    const int bt = s_b0[ci][0] + jt, by = s_b0[ci][1] + jy, bx = s_b0[ci][2] + jx;
    if (bt >= s_nblk[ci][0] || by >= s_nblk[ci][1] || bx >= s_nblk[ci][2]) continue;
    double u[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) u[e] = 0.0;
    for (int ct = s_bnd[ci][0][jt]; ct < s_bnd[ci][0][jt + 1]; ++ct)
      for (int cy = s_bnd[ci][1][jy]; cy < s_bnd[ci][1][jy + 1]; ++cy)
        for (int cx = s_bnd[ci][2][jx]; cx < s_bnd[ci][2][jx + 1]; ++cx) {
          const double* cs = cell_sum + ((ct * pl.ncell[1] + cy) * pl.ncell[2] + cx) * D + vec;
#pragma unroll
          for (int e = 0; e < 8; ++e) u[e] += cs[e * V];
        }
    double ss = 0.0;
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += u[e] * u[e];
    ss = row_group_sum<V>(ss);
    if (vec == 0) {
      const int NBc = s_nblk[ci][0] * s_nblk[ci][1] * s_nblk[ci][2];
      const int64_t blk = (int64_t(bt) * s_nblk[ci][1] + by) * s_nblk[ci][2] + bx;
      s_out[ci][bh * NBc + blk] = ss;
    }
  }
}

}  // namespace

hipError_t launch_candidate_sics(const DevGeom& g, const CandPlan& plan, const void* q,
                                 const void* k, hipStream_t s) {
  const int ncells = plan.ncell[0] * plan.ncell[1] * plan.ncell[2];
  const size_t lds = size_t(ncells) * g.d * sizeof(double);
  const dim3 grid(unsigned(plan.R[0] * plan.R[1] * plan.R[2]), unsigned(g.B * g.H), 2);
  const uint4* q4 = static_cast<const uint4*>(q);
  const uint4* k4 = static_cast<const uint4*>(k);
  if (g.d == 128) {
    const hipError_t e = ensure_dynamic_lds(
        reinterpret_cast<const void*>(&candidate_sics_kernel<128>), kMaxCellLds);
    if (e != hipSuccess) return e;
    candidate_sics_kernel<128><<<grid, kCandThreads, lds, s>>>(g, plan, q4, k4);
  } else if (g.d == 64) {
    const hipError_t e = ensure_dynamic_lds(
        reinterpret_cast<const void*>(&candidate_sics_kernel<64>), kMaxCellLds);
    if (e != hipSuccess) return e;
    candidate_sics_kernel<64><<<grid, kCandThreads, lds, s>>>(g, plan, q4, k4);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_choose_scheme(const double* as_qk, int C, int B, int H, int* choice,
                                double* best, hipStream_t s) {
  choose_scheme_kernel<<<dim3((H + kThreads - 1) / kThreads), kThreads, 0, s>>>(as_qk, C, B, H,
                                                                               choice, best);
  return hipGetLastError();
}

// Aggregation Score, Eq. (3): per head, the sum of its blocks' SICS, divided by
// sum_b n_b^2 (the value when every block's vectors are parallel) so that
// blockings with different block sizes or padding compare on one scale.
// One workgroup per head; each thread adds a fixed stride of blocks, then a
// fixed-shape tree, so the result does not depend on scheduling.
__global__ void __launch_bounds__(kThreads) aggregation_score_kernel(
    DevGeom g, const double* __restrict__ sics_q, const double* __restrict__ sics_k,
    double* __restrict__ as_q, double* __restrict__ as_k, double* __restrict__ as_sum) {
  __shared__ double red[3][kThreads];
  const int64_t bh = blockIdx.x;
  double sq = 0.0, sk = 0.0, norm = 0.0;
  for (int b = threadIdx.x; b < g.NB; b += kThreads) {
    const double n = double(block_ext(g, b).n);
    sq += sics_q[bh * g.NB + b];
    sk += sics_k[bh * g.NB + b];
    norm += n * n;
  }
  red[0][threadIdx.x] = sq;
  red[1][threadIdx.x] = sk;
  red[2][threadIdx.x] = norm;
  __syncthreads();
  for (int off = kThreads / 2; off > 0; off >>= 1) {
    if (threadIdx.x < off)
      for (int c = 0; c < 3; ++c) red[c][threadIdx.x] += red[c][threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double q = red[0][0] / red[2][0], k = red[1][0] / red[2][0];
    if (as_q) as_q[bh] = q;
    if (as_k) as_k[bh] = k;
    as_sum[bh] = q + k;
  }
}

hipError_t launch_aggregation_score(const DevGeom& g, const double* sics_q, const double* sics_k,
                                    double* as_q, double* as_k, double* as_sum, hipStream_t s) {
  aggregation_score_kernel<<<dim3(g.B * g.H), kThreads, 0, s>>>(g, sics_q, sics_k, as_q, as_k,
                                                                 as_sum);
  return hipGetLastError();
}

hipError_t launch_block_summarize(const DevGeom& g, const HeadMap& hm, const void* q,
                                  const void* k, void* qb, void* kb, double* qbar, double* kbar,
                                  double* sics_q, double* sics_k, hipStream_t s) {
  if (g.d == 128)
    return sics_q ? launch_bs<128, true>(g, hm, q, k, qb, kb, qbar, kbar, sics_q, sics_k, s)
                  : launch_bs<128, false>(g, hm, q, k, qb, kb, qbar, kbar, nullptr, nullptr, s);
  if (g.d == 64)
    return sics_q ? launch_bs<64, true>(g, hm, q, k, qb, kb, qbar, kbar, sics_q, sics_k, s)
                  : launch_bs<64, false>(g, hm, q, k, qb, kb, qbar, kbar, nullptr, nullptr, s);
  return hipErrorInvalidValue;
}

hipError_t launch_block_minmax(const DevGeom& g, const HeadMap& hm, const void* q, const void* k,
                               double* qmax, double* qmin, double* kmax, double* kmin,
                               double* sics_q, double* sics_k, hipStream_t s) {
  if (g.d == 128) return launch_mm<128>(g, hm, q, k, qmax, qmin, kmax, kmin, sics_q, sics_k, s);
  if (g.d == 64) return launch_mm<64>(g, hm, q, k, qmax, qmin, kmax, kmin, sics_q, sics_k, s);
  return hipErrorInvalidValue;
}

hipError_t launch_summarize(const DevGeom& g, const void* qb, const void* kb, double* qbar,
                            double* kbar, double* sics_q, double* sics_k, hipStream_t s) {
  if (g.d == 128) return launch_d<128>(g, qb, kb, qbar, kbar, sics_q, sics_k, s);
  if (g.d == 64) return launch_d<64>(g, qb, kb, qbar, kbar, sics_q, sics_k, s);
  return hipErrorInvalidValue;
}

}  // namespace spade
