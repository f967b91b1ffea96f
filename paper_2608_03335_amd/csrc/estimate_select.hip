// Inter-block Estimator + Top-K / Top-P index search (paper §3.3; Top-K/Top-P
// mode of §3.1), composed with the intra-block filter, the local window and the
// attention sink (§3.1 sparsity-ratio scheme and utility parameters; §3.3: intra
// scores broadcast and OR-combined with the inter ones, the result united with
// the window and sink masks), on gfx950.
//
// One workgroup (4 waves) owns 12 query-block rows of one head (the MFMA tiles of
// phase 1 span 16 rows; the 4 past the item are computed and dropped). Small
// workgroups keep three per CU, so a layer's items fit one round (Hunyuan: 720 items).
//  1. Scores, the 16 x NB tile parked in LDS, in fp64:
//     MEAN  S = qbar kbar^T * scale with v_mfma_f64_16x16x4. The contraction
//           index is permuted so each lane streams 16-byte pieces of the rows.
//     DSA   per channel max(q~ k_max, q~ k_min) with q~ the query block's
//           midpoint, summed: equal to <q~, k_c> + <|q~|, k_r> (k_c, k_r the key
//           box's centre and half width), so the same MFMA contraction runs
//           over 2d terms.
//     DSA2  per channel the largest product of a query and a key extreme: not
//           a contraction (the max is inside the sum), so plain fp64 VALU.
//  2. Selection: one wave per row. Each row's scores are mapped to order-
//     preserving 64-bit keys held in registers (element e = 64*s + lane). The
//     cut key t* = max{t : W(key >= t) >= need} is found by a most-significant-
//     digit radix search (8-bit digits, per-wave LDS histograms of weight and
//     count), stopping as soon as the chosen digit bucket holds one element.
//     Weights are 1 for Top-K (need = min(k, NB)); for Top-P they are the
//     softmax numerators exp(s - max) in 2^-53 fixed point, so bucket sums are
//     exact integers independent of summation order (need = ceil(tau * Z)).
//     Blocks with key > t* are kept; blocks tied at t* are taken in ascending
//     index order until the rule is met.
//  3. Composition: a block is kept when the inter rule keeps it, when its query
//     block or its key block is marked by the intra filter (incoherent: SICS/n^2
//     below a threshold, or among the k least coherent of the head, found with
//     the same radix cut), when it lies in the query block's window, or when it
//     holds one of the first `sink` raster tokens. Kept indices are written
//     ascending.
#include <climits>

#include "spade_internal.h"

namespace spade {
namespace {

constexpr int kRows = 12;
template <int D>
constexpr int kQsStride = D + 2;  // doubles per staged query row
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
// Register slots per lane of a row's keys (element e = 64 s + lane): SM slots
// hold rows of up to 64 SM blocks; launches pick the smallest of 4, 8, 16.
typedef double f64x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Total order on doubles as unsigned keys (larger score -> larger key); -0 is
// folded into +0 by the caller. Finite scores never map to key 0.
__device__ __forceinline__ uint64_t order_key(double s) {
  const uint64_t u = static_cast<uint64_t>(__double_as_longlong(s));
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Wave-wide reductions without LDS round trips: DPP moves within each 16-lane row
// (quad swaps, half-row and row mirrors: every lane ends with its row's total),
// then the four row totals are read into scalar registers. Integer sums and
// maxima are exact whatever the order.
template <int CTRL, int ROW_MASK = 0xf, int BANK_MASK = 0xf>
__device__ __forceinline__ uint32_t dpp32(uint32_t v) {
  return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), CTRL, ROW_MASK, BANK_MASK, true));
}
template <int CTRL, int ROW_MASK = 0xf, int BANK_MASK = 0xf>
__device__ __forceinline__ uint64_t dpp64(uint64_t v) {
  return (uint64_t(dpp32<CTRL, ROW_MASK, BANK_MASK>(uint32_t(v >> 32))) << 32) |
         dpp32<CTRL, ROW_MASK, BANK_MASK>(uint32_t(v));
}
__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
  return (uint64_t(uint32_t(__builtin_amdgcn_readlane(int(v >> 32), l))) << 32) |
         uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v)), l));
}
__device__ __forceinline__ double readlane_f64(double v, int l) {
  return __longlong_as_double((long long)readlane64(uint64_t(__double_as_longlong(v)), l));
}
// quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror, row_mirror
constexpr int kDppSwap1 = 0xB1, kDppSwap2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  v += dpp64<kDppSwap1>(v);
  v += dpp64<kDppSwap2>(v);
  v += dpp64<kDppHalfMirror>(v);
  v += dpp64<kDppMirror>(v);
  return readlane64(v, 0) + readlane64(v, 16) + readlane64(v, 32) + readlane64(v, 48);
}
__device__ __forceinline__ uint64_t max_u64(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
  v = max_u64(v, dpp64<kDppSwap1>(v));
  v = max_u64(v, dpp64<kDppSwap2>(v));
  v = max_u64(v, dpp64<kDppHalfMirror>(v));
  v = max_u64(v, dpp64<kDppMirror>(v));
  return max_u64(max_u64(readlane64(v, 0), readlane64(v, 16)),
                 max_u64(readlane64(v, 32), readlane64(v, 48)));
}
__device__ __forceinline__ double wave_max_f64(double v) {
  auto d = [](double x) { return uint64_t(__double_as_longlong(x)); };
  v = fmax(v, __longlong_as_double((long long)dpp64<kDppSwap1>(d(v))));
  v = fmax(v, __longlong_as_double((long long)dpp64<kDppSwap2>(d(v))));
  v = fmax(v, __longlong_as_double((long long)dpp64<kDppHalfMirror>(d(v))));
  v = fmax(v, __longlong_as_double((long long)dpp64<kDppMirror>(d(v))));
  return fmax(fmax(readlane_f64(v, 0), readlane_f64(v, 16)),
              fmax(readlane_f64(v, 32), readlane_f64(v, 48)));
}
// sum over lanes strictly above this one: the wave's inclusive prefix sum by DPP
// (row shifts 1, 2, 3 of the input, then 4 and 8 within the row, then the last lane
// of row 0 into row 1 and 3, of row 1 into rows 2 and 3), subtracted from the total
__device__ __forceinline__ uint64_t wave_suffix_excl_u64(uint64_t x, int lane) {
  (void)lane;
  uint64_t v = x + dpp64<0x111>(x);   // row_shr:1
  v += dpp64<0x112>(x);               // row_shr:2
  v += dpp64<0x113>(x);               // row_shr:3
  v += dpp64<0x114, 0xf, 0xe>(v);     // row_shr:4, banks 1-3
  v += dpp64<0x118, 0xf, 0xc>(v);     // row_shr:8, banks 2-3
  v += dpp64<0x142, 0xa, 0xf>(v);     // row_bcast:15 into rows 1 and 3
  v += dpp64<0x143, 0xc, 0xf>(v);     // row_bcast:31 into rows 2 and 3
  return readlane64(v, 63) - v;
}
__device__ __forceinline__ int lanes_below(uint64_t ballot) {
  return __builtin_amdgcn_mbcnt_hi(uint32_t(ballot >> 32),
                                   __builtin_amdgcn_mbcnt_lo(uint32_t(ballot), 0));
}

// Result of one wave's cut: keep keys > tstar, and the first `take` keys equal
// to tstar in ascending element order; all = keep every element.
struct Cut {
  uint64_t tstar;
  long long take;
  bool all;
};

// Radix search of one wave's keys (0 = no element) with weights w for the
// largest t with W(key >= t) >= need. count_rule: the tie group fills the count
// (Top-K); otherwise the mass (Top-P). hw: this wave's LDS histogram of weights
// (a bucket's element count, needed only to stop at a single element, comes from
// ballots, so the contended LDS atomics are the weights' alone).
template <int SM>
__device__ Cut find_cut(const uint64_t (&key)[SM], const uint64_t (&w)[SM], uint64_t need,
                        bool count_rule, uint64_t* hw, int lane) {
  uint64_t prefix = 0, above = 0, tstar = 0;
  for (int pass = 0; pass < 8; ++pass) {
    const int shift = 56 - 8 * pass;
#pragma unroll
    for (int q = 0; q < 4; ++q) hw[4 * lane + q] = 0;
    wave_sync();
#pragma unroll
    for (int s = 0; s < SM; ++s) {
      const bool cand =
          key[s] != 0 && (pass == 0 || (key[s] >> (shift + 8)) == (prefix >> (shift + 8)));
      if (cand) {
        const int dg = int((key[s] >> shift) & 255u);
        atomicAdd(reinterpret_cast<unsigned long long*>(&hw[dg]), (unsigned long long)w[s]);
      }
    }
    wave_sync();
    uint64_t bw[4], loc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) bw[q] = hw[4 * lane + q];
    loc[3] = bw[3];
    loc[2] = loc[3] + bw[2];
    loc[1] = loc[2] + bw[1];
    loc[0] = loc[1] + bw[0];
    const uint64_t E = wave_suffix_excl_u64(loc[0], lane);
    int bq = -1;
#pragma unroll
    for (int q = 3; q >= 0; --q)
      if (bq < 0 && above + E + loc[q] >= need) bq = q;
    const uint64_t has = __ballot(bq >= 0);
    if (has == 0) return {0, 0, true};  // total weight below need
    const int L = 63 - __builtin_clzll(has);
    uint64_t my_suf = 0, my_w = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (q == bq) {
        my_suf = E + loc[q];
        my_w = bw[q];
      }
    const int q_L = __builtin_amdgcn_readlane(bq, L);  // L is uniform (from a ballot)
    const uint64_t suf = readlane64(my_suf, L);
    const uint64_t wD = readlane64(my_w, L);
    const int Dg = 4 * L + q_L;
    prefix |= uint64_t(Dg) << shift;
    int cD = 0;  // elements in the chosen bucket
#pragma unroll
    for (int s = 0; s < SM; ++s)
      cD += __popcll(__ballot(key[s] != 0 && (key[s] >> shift) == (prefix >> shift)));
    if (cD == 1) {  // a single element in the bucket: its key is the cut
      uint64_t kk = 0;
#pragma unroll
      for (int s = 0; s < SM; ++s)
        if (key[s] != 0 && (key[s] >> shift) == (prefix >> shift)) kk = key[s];
      tstar = wave_max_u64(kk);
      break;
    }
    if (pass == 7) {  // all 64 bits fixed: a group of equal keys
      tstar = prefix;
      break;
    }
    above += suf - wD;
  }
  // elements strictly above the cut, and the tie group at the cut
  int n_above = 0, n_tie = 0;
  uint64_t w_above = 0, w_tie = 0;
#pragma unroll
  for (int s = 0; s < SM; ++s) {
    const bool gt = key[s] > tstar, eq = key[s] == tstar;
    n_above += __popcll(__ballot(gt));
    n_tie += __popcll(__ballot(eq));
    if (gt) w_above += w[s];
    if (eq) w_tie = w[s];
  }
  w_above = wave_sum_u64(w_above);
  w_tie = wave_max_u64(w_tie);
  long long take;
  if (count_rule) {
    take = (long long)need - n_above;
  } else {
    const uint64_t rem = need > w_above ? need - w_above : 0;
    take = w_tie > 0 ? (long long)((rem + w_tie - 1) / w_tie) : n_tie;
  }
  take = take < 1 ? 1 : (take > n_tie ? n_tie : take);
  return {tstar, take, false};
}

// Block-grid coordinates packed as (tb << 20) | (hb << 10) | wb (each < 1024
// because NB <= 1024).
__device__ __forceinline__ int pack_coords(const DevGeom& g, int b) {
  const int wb = b % g.nW, r = b / g.nW;
  return ((r / g.nH) << 20) | ((r % g.nH) << 10) | wb;
}

__device__ __forceinline__ bool in_window(int ci, int cj, int wt, int wh, int ww) {
  return abs((ci >> 20) - (cj >> 20)) <= wt && abs(((ci >> 10) & 1023) - ((cj >> 10) & 1023)) <= wh &&
         abs((ci & 1023) - (cj & 1023)) <= ww;
}

// coherence SICS / n^2 of block b (intra-block filter input)
__device__ __forceinline__ double coherence(const DevGeom& g, const double* sics, int b) {
  const double n = double(block_ext(g, b).n);
  return sics[b] / (n * n);
}

// Marks of the intra Top-K filter over one head's blocks: the `k` least
// coherent (ties to the lower index), written as 1s into mark[e - lo] for
// lo <= e < hi. One wave.
template <int SM>
__device__ void intra_topk_marks(const DevGeom& g, const double* sics, int k, int lo, int hi,
                                 unsigned char* mark, uint64_t* hw, int lane) {
  const int NB = g.NB;
  uint64_t key[SM], w[SM];
#pragma unroll
  for (int s = 0; s < SM; ++s) {
    const int e = s * 64 + lane;
    key[s] = e < NB ? order_key(-coherence(g, sics, e) + 0.0) : 0;  // least coherent first
    w[s] = key[s] != 0 ? 1 : 0;
  }
  const Cut c = find_cut<SM>(key, w, uint64_t(min(k, NB)), true, hw, lane);
  int tie_base = 0;
#pragma unroll
  for (int s = 0; s < SM; ++s) {
    const int e = s * 64 + lane;
    const bool eq = key[s] != 0 && key[s] == c.tstar;
    const uint64_t be = __ballot(eq);
    const int tr = tie_base + lanes_below(be);
    tie_base += __popcll(be);
    const bool kept = key[s] != 0 && (c.all || key[s] > c.tstar || (eq && tr < c.take));
    if (kept && e >= lo && e < hi) mark[e - lo] = 1;
  }
}

// Rows of up to 512 blocks (SM <= 8) fit in 128 VGPRs with the DSA2 estimator (up to
// four waves per SIMD) and in 168 with the mean estimator, whose score phase holds two
// key tiles (three waves per SIMD); the LDS (12 score rows + histograms) allows three
// workgroups per CU either way.
template <int D, int EST, int SM>
__global__ void __launch_bounds__(kThreads)
    __attribute__((amdgpu_waves_per_eu(SM <= 8 && EST != kEstDsa ? (EST == kEstMean ? 3 : 4) : 1)))
    select_kernel(DevGeom g, SelectSpec p) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int NB = g.NB;
  double* sc = reinterpret_cast<double*>(smem);                           // [kRows][NB]
  uint64_t* hist_w = reinterpret_cast<uint64_t*>(sc + kRows * NB);         // [kWaves][256]
  int* coord = reinterpret_cast<int*>(hist_w + kWaves * 256);             // [NB]
  unsigned char* colmark = reinterpret_cast<unsigned char*>(coord + NB);  // [NB]
  unsigned char* rowmark = colmark + NB;                                  // [kRows]

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // Workgroup w runs on XCD w % 8. The (head, row group) items are numbered head-major
  // and each XCD takes one contiguous eighth of them, so a head's row groups share
  // one XCD (two at a boundary) and its key summaries are fetched into that XCD's L2
  // once instead of into every XCD's.
  const int n_rg = (g.NB + kRows - 1) / kRows;
  const int64_t items = int64_t(g.B) * g.H * n_rg;
  const int64_t per_xcd = (items + 7) / 8;
  const int64_t item = int64_t(blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (item >= items) return;  // grid padding: the whole workgroup leaves together
  const int i0 = int(item % n_rg) * kRows;
  const int64_t bh = item / n_rg;
  const int h = int(bh % g.H);
  const double* q0 = p.q0 + bh * NB * D;
  const double* k0 = p.k0 + bh * NB * D;

  // ---------------- phase 1: scores ----------------
  constexpr int KQ = D / 8;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int ntiles = (NB + 15) / 16;
  if (EST != kEstDsa2) {
    // MFMA step (kq, h) contracts d = 8*kq + 2*g4 + h, g4 = lane/16 the k-slot.
    // DSA: A = q~ = (qmax + qmin)/2 against B = k_c, then |q~| against k_r.
    if (EST == kEstMean) {
      // The item's query summaries (16 rows: the tile's rows past the item zero) are
      // staged in LDS, in the area the selection phase later uses for its histograms:
      // the A operand is read from there, which leaves the registers to hold two key
      // tiles, so the next tile's loads are in flight while this one is contracted.
      // Rows padded to D + 2 doubles: the 16 rows a quarter wave reads hit distinct banks.
      double* qs = reinterpret_cast<double*>(hist_w);  // [16][kQsStride]
      for (int e = threadIdx.x; e < 16 * D; e += kThreads) {
        const int r = e / D, row = i0 + r;
        qs[r * kQsStride<D> + e % D] = (r < kRows && row < NB) ? q0[int64_t(row) * D + e % D] : 0.0;
      }
      __syncthreads();
      auto load_k = [&](double2 (&kv)[KQ], int jt) {
        const int col = jt * 16 + r16;
        const double2* pk = reinterpret_cast<const double2*>(k0 + int64_t(min(col, NB - 1)) * D) + g4;
#pragma unroll
        for (int kq = 0; kq < KQ; ++kq) kv[kq] = pk[4 * kq];
      };
      auto tile = [&](const double2 (&kv)[KQ], int jt) {
        const int col = jt * 16 + r16;
        const double* qrow = qs + r16 * kQsStride<D> + 2 * g4;
        f64x4 acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int kq = 0; kq < KQ; ++kq) {
          const double2 a = *reinterpret_cast<const double2*>(qrow + 8 * kq);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a.x, kv[kq].x, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a.y, kv[kq].y, acc, 0, 0, 0);
        }
        if (col < NB) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {  // acc[r] = S[4r + g4][r16]
            const int rr = 4 * r + g4;  // tile rows past kRows belong to the next item
            const double sv = acc[r] * p.scale + 0.0;  // + 0.0 folds -0 into +0
            if (rr < kRows) sc[rr * NB + col] = sv;
            if (p.scores && rr < kRows && i0 + rr < NB) p.scores[(bh * NB + i0 + rr) * NB + col] = sv;
          }
        }
      };
      double2 kA[KQ], kB[KQ];
      int jt = wave;
      if (jt < ntiles) load_k(kA, jt);
      for (; jt < ntiles; jt += 2 * kWaves) {
        const int jt1 = jt + kWaves;
        if (jt1 < ntiles) load_k(kB, jt1);
        tile(kA, jt);
        if (jt1 >= ntiles) break;
        if (jt1 + kWaves < ntiles) load_k(kA, jt1 + kWaves);
        tile(kB, jt1);
      }
    } else {
    double qa[2 * KQ];
    {
      const int row = i0 + r16;
      const int64_t ro = int64_t(min(row, NB - 1)) * D;
      const double2* p0 = reinterpret_cast<const double2*>(q0 + ro) + g4;
      const double2* p1 = EST == kEstDsa ? reinterpret_cast<const double2*>(p.q1 + bh * NB * D + ro) + g4
                                         : nullptr;
#pragma unroll
      for (int kq = 0; kq < KQ; ++kq) {
        double2 v = p0[4 * kq];
        if (EST == kEstDsa) {
          const double2 u = p1[4 * kq];
          v.x = (v.x + u.x) * 0.5;
          v.y = (v.y + u.y) * 0.5;
        }
        qa[2 * kq] = row < NB ? v.x : 0.0;
        qa[2 * kq + 1] = row < NB ? v.y : 0.0;
      }
    }
    for (int jt = wave; jt < ntiles; jt += kWaves) {
      const int col = jt * 16 + r16;
      const int64_t co = int64_t(min(col, NB - 1)) * D;
      const double2* pk = reinterpret_cast<const double2*>(k0 + co) + g4;
      f64x4 acc = {0.0, 0.0, 0.0, 0.0};
      if (EST == kEstMean) {
#pragma unroll
        for (int kq = 0; kq < KQ; ++kq) {
          const double2 kv = pk[4 * kq];
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[2 * kq], kv.x, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[2 * kq + 1], kv.y, acc, 0, 0, 0);
        }
      } else {
        const double2* pn = reinterpret_cast<const double2*>(p.k1 + bh * NB * D + co) + g4;
#pragma unroll
        for (int kq = 0; kq < KQ; ++kq) {
          const double2 a = pk[4 * kq], b = pn[4 * kq];
          const double cx = (a.x + b.x) * 0.5, cy = (a.y + b.y) * 0.5;  // centre (exact)
          const double rx = (a.x - b.x) * 0.5, ry = (a.y - b.y) * 0.5;  // half width (exact)
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[2 * kq], cx, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[2 * kq + 1], cy, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(fabs(qa[2 * kq]), rx, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64(fabs(qa[2 * kq + 1]), ry, acc, 0, 0, 0);
        }
      }
      if (col < NB) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {  // acc[r] = S[4r + g4][r16]
          const int rr = 4 * r + g4;  // tile rows past kRows belong to the next item
          const double s = acc[r] * p.scale + 0.0;  // + 0.0 folds -0 into +0
          if (rr < kRows) sc[rr * NB + col] = s;
          if (p.scores && rr < kRows && i0 + rr < NB) p.scores[(bh * NB + i0 + rr) * NB + col] = s;
        }
      }
    }
    }
  } else {
    // DSA2 on the VALU: lane (r16, g4) scores column jt*16 + r16 against rows
    // 4r + g4, summing channels in order.
    const double* q1 = p.q1 + bh * NB * D;
    const double* k1 = p.k1 + bh * NB * D;
    for (int jt = wave; jt < ntiles; jt += kWaves) {
      const int col = jt * 16 + r16;
      const int64_t co = int64_t(min(col, NB - 1)) * D;
      double acc[4] = {0.0, 0.0, 0.0, 0.0};
      int64_t ro[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) ro[r] = int64_t(min(i0 + 4 * r + g4, NB - 1)) * D;
      for (int c = 0; c < D; c += 2) {
        const double2 kx = *reinterpret_cast<const double2*>(k0 + co + c);
        const double2 kn = *reinterpret_cast<const double2*>(k1 + co + c);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const double2 qx = *reinterpret_cast<const double2*>(q0 + ro[r] + c);
          const double2 qn = *reinterpret_cast<const double2*>(q1 + ro[r] + c);
          acc[r] += fmax(fmax(qx.x * kx.x, qx.x * kn.x), fmax(qn.x * kx.x, qn.x * kn.x));
          acc[r] += fmax(fmax(qx.y * kx.y, qx.y * kn.y), fmax(qn.y * kx.y, qn.y * kn.y));
        }
      }
      if (col < NB) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int rr = 4 * r + g4;
          const double s = acc[r] * p.scale + 0.0;
          if (rr < kRows) sc[rr * NB + col] = s;
          if (p.scores && rr < kRows && i0 + rr < NB) p.scores[(bh * NB + i0 + rr) * NB + col] = s;
        }
      }
    }
  }

  __syncthreads();  // staged query rows dead: their area becomes the histograms
  // ---------------- composition inputs ----------------
  const bool window = p.wt >= 0;
  const bool extras = p.intra != kIntraNone || window || p.sink > 0;
  if (extras) {
    const double* sk = p.sics_k ? p.sics_k + bh * NB : nullptr;
    for (int j = threadIdx.x; j < NB; j += kThreads) {
      bool m = false;
      if (p.sink > 0) {
        const BlockExt e = block_ext(g, j);
        m = (int64_t(e.t0) * g.Hs + e.y0) * g.Ws + e.x0 < p.sink;  // its first raster token
      }
      if (p.intra == kIntraThreshold) m = m || coherence(g, sk, j) < p.intra_theta;
      colmark[j] = m;
      if (window) coord[j] = pack_coords(g, j);
    }
    if (threadIdx.x < kRows) {
      const int row = i0 + threadIdx.x;
      rowmark[threadIdx.x] = p.intra == kIntraThreshold && row < NB &&
                             coherence(g, p.sics_q + bh * NB, row) < p.intra_theta;
    }
  }
  __syncthreads();
  if (p.intra == kIntraTopk && p.intra_k > 0) {
    if (wave == 0)
      intra_topk_marks<SM>(g, p.sics_k + bh * NB, p.intra_k, 0, NB, colmark, hist_w, lane);
    else if (wave == 1)
      intra_topk_marks<SM>(g, p.sics_q + bh * NB, p.intra_k, i0, i0 + kRows, rowmark,
                           hist_w + 256, lane);
    __syncthreads();
  }

  // ---------------- phase 2: one wave per row ----------------
  const int S = (NB + 63) / 64;
  uint64_t* hw = hist_w + wave * 256;
  const int topk = p.topk_h ? min(max(p.topk_h[h], 1), NB) : p.topk;
  const double tau = p.tau_h ? p.tau_h[h] : p.tau;
  for (int rr = wave; rr < kRows; rr += kWaves) {
    const int row = i0 + rr;
    if (row >= NB) break;  // uniform per wave; no block barrier below
    const int64_t rowid = bh * NB + row;
    int* out = p.indices + rowid * NB;

    if ((p.mode == 1 && tau >= 1.0) || (extras && rowmark[rr])) {  // every block kept
      for (int e = lane; e < NB; e += 64) out[e] = e;
      if (lane == 0) p.counts[rowid] = NB;
      continue;
    }

    uint64_t key[SM], w[SM];
    double smax = -INFINITY;
#pragma unroll
    for (int s = 0; s < SM; ++s) {
      key[s] = 0;
      w[s] = 0;
      const int e = s * 64 + lane;
      if (s < S && e < NB) {
        const double v = sc[rr * NB + e];
        key[s] = order_key(v);
        smax = fmax(smax, v);
      }
    }
    uint64_t need;
    if (p.mode == 0) {
#pragma unroll
      for (int s = 0; s < SM; ++s) w[s] = key[s] != 0 ? 1 : 0;
      need = uint64_t(min(topk, NB));
    } else {
      smax = wave_max_f64(smax);
      uint64_t z = 0;
#pragma unroll
      for (int s = 0; s < SM; ++s) {
        const int e = s * 64 + lane;
        if (key[s] != 0) {
          const double ev = exp(sc[rr * NB + e] - smax);       // in (0, 1]
          w[s] = uint64_t(ev * 9007199254740992.0);            // 2^53 fixed point
          z += w[s];
        }
      }
      z = wave_sum_u64(z);
      const double t = tau > 0.0 ? tau : 0.0;  // NaN or <= 0: the top block only
      need = uint64_t(ceil(t * double(z)));
      need = need < 1 ? 1 : (need > z ? z : need);
    }
    const Cut c = find_cut<SM>(key, w, need, p.mode == 0, hw, lane);

    int cnt_out = 0;
    if (c.all) {
      for (int e = lane; e < NB; e += 64) out[e] = e;
      cnt_out = NB;
    } else {
      const int ci = window ? coord[row] : 0;
      int tie_base = 0;
#pragma unroll
      for (int s = 0; s < SM; ++s) {
        const int e = s * 64 + lane;
        const bool eq = key[s] == c.tstar;
        const uint64_t be = __ballot(eq);
        const int tr = tie_base + lanes_below(be);
        tie_base += __popcll(be);
        bool kept = key[s] > c.tstar || (eq && tr < c.take);
        if (extras && !kept && s < S && e < NB)
          kept = colmark[e] || (window && in_window(ci, coord[e], p.wt, p.wh, p.ww));
        const uint64_t bk = __ballot(kept);
        if (kept) out[cnt_out + lanes_below(bk)] = e;
        cnt_out += __popcll(bk);
      }
    }
    if (lane == 0) p.counts[rowid] = cnt_out;
  }
}

template <int D, int EST, int SM>
hipError_t launch_des(const DevGeom& g, const SelectSpec& p, hipStream_t s) {
  // after the score rows: the histograms and marks of the selection phase, sharing
  // their area with the staged query rows of the score phase
  auto tail = [](int NB) {
    const size_t sel = size_t(kWaves) * 256 * 8 + size_t(NB) * (4 + 1) + kRows;
    const size_t qst = EST == kEstMean ? size_t(16) * kQsStride<D> * sizeof(double) : 0;
    return sel > qst ? sel : qst;
  };
  const size_t lds = size_t(kRows) * g.NB * sizeof(double) + tail(g.NB);
  const hipError_t e = ensure_dynamic_lds(
      reinterpret_cast<const void*>(&select_kernel<D, EST, SM>),
      int(kRows * kMaxSelectNB * sizeof(double) + tail(kMaxSelectNB)));
  if (e != hipSuccess) return e;
  const int64_t items = int64_t(g.B) * g.H * ((g.NB + kRows - 1) / kRows);
  const dim3 grid(unsigned((items + 7) / 8 * 8));  // see the XCD mapping in the kernel
  select_kernel<D, EST, SM><<<grid, kThreads, lds, s>>>(g, p);
  return hipGetLastError();
}

template <int D, int EST>
hipError_t launch_de(const DevGeom& g, const SelectSpec& p, hipStream_t s) {
  if (g.NB <= 256) return launch_des<D, EST, 4>(g, p, s);
  if (g.NB <= 512) return launch_des<D, EST, 8>(g, p, s);
  return launch_des<D, EST, 16>(g, p, s);
}

template <int D>
hipError_t launch_d(const DevGeom& g, const SelectSpec& p, hipStream_t s) {
  switch (p.estimator) {
    case kEstMean: return launch_de<D, kEstMean>(g, p, s);
    case kEstDsa: return launch_de<D, kEstDsa>(g, p, s);
    case kEstDsa2: return launch_de<D, kEstDsa2>(g, p, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_select(const DevGeom& g, const SelectSpec& p, hipStream_t s) {
  if (g.d == 128) return launch_d<128>(g, p, s);
  if (g.d == 64) return launch_d<64>(g, p, s);
  return hipErrorInvalidValue;
}

}  // namespace spade

// Checks of block lists in the layout select_kernel writes (a debug aid: the
// attention kernels accept any lists). One wave per row (b, h, i); a failing row
// adds itself to the report with vector-memory atomics.
namespace spade {
namespace {

__global__ void __launch_bounds__(64) clear_report_kernel(int* __restrict__ report) {
  if (threadIdx.x < 4) report[threadIdx.x] = threadIdx.x == 1 ? INT_MAX : 0;
}

__global__ void __launch_bounds__(256) validate_lists_kernel(int NB, int rows,
                                                             const int* __restrict__ counts,
                                                             const int* __restrict__ indices,
                                                             int* __restrict__ report) {
  const int row = int(blockIdx.x) * 4 + int(threadIdx.x >> 6);
  if (row >= rows) return;
  const int lane = threadIdx.x & 63;
  const int c = counts[row];
  int bad = 0;
  if (c < 0 || c > NB) {
    bad = kListBadCount;
  } else {
    const int* ind = indices + int64_t(row) * NB;
    for (int e = lane; e < c; e += 64) {
      const int j = ind[e];
      if (j < 0 || j >= NB) bad |= kListBadIndex;
      if (e > 0 && ind[e - 1] >= j) bad |= kListNotAscending;
    }
    bad = (__ballot(bad & kListBadCount) ? kListBadCount : 0) |
          (__ballot(bad & kListBadIndex) ? kListBadIndex : 0) |
          (__ballot(bad & kListNotAscending) ? kListNotAscending : 0);
  }
  if (bad != 0 && lane == 0) {
    atomicAdd(report, 1);
    atomicMin(report + 1, row);
    atomicOr(report + 2, bad);
  }
}

}  // namespace

hipError_t launch_validate_lists(int NB, int rows, const int* counts, const int* indices,
                                 int* report, hipStream_t s) {
  clear_report_kernel<<<1, 64, 0, s>>>(report);
  if (rows > 0)
    validate_lists_kernel<<<dim3(unsigned((rows + 3) / 4)), 256, 0, s>>>(NB, rows, counts, indices,
                                                                         report);
  return hipGetLastError();
}

}  // namespace spade
