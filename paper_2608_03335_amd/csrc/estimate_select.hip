// Inter-block Estimator + Top-K / Top-P index search (paper §3.3; Top-K/Top-P
// mode of §3.1) on gfx950.
//
// One workgroup (8 waves) owns 16 query-block rows of one head.
//  1. Scores: the 16 x NB tile S = qbar kbar^T * scale is computed in fp64 with
//     v_mfma_f64_16x16x4 and parked in LDS. The contraction index is permuted so
//     each lane streams 16-byte pieces of the summary rows.
//  2. Selection: one wave per row. Each row's scores are mapped to order-
//     preserving 64-bit keys held in registers (element e = 64*s + lane). The
//     cut key t* = max{t : W(key >= t) >= need} is found by a most-significant-
//     digit radix search (8-bit digits, per-wave LDS histograms of weight and
//     count), stopping as soon as the chosen digit bucket holds one element.
//     Weights are 1 for Top-K (need = min(k, NB)); for Top-P they are the
//     softmax numerators exp(s - max) in 2^-53 fixed point, so bucket sums are
//     exact integers independent of summation order (need = ceil(tau * Z)).
//     Blocks with key > t* are kept; blocks tied at t* are taken in ascending
//     index order until the rule is met. Kept indices are written ascending.
#include "spade_internal.h"

namespace spade {
namespace {

constexpr int kRows = 16;
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxS = kMaxSelectNB / 64;  // register slots per lane
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

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const uint64_t o = __shfl_xor(v, m, 64);
    v = o > v ? o : v;
  }
  return v;
}
__device__ __forceinline__ double wave_max_f64(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmax(v, __shfl_xor(v, m, 64));
  return v;
}
// sum over lanes strictly above this one
__device__ __forceinline__ uint64_t wave_suffix_excl_u64(uint64_t x, int lane) {
  uint64_t v = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint64_t y = __shfl_down(v, off, 64);
    if (lane + off < 64) v += y;
  }
  return v - x;
}
__device__ __forceinline__ int lanes_below(uint64_t ballot) {
  return __builtin_amdgcn_mbcnt_hi(uint32_t(ballot >> 32),
                                   __builtin_amdgcn_mbcnt_lo(uint32_t(ballot), 0));
}

template <int D>
__global__ void __launch_bounds__(kThreads)
    estimate_select_kernel(DevGeom g, const double* __restrict__ qbar,
                           const double* __restrict__ kbar, int mode, int topk, double tau,
                           double scale, int* __restrict__ counts, int* __restrict__ indices,
                           double* __restrict__ scores_out) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int NB = g.NB;
  double* sc = reinterpret_cast<double*>(smem);                           // [kRows][NB]
  uint64_t* hist_w = reinterpret_cast<uint64_t*>(sc + kRows * NB);         // [kWaves][256]
  unsigned* hist_c = reinterpret_cast<unsigned*>(hist_w + kWaves * 256);  // [kWaves][256]

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i0 = blockIdx.x * kRows;
  const int64_t bh = blockIdx.y;
  const double* qh = qbar + bh * NB * D;
  const double* kh = kbar + bh * NB * D;

  // ---------------- phase 1: scores (fp64 MFMA) ----------------
  // MFMA step (kq, h) contracts d = 8*kq + 2*g4 + h, g4 = lane/16 the k-slot.
  constexpr int KQ = D / 8;
  const int r16 = lane & 15, g4 = lane >> 4;
  double qa[2 * KQ];
  {
    const int row = i0 + r16;
    const double2* p = reinterpret_cast<const double2*>(qh + int64_t(min(row, NB - 1)) * D) + g4;
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) {
      const double2 v = p[4 * kq];
      qa[2 * kq] = row < NB ? v.x : 0.0;
      qa[2 * kq + 1] = row < NB ? v.y : 0.0;
    }
  }
  const int ntiles = (NB + 15) / 16;
  for (int jt = wave; jt < ntiles; jt += kWaves) {
    const int col = jt * 16 + r16;
    const double2* p = reinterpret_cast<const double2*>(kh + int64_t(min(col, NB - 1)) * D) + g4;
    double2 kv[KQ];
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) kv[kq] = p[4 * kq];
    f64x4 acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) {
      acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[2 * kq], kv[kq].x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[2 * kq + 1], kv[kq].y, acc, 0, 0, 0);
    }
    if (col < NB) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {  // acc[r] = S[4r + g4][r16]
        const int rr = 4 * r + g4;
        const double s = acc[r] * scale + 0.0;  // + 0.0 folds -0 into +0
        sc[rr * NB + col] = s;
        if (scores_out && i0 + rr < NB) scores_out[(bh * NB + i0 + rr) * NB + col] = s;
      }
    }
  }
  __syncthreads();

  // ---------------- phase 2: one wave per row ----------------
  const int S = (NB + 63) / 64;
  uint64_t* hw = hist_w + wave * 256;
  unsigned* hc = hist_c + wave * 256;
  for (int rr = wave; rr < kRows; rr += kWaves) {
    const int row = i0 + rr;
    if (row >= NB) break;  // uniform per wave; no block barrier below
    const int64_t rowid = bh * NB + row;
    int* out = indices + rowid * NB;

    if (mode == 1 && tau >= 1.0) {  // Top-P with tau = 1 keeps every block
      for (int e = lane; e < NB; e += 64) out[e] = e;
      if (lane == 0) counts[rowid] = NB;
      continue;
    }

    uint64_t key[kMaxS], w[kMaxS];
    double smax = -INFINITY;
#pragma unroll
    for (int s = 0; s < kMaxS; ++s) {
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
    if (mode == 0) {
#pragma unroll
      for (int s = 0; s < kMaxS; ++s) w[s] = key[s] != 0 ? 1 : 0;
      need = uint64_t(min(topk, NB));
    } else {
      smax = wave_max_f64(smax);
      uint64_t z = 0;
#pragma unroll
      for (int s = 0; s < kMaxS; ++s) {
        const int e = s * 64 + lane;
        if (key[s] != 0) {
          const double ev = exp(sc[rr * NB + e] - smax);       // in (0, 1]
          w[s] = uint64_t(ev * 9007199254740992.0);            // 2^53 fixed point
          z += w[s];
        }
      }
      z = wave_sum_u64(z);
      need = uint64_t(ceil(tau * double(z)));
      need = need < 1 ? 1 : (need > z ? z : need);
    }

    // MSD radix search for t* = max{t : sum_{key >= t} w >= need}
    uint64_t prefix = 0, above = 0, tstar = 0;
    bool keep_all = false;
    for (int pass = 0; pass < 8; ++pass) {
      const int shift = 56 - 8 * pass;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        hw[4 * lane + q] = 0;
        hc[4 * lane + q] = 0;
      }
      wave_sync();
#pragma unroll
      for (int s = 0; s < kMaxS; ++s) {
        const bool cand = key[s] != 0 && (pass == 0 || (key[s] >> (shift + 8)) == (prefix >> (shift + 8)));
        if (cand) {
          const int dg = int((key[s] >> shift) & 255u);
          atomicAdd(reinterpret_cast<unsigned long long*>(&hw[dg]), (unsigned long long)w[s]);
          atomicAdd(&hc[dg], 1u);
        }
      }
      wave_sync();
      uint64_t bw[4], loc[4];
      unsigned bc[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        bw[q] = hw[4 * lane + q];
        bc[q] = hc[4 * lane + q];
      }
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
      if (has == 0) {  // total weight below need (cannot happen for valid rules)
        keep_all = true;
        break;
      }
      const int L = 63 - __builtin_clzll(has);
      // values of the chosen lane
      uint64_t my_suf = 0, my_w = 0;
      unsigned my_c = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (q == bq) {
          my_suf = E + loc[q];
          my_w = bw[q];
          my_c = bc[q];
        }
      const int q_L = __shfl(bq, L, 64);
      const uint64_t suf = __shfl(my_suf, L, 64);
      const uint64_t wD = __shfl(my_w, L, 64);
      const unsigned cD = __shfl(my_c, L, 64);
      const int Dg = 4 * L + q_L;
      prefix |= uint64_t(Dg) << shift;
      if (cD == 1) {  // a single element in the bucket: its key is the cut
        uint64_t kk = 0;
#pragma unroll
        for (int s = 0; s < kMaxS; ++s)
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

    int cnt_out = 0;
    if (keep_all) {
      for (int e = lane; e < NB; e += 64) out[e] = e;
      cnt_out = NB;
    } else {
      // elements strictly above the cut, and the tie group at the cut
      int n_above = 0, n_tie = 0;
      uint64_t w_above = 0, w_tie = 0;
#pragma unroll
      for (int s = 0; s < kMaxS; ++s) {
        const bool gt = key[s] > tstar, eq = key[s] == tstar;
        n_above += __popcll(__ballot(gt));
        n_tie += __popcll(__ballot(eq));
        if (gt) w_above += w[s];
        if (eq) w_tie = w[s];
      }
      w_above = wave_sum_u64(w_above);
      w_tie = wave_max_u64(w_tie);
      long long take;
      if (mode == 0) {
        take = (long long)need - n_above;
      } else {
        const uint64_t rem = need > w_above ? need - w_above : 0;
        take = w_tie > 0 ? (long long)((rem + w_tie - 1) / w_tie) : n_tie;
      }
      take = take < 1 ? 1 : (take > n_tie ? n_tie : take);
      int tie_base = 0;
#pragma unroll
      for (int s = 0; s < kMaxS; ++s) {
        const bool eq = key[s] == tstar;
        const uint64_t be = __ballot(eq);
        const int tr = tie_base + lanes_below(be);
        tie_base += __popcll(be);
        const bool kept = key[s] > tstar || (eq && tr < take);
        const uint64_t bk = __ballot(kept);
        if (kept) out[cnt_out + lanes_below(bk)] = s * 64 + lane;
        cnt_out += __popcll(bk);
      }
    }
    if (lane == 0) counts[rowid] = cnt_out;
  }
}

template <int D>
hipError_t launch_d(const DevGeom& g, const double* qbar, const double* kbar, int mode, int topk,
                    double tau, double scale, int* counts, int* indices, double* scores,
                    hipStream_t s) {
  const size_t lds = size_t(kRows) * g.NB * sizeof(double) + kWaves * 256 * (8 + 4);
  static bool attr_set = false;  // raising the dynamic-LDS cap once is idempotent
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&estimate_select_kernel<D>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       int(kRows * kMaxSelectNB * sizeof(double) + kWaves * 256 * 12));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const dim3 grid((g.NB + kRows - 1) / kRows, g.B * g.H);
  estimate_select_kernel<D><<<grid, kThreads, lds, s>>>(g, qbar, kbar, mode, topk, tau, scale,
                                                        counts, indices, scores);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_estimate_select(const DevGeom& g, const double* qbar, const double* kbar,
                                  int mode, int topk, double tau, double scale, int* counts,
                                  int* indices, double* scores, hipStream_t s) {
  if (g.d == 128) return launch_d<128>(g, qbar, kbar, mode, topk, tau, scale, counts, indices, scores, s);
  if (g.d == 64) return launch_d<64>(g, qbar, kbar, mode, topk, tau, scale, counts, indices, scores, s);
  return hipErrorInvalidValue;
}

}  // namespace spade
