// Flash block-sparse attention (paper Eq. (2), §3.3 optimisation (3)) on gfx950.
//
// One workgroup per query block (b, h, i); wave w owns query slots 32w..32w+31.
// The kept K/V blocks of row (b, h, i) are walked in ascending block order in
// chunks of 32 key slots (only chunks that contain real keys). Each chunk is
// staged in LDS, double-buffered: while the waves run MFMA on chunk c, the
// next chunk's K and V are already in flight from HBM into registers.
//
// Transposed formulation so that every softmax statistic is per lane:
//   S^T (32 keys x 32 queries) = K_chunk * Q^T   v_mfma_f32_32x32x16_bf16, d/16 steps
//   lane l then holds query row l%32 and 16 of the chunk's keys;
//   O^T (d x 32 queries) += V^T * P^T            P^T taken straight from the
//   S^T accumulators (rounded to bf16) as the B operand; the key order of the
//   contraction is permuted to match the accumulator layout, and V^T is laid
//   out in LDS so each lane reads two 8-byte runs of 4 keys.
// Row max needs one cross-lane exchange (lane l <-> l^32); the row sum is kept
// per lane and combined once at the end. Logits are scaled into base 2 so the
// exponentials are single v_exp_f32 instructions.
#include "spade_internal.h"

namespace spade {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kChunk = 32;  // key slots per chunk

template <int D>
struct Tile {
  static constexpr int KROW = D + 8;         // K rows, bf16 elements (16-byte pad)
  static constexpr int VROW = kChunk + 8;    // V^T rows (one per d), bf16 elements
  static constexpr int K_ELEMS = kChunk * KROW;
  static constexpr int V_ELEMS = D * VROW;
  static constexpr int BUF = K_ELEMS + V_ELEMS;
  static constexpr int ROW_VEC = D / 8;      // 16-byte vectors per token row
  static constexpr int K_LOADS = kChunk * ROW_VEC;      // 16-byte K loads per chunk
  static constexpr int V_UNITS = (kChunk / 4) * ROW_VEC;  // 4 keys x 8 d per unit
};

// Position in the kept-block walk: list entry jj, its block j and real-key count nj,
// and the chunk's first key slot c0.
struct Cursor {
  int jj, j, nj, c0;
};

__device__ __forceinline__ Cursor next_chunk(const DevGeom& g, const int* list, int cnt,
                                             Cursor c) {
  c.c0 += kChunk;
  while (c.c0 >= c.nj) {
    ++c.jj;
    if (c.jj >= cnt) {
      c.nj = 0;
      c.c0 = 0;
      return c;
    }
    const int j = list[c.jj];
    if (j >= 0 && j < g.NB) {
      c.j = j;
      c.nj = block_ext(g, j).n;
      c.c0 = 0;
    }
  }
  return c;
}

template <int D, int W>
__global__ void __launch_bounds__(64 * W)
    attn_kernel(DevGeom g, const uint4* __restrict__ qb, const uint4* __restrict__ kb,
                const uint4* __restrict__ vb, const int* __restrict__ counts,
                const int* __restrict__ indices, float scale_log2, __bf16* __restrict__ ob,
                float* __restrict__ lse) {
  using TL = Tile<D>;
  constexpr int NT = 64 * W;
  constexpr int KL = (TL::K_LOADS + NT - 1) / NT;
  constexpr int VU = (TL::V_UNITS + NT - 1) / NT;
  __shared__ __align__(16) __bf16 lds[2][TL::BUF];

  const int64_t item = blockIdx.x;
  const int64_t bh = item / g.NB;
  const int i = int(item % g.NB);
  const int n_i = block_ext(g, i).n;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q0 = wave * 32;
  const int half = lane >> 5;  // k-slot group of the MFMA operands
  const int r32 = lane & 31;
  const int64_t head_row = bh * g.NB * int64_t(g.BS);

  // Q^T fragments (B operand): query row q0 + r32, d = 16*kk + 8*half .. +8
  bf16x8 qf[D / 16];
  {
    const int qs = q0 + r32;
    const uint4* src = qb + (head_row + int64_t(i) * g.BS + qs) * TL::ROW_VEC + half;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (qs < n_i) v = src[2 * kk];
      qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  const int cnt = min(max(counts[bh * g.NB + i], 0), g.NB);
  const int* list = indices + (bh * g.NB + i) * int64_t(g.NB);

  uint4 kreg[KL];
  uint4 vreg[VU][4];
  auto load_chunk = [&](const Cursor& c) {
    const int64_t base = head_row + int64_t(c.j) * g.BS + c.c0;  // first key row of the chunk
#pragma unroll
    for (int u = 0; u < KL; ++u) {
      const int f = tid + u * NT;
      kreg[u] = make_uint4(0, 0, 0, 0);
      if (f < TL::K_LOADS) {
        const int key = f / TL::ROW_VEC, vec = f % TL::ROW_VEC;
        if (c.c0 + key < c.nj) kreg[u] = kb[(base + key) * TL::ROW_VEC + vec];
      }
    }
#pragma unroll
    for (int u = 0; u < VU; ++u) {
      const int f = tid + u * NT;
#pragma unroll
      for (int r = 0; r < 4; ++r) vreg[u][r] = make_uint4(0, 0, 0, 0);
      if (f < TL::V_UNITS) {
        const int kq = f % (kChunk / 4), dq = f / (kChunk / 4);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = 4 * kq + r;
          if (c.c0 + key < c.nj) vreg[u][r] = vb[(base + key) * TL::ROW_VEC + dq];
        }
      }
    }
  };
  auto store_chunk = [&](__bf16* buf) {
#pragma unroll
    for (int u = 0; u < KL; ++u) {
      const int f = tid + u * NT;
      if (f < TL::K_LOADS) {
        const int key = f / TL::ROW_VEC, vec = f % TL::ROW_VEC;
        *reinterpret_cast<uint4*>(buf + key * TL::KROW + vec * 8) = kreg[u];
      }
    }
    __bf16* vt = buf + TL::K_ELEMS;
#pragma unroll
    for (int u = 0; u < VU; ++u) {
      const int f = tid + u * NT;
      if (f < TL::V_UNITS) {
        const int kq = f % (kChunk / 4), dq = f / (kChunk / 4);
        // vreg[u][r] holds V[key 4kq+r][d 8dq .. 8dq+7]; write V^T rows d, keys 4kq..4kq+3
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          uint32_t lo = 0, hi = 0;
          const int sh = (e & 1) * 16;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const uint32_t w = (e >> 1) == 0 ? vreg[u][r].x : (e >> 1) == 1 ? vreg[u][r].y
                             : (e >> 1) == 2 ? vreg[u][r].z : vreg[u][r].w;
            const uint32_t h16 = (w >> sh) & 0xffffu;
            if (r < 2) lo |= h16 << (16 * r);
            else hi |= h16 << (16 * (r - 2));
          }
          *reinterpret_cast<uint2*>(vt + (8 * dq + e) * TL::VROW + 4 * kq) = make_uint2(lo, hi);
        }
      }
    }
  };

  f32x16 o[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
  float m = -INFINITY, l = 0.0f;
  const bool rows_live = q0 < n_i;

  Cursor cur = {-1, 0, 0, 0};
  cur.c0 = -kChunk;  // so that next_chunk starts at list entry 0, slot 0
  cur = next_chunk(g, list, cnt, cur);
  int buf = 0;
  if (cur.jj < cnt) {
    load_chunk(cur);
    store_chunk(lds[0]);
  }
  __syncthreads();
  while (cur.jj < cnt) {
    const Cursor nxt = next_chunk(g, list, cnt, cur);
    const bool more = nxt.jj < cnt;
    if (more) load_chunk(nxt);
    if (rows_live) {
      const __bf16* K = lds[buf];
      const __bf16* Vt = lds[buf] + TL::K_ELEMS;
      f32x16 s;
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(K + r32 * TL::KROW + 16 * kk + 8 * half);
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], s, 0, 0, 0);
      }
      // s[r]: key (r/4)*8 + 4*half + r%4 of the chunk, query row r32
      float mloc = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kr = (r >> 2) * 8 + 4 * half + (r & 3);
        const float v = (cur.c0 + kr < cur.nj) ? s[r] * scale_log2 : -INFINITY;
        s[r] = v;
        mloc = fmaxf(mloc, v);
      }
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
      const float mnew = fmaxf(m, mloc);
      const float alpha = __builtin_amdgcn_exp2f(m - mnew);
      float psum = 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = __builtin_amdgcn_exp2f(s[r] - mnew);
        psum += s[r];
      }
      l = l * alpha + psum;
      m = mnew;
      bf16x8 p[2];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[0][e] = __bf16(s[e]);
        p[1][e] = __bf16(s[8 + e]);
      }
#pragma unroll
      for (int t = 0; t < D / 32; ++t) {
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][r] *= alpha;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const __bf16* vrow = Vt + (32 * t + r32) * TL::VROW + 16 * u + 4 * half;
          const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vrow);
          const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vrow + 8);
          const bf16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, p[u], o[t], 0, 0, 0);
        }
      }
    }
    if (more) store_chunk(lds[buf ^ 1]);
    __syncthreads();
    buf ^= 1;
    cur = nxt;
  }

  // normalise and store: lane holds query row q0 + r32, d = 32t + 8*rq + 4*half + 0..3
  l += __shfl_xor(l, 32, 64);
  const int qs = q0 + r32;
  if (qs < g.BS) {
    const bool real = qs < n_i;
    const float inv = (real && l > 0.0f) ? 1.0f / l : 0.0f;
    __bf16* dst = ob + (head_row + int64_t(i) * g.BS + qs) * D + 4 * half;
#pragma unroll
    for (int t = 0; t < D / 32; ++t)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        bf16x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = __bf16(o[t][4 * rq + e] * inv);
        *reinterpret_cast<bf16x4*>(dst + 32 * t + 8 * rq) = v;
      }
    if (lse && real && half == 0)
      lse[head_row + int64_t(i) * g.BS + qs] =
          l > 0.0f ? (m + __log2f(l)) * 0.69314718055994530942f : -INFINITY;
  }
}

template <int D, int W>
hipError_t launch_dw(const DevGeom& g, const void* qb, const void* kb, const void* vb,
                     const int* counts, const int* indices, float scale_log2, void* ob, float* lse,
                     hipStream_t s) {
  const int64_t items = int64_t(g.B) * g.H * g.NB;
  attn_kernel<D, W><<<dim3(unsigned(items)), 64 * W, 0, s>>>(
      g, static_cast<const uint4*>(qb), static_cast<const uint4*>(kb),
      static_cast<const uint4*>(vb), counts, indices, scale_log2, static_cast<__bf16*>(ob), lse);
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(const DevGeom& g, const void* qb, const void* kb, const void* vb,
                    const int* counts, const int* indices, float scale_log2, void* ob, float* lse,
                    hipStream_t s) {
  switch ((g.BS + 31) / 32) {
    case 1: return launch_dw<D, 1>(g, qb, kb, vb, counts, indices, scale_log2, ob, lse, s);
    case 2: return launch_dw<D, 2>(g, qb, kb, vb, counts, indices, scale_log2, ob, lse, s);
    case 3: return launch_dw<D, 3>(g, qb, kb, vb, counts, indices, scale_log2, ob, lse, s);
    case 4: return launch_dw<D, 4>(g, qb, kb, vb, counts, indices, scale_log2, ob, lse, s);
    case 5: return launch_dw<D, 5>(g, qb, kb, vb, counts, indices, scale_log2, ob, lse, s);
    case 6: return launch_dw<D, 6>(g, qb, kb, vb, counts, indices, scale_log2, ob, lse, s);
    case 7: return launch_dw<D, 7>(g, qb, kb, vb, counts, indices, scale_log2, ob, lse, s);
    case 8: return launch_dw<D, 8>(g, qb, kb, vb, counts, indices, scale_log2, ob, lse, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

size_t attn_workspace_bytes(const DevGeom&) { return 0; }

hipError_t launch_block_sparse_attn(const DevGeom& g, const void* qb, const void* kb,
                                    const void* vb, const int* counts, const int* indices,
                                    float scale, void* ob, float* lse, void*, hipStream_t s) {
  const float scale_log2 = scale * 1.44269504088896340736f;
  if (g.d == 128) return launch_d<128>(g, qb, kb, vb, counts, indices, scale_log2, ob, lse, s);
  if (g.d == 64) return launch_d<64>(g, qb, kb, vb, counts, indices, scale_log2, ob, lse, s);
  return hipErrorInvalidValue;
}

}  // namespace spade
