// Flash block-sparse attention (paper Eq. (2), §3.3 optimisation (3)) on gfx950.
//
// One workgroup per query block (b, h, i). Three kernels share the data movement
// and the math below:
// - attn_sw_kernel, for blocks of 5 row tiles (129..160 slots) at d = 128: one
//   software-pipelined wave per 32-row tile, the fifth tile split over the four
//   DMA waves (see its comment);
// - attn_pp_kernel, for 5-tile blocks otherwise (d = 64, or kept lists too long
//   for the sw kernel's LDS): two waves per 32-row tile split the kept walk (even /
//   odd chunks) and alternate matrix and vector phases between barriers, so each
//   SIMD overlaps one wave's MFMAs with the other's softmax; the pair merges by
//   log-sum-exp;
// - attn_kernel for every other block size: wave w owns query slots 32w..32w+31;
//   for most block sizes one more wave only issues the K/V loads.
// Work items are dealt to the 8 XCDs so that all XCDs share one head at a time;
// each XCD starts its rows of a head heaviest first (heavy_first).
// The kept K/V blocks of row (b, h, i) are walked in ascending block order in
// chunks of 32 key slots (only chunks that hold real keys).
//
// Data movement: each chunk's K and V rows go straight from HBM into LDS with
// 16-byte global_load_lds (no register staging), double-buffered so chunk c+1
// is in flight while chunk c is computed. The loads are issued from inline asm:
// the compiler then schedules every LDS read with exact lgkmcnt tracking instead
// of draining the in-flight LDS-DMA load before each read (it cannot prove the
// load targets the other buffer); completion is ordered by the explicit wait and
// barrier at the end of each chunk. The work item's kept list is staged in LDS
// once, so the walk over kept blocks issues no vector-memory reads. Rows are stored unpadded with the
// 16-byte pieces XOR-swizzled per row, which keeps both LDS read patterns below
// free of bank conflicts. Key slots past a block's real tokens re-read the
// block's last real row (finite data; their logits are masked).
//
// Math, transposed so every softmax statistic is per lane:
//   S^T (32 keys x 32 queries) = K * Q^T        v_mfma_f32_32x32x16_bf16, d/16 steps;
//     lane l then holds query row l%32 and 16 keys of the chunk.
//   O^T (d x 32 queries) += V^T * P^T           P^T straight from the S^T registers
//     (rounded to bf16) as the B operand; the contraction's key order follows the
//     accumulator layout, and ds_read_b64_tr_b16 delivers V^T fragments in that
//     order from row-major V.
// Softmax: logits are scaled into base 2 (one FMA + v_exp_f32 per element); the
// row max pairs lanes l and l^32 with v_permlane32_swap; the running max is only
// raised (and O rescaled) when some row's max grows by more than 2^8, so most
// chunks skip the 64-register rescale; row sums use bf16 dot2 on the same packed
// P that feeds the MFMA.
#include <climits>
#include <mutex>
#include <type_traits>

#include "spade_internal.h"

// Scratch of the allocation-free raster attention call: the head ranking's keys
// and order, 16 bytes per (batch, head) pair for at most spade::kMaxRankedHeads
// pairs (beyond that the launch runs in grid order and needs none). Each GPU holds
// its own copy until the process ends; host code reaches it only through the
// address hipGetSymbolAddress returns on that device.
static __device__ __align__(256) unsigned char scratch[spade::kNoAllocScratchBytes];

namespace spade {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) int lds_int;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

constexpr int kChunk = 32;          // key slots per chunk
constexpr float kRescaleLog2 = 8.0f;  // lazy-rescale threshold (base-2 logits)

template <int D>
struct Tile {
  static constexpr int NCH = D / 8;                 // 16-byte pieces per row
  static constexpr int ROW_BYTES = D * 2;
  static constexpr int TILE_BYTES = kChunk * ROW_BYTES;
  static constexpr int RPI = 64 / NCH;              // rows per wave-wide 1 KB load
  static constexpr int LOADS = kChunk / RPI;        // wave loads per tile
  static constexpr int BUF_BYTES = 2 * TILE_BYTES;  // K tile then V tile
};

// swizzles: LDS piece c of tile row r holds global piece c ^ f(r)
template <int D>
__device__ __forceinline__ int swz_k(int r) { return r & (Tile<D>::NCH - 1); }
// V: in a transposing read, lanes 0-15 take pieces 4t + {0,1} and lanes 16-31 pieces
// 4t + {2,3} of rows 0-3; an XOR stride of 4 pieces (d = 128) keeps the two groups'
// pieces disjoint, so 32 lanes hit 64 distinct banks (no LDS bank conflicts)
template <int D>
__device__ __forceinline__ int swz_v(int r) { return D >= 128 ? 4 * (r & 3) : 2 * (r & 3); }

// Position in the kept-block walk: list entry jj, its block j and real-key count nj,
// the chunk's first key slot c0, and block j's extent (raster addressing).
struct Cursor {
  int jj, j, nj, c0;
  BlockExt e;
};

// Raster token of slot `slot` of a block of any extent (ragged edge blocks).
__device__ __forceinline__ int64_t ext_token(const DevGeom& g, const BlockExt& e, int slot) {
  return block_slot_token(g, e, __builtin_amdgcn_rcpf(float(e.ew)),
                          __builtin_amdgcn_rcpf(float(e.eh)), slot);
}

// Raster token of a block's first slot.
__device__ __forceinline__ int64_t block_origin(const DevGeom& g, const BlockExt& e) {
  return (int64_t(e.t0) * g.Hs + e.y0) * g.Ws + e.x0;
}

// Raster addressing of slot s of the cursor's block, relative to `base`: full
// blocks (every block away from the grid's far edges) share one slot -> token
// offset table `rel` (LDS, built once per workgroup), so a load costs one LDS
// read instead of the division-based map; ragged blocks take the map.
struct RasterRows {
  bool full;
  int64_t base;  // head_row + block origin (full), head_row (ragged)
};

__device__ __forceinline__ RasterRows raster_rows(const DevGeom& g, const Cursor& c,
                                                  int64_t head_row) {
  const bool full = c.e.n == g.BS;
  return {full, head_row + (full ? block_origin(g, c.e) : 0)};
}

__device__ __forceinline__ Cursor next_chunk(const DevGeom& g, const lds_int* list, int cnt,
                                             Cursor c) {
  c.c0 += kChunk;
  while (c.c0 >= c.nj) {
    ++c.jj;
    if (c.jj >= cnt) {
      c.nj = 0;
      c.c0 = 0;
      return c;
    }
    const int j = __builtin_amdgcn_readfirstlane(list[c.jj]);  // uniform: keep in SGPRs
    if (j >= 0 && j < g.NB) {
      c.j = j;
      c.e = block_ext(g, j);
      c.nj = c.e.n;
      c.c0 = 0;
    }
  }
  return c;
}

// Loads of one chunk without a loader wave: wave w issues loads w, w + W, ...
// of the 2*LOADS (K tiles, then V). wave_rows gives each of them its row
// relative to the chunk's base row (blocked: the block's first row; RASTER: the
// head's first raster row, plus the block origin for full blocks); it is called
// one chunk ahead, so its LDS table reads complete under the current chunk's math.
template <int D, int W>
struct WaveLoads {
  static constexpr int NQ = (2 * Tile<D>::LOADS + W - 1) / W;  // loads per wave (at most)
};

template <int D, int W, bool RASTER>
__device__ __forceinline__ void wave_rows(const DevGeom& g, const Cursor& c, const lds_int* rel,
                                          int wave, int lane, int (&rows)[WaveLoads<D, W>::NQ]) {
  using TL = Tile<D>;
  const int last = c.nj - 1 - c.c0;  // last real key slot of the chunk
  auto fill = [&](auto row_of) {
#pragma unroll
    for (int k = 0; k < WaveLoads<D, W>::NQ; ++k) {
      const int qq = (wave + k * W) % TL::LOADS;
      rows[k] = row_of(c.c0 + min(qq * TL::RPI + lane / TL::NCH, last));
    }
  };
  if (!RASTER)
    fill([](int s) { return s; });
  else if (c.e.n == g.BS)
    fill([&](int s) { return rel[s]; });
  else
    fill([&](int s) { return int(ext_token(g, c.e, s)); });
}

template <int D, int W, bool RASTER>
__device__ __forceinline__ void load_chunk(const DevGeom& g, const char* kb, const char* vb,
                                           int64_t head_row, const Cursor& c,
                                           const int (&rows)[WaveLoads<D, W>::NQ], lds_char* buf,
                                           int wave, int lane) {
  using TL = Tile<D>;
  const int64_t base = RASTER ? raster_rows(g, c, head_row).base
                              : head_row + int64_t(c.j) * g.BS;
  const int piece = lane % TL::NCH;
#pragma unroll
  for (int k = 0; k < WaveLoads<D, W>::NQ; ++k) {
    const int q = wave + k * W;
    if (q < 2 * TL::LOADS) {
      const bool is_v = q >= TL::LOADS;
      const int qq = is_v ? q - TL::LOADS : q;
      const int r = qq * TL::RPI + lane / TL::NCH;  // tile row (key slot in chunk)
      const int gp = piece ^ (is_v ? swz_v<D>(r) : swz_k<D>(r));
      const char* src = (is_v ? vb : kb) + (base + rows[k]) * TL::ROW_BYTES + gp * 16;
      const uint32_t dst =  // M0: LDS base of this wave-wide 1 KB load
          uint32_t(reinterpret_cast<uintptr_t>(buf)) + (is_v ? TL::TILE_BYTES : 0) + qq * 1024;
      asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(dst) : "memory");
    }
  }
}

// Loader-wave variant: one extra wave issues all 2*LOADS loads of a chunk, so
// the compute waves never wait on load issue or address arithmetic. The chunk
// base is uniform (an SGPR pair); each lane adds its 32-bit row/piece offset.
// RASTER: the base is the head's first raster row (plus the block origin for
// full blocks) and the offset carries the slot's raster token (the head's rows
// span < 2^31 bytes, checked on the host); a lane's K and V rows are the same,
// so each offset is computed once.
template <int D>
__device__ __forceinline__ void loader_issue(const char* kb, const char* vb, int64_t base_row,
                                             const uint32_t (&row_off)[Tile<D>::LOADS],
                                             uint32_t lds_buf, int lane);

template <int D, bool RASTER>
__device__ __forceinline__ void loader_chunk(const DevGeom& g, const char* kb, const char* vb,
                                             int64_t head_row, const Cursor& c, const lds_int* rel,
                                             uint32_t lds_buf, int lane) {
  using TL = Tile<D>;
  const int last = c.nj - 1 - c.c0;  // last real key slot of the chunk
  uint32_t row_off[TL::LOADS];       // byte offset of this lane's row in load qq
  int64_t base_row;
  auto fill = [&](auto row_of) {
#pragma unroll
    for (int qq = 0; qq < TL::LOADS; ++qq)
      row_off[qq] = uint32_t(row_of(min(qq * TL::RPI + lane / TL::NCH, last)) * TL::ROW_BYTES);
  };
  if (!RASTER) {
    base_row = head_row + int64_t(c.j) * g.BS + c.c0;
    fill([](int sr) { return sr; });
  } else {
    const RasterRows rr = raster_rows(g, c, head_row);
    base_row = rr.base;
    if (rr.full)
      fill([&](int sr) { return rel[c.c0 + sr]; });
    else
      fill([&](int sr) { return int(ext_token(g, c.e, c.c0 + sr)); });
  }
  loader_issue<D>(kb, vb, base_row, row_off, lds_buf, lane);
}

// The 2*LOADS wave-wide DMA loads of one chunk: K and V rows at base_row + the lane's
// row offsets (bytes), into the chunk's LDS buffer.
template <int D>
__device__ __forceinline__ void loader_issue(const char* kb, const char* vb, int64_t base_row,
                                             const uint32_t (&row_off)[Tile<D>::LOADS],
                                             uint32_t lds_buf, int lane) {
  using TL = Tile<D>;
  const char* kbase = kb + base_row * TL::ROW_BYTES;
  const char* vbase = vb + base_row * TL::ROW_BYTES;
#pragma unroll
  for (int q = 0; q < 2 * TL::LOADS; ++q) {
    const bool is_v = q >= TL::LOADS;
    const int qq = is_v ? q - TL::LOADS : q;
    const int r = qq * TL::RPI + lane / TL::NCH;  // tile row (key slot in chunk)
    const int gp = (lane % TL::NCH) ^ (is_v ? swz_v<D>(r) : swz_k<D>(r));
    const uint32_t off = row_off[qq] + uint32_t(gp * 16);
    const uint32_t dst = lds_buf + (is_v ? TL::TILE_BYTES : 0) + qq * 1024;  // M0
    asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(is_v ? vbase : kbase),
                 "{m0}"(dst)
                 : "memory");
  }
}

// W compute waves (32 query slots each), plus one loader wave when LD. The
// workgroup shapes are chosen so that a CU holds 12 waves at three waves per
// SIMD (<= 168 VGPRs): 4 compute waves without a loader (3 workgroups per CU),
// 5 compute waves with one (2 workgroups of 6).
// RASTER: q, k, v and o are raster [B,H,N,d] (and lse [B,H,N]); every row is
// addressed through the blocking's slot -> token map, so no blocked copies exist.
struct NoTable {};

// The work item of a workgroup: its geometry, (batch, head) pair, query block i
// (-1 for grid padding) and the source of its kept list.
// Workgroup w runs on XCD w % 8. Every XCD walks the heads in the same order
// and takes one contiguous eighth of each head's query blocks: the XCDs work
// on the same head at a time (its K/V stays in the MALL) and each XCD's L2
// serves spatially adjacent query blocks, whose kept K/V sets overlap.
// MULTI: the heads follow each other in the grid (per batch element), each
// padded to a multiple of 8 items, and are dealt to the XCDs the same way.
struct Item {
  DevGeom g;
  int64_t bh;
  int i;
  const int* cnt_src;
  const int* list_src;
};

// Row of rank r among the n query blocks c[0..n) of one XCD's share of a head, ordered
// by kept-block count (descending, ties to the lower index) within windows of 64. The
// XCD's CUs then start its rows heaviest first: rows of similar length walk the key
// blocks at a similar pace, so the K/V blocks they share meet in the XCD's L2, and long
// rows do not form the tail. Any order is correct: each row is one work item.
__device__ __forceinline__ int heavy_first(const int* __restrict__ c, int n, int r, int NB) {
  const int lane = int(threadIdx.x & 63);
  const int w0 = r & ~63, wn = min(64, n - w0);
  const int cl = min(max(c[w0 + min(lane, wn - 1)], 0), NB);  // lanes past the window re-read
  const int key = lane < wn ? cl : -1;
  int rank = 0;
  for (int t = 0; t < wn; ++t) {
    const int kt = __builtin_amdgcn_readlane(key, t);
    rank += (kt > key || (kt == key && t < lane)) ? 1 : 0;
  }
  const uint64_t hit = __ballot(lane < wn && rank == r - w0);
  return w0 + __builtin_amdgcn_readfirstlane(int(__builtin_ctzll(hit)));
}

template <bool MULTI, class Tab>
__device__ __forceinline__ Item work_item(const DevGeom& g_arg, const int* counts,
                                          const int* indices, const int* order, const Tab& tab) {
  Item it;
  it.g = g_arg;
  if constexpr (MULTI) {
    const int b = int(blockIdx.x) / tab.items_per_batch;
    const int w = int(blockIdx.x) - b * tab.items_per_batch;
    int k = 0, start;
    if (order) {
      // ranked: order holds per batch element the launch's heads by rank, then
      // their ascending first items; the item's rank is the number of first
      // items <= w, minus one (one load per lane and a ballot, n_heads <= 64)
      const int n = tab.n_heads;
      const int* ranked = order + int64_t(b) * 2 * n;
      const int ln = int(threadIdx.x & 63);
      const int first = ln < n ? ranked[n + ln] : INT_MAX;
      const int r = __popcll(__ballot(first <= w)) - 1;
      k = __builtin_amdgcn_readfirstlane(ranked[r]);
      start = __builtin_amdgcn_readfirstlane(ranked[n + r]);
    } else {
      while (k + 1 < tab.n_heads && tab.head[k + 1].start <= w) ++k;
      start = tab.head[k].start;
    }
    const MultiHead& mh = tab.head[k];
    it.g = tab.geo[mh.geom];
    const int local = w - start;  // same residue mod 8 as blockIdx.x
    const int per_xcd = (it.g.NB + 7) / 8;
    const int lo = (local & 7) * per_xcd, r = local >> 3;
    const int rows = min(per_xcd, it.g.NB - lo);
    if (r >= rows) {
      it.i = -1;
      return it;
    }
    const int* hc = mh.counts + int64_t(b) * mh.counts_bstride;
    it.i = lo + heavy_first(hc + lo, rows, r, it.g.NB);
    it.bh = int64_t(b) * it.g.H + mh.h;
    it.cnt_src = hc + it.i;
    it.list_src = mh.indices + int64_t(b) * mh.indices_bstride + int64_t(it.i) * it.g.NB;
  } else {
    const DevGeom& g = it.g;
    const int per_xcd = (g.NB + 7) / 8;
    const int64_t slot = int64_t(blockIdx.x) >> 3;
    it.bh = slot / per_xcd;
    if (order) it.bh = order[it.bh];  // heads in the ranked order (heaviest first)
    const int lo = int(blockIdx.x & 7) * per_xcd, r = int(slot % per_xcd);
    const int rows = min(per_xcd, g.NB - lo);
    if (r >= rows) {  // grid padding when NB is not a multiple of 8
      it.i = -1;
      return it;
    }
    it.i = lo + heavy_first(counts + it.bh * g.NB + lo, rows, r, g.NB);
    it.cnt_src = counts + it.bh * g.NB + it.i;
    it.list_src = indices + (it.bh * g.NB + it.i) * int64_t(g.NB);
  }
  return it;
}

// MULTI (raster only): one launch over heads with different blockings; the work
// item picks its head, and with it the geometry and block lists, from `tab`.
template <int D, int W, bool LD, bool RASTER, bool MULTI>
__global__ void __launch_bounds__(64 * (W + LD))
    __attribute__((amdgpu_waves_per_eu(W + LD >= 3 ? 3 : 2)))
    attn_kernel(DevGeom g_arg, const uint4* __restrict__ qb, const char* __restrict__ kb,
                const char* __restrict__ vb, const int* __restrict__ counts,
                const int* __restrict__ indices, float scale_log2, __bf16* __restrict__ ob,
                float* __restrict__ lse, const int* __restrict__ order,
                typename std::conditional<MULTI, MultiTable, NoTable>::type tab) {
  using TL = Tile<D>;
  __shared__ __align__(16) char lds_raw[2 * TL::BUF_BYTES];
  __shared__ int rel_raw[RASTER ? kMaxBS : 1];  // full-block slot -> raster token offset
  extern __shared__ int list_raw[];  // kept list of this work item, NB entries
  lds_char* const lds = (lds_char*)lds_raw;
  lds_int* const list = (lds_int*)list_raw;
  lds_int* const rel = (lds_int*)rel_raw;

  const Item it = work_item<MULTI>(g_arg, counts, indices, order, tab);
  if (it.i < 0) return;
  const DevGeom g = it.g;
  const int64_t bh = it.bh;
  const int i = it.i;
  const int* const cnt_src = it.cnt_src;
  const int* const list_src = it.list_src;
  const BlockExt e_i = block_ext(g, i);
  const int n_i = e_i.n;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: keep in an SGPR
  const bool loader = LD && wave == W;  // loader wave: q0 = 32 W >= BS, so no query rows
  const int q0 = wave * 32;
  const int half = lane >> 5;  // k-slot group of the MFMA operands
  const int r32 = lane & 31;
  const int64_t head_row = RASTER ? bh * g.N : bh * g.NB * int64_t(g.BS);
  // row of query slot qs < n_i of this item
  auto q_row = [&](int qs) -> int64_t {
    return RASTER ? head_row + ext_token(g, e_i, qs) : head_row + int64_t(i) * g.BS + qs;
  };

  // Q^T fragments (B operand): query row q0 + r32, d = 16*kk + 8*half .. +8
  bf16x8 qf[D / 16];
  {
    const int qs = q0 + r32;
    const uint4* src = qb + q_row(min(qs, n_i - 1)) * TL::NCH + half;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (qs < n_i) v = src[2 * kk];
      qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }

  const int cnt = min(max(*cnt_src, 0), g.NB);
  for (int e = threadIdx.x; e < cnt; e += 64 * (W + LD)) list[e] = list_src[e];
  if (RASTER) {
    for (int sl = threadIdx.x; sl < g.BS; sl += 64 * (W + LD)) {
      const int q = sl / g.bw;
      rel[sl] = ((q / g.bh) * g.Hs + q % g.bh) * g.Ws + sl % g.bw;
    }
  }
  __syncthreads();  // list and table visible to every wave (also completes the Q loads)

  // per-lane LDS byte offsets that do not depend on the chunk
  // K operand: tile row r32, global piece 2*kk + half
  const int k_off = r32 * TL::ROW_BYTES;
  const int k_sw = swz_k<D>(r32);
  // V^T operand via transposing reads: 16-lane group G, index s
  const int G = lane >> 4, s16 = lane & 15;
  const int v_row0 = 4 * (G >> 1) + (s16 >> 2);     // + 16u + 8h
  const int v_piece0 = 2 * (G & 1) + ((s16 & 3) >> 1);  // + 4t
  const int v_sub = (s16 & 1) * 8;

  f32x16 o[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
  float m = -INFINITY, l = 0.0f;
  const bool rows_live = q0 < n_i;
  const bf16x2 ones = {__bf16(1.0f), __bf16(1.0f)};

  const uint32_t lds_u32 = uint32_t(reinterpret_cast<uintptr_t>(lds));
  int rows[WaveLoads<D, W>::NQ];  // without a loader: this wave's rows of the next chunk
  // issue the loads of chunk c into buffer b (all of them from the loader wave,
  // or each wave its share at the rows prefetched into `rows`)
  auto issue = [&](const Cursor& c, int b) {
    if (LD) {
      if (loader)
        loader_chunk<D, RASTER>(g, kb, vb, head_row, c, rel, lds_u32 + b * TL::BUF_BYTES, lane);
    } else {
      load_chunk<D, W, RASTER>(g, kb, vb, head_row, c, rows, lds + b * TL::BUF_BYTES, wave, lane);
    }
  };
  auto prefetch = [&](const Cursor& c) {
    if (!LD) wave_rows<D, W, RASTER>(g, c, rel, wave, lane, rows);
  };
  Cursor cur = {-1, 0, 0, -kChunk, e_i};
  cur = next_chunk(g, list, cnt, cur);
  int buf = 0;
  if (cur.jj < cnt) {
    prefetch(cur);
    issue(cur, 0);
  }
  Cursor ahead = cur;  // without a loader: the chunk after the next, rows prefetched
  if (!LD) {
    ahead = next_chunk(g, list, cnt, cur);
    if (ahead.jj < cnt) prefetch(ahead);
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  while (cur.jj < cnt) {
    Cursor nxt;
    if (LD) {
      nxt = next_chunk(g, list, cnt, cur);
      if (nxt.jj < cnt) issue(nxt, buf ^ 1);
    } else {
      nxt = ahead;
      if (nxt.jj < cnt) {
        issue(nxt, buf ^ 1);
        ahead = next_chunk(g, list, cnt, nxt);
        if (ahead.jj < cnt) prefetch(ahead);
      }
    }
    if (rows_live) {
      lds_char* Kt = lds + buf * TL::BUF_BYTES;
      lds_char* Vt = Kt + TL::TILE_BYTES;
      f32x16 s;
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = 0.0f;
      {
        bf16x8 kf[D / 16];
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk)
          kf[kk] = *(lds_bf16x8*)(Kt + k_off + (((2 * kk + half) ^ k_sw) << 4));
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk)
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[kk], s, 0, 0, 0);
        // schedule: two K reads ahead of each pair of MFMAs
#pragma unroll
        for (int gi = 0; gi < D / 32; ++gi) {
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // LDS reads
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // MFMAs
        }
      }      // s[r]: key (r/4)*8 + 4*half + r%4 of the chunk, query row r32
      if (cur.c0 + kChunk > cur.nj) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kr = (r >> 2) * 8 + 4 * half + (r & 3);
          if (cur.c0 + kr >= cur.nj) s[r] = -INFINITY;
        }
      }
      float mx = s[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s[r]);
      {
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                         false, false);
        mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * scale_log2;
      }
      if (__any(mx > m + kRescaleLog2)) {
        const float mnew = fmaxf(m, mx);
        const float alpha = __builtin_amdgcn_exp2f(m - mnew);
        l *= alpha;
#pragma unroll
        for (int t = 0; t < D / 32; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[t][r] *= alpha;
        m = mnew;
      }
      bf16x8 p[2];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], scale_log2, -m));
        p[r >> 3][r & 7] = __bf16(e);
      }
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bf16x2 pr = {p[u][2 * e], p[u][2 * e + 1]};
          l = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, l, false);
        }
      {
        bf16x8 vf[D / 32][2];
#pragma unroll
        for (int t = 0; t < D / 32; ++t)
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            bf16x4 h2[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const int row = 16 * u + 8 * h + v_row0;
              const int piece = (4 * t + v_piece0) ^ swz_v<D>(row);
              h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                  (lds_bf16x4*)(Vt + row * TL::ROW_BYTES + piece * 16 + v_sub));
            }
            vf[t][u] = __builtin_shufflevector(h2[0], h2[1], 0, 1, 2, 3, 4, 5, 6, 7);
          }
#pragma unroll
        for (int t = 0; t < D / 32; ++t)
#pragma unroll
          for (int u = 0; u < 2; ++u)
            o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[t][u], p[u], o[t], 0, 0, 0);
        // schedule: the V^T reads of two output tiles ahead of their four MFMAs
#pragma unroll
        for (int gi = 0; gi < D / 64; ++gi) {
          __builtin_amdgcn_sched_group_barrier(0x100, 8, 1);  // LDS reads
          __builtin_amdgcn_sched_group_barrier(0x008, 4, 1);  // MFMAs
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    buf ^= 1;
    cur = nxt;
  }

  // normalise and store: lane holds query row q0 + r32, d = 32t + 8*rq + 4*half + 0..3
  {
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l), __float_as_uint(l),
                                                     false, false);
    l = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
  }
  const int qs = q0 + r32;
  // blocked output: every slot of the block (padding as zeros); raster: real rows only
  if (RASTER ? qs < n_i : qs < g.BS) {
    const bool real = qs < n_i;
    const float inv = (real && l > 0.0f) ? 1.0f / l : 0.0f;
    const int64_t orow = real ? q_row(qs) : head_row + int64_t(i) * g.BS + qs;
    __bf16* dst = ob + orow * D + 4 * half;
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
      lse[orow] = l > 0.0f ? (m + log2f(l)) * 0.69314718055994530942f : -INFINITY;
  }
}

// Paired kernel (blocks of 5 row tiles, i.e. 129..160 slots). The waves of a
// workgroup otherwise move through each chunk in step (LDS reads, S MFMAs,
// softmax VALU, P.V MFMAs, barrier), so a SIMD's matrix and vector units take
// turns instead of overlapping. Here each 32-row query tile has two compute
// waves, placed on the same SIMD (waves w and w + 4 of a workgroup share one):
// member A takes the even chunks of the kept walk, member B the odd ones, each
// with its own online-softmax state, and the pair merges by log-sum-exp at the
// end. A step has two halves separated by workgroup barriers:
//   half 0: A runs P.V(2s-2) and S(2s) (MFMA), B the softmax of 2s-1 (VALU) and
//           reads the V^T fragments of 2s-1 into registers;
//   half 1: B runs P.V(2s-1) and S(2s+1), A the softmax of 2s and its V^T reads;
// so on every SIMD one member's matrix work meets the other's vector work. Two
// loader waves (even / odd chunks) keep an 8-chunk LDS ring three chunks ahead;
// a slot is refilled in the half after its V^T was read.
// One workgroup (12 waves) fills a CU. With 4 row tiles the pairs would leave a
// CU at 8 compute waves instead of 12, which is slower, so smaller blocks keep
// the single-member kernel.
constexpr int kRing = 8;
constexpr int kPairTiles = 5;         // row tiles of the blocks the paired kernel takes
constexpr int kPairLds = 160 * 1024;  // LDS of one CU, all of it for one workgroup

template <int D>
struct PPLayout {
  static constexpr int RING_BYTES = kRing * Tile<D>::BUF_BYTES;
  static constexpr int REL_OFF = RING_BYTES;
  static constexpr int KVAL_OFF = RING_BYTES + kMaxBS * 4;  // real keys per ring slot
  static constexpr int LIST_OFF = KVAL_OFF + kRing * 4;
  static constexpr int LPC = 2 * Tile<D>::LOADS;  // loads per chunk (one loader wave)
  static constexpr int MERGE_FLOATS = D / 32 * 16 + 2;  // per lane: O, m, l
};

// (tile, phase) of compute wave w of 2T: full octets pair w with w + 4.
__device__ __forceinline__ void pp_role(int w, int T, int* tile, int* ph) {
  const int full = (2 * T) / 8 * 8;
  if (w < full) {
    *tile = (w / 8) * 4 + (w & 3);
    *ph = (w >> 2) & 1;
  } else {
    const int h = (2 * T - full) / 2, r = w - full;
    *tile = full / 2 + r % h;
    *ph = r >= h;
  }
}

// wait until at most n chunks' loads (n = 0, 1, 2) of this wave are in flight
template <int LPC>
__device__ __forceinline__ void wait_chunks(int n) {
  constexpr auto imm = [](int c) { return (c & 15) | (((c >> 4) & 3) << 14) | 0x70 | 0xF00; };
  if (n <= 0)
    __builtin_amdgcn_s_waitcnt(imm(0));
  else if (n == 1)
    __builtin_amdgcn_s_waitcnt(imm(LPC));
  else
    __builtin_amdgcn_s_waitcnt(imm(2 * LPC));
}

template <int D, int T, bool RASTER, bool MULTI>
__global__ void __launch_bounds__(64 * (2 * T + 2)) __attribute__((amdgpu_waves_per_eu(3)))
    attn_pp_kernel(DevGeom g_arg, const uint4* __restrict__ qb, const char* __restrict__ kb,
                   const char* __restrict__ vb, const int* __restrict__ counts,
                   const int* __restrict__ indices, float scale_log2, __bf16* __restrict__ ob,
                   float* __restrict__ lse, const int* __restrict__ order,
                   typename std::conditional<MULTI, MultiTable, NoTable>::type tab) {
  using TL = Tile<D>;
  using LY = PPLayout<D>;
  constexpr int NT = 64 * (2 * T + 2);
  extern __shared__ __align__(16) char smem_raw[];
  lds_char* const lds = (lds_char*)smem_raw;
  lds_int* const rel = (lds_int*)(smem_raw + LY::REL_OFF);
  lds_int* const list = (lds_int*)(smem_raw + LY::LIST_OFF);
  lds_int* const kval = (lds_int*)(smem_raw + LY::KVAL_OFF);

  const Item it = work_item<MULTI>(g_arg, counts, indices, order, tab);
  if (it.i < 0) return;
  const DevGeom g = it.g;
  const int64_t bh = it.bh;
  const int i = it.i;
  const BlockExt e_i = block_ext(g, i);
  const int n_i = e_i.n;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool loader = wave >= 2 * T;
  const int lp = wave - 2 * T;  // loader parity: 0 even chunks, 1 odd
  int tile = T, ph = 0;          // loaders own no rows (32 T >= BS)
  if (!loader) pp_role(wave, T, &tile, &ph);
  tile = __builtin_amdgcn_readfirstlane(tile);
  ph = __builtin_amdgcn_readfirstlane(ph);
  const int q0 = tile * 32;
  const int half = lane >> 5, r32 = lane & 31;
  const int64_t head_row = RASTER ? bh * g.N : bh * g.NB * int64_t(g.BS);
  auto q_row = [&](int qs) -> int64_t {
    return RASTER ? head_row + ext_token(g, e_i, qs) : head_row + int64_t(i) * g.BS + qs;
  };

  bf16x8 qf[D / 16];
  {
    const int qs = q0 + r32;
    const uint4* src = qb + q_row(min(qs, n_i - 1)) * TL::NCH + half;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (qs < n_i) v = src[2 * kk];
      qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }
  const int cnt = min(max(*it.cnt_src, 0), g.NB);
  for (int e = tid; e < cnt; e += NT) list[e] = it.list_src[e];
  if (RASTER) {
    for (int sl = tid; sl < g.BS; sl += NT) {
      const int q = sl / g.bw;
      rel[sl] = ((q / g.bh) * g.Hs + q % g.bh) * g.Ws + sl % g.bw;
    }
  }
  __syncthreads();

  // chunks of the kept walk (every wave computes the same count)
  int nch = 0;
  for (int e = lane; e < cnt; e += 64) {
    const int j = list[e];
    if (j >= 0 && j < g.NB) nch += (block_ext(g, j).n + kChunk - 1) / kChunk;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) nch += __shfl_xor(nch, off);
  nch = __builtin_amdgcn_readfirstlane(nch);

  const int v_row0 = 4 * ((lane >> 4) >> 1) + ((lane & 15) >> 2);
  const int v_piece0 = 2 * ((lane >> 4) & 1) + (((lane & 15) & 3) >> 1);
  const int v_sub = (lane & 1) * 8;
  const int k_off = r32 * TL::ROW_BYTES;
  const int k_sw = swz_k<D>(r32);

  f32x16 o[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
  float m = -INFINITY, l = 0.0f;
  const bool rows_live = !loader && q0 < n_i;
  const bf16x2 ones = {__bf16(1.0f), __bf16(1.0f)};
  const uint32_t lds_u32 = uint32_t(reinterpret_cast<uintptr_t>(lds));
  auto kbuf = [&](int k) { return lds + (k & (kRing - 1)) * TL::BUF_BYTES; };

  auto compute_s = [&](int k) {
    lds_char* Kt = kbuf(k);
    f32x16 sv;
#pragma unroll
    for (int r = 0; r < 16; ++r) sv[r] = 0.0f;
    bf16x8 kf[D / 16];
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
      kf[kk] = *(lds_bf16x8*)(Kt + k_off + (((2 * kk + half) ^ k_sw) << 4));
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
      sv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[kk], sv, 0, 0, 0);
#pragma unroll
    for (int gi = 0; gi < D / 32; ++gi) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    }
    return sv;
  };
  bf16x8 p[2];
  auto softmax = [&](f32x16 sv, int c0, int nj) {
    if (c0 + kChunk > nj) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kr = (r >> 2) * 8 + 4 * half + (r & 3);
        if (c0 + kr >= nj) sv[r] = -INFINITY;
      }
    }
    float mx = sv[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, sv[r]);
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                       false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * scale_log2;
    }
    if (__any(mx > m + kRescaleLog2)) {
      const float mnew = fmaxf(m, mx);
      const float alpha = __builtin_amdgcn_exp2f(m - mnew);
      l *= alpha;
#pragma unroll
      for (int t = 0; t < D / 32; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][r] *= alpha;
      m = mnew;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[r], scale_log2, -m));
      p[r >> 3][r & 7] = __bf16(e);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bf16x2 pr = {p[u][2 * e], p[u][2 * e + 1]};
        l = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, l, false);
      }
  };
  // V^T fragments of a chunk are read at the end of the vector phase that made its P
  // (S is dead by then), so the matrix phase starts on MFMAs instead of an LDS round
  // trip; they stay in registers across the barrier.
  bf16x8 vf[D / 32][2];
  auto read_v = [&](int k) {
    __builtin_amdgcn_sched_barrier(0);
    lds_char* Vt = kbuf(k) + TL::TILE_BYTES;
#pragma unroll
    for (int t = 0; t < D / 32; ++t)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        bf16x4 h2[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int row = 16 * u + 8 * h + v_row0;
          const int piece = (4 * t + v_piece0) ^ swz_v<D>(row);
          h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
              (lds_bf16x4*)(Vt + row * TL::ROW_BYTES + piece * 16 + v_sub));
        }
        vf[t][u] = __builtin_shufflevector(h2[0], h2[1], 0, 1, 2, 3, 4, 5, 6, 7);
      }
  };
  auto pv = [&]() {
#pragma unroll
    for (int t = 0; t < D / 32; ++t)
#pragma unroll
      for (int u = 0; u < 2; ++u)
        o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[t][u], p[u], o[t], 0, 0, 0);
  };

  // Loaders keep a cursor on chunk 2s + par of step s, three chunks ahead (the next
  // one they issue), and record each chunk's real keys beside its ring slot, so the
  // compute waves mask without walking the kept list themselves.
  const int par = loader ? lp : ph;
  auto next2 = [&](Cursor c) { return next_chunk(g, list, cnt, next_chunk(g, list, cnt, c)); };
  Cursor cur{};
  if (loader) {
    cur = next_chunk(g, list, cnt, {-1, 0, 0, -kChunk, e_i});
    if (par == 1) cur = next_chunk(g, list, cnt, cur);
  }
  auto record = [&](int k) {
    if (lane == 0) kval[k & (kRing - 1)] = min(cur.nj - cur.c0, kChunk);
  };
  auto issue = [&](int k) {
    record(k);
    loader_chunk<D, RASTER>(g, kb, vb, head_row, cur, rel,
                            lds_u32 + (k & (kRing - 1)) * TL::BUF_BYTES, lane);
  };
  if (loader) {
#pragma unroll 1
    for (int r = 0; r < 3; ++r) {
      if (par + 2 * r < nch) issue(par + 2 * r);
      cur = next2(cur);
    }
    if (par == 0) wait_chunks<LY::LPC>((2 < nch) + (4 < nch));
  }
  const f32x16 zero16 = {};
  const bf16x8 zero8 = {};
  const int sc0 = 0;  // the held S covers keys 0 .. snj - 1 of its chunk
  int snj = 0;
  f32x16 sv = zero16;
  const int steps = nch > 0 ? (nch + 1) / 2 + 1 : 0;
  // Each role runs its own loop (so S and P are never live across each other's
  // phases); all three execute the same two barriers per step. In the matrix
  // phase P.V of the previous own chunk (its V^T already in registers) runs before
  // S of this one.
  __syncthreads();
  if (loader) {
    // Raster layout: the row offsets of a full block's chunk depend only on the
    // chunk's position in the block (T positions), so they are read from the slot
    // table once here; the loop then issues full-block chunks without LDS reads,
    // which would queue behind the compute waves' K and V^T reads.
    uint32_t pre[RASTER ? T : 1][TL::LOADS];
    if (RASTER) {
#pragma unroll
      for (int ps = 0; ps < T; ++ps)
#pragma unroll
        for (int qq = 0; qq < TL::LOADS; ++qq) {
          const int sr = min(qq * TL::RPI + lane / TL::NCH, max(g.BS - 1 - ps * kChunk, 0));
          pre[ps][qq] = uint32_t(rel[min(ps * kChunk + sr, g.BS - 1)] * TL::ROW_BYTES);
        }
    }
    auto issue_loop = [&](int k) {
      record(k);
      const uint32_t buf = lds_u32 + (k & (kRing - 1)) * TL::BUF_BYTES;
      if (RASTER && cur.e.n == g.BS) {
        uint32_t ro[TL::LOADS];
        const int ps = cur.c0 / kChunk;
#pragma unroll
        for (int pp = 0; pp < T; ++pp)
          if (pp == ps)
#pragma unroll
            for (int qq = 0; qq < TL::LOADS; ++qq) ro[qq] = pre[RASTER ? pp : 0][qq];
        loader_issue<D>(kb, vb, head_row + block_origin(g, cur.e), ro, buf, lane);
      } else {
        loader_chunk<D, RASTER>(g, kb, vb, head_row, cur, rel, buf, lane);
      }
    };
#pragma unroll 1
    for (int st = 0; st < steps; ++st) {
      const int k = 2 * st + par;
      // half 0: loader 0 refills the slot of chunk 2s - 2 (its V^T was read in the
      // previous half 1); loader 1 makes sure chunk 2s + 1 (read in half 1) has landed
      if (par == 0 && k + 6 < nch) issue_loop(k + 6);
      if (par == 1 && k < nch) wait_chunks<LY::LPC>((k + 2 < nch) + (k + 4 < nch));
      __syncthreads();
      // half 1: loader 1 refills the slot of chunk 2s - 1 (V^T read in half 0); loader 0
      // makes sure chunk 2s + 2 (read in the next half 0) has landed
      if (par == 1 && k + 6 < nch) issue_loop(k + 6);
      if (par == 0 && k + 2 < nch) wait_chunks<LY::LPC>((k + 4 < nch) + (k + 6 < nch));
      __syncthreads();
      cur = next2(cur);
    }
  } else if (par == 0) {
#pragma unroll 1
    for (int st = 0; st < steps; ++st) {
      const int k = 2 * st;
      // half 0: matrix phase
      if (rows_live && k >= 2 && k - 2 < nch) pv();
      if (rows_live && k < nch) {
        sv = compute_s(k);
        snj = kval[k & (kRing - 1)];
      } else {
        sv = zero16;
      }
      __syncthreads();
      // half 1: vector phase
      if (rows_live && k < nch) {
        softmax(sv, sc0, snj);
        read_v(k);
      } else {
        p[0] = zero8;
        p[1] = zero8;
#pragma unroll
        for (int t = 0; t < D / 32; ++t) vf[t][0] = vf[t][1] = zero8;
      }
      __syncthreads();
    }
  } else {
#pragma unroll 1
    for (int st = 0; st < steps; ++st) {
      const int k = 2 * st + 1;
      // half 0: vector phase (the S computed in the previous step's half 1)
      if (rows_live && k >= 2 && k - 2 < nch) {
        softmax(sv, sc0, snj);
        read_v(k - 2);
      } else {
        p[0] = zero8;
        p[1] = zero8;
#pragma unroll
        for (int t = 0; t < D / 32; ++t) vf[t][0] = vf[t][1] = zero8;
      }
      __syncthreads();
      // half 1: matrix phase
      if (rows_live && k >= 2 && k - 2 < nch) pv();
      if (rows_live && k < nch) {
        sv = compute_s(k);
        snj = kval[k & (kRing - 1)];
      } else {
        sv = zero16;
      }
      __syncthreads();
    }
  }

  // merge: member B hands (O, m, l) to member A of its tile through LDS
  float* mg = reinterpret_cast<float*>(smem_raw) + tile * (LY::MERGE_FLOATS * 64);
  if (rows_live && ph == 1) {
#pragma unroll
    for (int t = 0; t < D / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) mg[(t * 16 + r) * 64 + lane] = o[t][r];
    mg[(D / 32 * 16) * 64 + lane] = m;
    mg[(D / 32 * 16 + 1) * 64 + lane] = l;
  }
  __syncthreads();
  if (loader || ph == 1) return;
  if (rows_live) {
    const float mB = mg[(D / 32 * 16) * 64 + lane];
    const float lB = mg[(D / 32 * 16 + 1) * 64 + lane];
    const float mm = fmaxf(m, mB);
    const bool none = mm == -INFINITY;
    const float aA = none ? 0.0f : __builtin_amdgcn_exp2f(m - mm);
    const float aB = none ? 0.0f : __builtin_amdgcn_exp2f(mB - mm);
#pragma unroll
    for (int t = 0; t < D / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] = o[t][r] * aA + mg[(t * 16 + r) * 64 + lane] * aB;
    l = l * aA + lB * aB;
    m = mm;
  }
  {
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l), __float_as_uint(l),
                                                     false, false);
    l = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
  }
  const int qs = q0 + r32;
  if (RASTER ? qs < n_i : qs < g.BS) {
    const bool real = qs < n_i;
    const float inv = (real && l > 0.0f) ? 1.0f / l : 0.0f;
    const int64_t orow = real ? q_row(qs) : head_row + int64_t(i) * g.BS + qs;
    __bf16* dst = ob + orow * D + 4 * half;
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
      lse[orow] = l > 0.0f ? (m + log2f(l)) * 0.69314718055994530942f : -INFINITY;
  }
}

template <int D, int T, bool RASTER, bool MULTI>
hipError_t launch_pp(const DevGeom& g, const void* qb, const void* kb, const void* vb,
                     const int* counts, const int* indices, float scale_log2, void* ob,
                     float* lse, hipStream_t s, const MultiTable* tab, const int* order,
                     int nb_max) {
  {  // the ring and the kept list exceed the 64 KB default
    const hipError_t e = ensure_dynamic_lds(
        reinterpret_cast<const void*>(&attn_pp_kernel<D, T, RASTER, MULTI>), kPairLds);
    if (e != hipSuccess) return e;
  }
  const size_t lds = size_t(PPLayout<D>::LIST_OFF) + size_t(nb_max) * sizeof(int);
  const uint4* q4 = static_cast<const uint4*>(qb);
  const char* k1 = static_cast<const char*>(kb);
  const char* v1 = static_cast<const char*>(vb);
  __bf16* o2 = static_cast<__bf16*>(ob);
  if constexpr (MULTI) {
    const int64_t items = int64_t(g.B) * tab->items_per_batch;
    attn_pp_kernel<D, T, RASTER, MULTI><<<dim3(unsigned(items)), 64 * (2 * T + 2), lds, s>>>(
        g, q4, k1, v1, nullptr, nullptr, scale_log2, o2, lse, order, *tab);
  } else {
    const int64_t items = int64_t(g.B) * g.H * ((g.NB + 7) / 8) * 8;  // see the XCD mapping
    attn_pp_kernel<D, T, RASTER, MULTI><<<dim3(unsigned(items)), 64 * (2 * T + 2), lds, s>>>(
        g, q4, k1, v1, counts, indices, scale_log2, o2, lse, order, NoTable{});
  }
  return hipGetLastError();
}

// Software-pipelined kernel (blocks of 5 row tiles, i.e. 129..160 slots, d = 128).
// Eight waves, two per SIMD (waves w and w + 4 share one):
// - wave X_s (s = 0..3) owns query tile s for the whole kept walk. Its chunk loop
//   is pipelined by one chunk: while the softmax of chunk c runs on the vector
//   unit, the matrix unit takes P.V of chunk c-1 and S of chunk c+1 (independent
//   of that softmax), and the K fragments of c+1 and the V^T fragments of c are
//   read from LDS in between. One wave issues its own MFMAs and vector work
//   interleaved; no barrier pairs it with another wave.
// - wave Y_s issues the DMA of every fourth chunk (s, s + 4, ...) and computes
//   tile 4 on those same chunks with its own online-softmax state; the four
//   partial states of tile 4 merge by log-sum-exp at the end in a fixed order. So
//   every SIMD carries 1.25 tiles of work.
// The waves meet at one barrier per window of four chunks. A 9-slot LDS ring
// holds the window being computed, the chunk before it and the next window in
// flight: chunk c lives in slot c % 9; Y_s issues window v + 1 right after the
// barrier that opens window v and waits for it before the next barrier. X's
// iteration c reads K of c + 1 and V^T of c, so the barrier that makes window v
// visible sits before X's iteration 4v - 1.
constexpr int kSwRing = 9;
constexpr int kSwWaves = 8;
constexpr int kSwTiles = 5;
constexpr int kSwLds = 160 * 1024;

template <int D>
struct SwLayout {
  static constexpr int RING_BYTES = kSwRing * Tile<D>::BUF_BYTES;
  static constexpr int REL_OFF = RING_BYTES;
  static constexpr int KVAL_OFF = REL_OFF + kMaxBS * 4;  // real keys per ring slot
  static constexpr int LIST_OFF = KVAL_OFF + 64;
  static constexpr int LPC = 2 * Tile<D>::LOADS;          // DMA loads per chunk
  static constexpr int MERGE_FLOATS = D / 32 * 16 + 2;    // per lane: O, m, l
};

template <int D, int T, bool RASTER, bool MULTI>
__global__ void __launch_bounds__(64 * kSwWaves) __attribute__((amdgpu_waves_per_eu(2)))
    attn_sw_kernel(DevGeom g_arg, const uint4* __restrict__ qb, const char* __restrict__ kb,
                   const char* __restrict__ vb, const int* __restrict__ counts,
                   const int* __restrict__ indices, float scale_log2, __bf16* __restrict__ ob,
                   float* __restrict__ lse, const int* __restrict__ order,
                   typename std::conditional<MULTI, MultiTable, NoTable>::type tab) {
  static_assert(T == kSwTiles, "blocks of 5 row tiles");
  using TL = Tile<D>;
  using LY = SwLayout<D>;
  constexpr int NT = 64 * kSwWaves;
  extern __shared__ __align__(16) char smem_raw[];
  lds_char* const lds = (lds_char*)smem_raw;
  lds_int* const rel = (lds_int*)(smem_raw + LY::REL_OFF);
  lds_int* const list = (lds_int*)(smem_raw + LY::LIST_OFF);
  lds_int* const kval = (lds_int*)(smem_raw + LY::KVAL_OFF);

  const Item it = work_item<MULTI>(g_arg, counts, indices, order, tab);
  if (it.i < 0) return;
  const DevGeom g = it.g;
  const int64_t bh = it.bh;
  const int i = it.i;
  const BlockExt e_i = block_ext(g, i);
  const int n_i = e_i.n;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool is_y = wave >= 4;
  const int sidx = wave & 3;          // X: tile; Y: chunk residue mod 4
  const int tile = is_y ? 4 : sidx;   // Y waves share tile 4
  const int q0 = tile * 32;
  const bool rows_live = tile < T && q0 < n_i;
  const int half = lane >> 5, r32 = lane & 31;
  const int64_t head_row = RASTER ? bh * g.N : bh * g.NB * int64_t(g.BS);
  auto q_row = [&](int qs) -> int64_t {
    return RASTER ? head_row + ext_token(g, e_i, qs) : head_row + int64_t(i) * g.BS + qs;
  };

  bf16x8 qf[D / 16];
  {
    const int qs = q0 + r32;
    const uint4* src = qb + q_row(min(qs, n_i - 1)) * TL::NCH + half;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (rows_live && qs < n_i) v = src[2 * kk];
      qf[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }
  const int cnt = min(max(*it.cnt_src, 0), g.NB);
  for (int e = tid; e < cnt; e += NT) list[e] = it.list_src[e];
  if (RASTER) {
    for (int sl = tid; sl < g.BS; sl += NT) {
      const int q = sl / g.bw;
      rel[sl] = ((q / g.bh) * g.Hs + q % g.bh) * g.Ws + sl % g.bw;
    }
  }
  __syncthreads();

  // chunks of the kept walk (every wave computes the same count)
  int nch = 0;
  for (int e = lane; e < cnt; e += 64) {
    const int j = list[e];
    if (j >= 0 && j < g.NB) nch += (block_ext(g, j).n + kChunk - 1) / kChunk;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) nch += __shfl_xor(nch, off);
  nch = __builtin_amdgcn_readfirstlane(nch);
  const int nbar = nch / 4 + 1;  // barriers of the chunk walk, the same for every wave

  const int v_row0 = 4 * ((lane >> 4) >> 1) + ((lane & 15) >> 2);
  const int v_piece0 = 2 * ((lane >> 4) & 1) + (((lane & 15) & 3) >> 1);
  const int v_sub = (lane & 1) * 8;
  const int k_off = r32 * TL::ROW_BYTES;
  const int k_sw = swz_k<D>(r32);

  f32x16 o[D / 32];
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;
  float m = -INFINITY, l = 0.0f;
  const bf16x2 ones = {__bf16(1.0f), __bf16(1.0f)};
  const uint32_t lds_u32 = uint32_t(reinterpret_cast<uintptr_t>(lds));
  auto slot = [](int c) { return c % kSwRing; };
  // the slot's base as an opaque uniform value: the compiler then adds it once per
  // distinct lane offset instead of folding the modulo into every read address
  auto kbuf = [&](int c) {
    return lds + __builtin_amdgcn_readfirstlane(slot(c) * TL::BUF_BYTES);
  };

  // per-lane LDS byte offsets of the fragment reads inside a ring slot, so each read
  // costs one add of the slot base: K fragment kk (row r32, piece 2 kk + half), and
  // the V^T fragments of output tile t (rows 16 u + 8 h + v_row0 share row & 3, so
  // their swizzle, and the (u, h) part goes into the instruction's offset field)
  int kofs[D / 16], vofs[D / 32];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) kofs[kk] = k_off + (((2 * kk + half) ^ k_sw) << 4);
#pragma unroll
  for (int t = 0; t < D / 32; ++t)
    vofs[t] = TL::TILE_BYTES + v_row0 * TL::ROW_BYTES +
              ((4 * t + v_piece0) ^ swz_v<D>(v_row0)) * 16 + v_sub;
  auto read_k = [&](int c, bf16x8 (&kf)[D / 16]) {
    lds_char* Kt = kbuf(c);
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) kf[kk] = *(lds_bf16x8*)(Kt + kofs[kk]);
  };
  auto read_v = [&](int c, bf16x8 (&vf)[D / 32][2]) {
    lds_char* Vb = kbuf(c);
#pragma unroll
    for (int t = 0; t < D / 32; ++t) {
      lds_char* Vt = Vb + vofs[t];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        bf16x4 h2[2];
#pragma unroll
        for (int h = 0; h < 2; ++h)
          h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
              (lds_bf16x4*)(Vt + (16 * u + 8 * h) * TL::ROW_BYTES));
        vf[t][u] = __builtin_shufflevector(h2[0], h2[1], 0, 1, 2, 3, 4, 5, 6, 7);
      }
    }
  };
  // keys past the chunk's real ones get -inf (key of s[r]: (r/4)*8 + 4*half + r%4)
  auto mask = [&](f32x16& sv, int kv) {
    if (kv < kChunk) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kr = (r >> 2) * 8 + 4 * half + (r & 3);
        if (kr >= kv) sv[r] = -INFINITY;
      }
    }
  };
  // online softmax of one chunk: P (bf16) and the new running max; returns the
  // factor that O must be scaled by (1 unless the max grew by more than 2^8)
  auto softmax = [&](const f32x16& sv, bf16x8 (&p)[2], bool* rescale) {
    float mx = sv[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, sv[r]);
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                       false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * scale_log2;
    }
    const bool rs = __any(mx > m + kRescaleLog2);
    const float mnew = rs ? fmaxf(m, mx) : m;
    const float alpha = __builtin_amdgcn_exp2f(m - mnew);
    m = mnew;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[r], scale_log2, -m));
      p[r >> 3][r & 7] = __bf16(e);
    }
    float ls = l * alpha;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bf16x2 pr = {p[u][2 * e], p[u][2 * e + 1]};
        ls = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, ls, false);
      }
    l = ls;
    *rescale = rs;
    return alpha;
  };
  auto scale_o = [&](float alpha) {
#pragma unroll
    for (int t = 0; t < D / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] *= alpha;
  };
  auto pv = [&](const bf16x8 (&vf)[D / 32][2], const bf16x8 (&p)[2]) {
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int t = 0; t < D / 32; ++t)
        o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[t][u], p[u], o[t], 0, 0, 0);
  };
  auto s_of = [&](const bf16x8 (&kf)[D / 16]) {
    f32x16 sv = {};
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
      sv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[kk], sv, 0, 0, 0);
    return sv;
  };

  if (!is_y) {
    // ---- X: tile `tile`, every chunk, pipelined by one chunk ----
    // One pipeline step for chunk c. In: S of c (svi), P and V^T of c - 1 (pi, vfi),
    // and the rescale that the softmax of c - 1 asked for. Out: S of c + 1 (svo), P
    // and V^T of c (po, vfo); the compiler folds most of the hand-over into the
    // register allocation (a loop unrolled by two with the sets swapped spilled).
    bool rs = false;
    float alpha = 1.0f;
    // kv: real keys of chunk c, read one step ahead and moved to a scalar register
    // beside the K fragments' wait, so the mask test at the top of a step waits on no
    // LDS read (a wait there would also drain the V^T reads just issued)
    int kv = 0;
    auto step = [&](int c, f32x16& svi, f32x16& svo, bf16x8 (&pi)[2], bf16x8 (&po)[2],
                    bf16x8 (&vfi)[D / 32][2], bf16x8 (&vfo)[D / 32][2]) {
      if ((c & 3) == 3) __syncthreads();  // window (c + 1) / 4 landed
      const int kv_next = kval[slot(c + 1)];
      if (rs) scale_o(alpha);  // O holds P.V up to c - 2; P of c - 1 used the new max
      mask(svi, kv);
      // part 1: the K fragments of c + 1 (past the walk's end the slot's stale
      // contents: that S is discarded); P.V of c - 1 on the matrix unit; on the
      // vector unit the row sum of P of c - 1, the row max of c and the first half of
      // its exponentials
      lds_char* Kt = kbuf(c + 1);
      bf16x8 kf[D / 16];
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) kf[kk] = *(lds_bf16x8*)(Kt + kofs[kk]);
      pv(vfi, pi);
      {
        float ls = l * alpha;
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bf16x2 pr = {pi[u][2 * e], pi[u][2 * e + 1]};
            ls = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, ls, false);
          }
        l = ls;
      }
      {
        float mx = svi[0];
#pragma unroll
        for (int r = 1; r < 16; ++r) mx = fmaxf(mx, svi[r]);
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx),
                                                         __float_as_uint(mx), false, false);
        mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * scale_log2;
        rs = __any(mx > m + kRescaleLog2);
        const float mnew = rs ? fmaxf(m, mx) : m;
        alpha = __builtin_amdgcn_exp2f(m - mnew);
        m = mnew;
      }
#pragma unroll
      for (int r = 0; r < 8; ++r)
        po[0][r] = __bf16(__builtin_amdgcn_exp2f(__builtin_fmaf(svi[r], scale_log2, -m)));
      // part 2: S of c + 1 (two accumulators: two short MFMA chains), the V^T
      // fragments of c and the second half of the exponentials
      read_v(c, vfo);
      f32x16 s0 = {}, s1 = {};
#pragma unroll
      for (int kk = 0; kk < D / 16; kk += 2) {
        s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[kk], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk + 1], qf[kk + 1], s1, 0, 0, 0);
      }
      kv = __builtin_amdgcn_readfirstlane(kv_next);
#pragma unroll
      for (int r = 8; r < 16; ++r)
        po[1][r - 8] = __bf16(__builtin_amdgcn_exp2f(__builtin_fmaf(svi[r], scale_log2, -m)));
#pragma unroll
      for (int r = 0; r < 16; ++r) svo[r] = s0[r] + s1[r];
    };
    __syncthreads();  // window 0 landed
    f32x16 svA = {}, svB = {};
    bf16x8 pA[2] = {}, pB[2] = {};              // P of the previous chunk (zero before 0)
    bf16x8 vfA[D / 32][2] = {}, vfB[D / 32][2] = {};  // V^T of the previous chunk
    if (rows_live && nch > 0) {
      bf16x8 kf[D / 16];
      read_k(0, kf);
      svA = s_of(kf);
      kv = __builtin_amdgcn_readfirstlane(kval[slot(0)]);
    }
    // the last chunk's P.V (after the rescale its softmax asked for)
    auto finish = [&](bf16x8 (&vfx)[D / 32][2], bf16x8 (&px)[2]) {
      if (rs) scale_o(alpha);
      pv(vfx, px);
      float ls = l * alpha;
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bf16x2 pr = {px[u][2 * e], px[u][2 * e + 1]};
          ls = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, ls, false);
        }
      l = ls;
    };
    if (rows_live) {
#pragma unroll 1
      for (int c = 0; c < nch; ++c) {
        step(c, svA, svB, pA, pB, vfA, vfB);
        svA = svB;
        pA[0] = pB[0];
        pA[1] = pB[1];
#pragma unroll
        for (int t = 0; t < D / 32; ++t) {
          vfA[t][0] = vfB[t][0];
          vfA[t][1] = vfB[t][1];
        }
      }
      if (nch > 0) finish(vfA, pA);
    } else {  // no query rows here: only the barriers of the walk
#pragma unroll 1
      for (int c = 3; c < nch; c += 4) __syncthreads();
    }
  } else {
    // ---- Y: DMA of chunks sidx, sidx + 4, ...; tile 4 on the same chunks ----
    Cursor cur = next_chunk(g, list, nch > 0 ? cnt : 0, {-1, 0, 0, -kChunk, e_i});
    auto advance4 = [&]() {
#pragma unroll 1
      for (int a = 0; a < 4; ++a) cur = next_chunk(g, list, cnt, cur);
    };
#pragma unroll 1
    for (int a = 0; a < sidx; ++a) cur = next_chunk(g, list, cnt, cur);
    int c_issue = sidx;  // next chunk this wave issues
    auto issue = [&]() {
      if (c_issue < nch) {
        if (lane == 0) kval[slot(c_issue)] = min(cur.nj - cur.c0, kChunk);
        loader_chunk<D, RASTER>(g, kb, vb, head_row, cur, rel,
                                lds_u32 + slot(c_issue) * TL::BUF_BYTES, lane);
        advance4();
      }
      c_issue += 4;
    };
    auto tile4 = [&](int c) {
      if (rows_live && c < nch) {
        bf16x8 kf[D / 16];
        read_k(c, kf);
        f32x16 sv = s_of(kf);
        mask(sv, kval[slot(c)]);
        bool rs;
        bf16x8 pc[2];
        const float alpha = softmax(sv, pc, &rs);
        if (rs) scale_o(alpha);
        bf16x8 vf[D / 32][2];
        read_v(c, vf);
        pv(vf, pc);
      }
    };
    issue();  // window 0
    issue();  // window 1
    wait_chunks<LY::LPC>(sidx + 4 < nch ? 1 : 0);
    __syncthreads();  // window 0 landed
#pragma unroll 1
    for (int w = 0; w + 1 < nbar; ++w) {
      tile4(4 * w + sidx);
      wait_chunks<LY::LPC>(0);
      __syncthreads();  // window w + 1 landed
      issue();          // window w + 2, into the slots of chunks 4w - 1 .. 4w + 2
    }
    tile4(4 * (nbar - 1) + sidx);
  }

  // tile 4: the Y waves' partial states merge in LDS (the ring is free once every
  // wave is past its walk)
  float* mg = reinterpret_cast<float*>(smem_raw);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (is_y && sidx > 0 && rows_live) {
    float* dst = mg + (sidx - 1) * (LY::MERGE_FLOATS * 64);
#pragma unroll
    for (int t = 0; t < D / 32; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) dst[(t * 16 + r) * 64 + lane] = o[t][r];
    dst[(D / 32 * 16) * 64 + lane] = m;
    dst[(D / 32 * 16 + 1) * 64 + lane] = l;
  }
  __syncthreads();
  if (is_y && sidx > 0) return;
  if (is_y && rows_live) {
#pragma unroll 1
    for (int k = 0; k < 3; ++k) {
      const float* src = mg + k * (LY::MERGE_FLOATS * 64);
      const float mB = src[(D / 32 * 16) * 64 + lane];
      const float lB = src[(D / 32 * 16 + 1) * 64 + lane];
      const float mm = fmaxf(m, mB);
      const bool none = mm == -INFINITY;
      const float aA = none ? 0.0f : __builtin_amdgcn_exp2f(m - mm);
      const float aB = none ? 0.0f : __builtin_amdgcn_exp2f(mB - mm);
#pragma unroll
      for (int t = 0; t < D / 32; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][r] = o[t][r] * aA + src[(t * 16 + r) * 64 + lane] * aB;
      l = l * aA + lB * aB;
      m = mm;
    }
  }
  if (tile >= T) return;
  {
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l), __float_as_uint(l),
                                                     false, false);
    l = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
  }
  const int qs = q0 + r32;
  if (RASTER ? qs < n_i : qs < g.BS) {
    const bool real = qs < n_i;
    const float inv = (real && l > 0.0f) ? 1.0f / l : 0.0f;
    const int64_t orow = real ? q_row(qs) : head_row + int64_t(i) * g.BS + qs;
    __bf16* dst = ob + orow * D + 4 * half;
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
      lse[orow] = l > 0.0f ? (m + log2f(l)) * 0.69314718055994530942f : -INFINITY;
  }
}

template <int D, int T, bool RASTER, bool MULTI>
hipError_t launch_sw(const DevGeom& g, const void* qb, const void* kb, const void* vb,
                     const int* counts, const int* indices, float scale_log2, void* ob,
                     float* lse, hipStream_t s, const MultiTable* tab, const int* order,
                     int nb_max) {
  {  // the ring and the kept list exceed the 64 KB default
    const hipError_t e = ensure_dynamic_lds(
        reinterpret_cast<const void*>(&attn_sw_kernel<D, T, RASTER, MULTI>), kSwLds);
    if (e != hipSuccess) return e;
  }
  const size_t lds = size_t(SwLayout<D>::LIST_OFF) + size_t(nb_max) * sizeof(int);
  const uint4* q4 = static_cast<const uint4*>(qb);
  const char* k1 = static_cast<const char*>(kb);
  const char* v1 = static_cast<const char*>(vb);
  __bf16* o2 = static_cast<__bf16*>(ob);
  if constexpr (MULTI) {
    const int64_t items = int64_t(g.B) * tab->items_per_batch;
    attn_sw_kernel<D, T, RASTER, MULTI><<<dim3(unsigned(items)), 64 * kSwWaves, lds, s>>>(
        g, q4, k1, v1, nullptr, nullptr, scale_log2, o2, lse, order, *tab);
  } else {
    const int64_t items = int64_t(g.B) * g.H * ((g.NB + 7) / 8) * 8;  // see the XCD mapping
    attn_sw_kernel<D, T, RASTER, MULTI><<<dim3(unsigned(items)), 64 * kSwWaves, lds, s>>>(
        g, q4, k1, v1, counts, indices, scale_log2, o2, lse, order, NoTable{});
  }
  return hipGetLastError();
}

template <int D, int W, bool LD, bool RASTER, bool MULTI>
hipError_t launch_dw(const DevGeom& g, const void* qb, const void* kb, const void* vb,
                     const int* counts, const int* indices, float scale_log2, void* ob, float* lse,
                     hipStream_t s, const MultiTable* tab = nullptr, const int* order = nullptr) {
  {  // allow the kept-list LDS beyond the 64 KB default
    const hipError_t e = ensure_dynamic_lds(
        reinterpret_cast<const void*>(&attn_kernel<D, W, LD, RASTER, MULTI>),
        int(kMaxAttnNB * sizeof(int)));
    if (e != hipSuccess) return e;
  }
  const uint4* q4 = static_cast<const uint4*>(qb);
  const char* k1 = static_cast<const char*>(kb);
  const char* v1 = static_cast<const char*>(vb);
  __bf16* o2 = static_cast<__bf16*>(ob);
  if constexpr (MULTI) {
    int nb_max = 0;
    for (int k = 0; k < tab->n_heads; ++k) nb_max = max(nb_max, tab->geo[tab->head[k].geom].NB);
    const int64_t items = int64_t(g.B) * tab->items_per_batch;
    attn_kernel<D, W, LD, RASTER, MULTI><<<dim3(unsigned(items)), 64 * (W + LD),
                                           size_t(nb_max) * sizeof(int), s>>>(
        g, q4, k1, v1, nullptr, nullptr, scale_log2, o2, lse, order, *tab);
  } else {
    const int64_t items = int64_t(g.B) * g.H * ((g.NB + 7) / 8) * 8;  // see the XCD mapping
    attn_kernel<D, W, LD, RASTER, MULTI><<<dim3(unsigned(items)), 64 * (W + LD),
                                           size_t(g.NB) * sizeof(int), s>>>(
        g, q4, k1, v1, counts, indices, scale_log2, o2, lse, order, NoTable{});
  }
  return hipGetLastError();
}

template <int D, bool RASTER, bool MULTI = false>
hipError_t launch_d(const DevGeom& g, const void* qb, const void* kb, const void* vb,
                    const int* counts, const int* indices, float scale_log2, void* ob, float* lse,
                    hipStream_t s, const MultiTable* tab = nullptr, const int* order = nullptr) {
  int nb_max = g.NB;
  if constexpr (MULTI) {
    nb_max = 0;
    for (int k = 0; k < tab->n_heads; ++k) nb_max = max(nb_max, tab->geo[tab->head[k].geom].NB);
  }
  // 5 row tiles: the software-pipelined kernel when its ring and the kept list fit
  // the LDS (4-tile blocks stay on attn_kernel: with one pipelined wave per tile
  // and idle DMA waves the sw form was 15% slower there)
  if constexpr (D == 128) {
    if ((g.BS + 31) / 32 == kSwTiles &&
        size_t(SwLayout<D>::LIST_OFF) + size_t(nb_max) * sizeof(int) <= size_t(kSwLds))
      return launch_sw<D, kSwTiles, RASTER, MULTI>(g, qb, kb, vb, counts, indices, scale_log2, ob,
                                                   lse, s, tab, order, nb_max);
  }
  // otherwise the paired kernel for 5 row tiles when its ring and the kept list fit
  if ((g.BS + 31) / 32 == kPairTiles &&
      size_t(PPLayout<D>::LIST_OFF) + size_t(nb_max) * sizeof(int) <= size_t(kPairLds))
    return launch_pp<D, kPairTiles, RASTER, MULTI>(g, qb, kb, vb, counts, indices, scale_log2, ob,
                                                   lse, s, tab, order, nb_max);
#define SPADE_ATTN_CASE(w, ld)                                                                  \
  case w:                                                                                       \
    return launch_dw<D, w, ld, RASTER, MULTI>(g, qb, kb, vb, counts, indices, scale_log2, ob, \
                                              lse, s, tab, order);
  // loader wave unless it would cost a workgroup per CU (4 or 6 compute waves)
  switch ((g.BS + 31) / 32) {
    SPADE_ATTN_CASE(1, true) SPADE_ATTN_CASE(2, true) SPADE_ATTN_CASE(3, true)
    SPADE_ATTN_CASE(4, false) SPADE_ATTN_CASE(5, true) SPADE_ATTN_CASE(6, false)
    SPADE_ATTN_CASE(7, true) SPADE_ATTN_CASE(8, true)
  }
#undef SPADE_ATTN_CASE
  return hipErrorInvalidValue;
}

// Ranked work order (§3.3 (3): rows preprocessed into a ranked layout, heads of
// similar density co-scheduled). The dispatch walks the (batch, head) pairs in
// the order of their heaviest row, then their total kept blocks (descending,
// ties to the lower index), so long rows start first instead of forming the
// tail; within a head each XCD takes its rows heaviest first (heavy_first).
constexpr int kRankThreads = 1024;

__global__ void __launch_bounds__(256) head_keys_kernel(DevGeom g, const int* __restrict__ counts,
                                                        uint64_t* __restrict__ keys) {
  __shared__ int smax[256];
  __shared__ uint32_t ssum[256];
  const int64_t bh = blockIdx.x;
  int mx = 0;
  uint32_t sum = 0;
  for (int i = threadIdx.x; i < g.NB; i += 256) {
    const int c = min(max(counts[bh * g.NB + i], 0), g.NB);
    mx = max(mx, c);
    sum += uint32_t(c);
  }
  smax[threadIdx.x] = mx;
  ssum[threadIdx.x] = sum;
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if (threadIdx.x < st) {
      smax[threadIdx.x] = max(smax[threadIdx.x], smax[threadIdx.x + st]);
      ssum[threadIdx.x] += ssum[threadIdx.x + st];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) keys[bh] = (uint64_t(uint32_t(smax[0])) << 32) | ssum[0];
}

__global__ void __launch_bounds__(kRankThreads) head_rank_kernel(const uint64_t* __restrict__ keys,
                                                                 int n, int* __restrict__ order) {
  for (int t = threadIdx.x; t < n; t += kRankThreads) {
    const uint64_t kt = keys[t];
    int rank = 0;
    for (int j = 0; j < n; ++j) {
      const uint64_t kj = keys[j];
      rank += (kj > kt || (kj == kt && j < t)) ? 1 : 0;
    }
    order[rank] = t;
  }
}

// The same ranking for one multi-scheme launch, per batch element over the
// launch's heads; the heads' first items follow as prefix sums of their padded
// item counts in rank order. Layout of `ranked`: per batch element, n head
// indices by rank, then n first items.
__global__ void __launch_bounds__(256) multi_keys_kernel(MultiTable tab,
                                                         uint64_t* __restrict__ keys) {
  __shared__ int smax[256];
  __shared__ uint32_t ssum[256];
  const int n = tab.n_heads;
  const int b = int(blockIdx.x) / n, k = int(blockIdx.x) - b * n;
  const MultiHead& mh = tab.head[k];
  const int NB = tab.geo[mh.geom].NB;
  const int* cnt = mh.counts + int64_t(b) * mh.counts_bstride;
  int mx = 0;
  uint32_t sum = 0;
  for (int i = threadIdx.x; i < NB; i += 256) {
    const int c = min(max(cnt[i], 0), NB);
    mx = max(mx, c);
    sum += uint32_t(c);
  }
  smax[threadIdx.x] = mx;
  ssum[threadIdx.x] = sum;
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if (threadIdx.x < st) {
      smax[threadIdx.x] = max(smax[threadIdx.x], smax[threadIdx.x + st]);
      ssum[threadIdx.x] += ssum[threadIdx.x + st];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) keys[blockIdx.x] = (uint64_t(uint32_t(smax[0])) << 32) | ssum[0];
}

__global__ void __launch_bounds__(64) multi_rank_kernel(MultiTable tab,
                                                        const uint64_t* __restrict__ keys,
                                                        int* __restrict__ ranked) {
  __shared__ int by_rank[kMaxMultiHeads];
  const int n = tab.n_heads, b = blockIdx.x;
  const uint64_t* kb = keys + int64_t(b) * n;
  const int t = threadIdx.x;
  if (t < n) {
    const uint64_t kt = kb[t];
    int rank = 0;
    for (int j = 0; j < n; ++j) {
      const uint64_t kj = kb[j];
      rank += (kj > kt || (kj == kt && j < t)) ? 1 : 0;
    }
    by_rank[rank] = t;
  }
  __syncthreads();
  if (t == 0) {
    int* out = ranked + int64_t(b) * 2 * n;
    int first = 0;
    for (int r = 0; r < n; ++r) {
      const int k = by_rank[r];
      out[r] = k;
      out[n + r] = first;
      first += (tab.geo[tab.head[k].geom].NB + 7) / 8 * 8;
    }
  }
}

size_t ranked_pairs(const DevGeom& g) {
  const int64_t n = int64_t(g.B) * g.H;
  return n > 0 && n <= kMaxRankedHeads ? size_t(n) : 0;
}

}  // namespace

hipError_t noalloc_scratch(void** ptr, size_t* bytes) {
  static std::mutex mu;
  static void* by_device[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (by_device[dev] == nullptr) {  // first call on this device: look the copy up once
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    by_device[dev] = p;
  }
  *ptr = by_device[dev];
  *bytes = kNoAllocScratchBytes;
  return hipSuccess;
}

size_t attn_workspace_bytes(const DevGeom& g) {
  // keys (8 B) of every pair, then the order (4 B; a multi-scheme launch also
  // keeps each head's first item, 4 B more)
  const size_t n = ranked_pairs(g);
  return n ? n * 16 : 0;
}

hipError_t launch_sparse_attn_multi(const DevGeom* geo, int n_geo, const MultiHead* heads,
                                    int n_heads, const void* q, const void* k, const void* v,
                                    float scale, void* o, float* lse, void* ws, hipStream_t s) {
  const float sl2 = scale * 1.44269504088896340736f;
  // each launch ranks its heads in its own part of the workspace (16 B per pair)
  const bool rank = ranked_pairs(geo[0]) > 0;
  char* wsp = static_cast<char*>(ws);
  // one launch per workgroup shape; the launch's geometry carries that shape's BS
  for (int w = 1; w <= kMaxBS / 32; ++w) {
    MultiTable tab = {};
    for (int c = 0; c < n_geo; ++c) tab.geo[c] = geo[c];
    int start = 0, widest = -1;
    for (int hh = 0; hh < n_heads; ++hh) {
      const DevGeom& gh = geo[heads[hh].geom];
      if ((gh.BS + 31) / 32 != w) continue;
      MultiHead mh = heads[hh];
      mh.start = start;
      start += (gh.NB + 7) / 8 * 8;
      tab.head[tab.n_heads++] = mh;
      if (widest < 0 || gh.BS > geo[widest].BS) widest = heads[hh].geom;
    }
    if (tab.n_heads == 0) continue;
    tab.items_per_batch = start;
    const DevGeom& gl = geo[widest];
    const int* order = nullptr;
    if (rank) {
      const int64_t pairs = int64_t(gl.B) * tab.n_heads;
      uint64_t* keys = reinterpret_cast<uint64_t*>(wsp);
      int* ranked = reinterpret_cast<int*>(keys + pairs);
      wsp += pairs * 16;
      multi_keys_kernel<<<dim3(unsigned(pairs)), 256, 0, s>>>(tab, keys);
      multi_rank_kernel<<<dim3(unsigned(gl.B)), 64, 0, s>>>(tab, keys, ranked);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      order = ranked;
    }
    const hipError_t e = gl.d == 128
        ? launch_d<128, true, true>(gl, q, k, v, nullptr, nullptr, sl2, o, lse, s, &tab, order)
        : launch_d<64, true, true>(gl, q, k, v, nullptr, nullptr, sl2, o, lse, s, &tab, order);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_block_sparse_attn(const DevGeom& g, const void* qb, const void* kb,
                                    const void* vb, const int* counts, const int* indices,
                                    float scale, void* ob, float* lse, void* ws, bool raster,
                                    hipStream_t s) {
  const float sl2 = scale * 1.44269504088896340736f;
  const int* order = nullptr;
  if (const size_t n = ranked_pairs(g)) {
    uint64_t* keys = static_cast<uint64_t*>(ws);
    int* ord = reinterpret_cast<int*>(keys + n);
    head_keys_kernel<<<dim3(unsigned(n)), 256, 0, s>>>(g, counts, keys);
    head_rank_kernel<<<1, kRankThreads, 0, s>>>(keys, int(n), ord);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    order = ord;
  }
  if (g.d == 128)
    return raster ? launch_d<128, true>(g, qb, kb, vb, counts, indices, sl2, ob, lse, s, nullptr, order)
                  : launch_d<128, false>(g, qb, kb, vb, counts, indices, sl2, ob, lse, s, nullptr, order);
  if (g.d == 64)
    return raster ? launch_d<64, true>(g, qb, kb, vb, counts, indices, sl2, ob, lse, s, nullptr, order)
                  : launch_d<64, false>(g, qb, kb, vb, counts, indices, sl2, ob, lse, s, nullptr, order);
  return hipErrorInvalidValue;
}

}  // namespace spade
