// Blocking (layout transform) and its inverse — paper §3.3 (rearrange Q/K/V
// into the blocked layout of a blocking scheme; restore the output layout).
//
// One workgroup per (block, head). Each 16-byte lane vector is one piece of a
// token row, so a row of d elements is moved by d*esize/16 consecutive lanes
// (one 256-byte transaction for bf16 d=128). The block's origin and extents are
// computed once per workgroup; a slot's (dt, dy, dx) is recovered with float
// reciprocals, exact because slots and extents are below 2^8 (see kMaxBS).
#include "spade_internal.h"

namespace spade {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

// raster [B, H, N, row] -> blocked [B, n, NB*BS, row]; padding slots get zeros.
template <int VPR>
__global__ void __launch_bounds__(kThreads) reorder_fwd(DevGeom g, HeadMap hm,
                                                        const uint4* __restrict__ x,
                                                        uint4* __restrict__ y) {
  const int b = blockIdx.x;
  int64_t bh_blk, bh_ras;
  head_pair(g, hm, &bh_blk, &bh_ras);
  const BlockExt e = block_ext(g, b);
  const float r_ew = 1.0f / float(e.ew), r_eh = 1.0f / float(e.eh);
  const uint4* src = x + bh_ras * g.N * VPR;
  uint4* dst = y + (bh_blk * g.NB + b) * int64_t(g.BS) * VPR;
  const int total = g.BS * VPR;
  const int valid = e.n * VPR;
  for (int f0 = threadIdx.x; f0 < total; f0 += kThreads * kUnroll) {
    uint4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int f = f0 + u * kThreads;
      v[u] = make_uint4(0, 0, 0, 0);
      if (f < valid) {
        const int slot = f / VPR, vec = f % VPR;
        v[u] = src[block_slot_token(g, e, r_ew, r_eh, slot) * VPR + vec];
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int f = f0 + u * kThreads;
      if (f < total) dst[f] = v[u];
    }
  }
}

// blocked [B, n, NB*BS, row] -> raster [B, H, N, row] (listed heads only);
// padding slots are not read.
template <int VPR>
__global__ void __launch_bounds__(kThreads) reorder_inv(DevGeom g, HeadMap hm,
                                                        const uint4* __restrict__ xb,
                                                        uint4* __restrict__ y) {
  const int b = blockIdx.x;
  int64_t bh_blk, bh_ras;
  head_pair(g, hm, &bh_blk, &bh_ras);
  const BlockExt e = block_ext(g, b);
  const float r_ew = 1.0f / float(e.ew), r_eh = 1.0f / float(e.eh);
  const uint4* src = xb + (bh_blk * g.NB + b) * int64_t(g.BS) * VPR;
  uint4* dst = y + bh_ras * g.N * VPR;
  const int valid = e.n * VPR;
  for (int f0 = threadIdx.x; f0 < valid; f0 += kThreads * kUnroll) {
    uint4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int f = f0 + u * kThreads;
      if (f < valid) v[u] = src[f];
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int f = f0 + u * kThreads;
      if (f < valid) {
        const int slot = f / VPR, vec = f % VPR;
        dst[block_slot_token(g, e, r_ew, r_eh, slot) * VPR + vec] = v[u];
      }
    }
  }
}

template <int VPR>
hipError_t launch_vpr(const DevGeom& g, const void* x, void* y, int inverse, const HeadMap& hm,
                      hipStream_t s) {
  const dim3 grid(g.NB, g.B * hm.n);
  if (inverse)
    reorder_inv<VPR><<<grid, kThreads, 0, s>>>(g, hm, static_cast<const uint4*>(x),
                                               static_cast<uint4*>(y));
  else
    reorder_fwd<VPR><<<grid, kThreads, 0, s>>>(g, hm, static_cast<const uint4*>(x),
                                               static_cast<uint4*>(y));
  return hipGetLastError();
}

}  // namespace

hipError_t launch_reorder(const DevGeom& g, const void* x, void* y, int esize, int inverse,
                          const HeadMap& hm, hipStream_t s) {
  switch (g.d * esize / 16) {
    case 8: return launch_vpr<8>(g, x, y, inverse, hm, s);
    case 16: return launch_vpr<16>(g, x, y, inverse, hm, s);
    case 32: return launch_vpr<32>(g, x, y, inverse, hm, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace spade
