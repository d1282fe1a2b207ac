// Workgroup-level building blocks for kernels that run one utterance per
// 1024-thread workgroup (16 wave64 wavefronts): ballot-aggregated appends,
// scans and reductions through LDS.
#pragma once

#include "wd_common.h"

namespace wd {

__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x & 63u; }

// v, through an empty asm: values derived from the result are computed where
// they are used instead of being hoisted out of a long loop and held (or
// spilled) across it.
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}
__device__ __forceinline__ uint32_t wave_id() { return threadIdx.x >> 6; }
// Set bits of m in the lanes below this one (the mbcnt instructions count
// them directly, with no lane mask to build or keep).
__device__ __forceinline__ uint32_t rank_in(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Wavefront scans and reductions by DPP (data-parallel primitives of the
// GFX9 vector ALU: a lane reads another lane's register within the same
// instruction), which take a few cycles per step where a shuffle through
// the LDS crossbar takes a round trip.  A wavefront is four rows of 16
// lanes: row shifts by 1, 2, 4 and 8 scan each row, then lane 15 of rows 0
// and 2 is broadcast into rows 1 and 3 and lane 31 into rows 2 and 3.
// Every lane of the wavefront must be active.
enum : int {
  kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118,
  kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143,
  // within each group of four lanes: swap neighbours (1,0,3,2), swap pairs (2,3,0,1)
  kDppQuadSwap1 = 0xb1, kDppQuadSwap2 = 0x4e
};

// Lane i reads the lane its DPP control names; `fill` where that lane is
// outside the row or the row is not in ROWS.
template <int CTRL, int ROWS = 0xf>
__device__ __forceinline__ uint32_t dpp32(uint32_t v, uint32_t fill) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)fill, (int)v, CTRL, ROWS, 0xf, false);
}

template <int CTRL, int ROWS = 0xf>
__device__ __forceinline__ uint64_t dpp64(uint64_t v, uint64_t fill) {
  const uint32_t lo = dpp32<CTRL, ROWS>((uint32_t)v, (uint32_t)fill);
  const uint32_t hi = dpp32<CTRL, ROWS>((uint32_t)(v >> 32), (uint32_t)(fill >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Inclusive scan over the wavefront with an associative op and its identity.
template <class T, class Op>
__device__ __forceinline__ T wave_scan_op(T v, T id, Op op) {
  if constexpr (sizeof(T) == 8) {
    v = op(v, (T)dpp64<kDppRowShr1>(v, id));
    v = op(v, (T)dpp64<kDppRowShr2>(v, id));
    v = op(v, (T)dpp64<kDppRowShr4>(v, id));
    v = op(v, (T)dpp64<kDppRowShr8>(v, id));
    v = op(v, (T)dpp64<kDppRowBcast15, 0xa>(v, id));
    v = op(v, (T)dpp64<kDppRowBcast31, 0xc>(v, id));
  } else {
    v = op(v, (T)dpp32<kDppRowShr1>(v, id));
    v = op(v, (T)dpp32<kDppRowShr2>(v, id));
    v = op(v, (T)dpp32<kDppRowShr4>(v, id));
    v = op(v, (T)dpp32<kDppRowShr8>(v, id));
    v = op(v, (T)dpp32<kDppRowBcast15, 0xa>(v, id));
    v = op(v, (T)dpp32<kDppRowBcast31, 0xc>(v, id));
  }
  return v;
}

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  return wave_scan_op<uint32_t>(v, 0u, [](uint32_t a, uint32_t b) { return a + b; });
}

__device__ __forceinline__ uint64_t wave_incl_scan64(uint64_t v) {
  return wave_scan_op<uint64_t>(v, 0ull, [](uint64_t a, uint64_t b) { return a + b; });
}

// Value of lane 63 in every lane (a scalar register).
__device__ __forceinline__ uint32_t lane63(uint32_t v) { return (uint32_t)__builtin_amdgcn_readlane((int)v, 63); }
__device__ __forceinline__ uint64_t lane63_64(uint64_t v) {
  return ((uint64_t)lane63((uint32_t)(v >> 32)) << 32) | lane63((uint32_t)v);
}

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int m) {
  uint32_t lo = __shfl_xor((uint32_t)v, m, 64);
  uint32_t hi = __shfl_xor((uint32_t)(v >> 32), m, 64);
  return ((uint64_t)hi << 32) | lo;
}

// Scratch a workgroup needs for its collectives.  Two buffers used in turn
// make each collective cost one barrier: a wave can only come back to a buffer
// after every wave has passed the barrier of the collective in between, i.e.
// after every wave has read it.  `par` is per thread, flipped by every
// collective; all threads call the same sequence of collectives.  NW is the
// workgroup's wavefront count (the scratch holds up to kWaves).
struct BlockScratch {
  uint32_t w32[2][kWaves];
  unsigned long long w64[2][kWaves];
};

// Exclusive prefix sum over the workgroup (thread order); *total = sum.
template <int NW = kWaves>
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, BlockScratch& bs, uint32_t& par,
                                                    uint32_t* total) {
  const uint32_t b = par;
  par ^= 1u;
  const uint32_t inc = wave_incl_scan(v);
  if (lane_id() == 63) bs.w32[b][wave_id()] = inc;
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint32_t x = bs.w32[b][i];
    before += (uint32_t)i < wave_id() ? x : 0u;
    tot += x;
  }
  *total = tot;
  return before + inc - v;
}

template <int NW = kWaves>
__device__ __forceinline__ uint64_t block_excl_scan64(uint64_t v, BlockScratch& bs, uint32_t& par,
                                                      uint64_t* total) {
  const uint32_t b = par;
  par ^= 1u;
  const uint64_t inc = wave_incl_scan64(v);
  if (lane_id() == 63) bs.w64[b][wave_id()] = inc;
  __syncthreads();
  uint64_t before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint64_t x = bs.w64[b][i];
    before += (uint32_t)i < wave_id() ? x : 0ull;
    tot += x;
  }
  *total = tot;
  return before + inc - v;
}

template <int NW = kWaves>
__device__ __forceinline__ uint64_t block_min64(uint64_t v, BlockScratch& bs, uint32_t& par) {
  const uint32_t b = par;
  par ^= 1u;
  v = wave_scan_op<uint64_t>(v, ~0ull, [](uint64_t a, uint64_t c) { return c < a ? c : a; });
  if (lane_id() == 63) bs.w64[b][wave_id()] = v;
  __syncthreads();
  uint64_t r = bs.w64[b][0];
#pragma unroll
  for (int i = 1; i < NW; ++i) r = bs.w64[b][i] < r ? bs.w64[b][i] : r;
  return r;
}

template <int NW = kWaves>
__device__ __forceinline__ uint64_t block_sum64(uint64_t v, BlockScratch& bs, uint32_t& par) {
  const uint32_t b = par;
  par ^= 1u;
  v = wave_incl_scan64(v);
  if (lane_id() == 63) bs.w64[b][wave_id()] = v;
  __syncthreads();
  uint64_t r = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) r += bs.w64[b][i];
  return r;
}

__device__ __forceinline__ uint32_t wave_or(uint32_t v) {
  return lane63(wave_scan_op<uint32_t>(v, 0u, [](uint32_t a, uint32_t c) { return a | c; }));
}

template <int NW = kWaves>
__device__ __forceinline__ uint32_t block_or(uint32_t v, BlockScratch& bs, uint32_t& par) {
  const uint32_t b = par;
  par ^= 1u;
  v = wave_scan_op<uint32_t>(v, 0u, [](uint32_t a, uint32_t c) { return a | c; });
  if (lane_id() == 63) bs.w32[b][wave_id()] = v;
  __syncthreads();
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) r |= bs.w32[b][i];
  return r;
}

// Append for every lane with `pred` set: one LDS atomic per wavefront, slot
// order by lane within the wave.  Must be reached by the whole wavefront.
__device__ __forceinline__ uint32_t wave_append(bool pred, uint32_t* counter) {
  uint64_t m = __ballot(pred);
  uint32_t base = 0;
  if (m) {
    int leader = __ffsll((unsigned long long)m) - 1;
    if ((int)lane_id() == leader) base = atomicAdd(counter, (uint32_t)__popcll(m));
    base = (uint32_t)__builtin_amdgcn_readlane((int)base, leader);
  }
  return base + rank_in(m);
}

// Last i in [0, n) with a[i] <= w, for a non-decreasing a with a[0] <= w.
__device__ __forceinline__ uint32_t search_le(const uint32_t* a, uint32_t n, uint32_t w) {
  uint32_t lo = 0, hi = n;
  while (hi - lo > 1) {
    uint32_t mid = (lo + hi) >> 1;
    if (a[mid] <= w) lo = mid;
    else hi = mid;
  }
  return lo;
}

__device__ __forceinline__ float canon(float x) { return x == 0.0f ? 0.0f : x; }

// Number of entries of the sorted a[0..n) below w.
__device__ __forceinline__ uint64_t lower_bound64(const uint64_t* a, uint64_t n, uint64_t w) {
  uint64_t lo = 0, hi = n;
  while (lo < hi) {
    uint64_t mid = (lo + hi) >> 1;
    if (a[mid] < w) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

}  // namespace wd
