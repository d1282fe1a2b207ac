// Workgroup-level building blocks for kernels that run one utterance per
// 1024-thread workgroup (16 wave64 wavefronts): ballot-aggregated appends,
// scans and reductions through LDS.
#pragma once

#include "wd_common.h"

namespace wd {

__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x & 63u; }
__device__ __forceinline__ uint32_t wave_id() { return threadIdx.x >> 6; }
__device__ __forceinline__ uint64_t lanemask_lt() {
  return (lane_id() == 0) ? 0ull : (~0ull >> (64u - lane_id()));
}

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t n = __shfl_up(v, o, 64);
    if ((int)lane_id() >= o) v += n;
  }
  return v;
}

__device__ __forceinline__ uint64_t shfl_up64(uint64_t v, int o) {
  uint32_t lo = __shfl_up((uint32_t)v, o, 64);
  uint32_t hi = __shfl_up((uint32_t)(v >> 32), o, 64);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_incl_scan64(uint64_t v) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint64_t n = shfl_up64(v, o);
    if ((int)lane_id() >= o) v += n;
  }
  return v;
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
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) {
    uint64_t o = shfl_xor64(v, m);
    v = o < v ? o : v;
  }
  if (lane_id() == 0) bs.w64[b][wave_id()] = v;
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
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) v += shfl_xor64(v, m);
  if (lane_id() == 0) bs.w64[b][wave_id()] = v;
  __syncthreads();
  uint64_t r = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) r += bs.w64[b][i];
  return r;
}

__device__ __forceinline__ uint32_t wave_or(uint32_t v) {
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) v |= __shfl_xor(v, m, 64);
  return v;
}

template <int NW = kWaves>
__device__ __forceinline__ uint32_t block_or(uint32_t v, BlockScratch& bs, uint32_t& par) {
  const uint32_t b = par;
  par ^= 1u;
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) v |= __shfl_xor(v, m, 64);
  if (lane_id() == 0) bs.w32[b][wave_id()] = v;
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
    base = __shfl(base, leader, 64);
  }
  return base + (uint32_t)__popcll(m & lanemask_lt());
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

}  // namespace wd
