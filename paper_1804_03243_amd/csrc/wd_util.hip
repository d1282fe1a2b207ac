// Small per-decode kernels around the decoder: input checks, fills, the lane
// frame ranges of a stream, and the packing of results for the host.
#include "wd_host.h"

namespace wd {

// Log-likelihood check: NaN, +inf and values above 1e30 are rejected.
// Rows of the frames this launch decodes, t0..T (frame t reads row t - 1).
// A streaming read: four independent loads per thread per step keep enough
// of them in flight to run at HBM speed.
__device__ __forceinline__ bool bad_loglike(float v) { return v != v || v > 1e30f; }

__global__ void k_check_loglikes(const LaneDesc* __restrict__ lanes, uint32_t P, uint32_t* bad) {
  const LaneDesc L = lanes[blockIdx.y];
  const uint64_t n = (uint64_t)L.T * P;
  const uint64_t r0 = (uint64_t)(L.t0 > 0 ? L.t0 - 1 : 0) * P;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  uint64_t i = r0 + (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool b = false;
  for (; i + 3 * stride < n; i += 4 * stride) {
    const float v0 = L.ll[i], v1 = L.ll[i + stride], v2 = L.ll[i + 2 * stride], v3 = L.ll[i + 3 * stride];
    b |= bad_loglike(v0) | bad_loglike(v1) | bad_loglike(v2) | bad_loglike(v3);
  }
  for (; i < n; i += stride) b |= bad_loglike(L.ll[i]);
  if (b) atomicOr(&bad[blockIdx.y], 1u);
}

__global__ void k_fill_u64(unsigned long long* p, uint64_t n, unsigned long long v) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

__global__ void k_fill_u32(uint32_t* p, uint64_t n, uint32_t v) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// Results of every finished utterance (links, nodes, words) packed into one
// contiguous buffer, so that the host copies them with one transfer: lane b
// starts after the lanes before it, each lane's part is its links, its nodes
// and its words padded to 16 bytes (packed_bytes; the host computes the same
// offsets).  One workgroup per lane.
__device__ __forceinline__ uint64_t packed_bytes(const LaneInfo& I) {
  if (I.status != 0 || I.tb_fail) return 0;
  return sizeof(OutLink) * I.kept + sizeof(OutNode) * I.out_nodes + ((4 * I.nwords + 15) & ~15ull);
}

__global__ void k_pack_results(const LaneDesc* __restrict__ lanes, int B, char* __restrict__ dst) {
  const int b = blockIdx.x;
  uint64_t off = 0;
  for (int k = 0; k < b; ++k) off += packed_bytes(*lanes[k].info);
  const LaneDesc& L = lanes[b];
  const LaneInfo& I = *L.info;
  if (!packed_bytes(I)) return;
  uint4* out = reinterpret_cast<uint4*>(dst + off);
  const uint64_t nl = I.kept * (sizeof(OutLink) / 16), nn = I.out_nodes;
  const uint4* ls = reinterpret_cast<const uint4*>(L.out_links);
  const uint4* ns = reinterpret_cast<const uint4*>(L.out_nodes);
  for (uint64_t i = threadIdx.x; i < nl; i += blockDim.x) out[i] = ls[i];
  for (uint64_t i = threadIdx.x; i < nn; i += blockDim.x) out[nl + i] = ns[i];
  uint32_t* w = reinterpret_cast<uint32_t*>(out + nl + nn);
  for (uint64_t i = threadIdx.x; i < I.nwords; i += blockDim.x) w[i] = (uint32_t)L.out_words[i];
}

void launch_pack_results(const LaneDesc* lanes, int B, void* dst, hipStream_t s) {
  hipLaunchKernelGGL(k_pack_results, dim3(B), dim3(256), 0, s, lanes, B, (char*)dst);
}

constexpr int kSetLanes = 128;
struct FrameSet {
  int32_t T[kSetLanes];
  int32_t t0[kSetLanes];
  int32_t b0, n, open;
};

__global__ void k_set_frames(LaneDesc* lanes, FrameSet f) {
  for (int i = (int)threadIdx.x; i < f.n; i += (int)blockDim.x) {
    LaneDesc& L = lanes[f.b0 + i];
    L.T = f.T[i];
    L.t0 = f.t0[i];
    L.open = f.open;
  }
}

void launch_set_frames(LaneDesc* lanes, int B, const int32_t* T, const int32_t* t0, int32_t open, hipStream_t s) {
  for (int b0 = 0; b0 < B; b0 += kSetLanes) {
    FrameSet f{};
    f.b0 = b0;
    f.n = B - b0 < kSetLanes ? B - b0 : kSetLanes;
    f.open = open;
    for (int i = 0; i < f.n; ++i) {
      f.T[i] = T[b0 + i];
      f.t0[i] = t0[b0 + i];
    }
    hipLaunchKernelGGL(k_set_frames, dim3(1), dim3(kSetLanes), 0, s, lanes, f);
  }
}


void launch_check_loglikes(const LaneDesc* lanes, int B, uint32_t P, uint32_t* bad, hipStream_t s) {
  // ~2048 workgroups in all (at least 16 per utterance)
  const int gx = B >= 128 ? 16 : 2048 / B;
  hipLaunchKernelGGL(k_check_loglikes, dim3(gx, B), dim3(256), 0, s, lanes, P, bad);
}

void launch_fill_u64(unsigned long long* p, uint64_t n, unsigned long long v, hipStream_t s) {
  if (n) hipLaunchKernelGGL(k_fill_u64, dim3(1024), dim3(256), 0, s, p, n, v);
}

void launch_fill_u32(uint32_t* p, uint64_t n, uint32_t v, hipStream_t s) {
  if (n) hipLaunchKernelGGL(k_fill_u32, dim3(1024), dim3(256), 0, s, p, n, v);
}

}  // namespace wd
