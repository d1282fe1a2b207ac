// Lattice links of the one-workgroup decode (Sec. 3.4), written after the
// forward pass from what it recorded, every frame at once.
//
// A link is a token-passing operation whose result is within the frame's
// final cutoff: an emitting arc out of a token of frame t-1 into frame t, or
// an epsilon arc out of a token of frame t.  Its cost is the same fp32 sum
// the forward pass formed (token cost, then the acoustic cost, then the arc
// weight, each addition rounded), so it can be formed again from the node
// store (each frame's tokens in state order, with their cost keys), the
// graph and the log-likelihoods; the forward pass keeps only the per-frame
// node records and cutoffs.  The links of frame t are its emitting links in
// work-item order (frontier of frame t-1 in state order, each token's arcs
// in arc order: arc-id order) followed by its epsilon links (frontier of
// frame t in state order, each token's epsilon arcs in order), exactly the
// layout the lattice pass reads.  Three launches: per-frame counts, one
// workgroup per utterance turning them into offsets (and checking the link
// store's capacity), then the links, each frame by one workgroup.
#include "wd_block.h"
#include "wd_host.h"

namespace wd {

constexpr int kLT = 256;              // threads per workgroup
constexpr int kLWv = kLT / 64;        // wavefronts
constexpr uint32_t kLinkBlocks = 256;  // workgroups per utterance (frames in turn)

struct LinkShared {
  BlockScratch bs;
  uint32_t pre[kLT];    // exclusive prefix of the tile's tokens' arc counts
  uint32_t beg[kLT];    // first arc of each token of the tile
  float cost[kLT];      // token cost
  uint32_t cls[kLT];    // token state's epsilon level (epsilon runs)
};

// The node of state s among one frame's nodes [n0, n1) (sorted by state), or
// ~0 when s has none.
__device__ __forceinline__ uint64_t node_of(const LaneDesc& L, uint64_t n0, uint64_t n1, uint32_t s) {
  uint64_t lo = n0, hi = n1;
  while (lo < hi) {
    const uint64_t mid = (lo + hi) >> 1;
    if (L.n_state[mid] < s) lo = mid + 1;
    else hi = mid;
  }
  return lo < n1 && L.n_state[lo] == s ? lo : ~0ull;
}

// One run of frame t: the emitting links (kEps false; sources: the nodes of
// frame t-1) or the epsilon links (sources: the nodes of frame t).  Counts
// them (kWrite false: returns the count in every thread) or writes them from
// link `at` on (returns the count, sets *xmask and *bad).
template <bool kEps, bool kWrite>
__device__ __forceinline__ uint32_t link_run(const DevGraph& g, const LaneDesc& L, LinkShared& sh, uint32_t& par,
                                             int t, uint32_t cut, uint64_t at, uint32_t* xmask, uint32_t* bad) {
  const uint32_t tid = threadIdx.x;
  const uint64_t p0 = L.node_off[kEps ? t : t - 1], p1 = L.node_off[kEps ? t + 1 : t];
  const uint64_t d0 = L.node_off[t], d1 = L.node_off[t + 1];  // destinations: frame t
  const float* row = L.ll + (size_t)(t > 0 ? t - 1 : 0) * g.P;
  uint32_t n = 0;  // links of the run so far (write mode: in every thread)
  uint32_t cnt = 0;  // count mode: this thread's links
  for (uint64_t q0 = p0; q0 < p1; q0 += kLT) {
    const uint32_t m = (uint32_t)(p1 - q0 < (uint64_t)kLT ? p1 - q0 : (uint64_t)kLT);
    uint32_t deg = 0, a0 = 0, c = 0;
    float cost = 0.0f;
    if (tid < m) {
      const uint32_t s = L.n_state[q0 + tid];
      cost = key_cost((uint32_t)(L.n_pack[q0 + tid] >> 32));
      const uint4 o0 = g.off[s], o1 = g.off[s + 1];
      a0 = kEps ? o0.y : o0.x;
      deg = kEps ? o1.y - o0.y : o1.x - o0.x;
      if (kEps) c = g.sclass[s];
    }
    uint32_t tot;
    const uint32_t ex = block_excl_scan<kLWv>(deg, sh.bs, par, &tot);
    sh.pre[tid] = ex;
    sh.beg[tid] = a0;
    sh.cost[tid] = cost;
    sh.cls[tid] = c;
    __syncthreads();
    for (uint32_t w0 = 0; w0 < tot; w0 += kLT) {
      const uint32_t w = w0 + tid;
      bool in = false;
      uint32_t j = 0, xb = 0;
      uint4 r = make_uint4(0, 0, 0, 0);
      if (w < tot) {
        j = search_le(sh.pre, m, w);
        const uint32_t a = sh.beg[j] + (w - sh.pre[j]);
        float x;
        if (kEps) {
          r = g.xarc[a];
          x = canon(sh.cost[j] + __uint_as_float(r.y));
        } else {
          r = g.earc[a];
          const float ac = -row[(r.z & 0xffffffu) - 1u];
          x = sh.cost[j] + ac;
          x = canon(x + __uint_as_float(r.y));
        }
        xb = __float_as_uint(x);
        const uint32_t xk = cost_key(x);
        in = xk <= cut && xk < kInfKey;
      }
      if (!kWrite) {
        cnt += in ? 1u : 0u;
        continue;
      }
      uint32_t nsub;
      const uint32_t pos = n + block_excl_scan<kLWv>(in ? 1u : 0u, sh.bs, par, &nsub);
      n += nsub;
      if (!in) continue;
      const uint64_t dn = node_of(L, d0, d1, r.x);
      if (dn == ~0ull) {
        *bad = 1;
        continue;
      }
      const uint32_t src = (uint32_t)(q0 + j);
      L.links[at + pos] = make_uint4(r.w, src, (uint32_t)dn, xb);
      if (kEps) {
        const uint32_t cls = sh.cls[j];
        L.link_lvl[at + pos] = (uint8_t)cls;
        *xmask |= 1u << (cls < 31u ? cls : 31u);
      }
      // the link that made the destination's token names its predecessor
      if (L.n_pack[dn] == pack_tok(cost_key(__uint_as_float(xb)), r.w)) L.n_pred[dn] = src;
    }
    __syncthreads();  // every read of the tile's arrays done before the next tile
  }
  if (!kWrite) {
    uint32_t all;
    (void)block_excl_scan<kLWv>(cnt, sh.bs, par, &all);
    return all;
  }
  return n;
}

// A decode whose forward pass stopped, or whose node store overflowed, gets
// no links (its status already says so).
__device__ __forceinline__ bool links_wanted(const LaneDesc& L) {
  return L.info->status == 0 && (L.info->overflow & kOvfNodes) == 0;
}

// Per frame: emitting links into link_xoff[t], epsilon links into link_end[t]
// (counts; the offset kernel turns them into offsets).
__global__ void __launch_bounds__(kLT) k_links_count(DevGraph g, const LaneDesc* __restrict__ lanes) {
  __shared__ LinkShared sh;
  const LaneDesc& L = lanes[blockIdx.y];
  if (!links_wanted(L)) return;
  uint32_t par = 0;
  for (int t = (int)blockIdx.x; t <= L.T; t += (int)gridDim.x) {
    const uint32_t cut = cost_key(L.cut[t]);
    const uint32_t ne = t > 0 ? link_run<false, false>(g, L, sh, par, t, cut, 0, nullptr, nullptr) : 0u;
    const uint32_t nx = link_run<true, false>(g, L, sh, par, t, cut, 0, nullptr, nullptr);
    if (threadIdx.x == 0) {
      L.link_xoff[t] = ne;
      L.link_end[t] = nx;
      // the step profile's frame record takes the frame's link count
      if (L.prof) {
        uint64_t& rec = L.prof[(size_t)t * kProfSlots + kProfStamps];
        rec = (rec & 0xffffffffull) | ((uint64_t)(ne + nx) << 32);
      }
    }
  }
}

// Per utterance: the frames' link offsets from their counts, the store's
// capacity check and the link totals.
__global__ void __launch_bounds__(kLT) k_links_offsets(const LaneDesc* __restrict__ lanes) {
  __shared__ BlockScratch bs;
  const LaneDesc& L = lanes[blockIdx.x];
  if (!links_wanted(L)) return;
  const uint32_t T1 = (uint32_t)L.T + 1;
  const uint32_t per = (T1 + kLT - 1) / kLT;
  const uint32_t f0 = threadIdx.x * per < T1 ? threadIdx.x * per : T1;
  const uint32_t f1 = f0 + per < T1 ? f0 + per : T1;
  uint64_t sum = 0;
  for (uint32_t t = f0; t < f1; ++t) sum += L.link_xoff[t] + L.link_end[t];
  uint32_t par = 0;
  uint64_t total;
  uint64_t base = block_excl_scan64<kLWv>(sum, bs, par, &total);
  for (uint32_t t = f0; t < f1; ++t) {
    const uint64_t ne = L.link_xoff[t], nx = L.link_end[t];
    L.link_off[t] = base;
    L.link_xoff[t] = base + ne;
    L.link_end[t] = base + ne + nx;
    base += ne + nx;
  }
  if (threadIdx.x == 0) {
    L.link_off[T1] = total;
    LaneInfo* I = L.info;
    I->links = total;
    I->need_links = total;
    if (total > L.link_cap) {
      I->overflow |= kOvfLinks;
      I->status = 4;  // WD_ECAPACITY
    }
  }
}

// Per frame: the links, at the frame's offsets; the frame's epsilon levels.
__global__ void __launch_bounds__(kLT) k_links_write(DevGraph g, const LaneDesc* __restrict__ lanes) {
  __shared__ LinkShared sh;
  const LaneDesc& L = lanes[blockIdx.y];
  if (!links_wanted(L)) return;
  uint32_t par = 0, bad = 0;
  for (int t = (int)blockIdx.x; t <= L.T; t += (int)gridDim.x) {
    const uint32_t cut = cost_key(L.cut[t]);
    uint32_t xmask = 0;
    if (t > 0) (void)link_run<false, true>(g, L, sh, par, t, cut, L.link_off[t], &xmask, &bad);
    (void)link_run<true, true>(g, L, sh, par, t, cut, L.link_xoff[t], &xmask, &bad);
    const uint32_t all = block_or<kLWv>(xmask, sh.bs, par);
    if (threadIdx.x == 0) L.xmask[t] = all;
  }
  if (bad) L.info->status = kStatusInternal;
}

void launch_links(const DevGraph& g, const LaneDesc* lanes, int B, hipStream_t s) {
  hipLaunchKernelGGL(k_links_count, dim3(kLinkBlocks, B), dim3(kLT), 0, s, g, lanes);
  hipLaunchKernelGGL(k_links_offsets, dim3(B), dim3(kLT), 0, s, lanes);
  hipLaunchKernelGGL(k_links_write, dim3(kLinkBlocks, B), dim3(kLT), 0, s, g, lanes);
}

}  // namespace wd
