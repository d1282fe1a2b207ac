// Chip-wide mode for utterances whose frames hold hundreds of thousands of
// tokens (wide beams, no max-active limit).
//
// The same per-frame steps as the one-workgroup forward pass (Sec. 3.2-3.4),
// each a kernel over 1024 workgroups per utterance, launched frame by frame on
// the caller's stream: emitting expansion with 64-bit atomicMin recombination
// on the per-state slot array (Alg. 1) over the prefix-sum work space of
// Sec. 3.3; one kernel per epsilon level; survivors of the beam cutoff with a
// global radix histogram for max-active; compaction in state order through the
// state bitmap; degree prefix sums; lattice links (Sec. 3.4).  Every position
// (frontier, links) comes from a two-level scan: per-workgroup sums, one
// workgroup scanning the sums, a per-workgroup rescan.  Frontier and link
// order are therefore the same as in the one-workgroup pass and the result is
// identical.  The backward pruning sweep of Sec. 3.5 has a chip-wide form too.
// Every kernel reads the frame's sizes from device memory, so the host never
// waits between frames; an utterance whose status is set skips the rest.
#include <mutex>

#include "wd_block.h"
#include "wd_host.h"
#include "../../include/wfstdec.h"

namespace wd {

constexpr int kGT = 256;          // threads per workgroup
constexpr int kGW = kGT / 64;     // wavefronts per workgroup
constexpr uint32_t kGB = 1024;    // workgroups per utterance
constexpr uint32_t kSeg = 4096;   // frontier prefix sums a workgroup keeps in LDS

// Incremental pruning runs in windows of this many frames, recorded in
// kSlots raw slots in turn; its sweep kernels use a quarter of the
// workgroups, leaving room for the decoding kernels.
constexpr int kPruneEvery = 32;
// A window is pruned kLookahead frames after its last frame (the sweep runs
// back from there), in one of kSlots raw slots.
constexpr int kLookahead = 8;
constexpr uint32_t kSlots = kLookahead < kPruneEvery ? 2u : 3u;
constexpr uint32_t kPB = kGB / 4;

// Incremental pruning state of one utterance, written only by the kernels on
// the pruning stream and, once the host has made the decoding stream wait for
// them, by the last window's gather.
struct PruneLane {
  uint64_t kend;      // links in the compacted region (still counted after an overflow)
  uint32_t go;        // the current window is pruned
  uint32_t ovf;       // the compacted region overflowed
  uint32_t next;      // first frame not yet pruned
  uint32_t pad0;
  unsigned long long part[kGB + 1];  // kept links per workgroup, then their prefix
};

// Per-utterance state carried from kernel to kernel.
struct GridLane {
  uint32_t stop;        // nonzero: skip every later kernel
  int32_t status;
  uint32_t ovf;
  uint32_t hist_ok;     // nodes and links still being stored
  uint32_t bad;         // a consistency check failed
  uint32_t frames;      // frames finished
  uint32_t W, n_prev, W_next, W_eps;
  uint32_t n_touched, n_surv, n_keep;
  uint32_t best_key, kcutb, cut_key;
  uint32_t best_pos;    // frontier position of a token with the frame's best cost
  uint32_t ub;          // cutoff prefilter bound of the frame being expanded (a key)
  uint32_t disp;        // dynamic load balancing: next frontier token to hand out
  uint32_t nbits, shift;
  uint32_t sel_active, sel_rank, sel_prefix, sel_less, sel_bits;
  uint32_t xmask;
  uint32_t final_used, best_total_key;
  unsigned long long best_total;  // (final cost key, node offset) of the best end token
  uint64_t node_base, node_base_prev, link_base;
  uint64_t arcs, eps_arcs, tokens, max_tokens, need_frame, need_arcs;
  uint64_t raw_total;              // links ever recorded
  uint64_t slot_lo, slot_hi;       // where links go: the whole store, or the window's slot
  uint64_t need_win;               // largest occupancy of the store (or of a slot)
  PruneLane pr;
  uint32_t nb[kMaxLevels + 1];
  uint32_t hist[kHistBins];
  // per-workgroup partial sums, then their exclusive prefix (+ total at kGB):
  // [0] frontier counts, [1] degree sums, [2] link counts, [3] kept links
  unsigned long long part[4][kGB + 1];
};

// ------------------------------------------------------- workgroup collectives

struct GScratch {
  unsigned long long w[kGW];
  unsigned long long w2[kGW][2];
  uint32_t u[4];
};

__device__ __forceinline__ unsigned long long gsum64(unsigned long long v, GScratch& s) {
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) v += shfl_xor64(v, m);
  __syncthreads();
  if (lane_id() == 0) s.w[wave_id()] = v;
  __syncthreads();
  unsigned long long r = 0;
#pragma unroll
  for (int i = 0; i < kGW; ++i) r += s.w[i];
  return r;
}

__device__ __forceinline__ unsigned long long gexcl64(unsigned long long v, GScratch& s,
                                                      unsigned long long* total) {
  const unsigned long long inc = wave_incl_scan64(v);
  __syncthreads();
  if (lane_id() == 63) s.w[wave_id()] = inc;
  __syncthreads();
  unsigned long long before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kGW; ++i) {
    before += (uint32_t)i < wave_id() ? s.w[i] : 0ull;
    tot += s.w[i];
  }
  *total = tot;
  return before + inc - v;
}

__device__ __forceinline__ unsigned long long gmin64(unsigned long long v, GScratch& s) {
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) {
    const unsigned long long o = shfl_xor64(v, m);
    v = o < v ? o : v;
  }
  __syncthreads();
  if (lane_id() == 0) s.w[wave_id()] = v;
  __syncthreads();
  unsigned long long r = s.w[0];
#pragma unroll
  for (int i = 1; i < kGW; ++i) r = s.w[i] < r ? s.w[i] : r;
  return r;
}

// [lo, hi) of workgroup b when n items are cut into kGB contiguous chunks.
__device__ __forceinline__ void chunk(uint64_t n, uint32_t b, uint64_t* lo, uint64_t* hi) {
  const uint64_t per = (n + kGB - 1) / kGB;
  const uint64_t a = (uint64_t)b * per;
  *lo = a < n ? a : n;
  *hi = a + per < n ? a + per : n;
}

// [lo, hi) of this thread inside the workgroup's [blo, bhi).
__device__ __forceinline__ void sub_chunk(uint64_t blo, uint64_t bhi, uint64_t* lo, uint64_t* hi) {
  const uint64_t n = bhi - blo, per = (n + kGT - 1) / kGT;
  const uint64_t a = (uint64_t)threadIdx.x * per;
  *lo = blo + (a < n ? a : n);
  *hi = blo + (a + per < n ? a + per : n);
}

// The frontier entries that own the work items [lo, hi) (lo < hi <= a[n]) of
// the exclusive prefix array a[0..n]: a[pl..pl+m), copied to LDS when it fits.
struct Seg {
  uint32_t pl, m;
  bool lds;
};

__device__ __forceinline__ Seg load_seg(const uint32_t* a, uint32_t n, uint32_t lo, uint32_t hi,
                                        uint32_t* seg, uint32_t* rng) {
  if (threadIdx.x < 2) rng[threadIdx.x] = search_le(a, n, threadIdx.x ? hi - 1u : lo);
  __syncthreads();
  Seg r;
  r.pl = rng[0];
  r.m = rng[1] - rng[0] + 1u;
  r.lds = r.m <= kSeg;
  if (r.lds)
    for (uint32_t i = threadIdx.x; i < r.m; i += kGT) seg[i] = a[r.pl + i];
  __syncthreads();
  return r;
}

__device__ __forceinline__ uint32_t seg_find(const Seg& sg, const uint32_t* seg, const uint32_t* a, uint32_t w) {
  return sg.pl + (sg.lds ? search_le(seg, sg.m, w) : search_le(a + sg.pl, sg.m, w));
}

// Exclusive scan of one utterance's kGB per-workgroup sums (+ total at kGB).
__device__ __forceinline__ void scan_parts(unsigned long long* part, GScratch& s) {
  constexpr uint32_t per = kGB / kGT;
  unsigned long long v[per], sum = 0;
#pragma unroll
  for (uint32_t i = 0; i < per; ++i) {
    v[i] = part[threadIdx.x * per + i];
    sum += v[i];
  }
  unsigned long long tot;
  unsigned long long ex = gexcl64(sum, s, &tot);
#pragma unroll
  for (uint32_t i = 0; i < per; ++i) {
    part[threadIdx.x * per + i] = ex;
    ex += v[i];
  }
  if (threadIdx.x == 0) part[kGB] = tot;
}

// Workgroup b's exclusive prefix among the kGB per-workgroup sums in part
// (as written by the kernel before: the consumer sums them itself rather
// than a separate one-workgroup scan launch) and their total.
__device__ __forceinline__ void part_prefix(const unsigned long long* part, uint32_t b, GScratch& s,
                                            unsigned long long* before, unsigned long long* total) {
  constexpr uint32_t per = kGB / kGT;
  unsigned long long lo = 0, all = 0;
#pragma unroll
  for (uint32_t i = 0; i < per; ++i) {
    const uint32_t j = threadIdx.x * per + i;
    const unsigned long long v = part[j];
    all += v;
    lo += j < b ? v : 0ull;
  }
  lo = wave_incl_scan64(lo);
  all = wave_incl_scan64(all);
  __syncthreads();
  if (lane_id() == 63) {
    s.w2[wave_id()][0] = lo;
    s.w2[wave_id()][1] = all;
  }
  __syncthreads();
  unsigned long long a = 0, c = 0;
#pragma unroll
  for (int i = 0; i < kGW; ++i) {
    a += s.w2[i][0];
    c += s.w2[i][1];
  }
  *before = a;
  *total = c;
}

// Exclusive scan of the kGB partial sums part[which] of each utterance
// (lattice != 0: after the forward pass has stopped, for utterances whose
// status is still WD_OK).
__global__ void __launch_bounds__(kGT) k_g_scan(const LaneDesc* __restrict__ lanes, GridLane* gl, int which,
                                                int lattice) {
  __shared__ GScratch s;
  GridLane& G = gl[blockIdx.y];
  if (lattice ? lanes[blockIdx.y].info->status != 0 : G.stop != 0) return;
  scan_parts(G.part[which], s);
}

// ---------------------------------------------------------------- forward pass

__global__ void k_g_init(const LaneDesc* __restrict__ lanes, GridLane* gl, const uint32_t* __restrict__ bad) {
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  uint32_t* w = reinterpret_cast<uint32_t*>(&G);
  for (uint32_t i = threadIdx.x; i < (uint32_t)(sizeof(GridLane) / 4); i += blockDim.x) w[i] = 0;
  __syncthreads();
  if (threadIdx.x == 0) {
    G.hist_ok = 1;
    // with incremental pruning, frames 0..31 go to the first window slot
    G.slot_lo = L.win_cap ? L.link_cap : 0;
    G.slot_hi = L.win_cap ? L.link_cap + L.win_cap : L.link_cap;
    G.link_base = G.slot_lo;
    if (bad[blockIdx.y]) {
      G.status = 1;  // WD_EINVAL
      G.stop = 1;
      lanes[blockIdx.y].info->status = 1;
    }
  }
}

// Frame 0: the start token.  One wavefront.
__global__ void k_g_begin(DevGraph g, const LaneDesc* __restrict__ lanes, GridLane* gl) {
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop || threadIdx.x != 0) return;
  const uint32_t s0 = g.start;
  L.slot[s0] = pack_tok(cost_key(0.0f), kNoArc);
  L.touched[0] = s0;
  G.n_touched = 1;
  const uint32_t c = g.sclass[s0];
  if (c != kNoEps) {
    L.bucket[g.level_base[c]] = s0;
    G.nb[c] = 1;
  }
  G.best_key = cost_key(0.0f);
}

// Start of the emitting expansion of frame t > 0, in every workgroup of the
// expansion kernel: the work capacity check (workgroup 0 records it and the
// frame's work) and the cutoff prefilter bound, which each workgroup
// computes for itself from the same inputs.  The bound (Sec. 4.3 prunes each
// transition against a beam as it is made): the best emitting candidate of
// one best token of frame t-1, plus the beam.  That candidate is one of all
// the frame's candidates, so the exact beam cutoff (best of all, plus the
// beam) is not above the bound, and a candidate above the bound can never
// survive or become a lattice link: expansion skips its recombination.
// Returns false when the frame does not fit (every workgroup stops).
__device__ __forceinline__ bool expand_begin(const DevGraph& g, const LaneDesc& L, GridLane& G, const Params& prm,
                                             int t, GScratch& s, uint32_t* ub) {
  const uint32_t W = G.W;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    G.need_arcs = W > G.need_arcs ? W : G.need_arcs;
    if (W > L.cand_cap) {
      G.status = 4;  // WD_ECAPACITY
      G.ovf |= kOvfArcs;
      G.stop = 1;
    } else {
      G.arcs += W;
    }
  }
  if (W > L.cand_cap) return false;
  if (threadIdx.x < 64u) {
    const uint32_t p = G.best_pos;
    uint32_t m = 0xffffffffu;
    if (p < G.n_prev) {
      const float c = key_cost(L.f_key[p]);
      const uint32_t a0 = L.f_ebeg[p], deg = L.f_edeg[p + 1] - L.f_edeg[p];
      const float* row = L.ll + (size_t)(t - 1) * g.P;
      for (uint32_t j = threadIdx.x; j < deg; j += 64) {
        const uint4 r = g.earc[a0 + j];
        const float ac = -row[(r.z & 0xffffffu) - 1u];
        float x = c + ac;
        x = canon(x + __uint_as_float(r.y));
        const uint32_t xk = cost_key(x);
        m = xk < m ? xk : m;
      }
    }
    m = lane63(wave_scan_op<uint32_t>(m, 0xffffffffu, [](uint32_t a, uint32_t b) { return b < a ? b : a; }));
    if (threadIdx.x == 0) s.u[0] = m < kInfKey ? cost_key(key_cost(m) + prm.beam) : 0xffffffffu;
  }
  __syncthreads();
  *ub = s.u[0];
  return true;
}

// First touches of a workgroup staged in LDS and published with one global
// reservation per list and round (touched states; the epsilon bucket of each
// level) instead of one atomic per wavefront or thread on a counter that every
// workgroup shares.  Entries that do not fit are appended directly.
constexpr uint32_t kStage = 1024;

template <uint32_t CAP>
struct TouchStageT {
  uint32_t nt, nbk, gt;
  uint32_t touched[CAP];
  uint32_t bk_state[CAP];
  uint32_t bk_tag[CAP];  // level << 16 | index among the level's staged entries
  uint32_t lcnt[kMaxLevels + 1];
  uint32_t lbase[kMaxLevels + 1];
};
using TouchStage = TouchStageT<kStage>;

template <uint32_t CAP>
__device__ __forceinline__ void stage_reset(TouchStageT<CAP>& ts, uint32_t nlevels) {
  for (uint32_t l = threadIdx.x; l < nlevels; l += kGT) ts.lcnt[l] = 0;
  if (threadIdx.x == 0) {
    ts.nt = 0;
    ts.nbk = 0;
  }
}

template <uint32_t CAP>
__device__ __forceinline__ void stage_touch(TouchStageT<CAP>& ts, GridLane& G, const LaneDesc& L, const DevGraph& g,
                                            uint32_t dst, uint32_t cls) {
  const uint32_t p = atomicAdd(&ts.nt, 1u);
  if (p < CAP) {
    ts.touched[p] = dst;
  } else {
    const uint32_t pos = atomicAdd(&G.n_touched, 1u);
    if (pos < L.frame_cap) L.touched[pos] = dst;
  }
  if (cls != kNoEps) {
    const uint32_t q = atomicAdd(&ts.nbk, 1u);
    if (q < CAP) {
      ts.bk_state[q] = dst;
      ts.bk_tag[q] = (cls << 16) | atomicAdd(&ts.lcnt[cls], 1u);
    } else {
      L.bucket[g.level_base[cls] + atomicAdd(&G.nb[cls], 1u)] = dst;
    }
  }
}

// Publishes the staged entries and empties the stage.  Whole workgroup.
template <uint32_t CAP>
__device__ __forceinline__ void stage_flush(TouchStageT<CAP>& ts, GridLane& G, const LaneDesc& L, const DevGraph& g) {
  __syncthreads();
  const uint32_t nt = ts.nt < CAP ? ts.nt : CAP, nbk = ts.nbk < CAP ? ts.nbk : CAP;
  if (threadIdx.x == 0 && nt) ts.gt = atomicAdd(&G.n_touched, nt);
  for (uint32_t l = threadIdx.x; l < g.nlevels; l += kGT)
    if (ts.lcnt[l]) ts.lbase[l] = atomicAdd(&G.nb[l], ts.lcnt[l]);
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < nt; i += kGT) {
    const uint32_t pos = ts.gt + i;
    if (pos < L.frame_cap) L.touched[pos] = ts.touched[i];
  }
  for (uint32_t i = threadIdx.x; i < nbk; i += kGT) {
    const uint32_t tag = ts.bk_tag[i], l = tag >> 16;
    L.bucket[g.level_base[l] + ts.lbase[l] + (tag & 0xffffu)] = ts.bk_state[i];
  }
  __syncthreads();
  stage_reset(ts, g.nlevels);
  __syncthreads();
}

// Emitting expansion of frame t: work item w is arc w - edeg[i] of frontier
// token i of frame t-1.  Writes the candidate of every work item.
__global__ void __launch_bounds__(kGT) k_g_expand(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                  GridLane* gl, Params prm, int t) {
  __shared__ GScratch s;
  __shared__ uint32_t seg[kSeg];
  __shared__ uint32_t rng[2];
  __shared__ TouchStage ts;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop || t == 0) return;
  uint32_t ub;
  if (!expand_begin(g, L, G, prm, t, s, &ub)) return;
  const uint32_t W = G.W, n_prev = G.n_prev;
  const uint64_t nbp = G.node_base_prev;
  const float* row = L.ll + (size_t)(t - 1) * g.P;
  uint64_t blo, bhi;
  chunk(W, blockIdx.x, &blo, &bhi);
  uint32_t my_best = 0xffffffffu;
  if (blo < bhi) {
    stage_reset(ts, g.nlevels);
    const Seg sg = load_seg(L.f_edeg, n_prev, (uint32_t)blo, (uint32_t)bhi, seg, rng);
    for (uint64_t r0 = blo; r0 < bhi; r0 += kStage) {
      const uint64_t r1 = r0 + kStage < bhi ? r0 + kStage : bhi;
      for (uint64_t base = r0; base < r1; base += kGT) {
        const uint32_t w = (uint32_t)base + threadIdx.x;
        if (w >= r1) continue;
        const uint32_t i = seg_find(sg, seg, L.f_edeg, w);
        const float c = key_cost(L.f_key[i]);
        const uint4 r = g.earc[L.f_ebeg[i] + (w - L.f_edeg[i])];
        const float ac = -row[(r.z & 0xffffffu) - 1u];
        float x = c + ac;
        x = canon(x + __uint_as_float(r.y));
        const uint32_t xk = cost_key(x);
        if (xk < kInfKey && xk <= ub) {
          const unsigned long long old = atomicMin(&L.slot[r.x], pack_tok(xk, r.w));
          my_best = xk < my_best ? xk : my_best;
          if (old == kEmpty) stage_touch(ts, G, L, g, r.x, r.z >> 24);
        }
        L.cand[w] = make_uint4(r.w, (uint32_t)(nbp + i), r.x, __float_as_uint(x));
      }
      stage_flush(ts, G, L, g);
    }
  }
  my_best = (uint32_t)gmin64(my_best, s);
  if (threadIdx.x == 0 && my_best != 0xffffffffu) atomicMin(&G.best_key, my_best);
}

// Dynamic load balancing (Alg. 2, Sec. 3.3), the A/B alternative to the
// prefix-sum work space above: a dispatcher counter hands out frontier tokens
// and a group of kDynGroup lanes expands all arcs of one token.  A wavefront
// takes kDynChunk tokens per dispatcher access: one access per token would
// serialise on the counter (same-address atomics measured at ~11.5 ns each on
// MI355X, against ~650k tokens per frame on the wide-beam workload).  Every
// candidate lands in the same work-item slot as with static balancing (its
// arc-id position), so the result is identical.
constexpr uint32_t kDynChunk = 256;
constexpr uint32_t kDynGroup = 8;
constexpr uint32_t kDynStage = 4096;

__global__ void __launch_bounds__(kGT) k_g_expand_dyn(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                      GridLane* gl, Params prm, int t) {
  __shared__ GScratch s;
  __shared__ TouchStageT<kDynStage> ts;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop || t == 0) return;
  uint32_t ub;
  if (!expand_begin(g, L, G, prm, t, s, &ub)) return;
  const uint32_t n_prev = G.n_prev;
  const uint64_t nbp = G.node_base_prev;
  const float* row = L.ll + (size_t)(t - 1) * g.P;
  stage_reset(ts, g.nlevels);
  __syncthreads();
  const uint32_t lane = lane_id(), grp = lane / kDynGroup, gln = lane % kDynGroup;
  constexpr uint32_t kGroups = 64 / kDynGroup;
  uint32_t my_best = 0xffffffffu;
  while (true) {
    uint32_t base = 0;
    if (lane == 0) base = atomicAdd(&G.disp, kDynChunk);
    base = __shfl(base, 0, 64);
    if (base >= n_prev) break;
    const uint32_t end = base + kDynChunk < n_prev ? base + kDynChunk : n_prev;
    for (uint32_t i = base + grp; i < end; i += kGroups) {
      const uint32_t w0 = L.f_edeg[i], deg = L.f_edeg[i + 1] - w0, a0 = L.f_ebeg[i];
      const float c = key_cost(L.f_key[i]);
      for (uint32_t j = gln; j < deg; j += kDynGroup) {
        const uint4 r = g.earc[a0 + j];
        const float ac = -row[(r.z & 0xffffffu) - 1u];
        float x = c + ac;
        x = canon(x + __uint_as_float(r.y));
        const uint32_t xk = cost_key(x);
        if (xk < kInfKey && xk <= ub) {
          const unsigned long long old = atomicMin(&L.slot[r.x], pack_tok(xk, r.w));
          my_best = xk < my_best ? xk : my_best;
          if (old == kEmpty) stage_touch(ts, G, L, g, r.x, r.z >> 24);
        }
        L.cand[w0 + j] = make_uint4(r.w, (uint32_t)(nbp + i), r.x, __float_as_uint(x));
      }
    }
  }
  stage_flush(ts, G, L, g);
  my_best = (uint32_t)gmin64(my_best, s);
  if (threadIdx.x == 0 && my_best != 0xffffffffu) atomicMin(&G.best_key, my_best);
}

// Epsilon closure, level `lvl`: states of that level within the cutoff relax
// their epsilon arcs; destinations sit on higher levels.  Per tile of bucket
// states the workgroup spreads the tile's arcs over its threads (a prefix sum
// of the states' epsilon degrees in LDS), so a state with many epsilon arcs
// does not serialise the kernel.  The tile is the smallest of 64, 128 and 256
// states that covers the level in one round of the grid: a level of a few
// thousand states then spreads over a hundred workgroups and more, each
// thread relaxing one or two arcs, instead of a few workgroups whose threads
// take several dependent arc-and-atomic round trips in turn (wide-beam frames:
// a frame 20 µs shorter; tiles of 32 states gain 4 µs less).
constexpr uint32_t kLvlMinTile = 64;

__global__ void __launch_bounds__(kGT) k_g_level(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                 GridLane* gl, Params prm, uint32_t lvl) {
  __shared__ GScratch s;
  __shared__ TouchStage ts;
  __shared__ uint32_t t_beg[kGT], t_ex[kGT], t_key[kGT];
  __shared__ uint32_t t_tot;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop) return;
  const uint32_t n = G.nb[lvl];
  uint32_t tile = kLvlMinTile;
  while (tile < (uint32_t)kGT && (uint64_t)tile * kGB < n) tile <<= 1;
  if (n == 0 || blockIdx.x * tile >= n) return;
  // beam cutoff from the best emitting candidate (inclusive); no candidate:
  // the survivor kernel reports it
  if (G.best_key >= kInfKey) return;
  const uint32_t kcutb = cost_key(key_cost(G.best_key) + prm.beam);
  const uint32_t* bk = L.bucket + g.level_base[lvl];
  stage_reset(ts, g.nlevels);
  unsigned long long eps = 0;
  for (uint32_t base = blockIdx.x * tile; base < n; base += kGB * tile) {
    const uint32_t i = base + threadIdx.x;
    uint32_t deg = 0, a0 = 0, k = 0;
    if (threadIdx.x < tile && i < n) {
      const uint32_t st = bk[i];
      // the state's epsilon arc range is loaded beside its token, not after
      // the cutoff test: one round trip instead of two
      const unsigned long long sv = L.slot[st];
      const uint32_t x0 = g.off[st].y, x1 = g.off[st + 1].y;
      k = (uint32_t)(sv >> 32);
      const bool live = k <= kcutb;  // (selects, so that the loads stay unconditional)
      a0 = live ? x0 : 0u;
      deg = live ? x1 - x0 : 0u;
    }
    uint32_t tot;
    if (tile <= 64u) {
      // the tile is one wavefront's: its scan needs no workgroup collective
      if (threadIdx.x < 64u) {
        const uint32_t inc = wave_incl_scan(deg);
        if (threadIdx.x < tile) {
          t_beg[threadIdx.x] = a0;
          t_ex[threadIdx.x] = inc - deg;
          t_key[threadIdx.x] = k;
        }
        if (threadIdx.x == 63u) t_tot = inc;
      }
      __syncthreads();
      tot = t_tot;
    } else {
      unsigned long long tt;
      const uint32_t ex = (uint32_t)gexcl64(deg, s, &tt);
      tot = (uint32_t)tt;
      if (threadIdx.x < tile) {
        t_beg[threadIdx.x] = a0;
        t_ex[threadIdx.x] = ex;
        t_key[threadIdx.x] = k;
      }
      __syncthreads();
    }
    eps += tot;
    for (uint32_t w = threadIdx.x; w < tot; w += kGT) {
      const uint32_t j = search_le(t_ex, tile, w);
      const uint4 r = g.xarc[t_beg[j] + (w - t_ex[j])];
      const uint32_t xk = cost_key(canon(key_cost(t_key[j]) + __uint_as_float(r.y)));
      if (xk > kcutb || xk >= kInfKey) continue;
      const unsigned long long old = atomicMin(&L.slot[r.x], pack_tok(xk, r.w));
      if (old == kEmpty) stage_touch(ts, G, L, g, r.x, r.z);
    }
    stage_flush(ts, G, L, g);
  }
  if (threadIdx.x == 0 && eps) atomicAdd((unsigned long long*)&G.eps_arcs, eps);
}

// A frame without max-active whose touched states are more than one in 32 of
// the graph's is dense: its survivors are found by one coalesced pass over
// the whole slot array (8 bytes per state) instead of a random slot read and
// a memory-side bitmap atomic per touched state.  Every kernel of the frame
// takes the same decision from the same values.
__device__ __forceinline__ bool dense_frame(const Params& prm, uint32_t nt, uint32_t S) {
  return prm.max_active == 0 && (uint64_t)nt * 32u > (uint64_t)S;
}

// Survivors of the beam cutoff; resets the touched slots; histogram of the
// top cost-key digit when max-active is on.  Costs never fall below the best
// emitting candidate (weights are >= 0), so the digit is in range.  Survivors
// and histogram counts are staged in LDS per workgroup.
__global__ void __launch_bounds__(kGT) k_g_count(DevGraph g, const LaneDesc* __restrict__ lanes, GridLane* gl,
                                                 Params prm) {
  __shared__ uint32_t n_st, gbase;
  __shared__ uint32_t st_state[kStage];
  __shared__ unsigned long long st_pack[kStage];
  __shared__ uint32_t hist[kHistBins];
  __shared__ GScratch s;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop) return;
  // After the closure: no candidate at all (no path), the frame capacity,
  // the beam cutoff and the digit layout of the histogram; every workgroup
  // takes them from the same values, workgroup 0 records them for the
  // kernels after this one.
  const uint32_t nt = G.n_touched, best = G.best_key;
  const bool nopath = best >= kInfKey, over = nt > L.frame_cap;
  const uint32_t kcutb = nopath ? 0u : cost_key(key_cost(best) + prm.beam);
  const uint32_t span = kcutb - best;
  const uint32_t nbits = span ? 32u - (uint32_t)__clz(span) : 0u;
  const uint32_t shift = nbits > 11u ? nbits - 11u : 0u;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    G.best_pos = 0xffffffffu;  // set again by this frame's compaction
    if (nopath) {
      G.status = 3;  // WD_ENOPATH
      G.stop = 1;
    } else {
      G.need_frame = nt > G.need_frame ? nt : G.need_frame;
      if (over) {
        G.status = 4;
        G.ovf |= kOvfFrame;
        G.stop = 1;
      } else {
        G.kcutb = kcutb;
        G.nbits = nbits;
        G.shift = shift;
      }
    }
  }
  if (nopath || over) return;
  if (prm.max_active == 0) {
    // dense frames: the state-bitmap kernel finds the survivors in the slot
    // array itself
    if (dense_frame(prm, nt, g.S)) return;
    // every survivor is kept: mark its state; its token stays in the slot,
    // where the compaction reads and resets it
    if (blockIdx.x * kGT >= nt) return;
    unsigned long long cnt = 0;
    for (uint32_t i = blockIdx.x * kGT + threadIdx.x; i < nt; i += kGB * kGT) {
      const uint32_t st = L.touched[i];
      if ((uint32_t)(L.slot[st] >> 32) <= kcutb) {
        atomicOr(&L.bitmap[st >> 5], 1u << (st & 31u));
        ++cnt;
      } else {
        L.slot[st] = kEmpty;
      }
    }
    cnt = gsum64(cnt, s);
    if (threadIdx.x == 0 && cnt) atomicAdd(&G.n_surv, (uint32_t)cnt);
    return;
  }
  if (blockIdx.x * kStage >= nt) return;
  const bool use_hist = true;
  if (use_hist)
    for (uint32_t i = threadIdx.x; i < (uint32_t)kHistBins; i += kGT) hist[i] = 0;
  if (threadIdx.x == 0) n_st = 0;
  __syncthreads();
  for (uint32_t r0 = blockIdx.x * kStage; r0 < nt; r0 += kGB * kStage) {
    const uint32_t r1 = r0 + kStage < nt ? r0 + kStage : nt;
    for (uint32_t i = r0 + threadIdx.x; i < r1; i += kGT) {
      const uint32_t st = L.touched[i];
      const unsigned long long v = L.slot[st];
      L.slot[st] = kEmpty;
      if ((uint32_t)(v >> 32) <= kcutb) {
        const uint32_t p = atomicAdd(&n_st, 1u);
        st_state[p] = st;
        st_pack[p] = v;
        if (use_hist) atomicAdd(&hist[((uint32_t)(v >> 32) - best) >> shift], 1u);
      }
    }
    __syncthreads();
    const uint32_t m = n_st;
    if (threadIdx.x == 0 && m) gbase = atomicAdd(&G.n_surv, m);
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < m; i += kGT) {
      L.surv_state[gbase + i] = st_state[i];
      L.surv_pack[gbase + i] = st_pack[i];
    }
    __syncthreads();
    if (threadIdx.x == 0) n_st = 0;
    __syncthreads();
  }
  if (use_hist)
    for (uint32_t i = threadIdx.x; i < (uint32_t)kHistBins; i += kGT)
      if (hist[i]) atomicAdd(&G.hist[i], hist[i]);
}

// Max-active by radix select: step 0 decides whether the limit binds; every
// step finds the histogram bin holding the rank-th smallest key and narrows
// the prefix by one digit (11, 11 and 10 bits at most).
__global__ void __launch_bounds__(kGT) k_g_select(GridLane* gl, Params prm, int step) {
  __shared__ GScratch s;
  __shared__ uint32_t sel[2];
  GridLane& G = gl[blockIdx.y];
  if (G.stop) return;
  if (step == 0) {
    if (threadIdx.x == 0) {
      const uint32_t ns = G.n_surv;
      G.cut_key = G.kcutb;
      G.n_keep = ns;
      G.sel_active = prm.max_active > 0 && ns > (uint32_t)prm.max_active;
      G.sel_rank = (uint32_t)prm.max_active;
      G.sel_prefix = 0;
      G.sel_less = 0;
      G.sel_bits = G.nbits - G.shift;
    }
    __syncthreads();
  }
  if (!G.sel_active) return;
  constexpr uint32_t per = kHistBins / kGT;
  uint32_t h[per], sum = 0;
#pragma unroll
  for (uint32_t i = 0; i < per; ++i) {
    h[i] = G.hist[threadIdx.x * per + i];
    sum += h[i];
  }
  unsigned long long tot;
  uint32_t ex = (uint32_t)gexcl64(sum, s, &tot);
  const uint32_t rank = G.sel_rank;
#pragma unroll
  for (uint32_t i = 0; i < per; ++i) {
    if (ex < rank && rank <= ex + h[i]) {
      sel[0] = threadIdx.x * per + i;
      sel[1] = ex;
    }
    ex += h[i];
  }
  __syncthreads();
  const uint32_t b = sel[0], before = sel[1], cnt = G.hist[b];
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < (uint32_t)kHistBins; i += kGT) G.hist[i] = 0;
  if (threadIdx.x == 0) {
    G.sel_prefix = (G.sel_prefix << G.sel_bits) | b;
    G.sel_less += before;
    G.sel_rank = rank - before;
    if (G.shift == 0) {
      const uint32_t vkey = G.best_key + G.sel_prefix;
      G.cut_key = vkey < G.kcutb ? vkey : G.kcutb;
      G.n_keep = G.sel_less + cnt;
      G.sel_active = 0;
    } else {
      const uint32_t nsh = G.shift > 11u ? G.shift - 11u : 0u;
      G.sel_bits = G.shift - nsh;
      G.shift = nsh;
    }
  }
}

// Histogram of the next digit over the survivors matching the prefix (per
// workgroup in LDS, then added to the utterance's histogram).
__global__ void __launch_bounds__(kGT) k_g_select_hist(const LaneDesc* __restrict__ lanes, GridLane* gl) {
  __shared__ uint32_t hist[kHistBins];
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop || !G.sel_active) return;
  const uint32_t ns = G.n_surv, best = G.best_key, prefix = G.sel_prefix, bits = G.sel_bits;
  const uint32_t nsh = G.shift, osh = nsh + bits;
  if (blockIdx.x * kGT >= ns) return;
  for (uint32_t i = threadIdx.x; i < (uint32_t)kHistBins; i += kGT) hist[i] = 0;
  __syncthreads();
  for (uint32_t i = blockIdx.x * kGT + threadIdx.x; i < ns; i += kGB * kGT) {
    const uint32_t d = (uint32_t)(L.surv_pack[i] >> 32) - best;
    if ((d >> osh) == prefix) atomicAdd(&hist[(d >> nsh) & ((1u << bits) - 1u)], 1u);
  }
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < (uint32_t)kHistBins; i += kGT)
    if (hist[i]) atomicAdd(&G.hist[i], hist[i]);
}

// Kept tokens mark their state in the bitmap; idx[state] = survivor index
// (max-active on; without it the survivor kernel marks them and the tokens
// stay in their slots).
__global__ void __launch_bounds__(kGT) k_g_mark(const LaneDesc* __restrict__ lanes, GridLane* gl) {
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop) return;
  const uint32_t ns = G.n_surv, cut = G.cut_key;
  for (uint32_t i = blockIdx.x * kGT + threadIdx.x; i < ns; i += kGB * kGT) {
    const unsigned long long v = L.surv_pack[i];
    if ((uint32_t)(v >> 32) <= cut) {
      const uint32_t st = L.surv_state[i];
      L.idx[st] = i;
      atomicOr(&L.bitmap[st >> 5], 1u << (st & 31u));
    }
  }
}

// Kept states per workgroup chunk of the bitmap; node capacity check.
__global__ void __launch_bounds__(kGT) k_g_bits(DevGraph g, const LaneDesc* __restrict__ lanes, GridLane* gl,
                                                Params prm) {
  __shared__ GScratch s;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop) return;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    // without max-active every survivor is kept (the select kernels set these
    // otherwise)
    if (prm.max_active == 0) {
      G.cut_key = G.kcutb;
      G.n_keep = G.n_surv;
    }
    const uint32_t n_keep = prm.max_active == 0 ? G.n_surv : G.n_keep;
    if (G.hist_ok && G.node_base + n_keep > L.node_cap) {
      G.hist_ok = 0;
      G.ovf |= kOvfNodes;
    }
  }
  uint64_t blo, bhi, lo, hi;
  chunk((g.S + 31u) >> 5, blockIdx.x, &blo, &bhi);
  unsigned long long c = 0;
  if (dense_frame(prm, G.n_touched, g.S)) {
    // the chunk's states in order, one per thread: a state survives when its
    // slot holds a token within the beam cutoff (other touched slots are
    // emptied here, the survivors' by the compaction); each half-wavefront's
    // ballot is one bitmap word, written whole
    const uint32_t kcutb = G.kcutb;
    const uint32_t s0 = (uint32_t)blo << 5, s1 = (uint32_t)bhi << 5;
    for (uint32_t base = s0; base < s1; base += kGT) {
      const uint32_t st = base + threadIdx.x;
      bool keep = false;
      if (st < s1 && st < g.S) {
        const unsigned long long v = L.slot[st];
        keep = (uint32_t)(v >> 32) <= kcutb;
        if (!keep && v != kEmpty) L.slot[st] = kEmpty;
      }
      const uint64_t m = __ballot(keep);
      const uint32_t half = lane_id() & 32u;
      if ((lane_id() & 31u) == 0 && base + (threadIdx.x & ~31u) < s1)
        L.bitmap[(base + (threadIdx.x & ~31u)) >> 5] = (uint32_t)(m >> half);
      if (lane_id() == 0) c += (uint32_t)__popcll(m);
    }
  } else {
    sub_chunk(blo, bhi, &lo, &hi);
    for (uint64_t w = lo; w < hi; ++w) c += (uint32_t)__popc(L.bitmap[w]);
  }
  c = gsum64(c, s);
  if (threadIdx.x == 0) G.part[0][blockIdx.x] = c;
}

// The frontier in state order: node store, frontier arrays, idx[state] = node
// id; per-workgroup (emitting, epsilon) out-degree sums of its frontier range.
// A workgroup takes its bitmap chunk 1024 words at a time into LDS with the
// words' exclusive bit counts, then one thread per state bit.
constexpr uint32_t kCW = 1024;

__global__ void __launch_bounds__(kGT) k_g_compact(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                   GridLane* gl, Params prm) {
  __shared__ GScratch s;
  __shared__ uint32_t wd[kCW], wp[kCW];
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop) return;
  uint64_t blo, bhi;
  chunk((g.S + 31u) >> 5, blockIdx.x, &blo, &bhi);
  unsigned long long pos0, n_all;
  part_prefix(G.part[0], blockIdx.x, s, &pos0, &n_all);
  const uint64_t nb = G.node_base;
  bool store = G.hist_ok != 0;
  if (dense_frame(prm, G.n_touched, g.S)) {
    // the survivors were counted by the bitmap kernel's workgroups: the
    // node capacity check and the frame's kept count happen here (every
    // workgroup decides alike; workgroup 0 records)
    const bool fits = nb + n_all <= L.node_cap;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      G.n_surv = (uint32_t)n_all;
      G.n_keep = (uint32_t)n_all;
      if (store && !fits) {
        G.hist_ok = 0;
        G.ovf |= kOvfNodes;
      }
    }
    store = store && fits;
  }
  const uint32_t best = G.best_key;
  const bool in_slot = prm.max_active == 0;  // the kept tokens are still in their slots
  unsigned long long deg = 0;
  constexpr uint32_t per = kCW / kGT;
  for (uint64_t r0 = blo; r0 < bhi; r0 += kCW) {
    const uint32_t m = (uint32_t)(bhi - r0 < kCW ? bhi - r0 : kCW);
    uint32_t c = 0;
#pragma unroll
    for (uint32_t j = 0; j < per; ++j) {
      const uint32_t q = threadIdx.x * per + j;
      uint32_t w = 0;
      if (q < m) {
        w = L.bitmap[r0 + q];
        if (w) L.bitmap[r0 + q] = 0;
      }
      wd[q] = w;
      wp[q] = c;
      c += (uint32_t)__popc(w);
    }
    unsigned long long tot;
    const uint32_t ex = (uint32_t)gexcl64(c, s, &tot);
#pragma unroll
    for (uint32_t j = 0; j < per; ++j) wp[threadIdx.x * per + j] += ex;
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < m * 32u; j += kGT) {
      const uint32_t word = wd[j >> 5], b = j & 31u;
      if (!((word >> b) & 1u)) continue;
      const uint64_t p = pos0 + wp[j >> 5] + (uint32_t)__popc(word & ((1u << b) - 1u));
      const uint32_t st = (uint32_t)((r0 << 5) + j);
      unsigned long long v;
      if (in_slot) {
        v = L.slot[st];
        L.slot[st] = kEmpty;
      } else {
        v = L.surv_pack[L.idx[st]];
      }
      const uint64_t node = nb + p;
      if (store) {
        L.n_state[node] = st;
        L.n_pack[node] = v;
        L.n_pred[node] = kNoArc;
      }
      L.idx[st] = (uint32_t)node;
      L.f_state[p] = st;
      L.f_key[p] = (uint32_t)(v >> 32);
      L.f_arc[p] = (uint32_t)v;
      if ((uint32_t)(v >> 32) == best) atomicMin(&G.best_pos, (uint32_t)p);
      // the token's arc ranges, its degrees for now (the degree kernel turns
      // them into prefix sums) and its epsilon level
      const uint4 o0 = g.off[st], o1 = g.off[st + 1];
      L.f_ebeg[p] = o0.x;
      L.f_xbeg[p] = o0.y;
      L.f_edeg[p] = o1.x - o0.x;
      L.f_xdeg[p] = o1.y - o0.y;
      L.f_cls[p] = g.sclass[st];
      deg += ((unsigned long long)(o1.y - o0.y) << 32) | (o1.x - o0.x);
    }
    pos0 += tot;
    __syncthreads();
  }
  deg = gsum64(deg, s);
  if (threadIdx.x == 0) G.part[1][blockIdx.x] = deg;
}

// Degree prefix sums of the frontier: each workgroup rescans the degrees of
// the frontier range it compacted.
__global__ void __launch_bounds__(kGT) k_g_degrees(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                   GridLane* gl) {
  __shared__ GScratch s;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop) return;
  unsigned long long blo, n_all, d_before, d_all;
  part_prefix(G.part[0], blockIdx.x, s, &blo, &n_all);
  part_prefix(G.part[1], blockIdx.x, s, &d_before, &d_all);
  const uint64_t bhi = blo + G.part[0][blockIdx.x];
  const uint32_t n = (uint32_t)n_all;
  uint64_t lo, hi;
  sub_chunk(blo, bhi, &lo, &hi);
  unsigned long long c = 0;
  for (uint64_t p = lo; p < hi; ++p) c += ((unsigned long long)L.f_xdeg[p] << 32) | L.f_edeg[p];
  unsigned long long tot;
  unsigned long long q = d_before + gexcl64(c, s, &tot);
  for (uint64_t p = lo; p < hi; ++p) {
    const unsigned long long d = ((unsigned long long)L.f_xdeg[p] << 32) | L.f_edeg[p];
    L.f_edeg[p] = (uint32_t)q;
    L.f_xdeg[p] = (uint32_t)(q >> 32);
    q += d;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const unsigned long long all = d_all;
    if (n != G.n_keep) G.bad = 1;
    G.W_next = (uint32_t)all;
    G.W_eps = (uint32_t)(all >> 32);
    L.f_edeg[n] = (uint32_t)all;
    L.f_xdeg[n] = (uint32_t)(all >> 32);
  }
}

// Lattice links of frame t over one item space: [0, W) the emitting
// candidates (arc-id order), [W, W + W_eps) the epsilon out-arcs of the
// frontier (arc-id order).  A link exists where the candidate is within the
// final cutoff.
struct LinkItem {
  uint32_t arc, src, dst, xbits, lvl;
};

__device__ __forceinline__ bool link_item(const DevGraph& g, const LaneDesc& L, uint32_t W, uint32_t cut,
                                          uint32_t it, const Seg& sg, const uint32_t* seg, LinkItem* o) {
  if (it < W) {
    const uint4 c = L.cand[it];
    const uint32_t xk = cost_key(__uint_as_float(c.w));
    *o = LinkItem{c.x, c.y, c.z, c.w, 0};
    return xk <= cut && xk < kInfKey;
  }
  const uint32_t e = it - W;
  const uint32_t p = seg_find(sg, seg, L.f_xdeg, e);
  const uint4 r = g.xarc[L.f_xbeg[p] + (e - L.f_xdeg[p])];
  const float x = canon(key_cost(L.f_key[p]) + __uint_as_float(r.y));
  const uint32_t xk = cost_key(x);
  *o = LinkItem{r.w, p, r.x, __float_as_uint(x), L.f_cls[p]};  // src: frontier position
  return xk <= cut && xk < kInfKey;
}

// Epsilon segment of a workgroup's item range [blo, bhi) (none below W).
__device__ __forceinline__ Seg link_seg(const LaneDesc& L, uint32_t W, uint32_t n, uint64_t blo, uint64_t bhi,
                                        uint32_t* seg, uint32_t* rng) {
  if (bhi <= W) return Seg{0, 0, true};
  const uint32_t e0 = (uint32_t)(blo > W ? blo - W : 0), e1 = (uint32_t)(bhi - W);
  return load_seg(L.f_xdeg, n, e0, e1, seg, rng);
}

__global__ void __launch_bounds__(kGT) k_g_link_count(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                      GridLane* gl, int t) {
  __shared__ GScratch s;
  __shared__ uint32_t seg[kSeg];
  __shared__ uint32_t rng[2];
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop) return;
  const uint32_t W = t > 0 ? G.W : 0, n = G.n_keep, cut = G.cut_key;
  uint64_t blo, bhi;
  chunk((uint64_t)W + G.W_eps, blockIdx.x, &blo, &bhi);
  unsigned long long c = 0;
  if (blo < bhi) {
    const Seg sg = link_seg(L, W, n, blo, bhi, seg, rng);
    for (uint64_t it = blo + threadIdx.x; it < bhi; it += kGT) {
      LinkItem o;
      if (link_item(g, L, W, cut, (uint32_t)it, sg, seg, &o)) c += it < W ? 1ull : (1ull << 32);
    }
  }
  c = gsum64(c, s);
  if (threadIdx.x == 0) G.part[2][blockIdx.x] = c;
}

// Writes the links in item order.  Items go kLinkBatch tiles of 256 at a time:
// every item's candidate or epsilon arc is read first, the tiles' (emitting,
// epsilon) flags are counted by wavefront ballots and one workgroup barrier,
// then the destinations' node ids and tokens are looked up for all items of
// the batch before the stores, so a thread has several independent chains of
// loads in flight instead of one per tile behind a workgroup scan.  Sets the
// predecessor node of each token from the link that produced it (same cost
// key and arc id).
constexpr uint32_t kLinkBatch = 4;

__global__ void __launch_bounds__(kGT) k_g_link_write(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                      GridLane* gl, int t) {
  __shared__ GScratch s;
  __shared__ uint32_t seg[kSeg];
  __shared__ uint32_t rng[2];
  __shared__ uint32_t wc[2][kLinkBatch][kGW][2];  // (batch parity, tile, wavefront): (emitting, epsilon) flags
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop) return;
  const uint32_t W = t > 0 ? G.W : 0, n = G.n_keep, cut = G.cut_key;
  unsigned long long run, all;
  part_prefix(G.part[2], blockIdx.x, s, &run, &all);
  const uint64_t nE = (uint32_t)all;
  const uint64_t lb = G.link_base, nb = G.node_base;
  if (!G.hist_ok || lb + nE + (all >> 32) > G.slot_hi) return;
  uint64_t blo, bhi;
  chunk((uint64_t)W + G.W_eps, blockIdx.x, &blo, &bhi);
  if (blo >= bhi) return;
  const Seg sg = link_seg(L, W, n, blo, bhi, seg, rng);
  uint32_t xm = 0, bad = 0, par = 0;
  uint32_t run_e = (uint32_t)run, run_x = (uint32_t)(run >> 32);
  for (uint64_t base = blo; base < bhi; base += kLinkBatch * kGT) {
    LinkItem o[kLinkBatch];
    bool on[kLinkBatch];
    uint64_t be[kLinkBatch], bx[kLinkBatch];
#pragma unroll
    for (uint32_t k = 0; k < kLinkBatch; ++k) {
      const uint64_t it = base + k * kGT + threadIdx.x;
      on[k] = it < bhi && link_item(g, L, W, cut, (uint32_t)it, sg, seg, &o[k]);
      be[k] = __ballot(on[k] && it < W);
      bx[k] = __ballot(on[k] && it >= W);
      if (lane_id() == 0) {
        wc[par][k][wave_id()][0] = (uint32_t)__popcll(be[k]);
        wc[par][k][wave_id()][1] = (uint32_t)__popcll(bx[k]);
      }
    }
    __syncthreads();  // (two count buffers: one barrier per batch)
    uint32_t pe[kLinkBatch], px[kLinkBatch], te = 0, tx = 0;
#pragma unroll
    for (uint32_t k = 0; k < kLinkBatch; ++k) {
      uint32_t ae = 0, ax = 0, se = 0, sx = 0;
#pragma unroll
      for (uint32_t i = 0; i < (uint32_t)kGW; ++i) {
        const uint32_t ce = wc[par][k][i][0], cx = wc[par][k][i][1];
        se += ce;
        sx += cx;
        ae += i < wave_id() ? ce : 0u;
        ax += i < wave_id() ? cx : 0u;
      }
      pe[k] = run_e + te + ae + rank_in(be[k]);
      px[k] = run_x + tx + ax + rank_in(bx[k]);
      te += se;
      tx += sx;
    }
    run_e += te;
    run_x += tx;
    par ^= 1u;
    uint32_t dn[kLinkBatch];
#pragma unroll
    for (uint32_t k = 0; k < kLinkBatch; ++k) dn[k] = on[k] ? L.idx[o[k].dst] : 0u;
    uint32_t fk[kLinkBatch], fa[kLinkBatch];
#pragma unroll
    for (uint32_t k = 0; k < kLinkBatch; ++k) {
      const uint32_t q = dn[k] - (uint32_t)nb;
      const bool ok = (uint64_t)dn[k] >= nb && q < n;
      if (on[k] && !ok) {
        bad = 1;
        on[k] = false;
      }
      fk[k] = on[k] ? L.f_key[q] : 0u;
      fa[k] = on[k] ? L.f_arc[q] : 0u;
    }
#pragma unroll
    for (uint32_t k = 0; k < kLinkBatch; ++k) {
      if (!on[k]) continue;
      const uint64_t it = base + k * kGT + threadIdx.x;
      const bool pred = fk[k] == cost_key(__uint_as_float(o[k].xbits)) && fa[k] == o[k].arc;
      if (it < W) {
        L.links[lb + pe[k]] = make_uint4(o[k].arc, o[k].src, dn[k], o[k].xbits);
        if (pred) L.n_pred[dn[k]] = o[k].src;
      } else {
        const uint64_t at = lb + nE + px[k];
        const uint32_t sn = (uint32_t)(nb + o[k].src);
        L.links[at] = make_uint4(o[k].arc, sn, dn[k], o[k].xbits);
        L.link_lvl[at] = (uint8_t)o[k].lvl;
        xm |= 1u << (o[k].lvl < 31u ? o[k].lvl : 31u);
        if (pred) L.n_pred[dn[k]] = sn;
      }
    }
  }
  if (xm) atomicOr(&G.xmask, xm);
  if (bad) atomicOr(&G.bad, 1u);
}

// End of frame t: per-frame records, counters, and the state of frame t+1.
__global__ void __launch_bounds__(kGT) k_g_end(const LaneDesc* __restrict__ lanes, GridLane* gl, int t) {
  __shared__ GScratch s;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (G.stop) return;
  unsigned long long none, all;
  part_prefix(G.part[2], 0, s, &none, &all);
  for (uint32_t i = threadIdx.x; i <= (uint32_t)kMaxLevels; i += kGT) G.nb[i] = 0;
  for (uint32_t i = threadIdx.x; i < (uint32_t)kHistBins; i += kGT) G.hist[i] = 0;
  if (threadIdx.x != 0) return;
  if (G.bad) {
    G.status = kStatusInternal;
    G.stop = 1;
    return;
  }
  const uint32_t n = G.n_keep;
  const uint64_t nE = (uint32_t)all, nX = all >> 32;
  const uint64_t end = G.link_base + nE + nX;
  G.raw_total += nE + nX;
  if (end - G.slot_lo > G.need_win) G.need_win = end - G.slot_lo;
  if (G.hist_ok && end > G.slot_hi) {
    G.hist_ok = 0;
    G.ovf |= kOvfLinks;
  }
  L.node_off[t] = G.node_base;
  L.node_off[t + 1] = G.node_base + n;
  L.link_off[t] = G.link_base;
  L.link_xoff[t] = G.link_base + nE;
  L.link_end[t] = end;
  L.link_off[t + 1] = end;
  L.xmask[t] = G.xmask;
  L.best[t] = key_cost(G.best_key);
  L.cutb[t] = key_cost(G.kcutb);
  L.cut[t] = key_cost(G.cut_key);
  G.tokens += n;
  G.max_tokens = n > G.max_tokens ? n : G.max_tokens;
  G.link_base = end;
  if (L.win_cap && (t + 1) % kPruneEvery == 0) {  // next window: the next slot
    G.slot_lo = L.link_cap + (((uint32_t)(t + 1) / kPruneEvery) % kSlots) * L.win_cap;
    G.slot_hi = G.slot_lo + L.win_cap;
    G.link_base = G.slot_lo;
  }
  G.node_base_prev = G.node_base;
  G.node_base += n;
  G.n_prev = n;
  G.W = G.W_next;
  G.n_touched = 0;
  G.n_surv = 0;
  G.xmask = 0;
  G.best_key = 0xffffffffu;  // the next frame's expansion takes the minimum
  G.disp = 0;
  G.frames = (uint32_t)t + 1u;
  if (t == L.T && !L.open) G.stop = 1;
}

// Final counters into the utterance's LaneInfo.
__global__ void k_g_finish(const LaneDesc* __restrict__ lanes, GridLane* gl) {
  const LaneDesc& L = lanes[blockIdx.y];
  const GridLane& G = gl[blockIdx.y];
  if (threadIdx.x != 0 || G.status == 1) return;
  LaneInfo* info = L.info;
  int32_t status = G.status;
  const uint32_t ovf = G.ovf | (G.pr.ovf ? (uint32_t)kOvfLinks : 0u);
  if (status == 0 && (ovf & (kOvfNodes | kOvfLinks))) status = 4;
  info->status = status;
  info->frames_done = (int32_t)G.frames;
  info->overflow = ovf;
  info->arcs_expanded = G.arcs + G.eps_arcs;
  info->eps_arcs = G.eps_arcs;
  info->tokens = G.tokens;
  info->max_tokens = G.max_tokens;
  info->links = G.raw_total;
  info->need_links = L.win_cap ? G.pr.kend : G.need_win;
  info->need_window = L.win_cap ? G.need_win : 0;
  info->need_frame_tokens = G.need_frame;
  info->need_frame_arcs = G.need_arcs;
}

// ------------------------------------------------------------- pruning sweep

// Whether a final state with a finite total cost was reached in the last frame.
__global__ void __launch_bounds__(kGT) k_gs_final_any(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                      GridLane* gl) {
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (L.info->status != 0) return;
  if (blockIdx.x == 0 && threadIdx.x == 0) G.best_total = kEmpty;
  if (!g.final_w) return;
  const uint64_t n0 = L.node_off[L.T], n1 = L.node_off[L.T + 1];
  bool any = false;
  for (uint64_t n = n0 + blockIdx.x * kGT + threadIdx.x; n < n1; n += (uint64_t)kGB * kGT) {
    const float fw = g.final_w[L.n_state[n]];
    const float c = key_cost((uint32_t)(L.n_pack[n] >> 32));
    any |= fw < INFINITY && (c + fw) < INFINITY;
  }
  if (__ballot(any) && lane_id() == 0) atomicOr(&G.final_used, 1u);
}

// The best final cost (lowest node on ties) of the last frame.
__global__ void __launch_bounds__(kGT) k_gs_final_min(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                      GridLane* gl) {
  __shared__ GScratch s;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (L.info->status != 0) return;
  const uint64_t n0 = L.node_off[L.T], n1 = L.node_off[L.T + 1];
  if (n0 + blockIdx.x * kGT >= n1) return;
  const bool any = G.final_used != 0;
  unsigned long long m = kEmpty;
  for (uint64_t n = n0 + blockIdx.x * kGT + threadIdx.x; n < n1; n += (uint64_t)kGB * kGT) {
    const float c = key_cost((uint32_t)(L.n_pack[n] >> 32));
    const float F = any ? canon(c + g.final_w[L.n_state[n]]) : c;
    const unsigned long long v = pack_tok(cost_key(F), (uint32_t)(n - n0));
    m = v < m ? v : m;
  }
  m = gmin64(m, s);
  if (threadIdx.x == 0) atomicMin(&G.best_total, m);
}

// Publishes the final-cost results for the lattice kernel.
__global__ void k_gs_final(const LaneDesc* __restrict__ lanes, GridLane* gl) {
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (threadIdx.x != 0 || L.info->status != 0) return;
  G.best_total_key = (uint32_t)(G.best_total >> 32);
  L.info->final_used = G.final_used ? 1 : 0;
  L.info->best_node = (uint32_t)(L.node_off[L.T] + (G.best_total & 0xffffffffu));
  L.info->best_cost = key_cost(G.best_total_key);
}

// Extra costs of all nodes before relaxation: the final extra cost for the
// last frame's nodes, +inf for the others.
__global__ void __launch_bounds__(kGT) k_gs_init(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                 const GridLane* gl) {
  const LaneDesc& L = lanes[blockIdx.y];
  const GridLane& G = gl[blockIdx.y];
  if (L.info->status != 0 || G.best_total_key >= kInfKey) return;
  const uint64_t nT = L.node_off[L.T], n1 = L.node_off[L.T + 1];
  const float best = key_cost(G.best_total_key);
  for (uint64_t n = (uint64_t)blockIdx.x * kGT + threadIdx.x; n < n1; n += (uint64_t)kGB * kGT) {
    uint32_t e = kInfKey;
    if (n >= nT) {
      const float c = key_cost((uint32_t)(L.n_pack[n] >> 32));
      const float F = G.final_used ? canon(c + g.final_w[L.n_state[n]]) : c;
      if (F < INFINITY) e = cost_key(F - best);
    }
    L.extra_key[n] = e;
  }
}

// Relaxes links into their source's extra cost: the emitting links that
// leave frame t (emit != 0), or frame t's epsilon links whose source is on
// level `lvl`.  extra(link) = extra(dst) + (x - cost(dst)).
// `prune`: the conservative sweep of incremental pruning, while decoding.
__global__ void __launch_bounds__(kGT) k_gs_relax(const LaneDesc* __restrict__ lanes, const GridLane* gl,
                                                  int t, int emit, int lvl, int prune) {
  const LaneDesc& L = lanes[blockIdx.y];
  const GridLane& G = gl[blockIdx.y];
  if (prune ? !G.pr.go : (L.info->status != 0 || t > L.T || G.best_total_key >= kInfKey)) return;
  uint64_t k0, k1;
  if (emit) {
    if (t == L.T) return;
    k0 = L.link_off[t + 1];
    k1 = L.link_xoff[t + 1];
  } else {
    if (((L.xmask[t] >> (lvl < 31 ? lvl : 31)) & 1u) == 0) return;
    k0 = L.link_xoff[t];
    k1 = L.link_end[t];
  }
  for (uint64_t k = k0 + blockIdx.x * kGT + threadIdx.x; k < k1; k += (uint64_t)gridDim.x * kGT) {
    if (!emit && L.link_lvl[k] != (uint8_t)lvl) continue;
    const uint4 v = L.links[k];
    const float exd = key_cost(L.extra_key[v.z]);
    const float c = key_cost((uint32_t)(L.n_pack[v.z] >> 32));
    const uint32_t le = cost_key(exd + (__uint_as_float(v.w) - c));
    L.le_key[k] = le;
    atomicMin(&L.extra_key[v.y], le);
  }
}

// Kept links (extra cost within the lattice beam) in link order: per-workgroup
// counts, then per 256-link tile a workgroup scan.  The count goes to the
// utterance's LaneInfo; the list is written only when it fits.
__device__ __forceinline__ bool kept_link(const LaneDesc& L, uint64_t k, uint32_t lb_key) {
  const uint32_t le = L.le_key[k];
  return le <= lb_key && le < kInfKey;
}

__global__ void __launch_bounds__(kGT) k_gk_count(const LaneDesc* __restrict__ lanes, GridLane* gl,
                                                  uint32_t lb_key) {
  __shared__ GScratch s;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (L.info->status != 0) return;
  uint64_t blo, bhi;
  chunk(L.link_off[L.T + 1], blockIdx.x, &blo, &bhi);
  unsigned long long c = 0;
  for (uint64_t k = blo + threadIdx.x; k < bhi; k += kGT) c += kept_link(L, k, lb_key);
  c = gsum64(c, s);
  if (threadIdx.x == 0) G.part[3][blockIdx.x] = c;
}

// Also writes each kept link's record for the forward-backward pass: {src
// node, dst node, the link's fp64 factor as two words (an epsilon link's with
// its source level in the low bits)}.
__global__ void __launch_bounds__(kGT) k_gk_write(DevGraph g, const LaneDesc* __restrict__ lanes, GridLane* gl,
                                                  uint32_t lb_key) {
  __shared__ GScratch s;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (L.info->status != 0) return;
  const uint64_t n_kept = G.part[3][kGB];
  if (blockIdx.x == 0 && threadIdx.x == 0) L.info->kept = n_kept;
  if (n_kept > L.kept_cap) return;
  uint64_t blo, bhi;
  chunk(L.link_off[L.T + 1], blockIdx.x, &blo, &bhi);
  unsigned long long run = G.part[3][blockIdx.x];
  for (uint64_t base = blo; base < bhi; base += kGT) {
    const uint64_t k = base + threadIdx.x;
    const bool on = k < bhi && kept_link(L, k, lb_key);
    unsigned long long tile;
    const unsigned long long ex = run + gexcl64(on ? 1ull : 0ull, s, &tile);
    run += tile;
    if (!on) continue;
    L.kept_idx[ex] = k;
    uint64_t lo = 0, hi = (uint64_t)L.T + 1;  // frame of link k: last t with link_off[t] <= k
    while (hi - lo > 1) {
      const uint64_t mid = (lo + hi) >> 1;
      if (L.link_off[mid] <= k) lo = mid;
      else hi = mid;
    }
    const uint4 v = L.links[k];
    const float w = g.weight_id[v.x];
    const bool eps = k >= L.link_xoff[lo];
    const double f = eps ? eps_factor(w)
                         : emit_factor(L.best[lo], L.best[lo - 1], w,
                                       -(double)L.ll[(size_t)(lo - 1) * g.P + (g.ilabel_id[v.x] - 1)]);
    const uint2 fb = factor_bits(f, eps, eps ? L.link_lvl[k] : 0u);
    L.post[ex] = make_uint4(v.y, v.z, fb.x, fb.y);
  }
}

// The linear-domain forward and backward sums of every node start at 0 (the
// lattice kernel then only adds into the nodes that kept links reach).
__global__ void __launch_bounds__(kGT) k_gs_fill_ab(const LaneDesc* __restrict__ lanes) {
  const LaneDesc& L = lanes[blockIdx.y];
  if (L.info->status != 0) return;
  const uint64_t n = L.node_off[L.T + 1];
  for (uint64_t i = (uint64_t)blockIdx.x * kGT + threadIdx.x; i < n; i += (uint64_t)kGB * kGT) {
    L.alpha[i] = 0.0;
    L.beta[i] = 0.0;
  }
  // per frame t: kept links start at kframe[2t], kept epsilon links at
  // kframe[2t+1] (the posterior passes' frame offsets); only when the list
  // was written
  const uint64_t nk = L.info->kept;
  if (nk > L.kept_cap) return;
  const int T = L.T;
  for (int t = (int)(blockIdx.x * kGT + threadIdx.x); t <= T + 1; t += kGB * kGT) {
    L.kframe[2 * t] = lower_bound64(L.kept_idx, nk, L.link_off[t]);
    L.kframe[2 * t + 1] = t <= T ? lower_bound64(L.kept_idx, nk, L.link_xoff[t]) : nk;
  }
}

// The lattice node list: nodes marked in the used bitmap, in node id order,
// which is (t, state) order.  Per-workgroup counts over bitmap chunks, a scan,
// then one thread per bit as in the frontier compaction.
__global__ void __launch_bounds__(kGT) k_gn_count(const LaneDesc* __restrict__ lanes, GridLane* gl) {
  __shared__ GScratch s;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (L.info->status != 0) return;
  uint64_t blo, bhi;
  chunk((L.node_off[L.T + 1] + 31) >> 5, blockIdx.x, &blo, &bhi);
  unsigned long long c = 0;
  for (uint64_t w = blo + threadIdx.x; w < bhi; w += kGT) c += (uint32_t)__popc(L.used[w]);
  c = gsum64(c, s);
  if (threadIdx.x == 0) G.part[0][blockIdx.x] = c;
}

__global__ void __launch_bounds__(kGT) k_gn_write(const LaneDesc* __restrict__ lanes, GridLane* gl) {
  __shared__ GScratch s;
  __shared__ uint32_t wd[kCW], wp[kCW];
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  LaneInfo* info = L.info;
  if (info->status != 0) return;
  if (blockIdx.x == 0 && threadIdx.x == 0) info->out_nodes = G.part[0][kGB];
  const uint64_t T2 = (uint64_t)L.T + 2;
  uint64_t blo, bhi;
  chunk((L.node_off[L.T + 1] + 31) >> 5, blockIdx.x, &blo, &bhi);
  uint64_t pos0 = G.part[0][blockIdx.x];
  constexpr uint32_t per = kCW / kGT;
  for (uint64_t r0 = blo; r0 < bhi; r0 += kCW) {
    const uint32_t m = (uint32_t)(bhi - r0 < kCW ? bhi - r0 : kCW);
    uint32_t c = 0;
#pragma unroll
    for (uint32_t j = 0; j < per; ++j) {
      const uint32_t q = threadIdx.x * per + j;
      const uint32_t w = q < m ? L.used[r0 + q] : 0u;
      wd[q] = w;
      wp[q] = c;
      c += (uint32_t)__popc(w);
    }
    unsigned long long tot;
    const uint32_t ex = (uint32_t)gexcl64(c, s, &tot);
#pragma unroll
    for (uint32_t j = 0; j < per; ++j) wp[threadIdx.x * per + j] += ex;
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < m * 32u; j += kGT) {
      const uint32_t word = wd[j >> 5], b = j & 31u;
      if (!((word >> b) & 1u)) continue;
      const uint64_t p = pos0 + wp[j >> 5] + (uint32_t)__popc(word & ((1u << b) - 1u));
      const uint64_t n = (r0 << 5) + j;
      // frame of node n: last t with node_off[t] <= n
      uint64_t lo = 0, hi = T2;
      while (hi - lo > 1) {
        const uint64_t mid = (lo + hi) >> 1;
        if (L.node_off[mid] <= n) lo = mid;
        else hi = mid;
      }
      OutNode o;
      o.t = (int32_t)lo;
      o.state = (int32_t)L.n_state[n];
      o.cost = key_cost((uint32_t)(L.n_pack[n] >> 32));
      o.extra = key_cost(L.extra_key[n]);
      L.out_nodes[p] = o;
    }
    pos0 += tot;
    __syncthreads();
  }
}

// ------------------------------------------------------ incremental pruning
//
// Frames are recorded in windows of kPruneEvery frames, window j in raw slot
// j mod kSlots of the link store.  Window j = [t0, t1] is pruned once frame
// tb = t1 + kLookahead is done too, by the pruning stream while decoding goes
// on: the nodes of frame tb get extra cost 0, the lowest an extra cost can
// be, and the sweep of Sec. 3.5 back from tb over window j then gives every
// node and link of window j a lower bound of its final extra cost (the
// recursion is monotone in the frame-tb values), one that already knows which
// paths die or fall behind within the kLookahead frames after the window.  A
// link of window j whose bound is above the lattice beam (or +inf: it leads
// nowhere) cannot be kept by the final pruning, and nothing it could decide
// survives either: a node's final extra cost is the minimum over its
// out-links, reached by a link within the beam whenever it matters.  Window
// j's other links are appended, in order, to the compacted region
// [0, link_cap), and its frame offsets move with them.  Decoding waits for
// window j's pruning only before window j + kSlots reuses its slot.  At the
// end, the frames after the last pruned window (at most two windows, the last
// of them partial) are gathered behind the compacted region, which then holds
// every frame in order, as the link store does without incremental pruning.
//
// Decoding and pruning touch disjoint data while they overlap: the window's
// links, link offsets, extra costs and le_key belong to the pruning stream;
// node offsets and costs of the window are final and only read.  The gate
// `go` is taken once per window from the decoding state: the window's frames
// are decoded (frames only grows), and status and hist_ok still say OK (they
// only ever change to a failure, whose result is not returned).

__global__ void k_gp_go(GridLane* gl, int t) {
  GridLane& G = gl[blockIdx.y];
  if (threadIdx.x != 0) return;
  const int32_t status = __hip_atomic_load(&G.status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t ok = __hip_atomic_load(&G.hist_ok, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t done = __hip_atomic_load(&G.frames, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  G.pr.go = ((uint32_t)t < done && status == 0 && ok) ? 1u : 0u;
}

__global__ void __launch_bounds__(kGT) k_gp_init(const LaneDesc* __restrict__ lanes, const GridLane* gl,
                                                 int t0, int t) {
  const LaneDesc& L = lanes[blockIdx.y];
  const GridLane& G = gl[blockIdx.y];
  if (!G.pr.go) return;
  const uint64_t n0 = L.node_off[t0], nt = L.node_off[t], n1 = L.node_off[t + 1];
  for (uint64_t n = n0 + (uint64_t)blockIdx.x * kGT + threadIdx.x; n < n1; n += (uint64_t)gridDim.x * kGT)
    L.extra_key[n] = n >= nt ? cost_key(0.0f) : kInfKey;
}

__device__ __forceinline__ bool gp_kept(const LaneDesc& L, uint64_t k, uint32_t lb_key) {
  const uint32_t le = L.le_key[k];
  return le <= lb_key && le < kInfKey;
}

__global__ void __launch_bounds__(kGT) k_gp_count(const LaneDesc* __restrict__ lanes, GridLane* gl, int t0,
                                                  int t, uint32_t lb_key) {
  __shared__ GScratch s;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (!G.pr.go) return;
  const uint64_t base = L.link_off[t0], end = L.link_end[t];
  uint64_t blo, bhi;
  chunk(end - base, blockIdx.x, &blo, &bhi);
  unsigned long long c = 0;
  for (uint64_t k = base + blo + threadIdx.x; k < base + bhi; k += kGT) c += gp_kept(L, k, lb_key);
  c = gsum64(c, s);
  if (threadIdx.x == 0) G.pr.part[blockIdx.x] = c;
}

__global__ void __launch_bounds__(kGT) k_gp_scan(GridLane* gl) {
  __shared__ GScratch s;
  GridLane& G = gl[blockIdx.y];
  if (!G.pr.go) return;
  scan_parts(G.pr.part, s);
}

// Kept links to the compacted region in order (when they fit); le_key[k] :=
// kept links of the window before k, for the offsets.
__global__ void __launch_bounds__(kGT) k_gp_write(const LaneDesc* __restrict__ lanes, GridLane* gl, int t0,
                                                  int t, uint32_t lb_key) {
  __shared__ GScratch s;
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (!G.pr.go) return;
  const uint64_t base = L.link_off[t0], end = L.link_end[t];
  const uint64_t k0 = G.pr.kend, nk = G.pr.part[kGB];
  const bool fits = !G.pr.ovf && k0 + nk <= L.link_cap;
  uint64_t blo, bhi;
  chunk(end - base, blockIdx.x, &blo, &bhi);
  unsigned long long run = G.pr.part[blockIdx.x];
  for (uint64_t b0 = base + blo; b0 < base + bhi; b0 += kGT) {
    const uint64_t k = b0 + threadIdx.x;
    const bool on = k < base + bhi && gp_kept(L, k, lb_key);
    unsigned long long tile;
    const unsigned long long ex = run + gexcl64(on ? 1ull : 0ull, s, &tile);
    run += tile;
    if (k >= base + bhi) continue;
    L.le_key[k] = (uint32_t)ex;
    if (on && fits) {
      L.links[k0 + ex] = L.links[k];
      L.link_lvl[k0 + ex] = L.link_lvl[k];
    }
  }
}

// The window's frame offsets in the compacted region, and its new end.
__global__ void __launch_bounds__(kGT) k_gp_fix(const LaneDesc* __restrict__ lanes, GridLane* gl, int t0, int t) {
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  if (!G.pr.go) return;
  const uint64_t end = L.link_end[t], k0 = G.pr.kend, nk = G.pr.part[kGB];
  __syncthreads();  // every thread has read link_end[t] before it moves
  auto moved = [&](uint64_t o) -> uint64_t { return k0 + (o < end ? (uint64_t)L.le_key[o] : nk); };
  for (int f = t0 + (int)threadIdx.x; f <= t; f += kGT) {
    L.link_off[f] = moved(L.link_off[f]);
    L.link_xoff[f] = moved(L.link_xoff[f]);
    L.link_end[f] = moved(L.link_end[f]);
  }
  if (threadIdx.x == 0) {
    if (k0 + nk > L.link_cap) G.pr.ovf = 1;
    G.pr.kend = k0 + nk;
    G.pr.next = (uint32_t)t + 1u;
  }
}

// The frames after the last pruned window (t0 .. T; none when it ended at
// T), behind the compacted region: frames t0 .. a1 of t0's window, then
// a1 + 1 .. T of the next one (empty when T ends t0's window), each
// contiguous in its slot.  On the decoding stream, after it has waited for
// the pruning stream.
struct Gather {
  int t0, a1;
  uint64_t srcA, nA, srcB, nB;
};

__device__ __forceinline__ bool gather_range(const LaneDesc& L, const GridLane& G, Gather* r) {
  if (!L.win_cap || G.status != 0 || !G.hist_ok) return false;
  const int t0 = (int)G.pr.next, T = L.T;
  r->t0 = t0;
  r->a1 = t0 + kPruneEvery - 1 < T ? t0 + kPruneEvery - 1 : T;
  r->srcA = t0 <= T ? L.link_off[t0] : 0;
  r->nA = t0 <= T ? L.link_end[r->a1] - r->srcA : 0;
  r->srcB = r->a1 < T ? L.link_off[r->a1 + 1] : 0;
  r->nB = r->a1 < T ? L.link_end[T] - r->srcB : 0;
  return true;
}

__global__ void __launch_bounds__(kGT) k_gp_gather(const LaneDesc* __restrict__ lanes, const GridLane* gl) {
  const LaneDesc& L = lanes[blockIdx.y];
  const GridLane& G = gl[blockIdx.y];
  Gather r;
  if (!gather_range(L, G, &r)) return;
  const uint64_t k0 = G.pr.kend, n = r.nA + r.nB;
  if (G.pr.ovf || k0 + n > L.link_cap) return;
  for (uint64_t i = (uint64_t)blockIdx.x * kGT + threadIdx.x; i < n; i += (uint64_t)kGB * kGT) {
    const uint64_t src = i < r.nA ? r.srcA + i : r.srcB + (i - r.nA);
    L.links[k0 + i] = L.links[src];
    L.link_lvl[k0 + i] = L.link_lvl[src];
  }
}

__global__ void __launch_bounds__(kGT) k_gp_gather_fix(const LaneDesc* __restrict__ lanes, GridLane* gl) {
  const LaneDesc& L = lanes[blockIdx.y];
  GridLane& G = gl[blockIdx.y];
  Gather r;
  if (!gather_range(L, G, &r)) return;
  const uint64_t k0 = G.pr.kend, n = r.nA + r.nB;
  const bool fits = !G.pr.ovf && k0 + n <= L.link_cap;
  __syncthreads();  // every thread has read the offsets before they move
  if (fits)
    for (int f = r.t0 + (int)threadIdx.x; f <= L.T; f += kGT) {
      const uint64_t dst = f <= r.a1 ? k0 - r.srcA : k0 + r.nA - r.srcB;  // (mod 2^64)
      L.link_off[f] = L.link_off[f] + dst;
      L.link_xoff[f] = L.link_xoff[f] + dst;
      L.link_end[f] = L.link_end[f] + dst;
    }
  if (threadIdx.x == 0) {
    if (fits) L.link_off[L.T + 1] = k0 + n;
    else G.pr.ovf = 1;
    G.pr.kend = k0 + n;
  }
}

// -------------------------------------------------------------------- launches

size_t grid_lane_bytes() { return sizeof(GridLane); }

uint32_t grid_window_slots() { return kSlots; }

// Decoding-state update for a stream's utterances: a workgroup per lane.
__global__ void k_g_bad(const LaneDesc* __restrict__ lanes, GridLane* gl, const uint32_t* __restrict__ bad) {
  GridLane& G = gl[blockIdx.y];
  if (threadIdx.x != 0 || !bad[blockIdx.y] || G.status != 0) return;
  G.status = 1;  // WD_EINVAL
  G.stop = 1;
  lanes[blockIdx.y].info->status = 1;
}

namespace {

// The library's pruning stream of each device (default priority, never
// blocking on the null stream).
hipError_t prune_stream(hipStream_t* out) {
  static std::mutex create;
  static hipStream_t per_dev[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(create);
  if (!per_dev[dev]) {
    hipStream_t q = nullptr;
    if ((e = hipStreamCreateWithFlags(&q, hipStreamNonBlocking)) != hipSuccess) return e;
    per_dev[dev] = q;
  }
  *out = per_dev[dev];
  return hipSuccess;
}

}  // namespace

void grid_release(GridRun* run) {
  // a run that did not reach grid_end may still have windows being pruned
  if (run->q && !run->ended && run->nwin > 0) (void)hipStreamSynchronize(run->q);
  for (int i = 0; i < 4; ++i) {
    if (run->ready[i]) (void)hipEventDestroy(run->ready[i]);
    if (run->done[i]) (void)hipEventDestroy(run->done[i]);
    run->ready[i] = run->done[i] = nullptr;
  }
  run->q = nullptr;
}

wd_status grid_begin(GridRun* run, const LaneDesc* lanes, void* glv, int B, bool prune, const uint32_t* bad,
                     hipStream_t st) {
  *run = GridRun{};
  if (prune) {
    hipError_t e = prune_stream(&run->q);
    for (int i = 0; i < 4 && e == hipSuccess; ++i) {
      e = hipEventCreateWithFlags(&run->ready[i], hipEventDisableTiming);
      if (e == hipSuccess) e = hipEventCreateWithFlags(&run->done[i], hipEventDisableTiming);
    }
    if (e != hipSuccess) {
      grid_release(run);
      return hip_check(e, "pruning stream");
    }
  }
  hipLaunchKernelGGL(k_g_init, dim3(1, B), dim3(kGT), 0, st, lanes, (GridLane*)glv, bad);
  return WD_OK;
}

// Frames t_from..t_to.  Window u's links go to slot u % kSlots: the first
// frame of window u waits for the pruning of window u - kSlots; kLookahead
// frames after the last frame of window j, an event hands window j to the
// pruning stream (ready[j % 4] / done[j % 4]; every wait is enqueued before
// its event is recorded again).
wd_status grid_frames(GridRun* run, const DevGraph& g, const LaneDesc* lanes, void* glv, int B, const Params& prm,
                      const uint32_t* bad, int t_from, int t_to, hipStream_t st) {
  GridLane* gl = (GridLane*)glv;
  const dim3 one(1, B), all(kGB, B), part(kPB, B), blk(kGT);
  const uint32_t lb_key = cost_key(prm.lattice_beam);
  hipError_t e = hipSuccess;
  hipLaunchKernelGGL(k_g_bad, one, dim3(64), 0, st, lanes, gl, bad);
  for (int t = t_from; t <= t_to && e == hipSuccess; ++t) {
    const int reuse = t / kPruneEvery - (int)kSlots;
    if (run->q && t % kPruneEvery == 0 && reuse >= 0 && reuse < run->nwin)
      e = hipStreamWaitEvent(st, run->done[reuse % 4], 0);
    // per frame: expansion (with the frame's start), epsilon levels,
    // survivors (with the cutoff and capacity checks), [max-active select],
    // kept-state counts, compaction, degrees, link counts, links, end
    if (t == 0) hipLaunchKernelGGL(k_g_begin, one, dim3(64), 0, st, g, lanes, gl);
    if (prm.flags & WD_FLAG_DYNAMIC_LB) hipLaunchKernelGGL(k_g_expand_dyn, all, blk, 0, st, g, lanes, gl, prm, t);
    else hipLaunchKernelGGL(k_g_expand, all, blk, 0, st, g, lanes, gl, prm, t);
    for (uint32_t l = 0; l < g.nlevels; ++l) hipLaunchKernelGGL(k_g_level, all, blk, 0, st, g, lanes, gl, prm, l);
    hipLaunchKernelGGL(k_g_count, all, blk, 0, st, g, lanes, gl, prm);
    if (prm.max_active > 0) {
      hipLaunchKernelGGL(k_g_select, one, blk, 0, st, gl, prm, 0);
      for (int step = 1; step < 3; ++step) {
        hipLaunchKernelGGL(k_g_select_hist, all, blk, 0, st, lanes, gl);
        hipLaunchKernelGGL(k_g_select, one, blk, 0, st, gl, prm, step);
      }
      hipLaunchKernelGGL(k_g_mark, all, blk, 0, st, lanes, gl);
    }
    hipLaunchKernelGGL(k_g_bits, all, blk, 0, st, g, lanes, gl, prm);
    hipLaunchKernelGGL(k_g_compact, all, blk, 0, st, g, lanes, gl, prm);
    hipLaunchKernelGGL(k_g_degrees, all, blk, 0, st, g, lanes, gl);
    hipLaunchKernelGGL(k_g_link_count, all, blk, 0, st, g, lanes, gl, t);
    hipLaunchKernelGGL(k_g_link_write, all, blk, 0, st, g, lanes, gl, t);
    hipLaunchKernelGGL(k_g_end, one, blk, 0, st, lanes, gl, t);
    if (run->q && (t + 1 - kLookahead) % kPruneEvery == 0 && t + 1 - kLookahead >= kPruneEvery) {
      // window j = [t0, t1] against frame t, kLookahead frames after it
      const int t1 = t - kLookahead, t0 = t1 + 1 - kPruneEvery, j = run->nwin++;
      hipStream_t q = run->q;
      e = hipEventRecord(run->ready[j % 4], st);
      if (e == hipSuccess) e = hipStreamWaitEvent(q, run->ready[j % 4], 0);
      if (e != hipSuccess) break;
      hipLaunchKernelGGL(k_gp_go, one, dim3(64), 0, q, gl, t);
      hipLaunchKernelGGL(k_gp_init, part, blk, 0, q, lanes, gl, t0, t);
      // frame f: the emitting links leaving it, then its epsilon levels; down
      // to f = t0 - 1 for the emitting links into t0 (the window's first run;
      // the extra costs this leaves on frame t0 - 1 are never read)
      for (int f = t; f >= t0 - 1 && f >= 0; --f) {
        if (f < t) hipLaunchKernelGGL(k_gs_relax, part, blk, 0, q, lanes, gl, f, 1, 0, 1);
        if (f >= t0)
          for (int l = (int)g.nlevels - 1; l >= 0; --l)
            hipLaunchKernelGGL(k_gs_relax, part, blk, 0, q, lanes, gl, f, 0, l, 1);
      }
      hipLaunchKernelGGL(k_gp_count, all, blk, 0, q, lanes, gl, t0, t1, lb_key);
      hipLaunchKernelGGL(k_gp_scan, one, blk, 0, q, gl);
      hipLaunchKernelGGL(k_gp_write, all, blk, 0, q, lanes, gl, t0, t1, lb_key);
      hipLaunchKernelGGL(k_gp_fix, one, blk, 0, q, lanes, gl, t0, t1);
      e = hipEventRecord(run->done[j % 4], q);
    }
  }
  return hip_check(e, "pruning stream");
}

// After the last frame: wait for the pruning stream, gather the frames after
// the last pruned window, final counters.
wd_status grid_end(GridRun* run, const LaneDesc* lanes, void* glv, int B, hipStream_t st) {
  GridLane* gl = (GridLane*)glv;
  const dim3 one(1, B), all(kGB, B), blk(kGT);
  hipError_t e = hipSuccess;
  if (run->q) {
    if (run->nwin > 0) e = hipStreamWaitEvent(st, run->done[(run->nwin - 1) % 4], 0);
    hipLaunchKernelGGL(k_gp_gather, all, blk, 0, st, lanes, gl);
    hipLaunchKernelGGL(k_gp_gather_fix, one, blk, 0, st, lanes, gl);
  }
  hipLaunchKernelGGL(k_g_finish, one, dim3(64), 0, st, lanes, gl);
  run->ended = e == hipSuccess;
  return hip_check(e, "pruning stream");
}

void launch_grid_nodes(const LaneDesc* lanes, void* glv, int B, hipStream_t st) {
  GridLane* gl = (GridLane*)glv;
  const dim3 one(1, B), all(kGB, B), blk(kGT);
  hipLaunchKernelGGL(k_gn_count, all, blk, 0, st, lanes, gl);
  hipLaunchKernelGGL(k_g_scan, one, blk, 0, st, lanes, gl, 0, 1);
  hipLaunchKernelGGL(k_gn_write, all, blk, 0, st, lanes, gl);
}

void launch_grid_sweep(const DevGraph& g, const LaneDesc* lanes, void* glv, int B, int maxT, float lattice_beam,
                       hipStream_t st) {
  GridLane* gl = (GridLane*)glv;
  const dim3 one(1, B), all(kGB, B), blk(kGT);
  hipLaunchKernelGGL(k_gs_final_any, all, blk, 0, st, g, lanes, gl);
  hipLaunchKernelGGL(k_gs_final_min, all, blk, 0, st, g, lanes, gl);
  hipLaunchKernelGGL(k_gs_final, one, dim3(64), 0, st, lanes, gl);
  hipLaunchKernelGGL(k_gs_init, all, blk, 0, st, g, lanes, gl);
  for (int t = maxT; t >= 0; --t) {
    hipLaunchKernelGGL(k_gs_relax, all, blk, 0, st, lanes, gl, t, 1, 0, 0);
    for (int l = (int)g.nlevels - 1; l >= 0; --l)
      hipLaunchKernelGGL(k_gs_relax, all, blk, 0, st, lanes, gl, t, 0, l, 0);
  }
  const uint32_t lb_key = cost_key(lattice_beam);
  hipLaunchKernelGGL(k_gk_count, all, blk, 0, st, lanes, gl, lb_key);
  hipLaunchKernelGGL(k_g_scan, one, blk, 0, st, lanes, gl, 3, 1);
  hipLaunchKernelGGL(k_gk_write, all, blk, 0, st, g, lanes, gl, lb_key);
  hipLaunchKernelGGL(k_gs_fill_ab, all, blk, 0, st, lanes);
}

}  // namespace wd
