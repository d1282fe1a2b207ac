// Lattice pass for one utterance per workgroup, after the forward pass.
//
// Final costs and the best end token; lattice pruning (Sec. 3.5): the extra
// cost of a node is the best complete path through it minus the best overall,
// of a link extra(dst) + (x - cost(dst)); nodes are updated with atomic
// minima on order-preserving keys, sweeping frames from the last one back (links
// only run from frame t to t or t+1) and, inside a frame, epsilon links from the
// highest source level down, so every value is final when it is read.  The
// 1-best path is traced back during the same sweep.  Then fp64 forward-backward
// posteriors over the kept links (Sec. 4.1 uses lattice posteriors) and the
// final merge of the kept links (Sec. 3.5) in (t, arc id) order.
#include "wd_block.h"

namespace wd {

constexpr uint32_t kWin = 4096;  // nodes of one frame held in LDS
// The lattice pass is a chain of small per-frame steps: 512 threads (8
// wavefronts, up to 256 VGPRs each) hold a frame's inputs loaded a frame
// ahead in registers and meet at cheaper barriers than 1024 would.
constexpr int kLT = 512;
constexpr int kLW = kLT / 64;

// Two-frame window of per-node values (frame t and t+1, or t-1 and t): extra
// costs and costs during the pruning sweep, alpha or beta during the
// posteriors.  Frames with more nodes use the workspace arrays directly.
// Small kept lattices (the usual case at a narrow lattice beam: a few kept
// links per frame) run their forward-backward sums entirely in LDS over the
// nodes the kept links touch, renumbered 0..K-1 (compact posteriors below).
constexpr uint32_t kCpNodes = 3584;   // touched nodes
constexpr uint32_t kCpLinks = 2560;   // kept links
constexpr uint32_t kCpFrames = 2048;  // frames + 1
constexpr uint32_t kCpWords = 2 * kCpNodes;  // node bitmap words (the bitmap in a, word ranks in b)
// Frames (+ 1) whose offsets the final merge and the node list read from LDS.
constexpr uint32_t kMgFrames = 2048;
// Staged pruning sweep: blocks of up to kSwK frames; rings of kSwRing links
// and nodes in LDS hold four blocks (one written back, one swept, one
// loaded, one loading), so a block may hold at most kSwRing / 4 of each.
constexpr int kSwK = 4;
constexpr uint32_t kSwRing = 4096;
constexpr uint32_t kSwCap = kSwRing / 4;
constexpr int kSwFrames = 4 * kSwK;  // per-frame table entries (a ring of frames)

struct LatShared {
  BlockScratch bs;
  union {
    struct {
      uint32_t ex[3][kWin];  // three frames: t+1 (read), t (relaxed), t-1 (being initialised)
      float cost[3][kWin];
    } p;
    struct {
      double a[2][kWin];  // alpha (wavefront 0)
      double b[2][kWin];  // beta (wavefront 1, concurrently)
    } ab;
    struct {
      // alpha and beta sums of the touched nodes; before them, the bitmap of
      // touched node ids (in a) and each bitmap word's rank (in b)
      double a[kCpNodes];
      double b[kCpNodes];
      uint4 link[kCpLinks];         // kept link records, source and destination renumbered
      uint32_t node[kCpNodes];      // node id of each compact number
      uint16_t kf[2 * kCpFrames];   // per-frame kept-link boundaries
      uint32_t lmask[kCpFrames];    // source levels of each frame's kept epsilon links
    } cp;
    struct {
      uint32_t sd[kSwRing];      // link: source | destination << 16, both as node ring positions
      float dl[kSwRing];         // link: forward cost minus its destination's cost
      uint8_t lvl[kSwRing];      // link: source level (epsilon links)
      uint32_t ex[kSwRing];      // node: extra-cost key
      uint32_t fm[kSwFrames];    // frame: source levels of its epsilon links
      // per frame u (u <= T; relative to frame 0's first epsilon link and first
      // node): first epsilon link, first emitting link out of it, one past its
      // last link, first node (u = T + 1: one past the last)
      uint32_t ox[kMgFrames], oe[kMgFrames], oz[kMgFrames], on[kMgFrames];
      int32_t top[kMgFrames];    // block b's highest frame (then -1)
      int32_t nblk;              // blocks (-1: a frame does not fit)
    } sw;
    struct {
      // per-frame offsets for the final merge and the node list
      uint64_t node_off[kMgFrames], link_off[kMgFrames], link_xoff[kMgFrames];
      uint64_t kf[2 * kMgFrames];
    } mg;
  } w;
};

__device__ __forceinline__ uint64_t search_le64(const uint64_t* a, uint64_t n, uint64_t w) {
  uint64_t lo = 0, hi = n;
  while (hi - lo > 1) {
    uint64_t mid = (lo + hi) >> 1;
    if (a[mid] <= w) lo = mid;
    else hi = mid;
  }
  return lo;
}


// Mass v moved into a node's linear-domain sum (the factor helpers beside
// cost_key define the sums): LDS windows add with the LDS unit's fp64 add,
// device-memory frames with the memory-side one.
__device__ __forceinline__ void mass_add(double* p, double v, bool lds) {
  if (!(v > 0.0)) return;
  if (lds) atomicAdd(p, v);
  else unsafeAtomicAdd(p, v);
}

__device__ __forceinline__ float node_cost(const LaneDesc& L, uint64_t n) {
  return key_cost((uint32_t)(L.n_pack[n] >> 32));
}

// The kept lattice's total cost Z = beta(start) = B - b(0) - log Sb(start),
// and the posteriors' normaliser: posterior = Sa(src) Sb(dst) factor
// exp(-b(0)) / Sb(start).
__device__ __forceinline__ double lattice_z(const LaneDesc& L, float best_total, uint64_t start_node) {
  return (double)best_total - (double)L.best[0] - log(L.beta[start_node]);
}
__device__ __forceinline__ double post_norm(const LaneDesc& L, uint64_t start_node) {
  return exp(-(double)L.best[0]) / L.beta[start_node];
}

// Node id of the start token: the start state among frame 0's tokens (sorted
// by state).
__device__ __forceinline__ uint64_t start_node_of(const LaneDesc& L, const DevGraph& g) {
  uint64_t lo = 0, hi = L.node_off[1];
  while (lo < hi) {
    const uint64_t mid = (lo + hi) >> 1;
    if (L.n_state[mid] < g.start) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

struct LinkView {
  uint32_t arc, src, dst;
  float x;
};
__device__ __forceinline__ LinkView link_at(const LaneDesc& L, uint64_t k) {
  const uint4 v = L.links[k];
  return LinkView{v.x, v.y, v.z, __uint_as_float(v.w)};
}

__device__ __forceinline__ bool kept(const LaneDesc& L, uint64_t k, uint32_t lb_key) {
  const uint32_t le = L.le_key[k];
  return le <= lb_key && le < kInfKey;
}

__device__ __forceinline__ double link_ac(const LaneDesc& L, const DevGraph& g, int t, uint32_t arc) {
  const int32_t il = g.ilabel_id[arc];
  return il ? -(double)L.ll[(size_t)(t - 1) * g.P + (il - 1)] : 0.0;
}

// Write the selected links (all links, or the kept ones listed in kept_idx)
// in (t, arc id) order.  Each frame holds an emitting run then an epsilon run,
// each already ascending in arc id; a link's slot is its rank in its own run
// plus the number of links of the other run with a smaller arc id.  The runs'
// bounds in selection order are the frame's link offsets (all links) or the
// per-frame kept-link boundaries kf.
// lo, xo, kf: the frame offsets (link_off, link_xoff, kframe), in LDS or
// device memory.
__device__ __forceinline__ void assemble(const LaneDesc& L, const DevGraph& g, bool all, uint64_t n_sel,
                         OutLink* out, uint32_t lb_key, double norm, bool with_post, bool mark_nodes,
                         uint64_t first, uint64_t stride, const uint64_t* lo_off, const uint64_t* xo_off,
                         const uint64_t* kf) {
  const int T = L.T;
  const uint64_t* kid = L.kept_idx;
  auto sel = [&](uint64_t j) -> uint64_t { return all ? j : kid[j]; };
  for (uint64_t j = first; j < n_sel; j += stride) {
    const uint64_t k = sel(j);
    const int t = (int)search_le64(lo_off, (uint64_t)T + 2, k);
    const uint64_t xo = xo_off[t];
    const bool eps = k >= xo;
    const uint64_t s0 = all ? lo_off[t] : kf[2 * t];
    const uint64_t sx = all ? xo : kf[2 * t + 1];
    const uint64_t s1 = all ? lo_off[t + 1] : kf[2 * t + 2];
    const LinkView l = link_at(L, k);
    // the other run [o0, o1) in selection order
    const uint64_t o0 = eps ? s0 : sx, o1 = eps ? sx : s1;
    uint64_t lo = o0, hi = o1;
    while (lo < hi) {
      const uint64_t mid = (lo + hi) >> 1;
      if (L.links[sel(mid)].x < l.arc) lo = mid + 1;
      else hi = mid;
    }
    const uint64_t rank = eps ? j - sx : j - s0;
    const uint64_t pos = s0 + rank + (lo - o0);
    if (pos >= n_sel) continue;  // cannot happen for consistent runs
    OutLink o;
    o.t = t;
    o.arc_id = l.arc;
    o.src_state = (int32_t)L.n_state[l.src];
    o.dst_state = (int32_t)L.n_state[l.dst];
    o.ilabel = g.ilabel_id[l.arc];
    o.olabel = g.olabel_id[l.arc];
    o.graph_cost = g.weight_id[l.arc];
    const double ac = link_ac(L, g, t, l.arc);
    o.ac_cost = (float)ac;
    o.fwd_cost = l.x;
    o.extra = key_cost(L.le_key[k]);
    o.posterior = 0.0;
    if (with_post && kept(L, k, lb_key)) {
      // exp(Z - alpha(src) - cost - beta(dst)) from the linear-domain sums
      const double f = eps ? eps_factor(o.graph_cost) : emit_factor(L.best[t], L.best[t - 1], o.graph_cost, ac);
      o.posterior = L.alpha[l.src] * L.beta[l.dst] * f * norm;
    }
    out[pos] = o;
    if (mark_nodes) {
      atomicOr(&L.used[l.src >> 5], 1u << (l.src & 31u));
      atomicOr(&L.used[l.dst >> 5], 1u << (l.dst & 31u));
    }
  }
}

// Lattice nodes (those marked in the used bitmap) in (t, state) order, which
// is node id order; returns their number.  Whole workgroup.
__device__ __forceinline__ uint64_t write_nodes(const LaneDesc& L, uint64_t nnodes, BlockScratch& bs, uint32_t& par,
                                                const uint64_t* no) {
  const uint32_t tid = threadIdx.x;
  const uint64_t nwd = (nnodes + 31) >> 5;
  const uint64_t per = (nwd + kLT - 1) / kLT;
  const uint64_t w0 = tid * per < nwd ? tid * per : nwd;
  const uint64_t w1 = w0 + per < nwd ? w0 + per : nwd;
  constexpr int kBatchW = 8;  // bitmap words read together
  uint64_t cnt = 0, n_out;
  for (uint64_t wb = w0; wb < w1; wb += kBatchW) {
    uint32_t v[kBatchW];
#pragma unroll
    for (int u = 0; u < kBatchW; ++u) v[u] = wb + u < w1 ? L.used[wb + u] : 0u;
#pragma unroll
    for (int u = 0; u < kBatchW; ++u) cnt += (uint64_t)__popc(v[u]);
  }
  uint64_t pos = block_excl_scan64<kLW>(cnt, bs, par, &n_out);
  // the frame of the thread's first node by a search, then walked forward
  // (node ids ascend in the thread's range)
  int t = -1;
  for (uint64_t w = w0; w < w1 && cnt; ++w) {
    uint32_t word = L.used[w];
    while (word) {
      const uint32_t b = (uint32_t)__ffs(word) - 1u;
      word &= word - 1u;
      const uint64_t n = (w << 5) | b;
      if (t < 0) t = (int)search_le64(no, (uint64_t)L.T + 2, n);
      while (no[t + 1] <= n) ++t;
      OutNode o;
      o.t = (int32_t)t;
      o.state = (int32_t)L.n_state[n];
      o.cost = node_cost(L, n);
      o.extra = key_cost(L.extra_key[n]);
      L.out_nodes[pos++] = o;
    }
  }
  return n_out;
}

// Levels present in a frame's epsilon links, highest first / lowest first.
__device__ __forceinline__ bool level_present(uint32_t mask, uint32_t lvl) {
  return (mask >> (lvl < 31u ? lvl : 31u)) & 1u;
}

// The per-frame chains (pruning sweep, alpha, beta) run on single
// wavefronts: a frame is a handful of dependent steps over tens of items, and
// the lanes of one wavefront need no workgroup barrier between steps.  Inputs
// of a frame that do not depend on the chain are loaded a frame ahead into
// registers, kAhead items per lane and run; further items are loaded in place.
constexpr int kAhead = 2;

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Synchronisation of the threads running a per-frame chain: one wavefront
// (GS = 64) or the whole workgroup.
template <int GS>
__device__ __forceinline__ void group_sync() {
  if (GS == 64) wave_sync();
  else __syncthreads();
}

// Loads of values other lanes update with atomics in device memory (frames
// too large for the LDS windows): served by L2, never by a stale L1 line.
__device__ __forceinline__ uint32_t load_fresh(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double load_fresh(const double* p) {
  const unsigned long long v = __hip_atomic_load(reinterpret_cast<const unsigned long long*>(p),
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return __longlong_as_double((long long)v);
}

// A frame's offsets (scalar loads, mostly scalar-cache hits) are read when
// its items are prefetched, a frame ahead of its processing.
// Offsets of frame u for the sweep, loaded two frames ahead of their use as
// vector loads: their waits count in issue order with the other loads, so a
// frame never waits for a load issued for a later one.
struct SweepFrame {
  uint64_t n0, n1, p0;  // nodes of frame u: [n0, n1); p0: first node of frame u-1 (n0 for u = 0)
  uint64_t k0, k1;      // emitting links out of frame u (empty for the last frame)
  uint64_t x0, x1;      // epsilon links of frame u
  uint32_t mask;        // their source levels
};
// A zero the compiler cannot see through.  Loads indexed with it are not known
// to be uniform, so their results stay in vector registers until `uniform`
// takes them; a load known to be uniform is moved to a scalar register, and
// waited for, right where it is issued.
__device__ __forceinline__ uint32_t opaque_zero() {
  uint32_t z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z));
  return z;
}
__device__ __forceinline__ uint64_t uni64(uint64_t v) {
  return ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(v >> 32)) << 32) |
         (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)v);
}

__device__ __forceinline__ void sweep_frame(const LaneDesc& L, int u, uint32_t z, SweepFrame& f) {
  const int T = L.T;
  const uint64_t* no = L.node_off + z;
  f.n0 = no[u];
  f.n1 = no[u + 1];
  f.p0 = no[u > 0 ? u - 1 : 0];
  f.x0 = L.link_xoff[u + z];
  f.x1 = L.link_off[u + 1 + z];
  f.k0 = f.x1;
  // the last frame's (empty) emitting run ends where it starts
  f.k1 = (u < T ? &L.link_xoff[u + 1] : &L.link_off[T + 1])[z];
  f.mask = L.xmask[u + z];
}
// The frame's offsets in scalar registers (their loads must have arrived).
__device__ __forceinline__ SweepFrame uniform(const SweepFrame& f) {
  SweepFrame u;
  u.n0 = uni64(f.n0);
  u.n1 = uni64(f.n1);
  u.p0 = uni64(f.p0);
  u.k0 = uni64(f.k0);
  u.k1 = uni64(f.k1);
  u.x0 = uni64(f.x0);
  u.x1 = u.k0;
  u.mask = __builtin_amdgcn_readfirstlane(f.mask);
  return u;
}

// extra(link) = extra(dst) + (x - cost(dst)) into le_key; extra(src) = min.
// exd/cd: the destination frame's window, or device memory (cd == nullptr).
__device__ __forceinline__ void sweep_relax(const LaneDesc& L, uint64_t k, uint4 v, const uint32_t* exd,
                                            const float* cd, uint64_t d0, uint32_t* ex, uint64_t n0) {
  const uint64_t d = v.z - d0;
  const float c = cd ? cd[d] : node_cost(L, v.z);
  const uint32_t e = cd ? exd[d] : load_fresh(&exd[d]);
  const uint32_t le = cost_key(key_cost(e) + (__uint_as_float(v.w) - c));
  L.le_key[k] = le;
  atomicMin(&ex[v.y - n0], le);
}

// The sweep: per frame the emitting links out of the frame (tens to
// hundreds) are relaxed by the whole workgroup; then wavefront 0 walks the
// frame's epsilon levels (a few tens of links) without workgroup barriers,
// while the other wavefronts write back frame t+1's window and initialise
// frame t-1's (three windows in turn).  Two workgroup barriers per frame.
struct SweepOne {
  uint32_t lvl, c;
  uint4 e, x;
};

// Index base + i when i < n, else some valid index (base + n - 1, or 0 for an
// empty range: every array holds at least one element).  Prefetches load
// unconditionally so that no merge copy waits for them.
__device__ __forceinline__ uint64_t safe_idx(uint64_t base, uint64_t i, uint64_t n) {
  return n ? base + (i < n ? i : n - 1) : 0;
}

// Links of frame u for this thread and the cost key of its node of frame
// u-1 (used only where that node exists).
__device__ __forceinline__ void sweep_one(const LaneDesc& L, const SweepFrame& f, uint32_t tid, SweepOne& it) {
  it.e = L.links[safe_idx(f.k0, tid, f.k1 - f.k0)];
  const uint64_t kx = safe_idx(f.x0, tid, f.x1 - f.x0);
  it.x = L.links[kx];
  it.lvl = L.link_lvl[kx];
  it.c = (uint32_t)(L.n_pack[safe_idx(f.p0, tid - 64, tid >= 64 ? f.n0 - f.p0 : 0)] >> 32);
}

// Extra costs (+inf, or the final extra cost for the last frame) and costs
// of frame t's nodes, by threads first, first + stride, ...; c0: the cost key
// of node `first`, loaded ahead (kNoKeyAhead: load it here).
constexpr uint32_t kNoKeyAhead = 0u;
__device__ __forceinline__ void sweep_init(const LaneDesc& L, const DevGraph& g, LatShared& sh, int t,
                                           const SweepFrame& a, uint32_t first, uint32_t stride, bool final_used,
                                           float best_total, uint32_t c0) {
  const uint64_t n0 = a.n0;
  const uint32_t nt = (uint32_t)(a.n1 - n0), buf = (uint32_t)t % 3u;
  auto init = [&](uint32_t* ex, float* cw) {
    for (uint32_t i = first; i < nt; i += stride) {
      const float c = (i == first && c0 != kNoKeyAhead) ? key_cost(c0) : node_cost(L, n0 + i);
      uint32_t e = kInfKey;
      if (t == L.T) {
        const float F = final_used ? canon(c + g.final_w[L.n_state[n0 + i]]) : c;
        if (F < INFINITY) e = cost_key(F - best_total);
      }
      ex[i] = e;
      if (cw) cw[i] = c;
    }
  };
  if (nt <= kWin) init(sh.w.p.ex[buf], sh.w.p.cost[buf]);
  else init(L.extra_key + n0, nullptr);
}

__device__ __forceinline__ void sweep_writeback(const LaneDesc& L, LatShared& sh, int t, const SweepFrame& a,
                                                uint32_t first, uint32_t stride) {
  const uint32_t nt = (uint32_t)(a.n1 - a.n0);
  if (nt > kWin) return;  // relaxed in device memory directly
  const uint32_t* ex = sh.w.p.ex[(uint32_t)t % 3u];
  for (uint32_t i = first; i < nt; i += stride) L.extra_key[a.n0 + i] = ex[i];
}

// Frame t.  sp, sa, sn: offsets of frames t+1, t and t-1 (t+1 unused for the
// last frame); those of frame t-2 are loaded into snn now.  cur: this
// thread's links of frame t and its node cost of frame t-1, loaded during
// frame t+1; those of frame t-1 (and t-2) are loaded into nxt now.  The
// caller rotates the sets, so no register with a load in flight is copied.
__device__ __forceinline__ void sweep_step(const LaneDesc& L, const DevGraph& g, LatShared& sh, uint32_t tid, int t,
                                           bool final_used, float best_total, const SweepFrame& sp_v,
                                           const SweepFrame& sa_v, const SweepFrame& sn_v, SweepFrame& snn,
                                           const SweepOne& cur, SweepOne& nxt, uint32_t z) {
  const int T = L.T;
  const SweepFrame sp = uniform(sp_v), sa = uniform(sa_v), sn = uniform(sn_v);
  sweep_frame(L, t > 1 ? t - 2 : 0, z, snn);
  sweep_one(L, sn, tid, nxt);
  const uint64_t n0 = sa.n0, n1 = sa.n1;
  const uint32_t buf = (uint32_t)t % 3u;
  const bool win = n1 - n0 <= kWin;
  // Each relaxation is written once per kind of window (LDS, device memory),
  // so that LDS windows are addressed as LDS: through a pointer that may be
  // either, every access would wait for all loads in flight.
  if (sa.k1 > sa.k0) {
    const uint64_t m0 = n1;
    const bool wn = sp.n1 - m0 <= kWin;
    const uint32_t nb = (uint32_t)(t + 1) % 3u;
    auto emitting = [&](const uint32_t* exn, const float* cn, uint32_t* ex) {
      if (sa.k0 + tid < sa.k1) sweep_relax(L, sa.k0 + tid, cur.e, exn, cn, m0, ex, n0);
      for (uint64_t k = sa.k0 + tid + kLT; k < sa.k1; k += kLT) sweep_relax(L, k, L.links[k], exn, cn, m0, ex, n0);
    };
    if (win && wn) emitting(sh.w.p.ex[nb], sh.w.p.cost[nb], sh.w.p.ex[buf]);
    else
      emitting(wn ? sh.w.p.ex[nb] : L.extra_key + m0, wn ? sh.w.p.cost[nb] : nullptr,
               win ? sh.w.p.ex[buf] : L.extra_key + n0);
  }
  __syncthreads();
  if (tid < 64) {
    auto epsilon = [&](uint32_t* ex, const float* cw) {
      for (int lvl = (int)g.nlevels - 1; lvl >= 0; --lvl) {
        if (!level_present(sa.mask, (uint32_t)lvl)) continue;
        if (sa.x0 + tid < sa.x1 && cur.lvl == (uint32_t)lvl) sweep_relax(L, sa.x0 + tid, cur.x, ex, cw, n0, ex, n0);
        for (uint64_t k = sa.x0 + tid + 64; k < sa.x1; k += 64)
          if (L.link_lvl[k] == (uint8_t)lvl) sweep_relax(L, k, L.links[k], ex, cw, n0, ex, n0);
        wave_sync();
      }
    };
    if (sa.x1 > sa.x0) {
      if (win) epsilon(sh.w.p.ex[buf], sh.w.p.cost[buf]);
      else epsilon(L.extra_key + n0, nullptr);
    }
  } else {
    if (t < T) sweep_writeback(L, sh, t + 1, sp, tid - 64, kLT - 64);
    if (t > 0) sweep_init(L, g, sh, t - 1, sn, tid - 64, kLT - 64, final_used, best_total, cur.c);
  }
  __syncthreads();
}

// Staged pruning sweep.  Frames are cut, from the last one down, into blocks
// of at most kSwK frames and kSwCap links and nodes.  The same relaxations
// as sweep_step, in the same order within each frame, but wavefront 0 walks
// the frames of a block with every operand already in LDS (links, node costs
// and extra costs in rings indexed by link and node id), its only global
// accesses the stores of the links' extra costs; meanwhile the other
// wavefronts load the block after next into the rings and write the block
// before back.  One workgroup barrier per block instead of two per frame.
// Returns false, before touching anything the other sweep needs, when a
// frame alone does not fit or the utterance is too long.  Whole workgroup.
__device__ __forceinline__ bool sweep_staged(const LaneDesc& L, const DevGraph& g, LatShared& sh, uint32_t tid,
                                             uint32_t& par, bool final_used, float best_total) {
  const int T = L.T;
  if ((uint64_t)T + 2 > kMgFrames) return false;
  // the frames' offsets, relative, into LDS
  const uint64_t kb = L.link_xoff[0], nb = L.node_off[0];
  for (int u = (int)tid; u <= T + 1; u += kLT) {
    if (u <= T) {
      sh.w.sw.ox[u] = (uint32_t)(L.link_xoff[u] - kb);
      sh.w.sw.oe[u] = (uint32_t)(L.link_off[u + 1] - kb);
      // one past frame u's last link: its emitting links run to the next
      // frame's epsilon run; the last frame has none
      sh.w.sw.oz[u] = (uint32_t)((u < T ? L.link_xoff[u + 1] : L.link_off[T + 1]) - kb);
    }
    sh.w.sw.on[u] = (uint32_t)(L.node_off[u] - nb);
  }
  __syncthreads();
  // blocks from the last frame down, cut greedily by one thread
  if (tid == 0) {
    int nblk = 0, u = T;
    bool fits = true;
    while (u >= 0 && fits) {
      const int hi = u;
      sh.w.sw.top[nblk++] = hi;
      while (u >= 0 && hi - u < kSwK && sh.w.sw.oz[hi] - sh.w.sw.ox[u] <= kSwCap &&
             sh.w.sw.on[hi + 1] - sh.w.sw.on[u] <= kSwCap)
        --u;
      fits = u < hi;  // the block holds at least its first frame
    }
    sh.w.sw.top[nblk] = -1;
    sh.w.sw.nblk = fits ? nblk : -1;
  }
  __syncthreads();
  const int nblk = sh.w.sw.nblk;
  if (nblk < 0) return false;
  auto hi_of = [&](int b) { return sh.w.sw.top[b]; };
  auto lo_of = [&](int b) { return sh.w.sw.top[b + 1] + 1; };
  constexpr uint32_t kM = kSwRing - 1;
  // block b into the rings (by the threads first, first + stride, ...)
  auto load = [&](int b, uint32_t first, uint32_t stride) {
    const int hi = hi_of(b), lo = lo_of(b);
    for (int u = lo + (int)first; u <= hi; u += (int)stride) sh.w.sw.fm[u % kSwFrames] = L.xmask[u];
    const uint64_t k0 = kb + sh.w.sw.ox[lo], k1 = kb + sh.w.sw.oz[hi];
    for (uint64_t k = k0 + first; k < k1; k += stride) {
      const uint4 v = L.links[k];
      const uint32_t r = (uint32_t)k & kM;
      sh.w.sw.sd[r] = (v.y & kM) | ((v.z & kM) << 16);
      sh.w.sw.dl[r] = __uint_as_float(v.w) - node_cost(L, v.z);
      sh.w.sw.lvl[r] = L.link_lvl[k];
    }
    const uint64_t n0 = nb + sh.w.sw.on[lo], n1 = nb + sh.w.sw.on[hi + 1], nT = nb + sh.w.sw.on[T];
    for (uint64_t n = n0 + first; n < n1; n += stride) {
      const float c = node_cost(L, n);
      uint32_t e = kInfKey;
      if (n >= nT) {
        const float F = final_used ? canon(c + g.final_w[L.n_state[n]]) : c;
        if (F < INFINITY) e = cost_key(F - best_total);
      }
      sh.w.sw.ex[(uint32_t)n & kM] = e;
    }
  };
  auto writeback = [&](int b, uint32_t first, uint32_t stride) {
    const uint64_t n0 = nb + sh.w.sw.on[lo_of(b)], n1 = nb + sh.w.sw.on[hi_of(b) + 1];
    for (uint64_t n = n0 + first; n < n1; n += stride) L.extra_key[n] = sh.w.sw.ex[(uint32_t)n & kM];
  };
  // link k (ring record sd, dl) relaxed into its source's extra cost (the
  // key array's address held in a register: a store through the lane
  // descriptor's field would make the compiler reload the field after every
  // store)
  uint32_t* const __restrict__ lek = L.le_key;
  auto relax_sd = [&](uint64_t k, uint32_t sd, float dl) {
    const uint32_t le = cost_key(key_cost(sh.w.sw.ex[sd >> 16]) + dl);
    lek[k] = le;
    atomicMin(&sh.w.sw.ex[sd & 0xffffu], le);
  };
  auto relax = [&](uint64_t k) {
    const uint32_t r = (uint32_t)k & kM;
    relax_sd(k, sh.w.sw.sd[r], sh.w.sw.dl[r]);
  };
  // levels present in a frame, one bit each (deeper graphs fold levels from
  // 31 up into bit 31 and take the per-level loop)
  const bool bitwise_levels = g.nlevels <= 31;
  load(0, tid, kLT);
  if (nblk > 1) load(1, tid, kLT);
  __syncthreads();
  for (int b = 0; b < nblk; ++b) {
    if (tid < 64) {
      for (int u = hi_of(b); u >= lo_of(b); --u) {
        const uint64_t x0 = kb + sh.w.sw.ox[u], e0 = kb + sh.w.sw.oe[u], z = kb + sh.w.sw.oz[u];
        const uint32_t mask = sh.w.sw.fm[u % kSwFrames];
        // emitting links out of the frame (none out of the last one)
        if (u < T) {
          for (uint64_t k = e0 + tid; k < z; k += 64) relax(k);
          wave_sync();
        }
        // epsilon links, from the highest source level down: with at most one
        // per lane, each lane's record is read once and kept for every level
        if (bitwise_levels && e0 - x0 <= 64) {
          const uint64_t k = x0 + tid;
          const bool has = k < e0;
          uint32_t sd = 0, lv = 0xffu;
          float dl = 0.0f;
          if (has) {
            const uint32_t r = (uint32_t)k & kM;
            sd = sh.w.sw.sd[r];
            dl = sh.w.sw.dl[r];
            lv = sh.w.sw.lvl[r];
          }
          for (uint32_t m = mask; m;) {
            const uint32_t lvl = 31u - (uint32_t)__clz(m);
            m &= ~(1u << lvl);
            if (lv == lvl) relax_sd(k, sd, dl);
            wave_sync();
          }
        } else {
          for (int lvl = (int)g.nlevels - 1; lvl >= 0; --lvl) {
            if (!level_present(mask, (uint32_t)lvl)) continue;
            for (uint64_t k = x0 + tid; k < e0; k += 64)
              if (sh.w.sw.lvl[(uint32_t)k & kM] == (uint8_t)lvl) relax(k);
            wave_sync();
          }
        }
      }
    } else {
      if (b + 2 < nblk) load(b + 2, tid - 64, kLT - 64);
      if (b >= 1) writeback(b - 1, tid - 64, kLT - 64);
    }
    __syncthreads();
  }
  writeback(nblk - 1, tid, kLT);
  return true;
}

// Backward extra-cost sweep over every frame: four sets of frame offsets and
// two of links in rotation (a loop of four frames, then up to three more).
__device__ __forceinline__ void sweep_block(const LaneDesc& L, const DevGraph& g, LatShared& sh,
                                            uint32_t tid, bool final_used, float best_total) {
  const int T = L.T;
  const uint32_t z = opaque_zero();
  SweepFrame A{}, B, C, D;
  SweepOne x, y;
  sweep_frame(L, T, z, B);
  sweep_frame(L, T > 0 ? T - 1 : 0, z, C);
  const SweepFrame fT = uniform(B);
  sweep_one(L, fT, tid, x);
  sweep_init(L, g, sh, T, fT, tid, kLT, final_used, best_total, kNoKeyAhead);
  __syncthreads();
  int t = T;
  for (; t >= 3; t -= 4) {
    sweep_step(L, g, sh, tid, t, final_used, best_total, A, B, C, D, x, y, z);
    sweep_step(L, g, sh, tid, t - 1, final_used, best_total, B, C, D, A, y, x, z);
    sweep_step(L, g, sh, tid, t - 2, final_used, best_total, C, D, A, B, x, y, z);
    sweep_step(L, g, sh, tid, t - 3, final_used, best_total, D, A, B, C, y, x, z);
  }
  if (t >= 0) sweep_step(L, g, sh, tid, t, final_used, best_total, A, B, C, D, x, y, z);
  if (t >= 1) sweep_step(L, g, sh, tid, t - 1, final_used, best_total, B, C, D, A, y, x, z);
  if (t >= 2) sweep_step(L, g, sh, tid, t - 2, final_used, best_total, C, D, A, B, x, y, z);
  SweepFrame f0;
  sweep_frame(L, 0, z, f0);
  sweep_writeback(L, sh, 0, uniform(f0), tid, kLT);
}

// Kept link j for the forward-backward pass: {src node, dst node, graph cost
// bits, acoustic cost bits (emitting) or source level (epsilon)}.
__device__ __forceinline__ uint4 post_link(const LaneDesc& L, uint64_t j) { return L.post[j]; }

// Record of kept link j (link k) of frame t; `eps`: an epsilon link.
// {src node, dst node, the link's factor (epsilon: with its source level in
// the low bits) as two words}.
__device__ __forceinline__ uint4 post_record(const LaneDesc& L, const DevGraph& g, uint64_t k, int t, bool eps) {
  const uint4 v = L.links[k];
  const float w = g.weight_id[v.x];
  double f;
  uint32_t lvl = 0;
  if (eps) {
    f = eps_factor(w);
    lvl = L.link_lvl[k];
  } else {
    f = emit_factor(L.best[t], L.best[t - 1], w, -(double)L.ll[(size_t)(t - 1) * g.P + (g.ilabel_id[v.x] - 1)]);
  }
  const uint2 fb = factor_bits(f, eps, lvl);
  return make_uint4(v.y, v.z, fb.x, fb.y);
}
__device__ __forceinline__ double rec_factor(uint4 l) { return __hiloint2double((int)l.w, (int)l.z); }
__device__ __forceinline__ uint32_t rec_level(uint4 l) { return l.z & 0xffu; }

// Kept links of a run beyond the prefetched ones, kBatch per lane per round
// trip: the loads of a batch are issued together, then the batch is applied.
constexpr int kBatch = 4;

template <int GS, typename F>
__device__ __forceinline__ void post_tail(const LaneDesc& L, uint64_t j0, uint64_t j1, uint32_t lane, F&& apply) {
  for (uint64_t jb = j0 + lane + (uint64_t)GS * kAhead; jb < j1; jb += (uint64_t)GS * kBatch) {
    uint4 lb[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      if (jb + (uint64_t)GS * u < j1) lb[u] = post_link(L, jb + (uint64_t)GS * u);
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      if (jb + (uint64_t)GS * u < j1) apply(lb[u]);
  }
}

// Offsets of frame u for a posterior pass, loaded two frames ahead of their
// use like the sweep's.
struct PostFrame {
  uint64_t n0, n1;  // nodes of frame u
  uint64_t m0, m1;  // nodes of the frame the emitting links come from (alpha: u-1) or go to (beta: u+1)
  uint64_t e0, e1;  // kept emitting links into u (alpha) or out of u (beta)
  uint64_t x0, x1;  // kept epsilon links of u
  uint32_t mask;    // their source levels
};
struct PostItems {
  uint4 e[kAhead], x[kAhead];
  float fw[kAhead];
};

__device__ __forceinline__ PostFrame uniform(const PostFrame& f) {
  PostFrame u;
  u.n0 = uni64(f.n0);
  u.n1 = uni64(f.n1);
  u.m0 = uni64(f.m0);
  u.m1 = uni64(f.m1);
  u.e0 = uni64(f.e0);
  u.e1 = uni64(f.e1);
  u.x0 = uni64(f.x0);
  u.x1 = uni64(f.x1);
  u.mask = __builtin_amdgcn_readfirstlane(f.mask);
  return u;
}

// Frame u of the alpha pass: emitting kept links into u (from u-1), epsilon
// kept links of u.
__device__ __forceinline__ void alpha_frame(const LaneDesc& L, int u, uint32_t z, PostFrame& f) {
  const uint64_t* no = L.node_off + z;
  const uint64_t* kf = L.kframe + z;
  f.n0 = no[u];
  f.n1 = no[u + 1];
  f.m0 = no[u > 0 ? u - 1 : 0];
  f.m1 = f.n0;
  f.e0 = kf[2 * u];
  f.e1 = kf[2 * u + 1];
  f.x0 = f.e1;
  f.x1 = kf[2 * u + 2];
  f.mask = L.xmask[u + z];
}

// Frame u of the beta pass: emitting kept links out of u (into u+1), epsilon
// kept links of u.
__device__ __forceinline__ void beta_frame(const LaneDesc& L, int u, uint32_t z, PostFrame& f) {
  const int T = L.T;
  const uint64_t* no = L.node_off + z;
  const uint64_t* kf = L.kframe + z;
  f.n0 = no[u];
  f.n1 = no[u + 1];
  f.m0 = f.n1;
  f.m1 = no[u < T ? u + 2 : u + 1];
  f.x0 = kf[2 * u + 1];
  f.x1 = kf[2 * u + 2];
  f.e0 = f.x1;
  f.e1 = kf[u < T ? 2 * u + 3 : 2 * u + 2];  // none out of the last frame
  f.mask = L.xmask[u + z];
}

// Kept links of a frame for this lane (loaded unconditionally, like the
// sweep's links); `fin`: also the final weights of the frame's first nodes
// (the last frame of the beta pass).
template <int GS>
__device__ __forceinline__ void post_items(const LaneDesc& L, const DevGraph& g, const PostFrame& a, uint32_t lane,
                                           bool fin, PostItems& it) {
#pragma unroll
  for (int q = 0; q < kAhead; ++q) {
    const uint64_t i = lane + (uint64_t)GS * q;
    it.e[q] = post_link(L, safe_idx(a.e0, i, a.e1 - a.e0));
    it.x[q] = post_link(L, safe_idx(a.x0, i, a.x1 - a.x0));
    if (fin && i < a.n1 - a.n0) it.fw[q] = g.final_w[L.n_state[a.n0 + i]];
  }
}

// Frame t of the alpha pass on a group of GS threads.  sa, sn: offsets of
// frames t and t+1; those of t+2 are loaded into snn now.  cur: kept links
// of frame t (loaded during t-1); those of t+1 are loaded into nxt now.
// `swept`: device-memory alpha is +inf already.
template <int GS>
__device__ __forceinline__ void alpha_step(const LaneDesc& L, const DevGraph& g, LatShared& sh, uint32_t lane,
                                           int t, bool swept, uint64_t start_node, double s_start, const PostFrame& sa_v,
                                           const PostFrame& sn_v, PostFrame& snn, const PostItems& cur,
                                           PostItems& nxt, uint32_t z) {
  const int T = L.T;
  const PostFrame pa = uniform(sa_v), pn = uniform(sn_v);
  alpha_frame(L, t + 2 <= T ? t + 2 : T, z, snn);
  post_items<GS>(L, g, pn, lane, false, nxt);
  const uint64_t n0 = pa.n0, n1 = pa.n1, m0 = pa.m0;
  const uint32_t nt = (uint32_t)(n1 - n0), buf = (uint32_t)t & 1u;
  const bool win = nt <= kWin, wp = n0 - m0 <= kWin;
  // written once per kind of window, as in the sweep
  auto frame = [&](double* a, const double* ap, bool lds_a, bool lds_ap) {
    if (lds_a || !swept) {
      for (uint32_t i = lane; i < nt; i += GS) a[i] = (n0 + i == start_node) ? s_start : 0.0;
    } else if (lane == 0 && start_node >= n0 && start_node < n1) {
      a[start_node - n0] = s_start;  // the rest is 0 already
    }
    group_sync<GS>();
    if (pa.e1 > pa.e0) {
      auto emit = [&](uint4 l) {
        const double av = lds_ap ? ap[l.x - m0] : load_fresh(&ap[l.x - m0]);
        mass_add(&a[l.y - n0], av * rec_factor(l), lds_a);
      };
#pragma unroll
      for (int q = 0; q < kAhead; ++q)
        if (pa.e0 + lane + (uint64_t)GS * q < pa.e1) emit(cur.e[q]);
      post_tail<GS>(L, pa.e0, pa.e1, lane, emit);
      group_sync<GS>();
    }
    if (pa.x1 > pa.x0)
      for (uint32_t lvl = 0; lvl < g.nlevels; ++lvl) {
        if (!level_present(pa.mask, lvl)) continue;
        auto eps = [&](uint4 l) {
          if (rec_level(l) != lvl) return;
          const double av = lds_a ? a[l.x - n0] : load_fresh(&a[l.x - n0]);
          mass_add(&a[l.y - n0], av * rec_factor(l), lds_a);
        };
#pragma unroll
        for (int q = 0; q < kAhead; ++q)
          if (pa.x0 + lane + (uint64_t)GS * q < pa.x1) eps(cur.x[q]);
        post_tail<GS>(L, pa.x0, pa.x1, lane, eps);
        group_sync<GS>();
      }
    if (lds_a)
      for (uint32_t i = lane; i < nt; i += GS) L.alpha[n0 + i] = a[i];
  };
  if (win && wp) frame(sh.w.ab.a[buf], sh.w.ab.a[buf ^ 1u], true, true);
  else frame(win ? sh.w.ab.a[buf] : L.alpha + n0, wp ? sh.w.ab.a[buf ^ 1u] : L.alpha + m0, win, wp);
}

// alpha over every frame, ascending; epsilon links of a frame by source
// level, on GS threads.  The look-ahead sets move down at the end of a step,
// when their loads (issued at its start) have had the step to arrive.
template <int GS>
__device__ __forceinline__ void alpha_wave(const LaneDesc& L, const DevGraph& g, LatShared& sh, uint32_t lane,
                                           bool swept, uint64_t start_node) {
  const int T = L.T;
  const uint32_t z = opaque_zero();
  PostFrame sa, sn, snn;
  PostItems cur{}, nxt{};
  alpha_frame(L, 0, z, sa);
  alpha_frame(L, T >= 1 ? 1 : 0, z, sn);
  post_items<GS>(L, g, uniform(sa), lane, false, cur);
  const double s_start = exp((double)L.best[0]);  // exp(b(0) - alpha(start)), alpha(start) = 0
  for (int t = 0; t <= T; ++t) {
    alpha_step<GS>(L, g, sh, lane, t, swept, start_node, s_start, sa, sn, snn, cur, nxt, z);
    sa = sn;
    sn = snn;
    cur = nxt;
  }
}

// Frame t of the beta pass on a group of GS threads.  sa, sn: offsets of
// frames t and t-1; those of t-2 are loaded into snn now.  cur: kept links
// of frame t (loaded during t+1); those of t-1 are loaded into nxt now.
template <int GS>
__device__ __forceinline__ void beta_step(const LaneDesc& L, const DevGraph& g, LatShared& sh, uint32_t lane,
                                          int t, bool swept, bool final_used, double ref_T, const PostFrame& sa_v,
                                          const PostFrame& sn_v, PostFrame& snn, const PostItems& cur,
                                          PostItems& nxt, uint32_t z) {
  const int T = L.T;
  const PostFrame pa = uniform(sa_v), pn = uniform(sn_v);
  beta_frame(L, t > 1 ? t - 2 : 0, z, snn);
  post_items<GS>(L, g, pn, lane, false, nxt);
  const uint64_t n0 = pa.n0, n1 = pa.n1, m0 = pa.m0;
  const uint32_t nt = (uint32_t)(n1 - n0), buf = (uint32_t)t & 1u;
  const bool win = nt <= kWin, wn = pa.m1 - m0 <= kWin;
  auto frame = [&](double* b, const double* bn, bool lds_b, bool lds_bn) {
    if (lds_b || !swept || t == T) {
#pragma unroll
      for (int q = 0; q <= kAhead; ++q)
        for (uint32_t i = lane + (uint32_t)(GS * q); i < nt; i += (q < kAhead ? nt : (uint32_t)GS)) {
          double v = 0.0;  // exp(B - b(T) - final weight) on the last frame
          if (t == T)
            v = exp(ref_T -
                    (final_used ? (double)(q < kAhead ? cur.fw[q < kAhead ? q : 0] : g.final_w[L.n_state[n0 + i]])
                                : 0.0));
          b[i] = v;
        }
    }
    group_sync<GS>();
    if (pa.e1 > pa.e0) {
      auto emit = [&](uint4 l) {
        const double bv = lds_bn ? bn[l.y - m0] : load_fresh(&bn[l.y - m0]);
        mass_add(&b[l.x - n0], rec_factor(l) * bv, lds_b);
      };
#pragma unroll
      for (int q = 0; q < kAhead; ++q)
        if (pa.e0 + lane + (uint64_t)GS * q < pa.e1) emit(cur.e[q]);
      post_tail<GS>(L, pa.e0, pa.e1, lane, emit);
      group_sync<GS>();
    }
    if (pa.x1 > pa.x0)
      for (int lvl = (int)g.nlevels - 1; lvl >= 0; --lvl) {
        if (!level_present(pa.mask, (uint32_t)lvl)) continue;
        auto eps = [&](uint4 l) {
          if (rec_level(l) != (uint32_t)lvl) return;
          const double bv = lds_b ? b[l.y - n0] : load_fresh(&b[l.y - n0]);
          mass_add(&b[l.x - n0], rec_factor(l) * bv, lds_b);
        };
#pragma unroll
        for (int q = 0; q < kAhead; ++q)
          if (pa.x0 + lane + (uint64_t)GS * q < pa.x1) eps(cur.x[q]);
        post_tail<GS>(L, pa.x0, pa.x1, lane, eps);
        group_sync<GS>();
      }
    if (lds_b)
      for (uint32_t i = lane; i < nt; i += GS) L.beta[n0 + i] = b[i];
  };
  if (win && wn) frame(sh.w.ab.b[buf], sh.w.ab.b[buf ^ 1u], true, true);
  else frame(win ? sh.w.ab.b[buf] : L.beta + n0, wn ? sh.w.ab.b[buf ^ 1u] : L.beta + m0, win, wn);
}

// beta over every frame, descending; epsilon links of a frame from the
// highest source level, on GS threads.
template <int GS>
__device__ __forceinline__ void beta_wave(const LaneDesc& L, const DevGraph& g, LatShared& sh, uint32_t lane,
                                          bool swept, bool final_used, float best_total) {
  const int T = L.T;
  const uint32_t z = opaque_zero();
  PostFrame sa, sn, snn;
  PostItems cur{}, nxt{};
  beta_frame(L, T, z, sa);
  beta_frame(L, T >= 1 ? T - 1 : 0, z, sn);
  post_items<GS>(L, g, uniform(sa), lane, final_used, cur);
  const double ref_T = (double)best_total - (double)L.best[T];  // B - b(T)
  for (int t = T; t >= 0; --t) {
    beta_step<GS>(L, g, sh, lane, t, swept, final_used, ref_T, sa, sn, snn, cur, nxt, z);
    sa = sn;
    sn = snn;
    cur = nxt;
  }
}

// Compact posteriors.  The nodes that kept links touch (and the start node)
// are numbered in node id order through a bitmap in LDS; the kept link
// records, the per-frame kept-link boundaries and each frame's kept epsilon
// levels are copied into LDS with those numbers; then wavefront 0 runs the
// alpha sums and wavefront 1 the beta sums frame by frame exactly as the
// windowed passes do (emitting links, then epsilon links by source level),
// with every value they read already in LDS.  A node's sums are only ever
// added to by links in its own frame's step, so starting every node at 0 (the
// start node at its alpha seed, the last frame's nodes at their final beta)
// equals the per-frame initialisation.  At the end the touched nodes' sums
// go to the workspace arrays, where the merge reads them.  Returns false
// (before touching anything the other path needs) when the lattice does not
// fit.  Whole workgroup.
__device__ __forceinline__ bool compact_fits(const LaneDesc& L, const DevGraph& g, uint64_t n_kept, uint64_t nnodes) {
  return n_kept <= kCpLinks && (uint64_t)L.T + 2 <= kCpFrames && ((nnodes + 31) >> 5) <= kCpWords &&
         g.nlevels <= 32;
}

__device__ __forceinline__ bool posteriors_compact(const LaneDesc& L, const DevGraph& g, LatShared& sh, uint32_t tid,
                                                   uint32_t& par, uint64_t n_kept, uint64_t nnodes,
                                                   uint64_t start_node, bool final_used, float best_total) {
  const int T = L.T;
  uint32_t* bits = reinterpret_cast<uint32_t*>(sh.w.cp.a);
  uint32_t* rank = reinterpret_cast<uint32_t*>(sh.w.cp.b);
  const uint32_t nwd = (uint32_t)((nnodes + 31) >> 5);
  for (uint32_t w = tid; w < nwd; w += kLT) bits[w] = 0;
  __syncthreads();
  for (uint64_t j = tid; j < n_kept; j += kLT) {
    const uint4 r = L.post[j];
    atomicOr(&bits[r.x >> 5], 1u << (r.x & 31u));
    atomicOr(&bits[r.y >> 5], 1u << (r.y & 31u));
  }
  if (tid == 0) atomicOr(&bits[start_node >> 5], 1u << (start_node & 31u));
  __syncthreads();
  // word ranks: a contiguous range of words per thread
  const uint32_t per = (nwd + kLT - 1) / kLT;
  const uint32_t w0 = tid * per < nwd ? tid * per : nwd;
  const uint32_t w1 = w0 + per < nwd ? w0 + per : nwd;
  uint64_t cnt = 0;
  for (uint32_t w = w0; w < w1; ++w) cnt += (uint32_t)__popc(bits[w]);
  uint64_t K;
  uint32_t r = (uint32_t)block_excl_scan64<kLW>(cnt, sh.bs, par, &K);
  if (K > kCpNodes) return false;  // (uniform)
  for (uint32_t w = w0; w < w1; ++w) {
    rank[w] = r;
    uint32_t word = bits[w];
    while (word) {
      const uint32_t b = (uint32_t)__ffs(word) - 1u;
      word &= word - 1u;
      sh.w.cp.node[r++] = (w << 5) | b;
    }
  }
  __syncthreads();
  auto cid = [&](uint32_t n) -> uint32_t {
    return rank[n >> 5] + (uint32_t)__popc(bits[n >> 5] & ((1u << (n & 31u)) - 1u));
  };
  for (uint64_t j = tid; j < n_kept; j += kLT) {
    const uint4 l = L.post[j];
    sh.w.cp.link[j] = make_uint4(cid(l.x), cid(l.y), l.z, l.w);
  }
  const uint64_t* kf = L.kframe;
  for (uint32_t i = tid; i < 2u * (uint32_t)(T + 2); i += kLT) sh.w.cp.kf[i] = (uint16_t)kf[i];
  for (int t = (int)tid; t <= T; t += kLT) {
    uint32_t m = 0;
    for (uint64_t j = kf[2 * t + 1]; j < kf[2 * t + 2]; ++j) m |= 1u << rec_level(L.post[j]);
    sh.w.cp.lmask[t] = m;
  }
  const uint32_t cstart = tid == 0 ? cid((uint32_t)start_node) : 0u;
  __syncthreads();  // every renumbering read of the bitmap is done
  const uint64_t nT = L.node_off[T];
  const double s_start = exp((double)L.best[0]);
  const double ref_T = (double)best_total - (double)L.best[T];  // B - b(T)
  for (uint32_t c = tid; c < (uint32_t)K; c += kLT) {
    const uint32_t n = sh.w.cp.node[c];
    sh.w.cp.a[c] = 0.0;
    double b = 0.0;
    if (n >= nT) b = exp(ref_T - (final_used ? (double)g.final_w[L.n_state[n]] : 0.0));
    sh.w.cp.b[c] = b;
  }
  __syncthreads();
  if (tid == 0) sh.w.cp.a[cstart] = s_start;
  __syncthreads();
  const uint4* lk = sh.w.cp.link;
  const uint16_t* kfs = sh.w.cp.kf;
  if (tid < 64) {
    // alpha, frames ascending; epsilon links from the lowest source level.
    // A frame's boundaries, level mask and first emitting and epsilon records
    // are read during the frame before (off the chain of adds).
    double* a = sh.w.cp.a;
    const uint4 none = make_uint4(0, 0, 0, 0);
    uint32_t e0 = kfs[0], x0 = kfs[1], x1 = kfs[2], m0 = sh.w.cp.lmask[0];
    uint4 le = e0 + tid < x0 ? lk[e0 + tid] : none, lx = x0 + tid < x1 ? lk[x0 + tid] : none;
    for (int t = 0; t <= T; ++t) {
      uint32_t ne0 = 0, nx0 = 0, nx1 = 0, nm = 0;
      uint4 nle = none, nlx = none;
      if (t < T) {
        ne0 = kfs[2 * t + 2];
        nx0 = kfs[2 * t + 3];
        nx1 = kfs[2 * t + 4];
        nm = sh.w.cp.lmask[t + 1];
        if (ne0 + tid < nx0) nle = lk[ne0 + tid];
        if (nx0 + tid < nx1) nlx = lk[nx0 + tid];
      }
      if (e0 + tid < x0) mass_add(&a[le.y], a[le.x] * rec_factor(le), true);
      for (uint32_t j = e0 + tid + 64; j < x0; j += 64) {
        const uint4 l = lk[j];
        mass_add(&a[l.y], a[l.x] * rec_factor(l), true);
      }
      wave_sync();
      for (uint32_t m = m0; m;) {
        const uint32_t lvl = (uint32_t)__ffs(m) - 1u;
        m &= m - 1u;
        if (x0 + tid < x1 && rec_level(lx) == lvl) mass_add(&a[lx.y], a[lx.x] * rec_factor(lx), true);
        for (uint32_t j = x0 + tid + 64; j < x1; j += 64) {
          const uint4 l = lk[j];
          if (rec_level(l) == lvl) mass_add(&a[l.y], a[l.x] * rec_factor(l), true);
        }
        wave_sync();
      }
      e0 = ne0;
      x0 = nx0;
      x1 = nx1;
      m0 = nm;
      le = nle;
      lx = nlx;
    }
  } else if (tid < 128) {
    // beta, frames descending; epsilon links from the highest source level;
    // read ahead like alpha
    const uint32_t lane = tid - 64;
    double* b = sh.w.cp.b;
    const uint4 none = make_uint4(0, 0, 0, 0);
    auto bounds = [&](int t, uint32_t& x0, uint32_t& x1, uint32_t& e1) {
      x0 = kfs[2 * t + 1];
      x1 = kfs[2 * t + 2];
      e1 = t < T ? kfs[2 * t + 3] : x1;  // emitting links out of t (into t+1)
    };
    uint32_t x0, x1, e1;
    bounds(T, x0, x1, e1);
    uint32_t m0 = sh.w.cp.lmask[T];
    uint4 le = x1 + lane < e1 ? lk[x1 + lane] : none, lx = x0 + lane < x1 ? lk[x0 + lane] : none;
    for (int t = T; t >= 0; --t) {
      uint32_t nx0 = 0, nx1 = 0, ne1 = 0, nm = 0;
      uint4 nle = none, nlx = none;
      if (t > 0) {
        bounds(t - 1, nx0, nx1, ne1);
        nm = sh.w.cp.lmask[t - 1];
        if (nx1 + lane < ne1) nle = lk[nx1 + lane];
        if (nx0 + lane < nx1) nlx = lk[nx0 + lane];
      }
      if (x1 + lane < e1) mass_add(&b[le.x], rec_factor(le) * b[le.y], true);
      for (uint32_t j = x1 + lane + 64; j < e1; j += 64) {
        const uint4 l = lk[j];
        mass_add(&b[l.x], rec_factor(l) * b[l.y], true);
      }
      wave_sync();
      for (uint32_t m = m0; m;) {
        const uint32_t lvl = 31u - (uint32_t)__clz(m);
        m &= ~(1u << lvl);
        if (x0 + lane < x1 && rec_level(lx) == lvl) mass_add(&b[lx.x], rec_factor(lx) * b[lx.y], true);
        for (uint32_t j = x0 + lane + 64; j < x1; j += 64) {
          const uint4 l = lk[j];
          if (rec_level(l) == lvl) mass_add(&b[l.x], rec_factor(l) * b[l.y], true);
        }
        wave_sync();
      }
      x0 = nx0;
      x1 = nx1;
      e1 = ne1;
      m0 = nm;
      le = nle;
      lx = nlx;
    }
  }
  __syncthreads();
  for (uint32_t c = tid; c < (uint32_t)K; c += kLT) {
    const uint32_t n = sh.w.cp.node[c];
    L.alpha[n] = sh.w.cp.a[c];
    L.beta[n] = sh.w.cp.b[c];
  }
  return true;
}

// blockIdx.y == 0: pruning, posteriors and the final merge; blockIdx.y == 1:
// the 1-best traceback (a serial walk over predecessor pointers, run
// concurrently by its own workgroup).
__global__ void __launch_bounds__(kLT) k_lattice(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                      Params prm) {
  __shared__ LatShared sh;
  const LaneDesc& L = lanes[blockIdx.x];
  LaneInfo* info = L.info;
  if (info->status != 0) return;
  const uint32_t tid = threadIdx.x;
  const int T = L.T;
  // step profile (WD_FLAG_PHASES): the wall clock at the pass's section
  // boundaries, in the profile row after the last frame's
  auto lstamp = [&](int k) {
    if (L.prof && tid == 0 && blockIdx.y == 0) L.prof[(size_t)(T + 1) * kProfSlots + (size_t)k] = wall_clock64();
  };
  lstamp(0);
  const uint64_t nT0 = L.node_off[T], nT1 = L.node_off[T + 1];
  const uint64_t nnodes = nT1;
  const uint64_t nlinks = L.link_off[T + 1];
  uint32_t par = 0;

  // ------------------------------------------------ final costs, best end token
  const bool swept = (prm.flags & kFlagSwept) != 0;
  bool final_used;
  uint32_t best_key;
  uint64_t bnode;
  if (swept) {
    // found by the chip-wide kernels
    final_used = info->final_used != 0;
    best_key = cost_key(info->best_cost);
    bnode = info->best_node;
  } else {
    uint32_t any = 0;
    if (g.final_w)
      for (uint64_t n = nT0 + tid; n < nT1; n += kLT) {
        const float fw = g.final_w[L.n_state[n]];
        const float c = node_cost(L, n);
        any |= (fw < INFINITY && (c + fw) < INFINITY) ? 1u : 0u;
      }
    final_used = block_or<kLW>(any, sh.bs, par) != 0;
    uint64_t m = kEmpty;
    for (uint64_t n = nT0 + tid; n < nT1; n += kLT) {
      const float c = node_cost(L, n);
      const float F = final_used ? canon(c + g.final_w[L.n_state[n]]) : c;
      const uint64_t v = pack_tok(cost_key(F), (uint32_t)(n - nT0));
      m = v < m ? v : m;
    }
    m = block_min64<kLW>(m, sh.bs, par);
    best_key = (uint32_t)(m >> 32);
    bnode = nT0 + (m & 0xffffffffu);
  }
  if (best_key >= kInfKey) {
    if (tid == 0 && blockIdx.y == 0) info->status = 3;
    return;
  }
  const float best_total = key_cost(best_key);

  if (blockIdx.y == 1) {
    // ------------------------------------------------------------ traceback
    if (tid != 0) return;
    uint64_t tb = bnode, nw = 0;
    bool ok = true;
    for (int t = T; t >= 0 && ok; --t) {
      const uint64_t n0 = L.node_off[t], n1 = L.node_off[t + 1];
      // epsilon predecessors stay in frame t; an emitting one goes back a frame
      for (uint32_t steps = 0;; ++steps) {
        if (tb < n0 || tb >= n1 || steps > g.nlevels) {
          ok = false;
          break;
        }
        const uint32_t arc = (uint32_t)L.n_pack[tb];
        if (arc == kNoArc) break;
        if (arc >= g.A) {
          ok = false;
          break;
        }
        const int32_t ol = g.olabel_id[arc];
        if (ol != 0) {
          if (nw < L.word_cap) L.out_words[nw] = ol;
          else ok = false;
          ++nw;
        }
        tb = L.n_pred[tb];
        if (g.ilabel_id[arc] != 0) break;
      }
    }
    if (ok)
      for (uint64_t i = 0; i < nw / 2; ++i) {  // collected last-first
        const int32_t a = L.out_words[i];
        L.out_words[i] = L.out_words[nw - 1 - i];
        L.out_words[nw - 1 - i] = a;
      }
    info->nwords = nw;
    info->tb_fail = ok ? 0u : 1u;
    return;
  }
  if (blockIdx.y == 2) {
    // chip-wide mode (links swept, kept links and their frame offsets listed
    // by the chip-wide kernels), wide lattice: beta here while workgroup 0
    // computes alpha; Z from it
    const uint64_t nk = info->kept;
    if (!swept || nk <= 64 * ((uint64_t)T + 1) || nk > L.kept_cap) return;
    beta_wave<kLT>(L, g, sh, tid, swept, final_used, best_total);
    __syncthreads();
    if (tid == 0) info->Z = lattice_z(L, best_total, start_node_of(L, g));
    return;
  }

  // ------------------------------------------------ backward extra-cost sweep
  lstamp(1);
  if (!swept && !sweep_staged(L, g, sh, tid, par, final_used, best_total)) sweep_block(L, g, sh, tid, final_used, best_total);
  __syncthreads();
  lstamp(2);

  // ------------------------------------------ kept links (final merge input)
  const uint32_t lb_key = cost_key(prm.lattice_beam);
  uint64_t n_kept = info->kept;  // counted and listed by the chip-wide kernels when swept
  if (!swept) {
    // a contiguous range of links per thread (a multiple of four, so that
    // whole 16-byte groups of extra-cost keys are read at once), kBatchK
    // groups in flight together
    constexpr int kBatchK = 4;
    const uint64_t per = (((nlinks + kLT - 1) / kLT) + 3) & ~(uint64_t)3;
    const uint64_t k0 = tid * per < nlinks ? tid * per : nlinks;
    const uint64_t k1 = k0 + per < nlinks ? k0 + per : nlinks;
    // end of the whole groups (none when the lane's key array is not 16-byte aligned)
    const bool al = ((uintptr_t)L.le_key & 15u) == 0;
    const uint64_t k4 = al ? k0 + ((k1 - k0) & ~(uint64_t)3) : k0;
    const uint4* le4 = reinterpret_cast<const uint4*>(L.le_key);
    auto in = [&](uint32_t le) -> uint32_t { return le <= lb_key && le < kInfKey ? 1u : 0u; };
    uint64_t cnt = 0;
    for (uint64_t kb = k0; kb < k4; kb += 4 * kBatchK) {
      uint4 v[kBatchK];
#pragma unroll
      for (int u = 0; u < kBatchK; ++u) v[u] = kb + 4 * u < k4 ? le4[(kb >> 2) + u] : make_uint4(kInfKey, kInfKey, kInfKey, kInfKey);
#pragma unroll
      for (int u = 0; u < kBatchK; ++u) cnt += in(v[u].x) + in(v[u].y) + in(v[u].z) + in(v[u].w);
    }
    for (uint64_t k = k4; k < k1; ++k) cnt += in(L.le_key[k]);
    uint64_t pos = block_excl_scan64<kLW>(cnt, sh.bs, par, &n_kept);
    if (n_kept <= L.kept_cap && cnt) {
      for (uint64_t kb = k0; kb < k4; kb += 4 * kBatchK) {
        uint4 v[kBatchK];
#pragma unroll
        for (int u = 0; u < kBatchK; ++u) v[u] = kb + 4 * u < k4 ? le4[(kb >> 2) + u] : make_uint4(kInfKey, kInfKey, kInfKey, kInfKey);
#pragma unroll
        for (int u = 0; u < kBatchK; ++u) {
          const uint64_t k = kb + 4 * u;
          if (in(v[u].x)) L.kept_idx[pos++] = k;
          if (in(v[u].y)) L.kept_idx[pos++] = k + 1;
          if (in(v[u].z)) L.kept_idx[pos++] = k + 2;
          if (in(v[u].w)) L.kept_idx[pos++] = k + 3;
        }
      }
      for (uint64_t k = k4; k < k1; ++k)
        if (in(L.le_key[k])) L.kept_idx[pos++] = k;
    }
  }
  const bool debug = (prm.flags & 1u) != 0;
  if (n_kept > L.kept_cap || (debug && nlinks > L.raw_cap)) {
    if (tid == 0) {
      info->status = 4;
      info->overflow |= kOvfKept;
      info->kept = n_kept;
    }
    return;
  }
  __syncthreads();
  lstamp(3);
  const uint64_t* kid = L.kept_idx;
  // per frame t: kept links start at kf[2t], kept epsilon links at kf[2t+1];
  // frame t ends where frame t+1 starts
  uint64_t* kf = L.kframe;
  if (!swept) {  // (chip-wide mode lists them beside the kept links)
    for (int t = (int)tid; t <= T + 1; t += kLT) {
      kf[2 * t] = lower_bound64(kid, n_kept, L.link_off[t]);
      kf[2 * t + 1] = t <= T ? lower_bound64(kid, n_kept, L.link_xoff[t]) : n_kept;
    }
    __syncthreads();
  }
  if (!swept) {
    // records of the kept links for forward-backward (chip-wide mode writes
    // them while listing the kept links): a thread takes a contiguous range,
    // finds the frame of its first link and walks the frame boundaries
    const uint64_t per = (n_kept + kLT - 1) / kLT;
    const uint64_t j0 = tid * per < n_kept ? tid * per : n_kept;
    const uint64_t j1 = j0 + per < n_kept ? j0 + per : n_kept;
    if (j0 < j1) {
      int lo = 0, hi = T + 1;  // last t with kf[2t] <= j0 (kf[2(T+1)] = n_kept)
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (kf[2 * mid] <= j0) lo = mid;
        else hi = mid;
      }
      int t = lo;
      for (uint64_t j = j0; j < j1; ++j) {
        while (kf[2 * t + 2] <= j) ++t;
        L.post[j] = post_record(L, g, kid[j], t, j >= kf[2 * t + 1]);
      }
    }
    __syncthreads();
  }

  // ----------------------------------------------------- posteriors (fp64)
  lstamp(4);
  const uint64_t start_node = start_node_of(L, g);
  const bool wide = n_kept > 64 * ((uint64_t)T + 1);  // (more than 64 kept links per frame)
  // small kept lattices: alpha on wavefront 0 and beta on wavefront 1,
  // concurrently; large ones (more than 64 kept links per frame on average):
  // the whole workgroup, alpha then beta, or in chip-wide mode alpha here and
  // beta on the utterance's third workgroup at the same time
  if (!wide && !swept && compact_fits(L, g, n_kept, nnodes) &&
      posteriors_compact(L, g, sh, tid, par, n_kept, nnodes, start_node, final_used, best_total)) {
    // (done in LDS)
  } else if (!wide) {
    __syncthreads();  // (a compact attempt that did not fit has used the LDS)
    if (tid < 64) alpha_wave<64>(L, g, sh, tid, swept, start_node);
    else if (tid < 128) beta_wave<64>(L, g, sh, tid - 64, swept, final_used, best_total);
  } else {
    alpha_wave<kLT>(L, g, sh, tid, swept, start_node);
    if (!swept) {
      __syncthreads();
      beta_wave<kLT>(L, g, sh, tid, swept, final_used, best_total);
    }
  }
  __syncthreads();
  lstamp(5);
  // (with a wide lattice in chip-wide mode, the third workgroup writes Z;
  // the merge runs as a chip-wide kernel after this one)
  const double norm = swept ? 0.0 : post_norm(L, start_node);
  if (tid == 0) {
    info->final_used = final_used ? 1 : 0;
    info->kept = n_kept;
    info->out_raw = debug ? nlinks : 0;
    info->start_node = (uint32_t)start_node;
    info->best_node = (uint32_t)bnode;
    info->best_cost = best_total;
    if (!(swept && wide)) info->Z = lattice_z(L, best_total, start_node);
  }
  // used-node bitmap is zero on entry (cleared by the host before the launch)
  if (tid == 0) atomicOr(&L.used[start_node >> 5], 1u << (start_node & 31u));
  if (swept) return;  // the merge and the node list run as chip-wide kernels

  // ------------------------------------------- final merge of the kept links
  // (the frame offsets copied to LDS when they fit: each link's and node's
  // frame is found by a binary search over them)
  const uint64_t *lo_off = L.link_off, *xo_off = L.link_xoff, *kfo = L.kframe, *no = L.node_off;
  if ((uint64_t)T + 2 <= kMgFrames) {
    for (uint32_t i = tid; i < (uint32_t)(T + 2); i += kLT) {
      sh.w.mg.node_off[i] = L.node_off[i];
      sh.w.mg.link_off[i] = L.link_off[i];
      sh.w.mg.link_xoff[i] = L.link_xoff[i];
      sh.w.mg.kf[2 * i] = L.kframe[2 * i];
      sh.w.mg.kf[2 * i + 1] = L.kframe[2 * i + 1];
    }
    __syncthreads();
    lo_off = sh.w.mg.link_off;
    xo_off = sh.w.mg.link_xoff;
    kfo = sh.w.mg.kf;
    no = sh.w.mg.node_off;
  }
  assemble(L, g, false, n_kept, L.out_links, lb_key, norm, true, true, tid, kLT, lo_off, xo_off, kfo);
  if (debug) assemble(L, g, true, nlinks, L.out_raw, lb_key, norm, true, false, tid, kLT, lo_off, xo_off, kfo);
  __syncthreads();
  lstamp(6);
  const uint64_t n_out = write_nodes(L, nnodes, sh.bs, par, no);
  if (tid == 0) info->out_nodes = n_out;
  if (L.prof) {
    __syncthreads();
    lstamp(7);
  }
}

// Chip-wide merge of the kept links (and of every raw link with the debug
// flag), after the lattice kernel has produced the posteriors' inputs.
__global__ void __launch_bounds__(256) k_lat_assemble(DevGraph g, const LaneDesc* __restrict__ lanes, Params prm) {
  const LaneDesc& L = lanes[blockIdx.y];
  const LaneInfo* info = L.info;
  if (info->status != 0) return;
  const uint32_t lb_key = cost_key(prm.lattice_beam);
  const uint64_t first = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const double norm = post_norm(L, info->start_node);
  assemble(L, g, false, info->kept, L.out_links, lb_key, norm, true, true, first, stride, L.link_off, L.link_xoff,
           L.kframe);
  if (prm.flags & 1u)
    assemble(L, g, true, L.link_off[L.T + 1], L.out_raw, lb_key, norm, true, false, first, stride, L.link_off,
             L.link_xoff, L.kframe);
}

void launch_lattice(const DevGraph& g, const LaneDesc* lanes, int B, const Params& prm, hipStream_t s) {
  hipLaunchKernelGGL(k_lattice, dim3(B, (prm.flags & kFlagSwept) ? 3 : 2), dim3(kLT), 0, s, g, lanes, prm);
  if (prm.flags & kFlagSwept) {
    hipLaunchKernelGGL(k_lat_assemble, dim3(1024, B), dim3(256), 0, s, g, lanes, prm);
  }
}

}  // namespace wd
