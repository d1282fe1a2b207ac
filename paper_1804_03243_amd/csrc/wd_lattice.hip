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

// -log(exp(-a) + exp(-b)) accumulated atomically into *p (fp64).
__device__ __forceinline__ void atomic_logadd(double* p, double v) {
  if (!(v < INFINITY)) return;
  unsigned long long* a = reinterpret_cast<unsigned long long*>(p);
  unsigned long long old = *a;
  while (true) {
    const double o = __longlong_as_double((long long)old);
    double n;
    if (!(o < INFINITY)) n = v;
    else n = fmin(o, v) - log1p(exp(-fabs(o - v)));
    const unsigned long long prev = atomicCAS(a, old, (unsigned long long)__double_as_longlong(n));
    if (prev == old) break;
    old = prev;
  }
}

__device__ __forceinline__ float node_cost(const LaneDesc& L, uint64_t n) {
  return key_cost((uint32_t)(L.n_pack[n] >> 32));
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
__device__ __forceinline__ void assemble(const LaneDesc& L, const DevGraph& g, bool all, uint64_t n_sel,
                         OutLink* out, uint32_t lb_key, double Z, bool with_post, bool mark_nodes,
                         uint64_t first, uint64_t stride) {
  const int T = L.T;
  const uint64_t* kid = L.kept_idx;
  const uint64_t* kf = L.kframe;
  auto sel = [&](uint64_t j) -> uint64_t { return all ? j : kid[j]; };
  for (uint64_t j = first; j < n_sel; j += stride) {
    const uint64_t k = sel(j);
    const int t = (int)search_le64(L.link_off, (uint64_t)T + 2, k);
    const uint64_t xo = L.link_xoff[t];
    const bool eps = k >= xo;
    const uint64_t s0 = all ? L.link_off[t] : kf[2 * t];
    const uint64_t sx = all ? xo : kf[2 * t + 1];
    const uint64_t s1 = all ? L.link_off[t + 1] : kf[2 * t + 2];
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
    if (with_post && kept(L, k, lb_key))
      o.posterior = exp(Z - L.alpha[l.src] - (double)o.graph_cost - ac - L.beta[l.dst]);
    out[pos] = o;
    if (mark_nodes) {
      atomicOr(&L.used[l.src >> 5], 1u << (l.src & 31u));
      atomicOr(&L.used[l.dst >> 5], 1u << (l.dst & 31u));
    }
  }
}

// Lattice nodes (those marked in the used bitmap) in (t, state) order, which
// is node id order; returns their number.  Whole workgroup.
__device__ __forceinline__ uint64_t write_nodes(const LaneDesc& L, uint64_t nnodes, BlockScratch& bs, uint32_t& par) {
  const uint32_t tid = threadIdx.x;
  const uint64_t nwd = (nnodes + 31) >> 5;
  const uint64_t per = (nwd + kLT - 1) / kLT;
  const uint64_t w0 = tid * per < nwd ? tid * per : nwd;
  const uint64_t w1 = w0 + per < nwd ? w0 + per : nwd;
  uint64_t cnt = 0, n_out;
  for (uint64_t w = w0; w < w1; ++w) cnt += (uint64_t)__popc(L.used[w]);
  uint64_t pos = block_excl_scan64<kLW>(cnt, bs, par, &n_out);
  for (uint64_t w = w0; w < w1; ++w) {
    uint32_t word = L.used[w];
    while (word) {
      const uint32_t b = (uint32_t)__ffs(word) - 1u;
      word &= word - 1u;
      const uint64_t n = (w << 5) | b;
      OutNode o;
      o.t = (int32_t)search_le64(L.node_off, (uint64_t)L.T + 2, n);
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
struct SweepScal {
  uint64_t n0, n1, k0, k1, x0, x1;
  uint32_t mask;
};
__device__ __forceinline__ void sweep_scal(const LaneDesc& L, int t, SweepScal& a) {
  a.n0 = L.node_off[t];
  a.n1 = L.node_off[t + 1];
  a.x0 = L.link_xoff[t];
  a.x1 = L.link_off[t + 1];
  a.mask = L.xmask[t];
  a.k0 = t < L.T ? L.link_off[t + 1] : 0;
  a.k1 = t < L.T ? L.link_xoff[t + 1] : 0;
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

__device__ __forceinline__ void sweep_one(const LaneDesc& L, const SweepScal& a, uint32_t tid, SweepOne& it) {
  if (tid < a.k1 - a.k0) it.e = L.links[a.k0 + tid];
  if (tid < a.x1 - a.x0) {
    it.x = L.links[a.x0 + tid];
    it.lvl = L.link_lvl[a.x0 + tid];
  }
}

// Extra costs (+inf, or the final extra cost for the last frame) and costs
// of frame t's nodes, by threads first, first + stride, ...; c0: the cost key
// of node `first`, loaded ahead (kNoKeyAhead: load it here).
constexpr uint32_t kNoKeyAhead = 0u;
__device__ __forceinline__ void sweep_init(const LaneDesc& L, const DevGraph& g, LatShared& sh, int t,
                                           const SweepScal& a, uint32_t first, uint32_t stride, bool final_used,
                                           float best_total, uint32_t c0) {
  const uint64_t n0 = a.n0;
  const uint32_t nt = (uint32_t)(a.n1 - n0), buf = (uint32_t)t % 3u;
  const bool win = nt <= kWin;
  uint32_t* ex = win ? sh.w.p.ex[buf] : L.extra_key + n0;
  for (uint32_t i = first; i < nt; i += stride) {
    const float c = (i == first && c0 != kNoKeyAhead) ? key_cost(c0) : node_cost(L, n0 + i);
    uint32_t e = kInfKey;
    if (t == L.T) {
      const float F = final_used ? canon(c + g.final_w[L.n_state[n0 + i]]) : c;
      if (F < INFINITY) e = cost_key(F - best_total);
    }
    ex[i] = e;
    if (win) sh.w.p.cost[buf][i] = c;
  }
}

__device__ __forceinline__ void sweep_writeback(const LaneDesc& L, LatShared& sh, int t, const SweepScal& a,
                                                uint32_t first, uint32_t stride) {
  const uint32_t nt = (uint32_t)(a.n1 - a.n0);
  if (nt > kWin) return;  // relaxed in device memory directly
  const uint32_t* ex = sh.w.p.ex[(uint32_t)t % 3u];
  for (uint32_t i = first; i < nt; i += stride) L.extra_key[a.n0 + i] = ex[i];
}

// Frame t: `cur` holds this thread's links of frame t (loaded during frame
// t+1) and the cost key of its node of frame t-1 (loaded during t+1); frame
// t-1's links and frame t-2's node cost are loaded into `nxt` now.  The
// caller alternates two sets, so no register with a load in flight is copied.
__device__ __forceinline__ void sweep_step(const LaneDesc& L, const DevGraph& g, LatShared& sh, uint32_t tid, int t,
                                           bool final_used, float best_total, const SweepOne& cur,
                                           SweepOne& nxt) {
  const int T = L.T;
  SweepScal sa, sp{}, sn{};
  sweep_scal(L, t, sa);
  if (t < T) sweep_scal(L, t + 1, sp);
  if (t > 0) {
    sweep_scal(L, t - 1, sn);
    sweep_one(L, sn, tid, nxt);
  }
  nxt.c = kNoKeyAhead;
  if (t > 1 && tid >= 64) {
    const uint64_t m0 = L.node_off[t - 2], m1 = L.node_off[t - 1];
    if (tid - 64 < m1 - m0) nxt.c = (uint32_t)(L.n_pack[m0 + tid - 64] >> 32);
  }
  const uint64_t n0 = sa.n0, n1 = sa.n1;
  const uint32_t buf = (uint32_t)t % 3u;
  const bool win = n1 - n0 <= kWin;
  uint32_t* ex = win ? sh.w.p.ex[buf] : L.extra_key + n0;
  float* cw = win ? sh.w.p.cost[buf] : nullptr;
  if (sa.k1 > sa.k0) {
    const uint64_t m0 = n1;
    const bool wn = sp.n1 - m0 <= kWin;
    const uint32_t nb = (uint32_t)(t + 1) % 3u;
    const uint32_t* exn = wn ? sh.w.p.ex[nb] : L.extra_key + m0;
    const float* cn = wn ? sh.w.p.cost[nb] : nullptr;
    if (sa.k0 + tid < sa.k1) sweep_relax(L, sa.k0 + tid, cur.e, exn, cn, m0, ex, n0);
    for (uint64_t k = sa.k0 + tid + kLT; k < sa.k1; k += kLT) sweep_relax(L, k, L.links[k], exn, cn, m0, ex, n0);
  }
  __syncthreads();
  if (tid < 64) {
    if (sa.x1 > sa.x0)
      for (int lvl = (int)g.nlevels - 1; lvl >= 0; --lvl) {
        if (!level_present(sa.mask, (uint32_t)lvl)) continue;
        if (sa.x0 + tid < sa.x1 && cur.lvl == (uint32_t)lvl) sweep_relax(L, sa.x0 + tid, cur.x, ex, cw, n0, ex, n0);
        for (uint64_t k = sa.x0 + tid + 64; k < sa.x1; k += 64)
          if (L.link_lvl[k] == (uint8_t)lvl) sweep_relax(L, k, L.links[k], ex, cw, n0, ex, n0);
        wave_sync();
      }
  } else {
    if (t < T) sweep_writeback(L, sh, t + 1, sp, tid - 64, kLT - 64);
    if (t > 0) sweep_init(L, g, sh, t - 1, sn, tid - 64, kLT - 64, final_used, best_total, cur.c);
  }
  __syncthreads();
}

// Backward extra-cost sweep over every frame.
__device__ __forceinline__ void sweep_block(const LaneDesc& L, const DevGraph& g, LatShared& sh,
                                            uint32_t tid, bool final_used, float best_total) {
  const int T = L.T;
  SweepOne x{}, y{};
  {
    SweepScal s0;
    sweep_scal(L, T, s0);
    sweep_one(L, s0, tid, x);
    sweep_init(L, g, sh, T, s0, tid, kLT, final_used, best_total, kNoKeyAhead);
    // node cost of frame T-1 for the first step's initialisation
    x.c = kNoKeyAhead;
    if (T > 0 && tid >= 64) {
      const uint64_t m0 = L.node_off[T - 1], m1 = L.node_off[T];
      if (tid - 64 < m1 - m0) x.c = (uint32_t)(L.n_pack[m0 + tid - 64] >> 32);
    }
  }
  __syncthreads();
  for (int t = T; t >= 0; t -= 2) {
    sweep_step(L, g, sh, tid, t, final_used, best_total, x, y);
    if (t >= 1) sweep_step(L, g, sh, tid, t - 1, final_used, best_total, y, x);
  }
  SweepScal s0;
  sweep_scal(L, 0, s0);
  sweep_writeback(L, sh, 0, s0, tid, kLT);
}

// Kept link j for the forward-backward pass: {src node, dst node, graph cost
// bits, acoustic cost bits (emitting) or source level (epsilon)}.
__device__ __forceinline__ uint4 post_link(const LaneDesc& L, uint64_t j) { return L.post[j]; }

// Record of kept link j (link k) of frame t; `eps`: an epsilon link.
__device__ __forceinline__ uint4 post_record(const LaneDesc& L, const DevGraph& g, uint64_t k, int t, bool eps) {
  const uint4 v = L.links[k];
  uint32_t aux;
  if (eps) aux = L.link_lvl[k];
  else aux = __float_as_uint(-L.ll[(size_t)(t - 1) * g.P + (g.ilabel_id[v.x] - 1)]);
  return make_uint4(v.y, v.z, __float_as_uint(g.weight_id[v.x]), aux);
}

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

struct PostScal {
  uint64_t n0, n1, m0, m1, e0, e1, x0, x1;
  uint32_t mask;
};
struct PostItems {
  uint4 e[kAhead], x[kAhead];
  float fw[kAhead];
};

// Frame t of the alpha pass: emitting kept links into t (from t-1), epsilon
// kept links of t.
__device__ __forceinline__ void alpha_scal(const LaneDesc& L, int t, PostScal& a) {
  a.n0 = L.node_off[t];
  a.n1 = L.node_off[t + 1];
  a.m0 = t > 0 ? L.node_off[t - 1] : 0;
  a.e0 = L.kframe[2 * t];
  a.e1 = L.kframe[2 * t + 1];
  a.x0 = a.e1;
  a.x1 = L.kframe[2 * t + 2];
  a.mask = L.xmask[t];
}

// Frame t of the beta pass: emitting kept links out of t (into t+1), epsilon
// kept links of t.
__device__ __forceinline__ void beta_scal(const LaneDesc& L, int t, PostScal& a) {
  const int T = L.T;
  a.n0 = L.node_off[t];
  a.n1 = L.node_off[t + 1];
  a.m0 = t < T ? L.node_off[t + 1] : 0;
  a.m1 = t < T ? L.node_off[t + 2] : 0;
  a.e0 = t < T ? L.kframe[2 * t + 2] : 0;
  a.e1 = t < T ? L.kframe[2 * t + 3] : 0;
  a.x0 = L.kframe[2 * t + 1];
  a.x1 = L.kframe[2 * t + 2];
  a.mask = L.xmask[t];
}

// Items of a frame; `fin`: the last frame of the beta pass (final weights).
template <int GS>
__device__ __forceinline__ void post_items(const LaneDesc& L, const DevGraph& g, const PostScal& a, uint32_t lane,
                                           bool fin, PostItems& it) {
#pragma unroll
  for (int q = 0; q < kAhead; ++q) {
    const uint64_t i = lane + (uint64_t)GS * q;
    if (i < a.e1 - a.e0) it.e[q] = post_link(L, a.e0 + i);
    if (i < a.x1 - a.x0) it.x[q] = post_link(L, a.x0 + i);
    if (fin && i < a.n1 - a.n0) it.fw[q] = g.final_w[L.n_state[a.n0 + i]];
  }
}

// Frame t of the alpha pass on a group of GS threads (items of t in `cur`; those of
// t+1 are loaded into `nxt`).  `swept`: device-memory alpha is +inf already.
template <int GS>
__device__ __forceinline__ void alpha_step(const LaneDesc& L, const DevGraph& g, LatShared& sh, uint32_t lane,
                                           int t, bool swept, uint64_t start_node, const PostItems& cur,
                                           PostItems& nxt) {
  const int T = L.T;
  PostScal pa;
  alpha_scal(L, t, pa);
  if (t < T) {
    PostScal pb;
    alpha_scal(L, t + 1, pb);
    post_items<GS>(L, g, pb, lane, false, nxt);
  }
  const uint64_t n0 = pa.n0, n1 = pa.n1;
  const uint32_t nt = (uint32_t)(n1 - n0), buf = (uint32_t)t & 1u;
  const bool win = nt <= kWin;
  double* a = win ? sh.w.ab.a[buf] : L.alpha + n0;
  if (win || !swept) {
    for (uint32_t i = lane; i < nt; i += GS) a[i] = (n0 + i == start_node) ? 0.0 : INFINITY;
  } else if (lane == 0 && start_node >= n0 && start_node < n1) {
    a[start_node - n0] = 0.0;  // the rest is +inf already
  }
  group_sync<GS>();
  if (pa.e1 > pa.e0) {
    const uint64_t m0 = pa.m0;
    const bool wp = n0 - m0 <= kWin;
    const double* ap = wp ? sh.w.ab.a[buf ^ 1u] : L.alpha + m0;
    auto emit = [&](uint4 l) {
      const double av = wp ? ap[l.x - m0] : load_fresh(&ap[l.x - m0]);
      atomic_logadd(&a[l.y - n0], av + (double)__uint_as_float(l.z) + (double)__uint_as_float(l.w));
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
        if (l.w != lvl) return;
        const double av = win ? a[l.x - n0] : load_fresh(&a[l.x - n0]);
        atomic_logadd(&a[l.y - n0], av + (double)__uint_as_float(l.z));
      };
#pragma unroll
      for (int q = 0; q < kAhead; ++q)
        if (pa.x0 + lane + (uint64_t)GS * q < pa.x1) eps(cur.x[q]);
      post_tail<GS>(L, pa.x0, pa.x1, lane, eps);
      group_sync<GS>();
    }
  if (win)
    for (uint32_t i = lane; i < nt; i += GS) L.alpha[n0 + i] = a[i];
}

// alpha over every frame, ascending; epsilon links of a frame by source
// level, on GS threads.
template <int GS>
__device__ __forceinline__ void alpha_wave(const LaneDesc& L, const DevGraph& g, LatShared& sh, uint32_t lane,
                                           bool swept, uint64_t start_node) {
  const int T = L.T;
  PostItems x{}, y{};
  {
    PostScal p0;
    alpha_scal(L, 0, p0);
    post_items<GS>(L, g, p0, lane, false, x);
  }
  for (int t = 0; t <= T; t += 2) {
    alpha_step<GS>(L, g, sh, lane, t, swept, start_node, x, y);
    if (t + 1 <= T) alpha_step<GS>(L, g, sh, lane, t + 1, swept, start_node, y, x);
  }
}

// Frame t of the beta pass on a group of GS threads (items of t in `cur`; those of
// t-1 are loaded into `nxt`).
template <int GS>
__device__ __forceinline__ void beta_step(const LaneDesc& L, const DevGraph& g, LatShared& sh, uint32_t lane,
                                          int t, bool swept, bool final_used, const PostItems& cur, PostItems& nxt) {
  const int T = L.T;
  PostScal pa;
  beta_scal(L, t, pa);
  if (t > 0) {
    PostScal pb;
    beta_scal(L, t - 1, pb);
    post_items<GS>(L, g, pb, lane, false, nxt);
  }
  const uint64_t n0 = pa.n0, n1 = pa.n1;
  const uint32_t nt = (uint32_t)(n1 - n0), buf = (uint32_t)t & 1u;
  const bool win = nt <= kWin;
  double* b = win ? sh.w.ab.b[buf] : L.beta + n0;
  if (win || !swept || t == T) {
#pragma unroll
    for (int q = 0; q <= kAhead; ++q)
      for (uint32_t i = lane + (uint32_t)(GS * q); i < nt; i += (q < kAhead ? nt : (uint32_t)GS)) {
        double v = INFINITY;
        if (t == T)
          v = final_used ? (double)(q < kAhead ? cur.fw[q < kAhead ? q : 0] : g.final_w[L.n_state[n0 + i]]) : 0.0;
        b[i] = v;
      }
  }
  group_sync<GS>();
  if (pa.e1 > pa.e0) {
    const uint64_t m0 = pa.m0;
    const bool wn = pa.m1 - m0 <= kWin;
    const double* bn = wn ? sh.w.ab.b[buf ^ 1u] : L.beta + m0;
    auto emit = [&](uint4 l) {
      const double bv = wn ? bn[l.y - m0] : load_fresh(&bn[l.y - m0]);
      atomic_logadd(&b[l.x - n0], (double)__uint_as_float(l.z) + (double)__uint_as_float(l.w) + bv);
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
        if (l.w != (uint32_t)lvl) return;
        const double bv = win ? b[l.y - n0] : load_fresh(&b[l.y - n0]);
        atomic_logadd(&b[l.x - n0], (double)__uint_as_float(l.z) + bv);
      };
#pragma unroll
      for (int q = 0; q < kAhead; ++q)
        if (pa.x0 + lane + (uint64_t)GS * q < pa.x1) eps(cur.x[q]);
      post_tail<GS>(L, pa.x0, pa.x1, lane, eps);
      group_sync<GS>();
    }
  if (win)
    for (uint32_t i = lane; i < nt; i += GS) L.beta[n0 + i] = b[i];
}

// beta over every frame, descending; epsilon links of a frame from the
// highest source level, on GS threads.
template <int GS>
__device__ __forceinline__ void beta_wave(const LaneDesc& L, const DevGraph& g, LatShared& sh, uint32_t lane,
                                          bool swept, bool final_used) {
  const int T = L.T;
  PostItems x{}, y{};
  {
    PostScal p0;
    beta_scal(L, T, p0);
    post_items<GS>(L, g, p0, lane, final_used, x);
  }
  for (int t = T; t >= 0; t -= 2) {
    beta_step<GS>(L, g, sh, lane, t, swept, final_used, x, y);
    if (t >= 1) beta_step<GS>(L, g, sh, lane, t - 1, swept, final_used, y, x);
  }
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

  // ------------------------------------------------ backward extra-cost sweep
  if (!swept) sweep_block(L, g, sh, tid, final_used, best_total);
  __syncthreads();

  // ------------------------------------------ kept links (final merge input)
  const uint32_t lb_key = cost_key(prm.lattice_beam);
  uint64_t n_kept = info->kept;  // counted and listed by the chip-wide kernels when swept
  if (!swept) {
    const uint64_t per = (nlinks + kLT - 1) / kLT;
    const uint64_t k0 = tid * per < nlinks ? tid * per : nlinks;
    const uint64_t k1 = k0 + per < nlinks ? k0 + per : nlinks;
    uint64_t cnt = 0;
    for (uint64_t k = k0; k < k1; ++k) cnt += kept(L, k, lb_key);
    uint64_t pos = block_excl_scan64<kLW>(cnt, sh.bs, par, &n_kept);
    if (n_kept <= L.kept_cap)
      for (uint64_t k = k0; k < k1; ++k)
        if (kept(L, k, lb_key)) L.kept_idx[pos++] = k;
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
  const uint64_t* kid = L.kept_idx;
  // per frame t: kept links start at kf[2t], kept epsilon links at kf[2t+1];
  // frame t ends where frame t+1 starts
  uint64_t* kf = L.kframe;
  for (int t = (int)tid; t <= T + 1; t += kLT) {
    kf[2 * t] = lower_bound64(kid, n_kept, L.link_off[t]);
    kf[2 * t + 1] = t <= T ? lower_bound64(kid, n_kept, L.link_xoff[t]) : n_kept;
  }
  __syncthreads();
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
  uint64_t start_node = 0;
  {
    // the start state among frame 0's tokens (sorted by state)
    uint64_t lo = 0, hi = L.node_off[1];
    while (lo < hi) {
      const uint64_t mid = (lo + hi) >> 1;
      if (L.n_state[mid] < g.start) lo = mid + 1;
      else hi = mid;
    }
    start_node = lo;
  }
  // small kept lattices: alpha on wavefront 0 and beta on wavefront 1,
  // concurrently; large ones (more than 64 kept links per frame on average):
  // the whole workgroup, alpha then beta
  if (n_kept <= 64 * ((uint64_t)T + 1)) {
    if (tid < 64) alpha_wave<64>(L, g, sh, tid, swept, start_node);
    else if (tid < 128) beta_wave<64>(L, g, sh, tid - 64, swept, final_used);
  } else {
    alpha_wave<kLT>(L, g, sh, tid, swept, start_node);
    __syncthreads();
    beta_wave<kLT>(L, g, sh, tid, swept, final_used);
  }
  __syncthreads();
  const double Z = L.beta[start_node];
  if (tid == 0) {
    info->final_used = final_used ? 1 : 0;
    info->kept = n_kept;
    info->out_raw = debug ? nlinks : 0;
    info->start_node = (uint32_t)start_node;
    info->best_node = (uint32_t)bnode;
    info->best_cost = best_total;
    info->Z = Z;
  }
  // used-node bitmap is zero on entry (cleared by the host before the launch)
  if (tid == 0) atomicOr(&L.used[start_node >> 5], 1u << (start_node & 31u));
  if (swept) return;  // the merge and the node list run as chip-wide kernels

  // ------------------------------------------- final merge of the kept links
  assemble(L, g, false, n_kept, L.out_links, lb_key, Z, true, true, tid, kLT);
  if (debug) assemble(L, g, true, nlinks, L.out_raw, lb_key, Z, true, false, tid, kLT);
  __syncthreads();
  const uint64_t n_out = write_nodes(L, nnodes, sh.bs, par);
  if (tid == 0) info->out_nodes = n_out;
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
  assemble(L, g, false, info->kept, L.out_links, lb_key, info->Z, true, true, first, stride);
  if (prm.flags & 1u)
    assemble(L, g, true, L.link_off[L.T + 1], L.out_raw, lb_key, info->Z, true, false, first, stride);
}

void launch_lattice(const DevGraph& g, const LaneDesc* lanes, int B, const Params& prm, hipStream_t s) {
  hipLaunchKernelGGL(k_lattice, dim3(B, 2), dim3(kLT), 0, s, g, lanes, prm);
  if (prm.flags & kFlagSwept) {
    hipLaunchKernelGGL(k_lat_assemble, dim3(1024, B), dim3(256), 0, s, g, lanes, prm);
  }
}

}  // namespace wd
