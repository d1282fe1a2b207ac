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

// Two-frame window of per-node values (frame t and t+1, or t-1 and t): extra
// costs and costs during the pruning sweep, alpha or beta during the
// posteriors.  Frames with more nodes use the workspace arrays directly.
struct LatShared {
  BlockScratch bs;
  union {
    struct {
      uint32_t ex[2][kWin];
      float cost[2][kWin];
    } p;
    double ab[2][kWin];
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
__device__ void assemble(const LaneDesc& L, const DevGraph& g, bool all, uint64_t n_sel,
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
__device__ uint64_t write_nodes(const LaneDesc& L, uint64_t nnodes, BlockScratch& bs, uint32_t& par) {
  const uint32_t tid = threadIdx.x;
  const uint64_t nwd = (nnodes + 31) >> 5;
  const uint64_t per = (nwd + kThreads - 1) / kThreads;
  const uint64_t w0 = tid * per < nwd ? tid * per : nwd;
  const uint64_t w1 = w0 + per < nwd ? w0 + per : nwd;
  uint64_t cnt = 0, n_out;
  for (uint64_t w = w0; w < w1; ++w) cnt += (uint64_t)__popc(L.used[w]);
  uint64_t pos = block_excl_scan64(cnt, bs, par, &n_out);
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

// blockIdx.y == 0: pruning, posteriors and the final merge; blockIdx.y == 1:
// the 1-best traceback (a serial walk over predecessor pointers, run
// concurrently by its own workgroup).
__global__ void __launch_bounds__(kThreads) k_lattice(DevGraph g, const LaneDesc* __restrict__ lanes,
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
      for (uint64_t n = nT0 + tid; n < nT1; n += kThreads) {
        const float fw = g.final_w[L.n_state[n]];
        const float c = node_cost(L, n);
        any |= (fw < INFINITY && (c + fw) < INFINITY) ? 1u : 0u;
      }
    final_used = block_or(any, sh.bs, par) != 0;
    uint64_t m = kEmpty;
    for (uint64_t n = nT0 + tid; n < nT1; n += kThreads) {
      const float c = node_cost(L, n);
      const float F = final_used ? canon(c + g.final_w[L.n_state[n]]) : c;
      const uint64_t v = pack_tok(cost_key(F), (uint32_t)(n - nT0));
      m = v < m ? v : m;
    }
    m = block_min64(m, sh.bs, par);
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
  for (int t = swept ? -1 : T; t >= 0; --t) {
    const uint64_t n0 = L.node_off[t], n1 = L.node_off[t + 1];
    const uint32_t nt = (uint32_t)(n1 - n0), buf = (uint32_t)t & 1u;
    const bool win = nt <= kWin;
    uint32_t* ex = win ? sh.w.p.ex[buf] : L.extra_key + n0;
    for (uint32_t i = tid; i < nt; i += kThreads) {
      const float c = node_cost(L, n0 + i);
      uint32_t e = kInfKey;
      if (t == T) {
        const float F = final_used ? canon(c + g.final_w[L.n_state[n0 + i]]) : c;
        if (F < INFINITY) e = cost_key(F - best_total);
      }
      ex[i] = e;
      if (win) sh.w.p.cost[buf][i] = c;
    }
    __syncthreads();
    // extra(link) = extra(dst) + (x - cost(dst)); extra(src) = min over links
    auto relax = [&](uint64_t k, const uint32_t* exd, const float* cd, uint64_t d0) {
      const LinkView l = link_at(L, k);
      const uint64_t d = l.dst - d0;
      const float c = cd ? cd[d] : node_cost(L, l.dst);
      const uint32_t le = cost_key(key_cost(exd[d]) + (l.x - c));
      L.le_key[k] = le;
      atomicMin(&ex[l.src - n0], le);
    };
    if (t < T) {
      const uint64_t k0 = L.link_off[t + 1], k1 = L.link_xoff[t + 1];
      if (k1 > k0) {
        const uint64_t m0 = L.node_off[t + 1];
        const bool wn = L.node_off[t + 2] - m0 <= kWin;
        const uint32_t* exn = wn ? sh.w.p.ex[buf ^ 1u] : L.extra_key + m0;
        const float* cn = wn ? sh.w.p.cost[buf ^ 1u] : nullptr;
        for (uint64_t k = k0 + tid; k < k1; k += kThreads) relax(k, exn, cn, m0);
        __syncthreads();
      }
    }
    const uint64_t x0 = L.link_xoff[t], x1 = L.link_off[t + 1];
    const uint32_t mask = L.xmask[t];
    if (x1 > x0)
      for (int lvl = (int)g.nlevels - 1; lvl >= 0; --lvl) {
        if (!level_present(mask, (uint32_t)lvl)) continue;
        for (uint64_t k = x0 + tid; k < x1; k += kThreads)
          if (L.link_lvl[k] == (uint8_t)lvl) relax(k, ex, win ? sh.w.p.cost[buf] : nullptr, n0);
        __syncthreads();
      }
    if (win)
      for (uint32_t i = tid; i < nt; i += kThreads) L.extra_key[n0 + i] = ex[i];
  }
  __syncthreads();

  // ------------------------------------------ kept links (final merge input)
  const uint32_t lb_key = cost_key(prm.lattice_beam);
  uint64_t n_kept = info->kept;  // counted and listed by the chip-wide kernels when swept
  if (!swept) {
    const uint64_t per = (nlinks + kThreads - 1) / kThreads;
    const uint64_t k0 = tid * per < nlinks ? tid * per : nlinks;
    const uint64_t k1 = k0 + per < nlinks ? k0 + per : nlinks;
    uint64_t cnt = 0;
    for (uint64_t k = k0; k < k1; ++k) cnt += kept(L, k, lb_key);
    uint64_t pos = block_excl_scan64(cnt, sh.bs, par, &n_kept);
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
  for (int t = (int)tid; t <= T + 1; t += kThreads) {
    kf[2 * t] = lower_bound64(kid, n_kept, L.link_off[t]);
    kf[2 * t + 1] = t <= T ? lower_bound64(kid, n_kept, L.link_xoff[t]) : n_kept;
  }
  __syncthreads();

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
  // alpha: frames ascending, epsilon links of a frame by source level
  for (int t = 0; t <= T; ++t) {
    const uint64_t n0 = L.node_off[t], n1 = L.node_off[t + 1];
    const uint32_t nt = (uint32_t)(n1 - n0), buf = (uint32_t)t & 1u;
    const bool win = nt <= kWin;
    double* a = win ? sh.w.ab[buf] : L.alpha + n0;
    if (win || !swept) {
      for (uint32_t i = tid; i < nt; i += kThreads) a[i] = (n0 + i == start_node) ? 0.0 : INFINITY;
    } else if (tid == 0 && start_node >= n0 && start_node < n1) {
      a[start_node - n0] = 0.0;  // the rest is +inf already
    }
    __syncthreads();
    const uint64_t e0 = kf[2 * t], e1 = kf[2 * t + 1], e2 = kf[2 * t + 2];
    if (e1 > e0) {
      const uint64_t m0 = L.node_off[t - 1];
      const double* ap = (n0 - m0 <= kWin) ? sh.w.ab[buf ^ 1u] : L.alpha + m0;
      for (uint64_t j = e0 + tid; j < e1; j += kThreads) {
        const LinkView l = link_at(L, kid[j]);
        atomic_logadd(&a[l.dst - n0], ap[l.src - m0] + (double)g.weight_id[l.arc] + link_ac(L, g, t, l.arc));
      }
      __syncthreads();
    }
    if (e2 > e1) {
      const uint32_t mask = L.xmask[t];
      for (uint32_t lvl = 0; lvl < g.nlevels; ++lvl) {
        if (!level_present(mask, lvl)) continue;
        for (uint64_t j = e1 + tid; j < e2; j += kThreads) {
          const uint64_t k = kid[j];
          if (L.link_lvl[k] != (uint8_t)lvl) continue;
          const LinkView l = link_at(L, k);
          atomic_logadd(&a[l.dst - n0], a[l.src - n0] + (double)g.weight_id[l.arc]);
        }
        __syncthreads();
      }
    }
    if (win)
      for (uint32_t i = tid; i < nt; i += kThreads) L.alpha[n0 + i] = a[i];
  }
  __syncthreads();
  // beta: frames descending, epsilon links of a frame from the highest level
  for (int t = T; t >= 0; --t) {
    const uint64_t n0 = L.node_off[t], n1 = L.node_off[t + 1];
    const uint32_t nt = (uint32_t)(n1 - n0), buf = (uint32_t)t & 1u;
    const bool win = nt <= kWin;
    double* b = win ? sh.w.ab[buf] : L.beta + n0;
    if (win || !swept || t == T)
      for (uint32_t i = tid; i < nt; i += kThreads)
        b[i] = t == T ? (final_used ? (double)g.final_w[L.n_state[n0 + i]] : 0.0) : INFINITY;
    __syncthreads();
    if (t < T) {
      const uint64_t e0 = kf[2 * t + 2], e1 = kf[2 * t + 3];
      if (e1 > e0) {
        const uint64_t m0 = L.node_off[t + 1];
        const double* bn = (L.node_off[t + 2] - m0 <= kWin) ? sh.w.ab[buf ^ 1u] : L.beta + m0;
        for (uint64_t j = e0 + tid; j < e1; j += kThreads) {
          const LinkView l = link_at(L, kid[j]);
          atomic_logadd(&b[l.src - n0],
                        (double)g.weight_id[l.arc] + link_ac(L, g, t + 1, l.arc) + bn[l.dst - m0]);
        }
        __syncthreads();
      }
    }
    const uint64_t e1 = kf[2 * t + 1], e2 = kf[2 * t + 2];
    if (e2 > e1) {
      const uint32_t mask = L.xmask[t];
      for (int lvl = (int)g.nlevels - 1; lvl >= 0; --lvl) {
        if (!level_present(mask, (uint32_t)lvl)) continue;
        for (uint64_t j = e1 + tid; j < e2; j += kThreads) {
          const uint64_t k = kid[j];
          if (L.link_lvl[k] != (uint8_t)lvl) continue;
          const LinkView l = link_at(L, k);
          atomic_logadd(&b[l.src - n0], (double)g.weight_id[l.arc] + b[l.dst - n0]);
        }
        __syncthreads();
      }
    }
    if (win)
      for (uint32_t i = tid; i < nt; i += kThreads) L.beta[n0 + i] = b[i];
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
  assemble(L, g, false, n_kept, L.out_links, lb_key, Z, true, true, tid, kThreads);
  if (debug) assemble(L, g, true, nlinks, L.out_raw, lb_key, Z, true, false, tid, kThreads);
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
  hipLaunchKernelGGL(k_lattice, dim3(B, 2), dim3(kThreads), 0, s, g, lanes, prm);
  if (prm.flags & kFlagSwept) {
    hipLaunchKernelGGL(k_lat_assemble, dim3(1024, B), dim3(256), 0, s, g, lanes, prm);
  }
}

}  // namespace wd
