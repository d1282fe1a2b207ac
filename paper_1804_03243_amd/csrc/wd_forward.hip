// Forward pass: frame-synchronous token passing for one utterance per
// workgroup, every frame and every phase inside one persistent launch.
//
// Per frame t (Sec. 3.2-3.4 of the paper, with the readings stated in the
// oracle): emitting expansion of the surviving tokens of frame t-1 over a flat,
// prefix-sum load-balanced arc work space (Sec. 3.3 static load balancing);
// recombination by a 64-bit atomicMin of (cost key, arc id) on the state's
// slot (Alg. 1); beam cutoff from the best emitting candidate; epsilon closure
// one epsilon level at a time; exact max-active cutoff by radix select over an
// LDS histogram; compaction of the survivors into a frontier sorted by state
// (which numbers the lattice nodes (t, i) of Sec. 3.5); lattice links for every
// surviving token-passing operation (Sec. 3.4).
#include "wd_block.h"

namespace wd {

struct FwdShared {
  BlockScratch bs;
  uint32_t n_touched;
  uint32_t n_surv;
  uint32_t n_rank;
  uint32_t sel_b;
  uint32_t sel_before;
  uint32_t nb[kMaxLevels + 1];
  uint32_t hist[kHistBins];
  uint32_t rs_state[kRankMax];
  unsigned long long rs_pack[kRankMax];
};

// Record a first touch of `dst` this frame: touched list (ballot-aggregated)
// and, if the state has epsilon out-arcs, the bucket of its epsilon level.
__device__ __forceinline__ void note_touch(bool first, uint32_t dst, uint32_t cls, FwdShared& sh,
                                           const DevGraph& g, const LaneDesc& L) {
  uint32_t pos = wave_append(first, &sh.n_touched);
  if (first) {
    if (pos < L.frame_cap) L.touched[pos] = dst;
    if (cls != kNoEps) {
      uint32_t b = atomicAdd(&sh.nb[cls], 1u);
      L.bucket[g.level_base[cls] + b] = dst;
    }
  }
}

// Same, for callers whose lanes are not converged (per-thread LDS atomics).
__device__ __forceinline__ void note_touch_div(uint32_t dst, uint32_t cls, FwdShared& sh,
                                               const DevGraph& g, const LaneDesc& L) {
  uint32_t pos = atomicAdd(&sh.n_touched, 1u);
  if (pos < L.frame_cap) L.touched[pos] = dst;
  if (cls != kNoEps) {
    uint32_t b = atomicAdd(&sh.nb[cls], 1u);
    L.bucket[g.level_base[cls] + b] = dst;
  }
}

// Find the bin holding the rank-th smallest key in sh.hist (1-based rank).
__device__ __forceinline__ void select_bin(uint32_t rank, FwdShared& sh, uint32_t* bin,
                                           uint32_t* before, uint32_t* count) {
  const uint32_t tid = threadIdx.x;
  uint32_t h0 = sh.hist[2 * tid], h1 = sh.hist[2 * tid + 1];
  uint32_t tot;
  uint32_t ex = block_excl_scan(h0 + h1, sh.bs, &tot);
  if (ex < rank && rank <= ex + h0) {
    sh.sel_b = 2 * tid;
    sh.sel_before = ex;
  } else if (ex + h0 < rank && rank <= ex + h0 + h1) {
    sh.sel_b = 2 * tid + 1;
    sh.sel_before = ex + h0;
  }
  __syncthreads();
  *bin = sh.sel_b;
  *before = sh.sel_before;
  *count = sh.hist[sh.sel_b];
  __syncthreads();
}

__global__ void __launch_bounds__(kThreads) k_forward(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                      Params prm, const uint32_t* __restrict__ bad) {
  __shared__ FwdShared sh;
  const LaneDesc& L = lanes[blockIdx.x];
  const uint32_t tid = threadIdx.x;
  if (bad[blockIdx.x]) {
    if (tid == 0) L.info->status = 1;  // WD_EINVAL
    return;
  }
  const int T = L.T;
  const uint32_t P = g.P;

  for (uint32_t i = tid; i <= (uint32_t)kMaxLevels; i += kThreads) sh.nb[i] = 0;
  for (uint32_t i = tid; i < (uint32_t)kHistBins; i += kThreads) sh.hist[i] = 0;
  if (tid == 0) {
    sh.n_touched = 0;
    sh.n_surv = 0;
    sh.n_rank = 0;
  }
  __syncthreads();
  // frame 0: the start token (cost 0, no predecessor)
  if (tid == 0) {
    const uint32_t s0 = g.start;
    L.slot[s0] = pack_tok(cost_key(0.0f), kNoArc);
    L.touched[0] = s0;
    sh.n_touched = 1;
    const uint32_t c = g.sclass[s0];
    if (c != kNoEps) {
      L.bucket[g.level_base[c]] = s0;
      sh.nb[c] = 1;
    }
  }
  __syncthreads();

  int status = 0;  // WD_OK
  uint32_t ovf = 0;
  uint32_t best_key = cost_key(0.0f);
  uint64_t node_base = 0, node_base_prev = 0, link_base = 0;
  uint32_t n_prev = 0, W = 0;
  int cur = 0;
  uint64_t my_arcs = 0, my_eps = 0, tokens = 0, max_tokens = 0, need_frame = 1, need_arcs = 0;
  bool hist_ok = true;  // history (nodes, links) still being stored
  int t = 0;

  for (t = 0; t <= T; ++t) {
    // ------------------------------------------------ emitting expansion
    if (t > 0) {
      need_arcs = W > need_arcs ? W : need_arcs;
      if (W > L.cand_cap) {
        status = 4;  // WD_ECAPACITY
        ovf |= kOvfArcs;
        break;
      }
      if (tid == 0) my_arcs += W;
      const int pb = cur ^ 1;
      const uint32_t* fs = L.f_state[pb];
      const uint32_t* fk = L.f_key[pb];
      const uint32_t* fe = L.f_edeg[pb];
      const float* row = L.ll + (size_t)(t - 1) * P;
      uint32_t my_best = 0xffffffffu;
      for (uint32_t base = 0; base < W; base += kThreads) {
        const uint32_t w = base + tid;
        bool first = false;
        uint32_t dst = 0, cls = kNoEps;
        if (w < W) {
          const uint32_t i = search_le(fe, n_prev, w);
          const uint32_t s = fs[i];
          const float c = key_cost(fk[i]);
          const uint4 r = g.earc[g.off[s].x + (w - fe[i])];
          dst = r.x;
          cls = r.z >> 24;
          const float ac = -row[(r.z & 0xffffffu) - 1u];
          float x = c + ac;
          x = canon(x + __uint_as_float(r.y));
          const uint32_t xk = cost_key(x);
          if (xk < kInfKey) {
            const unsigned long long old = atomicMin(&L.slot[dst], pack_tok(xk, r.w));
            first = old == kEmpty;
            my_best = xk < my_best ? xk : my_best;
          }
          L.cand[w] = make_uint4(r.w, (uint32_t)(node_base_prev + i), dst, __float_as_uint(x));
        }
        note_touch(first, dst, cls, sh, g, L);
      }
      best_key = (uint32_t)block_min64(my_best, sh.bs);
      if (best_key >= kInfKey) {
        status = 3;  // WD_ENOPATH
        break;
      }
    }
    // --------------------------------------------- beam cutoff, epsilon levels
    const float best = key_cost(best_key);
    const float cutb = best + prm.beam;
    const uint32_t kcutb = cost_key(cutb);
    for (uint32_t lvl = 0; lvl < g.nlevels; ++lvl) {
      const uint32_t n = sh.nb[lvl];
      const uint32_t* bk = L.bucket + g.level_base[lvl];
      for (uint32_t i = tid; i < n; i += kThreads) {
        const uint32_t s = bk[i];
        const uint32_t k = (uint32_t)(L.slot[s] >> 32);
        if (k > kcutb) continue;
        const float c = key_cost(k);
        const uint32_t a0 = g.off[s].y, a1 = g.off[s + 1].y;
        my_eps += a1 - a0;
        for (uint32_t a = a0; a < a1; ++a) {
          const uint4 r = g.xarc[a];
          const float x = canon(c + __uint_as_float(r.y));
          const uint32_t xk = cost_key(x);
          if (xk > kcutb || xk >= kInfKey) continue;
          const unsigned long long old = atomicMin(&L.slot[r.x], pack_tok(xk, r.w));
          if (old == kEmpty) note_touch_div(r.x, r.z, sh, g, L);
        }
      }
      __syncthreads();
    }
    // ------------------------------------ survivors of the beam cutoff + histogram
    const uint32_t nt = sh.n_touched;
    need_frame = nt > need_frame ? nt : need_frame;
    if (nt > L.frame_cap) {
      status = 4;
      ovf |= kOvfFrame;
      break;
    }
    const uint32_t span = kcutb - best_key;
    const uint32_t nbits = span ? 32u - (uint32_t)__clz(span) : 0u;
    uint32_t shift = nbits > 11u ? nbits - 11u : 0u;
    for (uint32_t base = 0; base < nt; base += kThreads) {
      const uint32_t i = base + tid;
      bool keep = false;
      uint32_t s = 0;
      unsigned long long v = kEmpty;
      if (i < nt) {
        s = L.touched[i];
        v = L.slot[s];
        L.slot[s] = kEmpty;
        keep = (uint32_t)(v >> 32) <= kcutb;
      }
      const uint32_t pos = wave_append(keep, &sh.n_surv);
      if (keep) {
        L.surv_state[pos] = s;
        L.surv_pack[pos] = v;
        atomicAdd(&sh.hist[((uint32_t)(v >> 32) - best_key) >> shift], 1u);
      }
    }
    __syncthreads();
    const uint32_t ns = sh.n_surv;
    // ------------------------------------------------ max-active cutoff
    uint32_t cut_key = kcutb;
    uint32_t n_keep = ns;
    if (prm.max_active > 0 && ns > (uint32_t)prm.max_active) {
      uint32_t rank = (uint32_t)prm.max_active, prefix = 0, less = 0;
      uint32_t bits = nbits - shift;
      while (true) {
        uint32_t b, before, cnt;
        select_bin(rank, sh, &b, &before, &cnt);
        prefix = (prefix << bits) | b;
        less += before;
        rank -= before;
        if (shift == 0) {
          n_keep = less + cnt;
          break;
        }
        const uint32_t nsh = shift > 11u ? shift - 11u : 0u;
        bits = shift - nsh;
        for (uint32_t i = tid; i < (uint32_t)kHistBins; i += kThreads) sh.hist[i] = 0;
        __syncthreads();
        for (uint32_t i = tid; i < ns; i += kThreads) {
          const uint32_t d = (uint32_t)(L.surv_pack[i] >> 32) - best_key;
          if ((d >> shift) == prefix) atomicAdd(&sh.hist[(d >> nsh) & ((1u << bits) - 1u)], 1u);
        }
        shift = nsh;
        __syncthreads();
      }
      const uint32_t vkey = best_key + prefix;
      cut_key = vkey < kcutb ? vkey : kcutb;
    }
    // -------------------------------- compaction into a frontier sorted by state
    uint32_t* fs = L.f_state[cur];
    uint32_t* fk = L.f_key[cur];
    if (hist_ok && node_base + n_keep > L.node_cap) {
      hist_ok = false;
      ovf |= kOvfNodes;
    }
    auto place = [&](uint32_t p, uint32_t s, unsigned long long v) {
      const uint64_t node = node_base + p;
      if (hist_ok) {
        L.n_state[node] = s;
        L.n_pack[node] = v;
        L.n_pred[node] = kNoArc;
      }
      L.idx[s] = (uint32_t)node;
      fs[p] = s;
      fk[p] = (uint32_t)(v >> 32);
    };
    if (n_keep <= (uint32_t)kRankMax) {
      for (uint32_t base = 0; base < ns; base += kThreads) {
        const uint32_t i = base + tid;
        bool keep = false;
        uint32_t s = 0;
        unsigned long long v = 0;
        if (i < ns) {
          v = L.surv_pack[i];
          s = L.surv_state[i];
          keep = (uint32_t)(v >> 32) <= cut_key;
        }
        const uint32_t pos = wave_append(keep, &sh.n_rank);
        if (keep && pos < (uint32_t)kRankMax) {
          sh.rs_state[pos] = s;
          sh.rs_pack[pos] = v;
        }
      }
      __syncthreads();
      if (sh.n_rank != n_keep) {
        status = kStatusInternal;
        break;
      }
      for (uint32_t j = tid; j < n_keep; j += kThreads) {
        const uint32_t s = sh.rs_state[j];
        uint32_t r = 0;
        for (uint32_t q = 0; q < n_keep; ++q) r += sh.rs_state[q] < s;
        place(r, s, sh.rs_pack[j]);
      }
    } else {
      for (uint32_t i = tid; i < ns; i += kThreads) {
        const unsigned long long v = L.surv_pack[i];
        if ((uint32_t)(v >> 32) <= cut_key) {
          const uint32_t s = L.surv_state[i];
          L.idx[s] = i;
          atomicOr(&L.bitmap[s >> 5], 1u << (s & 31u));
        }
      }
      __syncthreads();
      const uint32_t nw = (g.S + 31u) >> 5;
      const uint32_t per = (nw + kThreads - 1) / kThreads;
      const uint32_t w0 = tid * per < nw ? tid * per : nw;
      const uint32_t w1 = w0 + per < nw ? w0 + per : nw;
      uint32_t cnt = 0;
      for (uint32_t w = w0; w < w1; ++w) cnt += (uint32_t)__popc(L.bitmap[w]);
      uint32_t tot;
      uint32_t p = block_excl_scan(cnt, sh.bs, &tot);
      for (uint32_t w = w0; w < w1; ++w) {
        uint32_t word = L.bitmap[w];
        if (!word) continue;
        L.bitmap[w] = 0;
        while (word) {
          const uint32_t b = (uint32_t)__ffs(word) - 1u;
          word &= word - 1u;
          const uint32_t s = (w << 5) | b;
          place(p++, s, L.surv_pack[L.idx[s]]);
        }
      }
    }
    __syncthreads();
    // ------------------------------------- out-degree prefix sums of the frontier
    uint32_t* fe = L.f_edeg[cur];
    uint32_t* fx = L.f_xdeg[cur];
    uint8_t* fc = L.f_cls[cur];
    uint32_t W_next, W_eps;
    {
      const uint32_t per = (n_keep + kThreads - 1) / kThreads;
      const uint32_t p0 = tid * per < n_keep ? tid * per : n_keep;
      const uint32_t p1 = p0 + per < n_keep ? p0 + per : n_keep;
      uint32_t e = 0, x = 0;
      for (uint32_t p = p0; p < p1; ++p) {
        const uint32_t s = fs[p];
        const uint2 o0 = g.off[s], o1 = g.off[s + 1];
        e += o1.x - o0.x;
        x += o1.y - o0.y;
      }
      uint32_t eb = block_excl_scan(e, sh.bs, &W_next);
      uint32_t xb = block_excl_scan(x, sh.bs, &W_eps);
      for (uint32_t p = p0; p < p1; ++p) {
        const uint32_t s = fs[p];
        const uint2 o0 = g.off[s], o1 = g.off[s + 1];
        fe[p] = eb;
        fx[p] = xb;
        fc[p] = g.sclass[s];
        eb += o1.x - o0.x;
        xb += o1.y - o0.y;
      }
      if (tid == 0) {
        fe[n_keep] = W_next;
        fx[n_keep] = W_eps;
      }
    }
    __syncthreads();
    if (tid == 0) {
      L.node_off[t] = node_base;
      L.node_off[t + 1] = node_base + n_keep;
      L.best[t] = best;
      L.cutb[t] = cutb;
      L.cut[t] = key_cost(cut_key);
    }
    tokens += n_keep;
    max_tokens = n_keep > max_tokens ? n_keep : max_tokens;
    // -------------------------------------------------- lattice links of frame t
    // emitting run: candidates in work-item order are in arc-id order
    uint32_t nE = 0, nX = 0;
    uint32_t bad_idx = 0;
    {
      const uint32_t Wc = t > 0 ? W : 0;
      const uint32_t per = (Wc + kThreads - 1) / kThreads;
      const uint32_t w0 = tid * per < Wc ? tid * per : Wc;
      const uint32_t w1 = w0 + per < Wc ? w0 + per : Wc;
      uint32_t cnt = 0;
      for (uint32_t w = w0; w < w1; ++w) {
        const uint32_t xk = cost_key(__uint_as_float(L.cand[w].w));
        cnt += xk <= cut_key && xk < kInfKey;
      }
      uint32_t pos = block_excl_scan(cnt, sh.bs, &nE);
      // epsilon run: every epsilon out-arc of the frontier within the cutoff
      const uint32_t perx = (W_eps + kThreads - 1) / kThreads;
      const uint32_t e0 = tid * perx < W_eps ? tid * perx : W_eps;
      const uint32_t e1 = e0 + perx < W_eps ? e0 + perx : W_eps;
      uint32_t cntx = 0;
      if (e0 < e1) {
        uint32_t p = search_le(fx, n_keep, e0);
        for (uint32_t e = e0; e < e1; ++e) {
          while (fx[p + 1] <= e) ++p;
          const uint32_t s = fs[p];
          const uint4 r = g.xarc[g.off[s].y + (e - fx[p])];
          const uint32_t xk = cost_key(canon(key_cost(fk[p]) + __uint_as_float(r.y)));
          cntx += xk <= cut_key && xk < kInfKey;
        }
      }
      uint32_t posx = block_excl_scan(cntx, sh.bs, &nX);
      if (hist_ok && link_base + nE + nX > L.link_cap) {
        hist_ok = false;
        ovf |= kOvfLinks;
      }
      if (hist_ok) {
        for (uint32_t w = w0; w < w1; ++w) {
          const uint4 c = L.cand[w];
          const uint32_t xk = cost_key(__uint_as_float(c.w));
          if (!(xk <= cut_key && xk < kInfKey)) continue;
          const uint32_t dn = L.idx[c.z];
          if (dn < node_base || dn >= node_base + n_keep) {
            bad_idx = 1;
            continue;
          }
          L.links[link_base + pos] = make_uint4(c.x, c.y, dn, c.w);
          ++pos;
          if (L.n_pack[dn] == pack_tok(xk, c.x)) L.n_pred[dn] = c.y;
        }
        if (e0 < e1) {
          uint32_t p = search_le(fx, n_keep, e0);
          for (uint32_t e = e0; e < e1; ++e) {
            while (fx[p + 1] <= e) ++p;
            const uint32_t s = fs[p];
            const uint4 r = g.xarc[g.off[s].y + (e - fx[p])];
            const float x = canon(key_cost(fk[p]) + __uint_as_float(r.y));
            const uint32_t xk = cost_key(x);
            if (!(xk <= cut_key && xk < kInfKey)) continue;
            const uint32_t dn = L.idx[r.x];
            if (dn < node_base || dn >= node_base + n_keep) {
              bad_idx = 1;
              continue;
            }
            const uint32_t sn = (uint32_t)(node_base + p);
            const uint64_t at = link_base + nE + posx;
            L.links[at] = make_uint4(r.w, sn, dn, __float_as_uint(x));
            L.link_lvl[at] = fc[p];
            ++posx;
            if (L.n_pack[dn] == pack_tok(xk, r.w)) L.n_pred[dn] = sn;
          }
        }
      }
    }
    if (block_or(bad_idx, sh.bs)) {
      status = kStatusInternal;
      break;
    }
    if (tid == 0) {
      L.link_off[t] = link_base;
      L.link_xoff[t] = link_base + nE;
      L.link_off[t + 1] = link_base + nE + nX;
    }
    link_base += nE + nX;
    // ----------------------------------------------------- next frame
    node_base_prev = node_base;
    node_base += n_keep;
    n_prev = n_keep;
    W = W_next;
    cur ^= 1;
    for (uint32_t i = tid; i <= (uint32_t)kMaxLevels; i += kThreads) sh.nb[i] = 0;
    for (uint32_t i = tid; i < (uint32_t)kHistBins; i += kThreads) sh.hist[i] = 0;
    __syncthreads();
    if (tid == 0) {
      sh.n_touched = 0;
      sh.n_surv = 0;
      sh.n_rank = 0;
    }
    __syncthreads();
  }

  const uint64_t eps = block_sum64(my_eps, sh.bs);
  const uint64_t arcs = block_sum64(my_arcs, sh.bs) + eps;
  if (tid == 0) {
    LaneInfo* info = L.info;
    if (status == 0 && (ovf & (kOvfNodes | kOvfLinks))) status = 4;
    info->status = status;
    info->frames_done = t;
    info->overflow = ovf;
    info->arcs_expanded = arcs;
    info->eps_arcs = eps;
    info->tokens = tokens;
    info->max_tokens = max_tokens;
    info->links = link_base;
    info->need_frame_tokens = need_frame;
    info->need_frame_arcs = need_arcs;
  }
}

// Log-likelihood check: NaN, +inf and values above 1e30 are rejected.
__global__ void k_check_loglikes(const LaneDesc* __restrict__ lanes, uint32_t P, uint32_t* bad) {
  const LaneDesc L = lanes[blockIdx.y];
  const uint64_t n = (uint64_t)L.T * P;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x) {
    const float v = L.ll[i];
    if (v != v || v > 1e30f) {
      atomicOr(&bad[blockIdx.y], 1u);
      break;
    }
  }
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

void launch_forward(const DevGraph& g, const LaneDesc* lanes, int B, const Params& prm,
                    const uint32_t* bad, hipStream_t s) {
  hipLaunchKernelGGL(k_forward, dim3(B), dim3(kThreads), 0, s, g, lanes, prm, bad);
}

void launch_check_loglikes(const LaneDesc* lanes, int B, uint32_t P, uint32_t* bad, hipStream_t s) {
  hipLaunchKernelGGL(k_check_loglikes, dim3(64, B), dim3(256), 0, s, lanes, P, bad);
}

void launch_fill_u64(unsigned long long* p, uint64_t n, unsigned long long v, hipStream_t s) {
  if (n) hipLaunchKernelGGL(k_fill_u64, dim3(1024), dim3(256), 0, s, p, n, v);
}

void launch_fill_u32(uint32_t* p, uint64_t n, uint32_t v, hipStream_t s) {
  if (n) hipLaunchKernelGGL(k_fill_u32, dim3(1024), dim3(256), 0, s, p, n, v);
}

}  // namespace wd
