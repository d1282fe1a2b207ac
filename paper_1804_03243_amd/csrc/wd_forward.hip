// Forward pass: frame-synchronous token passing for one utterance per
// workgroup, every frame and every phase inside one persistent launch.
//
// Per frame t (Sec. 3.2-3.4 of the paper, with the readings stated in the
// oracle): emitting expansion of the surviving tokens of frame t-1 over a flat,
// prefix-sum load-balanced arc work space (Sec. 3.3 static load balancing);
// recombination by a 64-bit atomicMin of (cost key, arc id) on the state's
// token slot (Alg. 1); beam cutoff from the best emitting candidate; epsilon
// closure one epsilon level at a time; exact max-active cutoff by radix select
// over an LDS histogram; compaction of the survivors into a frontier sorted by
// state (which numbers the lattice nodes (t, i) of Sec. 3.5); lattice links for
// every surviving token-passing operation (Sec. 3.4).
//
// A frame's token table lives in LDS when the frame is small: an open-addressing
// hash of the touched states holding the packed tokens, so recombination,
// epsilon relaxation and the survivor scan are LDS operations.  A frame that
// touches more states than the table holds is redone from the same frontier on
// the global per-state slot array (its inputs are unchanged, so the result is
// identical).  The frontier itself is kept in LDS when it fits.
#include "../../include/wfstdec.h"
#include "wd_block.h"

namespace wd {

constexpr uint32_t kNoKey = 0xffffffffu;
constexpr uint16_t kNoSlot = 0xffffu;
// s_waitcnt operand: vector memory count 0, the export and LDS counts left open
constexpr int kWaitVm0 = 0x0f70;
constexpr uint32_t kLdsWork = 3 * kHashMax;  // emitting work above which a frame starts global
constexpr uint32_t kBkCap = 1024;            // LDS epsilon bucket entries before a frame spills
constexpr uint32_t kDirectRank = 256;        // survivors ranked directly, without the counting sort
// the thread that keeps the per-frame counters and records: the last one,
// whose wavefront is idle in small frames' steps
constexpr uint32_t kBook = kThreads - 1;
static_assert(kBkCap == (uint32_t)kThreads, "one bucket entry per thread in the epsilon level scan");

struct FwdShared {
  BlockScratch bs;
  // utterance counters, kept by thread 0 (in LDS to spare registers)
  unsigned long long c_arcs, c_tokens, c_max_tokens, c_need_frame, c_need_arcs;
  uint32_t n_touched;  // global table: touched states
  uint32_t n_surv;     // survivors of the beam cutoff
  uint32_t n_rank;
  uint32_t sel_b;
  uint32_t sel_before;
  uint32_t lvl_tot;    // LDS table: work items of the current epsilon level
  uint32_t lvl_wide;   // LDS table: first epsilon level the whole workgroup runs
  uint32_t lvl_live;   // LDS table: levels that may hold an entry within the cutoff (level_bit)
  unsigned long long deg_tot;  // frontier out-degree totals (epsilon << 32 | emitting), small frames
  uint32_t hcount;     // LDS table: reserved entries
  uint32_t spill;      // LDS table full: the frame goes global
  uint32_t n_bk;       // LDS table: epsilon bucket entries
  uint32_t nb[kMaxLevels + 1];  // global table: bucket sizes per level
  uint32_t nbl[kMaxLevels + 1]; // LDS table: bucket entries per level
  uint32_t hist[kHistBins];
  uint32_t rs_state[kRankMax];
  unsigned long long rs_pack[kRankMax];
  uint32_t rs_slot[kRankMax];
  alignas(16) uint32_t srt[kRankMax];  // states by bucket while sorting survivors
  uint32_t h_key[kHashCap];
  unsigned long long h_val[kHashCap];
  uint16_t h_used[kHashMax];  // slot claimed by the n-th insertion (kNoSlot: the state was there)
  uint4 bk[kBkCap];    // {table slot, first epsilon arc, end epsilon arc, level}
  uint32_t xp[kBkCap]; // epsilon arcs of the bucket entries before entry i (one level)
  uint32_t f_state[kFrontCap + 1];
  uint32_t f_key[kFrontCap + 1];
  uint32_t f_arc[kFrontCap + 1];
  uint32_t f_edeg[kFrontCap + 1];
  uint32_t f_xdeg[kFrontCap + 1];
  uint32_t f_ebeg[kFrontCap + 1];
  uint32_t f_xbeg[kFrontCap + 1];
  uint8_t f_cls[kFrontCap + 1];
};

// Frontier arrays of one frame, in LDS or in the workspace.
struct Front {
  uint32_t* state;
  uint32_t* key;
  uint32_t* arc;
  uint32_t* edeg;
  uint32_t* xdeg;
  uint32_t* ebeg;
  uint32_t* xbeg;
  uint8_t* cls;
};

__device__ __forceinline__ Front front_at(bool lds, FwdShared& sh, const LaneDesc& L) {
  if (lds) return Front{sh.f_state, sh.f_key, sh.f_arc, sh.f_edeg, sh.f_xdeg, sh.f_ebeg, sh.f_xbeg, sh.f_cls};
  return Front{L.f_state, L.f_key, L.f_arc, L.f_edeg, L.f_xdeg, L.f_ebeg, L.f_xbeg, L.f_cls};
}

// Emitting work item w of the previous frame's frontier: its arc index and
// (in *c) its token's cost.  With the owners in place the frontier is in
// LDS, and it is read there by name: accesses through a Front, which may
// point either way, are flat accesses, whose waits also take in every
// outstanding global load and store of the wavefront.
// (The LDS reads go through LDS-qualified pointers: plain ones would let
// the compiler merge them with the other branch's reads into flat ones.)
typedef __attribute__((address_space(3))) const uint32_t LdsU32;

__device__ __forceinline__ uint32_t item_arc(bool own, const uint16_t* own_e, FwdShared& sh, const Front& fp,
                                             uint32_t n_prev, uint32_t w, float* c) {
  if (own) {
    const uint32_t i = own_e[w];
    *c = key_cost(((LdsU32*)sh.f_key)[i]);
    return ((LdsU32*)sh.f_ebeg)[i] + (w - ((LdsU32*)sh.f_edeg)[i]);
  }
  const uint32_t i = search_le(fp.edeg, n_prev, w);
  *c = key_cost(fp.key[i]);
  return fp.ebeg[i] + (w - fp.edeg[i]);
}

// ---------------------------------------------------------------- LDS table

__device__ __forceinline__ uint32_t h_home(uint32_t s) { return (s * 0x9E3779B1u) >> 20; }  // 12 bits

// Find or insert state s; returns its slot, or kHashCap when the frame
// outgrows the table (sh.spill is then set and the frame goes to the global
// slot array).  *fresh: this call inserted s.  The probe reads up to s or an
// empty slot, where a compare-and-swap claims it (or finds s, put there
// meanwhile); the claimed slots are then counted, a wavefront at a time, and
// recorded for the survivor pass and the clear (the first kHashMax of them:
// more means a spill, after which the whole table is cleared).  The probe
// stops after kHashCap positions, so it ends even in a full table.
__device__ __forceinline__ uint32_t h_insert(FwdShared& sh, uint32_t s, bool* fresh) {
  uint32_t i = h_home(s), slot = kHashCap;
  bool ins = false;
  for (uint32_t n = 0; n < (uint32_t)kHashCap; ++n) {
    uint32_t k = sh.h_key[i];
    if (k == kNoKey) k = atomicCAS(&sh.h_key[i], kNoKey, s);
    if (k == kNoKey || k == s) {
      ins = k == kNoKey;
      slot = i;
      break;
    }
    i = (i + 1) & (kHashCap - 1);
  }
  const uint32_t c = wave_append(ins, &sh.hcount);
  if (ins) {
    if (c < (uint32_t)kHashMax) {
      sh.h_used[c] = (uint16_t)slot;
    } else {
      sh.spill = 1;
      slot = kHashCap;
    }
  }
  if (slot == kHashCap) sh.spill = 1;
  *fresh = ins && slot != kHashCap;
  return slot;
}

__device__ __forceinline__ uint32_t h_find(const FwdShared& sh, uint32_t s) {
  uint32_t i = h_home(s);
  while (true) {
    const uint32_t k = sh.h_key[i];
    if (k == s) return i;
    if (k == kNoKey) return kHashCap;
    i = (i + 1) & (kHashCap - 1);
  }
}

// Empties the table: every slot (used = kHashCap: its first use), or the
// slots claimed by the first `used` insertions (the count read before the
// last barrier; a frame that did not spill claims at most kHashMax slots).
__device__ __forceinline__ void h_clear(FwdShared& sh, uint32_t used) {
  if (used == (uint32_t)kHashCap) {
    for (uint32_t i = threadIdx.x; i < (uint32_t)kHashCap; i += kThreads) {
      sh.h_key[i] = kNoKey;
      sh.h_val[i] = kEmpty;
    }
  } else {
    for (uint32_t i = threadIdx.x; i < used; i += kThreads) {
      const uint32_t slot = sh.h_used[i];
      if (slot != kNoSlot) {
        sh.h_key[slot] = kNoKey;
        sh.h_val[slot] = kEmpty;
      }
    }
  }
  for (uint32_t i = threadIdx.x; i <= (uint32_t)kMaxLevels; i += kThreads) sh.nbl[i] = 0;
  if (threadIdx.x == 0) {
    sh.hcount = 0;
    sh.spill = 0;
    sh.n_bk = 0;
  }
}

// A first touch in the LDS table of a state with epsilon out-arcs: remember
// its slot, epsilon arc range and level for the epsilon passes.
__device__ __forceinline__ void lds_bucket(FwdShared& sh, uint32_t slot, uint4 o0, uint4 o1, uint32_t cls) {
  const uint32_t b = atomicAdd(&sh.n_bk, 1u);
  if (b < kBkCap) {
    sh.bk[b] = make_uint4(slot, o0.y, o1.y, cls);
    atomicAdd(&sh.nbl[cls], 1u);
  } else {
    sh.spill = 1;
  }
}

// The same with the graph's epsilon path table: the state's path range and
// its epsilon out-degree (empty range: a state reached by an epsilon path,
// whose own paths are extensions of that path).
__device__ __forceinline__ void lds_bucket_paths(FwdShared& sh, uint32_t slot, uint32_t p0, uint32_t p1,
                                                 uint32_t xdeg) {
  const uint32_t b = atomicAdd(&sh.n_bk, 1u);
  if (b < kBkCap) sh.bk[b] = make_uint4(slot, p0, p1, xdeg);
  else sh.spill = 1;
}

// Epsilon levels as bits of a mask: bit l for level l < 31, bit 31 for every
// level from 31 on.
__device__ __forceinline__ uint32_t level_bit(uint32_t l) { return 1u << (l < 31u ? l : 31u); }

// Lowest level >= from whose bit is set in mask (levels from 31 on are taken
// one after another while bit 31 is set); nlevels when there is none.
__device__ __forceinline__ uint32_t next_live(uint32_t mask, uint32_t from, uint32_t nlevels) {
  if (from >= nlevels) return nlevels;
  if (from < 31u) {
    const uint32_t m = mask & 0x7fffffffu & (~0u << from);
    if (m) {
      const uint32_t l = (uint32_t)__ffs(m) - 1u;
      return l < nlevels ? l : nlevels;
    }
    from = 31u;
    if (from >= nlevels) return nlevels;
  }
  return (mask & 0x80000000u) ? from : nlevels;
}

// ------------------------------------------------------------- global table

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
__device__ __forceinline__ void select_bin(uint32_t rank, FwdShared& sh, uint32_t& par, uint32_t* bin,
                                           uint32_t* before, uint32_t* count) {
  const uint32_t tid = threadIdx.x;
  uint32_t h0 = sh.hist[2 * tid], h1 = sh.hist[2 * tid + 1];
  uint32_t tot;
  uint32_t ex = block_excl_scan(h0 + h1, sh.bs, par, &tot);
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

__device__ __forceinline__ uint64_t uniform64(uint64_t v) {
  return ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(v >> 32)) << 32) |
         (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)v);
}

// kProf: the step-profile copy (WD_FLAG_PHASES), which stores the device
// wall clock at each step boundary of every frame (thread 0).
template <bool kProf>
__device__ __forceinline__ void forward_body(FwdShared& sh, const DevGraph& g, const LaneDesc* __restrict__ lanes,
                                             const Params& prm, const uint32_t* __restrict__ bad) {
  const LaneDesc& L = lanes[blockIdx.x];
  const uint32_t tid = threadIdx.x;
  // epsilon closure of LDS-table frames: every path at once, or level by level
  const bool paths = g.npaths != 0 && !(prm.flags & WD_FLAG_EPS_LEVELS);
  if (bad[blockIdx.x]) {
    if (tid == 0) L.info->status = 1;  // WD_EINVAL
    return;
  }
  const int T = L.T;
  const uint32_t P = g.P;

  for (uint32_t i = tid; i <= (uint32_t)kMaxLevels; i += kThreads) sh.nb[i] = 0;
  for (uint32_t i = tid; i < (uint32_t)kHistBins; i += kThreads) sh.hist[i] = 0;
  h_clear(sh, kHashCap);
  if (tid == 0) {
    sh.n_touched = 0;
    sh.n_surv = 0;
    sh.n_rank = 0;
  }
  __syncthreads();

  int status = 0;  // WD_OK
  uint32_t ovf = 0;
  uint32_t best_key = cost_key(0.0f);
  uint64_t node_base = 0;
  uint32_t n_prev = 0, W = 0;
  bool front_lds = true;  // where the frontier of the last finished frame is
  bool front_own = false; // its emitting work items' owners are in own_e
  // owners of the frontier's emitting work items, 16-bit, in rs_pack (free
  // from the degree pass until the next frame's survivor pass)
  uint16_t* const own_e = reinterpret_cast<uint16_t*>(sh.rs_pack);
  constexpr uint32_t kOwnE = 4u * (uint32_t)kRankMax;
  uint64_t my_eps = 0;
  if (tid == 0) {
    sh.c_arcs = 0;
    sh.c_tokens = 0;
    sh.c_max_tokens = 0;
    sh.c_need_frame = 1;
    sh.c_need_arcs = 0;
  }
  bool hist_ok = true;  // history (the node store) still being stored
  uint32_t warm_bad = 0;  // a warming load returned the sentinel payload (never)
  float warm_prev = 0.0f;  // the previous frame's warming values (read a frame late)
  uint32_t par = 0;     // scratch buffer parity of the workgroup collectives
  int t = L.t0;
  // step profile: slot k < kProfStamps of frame t gets the wall clock when
  // thread 0 passes step boundary k; the last two slots describe the frame
  auto stamp = [&](int k) {
    if constexpr (kProf) {
      if (tid == 0) L.prof[(size_t)t * kProfSlots + (size_t)k] = wall_clock64();
    }
  };
  auto note = [&](int k, uint64_t v) {
    if constexpr (kProf) {
      if (tid == 0) L.prof[(size_t)t * kProfSlots + (size_t)k] = v;
    }
  };
  if (t > 0) {
    // a stream resumes after frame t - 1: the state the last launch left in
    // LaneInfo, the frontier in the workspace.  A full node or link store
    // goes on (the decode still measures what it needs); a frame that
    // outgrew the per-frame capacities stopped mid-frame and stays stopped.
    // The values are the same in every lane; saying so keeps them out of
    // vector registers.
    const LaneInfo& I = *L.info;
    const bool go_on = I.status == 4 && (I.overflow & (kOvfFrame | kOvfArcs)) == 0;
    status = __builtin_amdgcn_readfirstlane(go_on ? 0 : I.status);
    if (status != 0) return;
    ovf = __builtin_amdgcn_readfirstlane(I.overflow);
    hist_ok = (ovf & kOvfNodes) == 0;
    node_base = uniform64(I.tokens);
    n_prev = __builtin_amdgcn_readfirstlane(I.last_tokens);
    W = __builtin_amdgcn_readfirstlane(L.f_edeg[n_prev]);
    front_lds = false;
    my_eps = tid == 0 ? I.eps_arcs : 0;
    if (tid == 0) {
      sh.c_arcs = I.arcs_expanded - I.eps_arcs;
      sh.c_tokens = I.tokens;
      sh.c_max_tokens = I.max_tokens;
      sh.c_need_frame = I.need_frame_tokens;
      sh.c_need_arcs = I.need_frame_arcs;
    }
  }

  for (; t <= T; ++t) {
    stamp(0);
    if (t > 0) {
      if (tid == kBook && W > sh.c_need_arcs) sh.c_need_arcs = W;
      if (W > L.cand_cap) {
        status = 4;  // WD_ECAPACITY
        ovf |= kOvfArcs;
        break;
      }
    }
    const Front fp = front_at(front_lds, sh, L);  // frontier of frame t-1
    const float* row = L.ll + (size_t)(t > 0 ? t - 1 : 0) * P;
    bool lds = t == 0 || W <= kLdsWork;
    uint32_t kcutb = 0, ns = 0;
    uint32_t nbits = 0, shift = 0;
    uint64_t eps_frame = 0;
    bool failed = false;
    float warm = 0.0f;  // values of cache-warming loads, read at the end of the next frame
    // ---------------------------------------------------- token passing
    for (int attempt = 0; attempt < 2; ++attempt) {
      eps_frame = 0;
      if (lds) {
        // ------------------------------------------ LDS token table
        if (t == 0) {
          if (tid == 0) {
            const uint32_t s0 = g.start;
            bool fresh;
            const uint32_t slot = h_insert(sh, s0, &fresh);
            sh.h_val[slot] = pack_tok(cost_key(0.0f), kNoArc);
            const uint32_t c = g.sclass[s0];
            if (c != kNoEps) {
              const uint4 o0 = g.off[s0], o1 = g.off[s0 + 1];
              if (paths) lds_bucket_paths(sh, slot, o0.z, o1.z, o1.y - o0.y);
              else lds_bucket(sh, slot, o0, o1, c);
            }
          }
          best_key = cost_key(0.0f);
          __syncthreads();
          stamp(1);
        } else {
          uint32_t my_best = 0xffffffffu;
          for (uint32_t base = 0; base < W; base += kThreads) {
            const uint32_t w = base + tid;
            if (w >= W) break;
            float c;
            const uint4 r = g.earc[item_arc(front_own, own_e, sh, fp, n_prev, w, &c)];
            const uint32_t dst = r.x, cls = r.z >> 24;
            // CSR offsets of the destination: the epsilon range for the bucket,
            // and warm in cache for the degree pass if the token survives;
            // with the path table, the range of its epsilon paths
            const uint4 o0 = g.off[dst], o1 = g.off[dst + 1];
            const float ac = -row[(r.z & 0xffffffu) - 1u];
            float x = c + ac;
            x = canon(x + __uint_as_float(r.y));
            const uint32_t xk = cost_key(x);
            if (xk < kInfKey) {
              my_best = xk < my_best ? xk : my_best;
              if (!sh.spill) {
                bool fresh;
                const uint32_t slot = h_insert(sh, dst, &fresh);
                if (slot < (uint32_t)kHashCap) {
                  atomicMin(&sh.h_val[slot], pack_tok(xk, r.w));
                  if (fresh && cls != kNoEps) {
                    if (paths) {
                      lds_bucket_paths(sh, slot, o0.z, o1.z, o1.y - o0.y);
                      // start the state's first epsilon paths on their way for the closure
                      warm = __uint_as_float(g.phead[2 * (size_t)o0.z].z);
                    } else {
                      lds_bucket(sh, slot, o0, o1, cls);
                      // start the state's first epsilon arc on its way for the closure
                      warm = __uint_as_float(g.xarc[o0.y].y);
                    }
                  }
                }
              }
            }
          }
          // (the collective's barrier also publishes the table writes)
          best_key = (uint32_t)block_min64(my_best, sh.bs, par);
          stamp(1);
          if (best_key >= kInfKey) {
            status = 3;  // WD_ENOPATH
            failed = true;
            break;
          }
        }
        if (sh.spill) {
          lds = false;
          continue;
        }
        const float cutb = key_cost(best_key) + prm.beam;
        kcutb = cost_key(cutb);
        // each entry writes its index at its work items, so a work item
        // finds its entry with one LDS read (rs_slot is free until the
        // closure ends)
        uint16_t* own = reinterpret_cast<uint16_t*>(sh.rs_slot);
        constexpr uint32_t kOwnCap = 2u * (uint32_t)kRankMax;
        if (paths) {
          // Every epsilon path of every bucket entry within the cutoff, all
          // levels at once: a path's cost adds its arcs' weights to the
          // entry's cost in path order, rounding after each addition, which
          // is what one pass per level computes for the path's last state
          // (rounding is monotone, so the minimum over the paths into a
          // state is the level-by-level token, arc ids included; an entry
          // whose cost later drops through another path only offers the
          // sums of longer paths that are themselves in the table).  One
          // round of dependent loads instead of one per level.
          auto relax_path = [&](uint32_t j, uint32_t w) {
            const uint4 e = sh.bk[j];
            const uint32_t pth = e.y + (w - sh.xp[j]);
            // the head and the first four tail weights: one 32-byte record
            const uint4 h = g.phead[2 * (size_t)pth], hw = g.phead[2 * (size_t)pth + 1];
            const uint32_t k = h.w & 0xffu;
            float x = key_cost((uint32_t)(sh.h_val[e.x] >> 32));
            if (k > 1u) {
              x = canon(x + __uint_as_float(hw.x));
              if (k > 2u) x = canon(x + __uint_as_float(hw.y));
              if (k > 3u) x = canon(x + __uint_as_float(hw.z));
              if (k > 4u) x = canon(x + __uint_as_float(hw.w));
              const float* tw = g.ptail + (size_t)pth * g.pstride;
              for (uint32_t i = 4; i + 1 < k; ++i) x = canon(x + tw[i]);
            }
            const uint32_t xk = cost_key(canon(x + __uint_as_float(h.z)));
            if (xk > kcutb || xk >= kInfKey || sh.spill) return;
            bool fresh;
            const uint32_t slot = h_insert(sh, h.x, &fresh);
            if (slot < (uint32_t)kHashCap) {
              atomicMin(&sh.h_val[slot], pack_tok(xk, h.y));
              if (fresh && (h.w >> 8)) lds_bucket_paths(sh, slot, 0, 0, h.w >> 8);
            }
          };
          const uint32_t n = sh.n_bk < kBkCap ? sh.n_bk : kBkCap;
          uint32_t d = 0;
          if (tid < n) {
            const uint4 e = sh.bk[tid];
            if ((uint32_t)(sh.h_val[e.x] >> 32) <= kcutb) d = e.z - e.y;
          }
          uint32_t tot;
          if (n <= 64u) {
            // every entry in the first wavefront: its scan needs no workgroup
            // barrier, and when the paths fit its lanes it relaxes them alone
            if (tid < 64u) {
              const uint32_t inc = wave_incl_scan(d), ex = inc - d;
              const uint32_t all = lane63(inc);
              sh.xp[tid] = ex;
              if (all <= kOwnCap)
                for (uint32_t k = 0; k < d; ++k) own[ex + k] = (uint16_t)tid;
              if (tid == 63u) sh.lvl_tot = all;
              __builtin_amdgcn_wave_barrier();
              if (all <= 64u && tid < all) relax_path(own[tid], tid);
            }
            __syncthreads();
            tot = sh.lvl_tot;
          } else {
            const uint32_t ex = block_excl_scan(d, sh.bs, par, &tot);
            sh.xp[tid] = ex;
            if (tot <= kOwnCap)
              for (uint32_t k = 0; k < d; ++k) own[ex + k] = (uint16_t)tid;
            __syncthreads();
          }
          // (uniform: n and tot are the same in every thread)
          if (n > 64u || tot > 64u) {
            const bool by_owner = tot <= kOwnCap;
            for (uint32_t w = tid; w < tot; w += kThreads)
              relax_path(by_owner ? (uint32_t)own[w] : search_le(sh.xp, n, w), w);
            __syncthreads();
          }
          if (sh.spill) {
            lds = false;
            continue;
          }
          // the epsilon out-arcs of the closure's states within the cutoff
          // (the arcs-expanded count); the entries' costs are final
          const uint32_t nb = sh.n_bk < kBkCap ? sh.n_bk : kBkCap;
          for (uint32_t j = tid; j < nb; j += kThreads) {
            const uint4 e = sh.bk[j];
            if ((uint32_t)(sh.h_val[e.x] >> 32) <= kcutb) eps_frame += e.w;
          }
        } else {
        // one epsilon arc of a level: work item w of bucket entry j
        auto relax_eps = [&](uint32_t j, uint32_t w) {
          const uint4 e = sh.bk[j];
          const uint32_t a = e.y + (w - sh.xp[j]);
          const uint4 r = g.xarc[a];
          const uint2 nx = g.xnext[a];  // the destination's epsilon arcs
          const float c = key_cost((uint32_t)(sh.h_val[e.x] >> 32));
          const uint32_t xk = cost_key(canon(c + __uint_as_float(r.y)));
          if (xk > kcutb || xk >= kInfKey || sh.spill) return;
          bool fresh;
          const uint32_t slot = h_insert(sh, r.x, &fresh);
          if (slot < (uint32_t)kHashCap) {
            atomicMin(&sh.h_val[slot], pack_tok(xk, r.w));
            if (r.z != kNoEps) {
              // the destination's level now holds an entry within the cutoff
              atomicOr(&sh.lvl_live, level_bit(r.z));
              if (fresh) lds_bucket(sh, slot, make_uint4(0, nx.x, 0, 0), make_uint4(0, nx.y, 0, 0), r.z);
            }
          }
        };
        // The levels that hold a bucket entry within the cutoff: only they
        // relax epsilon arcs (most frames have none, or one or two of the
        // graph's levels).  Every insertion within the cutoff into a state
        // with epsilon arcs adds its level.
        // (Wavefront 0 builds the mask when every entry is in its lanes and
        // reads it in program order; the others read it after the next
        // barrier.  With more entries every level is taken.)
        if (tid < 64u) {
          const uint32_t nbk0 = sh.n_bk;  // (published by the last barrier)
          uint32_t m = ~0u;
          if (nbk0 <= 64u) {
            m = 0;
            if (tid < nbk0) {
              const uint4 e = sh.bk[tid];
              if ((uint32_t)(sh.h_val[e.x] >> 32) <= kcutb) m = level_bit(e.w);
            }
            m = wave_or(m);
          }
          if (tid == 0) sh.lvl_live = m;
          __builtin_amdgcn_wave_barrier();
        }
        // Levels whose bucket entries and epsilon arcs each fit in one
        // wavefront run in wavefront 0 alone, one after another, with no
        // workgroup barrier: a wavefront's LDS accesses take effect in
        // program order, so each level sees the previous one's tokens.  The
        // first level that does not fit, and the levels after it, run on the
        // whole workgroup below.
        if (tid < 64u) {
          uint32_t lvl = next_live(sh.lvl_live, 0, g.nlevels);
          for (; lvl < g.nlevels; lvl = next_live(sh.lvl_live, lvl + 1, g.nlevels)) {
            if (sh.spill) {
              lvl = g.nlevels;
              break;
            }
            if (sh.nbl[lvl] == 0) continue;
            const uint32_t n = sh.n_bk < kBkCap ? sh.n_bk : kBkCap;
            if (n > 64u) break;
            uint32_t d = 0;
            if (tid < n) {
              const uint4 e = sh.bk[tid];
              if (e.w == lvl && (uint32_t)(sh.h_val[e.x] >> 32) <= kcutb) d = e.z - e.y;
            }
            const uint32_t inc = wave_incl_scan(d), ex = inc - d;
            const uint32_t all = lane63(inc);
            if (all > 64u) break;  // (nothing of this level done yet)
            eps_frame += d;
            sh.xp[tid] = ex;
            for (uint32_t k = 0; k < d; ++k) own[ex + k] = (uint16_t)tid;
            __builtin_amdgcn_wave_barrier();
            if (tid < all) relax_eps(own[tid], tid);
            __builtin_amdgcn_wave_barrier();
          }
          if (tid == 0) sh.lvl_wide = lvl;
        }
        __syncthreads();
        // (lvl_live changes only in a level's relaxation, after that level's
        // scan barrier, which every thread passes after reading it here)
        for (uint32_t lvl = next_live(sh.lvl_live, sh.lvl_wide, g.nlevels); lvl < g.nlevels;
             lvl = next_live(sh.lvl_live, lvl + 1, g.nlevels)) {
          if (sh.nbl[lvl] == 0) continue;  // uniform: written only by lower levels
          // this level's entries within the cutoff spread their epsilon arcs
          // over the workgroup: entry i (one per thread) owns arcs
          // [xp[i], xp[i] + its degree) of the level's work space.  Every
          // thread reads the entry count before the scan's barrier; entries
          // appended below (higher levels) come after it.
          const uint32_t n = sh.n_bk < kBkCap ? sh.n_bk : kBkCap;
          uint32_t d = 0;
          if (tid < n) {
            const uint4 e = sh.bk[tid];
            if (e.w == lvl && (uint32_t)(sh.h_val[e.x] >> 32) <= kcutb) d = e.z - e.y;
          }
          eps_frame += d;
          uint32_t tot;
          if (n <= 64u) {
            // every entry in the first wavefront: its scan needs no
            // workgroup barrier, and one barrier publishes the result
            if (tid < 64u) {
              const uint32_t inc = wave_incl_scan(d), ex = inc - d;
              const uint32_t all = lane63(inc);
              sh.xp[tid] = ex;
              if (all <= kOwnCap)
                for (uint32_t k = 0; k < d; ++k) own[ex + k] = (uint16_t)tid;
              if (tid == 63u) sh.lvl_tot = all;
            }
            __syncthreads();
            tot = sh.lvl_tot;
          } else {
            const uint32_t ex = block_excl_scan(d, sh.bs, par, &tot);
            sh.xp[tid] = ex;
            if (tot <= kOwnCap)
              for (uint32_t k = 0; k < d; ++k) own[ex + k] = (uint16_t)tid;
            __syncthreads();
          }
          const bool by_owner = tot <= kOwnCap;
          for (uint32_t w = tid; w < tot; w += kThreads)
            relax_eps(by_owner ? (uint32_t)own[w] : search_le(sh.xp, n, w), w);
          __syncthreads();
          if (sh.spill) break;
        }
        if (sh.spill) {
          lds = false;
          continue;
        }
        }  // level by level
        stamp(2);
        // survivors of the beam cutoff, straight from the table
        const uint32_t span = kcutb - best_key;
        nbits = span ? 32u - (uint32_t)__clz(span) : 0u;
        shift = nbits > 11u ? nbits - 11u : 0u;
        // (the table's entries are the slots its insertions claimed)
        const uint32_t hc = sh.hcount;  // <= kHashMax: the frame did not spill
        for (uint32_t base = 0; base < hc; base += kThreads) {
          const uint32_t i = base + tid;
          const uint32_t slot = i < hc ? (uint32_t)sh.h_used[i] : (uint32_t)kNoSlot;
          uint32_t s = kNoKey;
          unsigned long long v = kEmpty;
          if (slot != kNoSlot) {
            s = sh.h_key[slot];
            v = sh.h_val[slot];
          }
          const bool keep = s != kNoKey && (uint32_t)(v >> 32) <= kcutb;
          const uint32_t pos = wave_append(keep, &sh.n_surv);
          if (keep) {
            sh.rs_state[pos] = s;
            sh.rs_pack[pos] = v;
            sh.rs_slot[pos] = slot;
            sh.srt[pos] = s;  // the direct ranking's input when no max-active cut follows
            atomicAdd(&sh.hist[((uint32_t)(v >> 32) - best_key) >> shift], 1u);
          }
        }
        __syncthreads();
        ns = sh.n_surv;
        stamp(3);
        if (tid == kBook && sh.hcount > sh.c_need_frame) sh.c_need_frame = sh.hcount;
      } else {
        // --------------------------------------- global per-state slot array
        if (t == 0) {
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
          best_key = cost_key(0.0f);
          __syncthreads();
          stamp(1);
        } else {
          uint32_t my_best = 0xffffffffu;
          for (uint32_t base = 0; base < W; base += kThreads) {
            const uint32_t w = base + tid;
            bool first = false;
            uint32_t dst = 0, cls = kNoEps;
            if (w < W) {
              float c;
              const uint4 r = g.earc[item_arc(front_own, own_e, sh, fp, n_prev, w, &c)];
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
            }
            note_touch(first, dst, cls, sh, g, L);
          }
          best_key = (uint32_t)block_min64(my_best, sh.bs, par);
          stamp(1);
          if (best_key >= kInfKey) {
            status = 3;  // WD_ENOPATH
            failed = true;
            break;
          }
        }
        const float cutb = key_cost(best_key) + prm.beam;
        kcutb = cost_key(cutb);
        for (uint32_t lvl = 0; lvl < g.nlevels; ++lvl) {
          const uint32_t n = sh.nb[lvl];
          if (n == 0) continue;
          const uint32_t* bk = L.bucket + g.level_base[lvl];
          for (uint32_t i = tid; i < n; i += kThreads) {
            const uint32_t s = bk[i];
            const uint32_t k = (uint32_t)(L.slot[s] >> 32);
            if (k > kcutb) continue;
            const float c = key_cost(k);
            const uint32_t a0 = g.off[s].y, a1 = g.off[s + 1].y;
            eps_frame += a1 - a0;
            for (uint32_t a = a0; a < a1; ++a) {
              const uint4 r = g.xarc[a];
              const uint32_t xk = cost_key(canon(c + __uint_as_float(r.y)));
              if (xk > kcutb || xk >= kInfKey) continue;
              const unsigned long long old = atomicMin(&L.slot[r.x], pack_tok(xk, r.w));
              if (old == kEmpty) note_touch_div(r.x, r.z, sh, g, L);
            }
          }
          __syncthreads();
        }
        stamp(2);
        const uint32_t nt = sh.n_touched;
        if (tid == kBook && nt > sh.c_need_frame) sh.c_need_frame = nt;
        if (nt > L.frame_cap) {
          status = 4;
          ovf |= kOvfFrame;
          failed = true;
          break;
        }
        const uint32_t span = kcutb - best_key;
        nbits = span ? 32u - (uint32_t)__clz(span) : 0u;
        shift = nbits > 11u ? nbits - 11u : 0u;
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
        ns = sh.n_surv;
        stamp(3);
      }
      break;
    }
    if (failed) break;
    my_eps += eps_frame;
    if (t > 0 && tid == kBook) sh.c_arcs += W;
    const float best = key_cost(best_key);
    const float cutb = key_cost(kcutb);
    const unsigned long long* spack = lds ? sh.rs_pack : L.surv_pack;
    const uint32_t* sstate = lds ? sh.rs_state : L.surv_state;
    // ------------------------------------------------ max-active cutoff
    uint32_t cut_key = kcutb;
    uint32_t n_keep = ns;
    if (prm.max_active > 0 && ns > (uint32_t)prm.max_active) {
      uint32_t rank = (uint32_t)prm.max_active, prefix = 0, less = 0;
      uint32_t bits = nbits - shift;
      while (true) {
        uint32_t b, before, cnt;
        select_bin(rank, sh, par, &b, &before, &cnt);
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
          const uint32_t d = (uint32_t)(spack[i] >> 32) - best_key;
          if ((d >> shift) == prefix) atomicAdd(&sh.hist[(d >> nsh) & ((1u << bits) - 1u)], 1u);
        }
        shift = nsh;
        __syncthreads();
      }
      const uint32_t vkey = best_key + prefix;
      cut_key = vkey < kcutb ? vkey : kcutb;
    }
    stamp(4);
    // -------------------------------- compaction into a frontier sorted by state
    const bool fl = n_keep <= (uint32_t)kFrontCap;
    const Front f = front_at(fl, sh, L);
    // the LDS frontier by name, for the steps that run only when it is there
    // (its accesses are then LDS accesses, not flat ones)
    const Front fs = front_at(true, sh, L);
    bool deg_ready = false;  // the compaction filled the frontier's offsets and degrees
    if (hist_ok && node_base + n_keep > L.node_cap) {
      hist_ok = false;
      ovf |= kOvfNodes;
    }
    auto place = [&](const Front& F, uint32_t p, uint32_t s, unsigned long long v) {
      const uint64_t node = node_base + p;
      if (hist_ok) {
        L.n_state[node] = s;
        L.n_pack[node] = v;
        L.n_pred[node] = kNoArc;
      }
      F.state[p] = s;
      F.key[p] = (uint32_t)(v >> 32);
      F.arc[p] = (uint32_t)v;
    };
    if (lds || n_keep <= (uint32_t)kRankMax) {
      if (!lds) {
        // gather the kept survivors of the global table into rs_*
        for (uint32_t base = 0; base < ns; base += kThreads) {
          const uint32_t i = base + tid;
          bool keep = false;
          uint32_t s = 0;
          unsigned long long v = 0;
          if (i < ns) {
            v = spack[i];
            s = sstate[i];
            keep = (uint32_t)(v >> 32) <= cut_key;
          }
          const uint32_t pos = wave_append(keep, &sh.n_rank);
          if (keep && pos < (uint32_t)kRankMax) {
            sh.rs_state[pos] = s;
            sh.rs_pack[pos] = v;
            sh.rs_slot[pos] = kHashCap;
          }
        }
        __syncthreads();
        if (sh.n_rank != n_keep) {
          status = kStatusInternal;
          break;
        }
      }
      const uint32_t m = lds ? ns : n_keep;  // entries in rs_* (<= 2 * kThreads)
      if (m <= kDirectRank) {
        // few entries: each kept state's rank is the number of kept states
        // below it, counted by four lanes (each a quarter of the entries)
        // and summed across them.  Without a max-active cut the survivor pass
        // has put every entry into srt already; otherwise the entries it drops
        // read as ~0.  The quad's first lane also fills the frontier entry's
        // arc offsets, degrees and level (its loads overlap the ranking).
        static_assert(4 * kDirectRank <= kThreads, "four lanes per directly ranked entry");
        static_assert(kDirectRank <= kFrontCap, "a directly ranked frontier is in LDS");
        deg_ready = true;
        if (!(lds && cut_key == kcutb)) {
          if (tid < m) {
            uint32_t s = kNoKey;
            if ((uint32_t)(sh.rs_pack[tid] >> 32) <= cut_key) s = sh.rs_state[tid];
            sh.srt[tid] = s;
          }
          __syncthreads();
        }
        // the frontier's earlier stores have landed by now; saying so lets the
        // ranking loop read LDS without first waiting for the loads below
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        const uint32_t lane_q = opaque(tid);
        const uint32_t e = lane_q >> 2, sub = lane_q & 3u;
        if (e < m && sh.srt[e] != kNoKey) {  // (the same for the four lanes)
          const uint32_t s = sh.srt[e];
          uint4 o0 = make_uint4(0, 0, 0, 0), o1 = o0;
          uint8_t cls = 0;
          if (sub == 0) {
            o0 = g.off[s];
            o1 = g.off[s + 1];
            cls = g.sclass[s];
          }
          const uint4* q4 = reinterpret_cast<const uint4*>(sh.srt);
          uint32_t r = 0;
          for (uint32_t q = sub; q < m / 4u; q += 4u) {
            const uint4 v = q4[q];
            r += (v.x < s) + (v.y < s) + (v.z < s) + (v.w < s);
          }
          const uint32_t qt = (m & ~3u) + sub;
          if (qt < m) r += sh.srt[qt] < s;
          r += dpp32<kDppQuadSwap1>(r, 0u);
          r += dpp32<kDppQuadSwap2>(r, 0u);
          if (sub == 0) {
            place(fs, r, s, sh.rs_pack[e]);  // (at most kDirectRank tokens: in LDS)
            fs.ebeg[r] = o0.x;
            fs.xbeg[r] = o0.y;
            fs.edeg[r] = o1.x - o0.x;  // degrees for now, prefix sums below
            fs.xdeg[r] = o1.y - o0.y;
            fs.cls[r] = cls;
          }
        }
      } else {
        // counting sort on the top 11 bits of the state, then the few states
        // sharing a bucket are ranked among themselves
        const uint32_t S = opaque(g.S);
        const uint32_t sbits = 32u - (uint32_t)__clz(S > 1 ? S - 1 : 1u);
        const uint32_t ssh = sbits > 11u ? sbits - 11u : 0u;
        for (uint32_t i = tid; i < (uint32_t)kHistBins; i += kThreads) sh.hist[i] = 0;
        __syncthreads();
        uint32_t bb[2] = {0, 0}, loc[2] = {0, 0}, sv[2] = {0, 0};
        unsigned long long vv[2] = {0, 0};
        bool kp[2] = {false, false};
        for (int u = 0; u < 2; ++u) {
          const uint32_t j = tid + (uint32_t)u * kThreads;
          if (j >= m) continue;
          vv[u] = sh.rs_pack[j];
          if ((uint32_t)(vv[u] >> 32) > cut_key) continue;
          kp[u] = true;
          sv[u] = sh.rs_state[j];
          bb[u] = sv[u] >> ssh;
          loc[u] = atomicAdd(&sh.hist[bb[u]], 1u);
        }
        __syncthreads();
        uint32_t nk;
        {
          const uint32_t h0 = sh.hist[2 * tid], h1 = sh.hist[2 * tid + 1];
          const uint32_t ex = block_excl_scan(h0 + h1, sh.bs, par, &nk);
          __syncthreads();  // every count read before the starts overwrite them
          sh.hist[2 * tid] = ex;
          sh.hist[2 * tid + 1] = ex + h0;
        }
        if (nk != n_keep) {
          status = kStatusInternal;
          break;
        }
        __syncthreads();
        for (int u = 0; u < 2; ++u)
          if (kp[u]) sh.srt[sh.hist[bb[u]] + loc[u]] = sv[u];
        __syncthreads();
        for (int u = 0; u < 2; ++u) {
          if (!kp[u]) continue;
          const uint32_t b0 = sh.hist[bb[u]];
          const uint32_t b1 = bb[u] + 1 < (uint32_t)kHistBins ? sh.hist[bb[u] + 1] : n_keep;
          uint32_t r = b0;
          for (uint32_t q = b0; q < b1; ++q) r += sh.srt[q] < sv[u];
          place(f, r, sv[u], vv[u]);
        }
      }
    } else {
      for (uint32_t i = tid; i < ns; i += kThreads) {
        const unsigned long long v = spack[i];
        if ((uint32_t)(v >> 32) <= cut_key) {
          const uint32_t s = sstate[i];
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
      uint32_t p = block_excl_scan(cnt, sh.bs, par, &tot);
      for (uint32_t w = w0; w < w1; ++w) {
        uint32_t word = L.bitmap[w];
        if (!word) continue;
        L.bitmap[w] = 0;
        while (word) {
          const uint32_t b = (uint32_t)__ffs(word) - 1u;
          word &= word - 1u;
          const uint32_t s = (w << 5) | b;
          place(f, p, s, spack[L.idx[s]]);
          ++p;
        }
      }
    }
    __syncthreads();
    stamp(5);
    // the table's claimed slots, read before the degree pass's barrier (after
    // it, the frame end clears them and resets the count)
    const uint32_t h_used_n = sh.hcount > (uint32_t)kHashMax ? (uint32_t)kHashCap : sh.hcount;
    // ------------------------------- arc offsets and degree prefix sums
    uint32_t W_next, W_eps;
    if (deg_ready) {
      // at most kDirectRank tokens with their degrees in place: the last
      // wavefront sums them, four per lane, and publishes the totals
      static_assert(kDirectRank <= 4 * 64, "four tokens per lane");
      if (tid >= kThreads - 64u) {
        const uint32_t lane = lane_id();
        uint32_t de[4], dx[4];
        uint64_t sum = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t p = 4u * lane + (uint32_t)k;
          de[k] = p < n_keep ? fs.edeg[p] : 0u;
          dx[k] = p < n_keep ? fs.xdeg[p] : 0u;
          sum += ((uint64_t)dx[k] << 32) | de[k];
        }
        const uint64_t inc = wave_incl_scan64(sum);
        uint32_t eb = (uint32_t)(inc - sum), xb = (uint32_t)((inc - sum) >> 32);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t p = 4u * lane + (uint32_t)k;
          if (p < n_keep) {
            fs.edeg[p] = eb;
            fs.xdeg[p] = xb;
          }
          eb += de[k];
          xb += dx[k];
        }
        if (lane == 63u) {
          sh.deg_tot = inc;
          fs.edeg[n_keep] = (uint32_t)inc;
          fs.xdeg[n_keep] = (uint32_t)(inc >> 32);
        }
      }
      __syncthreads();
      W_next = (uint32_t)sh.deg_tot;
      W_eps = (uint32_t)(sh.deg_tot >> 32);
    } else {
      const uint32_t per = (n_keep + kThreads - 1) / kThreads;
      const uint32_t p0 = tid * per < n_keep ? tid * per : n_keep;
      const uint32_t p1 = p0 + per < n_keep ? p0 + per : n_keep;
      uint32_t e = 0, x = 0;
      for (uint32_t p = p0; p < p1; ++p) {
        const uint32_t s = f.state[p];
        const uint4 o0 = g.off[s], o1 = g.off[s + 1];
        e += o1.x - o0.x;
        x += o1.y - o0.y;
        f.ebeg[p] = o0.x;
        f.xbeg[p] = o0.y;
        f.edeg[p] = o1.x - o0.x;  // degrees for now, prefix sums below
        f.xdeg[p] = o1.y - o0.y;
        f.cls[p] = g.sclass[s];
      }
      uint64_t tot2;
      const uint64_t ex2 = block_excl_scan64(((uint64_t)x << 32) | e, sh.bs, par, &tot2);
      uint32_t eb = (uint32_t)ex2, xb = (uint32_t)(ex2 >> 32);
      W_next = (uint32_t)tot2;
      W_eps = (uint32_t)(tot2 >> 32);
      for (uint32_t p = p0; p < p1; ++p) {
        const uint32_t de = f.edeg[p], dx = f.xdeg[p];
        f.edeg[p] = eb;
        f.xdeg[p] = xb;
        eb += de;
        xb += dx;
      }
      if (tid == 0) {
        f.edeg[n_keep] = W_next;
        f.xdeg[n_keep] = W_eps;
      }
      __syncthreads();
    }
    stamp(6);
    // owners of the next frame's emitting work items, one item per thread
    // of the lower half (each found by a search of the degree prefix sums:
    // a token's own loop over its arcs would serialise a high out-degree)
    const bool own_e_ok = fl && W_next <= kOwnE;
    if (own_e_ok && tid < 512u)
      for (uint32_t k = tid; k < W_next; k += 512u) own_e[k] = (uint16_t)search_le(fs.edeg, n_keep, k);
    if (tid == kBook) {
      L.node_off[t] = node_base;
      L.node_off[t + 1] = node_base + n_keep;
      L.best[t] = best;
      L.cutb[t] = cutb;
      L.cut[t] = key_cost(cut_key);
    }
    if (tid == kBook) {
      sh.c_tokens += n_keep;
      if (n_keep > sh.c_max_tokens) sh.c_max_tokens = n_keep;
    }
    // Warm the caches for frame t+1: one load per 128-byte line of its
    // log-likelihood row and one per work item of its first 256 emitting
    // arcs, issued by the upper wavefronts (the lower half fills the owners).
    // Each value replaces the thread's last one rather than adding to it: an
    // addition would wait for the load here, before the frame's last barrier.
    if (t < T) {
      if (tid >= 768u) {
        const uint32_t k = (tid - 768u) * 32u;
        if (k < P) warm = L.ll[(size_t)t * P + k];
      } else if (fl && tid >= 512u && tid - 512u < W_next) {
        const uint32_t w = tid - 512u, p = search_le(fs.edeg, n_keep, w);
        warm = __uint_as_float(g.earc[fs.ebeg[p] + (w - fs.edeg[p])].y);
      }
    }
    // (the frame's lattice links are formed after the forward pass, from the
    // node store: every frame at once, off this chain)
    stamp(7);
    // a payload no sum of a finite weight and a log-likelihood has: keeps the
    // warming loads, whose values are read a frame later, so that no
    // wavefront waits for them before the frame's last barrier
    warm_bad |= __float_as_uint(warm_prev) == 0x7fc00001u ? 1u : 0u;
    warm_prev = warm;
    stamp(8);
    note(kProfStamps, (lds ? 1ull : 0ull) | ((uint64_t)n_keep << 8));
    note(kProfStamps + 1, (t > 0 ? (uint64_t)W : 0ull) | ((uint64_t)(lds ? sh.n_bk : 0u) << 32));
    // ----------------------------------------------------- next frame
    node_base += n_keep;
    n_prev = n_keep;
    W = W_next;
    front_lds = fl;
    front_own = own_e_ok;
    // (the frame's last reads of these counters came before the degree
    // pass's barrier)
    for (uint32_t i = tid; i <= (uint32_t)kMaxLevels; i += kThreads) sh.nb[i] = 0;
    for (uint32_t i = tid; i < (uint32_t)kHistBins; i += kThreads) sh.hist[i] = 0;
    h_clear(sh, h_used_n);
    if (tid == 0) {
      sh.n_touched = 0;
      sh.n_surv = 0;
      sh.n_rank = 0;
    }
    __syncthreads();
    stamp(9);
  }

  if (L.open && front_lds) {  // an open stream resumes from the workspace frontier
    for (uint32_t i = tid; i <= n_prev; i += kThreads) {
      L.f_edeg[i] = sh.f_edeg[i];
      L.f_xdeg[i] = sh.f_xdeg[i];
      if (i == n_prev) continue;
      L.f_state[i] = sh.f_state[i];
      L.f_key[i] = sh.f_key[i];
      L.f_arc[i] = sh.f_arc[i];
      L.f_ebeg[i] = sh.f_ebeg[i];
      L.f_xbeg[i] = sh.f_xbeg[i];
      L.f_cls[i] = sh.f_cls[i];
    }
  }
  warm_bad |= __float_as_uint(warm_prev) == 0x7fc00001u ? 1u : 0u;
  const uint32_t wb = block_or(warm_bad, sh.bs, par);
  const uint64_t eps = block_sum64(my_eps, sh.bs, par);
  const uint64_t arcs = sh.c_arcs + eps;  // (the bookkeeping thread's writes, before the barrier)
  if (tid == 0) {
    LaneInfo* info = L.info;
    if (status == 0 && wb) status = kStatusInternal;
    if (status == 0 && (ovf & kOvfNodes)) status = 4;
    info->status = status;
    info->frames_done = t;
    info->overflow = ovf;
    info->arcs_expanded = arcs;
    info->eps_arcs = eps;
    info->tokens = sh.c_tokens;
    info->max_tokens = sh.c_max_tokens;
    // (links, need_links: set by the link kernels after the forward pass)
    info->need_frame_tokens = sh.c_need_frame;
    info->need_frame_arcs = sh.c_need_arcs;
    info->last_tokens = n_prev;
  }
}

__global__ void __launch_bounds__(kThreads) k_forward(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                      Params prm, const uint32_t* __restrict__ bad) {
  __shared__ FwdShared sh;
  forward_body<false>(sh, g, lanes, prm, bad);
}

__global__ void __launch_bounds__(kThreads) k_forward_phases(DevGraph g, const LaneDesc* __restrict__ lanes,
                                                             Params prm, const uint32_t* __restrict__ bad) {
  __shared__ FwdShared sh;
  forward_body<true>(sh, g, lanes, prm, bad);
}

void launch_forward(const DevGraph& g, const LaneDesc* lanes, int B, const Params& prm,
                    const uint32_t* bad, hipStream_t s) {
  if (prm.flags & WD_FLAG_PHASES)
    hipLaunchKernelGGL(k_forward_phases, dim3(B), dim3(kThreads), 0, s, g, lanes, prm, bad);
  else
    hipLaunchKernelGGL(k_forward, dim3(B), dim3(kThreads), 0, s, g, lanes, prm, bad);
}

}  // namespace wd
