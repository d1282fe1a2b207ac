// Shared definitions of the wfstdec GPU library (host and device).
//
// Decoder state follows the paper's token passing (Sec. 3.2): every WFST state
// holds at most one token per frame; recombination keeps the candidate with the
// smallest (cost, arc id), packed into one 64-bit word so a single atomicMin
// decides it (Alg. 1).  Costs are fp32; the packing uses an order-preserving
// fp32 -> u32 key so negative costs order correctly.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wd {

constexpr uint64_t kEmpty = ~0ull;          // slot holds no token
constexpr uint32_t kNoArc = 0xffffffffu;    // predecessor of the start token
constexpr uint32_t kNoEps = 0xffu;          // class byte: state has no epsilon out-arcs
constexpr int kMaxLevels = 254;             // epsilon levels 0..253
constexpr int kThreads = 1024;              // one workgroup per utterance
constexpr int kWaves = kThreads / 64;
constexpr int kRankMax = 2048;              // survivors sorted in LDS up to this many
constexpr int kHashCap = 4096;              // LDS token table slots (power of two)
constexpr int kHashMax = 2048;              // LDS token table entries before a frame spills
constexpr int kFrontCap = 1024;             // frontier tokens held in LDS
constexpr int kHistBins = 2048;             // 11-bit radix digits for max-active
constexpr uint32_t kInfKey = 0xff800000u;   // key of +inf
constexpr uint32_t kPathMaxLen = 16;        // epsilon paths longer than this: no path table
constexpr uint64_t kPathMax = 1ull << 27;   // more epsilon paths than this: no path table
constexpr int kProfStamps = 10;             // step boundaries stamped per frame (WD_FLAG_PHASES)
constexpr int kProfSlots = kProfStamps + 2; // + two words describing the frame
constexpr int kLatStamps = 8;               // lattice-pass stamps (in the row after the last frame's)

// Order-preserving map of fp32 onto u32 (-0.0 folded onto +0.0): for non-NaN
// a, b: a < b  <=>  cost_key(a) < cost_key(b).
__host__ __device__ inline uint32_t cost_key(float x) {
  union { float f; uint32_t u; } v;
  v.f = (x == 0.0f) ? 0.0f : x;
  return (v.u & 0x80000000u) ? ~v.u : (v.u | 0x80000000u);
}

__host__ __device__ inline float key_cost(uint32_t k) {
  union { float f; uint32_t u; } v;
  v.u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return v.f;
}

__host__ __device__ inline uint64_t pack_tok(uint32_t key, uint32_t arc) {
  return ((uint64_t)key << 32) | arc;
}

// Forward-backward in the linear domain.  For frame t let b(t) be its best
// token cost and B the best total cost; the passes carry, per lattice node n
// of frame t, Sa(n) = exp(b(t) - alpha(n)) and Sb(n) = exp(B - b(t) -
// beta(n)).  Each kept link then moves mass by one factor, the same for both
// passes: exp(b(t) - b(t-1) - graph cost - acoustic cost) for an emitting
// link into frame t, exp(-graph cost) for an epsilon link.  Every term of a
// kept link lies within exp(-(beam + lattice beam)) .. exp(beam + log of the
// number of near-best paths), far inside fp64's range.
#if defined(__HIPCC__)
__device__ inline double emit_factor(float best_t, float best_prev, float graph, double ac) {
  return exp((double)best_t - (double)best_prev - (double)graph - ac);
}
__device__ inline double eps_factor(float graph) { return exp(-(double)graph); }
// An epsilon link's record keeps its source level in the factor's lowest 8
// mantissa bits (a relative change below 2^-44).
__device__ inline uint2 factor_bits(double f, bool eps, uint32_t lvl) {
  const uint64_t u = (uint64_t)__double_as_longlong(f);
  const uint64_t v = eps ? ((u & ~0xffull) | (lvl & 0xffu)) : u;
  return make_uint2((uint32_t)v, (uint32_t)(v >> 32));
}
#endif

// Device copy of the decoding graph, laid out in one caller-owned buffer.
//   off[s]  = {first emitting arc, first epsilon arc, first epsilon path, 0} of
//             state s (S+1 entries; the path index is 0 without a path table)
//   earc[i] = {dst, weight bits, ilabel | dst_class << 24, arc id}
//   xarc[j] = {dst, weight bits, dst_class, arc id}
//   xnext[j] = epsilon arc range {first, end} of xarc[j]'s destination
// Arcs of a state keep the caller's order, so within a state arc ids ascend.
// dst_class is the epsilon level of the destination state when it has
// epsilon out-arcs, else kNoEps.  Epsilon arcs always climb to a strictly
// higher level, so relaxing levels in order closes a frame exactly.
struct DevGraph {
  const uint4* off;
  const uint4* earc;
  const uint4* xarc;
  const uint2* xnext;
  const uint8_t* sclass;       // [S] class of every state
  const float* final_w;        // [S] or nullptr
  const int32_t* ilabel_id;    // [A] by caller arc id
  const int32_t* olabel_id;    // [A]
  const float* weight_id;      // [A]
  const uint32_t* level_base;  // [nlevels + 1] bucket offsets of the epsilon levels
  // Epsilon paths (every path of one or more epsilon arcs out of a state,
  // enumerated when the graph is loaded; npaths = 0 when the graph has too
  // many or too long ones).  Paths of state s: [off[s].z, off[s+1].z).
  //   phead[2p] = {last state, last arc id, last arc's weight bits, k | xdeg << 8}
  //     k = number of arcs, xdeg = epsilon out-degree of the last state
  //   phead[2p + 1] = bits of the weights of arcs 0..3 (those < k - 1; else 0),
  //     so that a path of up to five arcs is one 32-byte record
  //   ptail[p * pstride + i] = weight of arc i < k - 1 (pstride = longest path - 1)
  const uint4* phead;
  const float* ptail;
  uint64_t npaths;
  uint32_t pstride;
  uint32_t S;
  uint32_t start;
  uint32_t nlevels;
  uint32_t P;
  uint64_t Ae;
  uint64_t Ax;
  uint64_t A;
};

struct Params {
  float beam;
  int32_t max_active;
  float lattice_beam;
  uint32_t flags;
};

// Per-utterance counters and status, written by the kernels.
struct LaneInfo {
  int32_t status;              // WD_* code
  int32_t frames_done;
  int32_t final_used;
  uint32_t overflow;           // bit mask of exceeded capacities (kOvf*)
  uint64_t arcs_expanded;
  uint64_t eps_arcs;           // epsilon part of arcs_expanded
  uint64_t tokens;             // surviving tokens summed over frames (= nodes recorded)
  uint64_t max_tokens;
  uint64_t links;              // raw lattice links (all ever recorded)
  uint64_t need_links;         // link store capacity the decode needed (peak; with
                               // incremental pruning: the compacted region)
  uint64_t need_window;        // incremental pruning: raw links of the largest window
  uint64_t need_frame_tokens;  // largest per-frame touched-state count
  uint64_t need_frame_arcs;    // largest per-frame emitting work
  uint64_t kept;               // kept lattice links
  uint64_t out_nodes;
  uint64_t nwords;
  uint64_t out_raw;            // raw links written to the debug output
  uint32_t start_node;
  uint32_t best_node;
  float best_cost;
  uint32_t tb_fail;            // traceback met an inconsistent predecessor
  uint32_t last_tokens;        // surviving tokens of the last decoded frame
  uint32_t pad0;
  double Z;                    // total cost of the kept lattice (-log of its path sum)
};

enum : uint32_t { kOvfFrame = 1, kOvfArcs = 2, kOvfNodes = 4, kOvfLinks = 8, kOvfKept = 16 };
// Params::flags bit set by the host for the lattice kernel when the pruning
// sweep already ran as chip-wide kernels.
constexpr uint32_t kFlagSwept = 1u << 30;
// LaneInfo::status value for an internal consistency failure caught by a
// kernel's own bounds checks (reported as WD_EDEVICE).
constexpr int32_t kStatusInternal = 5;

// Device output records (match wd_lat_arc / wd_lat_node / wd_token of wfstdec.h).
struct OutLink {
  int32_t t;
  uint32_t arc_id;
  int32_t src_state;
  int32_t dst_state;
  int32_t ilabel;
  int32_t olabel;
  float graph_cost;
  float ac_cost;
  float fwd_cost;
  float extra;
  double posterior;
};
struct OutNode {
  int32_t t;
  int32_t state;
  float cost;
  float extra;
};

// Pointers into device memory seen from device code: in the global address
// space, so that every access through them is a global memory instruction.
// (A pointer of unknown address space compiles to flat instructions, and a
// wait for a flat load waits for every load in flight, which would stall the
// loads the kernels issue a frame ahead.)  Host code sees plain pointers;
// both views have the same layout.
#if defined(__HIP_DEVICE_COMPILE__)
#define WD_GLOBAL __attribute__((address_space(1)))
#else
#define WD_GLOBAL
#endif

// Everything one utterance needs on the device.  Built on the host; lives in
// the workspace.
struct LaneDesc {
  const WD_GLOBAL float* ll;             // T x P log-likelihoods (row t-1 belongs to frame t)
  int32_t T;                   // last frame (streaming: the last frame received so far)
  int32_t t0;                  // first frame this launch decodes; > 0 resumes a stream
  int32_t open;                // streaming: more frames may follow
  int32_t pad0;
  uint64_t frame_cap, cand_cap, node_cap, link_cap, kept_cap, word_cap;
  uint64_t win_cap;            // incremental pruning: links of one raw window slot (0: off)
  // per-frame scratch
  WD_GLOBAL unsigned long long* slot;    // [S] packed (cost key, arc id); kEmpty between frames
  WD_GLOBAL uint32_t* idx;               // [S] node id of a state in the current frame / scratch
  WD_GLOBAL uint32_t* bitmap;            // [ceil(S/32)] zero between frames
  WD_GLOBAL uint32_t* touched;           // [frame_cap] states touched this frame
  WD_GLOBAL uint32_t* bucket;            // [S] touched states with epsilon arcs, by level
  WD_GLOBAL uint32_t* surv_state;        // [frame_cap] tokens within the beam cutoff
  WD_GLOBAL unsigned long long* surv_pack;
  // frontier: surviving tokens of the last finished frame, sorted by state
  // (used when a frame has more survivors than the LDS frontier holds)
  WD_GLOBAL uint32_t* f_state;
  WD_GLOBAL uint32_t* f_key;             // cost key
  WD_GLOBAL uint32_t* f_arc;             // predecessor arc
  WD_GLOBAL uint32_t* f_edeg;            // exclusive prefix of emitting out-degree (+ total)
  WD_GLOBAL uint32_t* f_xdeg;            // exclusive prefix of epsilon out-degree (+ total)
  WD_GLOBAL uint32_t* f_ebeg;            // first emitting arc of the state
  WD_GLOBAL uint32_t* f_xbeg;            // first epsilon arc of the state
  WD_GLOBAL uint8_t* f_cls;
  WD_GLOBAL uint4* cand;                 // [cand_cap] emitting candidates {arc, src node, dst, x bits}
  // history
  WD_GLOBAL uint32_t* n_state;           // [node_cap]
  WD_GLOBAL unsigned long long* n_pack;  // [node_cap] (cost key, predecessor arc)
  WD_GLOBAL uint32_t* n_pred;            // [node_cap] predecessor node
  // link store [link_cap + 3*win_cap]: with incremental pruning, the compacted
  // region [0, link_cap) then three raw window slots of win_cap links each
  WD_GLOBAL uint4* links;                // {arc, src node, dst node, x bits}
  WD_GLOBAL uint8_t* link_lvl;           // epsilon level of the source (epsilon links)
  WD_GLOBAL uint64_t* node_off;          // [T+2]
  WD_GLOBAL uint64_t* link_off;          // [T+2] first link of frame t (emitting run)
  WD_GLOBAL uint64_t* link_xoff;         // [T+2] first epsilon link of frame t
  WD_GLOBAL uint64_t* link_end;          // [T+2] one past the last link of frame t
  WD_GLOBAL uint32_t* xmask;             // [T+2] levels of the epsilon links of frame t (bit 31: 31 or more)
  WD_GLOBAL float* best;                 // [T+1]
  WD_GLOBAL float* cutb;                 // [T+1]
  WD_GLOBAL float* cut;                  // [T+1]
  // lattice pass
  WD_GLOBAL uint32_t* extra_key;         // [node_cap]
  WD_GLOBAL uint32_t* le_key;            // [link_cap + 3*win_cap]
  WD_GLOBAL double* alpha;               // [node_cap] forward sums Sa (linear domain)
  WD_GLOBAL double* beta;                // [node_cap] backward sums Sb (linear domain)
  WD_GLOBAL uint32_t* used;              // [ceil(node_cap/32)+1] lattice-node bitmap
  WD_GLOBAL uint64_t* kept_idx;          // [kept_cap] kept link ids in link order
  WD_GLOBAL uint4* post;                 // [kept_cap] kept links for forward-backward:
                               //   {src node, dst node, factor bits lo, hi (| source level)}
  WD_GLOBAL uint64_t* kframe;            // [2*(T+2)] per frame: first kept link, first kept epsilon link
  // outputs
  WD_GLOBAL OutLink* out_links;          // [kept_cap]
  WD_GLOBAL OutLink* out_raw;            // [raw_cap] every raw link (debug output)
  uint64_t raw_cap;
  WD_GLOBAL OutNode* out_nodes;          // [2*kept_cap+1]
  WD_GLOBAL int32_t* out_words;          // [word_cap]
  WD_GLOBAL LaneInfo* info;
  WD_GLOBAL uint64_t* prof;              // [(T+1) * kProfSlots] step profile (WD_FLAG_PHASES)
};

}  // namespace wd
