// Decode entry points: workspace layout, launches, results.
//
// One workgroup decodes one utterance from the first frame to the last inside
// one launch (no per-frame host round trips; the paper's "other" time of
// launches and synchronisation, Sec. 4.3, is what this avoids).  A batch runs
// its utterances as concurrent workgroups sharing the resident graph, which is
// the paper's sequence parallelism (Sec. 4.2) done in one process.
#include <algorithm>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "wd_host.h"

namespace wd {

static thread_local std::string g_err;

void set_error(const std::string& msg) { g_err = msg; }

wd_status fail(wd_status st, const std::string& msg) {
  g_err = msg;
  return st;
}

wd_status hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return WD_OK;
  return fail(WD_EDEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

namespace {

struct Caps {
  uint64_t frame, arcs, nodes, links, kept, raw, words, win;
  uint64_t prof;  // step-profile words per utterance (WD_FLAG_PHASES)
};

// Execution mode: chip-wide kernels per frame for frames too large for one
// workgroup (no max-active limit, or a very large one).
bool chip_wide_mode(const wd_params* p) {
  return (p->flags & WD_FLAG_CHIP_WIDE) ||
         (!(p->flags & WD_FLAG_ONE_WORKGROUP) && (p->max_active == 0 || p->max_active >= WD_CHIP_WIDE_MAX_ACTIVE));
}

bool incremental_prune(const wd_params* p) {
  return chip_wide_mode(p) && !(p->flags & (WD_FLAG_DEBUG | WD_FLAG_NO_INCREMENTAL_PRUNE));
}

Caps resolve_caps(const wd_graph* g, int32_t max_T, const wd_params* p, const wd_caps* c) {
  Caps r{};
  const uint64_t S = (uint64_t)g->S;
  const uint64_t ma = p->max_active > 0 ? (uint64_t)p->max_active : 0;
  r.frame = (c && c->frame_tokens > 0) ? (uint64_t)c->frame_tokens
                                       : (ma ? std::min<uint64_t>(S, std::max<uint64_t>(65536, 16 * ma)) : S);
  r.frame = std::min<uint64_t>(r.frame, S);
  r.arcs = (c && c->frame_arcs > 0) ? (uint64_t)c->frame_arcs
                                    : (ma ? std::min<uint64_t>(g->Ae, std::max<uint64_t>(262144, 64 * ma)) : g->Ae);
  r.arcs = std::max<uint64_t>(std::min<uint64_t>(r.arcs, g->Ae), 1);
  const uint64_t T1 = (uint64_t)max_T + 1;
  r.nodes = (c && c->nodes > 0) ? (uint64_t)c->nodes : T1 * std::min<uint64_t>(S, 1024);
  r.nodes = std::min<uint64_t>(r.nodes, 0xfffffff0ull);
  r.links = (c && c->links > 0) ? (uint64_t)c->links : 4 * r.nodes;
  r.kept = (c && c->kept_links > 0) ? (uint64_t)c->kept_links : std::min<uint64_t>(r.links, 1u << 20);
  r.raw = (p->flags & WD_FLAG_DEBUG) ? r.links : 0;
  r.win = 0;
  if (incremental_prune(p))
    r.win = (c && c->window_links > 0) ? (uint64_t)c->window_links : std::max<uint64_t>(r.links / 4, 1);
  r.words = T1 * (g->nlevels + 1) + 1;
  // (one row per frame, then one for the lattice pass)
  r.prof = (p->flags & WD_FLAG_PHASES) ? (T1 + 1) * (uint64_t)kProfSlots : 0;
  return r;
}

// Lays every per-utterance array out as one region per array (all lanes side
// by side) so the per-decode resets are one fill each.  With base == nullptr
// only sizes the workspace.
struct Regions {
  LaneDesc* desc;
  LaneInfo* info;
  uint32_t* bad;
  unsigned long long* slot;
  uint32_t* bitmap;
  uint32_t* used;
  void* grid;
  uint64_t bitmap_words, used_words;
  uint64_t total;
};

Regions carve(const wd_graph* g, int B, int32_t max_T, const Caps& c, char* base, LaneDesc* lanes) {
  Regions R{};
  uint64_t p = 0;
  auto take = [&](uint64_t per_lane_bytes) -> char* {
    char* at = base ? base + p : nullptr;
    p = align_up(p + per_lane_bytes * (uint64_t)B, 256);
    return at;
  };
  const uint64_t S = (uint64_t)g->S;
  const uint64_t F1 = c.frame + 1;
  const uint64_t T2 = (uint64_t)max_T + 2;
  R.desc = (LaneDesc*)take(sizeof(LaneDesc));
  R.info = (LaneInfo*)take(sizeof(LaneInfo));
  R.bad = (uint32_t*)take(sizeof(uint32_t));
  R.grid = take(grid_lane_bytes());
  R.bitmap_words = (S + 31) / 32;
  R.used_words = (c.nodes + 31) / 32 + 1;
  char* slot = take(8 * S);
  char* idx = take(4 * S);
  char* bitmap = take(4 * R.bitmap_words);
  char* bucket = take(4 * S);
  char* touched = take(4 * c.frame);
  char* surv_state = take(4 * c.frame);
  char* surv_pack = take(8 * c.frame);
  char* f_state = take(4 * F1);
  char* f_key = take(4 * F1);
  char* f_arc = take(4 * F1);
  char* f_edeg = take(4 * F1);
  char* f_xdeg = take(4 * F1);
  char* f_ebeg = take(4 * F1);
  char* f_xbeg = take(4 * F1);
  char* f_cls = take(F1);
  char* cand = take(16 * c.arcs);
  char* n_state = take(4 * c.nodes);
  char* n_pack = take(8 * c.nodes);
  char* n_pred = take(4 * c.nodes);
  const uint64_t nlink = c.links + grid_window_slots() * c.win;  // compacted region + raw window slots
  char* links = take(16 * nlink);
  char* link_lvl = take(nlink);
  char* node_off = take(8 * T2);
  char* link_off = take(8 * T2);
  char* link_xoff = take(8 * T2);
  char* link_end = take(8 * T2);
  char* xmask = take(4 * T2);
  char* best = take(4 * T2);
  char* cutb = take(4 * T2);
  char* cut = take(4 * T2);
  char* extra_key = take(4 * c.nodes);
  char* le_key = take(4 * nlink);
  char* alpha = take(8 * c.nodes);
  char* beta = take(8 * c.nodes);
  char* used = take(4 * R.used_words);
  char* kept_idx = take(8 * c.kept);
  char* post = take(16 * c.kept);
  char* kframe = take(16 * T2);
  char* out_links = take(sizeof(OutLink) * c.kept);
  char* out_raw = take(sizeof(OutLink) * c.raw);
  char* out_nodes = take(sizeof(OutNode) * (2 * c.kept + 1));
  char* out_words = take(4 * c.words);
  char* prof = take(8 * c.prof);
  R.total = p;
  R.slot = (unsigned long long*)slot;
  R.bitmap = (uint32_t*)bitmap;
  R.used = (uint32_t*)used;
  if (lanes) {
    for (int b = 0; b < B; ++b) {
      LaneDesc& L = lanes[b];
      auto at = [&](char* region, uint64_t per_lane) { return region + (uint64_t)b * per_lane; };
      L.frame_cap = c.frame;
      L.cand_cap = c.arcs;
      L.node_cap = c.nodes;
      L.link_cap = c.links;
      L.win_cap = c.win;
      L.kept_cap = c.kept;
      L.raw_cap = c.raw;
      L.word_cap = c.words;
      L.slot = (decltype(L.slot))at(slot, 8 * S);
      L.idx = (decltype(L.idx))at(idx, 4 * S);
      L.bitmap = (decltype(L.bitmap))at(bitmap, 4 * R.bitmap_words);
      L.bucket = (decltype(L.bucket))at(bucket, 4 * S);
      L.touched = (decltype(L.touched))at(touched, 4 * c.frame);
      L.surv_state = (decltype(L.surv_state))at(surv_state, 4 * c.frame);
      L.surv_pack = (decltype(L.surv_pack))at(surv_pack, 8 * c.frame);
      L.f_state = (decltype(L.f_state))at(f_state, 4 * F1);
      L.f_key = (decltype(L.f_key))at(f_key, 4 * F1);
      L.f_arc = (decltype(L.f_arc))at(f_arc, 4 * F1);
      L.f_edeg = (decltype(L.f_edeg))at(f_edeg, 4 * F1);
      L.f_xdeg = (decltype(L.f_xdeg))at(f_xdeg, 4 * F1);
      L.f_ebeg = (decltype(L.f_ebeg))at(f_ebeg, 4 * F1);
      L.f_xbeg = (decltype(L.f_xbeg))at(f_xbeg, 4 * F1);
      L.f_cls = (decltype(L.f_cls))at(f_cls, F1);
      L.cand = (decltype(L.cand))at(cand, 16 * c.arcs);
      L.n_state = (decltype(L.n_state))at(n_state, 4 * c.nodes);
      L.n_pack = (decltype(L.n_pack))at(n_pack, 8 * c.nodes);
      L.n_pred = (decltype(L.n_pred))at(n_pred, 4 * c.nodes);
      L.links = (decltype(L.links))at(links, 16 * nlink);
      L.link_lvl = (decltype(L.link_lvl))at(link_lvl, nlink);
      L.node_off = (decltype(L.node_off))at(node_off, 8 * T2);
      L.link_off = (decltype(L.link_off))at(link_off, 8 * T2);
      L.link_xoff = (decltype(L.link_xoff))at(link_xoff, 8 * T2);
      L.link_end = (decltype(L.link_end))at(link_end, 8 * T2);
      L.xmask = (decltype(L.xmask))at(xmask, 4 * T2);
      L.best = (decltype(L.best))at(best, 4 * T2);
      L.cutb = (decltype(L.cutb))at(cutb, 4 * T2);
      L.cut = (decltype(L.cut))at(cut, 4 * T2);
      L.extra_key = (decltype(L.extra_key))at(extra_key, 4 * c.nodes);
      L.le_key = (decltype(L.le_key))at(le_key, 4 * nlink);
      L.alpha = (decltype(L.alpha))at(alpha, 8 * c.nodes);
      L.beta = (decltype(L.beta))at(beta, 8 * c.nodes);
      L.used = (decltype(L.used))at(used, 4 * R.used_words);
      L.kept_idx = (decltype(L.kept_idx))at(kept_idx, 8 * c.kept);
      L.post = (decltype(L.post))at(post, 16 * c.kept);
      L.kframe = (decltype(L.kframe))at(kframe, 16 * T2);
      L.out_links = (decltype(L.out_links))at(out_links, sizeof(OutLink) * c.kept);
      L.out_raw = (decltype(L.out_raw))at(out_raw, sizeof(OutLink) * c.raw);
      L.out_nodes = (decltype(L.out_nodes))at(out_nodes, sizeof(OutNode) * (2 * c.kept + 1));
      L.out_words = (decltype(L.out_words))at(out_words, 4 * c.words);
      L.prof = c.prof ? (decltype(L.prof))at(prof, 8 * c.prof) : nullptr;
      L.info = (decltype(L.info))(R.info + b);
    }
  }
  return R;
}

wd_status check_params(const wd_params* p) {
  if (!p) return fail(WD_EINVAL, "decode: null params");
  if (!(p->beam > 0.0f)) return fail(WD_EINVAL, "decode: beam must be > 0");
  if (p->max_active < 0) return fail(WD_EINVAL, "decode: max_active must be >= 0");
  if (!(p->lattice_beam >= 0.0f)) return fail(WD_EINVAL, "decode: lattice_beam must be >= 0");
  if ((p->flags & WD_FLAG_ONE_WORKGROUP) && (p->flags & WD_FLAG_CHIP_WIDE))
    return fail(WD_EINVAL, "decode: WD_FLAG_ONE_WORKGROUP and WD_FLAG_CHIP_WIDE are exclusive");
  if ((p->flags & WD_FLAG_PHASES) && chip_wide_mode(p))
    return fail(WD_EINVAL, "decode: WD_FLAG_PHASES profiles the one-workgroup forward pass only");
  return WD_OK;
}

}  // namespace

}  // namespace wd

struct wd_result {
  wd_status status = WD_OK;
  float cost = 0.0f;
  std::vector<int32_t> words;
  std::vector<wd_lat_arc> links, raw;
  std::vector<wd_lat_node> nodes;
  std::vector<wd_token> tokens;
  std::vector<float> best, cutb, cut;
  std::vector<uint64_t> prof;  // WD_FLAG_PHASES: (T+2) x WD_PHASE_SLOTS (the last row: the lattice pass)
  double tick_hz = 0.0;
  wd_stats stats{};
};

static_assert(sizeof(wd_lat_arc) == sizeof(wd::OutLink), "link record layout");
static_assert(wd::kLatStamps == WD_LATTICE_PHASE_STAMPS && wd::kLatStamps <= wd::kProfSlots, "lattice profile row");
static_assert(sizeof(wd_lat_node) == sizeof(wd::OutNode), "node record layout");

using namespace wd;

extern "C" wd_status wd_workspace_bytes(const wd_graph* g, int32_t lanes, int32_t max_T, const wd_params* p,
                                        const wd_caps* caps, size_t* bytes, wd_caps* caps_out) {
  if (!g || !bytes || lanes < 1 || max_T < 0 || max_T > (1 << 24))
    return fail(WD_EINVAL, "workspace_bytes: bad arguments");
  wd_status st = check_params(p);
  if (st != WD_OK) return st;
  const Caps c = resolve_caps(g, max_T, p, caps);
  *bytes = carve(g, lanes, max_T, c, nullptr, nullptr).total;
  if (caps_out) {
    caps_out->frame_tokens = (int64_t)c.frame;
    caps_out->frame_arcs = (int64_t)c.arcs;
    caps_out->nodes = (int64_t)c.nodes;
    caps_out->links = (int64_t)c.links;
    caps_out->kept_links = (int64_t)c.kept;
    caps_out->window_links = (int64_t)c.win;
  }
  return WD_OK;
}

// One decode of B utterances from setup to results: wd_decode_batch runs it
// in one call, a stream over several (begin, advances, end).
struct wd_stream {
  const wd_graph* g = nullptr;
  int B = 0;
  int32_t max_T = 0;
  wd_params p{};
  Params prm{};
  Caps c{};
  Regions R{};
  std::vector<LaneDesc> lanes;
  std::vector<int32_t> T;     // frames received per utterance
  std::vector<int32_t> next;  // first frame not yet decoded
  hipStream_t s = nullptr;
  bool chip = false, open = false;
  GridRun gr;
  hipEvent_t ev[3] = {nullptr, nullptr, nullptr};

  ~wd_stream() {
    grid_release(&gr);
    for (auto& e : ev)
      if (e) (void)hipEventDestroy(e);
  }
};

// Workspace layout, resets, the per-utterance state of the chosen mode.
static wd_status run_setup(wd_stream* run, const wd_graph* g, int32_t B, const float* const* ll, const int32_t* T,
                           int32_t max_T, const wd_params* p, const wd_caps* caps, void* ws, size_t ws_bytes,
                           void* stream, bool open) {
  run->g = g;
  run->B = B;
  run->max_T = max_T;
  run->p = *p;
  run->prm = Params{p->beam, p->max_active, p->lattice_beam, p->flags};
  run->c = resolve_caps(g, max_T, p, caps);
  run->lanes.assign((size_t)B, LaneDesc{});
  std::memset(run->lanes.data(), 0, sizeof(LaneDesc) * (size_t)B);
  run->R = carve(g, B, max_T, run->c, (char*)ws, run->lanes.data());
  const Regions& R = run->R;
  if (ws_bytes < R.total)
    return fail(WD_EINVAL, "decode: workspace of " + std::to_string(ws_bytes) + " bytes, need " +
                               std::to_string(R.total));
  run->T.assign(T, T + B);
  run->next.assign((size_t)B, 0);
  run->open = open;
  for (int b = 0; b < B; ++b) {
    run->lanes[b].ll = (decltype(run->lanes[b].ll))ll[b];
    run->lanes[b].T = T[b];
    run->lanes[b].t0 = 0;
    run->lanes[b].open = open ? 1 : 0;
  }
  run->s = (hipStream_t)stream;
  hipStream_t s = run->s;
  wd_status st;
  if ((st = hip_check(hipMemcpyAsync(R.desc, run->lanes.data(), sizeof(LaneDesc) * B, hipMemcpyHostToDevice, s),
                      "lane upload")))
    return st;
  const uint64_t S = (uint64_t)g->S;
  launch_fill_u32((uint32_t*)R.info, (uint64_t)B * sizeof(LaneInfo) / 4, 0u, s);
  launch_fill_u32(R.bad, (uint64_t)B, 0u, s);
  launch_fill_u64(R.slot, (uint64_t)B * S, kEmpty, s);
  launch_fill_u32(R.bitmap, (uint64_t)B * R.bitmap_words, 0u, s);
  launch_fill_u32(R.used, (uint64_t)B * R.used_words, 0u, s);
  if (p->flags & WD_FLAG_TIMING)
    for (auto& e : run->ev)
      if ((st = hip_check(hipEventCreate(&e), "event"))) return st;
  if (run->ev[0]) (void)hipEventRecord(run->ev[0], s);
  run->chip = chip_wide_mode(p);
  if (run->chip) return grid_begin(&run->gr, R.desc, R.grid, B, incremental_prune(p), R.bad, s);
  return WD_OK;
}

// Decodes every received frame not decoded yet (frame 0 in the first call).
static wd_status run_frames(wd_stream* run, bool update) {
  const Regions& R = run->R;
  hipStream_t s = run->s;
  const int B = run->B;
  if (update) launch_set_frames(R.desc, B, run->T.data(), run->next.data(), run->open ? 1 : 0, s);
  launch_check_loglikes(R.desc, B, run->g->P, R.bad, s);
  wd_status st = WD_OK;
  if (run->chip) {
    int lo = run->max_T + 1, hi = -1;
    for (int b = 0; b < B; ++b) {
      lo = std::min(lo, run->next[b]);
      hi = std::max(hi, run->T[b]);
    }
    st = grid_frames(&run->gr, run->g->dg, R.desc, R.grid, B, run->prm, R.bad, lo, hi, s);
  } else {
    launch_forward(run->g->dg, R.desc, B, run->prm, R.bad, s);
  }
  for (int b = 0; b < B; ++b) run->next[b] = run->T[b] + 1;
  if (st == WD_OK) st = hip_check(hipGetLastError(), "launch");
  return st;
}

static wd_stats lane_stats(const LaneInfo& I, int32_t T, float fwd_ms, float lat_ms, bool debug) {
  wd_stats stt{};
  stt.frames = T;
  stt.final_reached = I.final_used;
  stt.arcs_expanded = (int64_t)I.arcs_expanded;
  stt.tokens = (int64_t)I.tokens;
  stt.max_tokens = (int64_t)I.max_tokens;
  stt.raw_links = (int64_t)I.links;
  stt.kept_links = (int64_t)I.kept;
  stt.nodes = (int64_t)I.out_nodes;
  stt.eps_arcs_expanded = (int64_t)I.eps_arcs;
  stt.forward_ms = fwd_ms;
  stt.lattice_ms = lat_ms;
  stt.needed.frame_tokens = (int64_t)I.need_frame_tokens;
  stt.needed.frame_arcs = (int64_t)I.need_frame_arcs;
  stt.needed.nodes = (int64_t)I.tokens;
  stt.needed.links = (int64_t)I.need_links;
  stt.needed.window_links = (int64_t)I.need_window;
  stt.needed.kept_links = (int64_t)std::max<uint64_t>(I.kept, debug ? I.links : 0);
  return stt;
}

static const char* status_message(wd_status st) {
  return st == WD_ENOPATH     ? "decode: no token survived a frame"
         : st == WD_EINVAL    ? "decode: log-likelihoods contain NaN, +inf or values above 1e30"
         : st == WD_ECAPACITY ? "decode: workspace capacity exceeded; see stats.needed"
         : st == WD_EDEVICE   ? "decode: a kernel's internal consistency check failed"
                              : "decode failed";
}

// Lattice pass, then the results of every utterance (synchronises).
// Pinned host memory for result downloads, one buffer per device, grown on
// demand and kept until the process ends.  Its mutex is held from the copy
// until the results are unpacked (decodes on one device take turns there).
struct PinnedBuffer {
  std::mutex mu;
  char* p = nullptr;
  uint64_t cap = 0;
};

// Locks the current device's buffer (holding at least `bytes`) and returns it
// locked in *out.
static wd_status pinned_of_current_device(uint64_t bytes, PinnedBuffer** out) {
  static PinnedBuffer bufs[64];
  int dev = 0;
  wd_status st = hip_check(hipGetDevice(&dev), "device");
  if (st != WD_OK) return st;
  if (dev < 0 || dev >= 64) return fail(WD_EINVAL, "pinned buffer: device index out of range");
  PinnedBuffer& b = bufs[dev];
  b.mu.lock();
  if (b.cap < bytes) {
    if (b.p) (void)hipHostFree(b.p);
    b.p = nullptr;
    b.cap = 0;
    const uint64_t want = std::max<uint64_t>(bytes + bytes / 4, 1ull << 20);
    if ((st = hip_check(hipHostMalloc((void**)&b.p, want, hipHostMallocDefault), "pinned buffer"))) {
      b.p = nullptr;
      b.mu.unlock();
      return st;
    }
    b.cap = want;
  }
  *out = &b;
  return WD_OK;
}

static wd_status run_finish(wd_stream* run, wd_result** out) {
  const Regions& R = run->R;
  hipStream_t s = run->s;
  const int B = run->B;
  const wd_params* p = &run->p;
  wd_status st;
  if (run->chip && (st = grid_end(&run->gr, R.desc, R.grid, B, s))) return st;
  if (run->ev[1]) (void)hipEventRecord(run->ev[1], s);
  if (run->chip) {
    launch_grid_sweep(run->g->dg, R.desc, R.grid, B, run->max_T, p->lattice_beam, s);
    Params lp = run->prm;
    lp.flags |= kFlagSwept;
    launch_lattice(run->g->dg, R.desc, B, lp, s);
    launch_grid_nodes(R.desc, R.grid, B, s);
  } else {
    launch_links(run->g->dg, R.desc, B, s);
    launch_lattice(run->g->dg, R.desc, B, run->prm, s);
  }
  if (run->ev[2]) (void)hipEventRecord(run->ev[2], s);
  if ((st = hip_check(hipGetLastError(), "launch"))) return st;
  std::vector<LaneInfo> info((size_t)B);
  if ((st = hip_check(hipMemcpyAsync(info.data(), R.info, sizeof(LaneInfo) * B, hipMemcpyDeviceToHost, s),
                      "info download")) ||
      (st = hip_check(hipStreamSynchronize(s), "decode")))
    return st;

  float fwd_ms = 0.0f, lat_ms = 0.0f;
  if (run->ev[0]) {
    (void)hipEventElapsedTime(&fwd_ms, run->ev[0], run->ev[1]);
    (void)hipEventElapsedTime(&lat_ms, run->ev[1], run->ev[2]);
  }
  wd_status first_bad = WD_OK;
  const bool debug = (p->flags & WD_FLAG_DEBUG) != 0;
  // Without the debug outputs, the finished lanes' links, nodes and words
  // are packed on the device (into the candidate buffer, free after the
  // forward pass) and copied with one transfer instead of three per lane.
  std::vector<uint64_t> poff((size_t)B + 1, 0);
  for (int b = 0; b < B; ++b) {
    const LaneInfo& I = info[b];
    const uint64_t n = (I.status != 0 || I.tb_fail) ? 0
                       : sizeof(OutLink) * I.kept + sizeof(OutNode) * I.out_nodes + ((4 * I.nwords + 15) & ~15ull);
    poff[b + 1] = poff[b] + n;
  }
  const bool packed = !debug && poff[B] > 0 && poff[B] <= (uint64_t)B * run->c.arcs * 16;
  // the packed results land in the device's pinned download buffer (a DMA
  // straight into it; pageable memory would be copied through staging)
  PinnedBuffer* pin = nullptr;
  std::unique_lock<std::mutex> pin_lock;
  if (packed) {
    if ((st = pinned_of_current_device(poff[B], &pin))) return st;
    pin_lock = std::unique_lock<std::mutex>(pin->mu, std::adopt_lock);
    launch_pack_results(R.desc, B, run->lanes[0].cand, s);
    if ((st = hip_check(hipGetLastError(), "launch")) ||
        (st = hip_check(hipMemcpyAsync(pin->p, run->lanes[0].cand, poff[B], hipMemcpyDeviceToHost, s),
                        "result download")) ||
        (st = hip_check(hipStreamSynchronize(s), "result download")))
      return st;
  }
  for (int b = 0; b < B; ++b) {
    const LaneInfo& I = info[b];
    const LaneDesc& L = run->lanes[b];
    const int32_t Tb = run->T[b];
    const wd_status ls = (I.status == 0 && I.tb_fail) ? WD_EDEVICE : (wd_status)I.status;
    if (ls != WD_OK && first_bad == WD_OK) first_bad = ls;
    if (ls != WD_OK && ls != WD_ECAPACITY) continue;
    wd_result* r = new wd_result();
    r->status = ls;
    r->cost = I.best_cost;
    r->stats = lane_stats(I, Tb, fwd_ms, lat_ms, debug);
    out[b] = r;
    if (ls != WD_OK) continue;
    r->words.resize(I.nwords);
    r->links.resize(I.kept);
    r->nodes.resize(I.out_nodes);
    auto d2h = [&](void* dst, const void* src, uint64_t bytes) -> wd_status {
      if (!bytes) return WD_OK;
      return hip_check(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, s), "result download");
    };
    if (L.prof) {
      r->prof.resize(((size_t)Tb + 2) * kProfSlots);
      int khz = 0, dev = 0;
      if ((st = d2h(r->prof.data(), L.prof, 8 * r->prof.size())) ||
          (st = hip_check(hipGetDevice(&dev), "device")) ||
          (st = hip_check(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev), "clock rate")))
        return st;
      r->tick_hz = 1e3 * khz;
    }
    if (packed) continue;  // copied below, all lanes at once
    if ((st = d2h(r->words.data(), L.out_words, 4 * I.nwords)) ||
        (st = d2h(r->links.data(), L.out_links, sizeof(OutLink) * I.kept)) ||
        (st = d2h(r->nodes.data(), L.out_nodes, sizeof(OutNode) * I.out_nodes)))
      return st;
    if (debug) {
      const uint64_t nn = I.tokens;
      std::vector<uint32_t> ns(nn);
      std::vector<unsigned long long> np(nn);
      std::vector<uint64_t> noff((size_t)Tb + 2);
      r->raw.resize(I.out_raw);
      r->best.resize((size_t)Tb + 1);
      r->cutb.resize((size_t)Tb + 1);
      r->cut.resize((size_t)Tb + 1);
      if ((st = d2h(ns.data(), L.n_state, 4 * nn)) || (st = d2h(np.data(), L.n_pack, 8 * nn)) ||
          (st = d2h(noff.data(), L.node_off, 8 * ((uint64_t)Tb + 2))) ||
          (st = d2h(r->raw.data(), L.out_raw, sizeof(OutLink) * I.out_raw)) ||
          (st = d2h(r->best.data(), L.best, 4 * ((uint64_t)Tb + 1))) ||
          (st = d2h(r->cutb.data(), L.cutb, 4 * ((uint64_t)Tb + 1))) ||
          (st = d2h(r->cut.data(), L.cut, 4 * ((uint64_t)Tb + 1))) ||
          (st = hip_check(hipStreamSynchronize(s), "debug download")))
        return st;
      r->tokens.resize(nn);
      for (int t = 0; t <= Tb; ++t)
        for (uint64_t n = noff[t]; n < noff[t + 1]; ++n)
          r->tokens[n] = wd_token{t, (int32_t)ns[n], key_cost((uint32_t)(np[n] >> 32)), (uint32_t)np[n]};
    }
  }
  if (packed)
    for (int b = 0; b < B; ++b) {
      wd_result* r = out[b];
      if (!r || r->status != WD_OK) continue;
      const char* src = pin->p + poff[b];
      std::memcpy(r->links.data(), src, sizeof(OutLink) * r->links.size());
      src += sizeof(OutLink) * r->links.size();
      std::memcpy(r->nodes.data(), src, sizeof(OutNode) * r->nodes.size());
      src += sizeof(OutNode) * r->nodes.size();
      std::memcpy(r->words.data(), src, 4 * r->words.size());
    }
  if ((st = hip_check(hipStreamSynchronize(s), "result download"))) return st;
  if (first_bad != WD_OK) set_error(status_message(first_bad));
  return first_bad;
}

static wd_status check_lanes(const wd_graph* g, int32_t B, const float* const* ll, const int32_t* T,
                             wd_result** out) {
  if (!g || B < 1 || !ll || !T || !out) return fail(WD_EINVAL, "decode: bad arguments");
  for (int b = 0; b < B; ++b) out[b] = nullptr;
  for (int b = 0; b < B; ++b) {
    if (T[b] < 0 || T[b] > (1 << 24)) return fail(WD_EINVAL, "decode: T out of range");
    if (T[b] > 0 && !ll[b]) return fail(WD_EINVAL, "decode: null log-likelihoods");
  }
  return WD_OK;
}

static wd_status decode_impl(const wd_graph* g, int32_t B, const float* const* ll, const int32_t* T,
                             const wd_params* p, const wd_caps* caps, void* ws, size_t ws_bytes,
                             void* stream, wd_result** out) {
  wd_status st = check_lanes(g, B, ll, T, out);
  if (st != WD_OK) return st;
  if ((st = check_params(p)) != WD_OK) return st;
  int32_t max_T = 0;
  for (int b = 0; b < B; ++b) max_T = std::max(max_T, T[b]);
  if (!ws || ((uintptr_t)ws & 255u)) return fail(WD_EINVAL, "decode: workspace must be 256-byte aligned");
  wd_stream run;
  if ((st = run_setup(&run, g, B, ll, T, max_T, p, caps, ws, ws_bytes, stream, false)) ||
      (st = run_frames(&run, false))) {
    (void)hipStreamSynchronize(run.s);
    return st;
  }
  return run_finish(&run, out);
}

extern "C" wd_status wd_decode(const wd_graph* g, const float* loglikes, int32_t T, const wd_params* p,
                               const wd_caps* caps, void* ws, size_t ws_bytes, void* stream, wd_result** out) {
  return decode_impl(g, 1, &loglikes, &T, p, caps, ws, ws_bytes, stream, out);
}

extern "C" wd_status wd_decode_batch(const wd_graph* g, int32_t B, const float* const* loglikes, const int32_t* T,
                                     const wd_params* p, const wd_caps* caps, void* ws, size_t ws_bytes,
                                     void* stream, wd_result** out) {
  return decode_impl(g, B, loglikes, T, p, caps, ws, ws_bytes, stream, out);
}

extern "C" wd_status wd_stream_begin(const wd_graph* g, int32_t B, const float* const* frames, int32_t max_T,
                                     const wd_params* p, const wd_caps* caps, void* ws, size_t ws_bytes,
                                     void* stream, wd_stream** out) {
  if (!out) return fail(WD_EINVAL, "stream_begin: null output");
  *out = nullptr;
  if (!g || B < 1 || !frames || max_T < 0 || max_T > (1 << 24))
    return fail(WD_EINVAL, "stream_begin: bad arguments");
  for (int b = 0; b < B; ++b)
    if (max_T > 0 && !frames[b]) return fail(WD_EINVAL, "stream_begin: null frame store");
  wd_status st = check_params(p);
  if (st != WD_OK) return st;
  if (chip_wide_mode(p) && B != 1) return fail(WD_EINVAL, "stream_begin: chip-wide streams hold one utterance");
  if (!ws || ((uintptr_t)ws & 255u)) return fail(WD_EINVAL, "stream_begin: workspace must be 256-byte aligned");
  wd_stream* run = new wd_stream();
  std::vector<int32_t> zero((size_t)B, 0);
  if ((st = run_setup(run, g, B, frames, zero.data(), max_T, p, caps, ws, ws_bytes, stream, true))) {
    (void)hipStreamSynchronize((hipStream_t)stream);
    delete run;
    return st;
  }
  *out = run;
  return WD_OK;
}

extern "C" wd_status wd_stream_advance(wd_stream* run, const int32_t* n_frames) {
  if (!run || !n_frames) return fail(WD_EINVAL, "stream_advance: bad arguments");
  for (int b = 0; b < run->B; ++b)
    if (n_frames[b] < 0 || (int64_t)run->T[b] + n_frames[b] > run->max_T)
      return fail(WD_EINVAL, "stream_advance: frame count beyond max_T");
  for (int b = 0; b < run->B; ++b) run->T[b] += n_frames[b];
  return run_frames(run, true);
}

extern "C" wd_status wd_stream_end(wd_stream* run, wd_result** out) {
  if (!run || !out) return fail(WD_EINVAL, "stream_end: bad arguments");
  for (int b = 0; b < run->B; ++b) out[b] = nullptr;
  run->open = false;
  wd_status st = run_frames(run, true);
  if (st == WD_OK) st = run_finish(run, out);
  (void)hipStreamSynchronize(run->s);  // nothing of the stream's may run after it is freed
  delete run;
  return st;
}

extern "C" void wd_stream_free(wd_stream* run) {
  if (!run) return;
  (void)hipStreamSynchronize(run->s);
  delete run;
}

// ------------------------------------------------------ decode without allocation
//
// The workspace of wd_decode_noalloc: a fixed array in every device's memory
// (held from the library's first use on that device until the process ends).
// In host code `scratch` names a host-side stand-in, never the device
// memory; the device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[WD_NOALLOC_SCRATCH_BYTES];

static wd_status scratch_of_current_device(char** out) {
  static std::mutex mu;
  static char* per_dev[64] = {};
  int dev = 0;
  wd_status st = hip_check(hipGetDevice(&dev), "noalloc: device");
  if (st != WD_OK) return st;
  if (dev < 0 || dev >= 64) return fail(WD_EDEVICE, "noalloc: device index out of range");
  std::lock_guard<std::mutex> lk(mu);
  if (!per_dev[dev]) {
    void* ptr = nullptr;
    if ((st = hip_check(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)), "noalloc: scratch address"))) return st;
    if (!ptr || ((uintptr_t)ptr & 255u)) return fail(WD_EDEVICE, "noalloc: scratch misaligned");
    per_dev[dev] = (char*)ptr;
  }
  *out = per_dev[dev];
  return WD_OK;
}

extern "C" wd_status wd_decode_noalloc(const wd_graph* g, const float* loglikes, int32_t T, const wd_params* p,
                                       const wd_caps* caps, void* stream, float* cost, int32_t* words,
                                       int32_t words_cap, int32_t* n_words, wd_lat_arc* links, int64_t links_cap,
                                       wd_lat_node* nodes, int64_t nodes_cap, wd_stats* stats) {
  if (!g || T < 0 || T > (1 << 24) || (T > 0 && !loglikes) || !cost || !n_words || !stats ||
      words_cap < 0 || links_cap < 0 || nodes_cap < 0 || (words_cap && !words) || (links_cap && !links) ||
      (nodes_cap && !nodes))
    return fail(WD_EINVAL, "decode_noalloc: bad arguments");
  wd_status st = check_params(p);
  if (st != WD_OK) return st;
  const uint32_t allowed = WD_FLAG_ONE_WORKGROUP;
  if ((p->flags & ~allowed) || chip_wide_mode(p))
    return fail(WD_EINVAL, "decode_noalloc: one-workgroup decodes only, without debug, timing or profile flags "
                           "(set WD_FLAG_ONE_WORKGROUP when max_active is 0 or >= WD_CHIP_WIDE_MAX_ACTIVE)");
  *n_words = 0;
  *cost = 0.0f;
  std::memset(stats, 0, sizeof(*stats));
  const Caps c = resolve_caps(g, T, p, caps);
  const uint64_t need = carve(g, 1, T, c, nullptr, nullptr).total;
  if (need > (uint64_t)WD_NOALLOC_SCRATCH_BYTES)
    return fail(WD_EINVAL, "decode_noalloc: this decode needs a workspace of " + std::to_string(need) +
                               " bytes, more than the " + std::to_string((uint64_t)WD_NOALLOC_SCRATCH_BYTES) +
                               "-byte scratch (pass smaller capacities, or use wd_decode)");
  char* base = nullptr;
  if ((st = scratch_of_current_device(&base))) return st;
  hipStream_t s = (hipStream_t)stream;
  LaneDesc lane;
  std::memset(&lane, 0, sizeof(lane));
  const Regions R = carve(g, 1, T, c, base, &lane);
  lane.ll = (decltype(lane.ll))loglikes;
  lane.T = T;
  // the scratch keeps the last call's contents: every region a decode reads
  // before writing is reset here, as for a caller's workspace
  if ((st = hip_check(hipMemcpyAsync(R.desc, &lane, sizeof(LaneDesc), hipMemcpyHostToDevice, s), "lane upload")))
    return st;
  launch_fill_u32((uint32_t*)R.info, sizeof(LaneInfo) / 4, 0u, s);
  launch_fill_u32(R.bad, 1, 0u, s);
  launch_fill_u64(R.slot, (uint64_t)g->S, kEmpty, s);
  launch_fill_u32(R.bitmap, R.bitmap_words, 0u, s);
  launch_fill_u32(R.used, R.used_words, 0u, s);
  const Params prm{p->beam, p->max_active, p->lattice_beam, p->flags};
  launch_check_loglikes(R.desc, 1, g->P, R.bad, s);
  launch_forward(g->dg, R.desc, 1, prm, R.bad, s);
  launch_links(g->dg, R.desc, 1, s);
  launch_lattice(g->dg, R.desc, 1, prm, s);
  LaneInfo I;
  if ((st = hip_check(hipGetLastError(), "launch")) ||
      (st = hip_check(hipMemcpyAsync(&I, R.info, sizeof(LaneInfo), hipMemcpyDeviceToHost, s), "info download")) ||
      (st = hip_check(hipStreamSynchronize(s), "decode")))
    return st;
  const wd_status ls = (I.status == 0 && I.tb_fail) ? WD_EDEVICE : (wd_status)I.status;
  *stats = lane_stats(I, T, 0.0f, 0.0f, false);
  if (ls != WD_OK) return fail(ls, status_message(ls));
  *cost = I.best_cost;
  *n_words = (int32_t)I.nwords;
  if ((int64_t)I.nwords > words_cap || (int64_t)I.kept > links_cap || (int64_t)I.out_nodes > nodes_cap)
    return fail(WD_ECAPACITY, "decode_noalloc: output buffers too small (need " + std::to_string(I.nwords) +
                                  " words, " + std::to_string(I.kept) + " links, " + std::to_string(I.out_nodes) +
                                  " nodes; see n_words and stats)");
  auto d2h = [&](void* dst, const void* src, uint64_t bytes) -> wd_status {
    if (!bytes) return WD_OK;
    return hip_check(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, s), "result download");
  };
  if ((st = d2h(words, lane.out_words, 4 * I.nwords)) ||
      (st = d2h(links, lane.out_links, sizeof(OutLink) * I.kept)) ||
      (st = d2h(nodes, lane.out_nodes, sizeof(OutNode) * I.out_nodes)) ||
      (st = hip_check(hipStreamSynchronize(s), "result download")))
    return st;
  return WD_OK;
}

extern "C" wd_status wd_result_status(const wd_result* r) { return r->status; }
extern "C" float wd_result_cost(const wd_result* r) { return r->cost; }
extern "C" int32_t wd_result_words(const wd_result* r, const int32_t** w) {
  *w = r->words.data();
  return (int32_t)r->words.size();
}
extern "C" int64_t wd_result_lattice(const wd_result* r, const wd_lat_arc** a) {
  *a = r->links.data();
  return (int64_t)r->links.size();
}
extern "C" int64_t wd_result_nodes(const wd_result* r, const wd_lat_node** n) {
  *n = r->nodes.data();
  return (int64_t)r->nodes.size();
}
extern "C" int64_t wd_result_tokens(const wd_result* r, const wd_token** t) {
  *t = r->tokens.data();
  return (int64_t)r->tokens.size();
}
extern "C" int64_t wd_result_raw_lattice(const wd_result* r, const wd_lat_arc** a) {
  *a = r->raw.data();
  return (int64_t)r->raw.size();
}
extern "C" int32_t wd_result_cutoffs(const wd_result* r, const float** b, const float** cb, const float** c) {
  *b = r->best.data();
  *cb = r->cutb.data();
  *c = r->cut.data();
  return (int32_t)r->best.size();
}
extern "C" int32_t wd_result_phases(const wd_result* r, const uint64_t** stamps, double* tick_hz) {
  *stamps = r->prof.data();
  if (tick_hz) *tick_hz = r->tick_hz;
  const size_t rows = r->prof.size() / kProfSlots;
  return rows ? (int32_t)(rows - 1) : 0;
}
extern "C" int32_t wd_result_lattice_phases(const wd_result* r, const uint64_t** stamps) {
  const size_t rows = r->prof.size() / kProfSlots;
  *stamps = rows ? r->prof.data() + (rows - 1) * kProfSlots : nullptr;
  return rows ? (int32_t)kLatStamps : 0;
}
extern "C" void wd_result_stats(const wd_result* r, wd_stats* s) { *s = r->stats; }
extern "C" void wd_result_free(wd_result* r) { delete r; }
extern "C" const char* wd_last_error(void) { return g_err.c_str(); }
