// Graph loading: validation, epsilon levels, and the device layout.
//
// The graph stays resident in GPU memory for every decode (the paper decodes
// graphs held entirely in GPU memory, Sec. 4.3).  Emitting and epsilon arcs are
// split into two CSRs of 16-byte records so the emitting expansion reads only
// the arcs it uses, each with one 16-byte load.  Epsilon levels (longest
// epsilon path into a state) order the epsilon closure: an epsilon arc always
// climbs to a higher level.  Beside each epsilon arc sits its destination's
// epsilon arc range, so a closure step that reaches a state with epsilon arcs
// needs no second, dependent read of the offsets.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "wd_host.h"

namespace wd {

namespace {

struct Prepared {
  std::vector<uint4> off;
  std::vector<uint4> earc, xarc;
  std::vector<uint2> xnext;
  std::vector<uint8_t> sclass;
  std::vector<uint32_t> level_base;
  uint32_t nlevels = 0;
  bool paths = false;            // epsilon path table (its first path per state in off[s].z)
  std::vector<uint4> phead;
  std::vector<float> ptail;
  uint32_t pstride = 0;
};

struct Layout {
  uint64_t off, earc, xarc, xnext, sclass, final_w, ilabel, olabel, weight, level_base, phead, ptail, total;
};

Layout layout(int64_t S, int64_t A, uint64_t Ae, uint64_t Ax, uint32_t nlevels, bool finals, uint64_t npaths,
              uint32_t pstride) {
  Layout l{};
  uint64_t p = 0;
  auto take = [&](uint64_t bytes) {
    uint64_t at = p;
    p = align_up(p + bytes, 256);
    return at;
  };
  l.off = take(sizeof(uint4) * (uint64_t)(S + 1));
  l.earc = take(sizeof(uint4) * (Ae ? Ae : 1));
  l.xarc = take(sizeof(uint4) * (Ax ? Ax : 1));
  l.xnext = take(sizeof(uint2) * (Ax ? Ax : 1));
  l.sclass = take((uint64_t)S);
  l.final_w = finals ? take(sizeof(float) * (uint64_t)S) : 0;
  l.ilabel = take(sizeof(int32_t) * (uint64_t)(A ? A : 1));
  l.olabel = take(sizeof(int32_t) * (uint64_t)(A ? A : 1));
  l.weight = take(sizeof(float) * (uint64_t)(A ? A : 1));
  l.level_base = take(sizeof(uint32_t) * (uint64_t)(nlevels + 1));
  l.phead = npaths ? take(sizeof(uint4) * 2 * npaths) : 0;
  l.ptail = npaths && pstride ? take(sizeof(float) * npaths * pstride) : 0;
  l.total = p;
  return l;
}

wd_status validate(const wd_graph_desc* d) {
  if (!d) return fail(WD_EINVAL, "graph: null descriptor");
  const int64_t S = d->num_states, A = d->num_arcs;
  if (S < 1) return fail(WD_EINVAL, "graph: num_states must be >= 1");
  if (A < 0 || A >= (int64_t)0xffffffffu) return fail(WD_EINVAL, "graph: num_arcs out of range");
  if (d->start_state < 0 || d->start_state >= S) return fail(WD_EINVAL, "graph: start_state out of range");
  if (d->num_pdfs < 1 || d->num_pdfs >= (1 << 24)) return fail(WD_EINVAL, "graph: num_pdfs out of range");
  if (!d->row_ptr) return fail(WD_EINVAL, "graph: null row_ptr");
  if (A > 0 && (!d->dst || !d->ilabel || !d->olabel || !d->weight))
    return fail(WD_EINVAL, "graph: null arc array");
  if (d->row_ptr[0] != 0 || (int64_t)d->row_ptr[S] != A)
    return fail(WD_EINVAL, "graph: row_ptr must start at 0 and end at num_arcs");
  for (int64_t s = 0; s < S; ++s)
    if (d->row_ptr[s] > d->row_ptr[s + 1]) return fail(WD_EINVAL, "graph: row_ptr decreases");
  for (int64_t a = 0; a < A; ++a) {
    if ((int64_t)d->dst[a] >= S) return fail(WD_EINVAL, "graph: dst out of range at arc " + std::to_string(a));
    if (d->ilabel[a] < 0 || d->ilabel[a] > d->num_pdfs)
      return fail(WD_EINVAL, "graph: ilabel out of range at arc " + std::to_string(a));
    if (d->olabel[a] < 0) return fail(WD_EINVAL, "graph: negative olabel at arc " + std::to_string(a));
    const float w = d->weight[a];
    if (!(w >= 0.0f) || std::isinf(w))
      return fail(WD_EINVAL, "graph: weight must be finite and >= 0 at arc " + std::to_string(a));
  }
  if (d->final_weight)
    for (int64_t s = 0; s < S; ++s)
      if (!(d->final_weight[s] >= 0.0f)) return fail(WD_EINVAL, "graph: final weight must be >= 0 or +inf");
  return WD_OK;
}

// Longest epsilon path into every state, by Kahn's order over epsilon arcs;
// WD_ECYCLE when some state is never freed.
wd_status eps_levels(const wd_graph_desc* d, std::vector<uint32_t>& level, std::vector<uint32_t>& queue) {
  const int64_t S = d->num_states;
  std::vector<uint32_t> indeg((size_t)S, 0);
  for (int64_t a = 0; a < d->num_arcs; ++a)
    if (d->ilabel[a] == 0) indeg[d->dst[a]]++;
  queue.clear();
  queue.reserve((size_t)S);
  level.assign((size_t)S, 0);
  for (int64_t s = 0; s < S; ++s)
    if (!indeg[s]) queue.push_back((uint32_t)s);
  for (size_t h = 0; h < queue.size(); ++h) {
    const uint32_t s = queue[h];
    for (uint32_t a = d->row_ptr[s]; a < d->row_ptr[s + 1]; ++a) {
      if (d->ilabel[a] != 0) continue;
      const uint32_t v = d->dst[a];
      if (level[v] < level[s] + 1) level[v] = level[s] + 1;
      if (--indeg[v] == 0) queue.push_back(v);
    }
  }
  if ((int64_t)queue.size() != S) return fail(WD_ECYCLE, "graph: epsilon arcs contain a cycle");
  return WD_OK;
}

// Every epsilon path out of every state (the closure's alternative to one
// pass per level: a token's epsilon paths are relaxed all at once, each
// path's weights added in path order).  Left empty when the graph has more
// than kPathMax paths or one longer than kPathMaxLen arcs.  Per state the
// paths are listed depth first, arcs in the caller's order.
void eps_paths(const wd_graph_desc* d, const std::vector<uint32_t>& topo, Prepared& p) {
  const int64_t S = d->num_states;
  std::vector<uint64_t> npath((size_t)S, 0);
  std::vector<uint32_t> maxlen((size_t)S, 0), xdeg((size_t)S, 0);
  uint64_t total = 0;
  uint32_t longest = 0;
  // destinations before sources: the reverse of a topological order
  for (size_t h = topo.size(); h-- > 0;) {
    const uint32_t s = topo[h];
    uint64_t n = 0;
    uint32_t len = 0;
    for (uint32_t a = d->row_ptr[s]; a < d->row_ptr[s + 1]; ++a) {
      if (d->ilabel[a] != 0) continue;
      const uint32_t v = d->dst[a];
      xdeg[s]++;
      n += 1 + npath[v];
      if (n > kPathMax) n = kPathMax + 1;  // (saturates: the table will not be built)
      len = std::max(len, 1 + maxlen[v]);
    }
    npath[s] = n;
    maxlen[s] = len;
    total = std::min<uint64_t>(total + n, kPathMax + 1);
    longest = std::max(longest, len);
  }
  if (total == 0 || total > kPathMax || longest > kPathMaxLen) return;
  for (int64_t s = 0; s < S; ++s)
    if (xdeg[s] >= (1u << 24)) return;
  p.pstride = longest - 1;
  p.paths = true;
  for (int64_t s = 0; s < S; ++s) p.off[s + 1].z = p.off[s].z + (uint32_t)npath[s];
  p.phead.assign(2 * total, make_uint4(0, 0, 0, 0));
  p.ptail.assign(total * p.pstride, 0.0f);
  // depth-first walk of the epsilon arcs out of s: stack of (state, next arc)
  std::vector<std::pair<uint32_t, uint32_t>> stack;
  std::vector<float> wpath;  // weights of the current path's arcs
  for (int64_t s = 0; s < S; ++s) {
    if (!npath[s]) continue;
    uint64_t at = p.off[s].z;
    stack.assign(1, {(uint32_t)s, d->row_ptr[s]});
    wpath.clear();
    while (!stack.empty()) {
      auto& top = stack.back();
      const uint32_t u = top.first;
      uint32_t a = top.second;
      while (a < d->row_ptr[u + 1] && d->ilabel[a] != 0) ++a;
      if (a >= d->row_ptr[u + 1]) {
        stack.pop_back();
        if (!wpath.empty()) wpath.pop_back();
        continue;
      }
      top.second = a + 1;
      const uint32_t v = d->dst[a];
      const uint32_t k = (uint32_t)wpath.size() + 1;
      uint32_t wbits;
      std::memcpy(&wbits, &d->weight[a], 4);
      p.phead[2 * at] = make_uint4(v, a, wbits, k | (xdeg[v] << 8));
      uint32_t tw[4] = {0, 0, 0, 0};  // the first tail weights, beside the head
      for (uint32_t i = 0; i + 1 < k && i < 4; ++i) std::memcpy(&tw[i], &wpath[i], 4);
      p.phead[2 * at + 1] = make_uint4(tw[0], tw[1], tw[2], tw[3]);
      for (uint32_t i = 0; i + 1 < k; ++i) p.ptail[at * p.pstride + i] = wpath[i];
      ++at;
      if (xdeg[v]) {
        wpath.push_back(d->weight[a]);
        stack.push_back({v, d->row_ptr[v]});
      }
    }
  }
}

wd_status prepare(const wd_graph_desc* d, Prepared& p, uint64_t* Ae_out, uint64_t* Ax_out) {
  wd_status st = validate(d);
  if (st != WD_OK) return st;
  const int64_t S = d->num_states, A = d->num_arcs;
  std::vector<uint32_t> level, topo;
  st = eps_levels(d, level, topo);
  if (st != WD_OK) return st;
  p.sclass.assign((size_t)S, (uint8_t)kNoEps);
  std::vector<uint32_t> count(kMaxLevels + 1, 0);
  uint32_t maxcls = 0;
  bool any_eps = false;
  uint64_t Ae = 0, Ax = 0;
  p.off.resize((size_t)S + 1);
  for (int64_t s = 0; s < S; ++s) {
    p.off[s] = make_uint4((uint32_t)Ae, (uint32_t)Ax, 0, 0);
    uint32_t ne = 0, nx = 0;
    for (uint32_t a = d->row_ptr[s]; a < d->row_ptr[s + 1]; ++a) (d->ilabel[a] ? ne : nx)++;
    Ae += ne;
    Ax += nx;
    if (nx) {
      if (level[s] >= (uint32_t)kMaxLevels)
        return fail(WD_EINVAL, "graph: epsilon chains deeper than " + std::to_string(kMaxLevels));
      p.sclass[s] = (uint8_t)level[s];
      count[level[s]]++;
      maxcls = level[s] > maxcls ? level[s] : maxcls;
      any_eps = true;
    }
  }
  p.off[S] = make_uint4((uint32_t)Ae, (uint32_t)Ax, 0, 0);
  p.nlevels = any_eps ? maxcls + 1 : 0;
  p.level_base.assign(p.nlevels + 1, 0);
  for (uint32_t l = 0; l < p.nlevels; ++l) p.level_base[l + 1] = p.level_base[l] + count[l];
  p.earc.resize(Ae);
  p.xarc.resize(Ax);
  uint64_t ie = 0, ix = 0;
  for (int64_t s = 0; s < S; ++s)
    for (uint32_t a = d->row_ptr[s]; a < d->row_ptr[s + 1]; ++a) {
      const uint32_t v = d->dst[a];
      uint32_t wbits;
      std::memcpy(&wbits, &d->weight[a], 4);
      if (d->ilabel[a])
        p.earc[ie++] = make_uint4(v, wbits, (uint32_t)d->ilabel[a] | ((uint32_t)p.sclass[v] << 24), a);
      else
        p.xarc[ix++] = make_uint4(v, wbits, p.sclass[v], a);
    }
  p.xnext.resize(Ax);
  for (uint64_t j = 0; j < Ax; ++j) {
    const uint32_t v = p.xarc[j].x;
    p.xnext[j] = make_uint2(p.off[v].y, p.off[v + 1].y);
  }
  eps_paths(d, topo, p);
  (void)A;
  *Ae_out = Ae;
  *Ax_out = Ax;
  return WD_OK;
}

}  // namespace

}  // namespace wd

using namespace wd;

extern "C" wd_status wd_graph_bytes(const wd_graph_desc* d, size_t* bytes) {
  if (!bytes) return fail(WD_EINVAL, "graph_bytes: null output");
  Prepared p;
  uint64_t Ae, Ax;
  wd_status st = prepare(d, p, &Ae, &Ax);
  if (st != WD_OK) return st;
  *bytes = layout(d->num_states, d->num_arcs, Ae, Ax, p.nlevels, d->final_weight != nullptr, p.phead.size() / 2,
                  p.pstride).total;
  return WD_OK;
}

extern "C" wd_status wd_graph_load(const wd_graph_desc* d, void* dev_buf, size_t dev_bytes, void* stream,
                                   wd_graph** out) {
  if (!out) return fail(WD_EINVAL, "graph_load: null output");
  *out = nullptr;
  if (!dev_buf || ((uintptr_t)dev_buf & 255u)) return fail(WD_EINVAL, "graph_load: dev_buf must be 256-byte aligned");
  Prepared p;
  uint64_t Ae, Ax;
  wd_status st = prepare(d, p, &Ae, &Ax);
  if (st != WD_OK) return st;
  const int64_t S = d->num_states, A = d->num_arcs;
  const bool finals = d->final_weight != nullptr;
  const uint64_t npaths = p.phead.size() / 2;
  const Layout l = layout(S, A, Ae, Ax, p.nlevels, finals, npaths, p.pstride);
  if (dev_bytes < l.total) return fail(WD_EINVAL, "graph_load: dev_buf smaller than wd_graph_bytes");
  hipStream_t s = (hipStream_t)stream;
  char* base = (char*)dev_buf;
  auto put = [&](uint64_t at, const void* src, uint64_t bytes) -> wd_status {
    if (!bytes) return WD_OK;
    return hip_check(hipMemcpyAsync(base + at, src, bytes, hipMemcpyHostToDevice, s), "graph upload");
  };
  if ((st = put(l.off, p.off.data(), sizeof(uint4) * (S + 1))) ||
      (st = put(l.earc, p.earc.data(), sizeof(uint4) * Ae)) ||
      (st = put(l.xarc, p.xarc.data(), sizeof(uint4) * Ax)) ||
      (st = put(l.xnext, p.xnext.data(), sizeof(uint2) * Ax)) ||
      (st = put(l.sclass, p.sclass.data(), (uint64_t)S)) ||
      (finals && (st = put(l.final_w, d->final_weight, sizeof(float) * S))) ||
      (st = put(l.ilabel, d->ilabel, sizeof(int32_t) * A)) ||
      (st = put(l.olabel, d->olabel, sizeof(int32_t) * A)) ||
      (st = put(l.weight, d->weight, sizeof(float) * A)) ||
      (st = put(l.level_base, p.level_base.data(), sizeof(uint32_t) * (p.nlevels + 1))) ||
      (npaths && (st = put(l.phead, p.phead.data(), sizeof(uint4) * 2 * npaths))) ||
      (npaths && p.pstride && (st = put(l.ptail, p.ptail.data(), sizeof(float) * npaths * p.pstride))))
    return st;
  if ((st = hip_check(hipStreamSynchronize(s), "graph upload sync"))) return st;
  wd_graph* g = new wd_graph();
  g->S = (int32_t)S;
  g->A = A;
  g->Ae = Ae;
  g->Ax = Ax;
  g->nlevels = p.nlevels;
  g->P = (uint32_t)d->num_pdfs;
  g->level_base = p.level_base;
  g->bytes = l.total;
  DevGraph& dg = g->dg;
  dg.off = (const uint4*)(base + l.off);
  dg.earc = (const uint4*)(base + l.earc);
  dg.xarc = (const uint4*)(base + l.xarc);
  dg.xnext = (const uint2*)(base + l.xnext);
  dg.sclass = (const uint8_t*)(base + l.sclass);
  dg.final_w = finals ? (const float*)(base + l.final_w) : nullptr;
  dg.ilabel_id = (const int32_t*)(base + l.ilabel);
  dg.olabel_id = (const int32_t*)(base + l.olabel);
  dg.weight_id = (const float*)(base + l.weight);
  dg.level_base = (const uint32_t*)(base + l.level_base);
  dg.phead = npaths ? (const uint4*)(base + l.phead) : nullptr;
  dg.ptail = npaths && p.pstride ? (const float*)(base + l.ptail) : nullptr;
  dg.npaths = npaths;
  dg.pstride = p.pstride;
  dg.S = (uint32_t)S;
  dg.start = (uint32_t)d->start_state;
  dg.nlevels = p.nlevels;
  dg.P = (uint32_t)d->num_pdfs;
  dg.Ae = Ae;
  dg.Ax = Ax;
  dg.A = (uint64_t)A;
  *out = g;
  return WD_OK;
}

extern "C" void wd_graph_free(wd_graph* g) { delete g; }

extern "C" int32_t wd_graph_eps_levels(const wd_graph* g) { return g ? (int32_t)g->nlevels : 0; }

extern "C" int64_t wd_graph_eps_paths(const wd_graph* g) { return g ? (int64_t)g->dg.npaths : 0; }
