// Lattice determinisation on the host: the compact "exact lattice" of the
// method (Sec. 3.4, after Povey et al. 2012), built from the pruned
// state-level lattice the decoder returns, on the CPU as the paper does.
//
// The input is an acceptor over words: a link with olabel 0 carries no word.
// Every path carries a weight, the pair (graph cost, acoustic cost), and a
// string, the input labels (pdf + 1) of its emitting links in frame order.
// The output is deterministic on words and has, for every word sequence of
// the input, exactly one path, whose total weight and string are those of
// the best input path with that word sequence.  "Best" is the order used
// throughout: lower total cost (graph + acoustic), then the lexicographically
// smaller string, then the lower graph cost.
//
// Weighted subset construction in the semiring of (weight, string) pairs:
// a state of the output is a set of (input node, residual weight, residual
// string), closed under the links that carry no word; the transition on word
// w follows the links with olabel w from every element, keeps the best
// element per input node, closes the set again and divides it by its common
// part, the best weight and the longest common prefix of the strings, which
// go onto the output arc.  The start set is not divided.  A set's final
// weight is the best of its elements' residuals extended by their nodes'
// final costs.  The input is acyclic (frames only grow, epsilon links climb
// levels inside a frame), so the construction ends; closures visit nodes in
// a topological order of the input, each node once.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <queue>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/wfstdec.h"

namespace wd {
wd_status fail(wd_status st, const std::string& msg);
}

struct wd_clat {
  int32_t states = 0;
  std::vector<wd_clat_arc> arcs;
  std::vector<wd_clat_final> finals;
  std::vector<int32_t> align;
};

namespace {

using Str = std::vector<int32_t>;

struct InArc {
  int32_t dst, word, ilabel;
  double g, a;
};

struct Input {
  int32_t n = 0, start = -1;
  std::vector<int64_t> off;     // CSR over nodes
  std::vector<InArc> arcs;
  std::vector<double> fin;      // final graph cost, +inf if not final
  std::vector<int32_t> rank;    // position in a topological order
};

struct Elem {
  int32_t node;
  double g, a;
  Str s;
};

bool better(double g1, double a1, const Str& s1, double g2, double a2, const Str& s2) {
  const double t1 = g1 + a1, t2 = g2 + a2;
  if (t1 != t2) return t1 < t2;
  if (s1 != s2) return s1 < s2;
  return g1 < g2;
}

bool better(const Elem& x, const Elem& y) { return better(x.g, x.a, x.s, y.g, y.a, y.s); }

// Best completion cost of every node (graph + acoustic + final), by the
// reverse of the topological order; +inf for a node that reaches no final.
std::vector<double> completion(const Input& in) {
  std::vector<int32_t> order((size_t)in.n);
  for (int32_t u = 0; u < in.n; ++u) order[(size_t)in.rank[u]] = u;
  std::vector<double> beta((size_t)in.n, INFINITY);
  for (int32_t h = in.n - 1; h >= 0; --h) {
    const int32_t u = order[(size_t)h];
    double b = in.fin[u];
    for (int64_t k = in.off[u]; k < in.off[u + 1]; ++k) {
      const InArc& a = in.arcs[k];
      const double c = a.g + a.a + beta[a.dst];
      b = c < b ? c : b;
    }
    beta[u] = b;
  }
  return beta;
}

// Closure of `m` (input node -> element) under the links without a word.
// With a finite `limit`, an element whose residual plus its node's best
// completion exceeds it is neither added nor followed (no path through it
// is within the beam).
void closure(const Input& in, std::unordered_map<int32_t, Elem>& m, const std::vector<double>& beta,
             double limit) {
  using Item = std::pair<int32_t, int32_t>;  // (rank, node)
  std::priority_queue<Item, std::vector<Item>, std::greater<Item>> q;
  for (auto& kv : m) q.push({in.rank[kv.first], kv.first});
  int32_t last = -1;
  while (!q.empty()) {
    const int32_t u = q.top().second;
    q.pop();
    if (u == last) continue;  // queued more than once
    last = u;
    const Elem e = m.at(u);
    for (int64_t k = in.off[u]; k < in.off[u + 1]; ++k) {
      const InArc& r = in.arcs[k];
      if (r.word != 0) continue;
      if (e.g + r.g + e.a + r.a + beta[r.dst] > limit) continue;
      Elem c{r.dst, e.g + r.g, e.a + r.a, e.s};
      if (r.ilabel != 0) c.s.push_back(r.ilabel);
      auto it = m.find(r.dst);
      if (it == m.end()) {
        m.emplace(r.dst, std::move(c));
        q.push({in.rank[r.dst], r.dst});
      } else if (better(c, it->second)) {
        it->second = std::move(c);
      }
    }
  }
}

std::vector<Elem> sorted(std::unordered_map<int32_t, Elem>& m) {
  std::vector<Elem> v;
  v.reserve(m.size());
  for (auto& kv : m) v.push_back(std::move(kv.second));
  std::sort(v.begin(), v.end(), [](const Elem& x, const Elem& y) { return x.node < y.node; });
  return v;
}

struct KeyHash {
  size_t operator()(const std::vector<int64_t>& k) const {
    uint64_t h = 1469598103934665603ull;
    for (int64_t x : k) {
      h ^= (uint64_t)x;
      h *= 1099511628211ull;
    }
    return (size_t)h;
  }
};

std::vector<int64_t> key_of(const std::vector<Elem>& v) {
  std::vector<int64_t> k;
  for (const Elem& e : v) {
    int64_t gb, ab;
    std::memcpy(&gb, &e.g, 8);
    std::memcpy(&ab, &e.a, 8);
    k.push_back(e.node);
    k.push_back(gb);
    k.push_back(ab);
    k.push_back((int64_t)e.s.size());
    k.insert(k.end(), e.s.begin(), e.s.end());
  }
  return k;
}

wd_status build_input(const wd_lat_arc* arcs, int64_t n_arcs, const wd_lat_node* nodes, int64_t n_nodes,
                      int32_t start_state, const float* node_final, Input* in) {
  if (n_nodes > INT32_MAX - 1) return wd::fail(WD_EINVAL, "determinize: too many nodes");
  in->n = (int32_t)n_nodes;
  auto key = [](int32_t t, int32_t s) { return ((int64_t)t << 32) | (uint32_t)s; };
  std::vector<int64_t> nk((size_t)n_nodes);
  int32_t t_last = 0;
  for (int64_t i = 0; i < n_nodes; ++i) {
    nk[i] = key(nodes[i].t, nodes[i].state);
    if (i > 0 && nk[i] <= nk[i - 1]) return wd::fail(WD_EINVAL, "determinize: nodes not sorted by (t, state)");
    t_last = std::max(t_last, nodes[i].t);
  }
  auto find = [&](int32_t t, int32_t s) -> int32_t {
    auto it = std::lower_bound(nk.begin(), nk.end(), key(t, s));
    return (it != nk.end() && *it == key(t, s)) ? (int32_t)(it - nk.begin()) : -1;
  };
  in->start = n_nodes ? find(0, start_state) : -1;
  if (n_nodes && in->start < 0) return wd::fail(WD_EINVAL, "determinize: no node for the start state at t = 0");
  std::vector<int32_t> src((size_t)n_arcs), dst((size_t)n_arcs);
  std::vector<int64_t> deg((size_t)n_nodes + 1, 0);
  for (int64_t k = 0; k < n_arcs; ++k) {
    const wd_lat_arc& l = arcs[k];
    src[k] = find(l.ilabel != 0 ? l.t - 1 : l.t, l.src_state);
    dst[k] = find(l.t, l.dst_state);
    if (src[k] < 0 || dst[k] < 0) return wd::fail(WD_EINVAL, "determinize: a link's endpoint is not a node");
    if (l.olabel < 0 || l.ilabel < 0) return wd::fail(WD_EINVAL, "determinize: negative label");
    ++deg[src[k] + 1];
  }
  in->off.assign((size_t)n_nodes + 1, 0);
  for (int64_t i = 0; i < n_nodes; ++i) in->off[i + 1] = in->off[i] + deg[i + 1];
  in->arcs.resize((size_t)n_arcs);
  std::vector<int64_t> pos(in->off.begin(), in->off.end() - (n_nodes ? 1 : 0));
  std::vector<int32_t> indeg((size_t)n_nodes, 0);
  for (int64_t k = 0; k < n_arcs; ++k) {
    const wd_lat_arc& l = arcs[k];
    in->arcs[pos[src[k]]++] = InArc{dst[k], l.olabel, l.ilabel, (double)l.graph_cost, (double)l.ac_cost};
    ++indeg[dst[k]];
  }
  in->fin.assign((size_t)n_nodes, INFINITY);
  for (int64_t i = 0; i < n_nodes; ++i) {
    if (node_final) in->fin[i] = node_final[i];
    else if (nodes[i].t == t_last) in->fin[i] = 0.0;
  }
  // topological order (Kahn); a cycle is an error
  in->rank.assign((size_t)n_nodes, -1);
  std::vector<int32_t> q;
  for (int32_t i = 0; i < (int32_t)n_nodes; ++i)
    if (!indeg[i]) q.push_back(i);
  for (size_t h = 0; h < q.size(); ++h) {
    const int32_t u = q[h];
    in->rank[u] = (int32_t)h;
    for (int64_t k = in->off[u]; k < in->off[u + 1]; ++k)
      if (--indeg[in->arcs[k].dst] == 0) q.push_back(in->arcs[k].dst);
  }
  if ((int64_t)q.size() != n_nodes) return wd::fail(WD_EINVAL, "determinize: the lattice has a cycle");
  return WD_OK;
}

double best_rest(const std::vector<Elem>& S, const std::vector<double>& beta) {
  double m = INFINITY;
  for (const Elem& e : S) {
    const double c = e.g + e.a + beta[e.node];
    m = c < m ? c : m;
  }
  return m;
}

}  // namespace

extern "C" wd_status wd_lattice_determinize(const wd_lat_arc* arcs, int64_t n_arcs, const wd_lat_node* nodes,
                                            int64_t n_nodes, int32_t start_state, const float* node_final,
                                            double beam, int64_t max_states, wd_clat** out) {
  if (!out || n_arcs < 0 || n_nodes < 0 || (n_arcs && !arcs) || (n_nodes && !nodes) || !(beam >= 0.0))
    return wd::fail(WD_EINVAL, "determinize: bad arguments");
  *out = nullptr;
  Input in;
  wd_status st = build_input(arcs, n_arcs, nodes, n_nodes, start_state, node_final, &in);
  if (st != WD_OK) return st;
  wd_clat* r = new wd_clat();
  if (!in.n) {
    *out = r;
    return WD_OK;
  }
  if (max_states <= 0) max_states = 1 << 22;
  const std::vector<double> beta = completion(in);
  // Output states are expanded in the order of (forward cost of the best
  // output path reaching them + best completion of their elements): the
  // completion cost is exact, so this order never decreases along an arc
  // and a state's forward cost is final when it is expanded.  With a finite
  // beam, word links and closure elements whose best complete path costs
  // more than the best path plus `beam` are left out, so no state beyond
  // the beam is created and subsets hold only nodes within it; the paths
  // within the beam are all still there, each with its own best weight.
  std::unordered_map<std::vector<int64_t>, int32_t, KeyHash> ids;
  std::vector<std::vector<Elem>> todo;  // subsets by state id, freed once expanded
  std::vector<double> fwd;              // forward cost (graph + acoustic) of each state
  using Item = std::pair<double, int32_t>;
  std::priority_queue<Item, std::vector<Item>, std::greater<Item>> heap;
  double cutoff;
  {
    std::unordered_map<int32_t, Elem> m;
    m.emplace(in.start, Elem{in.start, 0.0, 0.0, {}});
    const double f0 = beta[in.start];
    cutoff = f0 + beam;
    closure(in, m, beta, cutoff);
    todo.push_back(sorted(m));
    ids.emplace(key_of(todo[0]), 0);
    fwd.push_back(0.0);
    heap.push({f0, 0});
  }
  std::vector<char> done(1, 0);
  while (!heap.empty()) {
    const int32_t id = heap.top().second;
    heap.pop();
    if (done[(size_t)id]) continue;
    done[(size_t)id] = 1;
    const std::vector<Elem> S = std::move(todo[id]);
    todo[id].clear();
    todo[id].shrink_to_fit();
    // final weight
    const Elem* bf = nullptr;
    Elem fe{};
    for (const Elem& e : S) {
      if (!std::isfinite(in.fin[e.node])) continue;
      Elem c{e.node, e.g + in.fin[e.node], e.a, e.s};
      if (!bf || better(c, fe)) {
        fe = std::move(c);
        bf = &fe;
      }
    }
    if (bf) {
      r->finals.push_back(wd_clat_final{id, (int32_t)fe.s.size(), fe.g, fe.a, (int64_t)r->align.size()});
      r->align.insert(r->align.end(), fe.s.begin(), fe.s.end());
    }
    // the word links leaving the set, by word (then element and link order);
    // links that cannot be within the beam are left out
    const double limit = cutoff - fwd[(size_t)id];
    std::vector<std::pair<int32_t, std::pair<uint32_t, int64_t>>> out_links;  // (word, (elem, link))
    for (uint32_t ei = 0; ei < (uint32_t)S.size(); ++ei) {
      const Elem& e = S[ei];
      for (int64_t k = in.off[e.node]; k < in.off[e.node + 1]; ++k) {
        const InArc& a = in.arcs[k];
        if (a.word != 0 && !(e.g + a.g + e.a + a.a + beta[a.dst] > limit)) out_links.push_back({a.word, {ei, k}});
      }
    }
    std::sort(out_links.begin(), out_links.end());
    for (size_t q0 = 0; q0 < out_links.size();) {
      const int32_t w = out_links[q0].first;
      size_t q1 = q0;
      while (q1 < out_links.size() && out_links[q1].first == w) ++q1;
      std::unordered_map<int32_t, Elem> m;
      for (size_t q = q0; q < q1; ++q) {
        const Elem& e = S[out_links[q].second.first];
        const InArc& a = in.arcs[out_links[q].second.second];
        Elem c{a.dst, e.g + a.g, e.a + a.a, e.s};
        if (a.ilabel != 0) c.s.push_back(a.ilabel);
        auto it = m.find(a.dst);
        if (it == m.end()) m.emplace(a.dst, std::move(c));
        else if (better(c, it->second)) it->second = std::move(c);
      }
      q0 = q1;
      closure(in, m, beta, limit);
      std::vector<Elem> T = sorted(m);
      // divide by the common part: best weight, longest common string prefix
      const Elem* b = &T[0];
      for (const Elem& e : T)
        if (better(e, *b)) b = &e;
      const double g0 = b->g, a0 = b->a;
      size_t pre = T[0].s.size();
      for (const Elem& e : T) {
        size_t i = 0;
        while (i < pre && i < e.s.size() && e.s[i] == T[0].s[i]) ++i;
        pre = i;
      }
      const Str common(T[0].s.begin(), T[0].s.begin() + (std::ptrdiff_t)pre);
      for (Elem& e : T) {
        e.g -= g0;
        e.a -= a0;
        e.s.erase(e.s.begin(), e.s.begin() + (std::ptrdiff_t)pre);
      }
      const double fT = fwd[(size_t)id] + (g0 + a0);
      const double f = fT + best_rest(T, beta);
      std::vector<int64_t> k = key_of(T);
      auto it = ids.find(k);
      int32_t to;
      if (it != ids.end()) {
        to = it->second;
        if (!done[(size_t)to] && fT < fwd[(size_t)to]) {
          fwd[(size_t)to] = fT;
          heap.push({f, to});
        }
      } else {
        if ((int64_t)todo.size() >= max_states) {
          delete r;
          return wd::fail(WD_ECAPACITY, "determinize: more output states than max_states");
        }
        to = (int32_t)todo.size();
        ids.emplace(std::move(k), to);
        todo.push_back(std::move(T));
        fwd.push_back(fT);
        done.push_back(0);
        heap.push({f, to});
      }
      r->arcs.push_back(wd_clat_arc{id, to, w, (int32_t)common.size(), g0, a0, (int64_t)r->align.size()});
      r->align.insert(r->align.end(), common.begin(), common.end());
    }
  }
  r->states = (int32_t)todo.size();
  std::sort(r->arcs.begin(), r->arcs.end(), [](const wd_clat_arc& x, const wd_clat_arc& y) {
    return x.src != y.src ? x.src < y.src : x.word < y.word;
  });
  std::sort(r->finals.begin(), r->finals.end(),
            [](const wd_clat_final& x, const wd_clat_final& y) { return x.state < y.state; });
  *out = r;
  return WD_OK;
}

extern "C" int32_t wd_clat_states(const wd_clat* c) { return c->states; }
extern "C" int64_t wd_clat_arcs(const wd_clat* c, const wd_clat_arc** arcs) {
  *arcs = c->arcs.data();
  return (int64_t)c->arcs.size();
}
extern "C" int64_t wd_clat_finals(const wd_clat* c, const wd_clat_final** finals) {
  *finals = c->finals.data();
  return (int64_t)c->finals.size();
}
extern "C" int64_t wd_clat_alignment(const wd_clat* c, const int32_t** labels) {
  *labels = c->align.data();
  return (int64_t)c->align.size();
}
extern "C" void wd_clat_free(wd_clat* c) { delete c; }
