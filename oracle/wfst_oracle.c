/*
 * CPU oracle: frame-synchronous Viterbi token passing over a WFST with exact
 * lattice generation, lattice pruning and fp64 arc posteriors.
 *
 * TEST INFRASTRUCTURE ONLY (see wfst_oracle.h).  Plain, sequential and slow on
 * purpose; every step follows the paper in its own order:
 *   - token passing and recombination: Sec. 3.2 (each state holds one token per
 *     frame; recombination keeps the minimum over incoming arcs together with
 *     the winning arc; Alg. 1 orders candidates by (cost, arc id));
 *   - lattice generation: Sec. 3.4 (one lattice link per token-passing
 *     operation that survives);
 *   - lattice pruning: Sec. 3.5 (extra costs of nodes and links updated until
 *     they stop changing; links whose extra cost exceeds the lattice beam are
 *     dropped; nodes are implied by the remaining links);
 *   - posteriors: Sec. 4.1 uses lattice arc posteriors for confidence.
 * Where the paper is silent (epsilon closure, beam and max-active cutoffs,
 * tie-breaks, fp32 summation order, final states) the readings are:
 *   emitting candidate x = fl(fl(c + ac) + w), ac = -loglike[t-1][ilabel-1];
 *   epsilon candidate   x = fl(c + w);
 *   candidates compare by (x, arc id), lowest arc id wins a cost tie;
 *   beam cutoff = fl(best emitting candidate + beam), inclusive;
 *   epsilon closure after the emitting step, bounded by the beam cutoff;
 *   max-active cutoff = the max_active-th smallest cost after the closure
 *   (ties kept); final cutoff = min of the two;
 *   lattice links = candidates from surviving sources whose x is within the
 *   final cutoff; -0.0 costs are stored as +0.0.
 */
#include "wfst_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define NONE 0xffffffffu

/* ---------------------------------------------------------------- utils -- */

static int grow(void** p, int64_t* cap, int64_t need, size_t elem) {
  if (need <= *cap) return 0;
  int64_t nc = *cap ? *cap : 1024;
  while (nc < need) nc *= 2;
  void* q = realloc(*p, (size_t)nc * elem);
  if (!q) return -1;
  *p = q;
  *cap = nc;
  return 0;
}

/* -0.0 and +0.0 are the same cost; store the latter. */
static float canon(float x) { return x == 0.0f ? 0.0f : x; }

/* Alg. 1 orders candidates by cost first and arc id second. */
static int better(float x, uint32_t a, float y, uint32_t b) {
  return x < y || (x == y && a < b);
}

static int cmp_float(const void* a, const void* b) {
  float x = *(const float*)a, y = *(const float*)b;
  return (x > y) - (x < y);
}

static int cmp_u32(const void* a, const void* b) {
  uint32_t x = *(const uint32_t*)a, y = *(const uint32_t*)b;
  return (x > y) - (x < y);
}

/* --------------------------------------------------------------- result -- */

struct wdo_result {
  float cost;
  int32_t* words;
  int32_t nwords;
  wdo_link* links;
  int64_t nlinks;
  wdo_node* nodes;
  int64_t nnodes;
  wdo_stats stats;
  wdo_token* toks;
  int64_t ntoks;
  wdo_link* raw;
  int64_t nraw;
  float* best;
  float* cutb;
  float* cut;
  int32_t ncut;
};

void wdo_result_free(wdo_result* r) {
  if (!r) return;
  free(r->words);
  free(r->links);
  free(r->nodes);
  free(r->toks);
  free(r->raw);
  free(r->best);
  free(r->cutb);
  free(r->cut);
  free(r);
}

float wdo_result_cost(const wdo_result* r) { return r->cost; }
int32_t wdo_result_words(const wdo_result* r, const int32_t** w) { *w = r->words; return r->nwords; }
int64_t wdo_result_links(const wdo_result* r, const wdo_link** l) { *l = r->links; return r->nlinks; }
int64_t wdo_result_nodes(const wdo_result* r, const wdo_node** n) { *n = r->nodes; return r->nnodes; }
void wdo_result_stats(const wdo_result* r, wdo_stats* s) { *s = r->stats; }
int64_t wdo_result_tokens(const wdo_result* r, const wdo_token** t) { *t = r->toks; return r->ntoks; }
int64_t wdo_result_raw_links(const wdo_result* r, const wdo_link** l) { *l = r->raw; return r->nraw; }
int32_t wdo_result_cutoffs(const wdo_result* r, const float** b, const float** cb, const float** c) {
  *b = r->best;
  *cb = r->cutb;
  *c = r->cut;
  return r->ncut;
}

const char* wdo_error_message(int code) {
  switch (code) {
    case WDO_OK: return "ok";
    case WDO_EINVAL: return "invalid argument";
    case WDO_ECYCLE: return "epsilon cycle in graph";
    case WDO_ENOPATH: return "no surviving token";
    case WDO_ENOMEM: return "out of memory";
    default: return "unknown";
  }
}

/* ----------------------------------------------------------- validation -- */

static int validate(const wdo_graph* g, const float* L, int32_t T, int32_t P, const wdo_params* p) {
  if (!g || !p || !g->row_ptr) return WDO_EINVAL;
  if (g->num_states < 1 || g->num_arcs < 0 || g->num_arcs >= (int64_t)NONE) return WDO_EINVAL;
  if (g->start_state < 0 || g->start_state >= g->num_states) return WDO_EINVAL;
  if (g->num_arcs > 0 && (!g->dst || !g->ilabel || !g->olabel || !g->weight)) return WDO_EINVAL;
  if (T < 0 || T > (1 << 24) || P < 1 || (T > 0 && !L)) return WDO_EINVAL;
  if (!(p->beam > 0.0f) || !(p->lattice_beam >= 0.0f) || p->max_active < 0) return WDO_EINVAL;
  const int64_t S = g->num_states, A = g->num_arcs;
  if (g->row_ptr[0] != 0 || (int64_t)g->row_ptr[S] != A) return WDO_EINVAL;
  for (int64_t s = 0; s < S; ++s)
    if (g->row_ptr[s] > g->row_ptr[s + 1]) return WDO_EINVAL;
  for (int64_t a = 0; a < A; ++a) {
    if ((int64_t)g->dst[a] >= S) return WDO_EINVAL;
    if (g->ilabel[a] < 0 || g->olabel[a] < 0) return WDO_EINVAL;
    if (g->ilabel[a] > P) return WDO_EINVAL;
    float w = g->weight[a];
    if (!(w >= 0.0f) || isinf(w)) return WDO_EINVAL;
  }
  if (g->final_weight)
    for (int64_t s = 0; s < S; ++s)
      if (!(g->final_weight[s] >= 0.0f)) return WDO_EINVAL;
  for (int64_t i = 0; i < (int64_t)T * P; ++i) {
    float v = L[i];
    if (isnan(v) || v > 1e30f) return WDO_EINVAL;
  }
  return WDO_OK;
}

/* Topological rank of every state in the epsilon subgraph (Kahn's algorithm);
 * WDO_ECYCLE if the epsilon arcs contain a cycle. */
static int eps_topo_rank(const wdo_graph* g, int32_t* rank) {
  const int64_t S = g->num_states;
  int32_t* indeg = calloc((size_t)S, sizeof(int32_t));
  int32_t* queue = malloc((size_t)S * sizeof(int32_t));
  if (!indeg || !queue) { free(indeg); free(queue); return WDO_ENOMEM; }
  for (int64_t a = 0; a < g->num_arcs; ++a)
    if (g->ilabel[a] == 0) indeg[g->dst[a]]++;
  int64_t head = 0, tail = 0;
  for (int64_t s = 0; s < S; ++s)
    if (indeg[s] == 0) queue[tail++] = (int32_t)s;
  while (head < tail) {
    int32_t s = queue[head];
    rank[s] = (int32_t)head;
    head++;
    for (uint32_t a = g->row_ptr[s]; a < g->row_ptr[s + 1]; ++a)
      if (g->ilabel[a] == 0 && --indeg[g->dst[a]] == 0) queue[tail++] = (int32_t)g->dst[a];
  }
  free(indeg);
  free(queue);
  return head == S ? WDO_OK : WDO_ECYCLE;
}

/* ------------------------------------------------------- decoder state -- */

typedef struct {
  uint32_t arc;
  uint32_t src;   /* global node index of the source token */
  uint32_t dst;   /* global node index of the destination token */
  float x;
  float le;       /* extra cost after pruning */
  int32_t t;
} rlink;

typedef struct {
  const wdo_graph* g;
  const float* L;
  int32_t P;
  wdo_params p;
  /* token table of the frame being built (Sec. 3.2: one token per state) */
  float* cost;
  uint32_t* pred;
  uint32_t* mark;       /* == stamp: the state holds a token this frame */
  uint32_t stamp;
  uint32_t* list;       /* states holding a token, in insertion order */
  int64_t nlist;
  float* sortbuf;
  /* surviving tokens of all frames, each frame sorted by state */
  wdo_token* toks;
  int64_t ntoks, captoks;
  int64_t* frame_off;   /* [T+2] */
  /* lattice links of all frames */
  rlink* links;
  int64_t nlinks, caplinks;
  int64_t* link_off;    /* [T+2] */
  float *best, *cutb, *cut;
  wdo_stats st;
} dec;

static uint32_t emit_deg(const wdo_graph* g, uint32_t s) {
  uint32_t n = 0;
  for (uint32_t a = g->row_ptr[s]; a < g->row_ptr[s + 1]; ++a) n += g->ilabel[a] != 0;
  return n;
}

static uint32_t eps_deg(const wdo_graph* g, uint32_t s) {
  uint32_t n = 0;
  for (uint32_t a = g->row_ptr[s]; a < g->row_ptr[s + 1]; ++a) n += g->ilabel[a] == 0;
  return n;
}

/* Recombination (Sec. 3.2, Alg. 1): keep the better of the held token and the
 * candidate (x, a).  Returns 1 if the candidate won. */
static int recombine(dec* d, uint32_t s, float x, uint32_t a) {
  if (d->mark[s] != d->stamp) {
    d->mark[s] = d->stamp;
    d->cost[s] = x;
    d->pred[s] = a;
    d->list[d->nlist++] = s;
    return 1;
  }
  if (better(x, a, d->cost[s], d->pred[s])) {
    d->cost[s] = x;
    d->pred[s] = a;
    return 1;
  }
  return 0;
}

/* Epsilon closure at one frame: relax the epsilon arcs of every held token
 * until no token changes; candidates above the beam cutoff are not offered.
 * The fixpoint does not depend on the visiting order because fp32 addition is
 * monotone. */
static void eps_closure(dec* d, float cutb) {
  const wdo_graph* g = d->g;
  int changed = 1;
  while (changed) {
    changed = 0;
    for (int64_t i = 0; i < d->nlist; ++i) {
      uint32_t s = d->list[i];
      float c = d->cost[s];
      for (uint32_t a = g->row_ptr[s]; a < g->row_ptr[s + 1]; ++a) {
        if (g->ilabel[a] != 0) continue;
        float x = canon(c + g->weight[a]);
        if (isinf(x) || !(x <= cutb)) continue;
        if (recombine(d, g->dst[a], x, a)) changed = 1;
      }
    }
  }
}

/* Drop held tokens whose cost exceeds `cut` (inclusive cutoff). */
static void prune_list(dec* d, float cut) {
  int64_t k = 0;
  for (int64_t i = 0; i < d->nlist; ++i) {
    uint32_t s = d->list[i];
    if (d->cost[s] <= cut) d->list[k++] = s;
    else d->mark[s] = d->stamp - 1;
  }
  d->nlist = k;
}

/* Finish frame t: epsilon closure, max-active, record the surviving set. */
static int finish_frame(dec* d, int32_t t, float best) {
  const wdo_graph* g = d->g;
  float cutb = best + d->p.beam;
  prune_list(d, cutb);
  eps_closure(d, cutb);
  for (int64_t i = 0; i < d->nlist; ++i) {
    d->st.arcs_expanded += eps_deg(g, d->list[i]);
    d->st.eps_arcs_expanded += eps_deg(g, d->list[i]);
  }
  float cut = cutb;
  if (d->p.max_active > 0 && d->nlist > d->p.max_active) {
    for (int64_t i = 0; i < d->nlist; ++i) d->sortbuf[i] = d->cost[d->list[i]];
    qsort(d->sortbuf, (size_t)d->nlist, sizeof(float), cmp_float);
    float v = d->sortbuf[d->p.max_active - 1];
    if (v < cut) cut = v;
  }
  prune_list(d, cut);
  qsort(d->list, (size_t)d->nlist, sizeof(uint32_t), cmp_u32);
  if (grow((void**)&d->toks, &d->captoks, d->ntoks + d->nlist, sizeof(wdo_token))) return WDO_ENOMEM;
  d->frame_off[t] = d->ntoks;
  for (int64_t i = 0; i < d->nlist; ++i) {
    uint32_t s = d->list[i];
    wdo_token tk = {t, (int32_t)s, d->cost[s], d->pred[s]};
    d->toks[d->ntoks++] = tk;
  }
  d->frame_off[t + 1] = d->ntoks;
  if (d->ntoks >= (int64_t)NONE) return WDO_ENOMEM;
  d->best[t] = best;
  d->cutb[t] = cutb;
  d->cut[t] = cut;
  d->st.tokens += d->nlist;
  if (d->nlist > d->st.max_tokens) d->st.max_tokens = d->nlist;
  return WDO_OK;
}

/* Index of `state` among the surviving tokens of frame t, or -1. */
static int64_t find_node(const dec* d, int32_t t, uint32_t state) {
  int64_t lo = d->frame_off[t], hi = d->frame_off[t + 1];
  while (lo < hi) {
    int64_t mid = lo + (hi - lo) / 2;
    if ((uint32_t)d->toks[mid].state < state) lo = mid + 1;
    else hi = mid;
  }
  if (lo < d->frame_off[t + 1] && (uint32_t)d->toks[lo].state == state) return lo;
  return -1;
}

static int add_link(dec* d, int32_t t, uint32_t arc, int64_t src, int64_t dst, float x) {
  if (dst < 0) return WDO_EINVAL; /* cannot happen: the destination is within the cutoff */
  if (grow((void**)&d->links, &d->caplinks, d->nlinks + 1, sizeof(rlink))) return WDO_ENOMEM;
  rlink l = {arc, (uint32_t)src, (uint32_t)dst, x, INFINITY, t};
  d->links[d->nlinks++] = l;
  return WDO_OK;
}

/* Lattice links of frame t (Sec. 3.4): emitting links from the survivors of
 * frame t-1 and epsilon links from the survivors of frame t whose candidate
 * cost lies within the final cutoff of frame t. */
static int record_links(dec* d, int32_t t) {
  const wdo_graph* g = d->g;
  const float cut = d->cut[t];
  d->link_off[t] = d->nlinks;
  if (t > 0) {
    const float* row = d->L + (int64_t)(t - 1) * d->P;
    for (int64_t i = d->frame_off[t - 1]; i < d->frame_off[t]; ++i) {
      uint32_t s = (uint32_t)d->toks[i].state;
      float c = d->toks[i].cost;
      for (uint32_t a = g->row_ptr[s]; a < g->row_ptr[s + 1]; ++a) {
        if (g->ilabel[a] == 0) continue;
        float ac = -row[g->ilabel[a] - 1];
        float x = c + ac;
        x = canon(x + g->weight[a]);
        if (isinf(x) || !(x <= cut)) continue;
        int rc = add_link(d, t, a, i, find_node(d, t, g->dst[a]), x);
        if (rc) return rc;
      }
    }
  }
  for (int64_t i = d->frame_off[t]; i < d->frame_off[t + 1]; ++i) {
    uint32_t s = (uint32_t)d->toks[i].state;
    float c = d->toks[i].cost;
    for (uint32_t a = g->row_ptr[s]; a < g->row_ptr[s + 1]; ++a) {
      if (g->ilabel[a] != 0) continue;
      float x = canon(c + g->weight[a]);
      if (isinf(x) || !(x <= cut)) continue;
      int rc = add_link(d, t, a, i, find_node(d, t, g->dst[a]), x);
      if (rc) return rc;
    }
  }
  d->link_off[t + 1] = d->nlinks;
  d->st.raw_links = d->nlinks;
  return WDO_OK;
}

/* Source state of an arc: the state whose CSR range holds it. */
static uint32_t arc_src(const wdo_graph* g, uint32_t a) {
  int64_t lo = 0, hi = g->num_states; /* first s with row_ptr[s] > a, minus one */
  while (lo < hi) {
    int64_t mid = lo + (hi - lo) / 2;
    if (g->row_ptr[mid] <= a) lo = mid + 1;
    else hi = mid;
  }
  return (uint32_t)(lo - 1);
}

/* ---------------------------------------------------- lattice pruning -- */

/* Sec. 3.5: extra cost of a node = best complete-path cost through it minus
 * the best overall; of a link = extra(dst) + (x - cost(dst)).  Updated until
 * nothing changes, frame by frame from the last one (links only go from frame
 * t to t or t+1), emitting out-links before the epsilon links of the frame. */
static float* prune_lattice(dec* d, int32_t T, const float* F, float best_total) {
  float* ex = malloc((size_t)(d->ntoks + 1) * sizeof(float));
  if (!ex) return NULL;
  for (int64_t n = 0; n < d->ntoks; ++n) ex[n] = INFINITY;
  for (int64_t n = d->frame_off[T]; n < d->frame_off[T + 1]; ++n)
    if (!isinf(F[n - d->frame_off[T]])) ex[n] = F[n - d->frame_off[T]] - best_total;
  for (int32_t t = T; t >= 0; --t) {
    if (t < T)
      for (int64_t k = d->link_off[t + 1]; k < d->link_off[t + 2]; ++k) {
        rlink* l = &d->links[k];
        if (d->g->ilabel[l->arc] == 0) continue;
        float le = ex[l->dst] + (l->x - d->toks[l->dst].cost);
        if (le < ex[l->src]) ex[l->src] = le;
      }
    int changed = 1;
    while (changed) {
      changed = 0;
      for (int64_t k = d->link_off[t]; k < d->link_off[t + 1]; ++k) {
        rlink* l = &d->links[k];
        if (d->g->ilabel[l->arc] != 0) continue;
        float le = ex[l->dst] + (l->x - d->toks[l->dst].cost);
        if (le < ex[l->src]) { ex[l->src] = le; changed = 1; }
      }
    }
  }
  for (int64_t k = 0; k < d->nlinks; ++k) {
    rlink* l = &d->links[k];
    l->le = ex[l->dst] + (l->x - d->toks[l->dst].cost);
  }
  return ex; /* node extras, indexed by global node */
}

/* ------------------------------------------------------- posteriors -- */

/* Streaming -log(sum exp(-v)): m = smallest term so far, s = sum exp(-(v-m)). */
typedef struct { double m, s; } lse;
static void lse_add(lse* a, double v) {
  if (isinf(v)) return;
  if (a->s == 0.0) { a->m = v; a->s = 1.0; return; }
  if (v < a->m) { a->s = a->s * exp(-(a->m - v)) + 1.0; a->m = v; }
  else a->s += exp(-(v - a->m));
}
static double lse_val(const lse* a) { return a->s == 0.0 ? INFINITY : a->m - log(a->s); }

typedef struct { int64_t k; int32_t r; } kr;
static int cmp_kr_up(const void* a, const void* b) {
  const kr *x = a, *y = b;
  if (x->r != y->r) return (x->r > y->r) - (x->r < y->r);
  return (x->k > y->k) - (x->k < y->k);
}

/* Forward-backward over the kept links (fp64): alpha(n) = -log sum over
 * incoming links of exp(-(alpha(src) + w + ac)); beta likewise backwards with
 * the final cost at the last frame; posterior = exp(Z - alpha - w - ac - beta).
 * Nodes of a frame are taken in epsilon-topological order. */
static int posteriors(dec* d, int32_t T, const uint8_t* keep, const int32_t* rank, int final_used,
                      double* post) {
  const wdo_graph* g = d->g;
  lse* al = calloc((size_t)d->ntoks, sizeof(lse));
  lse* be = calloc((size_t)d->ntoks, sizeof(lse));
  kr* order = malloc((size_t)(d->nlinks + 1) * sizeof(kr));
  if (!al || !be || !order) { free(al); free(be); free(order); return WDO_ENOMEM; }
  int64_t start = find_node(d, 0, (uint32_t)g->start_state);
  lse_add(&al[start], 0.0);
  /* forward */
  for (int32_t t = 0; t <= T; ++t) {
    for (int64_t k = d->link_off[t]; k < d->link_off[t + 1]; ++k) {
      const rlink* l = &d->links[k];
      if (!keep[k] || g->ilabel[l->arc] == 0) continue;
      double ac = -(double)d->L[(int64_t)(t - 1) * d->P + g->ilabel[l->arc] - 1];
      lse_add(&al[l->dst], lse_val(&al[l->src]) + (double)g->weight[l->arc] + ac);
    }
    int64_t n = 0;
    for (int64_t k = d->link_off[t]; k < d->link_off[t + 1]; ++k)
      if (keep[k] && g->ilabel[d->links[k].arc] == 0) {
        kr e = {k, rank[d->toks[d->links[k].src].state]};
        order[n++] = e;
      }
    qsort(order, (size_t)n, sizeof(kr), cmp_kr_up);
    for (int64_t i = 0; i < n; ++i) {
      const rlink* l = &d->links[order[i].k];
      lse_add(&al[l->dst], lse_val(&al[l->src]) + (double)g->weight[l->arc]);
    }
  }
  /* backward */
  for (int32_t t = T; t >= 0; --t) {
    if (t == T)
      for (int64_t n = d->frame_off[T]; n < d->frame_off[T + 1]; ++n) {
        double fo = 0.0;
        if (final_used) fo = (double)g->final_weight[d->toks[n].state];
        lse_add(&be[n], fo);
      }
    if (t < T)
      for (int64_t k = d->link_off[t + 1]; k < d->link_off[t + 2]; ++k) {
        const rlink* l = &d->links[k];
        if (!keep[k] || g->ilabel[l->arc] == 0) continue;
        double ac = -(double)d->L[(int64_t)t * d->P + g->ilabel[l->arc] - 1];
        lse_add(&be[l->src], (double)g->weight[l->arc] + ac + lse_val(&be[l->dst]));
      }
    int64_t n = 0;
    for (int64_t k = d->link_off[t]; k < d->link_off[t + 1]; ++k)
      if (keep[k] && g->ilabel[d->links[k].arc] == 0) {
        kr e = {k, rank[d->toks[d->links[k].src].state]};
        order[n++] = e;
      }
    qsort(order, (size_t)n, sizeof(kr), cmp_kr_up);
    for (int64_t i = n - 1; i >= 0; --i) {
      const rlink* l = &d->links[order[i].k];
      lse_add(&be[l->src], (double)g->weight[l->arc] + lse_val(&be[l->dst]));
    }
  }
  double Z = lse_val(&be[start]);
  for (int64_t k = 0; k < d->nlinks; ++k) {
    post[k] = 0.0;
    if (!keep[k]) continue;
    const rlink* l = &d->links[k];
    double ac = g->ilabel[l->arc] ? -(double)d->L[(int64_t)(l->t - 1) * d->P + g->ilabel[l->arc] - 1] : 0.0;
    post[k] = exp(Z - lse_val(&al[l->src]) - (double)g->weight[l->arc] - ac - lse_val(&be[l->dst]));
  }
  free(al);
  free(be);
  free(order);
  return WDO_OK;
}

/* ----------------------------------------------------------- decode -- */

static int cmp_link_out(const void* a, const void* b) {
  const wdo_link *x = a, *y = b;
  if (x->t != y->t) return (x->t > y->t) - (x->t < y->t);
  return (x->arc_id > y->arc_id) - (x->arc_id < y->arc_id);
}

static void fill_link(const dec* d, const rlink* l, wdo_link* o) {
  const wdo_graph* g = d->g;
  o->t = l->t;
  o->arc_id = l->arc;
  o->src_state = d->toks[l->src].state;
  o->dst_state = d->toks[l->dst].state;
  o->ilabel = g->ilabel[l->arc];
  o->olabel = g->olabel[l->arc];
  o->graph_cost = g->weight[l->arc];
  o->ac_cost = o->ilabel ? -d->L[(int64_t)(l->t - 1) * d->P + o->ilabel - 1] : 0.0f;
  o->fwd_cost = l->x;
  o->extra = l->le;
  o->posterior = 0.0;
}

static void dec_free(dec* d) {
  free(d->cost);
  free(d->pred);
  free(d->mark);
  free(d->list);
  free(d->sortbuf);
  free(d->toks);
  free(d->frame_off);
  free(d->links);
  free(d->link_off);
  free(d->best);
  free(d->cutb);
  free(d->cut);
}

int wdo_decode(const wdo_graph* g, const float* L, int32_t T, int32_t P, const wdo_params* p,
               wdo_result** out) {
  if (!out) return WDO_EINVAL;
  *out = NULL;
  int rc = validate(g, L, T, P, p);
  if (rc) return rc;
  const int64_t S = g->num_states;
  int32_t* rank = malloc((size_t)S * sizeof(int32_t));
  if (!rank) return WDO_ENOMEM;
  rc = eps_topo_rank(g, rank);
  if (rc) { free(rank); return rc; }

  dec d;
  memset(&d, 0, sizeof d);
  d.g = g;
  d.L = L;
  d.P = P;
  d.p = *p;
  d.cost = malloc((size_t)S * sizeof(float));
  d.pred = malloc((size_t)S * sizeof(uint32_t));
  d.mark = calloc((size_t)S, sizeof(uint32_t));
  d.list = malloc((size_t)S * sizeof(uint32_t));
  d.sortbuf = malloc((size_t)S * sizeof(float));
  d.frame_off = calloc((size_t)T + 3, sizeof(int64_t));
  d.link_off = calloc((size_t)T + 3, sizeof(int64_t));
  d.best = malloc(((size_t)T + 1) * sizeof(float));
  d.cutb = malloc(((size_t)T + 1) * sizeof(float));
  d.cut = malloc(((size_t)T + 1) * sizeof(float));
  wdo_result* r = calloc(1, sizeof(wdo_result));
  if (!d.cost || !d.pred || !d.mark || !d.list || !d.sortbuf || !d.frame_off || !d.link_off ||
      !d.best || !d.cutb || !d.cut || !r) {
    rc = WDO_ENOMEM;
    goto fail;
  }
  d.stamp = 2;

  /* frame 0: the start token, then closure and max-active */
  d.nlist = 0;
  recombine(&d, (uint32_t)g->start_state, 0.0f, NONE);
  if ((rc = finish_frame(&d, 0, 0.0f))) goto fail;
  if ((rc = record_links(&d, 0))) goto fail;

  for (int32_t t = 1; t <= T; ++t) {
    d.stamp += 2;
    d.nlist = 0;
    const float* row = L + (int64_t)(t - 1) * P;
    /* emitting step: every out-arc of every surviving token of frame t-1 */
    for (int64_t i = d.frame_off[t - 1]; i < d.frame_off[t]; ++i) {
      uint32_t s = (uint32_t)d.toks[i].state;
      float c = d.toks[i].cost;
      d.st.arcs_expanded += emit_deg(g, s);
      for (uint32_t a = g->row_ptr[s]; a < g->row_ptr[s + 1]; ++a) {
        if (g->ilabel[a] == 0) continue;
        float ac = -row[g->ilabel[a] - 1];
        float x = c + ac;
        x = canon(x + g->weight[a]);
        if (isinf(x)) continue;
        recombine(&d, g->dst[a], x, a);
      }
    }
    if (d.nlist == 0) { rc = WDO_ENOPATH; goto fail; }
    float best = INFINITY;
    for (int64_t i = 0; i < d.nlist; ++i)
      if (d.cost[d.list[i]] < best) best = d.cost[d.list[i]];
    if ((rc = finish_frame(&d, t, best))) goto fail;
    if ((rc = record_links(&d, t))) goto fail;
  }

  /* final costs and the best end state (lowest state id on ties) */
  const int64_t nT = d.frame_off[T + 1] - d.frame_off[T];
  float* F = malloc((size_t)(nT > 0 ? nT : 1) * sizeof(float));
  if (!F) { rc = WDO_ENOMEM; goto fail; }
  int final_used = 0;
  if (g->final_weight)
    for (int64_t i = 0; i < nT; ++i) {
      const wdo_token* tk = &d.toks[d.frame_off[T] + i];
      float fw = g->final_weight[tk->state];
      if (!isinf(fw) && !isinf(tk->cost + fw)) final_used = 1;
    }
  float best_total = INFINITY;
  int64_t bnode = -1;
  for (int64_t i = 0; i < nT; ++i) {
    const wdo_token* tk = &d.toks[d.frame_off[T] + i];
    F[i] = final_used ? canon(tk->cost + g->final_weight[tk->state]) : tk->cost;
    if (F[i] < best_total) { best_total = F[i]; bnode = d.frame_off[T] + i; }
  }
  if (bnode < 0) { free(F); rc = WDO_ENOPATH; goto fail; }
  r->cost = best_total;

  /* traceback: an epsilon arc stays in its frame, an emitting arc goes back one */
  {
    int64_t cap = 0;
    int32_t t = T;
    int64_t n = bnode;
    while (d.toks[n].pred_arc != NONE) {
      uint32_t a = d.toks[n].pred_arc;
      if (g->olabel[a] != 0) {
        if (grow((void**)&r->words, &cap, r->nwords + 1, sizeof(int32_t))) { free(F); rc = WDO_ENOMEM; goto fail; }
        r->words[r->nwords++] = g->olabel[a];
      }
      if (g->ilabel[a] != 0) t--;
      n = find_node(&d, t, arc_src(g, a));
      if (n < 0) { free(F); rc = WDO_EINVAL; goto fail; }
    }
    for (int32_t i = 0; i < r->nwords / 2; ++i) {
      int32_t tmp = r->words[i];
      r->words[i] = r->words[r->nwords - 1 - i];
      r->words[r->nwords - 1 - i] = tmp;
    }
  }

  float* node_extra = prune_lattice(&d, T, F, best_total);
  free(F);
  uint8_t* keep = malloc((size_t)(d.nlinks + 1));
  double* post = malloc((size_t)(d.nlinks + 1) * sizeof(double));
  uint8_t* used = calloc((size_t)d.ntoks + 1, 1);
  if (!node_extra || !keep || !post || !used) {
    free(node_extra); free(keep); free(post); free(used);
    rc = WDO_ENOMEM;
    goto fail;
  }
  int64_t nkeep = 0;
  for (int64_t k = 0; k < d.nlinks; ++k) {
    float le = d.links[k].le;
    keep[k] = !isinf(le) && le <= p->lattice_beam;
    nkeep += keep[k];
  }
  if ((rc = posteriors(&d, T, keep, rank, final_used, post)) ||
      !(r->links = malloc((size_t)(nkeep + 1) * sizeof(wdo_link)))) {
    if (!rc) rc = WDO_ENOMEM;
    free(node_extra); free(keep); free(post); free(used);
    goto fail;
  }
  used[find_node(&d, 0, (uint32_t)g->start_state)] = 1;
  for (int64_t k = 0; k < d.nlinks; ++k) {
    if (!keep[k]) continue;
    wdo_link* o = &r->links[r->nlinks++];
    fill_link(&d, &d.links[k], o);
    o->posterior = post[k];
    used[d.links[k].src] = 1;
    used[d.links[k].dst] = 1;
  }
  qsort(r->links, (size_t)r->nlinks, sizeof(wdo_link), cmp_link_out);
  int64_t nn = 0;
  for (int64_t n = 0; n < d.ntoks; ++n) nn += used[n];
  r->nodes = malloc((size_t)(nn + 1) * sizeof(wdo_node));
  if (!r->nodes) { free(node_extra); free(keep); free(post); free(used); rc = WDO_ENOMEM; goto fail; }
  for (int64_t n = 0; n < d.ntoks; ++n) /* tokens are already in (t, state) order */
    if (used[n]) {
      wdo_node o = {d.toks[n].t, d.toks[n].state, d.toks[n].cost, node_extra[n]};
      r->nodes[r->nnodes++] = o;
    }
  free(used);
  free(node_extra);

  d.st.frames = T;
  d.st.final_reached = final_used;
  d.st.kept_links = r->nlinks;
  d.st.nodes = r->nnodes;
  r->stats = d.st;

  if (p->debug) {
    r->raw = malloc((size_t)(d.nlinks + 1) * sizeof(wdo_link));
    if (!r->raw) { free(keep); free(post); rc = WDO_ENOMEM; goto fail; }
    for (int64_t k = 0; k < d.nlinks; ++k) {
      fill_link(&d, &d.links[k], &r->raw[k]);
      r->raw[k].posterior = post[k];
    }
    r->nraw = d.nlinks;
    qsort(r->raw, (size_t)r->nraw, sizeof(wdo_link), cmp_link_out);
    r->toks = d.toks;
    r->ntoks = d.ntoks;
    d.toks = NULL;
    r->best = d.best;
    r->cutb = d.cutb;
    r->cut = d.cut;
    r->ncut = T + 1;
    d.best = d.cutb = d.cut = NULL;
  }
  free(keep);
  free(post);
  free(rank);
  dec_free(&d);
  *out = r;
  return WDO_OK;

fail:
  free(rank);
  dec_free(&d);
  wdo_result_free(r);
  return rc;
}
