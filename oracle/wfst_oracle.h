/*
 * CPU oracle for frame-synchronous Viterbi token passing with exact lattice
 * generation, lattice pruning and arc posteriors.
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, sequential, deliberately slow
 * restatement of what the decoder computes.  Only the test-suite, the smoke
 * check and the CPU-baseline leg of the benchmark may load it; the GPU library
 * never links, calls or includes it, and it shares no code with that library.
 *
 * All costs are IEEE fp32 with round-to-nearest-even, accumulated in the order
 * stated per function (no FMA, no re-association); only posteriors are fp64.
 * Build with: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fPIC -shared
 */
#ifndef WFST_ORACLE_H
#define WFST_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { WDO_OK = 0, WDO_EINVAL = 1, WDO_ECYCLE = 2, WDO_ENOPATH = 3, WDO_ENOMEM = 6 };

/* Decoding graph in CSR form; arc id = index into the arc arrays. */
typedef struct {
  int32_t num_states;
  int64_t num_arcs;
  int32_t start_state;
  const uint32_t* row_ptr;     /* [S+1] */
  const uint32_t* dst;         /* [A]   */
  const int32_t* ilabel;       /* [A]  0 = epsilon, k >= 1 -> log-likelihood column k-1 */
  const int32_t* olabel;       /* [A]  0 = no output word */
  const float* weight;         /* [A]  finite, >= 0 */
  const float* final_weight;   /* [S] or NULL (NULL: every state final with cost 0) */
} wdo_graph;

typedef struct {
  float beam;          /* > 0, may be +inf */
  int32_t max_active;  /* 0 = unlimited */
  float lattice_beam;  /* >= 0, may be +inf */
  int32_t debug;       /* nonzero: keep per-frame token sets and the raw lattice */
} wdo_params;

/* One lattice link (a token-passing operation that survived). */
typedef struct {
  int32_t t;            /* frame of the destination token (1..T for emitting, 0..T for epsilon) */
  uint32_t arc_id;
  int32_t src_state;    /* source token is at frame t-1 (emitting) or t (epsilon) */
  int32_t dst_state;
  int32_t ilabel;
  int32_t olabel;
  float graph_cost;     /* arc weight */
  float ac_cost;        /* -loglike[t-1][ilabel-1] for emitting links, 0 for epsilon */
  float fwd_cost;       /* the candidate cost x this link offered its destination */
  float extra;          /* extra cost of the link after pruning */
  double posterior;     /* fp64 arc posterior on the pruned lattice */
} wdo_link;

typedef struct {
  int32_t t;
  int32_t state;
  float cost;           /* Viterbi forward cost of the token */
  float extra;          /* node extra cost */
} wdo_node;

typedef struct {
  int32_t t;
  int32_t state;
  float cost;
  uint32_t pred_arc;    /* 0xffffffff for the start token */
} wdo_token;

typedef struct {
  int32_t frames;
  int32_t final_reached;    /* 1 if final weights were used at the last frame */
  int64_t arcs_expanded;    /* emitting out-arcs of every surviving token + epsilon out-arcs
                               of every token that took part in the epsilon closure */
  int64_t tokens;           /* sum over frames of surviving tokens */
  int64_t max_tokens;       /* max over frames */
  int64_t raw_links;        /* links recorded before pruning */
  int64_t kept_links;
  int64_t nodes;
  int64_t eps_arcs_expanded;  /* the epsilon part of arcs_expanded */
} wdo_stats;

typedef struct wdo_result wdo_result;

/* Decode one utterance.  loglikes: host, T x P row-major fp32.  On success
 * *out is a result owned by the caller (free with wdo_result_free). */
int wdo_decode(const wdo_graph* g, const float* loglikes, int32_t T, int32_t P,
               const wdo_params* p, wdo_result** out);

float   wdo_result_cost(const wdo_result* r);
int32_t wdo_result_words(const wdo_result* r, const int32_t** words);
int64_t wdo_result_links(const wdo_result* r, const wdo_link** links);   /* sorted by (t, arc_id) */
int64_t wdo_result_nodes(const wdo_result* r, const wdo_node** nodes);   /* sorted by (t, state) */
void    wdo_result_stats(const wdo_result* r, wdo_stats* s);
/* debug only (params.debug != 0): all surviving tokens of every frame, sorted
 * by (t, state); the raw lattice (every recorded link, kept or not, with its
 * extra cost, posterior 0); per-frame best cost, beam cutoff and final cutoff. */
int64_t wdo_result_tokens(const wdo_result* r, const wdo_token** toks);
int64_t wdo_result_raw_links(const wdo_result* r, const wdo_link** links);
int32_t wdo_result_cutoffs(const wdo_result* r, const float** best, const float** cutoff_beam,
                           const float** cutoff);
void    wdo_result_free(wdo_result* r);
const char* wdo_error_message(int code);

#ifdef __cplusplus
}
#endif
#endif
