/*
 * wfstdec: frame-synchronous Viterbi token passing over a WFST decoding graph
 * with exact lattice generation, lattice pruning and arc posteriors, on one
 * AMD Instinct MI355X (gfx950).
 *
 * Method: Chen, Luitjens, Xu, Wang, Povey, Khudanpur, "A GPU-based WFST
 * Decoder with Exact Lattice Generation", Interspeech 2018 -- token passing
 * and atomic recombination (Sec. 3.2, Alg. 1), load-balanced arc expansion
 * (Sec. 3.3, Alg. 2), lattice-arc recording (Sec. 3.4), lattice pruning and
 * final merge (Sec. 3.5, also incrementally on a second stream, Sec. 3.1),
 * lattice posteriors (Sec. 4.1), the compact exact lattice (Sec. 3.4, on the
 * host), streaming decodes (the integration with acoustic inference the
 * paper leaves to future work, Sec. 5).
 *
 * Conventions for every entry point:
 *  - Return a wd_status; no exception crosses this boundary.  On a non-OK
 *    status, wd_last_error() returns a message for the calling thread.
 *  - "device" pointers are HIP device memory owned by the caller (e.g. torch
 *    tensors).  The library borrows them for the duration of the call (a
 *    stream: until wd_stream_end / wd_stream_free returns) and never
 *    allocates device memory itself; its only device resources are one
 *    pruning stream per device (created on first use, kept for the process)
 *    and a few events per chip-wide decode.
 *  - Work is enqueued on the caller's stream; wd_decode / wd_decode_batch
 *    return after the results have been copied to host memory.
 *  - Results are deterministic: identical inputs give identical outputs,
 *    bit for bit (posteriors: see wd_lat_arc).
 */
#ifndef WFSTDEC_H
#define WFSTDEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WD_OK = 0,
  WD_EINVAL = 1,     /* malformed graph, log-likelihoods or parameters */
  WD_ECYCLE = 2,     /* the epsilon arcs of the graph contain a cycle */
  WD_ENOPATH = 3,    /* no token survived some frame */
  WD_ECAPACITY = 4,  /* the workspace was too small; wd_result_stats reports
                        the capacities needed, retry with a larger workspace */
  WD_EDEVICE = 5     /* a HIP call failed */
} wd_status;

/* Decoding graph (host memory, CSR; arc id = index into the arc arrays).
 * Arc ids order recombination ties (Sec. 3.2, Alg. 1 packs the arc id under
 * the cost), so they are part of the result. */
typedef struct {
  int32_t num_states;          /* S >= 1 */
  int64_t num_arcs;            /* A, 0 <= A < 2^32 - 1 */
  int32_t start_state;         /* 0 <= start < S */
  const uint32_t* row_ptr;     /* [S+1], row_ptr[0] = 0, non-decreasing, row_ptr[S] = A */
  const uint32_t* dst;         /* [A] < S */
  const int32_t* ilabel;       /* [A] 0 = epsilon; k >= 1 reads log-likelihood column k-1 */
  const int32_t* olabel;       /* [A] >= 0; 0 = no output word */
  const float* weight;         /* [A] finite, >= 0 */
  const float* final_weight;   /* [S] >= 0 or +inf (not final); NULL = every state final, cost 0 */
  int32_t num_pdfs;            /* P: every ilabel must be <= P, 1 <= P < 2^24 */
} wd_graph_desc;

typedef struct wd_graph wd_graph;

/* Decoding parameters. */
typedef struct {
  float beam;          /* > 0, may be +inf: keep tokens within best + beam */
  int32_t max_active;  /* >= 0; 0 = unlimited; else keep the max_active best (ties kept) */
  float lattice_beam;  /* >= 0, may be +inf: keep lattice links within this extra cost */
  uint32_t flags;      /* WD_FLAG_* */
} wd_params;

/* Debug output: every surviving token of every frame (wd_result_tokens), the
 * raw lattice before pruning (wd_result_raw_lattice) and the per-frame cutoffs
 * (wd_result_cutoffs).  Needs workspace capacity for the raw lattice. */
#define WD_FLAG_DEBUG 1u
/* Time the forward (token passing) and lattice kernels with HIP events on the
 * caller's stream and report them in wd_stats (whole launch: all utterances
 * of a batch). */
#define WD_FLAG_TIMING 2u
/* Execution mode.  One workgroup per utterance runs every frame inside one
 * launch: best while frames hold up to a few thousand tokens.  Chip-wide mode
 * runs every step of a frame as a kernel over the whole GPU (1024 workgroups
 * per utterance, launched frame by frame on the caller's stream): for frames
 * of 10^5..10^6 tokens.  Results are identical.  With neither flag the
 * library picks chip-wide when max_active is 0 (no limit) or at least
 * WD_CHIP_WIDE_MAX_ACTIVE, else one workgroup.  Both flags: WD_EINVAL. */
#define WD_FLAG_ONE_WORKGROUP 4u
#define WD_FLAG_CHIP_WIDE 8u
#define WD_CHIP_WIDE_MAX_ACTIVE 32768
/* Chip-wide mode only (ignored by one-workgroup decodes): expand emitting
 * arcs with the paper's dynamic load balancing (Alg. 2, Sec. 3.3: a
 * dispatcher counter hands out frontier tokens; a group of lanes expands all
 * arcs of one token) instead of the static prefix-sum work space.  The
 * result is identical; the flag exists for the A/B comparison. */
#define WD_FLAG_DYNAMIC_LB 16u
/* Chip-wide mode prunes the lattice conservatively while decoding, on a
 * second stream of the library's own (Fig. 1 of the paper prunes on a second
 * stream as decoding goes): frames are recorded in windows of 32 into two raw
 * window slots taken in turn; 8 frames after a window's last frame, its links
 * (and those of the 8 frames after it) are swept with the lowest possible
 * extra cost (0) on the 8th frame's tokens, and the window's links that cannot
 * be kept by the final pruning are dropped while the rest are appended to the
 * compacted region of the link store.  Decoding goes on meanwhile and only
 * waits for a window's pruning before it reuses that window's slot.  The link
 * store then holds the compacted region (capacity `links`) plus the two slots
 * (`window_links` each) instead of every raw link.  The result is identical.
 * This flag turns it off (A/B).  Never done with WD_FLAG_DEBUG, which returns
 * the raw lattice.  Decodes on one device share the library's pruning stream
 * and are ordered on it by events. */
#define WD_FLAG_NO_INCREMENTAL_PRUNE 32u
/* Step profile of the one-workgroup forward pass (a measurement aid, off in
 * timed runs; WD_EINVAL in chip-wide mode): a separately compiled copy of the
 * forward kernel stores the device wall clock each time its first thread
 * passes a step boundary of a frame (wd_result_phases).  The result is the
 * same; the stores add a little time to each frame. */
#define WD_FLAG_PHASES 64u
/* One-workgroup mode: take the epsilon closure level by level (one pass per
 * epsilon level, each a round of dependent memory reads) even when the graph
 * has an epsilon path table (wd_graph_eps_paths), where by default every
 * epsilon path of a state within the beam is relaxed at once.  The result is
 * identical; the flag exists for the A/B comparison. */
#define WD_FLAG_EPS_LEVELS 128u
/* Words per frame of wd_result_phases: WD_PHASE_STAMPS wall-clock stamps, at
 * (0) the frame's start, the end of (1) the emitting expansion and its best
 * cost, (2) the epsilon closure, (3) the survivor pass, (4) the max-active
 * cutoff, (5) the compaction into the state-sorted frontier, (6) the degree
 * prefix sums, (7) the next frame's work-item owners and cache warming, (8)
 * the frame's bookkeeping, (9) the frame (table reset); then word 10 = (1 if
 * the frame's token table was in LDS) | surviving tokens << 8 | lattice
 * links << 32 (the links are formed after the forward pass, every frame at
 * once, and their count is filled in then), and word 11 = emitting work
 * items | LDS-table epsilon bucket entries << 32 (touched states with
 * epsilon arcs). */
#define WD_PHASE_STAMPS 10
#define WD_PHASE_SLOTS 12
/* Stamps of the lattice pass (wd_result_lattice_phases, WD_FLAG_PHASES): at
 * (0) its start, the end of (1) the final costs and best end token, (2) the
 * backward pruning sweep (Sec. 3.5), (3) the kept-link list, (4) the kept
 * links' per-frame offsets and records, (5) the fp64 forward-backward
 * posteriors, (6) the merge of the kept links into (t, arc id) order, (7) the
 * node list. */
#define WD_LATTICE_PHASE_STAMPS 8

/* Workspace capacities (per utterance).  0 selects a default.  A decode that
 * outgrows a capacity fails with WD_ECAPACITY and reports what it needed. */
typedef struct {
  int64_t frame_tokens;   /* tokens touched in one frame (<= S) */
  int64_t frame_arcs;     /* emitting arcs expanded in one frame */
  int64_t nodes;          /* surviving tokens summed over all frames (< 2^32) */
  int64_t links;          /* lattice links recorded before pruning (the link store; with
                             chip-wide incremental pruning its compacted region) */
  int64_t kept_links;     /* lattice links returned (after pruning; raw links with WD_FLAG_DEBUG) */
  int64_t window_links;   /* chip-wide incremental pruning: raw links of one 32-frame window
                             (`links` is then the compacted region); unused otherwise */
} wd_caps;

/* One lattice link of the pruned lattice, i.e. one token-passing operation
 * that survived (Sec. 3.4-3.5).  Links are sorted by (t, arc_id); the pair
 * is unique.  posterior is computed in fp64 on the pruned lattice; every other
 * field is exact.  Posteriors agree across runs to within fp64 rounding of the
 * summation order (<< 1e-9), not necessarily bit for bit. */
typedef struct {
  int32_t t;            /* frame of the destination token */
  uint32_t arc_id;
  int32_t src_state;    /* source token at frame t-1 (emitting) or t (epsilon) */
  int32_t dst_state;
  int32_t ilabel;
  int32_t olabel;
  float graph_cost;     /* arc weight */
  float ac_cost;        /* -loglike[t-1][ilabel-1]; 0 for epsilon links */
  float fwd_cost;       /* x: cost offered to the destination token */
  float extra;          /* extra cost of the link (<= lattice_beam) */
  double posterior;
} wd_lat_arc;

/* One lattice node: an endpoint of a kept link, or the start token. Sorted by
 * (t, state). */
typedef struct {
  int32_t t;
  int32_t state;
  float cost;           /* Viterbi forward cost */
  float extra;          /* node extra cost */
} wd_lat_node;

/* One surviving token (WD_FLAG_DEBUG). Sorted by (t, state). */
typedef struct {
  int32_t t;
  int32_t state;
  float cost;
  uint32_t pred_arc;    /* 0xffffffff for the start token */
} wd_token;

typedef struct {
  int32_t frames;
  int32_t final_reached;     /* 1 if final weights were used at the last frame */
  int64_t arcs_expanded;     /* emitting out-arcs of every surviving token plus the
                                epsilon out-arcs of every token in the epsilon closure */
  int64_t tokens;            /* surviving tokens summed over frames */
  int64_t max_tokens;        /* largest surviving set of one frame */
  int64_t raw_links;         /* lattice links recorded before pruning */
  int64_t kept_links;
  int64_t nodes;             /* lattice nodes returned */
  int64_t eps_arcs_expanded; /* the epsilon part of arcs_expanded */
  float forward_ms;          /* WD_FLAG_TIMING: token-passing kernel time(s) */
  float lattice_ms;          /* WD_FLAG_TIMING: lattice kernel time(s) */
  wd_caps needed;            /* capacities this decode needed (also on WD_ECAPACITY) */
} wd_stats;

typedef struct wd_result wd_result;

/* ---- graph ------------------------------------------------------------ */

/* Validate `d` (CSR shape, labels, weights, acyclic epsilon arcs) and return
 * the device bytes wd_graph_load needs in *bytes.  WD_EINVAL / WD_ECYCLE.
 * Epsilon depth limit: the epsilon closure runs one pass per epsilon level
 * (the longest epsilon path into a state; the paper leaves epsilon handling
 * open), and a level is stored in one byte, so every state that HAS epsilon
 * out-arcs must sit at level <= 253 (a chain of at most 254 epsilon arcs);
 * a deeper graph is rejected with WD_EINVAL (message "epsilon chains deeper
 * than 254") although its decode would be defined.  States reached by longer
 * chains but without epsilon arcs of their own are accepted. */
wd_status wd_graph_bytes(const wd_graph_desc* d, size_t* bytes);

/* Lay the graph out in `dev_buf` (device, >= wd_graph_bytes, 256-byte
 * aligned, owned by the caller, must outlive the handle) on `stream`, and
 * return a host handle in *out.  The graph stays resident in GPU memory
 * (Sec. 4.3 decodes graphs held entirely in GPU memory).  Synchronous. */
wd_status wd_graph_load(const wd_graph_desc* d, void* dev_buf, size_t dev_bytes, void* stream,
                        wd_graph** out);

/* Frees the host handle only; the caller frees dev_buf. */
void wd_graph_free(wd_graph* g);

/* Number of epsilon levels (longest epsilon chain + 1, 0 without epsilon arcs). */
int32_t wd_graph_eps_levels(const wd_graph* g);

/* Epsilon paths in the graph's path table: every path of one or more
 * epsilon arcs out of every state, enumerated at load (with their weights
 * and last arcs) so that the one-workgroup epsilon closure relaxes all
 * levels in one round (see WD_FLAG_EPS_LEVELS); 0 when the graph has no
 * epsilon arcs, more than 2^27 such paths or one longer than 16 arcs (the
 * closure then goes level by level).  The table takes 16 + 4 * (longest
 * path - 1) bytes per path of device memory (part of wd_graph_bytes; the
 * first path of each state sits beside its arc offsets). */
int64_t wd_graph_eps_paths(const wd_graph* g);

/* ---- decoding --------------------------------------------------------- */

/* Device workspace bytes for decoding `lanes` utterances of at most `max_T`
 * frames each with capacities `caps` (NULL or zero fields: defaults derived
 * from the graph, max_T and p).  *caps_out (may be NULL) receives the
 * capacities the layout uses. */
wd_status wd_workspace_bytes(const wd_graph* g, int32_t lanes, int32_t max_T, const wd_params* p,
                             const wd_caps* caps, size_t* bytes, wd_caps* caps_out);

/* Decode one utterance.  loglikes: device, T x P row-major fp32 with
 * P = num_pdfs of the graph; values must not be NaN or +inf and must be
 * <= 1e30 (-inf marks an impossible pdf).  ws: device workspace of
 * ws_bytes >= wd_workspace_bytes(g, 1, T, p, caps).  On WD_OK or
 * WD_ECAPACITY, *out receives a host result to free with wd_result_free. */
wd_status wd_decode(const wd_graph* g, const float* loglikes, int32_t T, const wd_params* p,
                    const wd_caps* caps, void* ws, size_t ws_bytes, void* stream, wd_result** out);

/* Decode B independent utterances concurrently against one graph (sequence
 * parallelism, Sec. 4.2, done as in-process lanes).  loglikes[i] is a device
 * pointer to T[i] x P fp32.  out[i] receives utterance i's result (lane i
 * equals wd_decode of utterance i, bit for bit).  The status is the first
 * non-OK lane status, else WD_OK; every out[i] is filled whenever it is
 * WD_OK or WD_ECAPACITY for that lane. */
wd_status wd_decode_batch(const wd_graph* g, int32_t B, const float* const* loglikes,
                          const int32_t* T, const wd_params* p, const wd_caps* caps, void* ws,
                          size_t ws_bytes, void* stream, wd_result** out);

/* ---- decoding without allocation -------------------------------------- */

/* For callers that cannot allocate device memory (code that must not call
 * hipMalloc, e.g. under HIP graph capture, in tight serving loops, or in
 * harnesses that forbid it): wd_decode of one utterance in one-workgroup
 * mode whose workspace is a fixed device array inside the library,
 * WD_NOALLOC_SCRATCH_BYTES on every device the library runs on (held until
 * the process ends), and whose results go into the caller's host buffers.
 * It calls no hipMalloc, hipFree or other allocating routine, and creates no
 * stream or event.
 *  - p->flags: 0 or WD_FLAG_ONE_WORKGROUP only (debug, timing, profile and
 *    chip-wide flags: WD_EINVAL; with max_active 0 or >= WD_CHIP_WIDE_MAX_ACTIVE
 *    WD_FLAG_ONE_WORKGROUP must be set).  caps as for wd_workspace_bytes.
 *  - WD_EINVAL, before any device work, when the workspace these
 *    capacities need (wd_workspace_bytes with lanes = 1) exceeds the scratch;
 *    the per-state arrays take 16.5 bytes per graph state, so graphs beyond
 *    ~15M states do not fit.
 *  - Outputs (host memory, caller-owned): *cost, words[words_cap] with the
 *    count in *n_words, links[links_cap] (sorted by (t, arc_id)) and
 *    nodes[nodes_cap] (sorted by (t, state)) with their counts in
 *    stats->kept_links and stats->nodes, and *stats (forward_ms/lattice_ms 0).
 *    WD_ECAPACITY when the workspace capacities or an output buffer were too
 *    small; *n_words and *stats (its `needed` capacities, kept_links, nodes)
 *    then say what is needed.
 *  - Synchronous on `stream`.  Every call on a device uses the same scratch,
 *    which keeps the last call's contents: calls that overlap on one device
 *    (other threads, other streams) race and must not be issued. */
#define WD_NOALLOC_SCRATCH_BYTES (256u << 20)
wd_status wd_decode_noalloc(const wd_graph* g, const float* loglikes, int32_t T, const wd_params* p,
                            const wd_caps* caps, void* stream, float* cost, int32_t* words, int32_t words_cap,
                            int32_t* n_words, wd_lat_arc* links, int64_t links_cap, wd_lat_node* nodes,
                            int64_t nodes_cap, wd_stats* stats);

/* ---- streaming -------------------------------------------------------- */

/* Frame-synchronous decoding as the log-likelihoods arrive, e.g. chunk by
 * chunk from an acoustic model on the same stream (the paper's closing
 * sections name the integration of acoustic inference with decoding on the
 * GPU as future work).  The result equals wd_decode_batch of the complete
 * utterances, bit for bit.
 *
 * wd_stream_begin: B utterances of at most max_T frames each.  frames[i] is
 * utterance i's frame store: device, max_T x P fp32 row-major, owned by the
 * caller and valid until wd_stream_end/free returns; row t-1 holds frame t.
 * A row must be written (on `stream`, or before) before the advance that
 * covers it and left unchanged afterwards.  ws: as for wd_decode_batch with
 * (B, max_T).  Chip-wide mode (see the mode flags) takes B = 1.  The decoder
 * carries each utterance's frontier and counters in the workspace between
 * launches.  *out receives the stream handle.
 *
 * wd_stream_advance: n_frames[i] >= 0 more rows of utterance i are ready;
 * decodes them (asynchronously on `stream`: the call only enqueues work).
 * WD_EINVAL if a count would pass max_T.  Decoding errors (invalid values,
 * no surviving token, capacity) are reported by wd_stream_end.
 *
 * wd_stream_end: the utterances end after the frames received; final costs,
 * lattice pruning and posteriors as in wd_decode_batch, whose status and
 * out[i] rules apply.  Synchronises and frees the handle.
 *
 * wd_stream_free: abandons a stream (waits for its work, frees the handle). */
typedef struct wd_stream wd_stream;
wd_status wd_stream_begin(const wd_graph* g, int32_t B, const float* const* frames, int32_t max_T,
                          const wd_params* p, const wd_caps* caps, void* ws, size_t ws_bytes, void* stream,
                          wd_stream** out);
wd_status wd_stream_advance(wd_stream* s, const int32_t* n_frames);
wd_status wd_stream_end(wd_stream* s, wd_result** out);
void      wd_stream_free(wd_stream* s);

/* ---- lattice determinisation (host) ----------------------------------- */

/* The compact "exact lattice" (Sec. 3.4, after Povey et al. 2012) of a pruned
 * state-level lattice, computed on the CPU as the paper does after the copy
 * to the host.  Input: the links and nodes of a result (wd_result_lattice,
 * wd_result_nodes: nodes sorted by (t, state); a link runs from node
 * (t-1, src_state) if ilabel != 0, else (t, src_state), to (t, dst_state)),
 * the start state (its node at t = 0 starts every path), and node_final[i],
 * the final graph cost of node i (+inf: not final; NULL: the nodes of the
 * last frame, cost 0).  A path's weight is the pair (sum of graph costs, sum
 * of acoustic costs), in double; its string is the ilabels of its emitting
 * links in order; its words are its nonzero olabels.
 * Output: a lattice deterministic on words (state 0 starts; no arc has word
 * 0; arcs sorted by (source state, word)) with exactly one path per word
 * sequence of the input; that path's weight and string are those of the best
 * input path with the same words (best: lower graph + acoustic total, then
 * the lexicographically smaller string, then the lower graph cost).  An arc's
 * alignment is its part of the path's string; a final state's alignment
 * ends it.  beam (>= 0, +inf: none) prunes inside the construction: output
 * states are built best first (forward cost plus the exact best completion
 * of their lattice nodes) and a state whose best complete path costs more
 * than the lattice's best path plus beam is not built, and the subsets
 * leave out lattice nodes that no path within the beam crosses.  Every word
 * sequence within the beam is then kept, with its exact best path; a
 * sequence beyond it may be kept too, with some path of its words beyond
 * the beam.  State numbers follow the construction order.  WD_EINVAL for unsorted nodes,
 * dangling links, a cycle or a negative or NaN beam; WD_ECAPACITY beyond
 * max_states output states (<= 0: 4M).  Residual weights are kept in double;
 * output states whose residuals differ in their last bits are not merged
 * (the lattice stays deterministic and exact). */
typedef struct {
  int32_t src, dst;
  int32_t word;         /* olabel, never 0 */
  int32_t align_len;
  double graph_cost, ac_cost;
  int64_t align_off;    /* into wd_clat_alignment */
} wd_clat_arc;
typedef struct {
  int32_t state;
  int32_t align_len;
  double graph_cost, ac_cost;
  int64_t align_off;
} wd_clat_final;
typedef struct wd_clat wd_clat;
wd_status wd_lattice_determinize(const wd_lat_arc* arcs, int64_t n_arcs, const wd_lat_node* nodes,
                                 int64_t n_nodes, int32_t start_state, const float* node_final,
                                 double beam, int64_t max_states, wd_clat** out);
int32_t wd_clat_states(const wd_clat* c);
int64_t wd_clat_arcs(const wd_clat* c, const wd_clat_arc** arcs);
int64_t wd_clat_finals(const wd_clat* c, const wd_clat_final** finals);
int64_t wd_clat_alignment(const wd_clat* c, const int32_t** labels);
void    wd_clat_free(wd_clat* c);

/* ---- results (host memory owned by the result) ------------------------ */

wd_status wd_result_status(const wd_result* r);
float   wd_result_cost(const wd_result* r);
int32_t wd_result_words(const wd_result* r, const int32_t** words);
int64_t wd_result_lattice(const wd_result* r, const wd_lat_arc** arcs);
int64_t wd_result_nodes(const wd_result* r, const wd_lat_node** nodes);
int64_t wd_result_tokens(const wd_result* r, const wd_token** toks);          /* WD_FLAG_DEBUG */
int64_t wd_result_raw_lattice(const wd_result* r, const wd_lat_arc** arcs);    /* WD_FLAG_DEBUG */
/* WD_FLAG_DEBUG: per frame t = 0..T the best cost after the emitting step,
 * the beam cutoff and the final cutoff; returns T+1. */
int32_t wd_result_cutoffs(const wd_result* r, const float** best, const float** cutoff_beam,
                          const float** cutoff);
/* WD_FLAG_PHASES: per decoded frame t = 0..T (streams: every frame) the
 * WD_PHASE_SLOTS words above, frame after frame, in *stamps; *tick_hz (may be
 * NULL) receives the stamps' clock rate.  Returns the number of frames (0
 * without the flag). */
int32_t wd_result_phases(const wd_result* r, const uint64_t** stamps, double* tick_hz);
/* WD_FLAG_PHASES: the lattice pass's WD_LATTICE_PHASE_STAMPS wall-clock
 * stamps (same clock as wd_result_phases); returns their number, 0 without
 * the flag. */
int32_t wd_result_lattice_phases(const wd_result* r, const uint64_t** stamps);
void    wd_result_stats(const wd_result* r, wd_stats* s);
void    wd_result_free(wd_result* r);

/* Message for the last non-OK status returned on this thread. */
const char* wd_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* WFSTDEC_H */
