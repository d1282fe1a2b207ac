// Host-side declarations shared by the library's translation units.
#pragma once

#include <string>
#include <vector>

#include "../../include/wfstdec.h"
#include "wd_common.h"

struct wd_graph {
  wd::DevGraph dg;
  int32_t S = 0;
  int64_t A = 0;
  uint64_t Ae = 0, Ax = 0;
  uint32_t nlevels = 0;
  uint32_t P = 0;
  std::vector<uint32_t> level_base;  // host copy, nlevels + 1 entries
  size_t bytes = 0;
};

namespace wd {

void set_error(const std::string& msg);
wd_status fail(wd_status st, const std::string& msg);
wd_status hip_check(hipError_t e, const char* what);

void launch_forward(const DevGraph& g, const LaneDesc* lanes, int B, const Params& prm,
                    const uint32_t* bad, hipStream_t s);
// Lattice links of one-workgroup decodes, from the node store, after the
// forward pass (all frames at once); before launch_lattice.
void launch_links(const DevGraph& g, const LaneDesc* lanes, int B, hipStream_t s);
void launch_lattice(const DevGraph& g, const LaneDesc* lanes, int B, const Params& prm, hipStream_t s);
size_t grid_lane_bytes();
// Raw window slots of the link store with incremental pruning.
uint32_t grid_window_slots();
// Chip-wide forward pass in three steps, so that a stream can decode frames as
// they arrive: begin (per-utterance state; with `prune`, incremental lattice
// pruning on the library's pruning stream of the current device, ordered
// against `s` by the run's events), frames t_from..t_to (any number of calls,
// in order), end.  Errors are HIP errors of the pruning stream or its events.
// grid_release frees the events (after waiting for the pruning stream if the
// run did not reach grid_end).
struct GridRun {
  hipStream_t q = nullptr;  // pruning stream, or nullptr
  hipEvent_t ready[4] = {}, done[4] = {};
  int nwin = 0;             // windows handed to the pruning stream
  bool ended = false;       // grid_end made the decoding stream wait for them
};
wd_status grid_begin(GridRun* run, const LaneDesc* lanes, void* grid, int B, bool prune, const uint32_t* bad,
                     hipStream_t s);
wd_status grid_frames(GridRun* run, const DevGraph& g, const LaneDesc* lanes, void* grid, int B, const Params& prm,
                      const uint32_t* bad, int t_from, int t_to, hipStream_t s);
wd_status grid_end(GridRun* run, const LaneDesc* lanes, void* grid, int B, hipStream_t s);
void grid_release(GridRun* run);
void launch_grid_sweep(const DevGraph& g, const LaneDesc* lanes, void* grid, int B, int maxT, float lattice_beam,
                       hipStream_t s);
void launch_grid_nodes(const LaneDesc* lanes, void* grid, int B, hipStream_t s);
void launch_check_loglikes(const LaneDesc* lanes, int B, uint32_t P, uint32_t* bad, hipStream_t s);
// Packs the links, nodes and words of every finished lane into dst (device),
// lane after lane, each lane's part 16-byte aligned.
void launch_pack_results(const LaneDesc* lanes, int B, void* dst, hipStream_t s);
// Sets T, t0 and open of lanes[0..B) (streaming) from host values passed as
// kernel arguments.
void launch_set_frames(LaneDesc* lanes, int B, const int32_t* T, const int32_t* t0, int32_t open, hipStream_t s);
void launch_fill_u64(unsigned long long* p, uint64_t n, unsigned long long v, hipStream_t s);
void launch_fill_u32(uint32_t* p, uint64_t n, uint32_t v, hipStream_t s);

inline uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

}  // namespace wd
