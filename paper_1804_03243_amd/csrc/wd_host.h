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
void launch_lattice(const DevGraph& g, const LaneDesc* lanes, int B, const Params& prm, hipStream_t s);
size_t grid_lane_bytes();
// `prune`: incremental lattice pruning on the library's pruning stream of the
// current device (ordered against `s` by events).  Fails only on a HIP error
// of that stream or its events.
wd_status launch_grid_forward(const DevGraph& g, const LaneDesc* lanes, void* grid, int B, const Params& prm,
                              bool prune, const uint32_t* bad, int maxT, hipStream_t s);
void launch_grid_sweep(const DevGraph& g, const LaneDesc* lanes, void* grid, int B, int maxT, float lattice_beam,
                       hipStream_t s);
void launch_grid_nodes(const LaneDesc* lanes, void* grid, int B, hipStream_t s);
void launch_check_loglikes(const LaneDesc* lanes, int B, uint32_t P, uint32_t* bad, hipStream_t s);
void launch_fill_u64(unsigned long long* p, uint64_t n, unsigned long long v, hipStream_t s);
void launch_fill_u32(uint32_t* p, uint64_t n, uint32_t v, hipStream_t s);

inline uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

}  // namespace wd
