// Internal structures of the out-of-core training library.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/ooc.h"

namespace ooc {

enum State : uint8_t { UNMAT = 0, HOST = 1, DEV = 2, PEND = 3 };

struct Var {
  uint64_t bytes;
  int32_t kind;
};

struct FnVar {
  int64_t var;
  uint8_t access;
};

struct Fn {
  int32_t op;
  std::vector<FnVar> vars;      // merged: first position kept, accesses or-ed
  std::vector<int64_t> attrs;
};

struct Op {
  int32_t fn;
  uint8_t phase;
  uint8_t kind;
  int64_t var;
  uint64_t held;
};

struct Schedule {
  std::vector<Op> ops;
  std::vector<int64_t> windows;
  uint64_t peak = 0, h2d = 0, d2h = 0;
};

// Residency interval: one device copy of one variable (Section 4: one
// virtual range per allocation request).
struct Interval {
  int64_t var;
  int64_t open;    // op index, -1 = resident for the whole step
  int64_t close;   // op index, -1 = never closed
  std::vector<int32_t> chunks;
};

struct Plan {
  std::vector<Interval> intervals;
  std::vector<int64_t> op_interval;   // per op: the interval it opens / closes / touches (-1)
  uint64_t max_chunks_used = 0;
  uint64_t n_chunks = 0;              // chunks the pool must own
};

// The plan's intervals served by one contiguous best-fit heap (the allocator
// the chunk pool is compared with): highest address used and peak live bytes.
void bestfit_extent(const std::vector<Var>& vars, const Plan& plan, uint64_t align,
                    uint64_t* extent, uint64_t* peak_live,
                    std::vector<uint64_t>* offsets = nullptr);
// Lays the plan's intervals out in that heap: offsets per interval, the heap's
// extent, and each interval's chunk list replaced by the heap segments it
// covers (the heap cut at every interval boundary).
void bestfit_layout(const std::vector<Var>& vars, uint64_t align, Plan* plan,
                    std::vector<uint64_t>* offsets, uint64_t* extent);
// Scheduler (Section 3, Fig. 2).  Returns OOC_OK, OOC_E_INFEASIBLE.  With
// ahead >= 0 the fixed-distance rule of LMS (Section 2) replaces the byte
// window: the window ends with f_{i+ahead} and a variable whose next use is
// at most `threshold` functions away is kept.  wait_order: OOC_WAIT_OLDEST or
// OOC_WAIT_FURTHEST (which pending swap-out a budget wait completes).
ooc_status build_schedule(const std::vector<Var>& vars, const std::vector<Fn>& fns,
                          uint64_t budget, uint64_t window, uint64_t chunk, int policy,
                          Schedule* out, std::string* err, int64_t ahead = -1,
                          int64_t threshold = -1, int wait_order = OOC_WAIT_OLDEST);
// In-core plan: persistent variables resident for the whole step, TEMPs from
// first to last use, no transfers.
void build_incore(const std::vector<Var>& vars, const std::vector<Fn>& fns, uint64_t chunk,
                  Schedule* out);
uint64_t incore_peak(const std::vector<Var>& vars, const std::vector<Fn>& fns, uint64_t chunk);
uint64_t working_set_max(const std::vector<Var>& vars, const std::vector<Fn>& fns,
                         uint64_t chunk);
// Chunk plan: replays the schedule through the pool (freed chunks reused in the order
// they were freed; a new chunk only when none is free).
void build_plan(const std::vector<Var>& vars, const Schedule& s, bool incore, uint64_t chunk,
                Plan* out);

// Function-sequence rules and operation signatures; returns "" when valid.
std::string check_fn(const std::vector<Var>& vars, const Fn& fn);

inline uint64_t round_up(uint64_t b, uint64_t c) { return (b + c - 1) / c * c; }

}  // namespace ooc
