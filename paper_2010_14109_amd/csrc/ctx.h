// Library context: registration, schedule, pool, arena, streams and the
// compiled step program.
#pragma once

#include <hip/hip_runtime.h>

#include <string>
#include <vector>

#include "internal.h"

namespace ooc {

// One host<->device copy of the step program (addresses resolved once the
// host arena exists).
struct Copy {
  int64_t var;
  int64_t iv;                   // device interval copied to or from
  void* dst;
  const void* src;
  uint64_t bytes;
  std::vector<int32_t> waits;   // event ids the copy stream waits for first
  int32_t ev_start, ev_done;
};

// What the executor does around function f_i.
struct FnProgram {
  std::vector<Copy> h2d;        // swap-ins issued in f_i's PRE phase
  std::vector<int32_t> cwaits;  // compute stream waits before f_i's kernels
  std::vector<void*> ptrs;      // device address of each of f_i's variables
  std::vector<uint64_t> sizes;  // and its size in bytes
  std::vector<Copy> d2h;        // swap-outs issued in f_i's POST phase
  int32_t ev_pre, ev_fn;        // compute stream, around f_i's kernels
};

enum Stage { REGISTERING = 0, BUILT = 1, PREPARED = 2 };

}  // namespace ooc

struct ooc_ctx {
  int32_t device = -1;
  std::string err;
  ooc::Stage stage = ooc::REGISTERING;

  std::vector<ooc::Var> vars;
  std::vector<ooc::Fn> fns;
  std::vector<uint8_t> produced;   // a value exists for the variable at this point of the sequence

  uint64_t budget = OOC_UNLIMITED;
  uint64_t window = 0;
  int64_t ahead = -1, threshold = -1;     // fixed-distance rule when ahead >= 0
  bool window_set = false;
  uint64_t chunk = 2ull << 20;
  int32_t policy = OOC_POLICY_CANCEL;
  int32_t wait_order = OOC_WAIT_OLDEST;    // see ooc_set_wait_order
  int64_t swapout_depth = 4;               // see ooc_set_swapout_depth
  bool incore = true;

  ooc::Schedule sched;
  ooc::Plan plan;

  // device resources
  std::vector<hipMemGenericAllocationHandle_t> chunks;
  void* va_base = nullptr;
  uint64_t va_bytes = 0;
  std::vector<char*> iv_ptr;              // per interval: start of its virtual range
  std::vector<int64_t> resident;          // in-core mode: per variable, its resident interval
  char* arena = nullptr;
  uint64_t arena_bytes = 0;
  std::vector<char*> host_slot;           // per variable, or nullptr
  hipStream_t cs = nullptr, hs = nullptr, ds = nullptr;
  std::vector<hipEvent_t> events;
  std::vector<int8_t> event_stream;       // 0 compute, 1 h2d, 2 d2h
  std::vector<ooc::FnProgram> prog;
  int32_t ev_begin = -1, ev_end = -1;
  int64_t loss_var = -1;
  uint64_t prog_h2d = 0, prog_d2h = 0;

  ooc_stats stats{};
  std::vector<double> fn_ms;              // last step, per function
};
