// Library context: registration, schedule, pool, arena, streams and the
// compiled step program.
#pragma once

#include <hip/hip_runtime.h>

#include <string>
#include <vector>

#include "internal.h"

namespace ooc {

// A piece of a staged copy (see Copy::staged): bytes [off, off + bytes) of
// the variable, moved through staging slot seq mod the slot count.
struct Piece {
  uint64_t off, bytes;
  int32_t ev_start, ev_done;    // the first piece's ev_start and the last one's ev_done
  int64_t seq;                  // are the copy's; seq numbers the pieces of one direction
};

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
  // A variable whose host home is pageable memory is copied in pieces through
  // pinned staging slots; host threads move each piece between its slot and
  // the pageable home.  gen: a swap-out writes the variable's gen-th host
  // copy of the step; a swap-in needs its gen-th copy.
  bool staged = false;
  int64_t gen = 0;
  std::vector<Piece> pieces;
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
  mutable std::string err;                // message of the last failing call
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
  uint64_t host_limit = OOC_UNLIMITED;     // see ooc_set_host_limit
  int32_t layout = OOC_LAYOUT_POOL;        // see ooc_set_layout
  bool incore = true;

  ooc::Schedule sched;
  ooc::Plan plan;

  // device resources
  std::vector<hipMemGenericAllocationHandle_t> chunks;
  void* va_base = nullptr;
  uint64_t va_bytes = 0;
  std::vector<char*> iv_ptr;              // per interval: start of its virtual range
  // OOC_LAYOUT_BESTFIT: one allocation; each interval at its offset in it
  std::vector<uint64_t> iv_off;
  uint64_t heap_extent = 0;
  void* heap = nullptr;
  std::vector<int64_t> resident;          // in-core mode: per variable, its resident interval
  char* arena = nullptr;
  uint64_t arena_bytes = 0;
  std::vector<char*> host_slot;           // per variable, or nullptr
  // pageable overflow of the host arena (TEMP homes beyond the host limit)
  char* spill = nullptr;
  uint64_t spill_bytes = 0;
  char* stage_in = nullptr;               // pinned staging slots, inside the arena
  char* stage_out = nullptr;
  std::vector<const ooc::Copy*> in_copy, out_copy;   // per staged piece seq: its copy
  std::vector<int32_t> in_piece, out_piece;          // and the piece's index in it
  uint64_t staged_h2d = 0, staged_d2h = 0;
  hipStream_t cs = nullptr, hs = nullptr, ds = nullptr;
  hipStream_t ss = nullptr;               // staged swap-ins (pageable homes)
  std::vector<hipEvent_t> events;
  std::vector<int8_t> event_stream;       // 0 compute, 1 h2d, 2 d2h, 3 staged h2d
  std::vector<int64_t> ev_staged_in;      // per event: the staged swap-in it completes, or -1
  std::vector<ooc::FnProgram> prog;
  int32_t ev_begin = -1, ev_end = -1;
  int64_t loss_var = -1;
  uint64_t prog_h2d = 0, prog_d2h = 0;

  ooc_stats stats{};
  std::vector<double> fn_ms;              // last step, per function
};
