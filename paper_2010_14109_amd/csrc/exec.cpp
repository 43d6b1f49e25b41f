// Executor: builds the virtual-address pool and the pinned host arena, turns
// the schedule into a stream program, and runs one training step.
//
// Pool (Section 4).  The pool owns exactly as many physical chunks of m_c
// bytes as the plan ever has in use (never more than budget / m_c).  Every
// residency interval -- one device copy of one variable -- gets its own
// contiguous virtual range, onto which its chunks are mapped in plan order.
// The schedule is fixed, so all ranges are reserved and mapped once, here;
// a step only looks up addresses.  A chunk may therefore be mapped at several
// virtual addresses, one per interval that uses it at some time.
//
// Streams.  Kernels run on the compute stream; swap-ins on the h2d stream,
// swap-outs on the d2h stream.  Events order them:
//  * a kernel waits for the swap-in of each variable it reads;
//  * a swap-out waits for the function after which it was reserved;
//  * whoever first writes an interval (its swap-in copy, or the first kernel
//    using an allocated one) waits until every interval that used the same
//    chunks before is released: its last kernel finished and its last
//    swap-out copy completed (the device-side form of step (b) of Section 3,
//    which completes the oldest swap-outs before f_i runs);
//  * a swap-in waits for the last swap-out copy into the same host slot.
// Two kinds of swap-out need no copy and are not issued: one that is later
// cancelled (its host copy is never read: the variable is kept on the device
// and any later swap-out writes a newer copy) and one of a variable whose
// host copy is still current (not written since it was swapped in).
#include <sys/mman.h>

#include <algorithm>
#include <chrono>
#include <condition_variable>
#include <cstdio>
#include <cstring>
#include <functional>
#include <mutex>
#include <queue>
#include <set>
#include <thread>

#include "ctx.h"
#include "kernels.h"

namespace ooc {

static const uint64_t kSlotAlign = 4096;
// Pageable overflow (see ooc_set_host_limit): pieces of at most kPiece bytes
// move through kSlots pinned staging slots per direction, copied between slot
// and pageable home by kThreads host threads per direction.
static const uint64_t kPiece = 32ull << 20;
static const int64_t kSlots = 32;
static const int kThreads = 8;

#define HIPCK(call)                                                               \
  do {                                                                            \
    hipError_t e_ = (call);                                                       \
    if (e_ != hipSuccess) {                                                       \
      ctx->err = std::string(#call) + " failed: " + hipGetErrorString(e_);        \
      return OOC_E_DEVICE;                                                        \
    }                                                                             \
  } while (0)

void release_device(ooc_ctx* ctx) {
  if (ctx->device < 0) return;
  // teardown: an error here cannot be acted on, and every resource is released regardless
  (void)hipSetDevice(ctx->device);
  if (ctx->cs) (void)hipStreamSynchronize(ctx->cs);
  if (ctx->hs) (void)hipStreamSynchronize(ctx->hs);
  if (ctx->ds) (void)hipStreamSynchronize(ctx->ds);
  if (ctx->ss) (void)hipStreamSynchronize(ctx->ss);
  for (hipEvent_t e : ctx->events) (void)hipEventDestroy(e);
  ctx->events.clear();
  if (ctx->cs) (void)hipStreamDestroy(ctx->cs);
  if (ctx->hs) (void)hipStreamDestroy(ctx->hs);
  if (ctx->ds) (void)hipStreamDestroy(ctx->ds);
  if (ctx->ss) (void)hipStreamDestroy(ctx->ss);
  ctx->cs = ctx->hs = ctx->ds = ctx->ss = nullptr;
  if (ctx->heap) (void)hipFree(ctx->heap);
  ctx->heap = nullptr;
  if (ctx->va_base) {
    (void)hipMemUnmap(ctx->va_base, ctx->va_bytes);
    (void)hipMemAddressFree(ctx->va_base, ctx->va_bytes);
    ctx->va_base = nullptr;
  }
  for (auto h : ctx->chunks) (void)hipMemRelease(h);
  ctx->chunks.clear();
  if (ctx->arena) (void)hipHostFree(ctx->arena);
  ctx->arena = nullptr;
  if (ctx->spill) munmap(ctx->spill, ctx->spill_bytes);
  ctx->spill = nullptr;
  ctx->spill_bytes = 0;
}

// Entries of the process memory-map table still free (-1 if unknown).
static int64_t map_entries_left() {
  FILE* f = std::fopen("/proc/sys/vm/max_map_count", "r");
  if (!f) return -1;
  long long limit = -1;
  if (std::fscanf(f, "%lld", &limit) != 1) limit = -1;
  std::fclose(f);
  if (limit < 0) return -1;
  f = std::fopen("/proc/self/maps", "r");
  if (!f) return -1;
  int64_t used = 0;
  for (int c; (c = std::fgetc(f)) != EOF;)
    if (c == '\n') ++used;
  std::fclose(f);
  return limit - used;
}

static int32_t new_event(ooc_ctx* ctx, int8_t stream) {
  ctx->event_stream.push_back(stream);
  return (int32_t)ctx->event_stream.size() - 1;
}

// Turns the schedule and the chunk plan into per-function stream programs.
static ooc_status compile(ooc_ctx* ctx) {
  const auto& ops = ctx->sched.ops;
  const auto& plan = ctx->plan;
  const int64_t N = (int64_t)ctx->fns.size();
  const int64_t NI = (int64_t)plan.intervals.size();
  const int64_t nv = (int64_t)ctx->vars.size();
  ctx->prog.assign(N, FnProgram{});
  ctx->event_stream.clear();
  ctx->ev_begin = new_event(ctx, 0);
  for (int64_t i = 0; i < N; ++i) {
    ctx->prog[i].ev_pre = new_event(ctx, 0);
    ctx->prog[i].ev_fn = new_event(ctx, 0);
  }
  ctx->ev_end = new_event(ctx, 0);

  // swap-outs that a later CANCEL undoes
  std::vector<uint8_t> cancelled(ops.size(), 0);
  {
    std::vector<int64_t> pend_op(nv, -1);
    for (int64_t k = 0; k < (int64_t)ops.size(); ++k) {
      if (ops[k].kind == OOC_SWAPOUT) pend_op[ops[k].var] = k;
      if (ops[k].kind == OOC_CANCEL && pend_op[ops[k].var] >= 0) {
        cancelled[pend_op[ops[k].var]] = 1;
        pend_op[ops[k].var] = -1;
      }
      if (ops[k].kind == OOC_WAIT_OUT) pend_op[ops[k].var] = -1;
    }
  }

  std::vector<int64_t> working(nv, -1);
  std::vector<uint8_t> acquired(NI, 0), host_valid(nv, 0);
  std::vector<int64_t> last_fn(NI, -1), last_d2h(NI, -1), in_ev(NI, -1), var_d2h(nv, -1);
  std::vector<std::vector<int32_t>> release(NI), preds(NI);
  std::vector<int64_t> owner(plan.n_chunks, -1);
  for (int64_t v = 0; v < nv; ++v)
    host_valid[v] = ctx->vars[v].kind == OOC_INPUT || ctx->vars[v].kind == OOC_PARAM ||
                    ctx->vars[v].kind == OOC_STATE;

  auto opened = [&](int64_t J) {
    std::set<int64_t> ps;
    for (int32_t c : plan.intervals[J].chunks) {
      if (owner[c] >= 0) ps.insert(owner[c]);
      owner[c] = J;
    }
    for (int64_t p : ps)
      for (int32_t e : release[p]) preds[J].push_back(e);
  };
  auto closed = [&](int64_t J) {
    release[J].clear();
    if (last_fn[J] >= 0) release[J].push_back(ctx->prog[last_fn[J]].ev_fn);
    if (last_d2h[J] >= 0) release[J].push_back((int32_t)last_d2h[J]);
    if (in_ev[J] >= 0) release[J].push_back((int32_t)in_ev[J]);   // its swap-in copy, if unused
  };
  auto add_waits = [&](std::vector<int32_t>* w, const std::vector<int32_t>& evs, int8_t stream) {
    for (int32_t e : evs)
      if (ctx->event_stream[e] != stream) w->push_back(e);
  };
  // in-core mode: persistent variables are resident from the start
  ctx->resident.assign(nv, -1);
  for (int64_t J = 0; J < NI; ++J)
    if (plan.intervals[J].open < 0) {
      opened(J);
      acquired[J] = 1;
      working[plan.intervals[J].var] = J;
      ctx->resident[plan.intervals[J].var] = J;
    }

  ctx->prog_h2d = ctx->prog_d2h = 0;
  int64_t k = 0;
  const int64_t K = (int64_t)ops.size();
  for (int64_t i = 0; i <= N; ++i) {
    // PRE ops of f_i (END ops when i == N)
    while (k < K && ops[k].fn == i && ops[k].phase != OOC_POST) {
      const Op& o = ops[k];
      const int64_t J = plan.op_interval[k];
      switch (o.kind) {
        case OOC_SWAPIN: {
          opened(J);
          working[o.var] = J;
          Copy c{o.var, J, nullptr, nullptr, ctx->vars[o.var].bytes, {}, 0, 0};
          // every release event, same stream included: a swap-in whose variable ends up with
          // a pageable home moves to the staged stream
          add_waits(&c.waits, preds[J], -1);
          if (var_d2h[o.var] >= 0) add_waits(&c.waits, {(int32_t)var_d2h[o.var]}, -1);
          c.ev_start = new_event(ctx, 1);
          c.ev_done = new_event(ctx, 1);
          in_ev[J] = c.ev_done;
          ctx->prog_h2d += c.bytes;
          ctx->prog[i].h2d.push_back(std::move(c));
          break;
        }
        case OOC_ALLOC:
          opened(J);
          working[o.var] = J;
          break;
        case OOC_CANCEL:
          working[o.var] = J;
          break;
        case OOC_WAIT_OUT:
        case OOC_FREE:
          closed(J);
          break;
      }
      ++k;
    }
    if (i == N) break;
    // f_i's kernels
    FnProgram& fp = ctx->prog[i];
    for (const FnVar& fv : ctx->fns[i].vars) {
      const int64_t J = working[fv.var];
      if (J < 0) {
        ctx->err = "schedule leaves variable " + std::to_string(fv.var) + " of function " +
                   std::to_string(i) + " off the device";
        return OOC_E_INVALID;
      }
      if (!acquired[J]) {
        if (in_ev[J] >= 0)
          add_waits(&fp.cwaits, {(int32_t)in_ev[J]}, 0);
        else
          add_waits(&fp.cwaits, preds[J], 0);
        acquired[J] = 1;
      }
      fp.ptrs.push_back(ctx->iv_ptr[J]);
      fp.sizes.push_back(ctx->vars[fv.var].bytes);
      last_fn[J] = i;
      if (fv.access & OOC_W) host_valid[fv.var] = 0;
    }
    // POST ops of f_i
    while (k < K && ops[k].fn == i && ops[k].phase == OOC_POST) {
      const Op& o = ops[k];
      const int64_t J = plan.op_interval[k];
      if (o.kind == OOC_SWAPOUT) {
        working[o.var] = -1;
        if (!cancelled[k] && !host_valid[o.var]) {
          Copy c{o.var, J, nullptr, nullptr, ctx->vars[o.var].bytes, {}, 0, 0};
          c.waits.push_back(fp.ev_fn);
          c.ev_start = new_event(ctx, 2);
          c.ev_done = new_event(ctx, 2);
          last_d2h[J] = c.ev_done;
          var_d2h[o.var] = c.ev_done;
          host_valid[o.var] = 1;
          ctx->prog_d2h += c.bytes;
          fp.d2h.push_back(std::move(c));
        }
      } else if (o.kind == OOC_FREE) {
        working[o.var] = -1;
        closed(J);
      }
      ++k;
    }
  }
  return OOC_OK;
}

// A stream gets its DMA-engine queue from the runtime at its first copy large
// enough for the engine (smaller copies run as a copy kernel instead), and that
// copy blocks the host thread for several milliseconds (measured 6-7 ms on
// each copy stream in the first out-of-core steps).  One such copy each way on
// every copy stream at prepare takes that delay out of the steps.
static ooc_status warm_copy_streams(ooc_ctx* ctx) {
  constexpr size_t kWarm = 8u << 20;
  void* h = nullptr;
  void* d = nullptr;
  // best effort: with no 8 MiB to spare on either side the steps simply pay the delay
  if (hipHostMalloc(&h, kWarm, hipHostMallocDefault) != hipSuccess ||
      hipMalloc(&d, kWarm) != hipSuccess) {
    (void)hipGetLastError();
    if (h) (void)hipHostFree(h);
    return OOC_OK;
  }
  hipError_t e = hipSuccess;
  for (hipStream_t s : {ctx->hs, ctx->ds, ctx->ss}) {
    if (e == hipSuccess) e = hipMemcpyAsync(d, h, kWarm, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(h, d, kWarm, hipMemcpyDeviceToHost, s);
  }
  for (hipStream_t s : {ctx->hs, ctx->ds, ctx->ss})
    if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (d) (void)hipFree(d);
  if (h) (void)hipHostFree(h);
  if (e != hipSuccess) {
    ctx->err = std::string("warm-up copy on the copy streams failed: ") + hipGetErrorString(e);
    return OOC_E_DEVICE;
  }
  return OOC_OK;
}

ooc_status prepare(ooc_ctx* ctx) {
  auto t0 = std::chrono::steady_clock::now();
  HIPCK(hipSetDevice(ctx->device));
  hipMemAllocationProp prop = {};
  prop.type = hipMemAllocationTypePinned;
  prop.location.type = hipMemLocationTypeDevice;
  prop.location.id = ctx->device;
  size_t gran = 0;
  HIPCK(hipMemGetAllocationGranularity(&gran, &prop, hipMemAllocationGranularityMinimum));
  if (gran == 0 || ctx->chunk % gran != 0) {
    ctx->err = "chunk size " + std::to_string(ctx->chunk) +
               " is not a multiple of the allocation granularity " + std::to_string(gran);
    return OOC_E_INVALID;
  }
  size_t free0 = 0, total0 = 0, free1 = 0, total1 = 0;
  HIPCK(hipMemGetInfo(&free0, &total0));

  const Plan& plan = ctx->plan;
  const int64_t NI = (int64_t)plan.intervals.size();
  if (ctx->layout == OOC_LAYOUT_BESTFIT) {
    // the comparison allocator: one contiguous heap, intervals at their best-fit offsets
    HIPCK(hipMalloc(&ctx->heap, std::max<uint64_t>(ctx->heap_extent, 256)));
    ctx->iv_ptr.assign(NI, nullptr);
    for (int64_t J = 0; J < NI; ++J) ctx->iv_ptr[J] = (char*)ctx->heap + ctx->iv_off[J];
    ctx->stats.n_mappings = 0;
  }
  // Every physical chunk and every mapping of a chunk takes one entry of the
  // process's memory-map table (vm.max_map_count); beyond it the driver
  // rejects further access grants.  Refuse plans that cannot fit.
  if (ctx->layout == OOC_LAYOUT_POOL) {
    uint64_t maps = ctx->plan.n_chunks;
    for (const Interval& iv : ctx->plan.intervals) maps += iv.chunks.size();
    const int64_t room = map_entries_left();
    if (room >= 0 && maps + 2048 > (uint64_t)room) {
      ctx->err = "the plan needs " + std::to_string(maps) +
                 " memory-map entries (chunks + mappings) but the process has " +
                 std::to_string(room) + " left; use a larger chunk size";
      return OOC_E_UNSUPPORTED;
    }
  }

  // physical chunks
  ctx->chunks.resize(ctx->layout == OOC_LAYOUT_POOL ? plan.n_chunks : 0);
  for (uint64_t c = 0; c < ctx->chunks.size(); ++c) {
    hipError_t e = hipMemCreate(&ctx->chunks[c], ctx->chunk, &prop, 0);
    if (e != hipSuccess) {
      ctx->chunks.resize(c);
      ctx->err = "hipMemCreate of chunk " + std::to_string(c) + " failed: " +
                 hipGetErrorString(e);
      return OOC_E_DEVICE;
    }
  }
  // one virtual range per interval, carved out of one reservation
  uint64_t total = 0;
  std::vector<uint64_t> off(NI);
  for (int64_t J = 0; J < NI; ++J) {
    off[J] = total;
    total += plan.intervals[J].chunks.size() * ctx->chunk;
  }
  if (ctx->layout == OOC_LAYOUT_POOL) ctx->iv_ptr.assign(NI, nullptr);
  if (ctx->layout == OOC_LAYOUT_POOL && total > 0) {
    HIPCK(hipMemAddressReserve(&ctx->va_base, total, ctx->chunk, nullptr, 0));
    ctx->va_bytes = total;
    uint64_t maps = 0;
    for (int64_t J = 0; J < NI; ++J) {
      char* base = (char*)ctx->va_base + off[J];
      ctx->iv_ptr[J] = base;
      const auto& cs = plan.intervals[J].chunks;
      for (size_t j = 0; j < cs.size(); ++j) {
        HIPCK(hipMemMap(base + j * ctx->chunk, ctx->chunk, 0, ctx->chunks[cs[j]], 0));
        ++maps;
      }
    }
    // read/write access, set per interval in pieces of at most 1 GiB (one call
    // over a reservation of ~100 GiB is rejected as an invalid argument)
    hipMemAccessDesc ad = {};
    ad.location.type = hipMemLocationTypeDevice;
    ad.location.id = ctx->device;
    ad.flags = hipMemAccessFlagsProtReadWrite;
    const uint64_t piece = std::max<uint64_t>(ctx->chunk, (1ull << 30) / ctx->chunk * ctx->chunk);
    for (int64_t J = 0; J < NI; ++J) {
      const uint64_t len = plan.intervals[J].chunks.size() * ctx->chunk;
      for (uint64_t o = 0; o < len; o += piece)
        HIPCK(hipMemSetAccess(ctx->iv_ptr[J] + o, std::min(piece, len - o), &ad, 1));
    }
    ctx->stats.n_mappings = maps;
  }
  HIPCK(hipMemGetInfo(&free1, &total1));

  HIPCK(hipStreamCreateWithFlags(&ctx->cs, hipStreamNonBlocking));
  HIPCK(hipStreamCreateWithFlags(&ctx->hs, hipStreamNonBlocking));
  HIPCK(hipStreamCreateWithFlags(&ctx->ds, hipStreamNonBlocking));
  HIPCK(hipStreamCreateWithFlags(&ctx->ss, hipStreamNonBlocking));

  {
    ooc_status s = compile(ctx);
    if (s) return s;
  }

  // pinned host arena.  A persistent variable (INPUT, PARAM, STATE, OUTPUT)
  // owns its slot for the whole step: the caller reads and writes it there.
  // A TEMP needs host memory only from its first swap-out to its last
  // swap-in, so TEMP slots are packed by lifetime: best fit over the holes
  // left by TEMPs whose last swap-in was issued before.  The first swap-out
  // into reused bytes waits for the last swap-in of every earlier occupant of
  // those bytes; the variable's later swap-outs follow it on the same stream.
  const int64_t nv = (int64_t)ctx->vars.size();
  std::vector<uint8_t> backed(nv, 0);
  std::vector<uint64_t> hoff(nv, 0);
  uint64_t hb = 0;
  for (int64_t v = 0; v < nv; ++v)
    if (ctx->vars[v].kind != OOC_TEMP) {
      backed[v] = 1;
      hoff[v] = hb;
      hb += round_up(ctx->vars[v].bytes, kSlotAlign);
    }
  const uint64_t pers = hb;
  // With a host limit, TEMP slots get pinned bytes up to the limit (less the
  // staging slots); the rest get pageable homes, one each, no reuse.
  const uint64_t stage_bytes = 2 * kSlots * kPiece;
  uint64_t cap = UINT64_MAX;
  if (ctx->host_limit != OOC_UNLIMITED) {
    if (ctx->host_limit < pers + stage_bytes) {
      ctx->err = "host limit " + std::to_string(ctx->host_limit) + " is below the " +
                 std::to_string(pers) + " bytes of persistent slots plus " +
                 std::to_string(stage_bytes) + " bytes of staging slots";
      return OOC_E_HOST_OOM;
    }
    cap = ctx->host_limit - pers - stage_bytes;
  }
  std::vector<uint8_t> spilled(nv, 0);
  std::vector<uint64_t> soff(nv, 0);
  uint64_t spill_top = 0;
  // lifetimes in issue order: swap-ins of f_i at 3 i, swap-outs at 3 i + 2
  std::vector<int64_t> born(nv, -1), dies(nv, -1);
  std::vector<int32_t> last_in(nv, -1);
  std::vector<Copy*> first_out(nv, nullptr);
  for (size_t i = 0; i < ctx->prog.size(); ++i) {
    for (Copy& c : ctx->prog[i].h2d) {
      if (backed[c.var]) continue;
      if (born[c.var] < 0) {
        ctx->err = "swap-in of variable " + std::to_string(c.var) + " with no host copy";
        return OOC_E_INVALID;
      }
      dies[c.var] = std::max<int64_t>(dies[c.var], 3 * (int64_t)i);
      last_in[c.var] = c.ev_done;
    }
    for (Copy& c : ctx->prog[i].d2h) {
      if (backed[c.var]) continue;
      if (born[c.var] < 0) {
        born[c.var] = 3 * (int64_t)i + 2;
        first_out[c.var] = &c;
      }
      dies[c.var] = std::max<int64_t>(dies[c.var], 3 * (int64_t)i + 2);
    }
  }
  std::vector<int64_t> order;
  for (int64_t v = 0; v < nv; ++v)
    if (born[v] >= 0) order.push_back(v);
  std::stable_sort(order.begin(), order.end(),
                   [&](int64_t x, int64_t y) { return born[x] < born[y]; });
  struct Span { uint64_t off, size; };
  struct Freed { uint64_t off, size; int32_t ev; };
  std::vector<Span> holes;     // sorted by offset, disjoint, not adjacent
  std::vector<Freed> freed;    // released occupants whose last swap-in later copies wait for
  std::priority_queue<std::pair<int64_t, int64_t>, std::vector<std::pair<int64_t, int64_t>>,
                      std::greater<>> live;   // (dies, var)
  uint64_t top = 0;
  auto release = [&](int64_t u) {
    const uint64_t off = hoff[u] - pers, size = round_up(ctx->vars[u].bytes, kSlotAlign);
    if (last_in[u] >= 0) freed.push_back(Freed{off, size, last_in[u]});
    auto it = std::lower_bound(holes.begin(), holes.end(), off,
                               [](const Span& h, uint64_t o) { return h.off < o; });
    it = holes.insert(it, Span{off, size});
    if (it + 1 != holes.end() && it->off + it->size == (it + 1)->off) {
      it->size += (it + 1)->size;
      holes.erase(it + 1);
    }
    if (it != holes.begin() && (it - 1)->off + (it - 1)->size == it->off) {
      (it - 1)->size += it->size;
      holes.erase(it);
    }
  };
  for (int64_t v : order) {
    while (!live.empty() && live.top().first < born[v]) {
      release(live.top().second);
      live.pop();
    }
    const uint64_t size = round_up(ctx->vars[v].bytes, kSlotAlign);
    size_t best = holes.size();
    for (size_t h = 0; h < holes.size(); ++h)
      if (holes[h].size >= size && (best == holes.size() || holes[h].size < holes[best].size))
        best = h;
    uint64_t off;
    if (best < holes.size()) {
      off = holes[best].off;
      holes[best].off += size;
      holes[best].size -= size;
      if (holes[best].size == 0) holes.erase(holes.begin() + best);
    } else if (size <= cap && top <= cap - size) {
      off = top;
      top += size;
    } else {
      spilled[v] = 1;
      soff[v] = spill_top;
      spill_top += size;
      backed[v] = 1;
      continue;
    }
    backed[v] = 1;
    hoff[v] = pers + off;
    std::vector<int32_t>& w = first_out[v]->waits;
    for (size_t f = 0; f < freed.size();) {
      const Freed& fr = freed[f];
      if (fr.off < off + size && off < fr.off + fr.size) {
        if (std::find(w.begin(), w.end(), fr.ev) == w.end()) w.push_back(fr.ev);
        if (fr.off >= off && fr.off + fr.size <= off + size) {
          freed.erase(freed.begin() + f);
          continue;
        }
      }
      ++f;
    }
    live.push({dies[v], v});
  }
  hb = pers + top;
  const uint64_t stage_off = hb;
  if (spill_top > 0) hb += stage_bytes;
  ctx->host_slot.assign(nv, nullptr);
  if (hb > 0) {
    hipError_t e = hipHostMalloc((void**)&ctx->arena, hb, hipHostMallocDefault);
    if (e != hipSuccess) {
      (void)hipGetLastError();   // the refusal must not surface at a later launch check
      ctx->arena = nullptr;
      ctx->err = "pinned host arena of " + std::to_string(hb) + " bytes: " + hipGetErrorString(e);
      return OOC_E_HOST_OOM;
    }
    ctx->arena_bytes = hb;
    for (int64_t v = 0; v < nv; ++v)
      if (backed[v] && !spilled[v]) ctx->host_slot[v] = ctx->arena + hoff[v];
  }
  ctx->in_copy.clear();
  ctx->out_copy.clear();
  ctx->ev_staged_in.clear();
  ctx->in_piece.clear();
  ctx->out_piece.clear();
  ctx->staged_h2d = ctx->staged_d2h = 0;
  if (spill_top > 0) {
    // pageable homes: populated now (transparent huge pages where the kernel
    // gives them), so that no page fault lands inside a step
    void* m = mmap(nullptr, spill_top, PROT_READ | PROT_WRITE, MAP_PRIVATE | MAP_ANONYMOUS, -1, 0);
    if (m == MAP_FAILED) {
      ctx->err = "pageable host overflow of " + std::to_string(spill_top) + " bytes: mmap failed";
      return OOC_E_HOST_OOM;
    }
    ctx->spill = (char*)m;
    ctx->spill_bytes = spill_top;
    madvise(m, spill_top, MADV_HUGEPAGE);
    {
      std::vector<std::thread> ts;
      const uint64_t part = round_up((spill_top + 7) / 8, kSlotAlign);
      for (uint64_t o = 0; o < spill_top; o += part)
        ts.emplace_back([=] { std::memset(ctx->spill + o, 0, std::min(part, spill_top - o)); });
      for (auto& t : ts) t.join();
    }
    ctx->stage_in = ctx->arena + stage_off;
    ctx->stage_out = ctx->stage_in + kSlots * kPiece;
    for (int64_t v = 0; v < nv; ++v)
      if (spilled[v]) ctx->host_slot[v] = ctx->spill + soff[v];
    // staged copies in pieces, numbered per direction in issue order; a
    // swap-in needs the host copy written by the latest swap-out before it
    std::vector<int64_t> outs(nv, 0);
    auto split = [&](Copy& c, int8_t stream, std::vector<const Copy*>* owner,
                     std::vector<int32_t>* index) {
      c.staged = true;
      const uint64_t n = (c.bytes + kPiece - 1) / kPiece;
      for (uint64_t k = 0; k < n; ++k) {
        Piece pc;
        pc.off = k * kPiece;
        pc.bytes = std::min(kPiece, c.bytes - pc.off);
        pc.ev_start = k == 0 ? c.ev_start : new_event(ctx, stream);
        pc.ev_done = k + 1 == n ? c.ev_done : new_event(ctx, stream);
        pc.seq = (int64_t)owner->size();
        owner->push_back(&c);
        index->push_back((int32_t)k);
        c.pieces.push_back(pc);
      }
    };
    int64_t staged_in = 0;
    for (FnProgram& fp : ctx->prog) {
      for (Copy& c : fp.h2d)
        if (spilled[c.var]) {
          c.gen = outs[c.var];
          // staged swap-ins run on their own stream (3)
          ctx->event_stream[c.ev_start] = ctx->event_stream[c.ev_done] = 3;
          split(c, 3, &ctx->in_copy, &ctx->in_piece);
          ctx->staged_h2d += c.bytes;
          if ((int64_t)ctx->ev_staged_in.size() < (int64_t)ctx->event_stream.size())
            ctx->ev_staged_in.resize(ctx->event_stream.size(), -1);
          ctx->ev_staged_in[c.ev_done] = staged_in++;
        }
      for (Copy& c : fp.d2h)
        if (spilled[c.var]) {
          c.gen = ++outs[c.var];
          split(c, 2, &ctx->out_copy, &ctx->out_piece);
          ctx->staged_d2h += c.bytes;
        }
    }
  }
  for (FnProgram& fp : ctx->prog) {
    for (Copy& c : fp.h2d) {
      c.dst = ctx->iv_ptr[c.iv];
      c.src = ctx->host_slot[c.var];
    }
    for (Copy& c : fp.d2h) {
      c.dst = ctx->host_slot[c.var];
      c.src = ctx->iv_ptr[c.iv];
    }
  }

  ctx->ev_staged_in.resize(ctx->event_stream.size(), -1);
  // Compute-stream events that no stream waits for only time the step: they are
  // created without the system-scope fence that recording an event otherwise
  // performs (a cache writeback and invalidation after every function, measured
  // at ~6 % of the plain CNN's in-core step).  Events another stream waits for
  // keep it.
  std::vector<uint8_t> waited(ctx->event_stream.size(), 0);
  for (const FnProgram& fp : ctx->prog) {
    for (int32_t w : fp.cwaits) waited[w] = 1;
    for (const Copy& c : fp.h2d)
      for (int32_t w : c.waits) waited[w] = 1;
    for (const Copy& c : fp.d2h)
      for (int32_t w : c.waits) waited[w] = 1;
  }
  ctx->events.resize(ctx->event_stream.size(), nullptr);
  for (size_t j = 0; j < ctx->events.size(); ++j) {
    const bool timing_only = ctx->event_stream[j] == 0 && !waited[j];
    hipError_t e = timing_only ? hipEventCreateWithFlags(&ctx->events[j], hipEventDisableSystemFence)
                               : hipEventCreate(&ctx->events[j]);
    if (e != hipSuccess) {
      ctx->events.resize(j);
      ctx->err = std::string("hipEventCreate failed: ") + hipGetErrorString(e);
      return OOC_E_DEVICE;
    }
  }
  for (int64_t i = (int64_t)ctx->fns.size() - 1; i >= 0; --i)
    if (ctx->fns[i].op == OOC_OP_SOFTMAX_CE) {
      ctx->loss_var = ctx->fns[i].vars[2].var;
      break;
    }
  if (!ctx->incore) {
    ooc_status s = warm_copy_streams(ctx);
    if (s) return s;
  }

  auto t1 = std::chrono::steady_clock::now();
  ooc_stats& st = ctx->stats;
  st.pool_chunks = ctx->chunks.size();
  st.pool_bytes = ctx->layout == OOC_LAYOUT_POOL ? plan.n_chunks * ctx->chunk : ctx->heap_extent;
  st.max_chunks_used = plan.max_chunks_used;
  st.device_bytes_delta = free0 > free1 ? (uint64_t)(free0 - free1) : 0;
  st.host_bytes = hb;
  st.spill_bytes = ctx->spill_bytes;
  st.staged_h2d_bytes = ctx->staged_h2d;
  st.staged_d2h_bytes = ctx->staged_d2h;
  st.n_intervals = (uint64_t)NI;
  st.prepare_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
  return OOC_OK;
}

static ooc_status enqueue_copy(ooc_ctx* ctx, const Copy& c, hipStream_t s, hipMemcpyKind kind) {
  for (int32_t w : c.waits) HIPCK(hipStreamWaitEvent(s, ctx->events[w], 0));
  HIPCK(hipEventRecord(ctx->events[c.ev_start], s));
  HIPCK(hipMemcpyAsync(c.dst, c.src, c.bytes, kind, s));
  HIPCK(hipEventRecord(ctx->events[c.ev_done], s));
  return OOC_OK;
}

ooc_status timeline(ooc_ctx* ctx, std::vector<ooc_span>* out) {
  out->clear();
  if (ctx->fn_ms.empty()) {
    ctx->err = "no step has run";
    return OOC_E_STATE;
  }
  const hipEvent_t t0 = ctx->events[ctx->ev_begin];
  auto span = [&](int32_t kind, int32_t fn, int64_t var, uint64_t bytes, int32_t a,
                  int32_t b) -> ooc_status {
    float s = 0, d = 0;
    HIPCK(hipEventElapsedTime(&s, t0, ctx->events[a]));
    HIPCK(hipEventElapsedTime(&d, ctx->events[a], ctx->events[b]));
    out->push_back(ooc_span{kind, fn, var, bytes, s, d});
    return OOC_OK;
  };
  const int32_t N = (int32_t)ctx->fns.size();
  for (int32_t i = 0; i < N; ++i) {
    ooc_status r = span(0, i, -1, 0, ctx->prog[i].ev_pre, ctx->prog[i].ev_fn);
    if (r) return r;
  }
  for (int32_t i = 0; i < N; ++i) {
    for (const Copy& c : ctx->prog[i].h2d) {
      ooc_status r = span(1, i, c.var, c.bytes, c.ev_start, c.ev_done);
      if (r) return r;
    }
    for (const Copy& c : ctx->prog[i].d2h) {
      ooc_status r = span(2, i, c.var, c.bytes, c.ev_start, c.ev_done);
      if (r) return r;
    }
  }
  return OOC_OK;
}

namespace {

// Host side of the staged copies of one step (pageable homes, see
// ooc_set_host_limit).
//  * Swap-in piece p: a fill thread copies the pageable home into staging
//    slot p mod kSlots once the slot's previous piece has reached the device
//    and the variable's host copy has been written; an issuer thread, in
//    program order, enqueues each staged swap-in on its own stream once the
//    step loop has reached it, piece by piece as the slots fill.  The step
//    loop only waits for the issuer when a kernel needs a staged swap-in
//    whose copy is not enqueued yet, so it keeps running ahead of the device.
//  * Swap-out piece q: the step loop enqueues the device copy into slot
//    q mod kSlots once a drain thread has emptied the slot's previous piece
//    into its pageable home.
// Every wait is for work that comes earlier in the step's order, so all of
// them end.
struct Stager {
  ooc_ctx* ctx;
  hipStream_t s;                    // stream of the staged swap-ins
  std::mutex m;
  std::condition_variable cv;
  std::vector<uint8_t> in_ready, out_free;
  std::vector<int64_t> written;     // per variable: host copies completed this step
  std::vector<int32_t> left;        // per swap-out copy (seq of its first piece): pieces to drain
  int64_t in_enq = 0;               // swap-in pieces enqueued by the issuer
  int64_t out_pushed = 0;           // swap-out pieces enqueued by the step loop
  int64_t posted = 0;               // staged swap-in copies the step loop has reached
  int64_t recorded = 0;             // staged swap-in copies the issuer has enqueued
  bool failed = false, finished = false;
  std::string err;
  std::vector<std::thread> threads;

  Stager(ooc_ctx* c, hipStream_t stream) : ctx(c), s(stream) {
    const int64_t ni = (int64_t)ctx->in_copy.size(), no = (int64_t)ctx->out_copy.size();
    if (ni == 0 && no == 0) return;
    in_ready.assign(ni, 0);
    out_free.assign(no, 0);
    written.assign(ctx->vars.size(), 0);
    left.assign(no, 0);
    for (int64_t q = 0; q < no; ++q) {
      const Copy& cp = *ctx->out_copy[q];
      left[cp.pieces[0].seq] = (int32_t)cp.pieces.size();
    }
    for (int t = 0; t < kThreads; ++t) {
      if (t < ni) threads.emplace_back([this, t] { fill(t); });
      if (t < no) threads.emplace_back([this, t] { drain(t); });
    }
    if (ni > 0) threads.emplace_back([this] { issue(); });
  }
  ~Stager() { finish(true); }

  char* in_slot(int64_t p) const { return ctx->stage_in + (p % kSlots) * kPiece; }
  char* out_slot(int64_t q) const { return ctx->stage_out + (q % kSlots) * kPiece; }

  void fail(const std::string& e) {
    {
      std::lock_guard<std::mutex> lk(m);
      if (!failed) err = e;
      failed = true;
    }
    cv.notify_all();
  }
  template <class Pred>
  bool wait(Pred pred) {
    std::unique_lock<std::mutex> lk(m);
    cv.wait(lk, [&] { return failed || pred(); });
    return !failed;
  }
  void bump(int64_t* counter, int64_t v) {
    {
      std::lock_guard<std::mutex> lk(m);
      *counter = v;
    }
    cv.notify_all();
  }
  // joins the threads; abort: make every wait end first
  void finish(bool abort) {
    if (finished) return;
    finished = true;
    if (abort) {
      {
        std::lock_guard<std::mutex> lk(m);
        if (!failed) err = "step aborted";
        failed = true;
      }
      cv.notify_all();
    }
    for (auto& t : threads) t.join();
  }

  void fill(int t) {
    if (const hipError_t e = hipSetDevice(ctx->device); e != hipSuccess)
      return fail(std::string("staging: ") + hipGetErrorString(e));
    const int64_t n = (int64_t)ctx->in_copy.size();
    for (int64_t p = t; p < n; p += kThreads) {
      const Copy& c = *ctx->in_copy[p];
      const Piece& pc = c.pieces[ctx->in_piece[p]];
      if (p >= kSlots) {
        if (!wait([&] { return in_enq > p - kSlots; })) return;
        const Copy& prev = *ctx->in_copy[p - kSlots];
        const hipError_t e =
            hipEventSynchronize(ctx->events[prev.pieces[ctx->in_piece[p - kSlots]].ev_done]);
        if (e != hipSuccess) return fail(std::string("staging: ") + hipGetErrorString(e));
      }
      if (!wait([&] { return written[c.var] >= c.gen; })) return;
      std::memcpy(in_slot(p), ctx->host_slot[c.var] + pc.off, pc.bytes);
      {
        std::lock_guard<std::mutex> lk(m);
        in_ready[p] = 1;
      }
      cv.notify_all();
    }
  }

  void issue() {
    if (const hipError_t e = hipSetDevice(ctx->device); e != hipSuccess)
      return fail(std::string("staging: ") + hipGetErrorString(e));
    const int64_t n = (int64_t)ctx->in_copy.size();
    int64_t ci = 0;
    for (int64_t p = 0; p < n; ++ci) {
      const Copy& c = *ctx->in_copy[p];
      if (!wait([&] { return posted > ci; })) return;
      for (int32_t w : c.waits) {
        const hipError_t e = hipStreamWaitEvent(s, ctx->events[w], 0);
        if (e != hipSuccess) return fail(std::string("staging: ") + hipGetErrorString(e));
      }
      for (const Piece& pc : c.pieces) {
        if (!wait([&] { return in_ready[pc.seq] != 0; })) return;
        hipError_t e = hipEventRecord(ctx->events[pc.ev_start], s);
        if (e == hipSuccess)
          e = hipMemcpyAsync((char*)c.dst + pc.off, in_slot(pc.seq), pc.bytes,
                             hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = hipEventRecord(ctx->events[pc.ev_done], s);
        if (e != hipSuccess) return fail(std::string("staging: ") + hipGetErrorString(e));
        bump(&in_enq, pc.seq + 1);
      }
      p += (int64_t)c.pieces.size();
      bump(&recorded, ci + 1);
    }
  }

  void drain(int t) {
    if (const hipError_t e = hipSetDevice(ctx->device); e != hipSuccess)
      return fail(std::string("staging: ") + hipGetErrorString(e));
    const int64_t n = (int64_t)ctx->out_copy.size();
    for (int64_t q = t; q < n; q += kThreads) {
      const Copy& c = *ctx->out_copy[q];
      const Piece& pc = c.pieces[ctx->out_piece[q]];
      if (!wait([&] { return out_pushed > q; })) return;
      const hipError_t e = hipEventSynchronize(ctx->events[pc.ev_done]);
      if (e != hipSuccess) return fail(std::string("staging: ") + hipGetErrorString(e));
      std::memcpy(ctx->host_slot[c.var] + pc.off, out_slot(q), pc.bytes);
      {
        std::lock_guard<std::mutex> lk(m);
        out_free[q] = 1;
        if (--left[c.pieces[0].seq] == 0) written[c.var] = std::max(written[c.var], c.gen);
      }
      cv.notify_all();
    }
  }
};

}  // namespace

// Enqueues a staged swap-out piece by piece (see Stager).
static ooc_status enqueue_staged_out(ooc_ctx* ctx, Stager* sg, const Copy& c) {
  hipStream_t s = ctx->ds;
  for (size_t k = 0; k < c.pieces.size(); ++k) {
    const Piece& pc = c.pieces[k];
    const int64_t q = pc.seq;
    if (q >= kSlots && !sg->wait([&] { return sg->out_free[q - kSlots] != 0; })) {
      ctx->err = sg->err;
      return OOC_E_DEVICE;
    }
    if (k == 0)
      for (int32_t w : c.waits) HIPCK(hipStreamWaitEvent(s, ctx->events[w], 0));
    HIPCK(hipEventRecord(ctx->events[pc.ev_start], s));
    HIPCK(hipMemcpyAsync(sg->out_slot(q), (const char*)c.src + pc.off, pc.bytes,
                         hipMemcpyDeviceToHost, s));
    HIPCK(hipEventRecord(ctx->events[pc.ev_done], s));
    sg->bump(&sg->out_pushed, q + 1);
  }
  return OOC_OK;
}

ooc_status step(ooc_ctx* ctx, float lr, float mu, float* loss_out) {
  HIPCK(hipSetDevice(ctx->device));
  auto t0 = std::chrono::steady_clock::now();
  Stager stager(ctx, ctx->ss);
  int64_t staged_in = 0;         // staged swap-in copies reached so far
  hipStream_t cs = ctx->cs;
  HIPCK(hipEventRecord(ctx->events[ctx->ev_begin], cs));
  const int64_t N = (int64_t)ctx->fns.size();
  const int64_t depth = ctx->swapout_depth;
  std::vector<int32_t> issued;   // done events of the swap-outs issued so far
  for (int64_t i = 0; i < N; ++i) {
    const FnProgram& fp = ctx->prog[i];
    // an event of a staged swap-in is recorded by the issuer thread: wait until it has
    // been, before a stream of this loop waits for it
    auto issued_by_stager = [&](const std::vector<int32_t>& evs) -> bool {
      for (int32_t w : evs) {
        const int64_t sc = ctx->ev_staged_in[w];   // staged swap-in it completes, or -1
        if (sc >= 0 && !stager.wait([&] { return stager.recorded > sc; })) {
          ctx->err = stager.err;
          return false;
        }
      }
      return true;
    };
    for (const Copy& c : fp.h2d) {
      if (c.staged) {
        stager.bump(&stager.posted, ++staged_in);
        continue;
      }
      if (!issued_by_stager(c.waits)) return OOC_E_DEVICE;
      ooc_status s = enqueue_copy(ctx, c, ctx->hs, hipMemcpyHostToDevice);
      if (s) return s;
    }
    if (!issued_by_stager(fp.cwaits)) return OOC_E_DEVICE;
    for (int32_t w : fp.cwaits) HIPCK(hipStreamWaitEvent(cs, ctx->events[w], 0));
    HIPCK(hipEventRecord(ctx->events[fp.ev_pre], cs));
    hipError_t e = launch_fn(ctx->fns[i], fp.ptrs.data(), fp.sizes.data(), lr, mu, cs);
    if (e != hipSuccess) {
      ctx->err = "kernel launch of function " + std::to_string(i) + " failed: " +
                 hipGetErrorString(e);
      return OOC_E_DEVICE;
    }
    HIPCK(hipEventRecord(ctx->events[fp.ev_fn], cs));
    for (const Copy& c : fp.d2h) {
      // bounded queue of swap-outs (see ooc_set_swapout_depth); the compute
      // stream already holds the work up to f_i, so it keeps running meanwhile
      if (depth > 0 && (int64_t)issued.size() >= depth)
        HIPCK(hipEventSynchronize(ctx->events[issued[issued.size() - depth]]));
      ooc_status s = c.staged ? enqueue_staged_out(ctx, &stager, c)
                              : enqueue_copy(ctx, c, ctx->ds, hipMemcpyDeviceToHost);
      if (s) return s;
      issued.push_back(c.ev_done);
    }
  }
  HIPCK(hipEventRecord(ctx->events[ctx->ev_end], cs));
  HIPCK(hipStreamSynchronize(cs));
  HIPCK(hipStreamSynchronize(ctx->hs));
  HIPCK(hipStreamSynchronize(ctx->ds));
  stager.finish(false);
  HIPCK(hipStreamSynchronize(ctx->ss));
  if (stager.failed) {
    ctx->err = stager.err;
    return OOC_E_DEVICE;
  }
  auto t1 = std::chrono::steady_clock::now();

  ooc_stats& st = ctx->stats;
  st.step_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
  float ms = 0;
  HIPCK(hipEventElapsedTime(&ms, ctx->events[ctx->ev_begin], ctx->events[ctx->ev_end]));
  st.step_gpu_ms = ms;
  double hbusy = 0, dbusy = 0, cbusy = 0;
  ctx->fn_ms.assign(N, 0.0);
  for (int64_t i = 0; i < N; ++i) {
    const FnProgram& fp = ctx->prog[i];
    for (const Copy& c : fp.h2d) {
      HIPCK(hipEventElapsedTime(&ms, ctx->events[c.ev_start], ctx->events[c.ev_done]));
      hbusy += ms;
    }
    for (const Copy& c : fp.d2h) {
      HIPCK(hipEventElapsedTime(&ms, ctx->events[c.ev_start], ctx->events[c.ev_done]));
      dbusy += ms;
    }
    HIPCK(hipEventElapsedTime(&ms, ctx->events[fp.ev_pre], ctx->events[fp.ev_fn]));
    cbusy += ms;
    ctx->fn_ms[i] = ms;
  }
  st.h2d_busy_ms = hbusy;
  st.d2h_busy_ms = dbusy;
  st.compute_busy_ms = cbusy;
  st.h2d_bytes = ctx->prog_h2d;
  st.d2h_bytes = ctx->prog_d2h;

  if (loss_out) {
    float loss = __builtin_nanf("");
    if (ctx->loss_var >= 0) {
      const uint64_t b = ctx->vars[ctx->loss_var].bytes;
      if (ctx->incore) {
        const char* d = ctx->iv_ptr[ctx->resident[ctx->loss_var]];
        HIPCK(hipMemcpy(&loss, d + b - 4, 4, hipMemcpyDeviceToHost));
      } else {
        std::memcpy(&loss, ctx->host_slot[ctx->loss_var] + b - 4, 4);
      }
    }
    *loss_out = loss;
  }
  return OOC_OK;
}

ooc_status transfer_resident(ooc_ctx* ctx, bool to_device) {
  if (!ctx->incore) return OOC_OK;
  HIPCK(hipSetDevice(ctx->device));
  for (int64_t v = 0; v < (int64_t)ctx->vars.size(); ++v) {
    const int32_t kind = ctx->vars[v].kind;
    if (kind == OOC_TEMP || ctx->resident[v] < 0) continue;
    char* d = ctx->iv_ptr[ctx->resident[v]];
    if (to_device && (kind == OOC_INPUT || kind == OOC_PARAM || kind == OOC_STATE))
      HIPCK(hipMemcpy(d, ctx->host_slot[v], ctx->vars[v].bytes, hipMemcpyHostToDevice));
    if (!to_device && kind != OOC_INPUT)
      HIPCK(hipMemcpy(ctx->host_slot[v], d, ctx->vars[v].bytes, hipMemcpyDeviceToHost));
  }
  HIPCK(hipDeviceSynchronize());
  return OOC_OK;
}

ooc_status link_probe(int32_t device, uint64_t bytes, int32_t reps, double* h2d, double* d2h,
                      double* both, std::string* err) {
  ooc_ctx dummy;
  ooc_ctx* ctx = &dummy;
  void *hp1 = nullptr, *hp2 = nullptr, *d1 = nullptr, *d2 = nullptr;
  hipStream_t s1 = nullptr, s2 = nullptr;
  hipEvent_t e[4] = {};
  ooc_status st = OOC_OK;
  auto run = [&]() -> ooc_status {
    HIPCK(hipSetDevice(device));
    HIPCK(hipHostMalloc(&hp1, bytes, hipHostMallocDefault));
    HIPCK(hipHostMalloc(&hp2, bytes, hipHostMallocDefault));
    HIPCK(hipMalloc(&d1, bytes));
    HIPCK(hipMalloc(&d2, bytes));
    std::memset(hp1, 1, bytes);
    std::memset(hp2, 2, bytes);
    HIPCK(hipStreamCreateWithFlags(&s1, hipStreamNonBlocking));
    HIPCK(hipStreamCreateWithFlags(&s2, hipStreamNonBlocking));
    for (auto& x : e) HIPCK(hipEventCreate(&x));
    double bh = 0, bd = 0, bb = 0;
    for (int r = 0; r < reps; ++r) {
      float ms = 0;
      HIPCK(hipEventRecord(e[0], s1));
      HIPCK(hipMemcpyAsync(d1, hp1, bytes, hipMemcpyHostToDevice, s1));
      HIPCK(hipEventRecord(e[1], s1));
      HIPCK(hipEventSynchronize(e[1]));
      HIPCK(hipEventElapsedTime(&ms, e[0], e[1]));
      bh = std::max(bh, bytes / (ms * 1e6));
      HIPCK(hipEventRecord(e[0], s2));
      HIPCK(hipMemcpyAsync(hp2, d2, bytes, hipMemcpyDeviceToHost, s2));
      HIPCK(hipEventRecord(e[1], s2));
      HIPCK(hipEventSynchronize(e[1]));
      HIPCK(hipEventElapsedTime(&ms, e[0], e[1]));
      bd = std::max(bd, bytes / (ms * 1e6));
      HIPCK(hipDeviceSynchronize());
      auto t0 = std::chrono::steady_clock::now();
      HIPCK(hipMemcpyAsync(d1, hp1, bytes, hipMemcpyHostToDevice, s1));
      HIPCK(hipMemcpyAsync(hp2, d2, bytes, hipMemcpyDeviceToHost, s2));
      HIPCK(hipStreamSynchronize(s1));
      HIPCK(hipStreamSynchronize(s2));
      auto t1 = std::chrono::steady_clock::now();
      bb = std::max(bb, 2.0 * bytes / (std::chrono::duration<double>(t1 - t0).count() * 1e9));
    }
    *h2d = bh;
    *d2h = bd;
    *both = bb;
    return OOC_OK;
  };
  st = run();
  *err = ctx->err;
  // clean-up after the probe: its result stands whatever these return
  for (auto x : e)
    if (x) (void)hipEventDestroy(x);
  if (s1) (void)hipStreamDestroy(s1);
  if (s2) (void)hipStreamDestroy(s2);
  if (d1) (void)hipFree(d1);
  if (d2) (void)hipFree(d2);
  if (hp1) (void)hipHostFree(hp1);
  if (hp2) (void)hipHostFree(hp2);
  return st;
}

}  // namespace ooc
