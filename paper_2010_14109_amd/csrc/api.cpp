// C interface: argument checks, the call-order state machine and error
// reporting around the scheduler, the chunk plan and the executor.
#include <cmath>
#include <cstring>
#include <new>

#include "ctx.h"
#include "kernels.h"

namespace ooc {
ooc_status prepare(ooc_ctx* ctx);
ooc_status step(ooc_ctx* ctx, float lr, float mu, float* loss_out);
ooc_status timeline(ooc_ctx* ctx, std::vector<ooc_span>* out);
ooc_status transfer_resident(ooc_ctx* ctx, bool to_device);
void release_device(ooc_ctx* ctx);
ooc_status link_probe(int32_t device, uint64_t bytes, int32_t reps, double* h2d, double* d2h,
                      double* both, std::string* err);
}  // namespace ooc

using namespace ooc;

static thread_local std::string g_create_error;

// Records msg as the context's last error (readable with ooc_last_error) and
// returns s.  The message lives in the context, so const queries set it too.
static ooc_status fail(const ooc_ctx* ctx, ooc_status s, const std::string& msg) {
  ctx->err = msg;
  return s;
}

#define REQUIRE_CTX(ctx)                                 \
  if (!(ctx)) {                                          \
    g_create_error = std::string(__func__) + ": NULL context"; \
    return OOC_E_INVALID;                                \
  }
// queries valid once the schedule is built
#define REQUIRE_BUILT(ctx)                                                          \
  if ((ctx)->stage < BUILT)                                                         \
  return fail((ctx), OOC_E_STATE, std::string(__func__) + " before ooc_build_schedule")
#define REQUIRE_OUT(ctx, p)                                                        \
  if (!(p))                                                                          \
  return fail((ctx), OOC_E_INVALID, std::string(__func__) + ": " #p " is NULL")
#define REQUIRE_BUF(ctx, buf, cap)                                                 \
  if ((cap) > 0 && !(buf))                                                           \
  return fail((ctx), OOC_E_INVALID, std::string(__func__) + ": " #buf " is NULL with cap > 0")
#define REQUIRE_STAGE(ctx, st, what)                                              \
  if ((ctx)->stage != (st)) return fail((ctx), OOC_E_STATE, std::string(what) +   \
                                         " is not allowed at this point")

extern "C" {

ooc_status ooc_create(int32_t hip_device, ooc_ctx** out) {
  if (!out) {
    g_create_error = "ooc_create: out is NULL";
    return OOC_E_INVALID;
  }
  *out = nullptr;
  if (hip_device < -1) {
    g_create_error = "device id must be >= -1";
    return OOC_E_INVALID;
  }
  if (hip_device >= 0) {
    int n = 0;
    hipError_t e = hipGetDeviceCount(&n);
    if (e != hipSuccess || hip_device >= n) {
      g_create_error = std::string("HIP device ") + std::to_string(hip_device) +
                       " is not available" + (e != hipSuccess ? std::string(": ") +
                       hipGetErrorString(e) : std::string());
      return OOC_E_DEVICE;
    }
  }
  ooc_ctx* ctx = new (std::nothrow) ooc_ctx();
  if (!ctx) {
    g_create_error = "ooc_create: out of host memory";
    return OOC_E_HOST_OOM;
  }
  ctx->device = hip_device;
  *out = ctx;
  return OOC_OK;
}

void ooc_destroy(ooc_ctx* ctx) {
  if (!ctx) return;
  release_device(ctx);
  delete ctx;
}

const char* ooc_last_error(const ooc_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_create_error.c_str();
}

ooc_status ooc_add_var(ooc_ctx* ctx, uint64_t bytes, int32_t kind, int64_t* out_id) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, REGISTERING, "ooc_add_var");
  if (bytes == 0) return fail(ctx, OOC_E_INVALID, "a variable needs at least one byte");
  if (bytes > (1ull << 50)) return fail(ctx, OOC_E_INVALID, "variable too large");
  if (kind < OOC_INPUT || kind > OOC_TEMP) return fail(ctx, OOC_E_INVALID, "unknown kind");
  ctx->vars.push_back(Var{bytes, kind});
  ctx->produced.push_back(kind == OOC_INPUT || kind == OOC_PARAM || kind == OOC_STATE);
  if (out_id) *out_id = (int64_t)ctx->vars.size() - 1;
  return OOC_OK;
}

ooc_status ooc_add_fn(ooc_ctx* ctx, int32_t op, const int64_t* vars, const uint8_t* access,
                      int32_t n, const int64_t* attrs, int32_t n_attrs, int64_t* out_id) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, REGISTERING, "ooc_add_fn");
  if (n <= 0 || !vars || !access) return fail(ctx, OOC_E_INVALID, "a function needs variables");
  if (n_attrs < 0 || (n_attrs > 0 && !attrs)) return fail(ctx, OOC_E_INVALID, "bad attributes");
  Fn fn;
  fn.op = op;
  for (int32_t j = 0; j < n; ++j) {
    const int64_t v = vars[j];
    if (v < 0 || v >= (int64_t)ctx->vars.size())
      return fail(ctx, OOC_E_INVALID, "unknown variable " + std::to_string(v));
    if (access[j] < OOC_R || access[j] > OOC_RW)
      return fail(ctx, OOC_E_INVALID, "bad access flag");
    bool merged = false;
    for (FnVar& fv : fn.vars)
      if (fv.var == v) {
        fv.access |= access[j];
        merged = true;
      }
    if (!merged) fn.vars.push_back(FnVar{v, access[j]});
  }
  fn.attrs.assign(attrs, attrs + n_attrs);
  for (const FnVar& fv : fn.vars) {
    if (ctx->vars[fv.var].kind == OOC_INPUT && (fv.access & OOC_W))
      return fail(ctx, OOC_E_INVALID, "function writes input variable " + std::to_string(fv.var));
    if (!ctx->produced[fv.var] && fv.access != OOC_W)
      return fail(ctx, OOC_E_INVALID,
                  "function reads variable " + std::to_string(fv.var) + " before it is written");
  }
  std::string e = check_fn(ctx->vars, fn);
  if (!e.empty()) return fail(ctx, OOC_E_INVALID, e);
  for (const FnVar& fv : fn.vars) ctx->produced[fv.var] = 1;
  ctx->fns.push_back(std::move(fn));
  if (out_id) *out_id = (int64_t)ctx->fns.size() - 1;
  return OOC_OK;
}

ooc_status ooc_set_budget(ooc_ctx* ctx, uint64_t bytes) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, REGISTERING, "ooc_set_budget");
  if (bytes == 0) return fail(ctx, OOC_E_INVALID, "budget must be positive");
  ctx->budget = bytes;
  return OOC_OK;
}

ooc_status ooc_set_window(ooc_ctx* ctx, uint64_t bytes) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, REGISTERING, "ooc_set_window");
  ctx->window = bytes;
  ctx->window_set = true;
  return OOC_OK;
}

ooc_status ooc_set_chunk(ooc_ctx* ctx, uint64_t bytes) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, REGISTERING, "ooc_set_chunk");
  if (bytes == 0 || bytes > (1ull << 40)) return fail(ctx, OOC_E_INVALID, "bad chunk size");
  ctx->chunk = bytes;
  return OOC_OK;
}

ooc_status ooc_set_policy(ooc_ctx* ctx, int32_t policy) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, REGISTERING, "ooc_set_policy");
  if (policy != OOC_POLICY_CANCEL && policy != OOC_POLICY_LITERAL)
    return fail(ctx, OOC_E_INVALID, "unknown policy");
  ctx->policy = policy;
  return OOC_OK;
}

ooc_status ooc_set_wait_order(ooc_ctx* ctx, int32_t order) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, REGISTERING, "ooc_set_wait_order");
  if (order != OOC_WAIT_OLDEST && order != OOC_WAIT_FURTHEST)
    return fail(ctx, OOC_E_INVALID, "unknown wait order");
  ctx->wait_order = order;
  return OOC_OK;
}

ooc_status ooc_set_layout(ooc_ctx* ctx, int32_t layout) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, REGISTERING, "ooc_set_layout");
  if (layout != OOC_LAYOUT_POOL && layout != OOC_LAYOUT_BESTFIT)
    return fail(ctx, OOC_E_INVALID, "unknown device layout");
  ctx->layout = layout;
  return OOC_OK;
}

ooc_status ooc_set_host_limit(ooc_ctx* ctx, uint64_t bytes) {
  REQUIRE_CTX(ctx);
  if (ctx->stage == PREPARED) return fail(ctx, OOC_E_STATE, "ooc_set_host_limit after ooc_prepare");
  if (bytes == 0) return fail(ctx, OOC_E_INVALID, "host limit of 0 bytes");
  ctx->host_limit = bytes;
  return OOC_OK;
}

ooc_status ooc_set_swapout_depth(ooc_ctx* ctx, int64_t depth) {
  REQUIRE_CTX(ctx);
  if (depth < 0) return fail(ctx, OOC_E_INVALID, "negative swap-out depth");
  ctx->swapout_depth = depth;
  return OOC_OK;
}

ooc_status ooc_set_fixed_distance(ooc_ctx* ctx, int64_t swapin_ahead, int64_t swapout_threshold) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, REGISTERING, "ooc_set_fixed_distance");
  const bool off = swapin_ahead == -1 && swapout_threshold == -1;
  if (!off && (swapin_ahead < 0 || swapout_threshold < 0))
    return fail(ctx, OOC_E_INVALID, "swapin_ahead and swapout_threshold must both be >= 0, "
                                    "or both -1");
  ctx->ahead = swapin_ahead;
  ctx->threshold = swapout_threshold;
  return OOC_OK;
}

ooc_status ooc_build_schedule(ooc_ctx* ctx) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, REGISTERING, "ooc_build_schedule");
  if (ctx->fns.empty()) return fail(ctx, OOC_E_INVALID, "empty function sequence");
  ctx->incore = ctx->budget == OOC_UNLIMITED;
  Schedule s;
  if (ctx->incore) {
    build_incore(ctx->vars, ctx->fns, ctx->chunk, &s);
  } else {
    const uint64_t window = ctx->window_set ? ctx->window : ctx->budget / 2;
    std::string err;
    ooc_status st = build_schedule(ctx->vars, ctx->fns, ctx->budget, window, ctx->chunk,
                                   ctx->policy, &s, &err, ctx->ahead, ctx->threshold,
                                   ctx->wait_order);
    if (st) return fail(ctx, st, err);
  }
  ctx->sched = std::move(s);
  build_plan(ctx->vars, ctx->sched, ctx->incore, ctx->chunk, &ctx->plan);
  const uint64_t pool_chunks_used = ctx->plan.max_chunks_used;
  if (ctx->layout == OOC_LAYOUT_BESTFIT)
    bestfit_layout(ctx->vars, 256, &ctx->plan, &ctx->iv_off, &ctx->heap_extent);
  ooc_stats& st = ctx->stats;
  st = ooc_stats{};
  st.budget = ctx->budget;
  st.chunk = ctx->chunk;
  st.peak_accounted = ctx->sched.peak;
  st.sched_h2d_bytes = ctx->sched.h2d;
  st.sched_d2h_bytes = ctx->sched.d2h;
  st.max_chunks_used = pool_chunks_used;
  st.n_intervals = ctx->plan.intervals.size();
  st.incore = ctx->incore;
  st.policy = ctx->policy;
  ctx->stage = BUILT;
  return OOC_OK;
}

ooc_status ooc_schedule_get(const ooc_ctx* ctx, ooc_op* buf, uint64_t cap, uint64_t* n) {
  REQUIRE_CTX(ctx);
  REQUIRE_OUT(ctx, n);
  REQUIRE_BUF(ctx, buf, cap);
  REQUIRE_BUILT(ctx);
  *n = ctx->sched.ops.size();
  for (uint64_t k = 0; k < cap && k < *n; ++k) {
    const Op& o = ctx->sched.ops[k];
    buf[k] = ooc_op{o.fn, o.phase, o.kind, 0, o.var, o.held};
  }
  return OOC_OK;
}

ooc_status ooc_schedule_windows(const ooc_ctx* ctx, int64_t* buf, uint64_t cap, uint64_t* n) {
  REQUIRE_CTX(ctx);
  REQUIRE_OUT(ctx, n);
  REQUIRE_BUF(ctx, buf, cap);
  REQUIRE_BUILT(ctx);
  *n = ctx->sched.windows.size();
  for (uint64_t k = 0; k < cap && k < *n; ++k) buf[k] = ctx->sched.windows[k];
  return OOC_OK;
}

ooc_status ooc_incore_peak(const ooc_ctx* ctx, uint64_t* bytes) {
  REQUIRE_CTX(ctx);
  REQUIRE_OUT(ctx, bytes);
  *bytes = incore_peak(ctx->vars, ctx->fns, ctx->chunk);
  return OOC_OK;
}

ooc_status ooc_working_set_max(const ooc_ctx* ctx, uint64_t* bytes) {
  REQUIRE_CTX(ctx);
  REQUIRE_OUT(ctx, bytes);
  *bytes = working_set_max(ctx->vars, ctx->fns, ctx->chunk);
  return OOC_OK;
}

ooc_status ooc_bestfit_extent(const ooc_ctx* ctx, uint64_t align, uint64_t* extent,
                              uint64_t* peak_live) {
  REQUIRE_CTX(ctx);
  REQUIRE_OUT(ctx, extent);
  REQUIRE_OUT(ctx, peak_live);
  REQUIRE_BUILT(ctx);
  if (align == 0 || (align & (align - 1)))
    return fail(ctx, OOC_E_INVALID, "ooc_bestfit_extent: align must be a power of two");
  bestfit_extent(ctx->vars, ctx->plan, align, extent, peak_live);
  return OOC_OK;
}

ooc_status ooc_plan_intervals(const ooc_ctx* ctx, ooc_interval* buf, uint64_t cap, uint64_t* n) {
  REQUIRE_CTX(ctx);
  REQUIRE_OUT(ctx, n);
  REQUIRE_BUF(ctx, buf, cap);
  REQUIRE_BUILT(ctx);
  *n = ctx->plan.intervals.size();
  int64_t first = 0;
  for (uint64_t k = 0; k < *n; ++k) {
    const Interval& iv = ctx->plan.intervals[k];
    if (k < cap)
      buf[k] = ooc_interval{iv.var, iv.open, iv.close, first, (int64_t)iv.chunks.size()};
    first += (int64_t)iv.chunks.size();
  }
  return OOC_OK;
}

ooc_status ooc_plan_chunks(const ooc_ctx* ctx, int32_t* buf, uint64_t cap, uint64_t* n) {
  REQUIRE_CTX(ctx);
  REQUIRE_OUT(ctx, n);
  REQUIRE_BUF(ctx, buf, cap);
  REQUIRE_BUILT(ctx);
  uint64_t k = 0;
  for (const Interval& iv : ctx->plan.intervals)
    for (int32_t c : iv.chunks) {
      if (k < cap) buf[k] = c;
      ++k;
    }
  *n = k;
  return OOC_OK;
}

ooc_status ooc_prepare(ooc_ctx* ctx) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, BUILT, "ooc_prepare");
  if (ctx->device < 0)
    return fail(ctx, OOC_E_UNSUPPORTED, "host-only context: no device to prepare");
  ooc_status s = prepare(ctx);
  if (s) {
    std::string keep = ctx->err;
    release_device(ctx);
    ctx->err = keep;
    return s;
  }
  ctx->stage = PREPARED;
  return OOC_OK;
}

ooc_status ooc_host_ptr(ooc_ctx* ctx, int64_t var, void** p) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, PREPARED, "ooc_host_ptr");
  REQUIRE_OUT(ctx, p);
  if (var < 0 || var >= (int64_t)ctx->vars.size())
    return fail(ctx, OOC_E_INVALID, "ooc_host_ptr: unknown variable " + std::to_string(var));
  if (ctx->vars[var].kind == OOC_TEMP)
    return fail(ctx, OOC_E_INVALID, "a TEMP variable has no host slot");
  *p = ctx->host_slot[var];
  return OOC_OK;
}

ooc_status ooc_upload(ooc_ctx* ctx) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, PREPARED, "ooc_upload");
  return transfer_resident(ctx, true);
}

ooc_status ooc_download(ooc_ctx* ctx) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, PREPARED, "ooc_download");
  return transfer_resident(ctx, false);
}

ooc_status ooc_step(ooc_ctx* ctx, float lr, float momentum, float* loss_out) {
  REQUIRE_CTX(ctx);
  REQUIRE_STAGE(ctx, PREPARED, "ooc_step");
  if (!std::isfinite(lr) || !std::isfinite(momentum))
    return fail(ctx, OOC_E_INVALID, "lr and momentum must be finite");
  return step(ctx, lr, momentum, loss_out);
}

ooc_status ooc_get_stats(const ooc_ctx* ctx, ooc_stats* out) {
  REQUIRE_CTX(ctx);
  REQUIRE_OUT(ctx, out);
  REQUIRE_BUILT(ctx);
  *out = ctx->stats;
  return OOC_OK;
}

ooc_status ooc_link_probe(int32_t hip_device, uint64_t bytes, int32_t reps, double* h2d_gbs,
                          double* d2h_gbs, double* both_gbs) {
  if (!h2d_gbs || !d2h_gbs || !both_gbs || bytes == 0 || reps <= 0 || hip_device < 0) {
    g_create_error = "ooc_link_probe: bad arguments";
    return OOC_E_INVALID;
  }
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || hip_device >= n) {
    g_create_error = "ooc_link_probe: device not available";
    return OOC_E_DEVICE;
  }
  std::string err;
  ooc_status s = link_probe(hip_device, bytes, reps, h2d_gbs, d2h_gbs, both_gbs, &err);
  if (s) g_create_error = err;
  return s;
}

ooc_status ooc_wgrad_slices(int32_t op, const int64_t* attrs, int32_t n_attrs, int64_t* slices) {
  if (!slices || !attrs) {
    g_create_error = "ooc_wgrad_slices: NULL argument";
    return OOC_E_INVALID;
  }
  for (int32_t j = 0; j < n_attrs; ++j)
    if (attrs[j] < 0 || attrs[j] > (int64_t(1) << 40)) {
      g_create_error = "ooc_wgrad_slices: attribute out of range";
      return OOC_E_INVALID;
    }
  if (op == OOC_OP_CONV_BWD_W && n_attrs >= 11) {
    const int64_t* a = attrs;   // N H W C K R S stride pad P Q
    if (a[0] < 1 || a[3] < 1 || a[4] < 1 || a[5] < 1 || a[6] < 1 || a[9] < 1 || a[10] < 1) {
      g_create_error = "ooc_wgrad_slices: empty convolution";
      return OOC_E_INVALID;
    }
    *slices = wgrad_slices(a[4], a[5] * a[6] * a[3], a[0] * a[9] * a[10], a[3]);
    return OOC_OK;
  }
  if (op == OOC_OP_LINEAR_BWD_W && n_attrs >= 3) {
    const int64_t* a = attrs;   // M K N: dW [N][K] reduced over M rows
    if (a[0] < 1 || a[1] < 1 || a[2] < 1) {
      g_create_error = "ooc_wgrad_slices: empty dense layer";
      return OOC_E_INVALID;
    }
    *slices = wgrad_slices(a[2], a[1], a[0], -1);
    return OOC_OK;
  }
  g_create_error = "ooc_wgrad_slices: op must be CONV_BWD_W (11 attributes) or LINEAR_BWD_W (3)";
  return OOC_E_INVALID;
}

ooc_status ooc_fn_times(const ooc_ctx* ctx, double* buf, uint64_t cap, uint64_t* n) {
  REQUIRE_CTX(ctx);
  REQUIRE_OUT(ctx, n);
  REQUIRE_BUF(ctx, buf, cap);
  if (ctx->fn_ms.empty()) return fail(ctx, OOC_E_STATE, "ooc_fn_times before the first step");
  *n = ctx->fn_ms.size();
  for (uint64_t k = 0; k < cap && k < *n; ++k) buf[k] = ctx->fn_ms[k];
  return OOC_OK;
}

ooc_status ooc_timeline(ooc_ctx* ctx, ooc_span* buf, uint64_t cap, uint64_t* n) {
  REQUIRE_CTX(ctx);
  REQUIRE_OUT(ctx, n);
  REQUIRE_BUF(ctx, buf, cap);
  std::vector<ooc_span> t;
  ooc_status st = timeline(ctx, &t);
  if (st) return st;
  *n = t.size();
  for (uint64_t k = 0; k < cap && k < *n; ++k) buf[k] = t[k];
  return OOC_OK;
}

}  // extern "C"
