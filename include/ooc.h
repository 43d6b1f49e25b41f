/*
 * ooc.h -- out-of-core training step on one MI355X (gfx950).
 *
 * C interface of the method of Hayakawa & Narihira, "Out-of-core training for
 * extremely large-scale neural networks with adaptive window-based
 * scheduling": a network is given as a topologically ordered function
 * sequence f_1..f_N, each function using a set of variables with known byte
 * sizes (Section 2; Section 3, variable-sequence); under a device-memory
 * budget the library schedules swap-ins and swap-outs with the adaptive
 * schedule-window (Section 3, Fig. 2), backs device memory with a pool of
 * equal physical chunks mapped into per-allocation virtual ranges
 * (Section 4, eq. 1 and 2), and runs forward, backward and SGD update of one
 * training step with its own HIP kernels while the swaps run on two copy
 * streams.
 *
 * Conventions (every call):
 *  - No exception or signal crosses this interface.  Every failure returns a
 *    negative ooc_status and sets a message readable with ooc_last_error():
 *    on the context for calls that take one (const queries included), else
 *    (a NULL context, ooc_create, ooc_link_probe, ooc_wgrad_slices) on
 *    ooc_last_error(NULL).  A NULL out-pointer, or a NULL buffer with a
 *    nonzero capacity, is OOC_E_INVALID; a query made before the stage it
 *    needs is OOC_E_STATE.
 *  - A context is driven in this order: create -> add_var / add_fn ->
 *    set_* -> build_schedule -> prepare -> (host_ptr, upload, step,
 *    download, get_stats)* -> destroy.  A call out of order returns
 *    OOC_E_STATE and changes nothing.  set_* after build_schedule returns
 *    OOC_E_STATE.
 *  - A context is not thread-safe; two contexts may be used from two threads.
 *  - The library owns all device memory (the chunk pool), all pinned host
 *    memory (one slot per host-backed variable) and its three non-blocking
 *    streams (compute, host-to-device, device-to-host; default priority).
 *    Buffers passed in by the caller (ids, access flags, attributes, op and
 *    plan buffers) are read or written only during the call.
 *  - Sizes are bytes; ids are 0-based in registration order.
 */
#ifndef OOC_H
#define OOC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OOC_API_VERSION 1

typedef struct ooc_ctx ooc_ctx;
typedef int32_t ooc_status;

enum {
  OOC_OK = 0,
  OOC_E_INVALID = -1,     /* bad argument or ill-formed function sequence */
  OOC_E_STATE = -2,       /* call out of order */
  OOC_E_INFEASIBLE = -3,  /* budget below the footprint of one function */
  OOC_E_HOST_OOM = -4,    /* pinned host memory could not be allocated */
  OOC_E_DEVICE = -5,      /* a HIP call failed (message names it) */
  OOC_E_UNSUPPORTED = -6  /* valid request this build cannot serve */
};

/* Variable kinds.  INPUT, PARAM and STATE hold a value on the host when a
 * step starts; PARAM, STATE and OUTPUT must hold their final value on the
 * host when it ends; TEMP lives only inside a step. */
enum { OOC_INPUT = 0, OOC_PARAM = 1, OOC_STATE = 2, OOC_OUTPUT = 3, OOC_TEMP = 4 };

/* Access of a function to one of its variables. */
enum { OOC_R = 1, OOC_W = 2, OOC_RW = 3 };

/* What happens when a variable re-enters the window while its swap-out is
 * still pending (the paper is silent, Section 3): CANCEL keeps the device
 * copy; LITERAL treats the variable as already on the host (binary state of
 * Section 3) and swaps it in again into fresh memory. */
enum { OOC_POLICY_CANCEL = 0, OOC_POLICY_LITERAL = 1 };
enum { OOC_WAIT_OLDEST = 0, OOC_WAIT_FURTHEST = 1 };

/* Schedule ops and the phase of f_i they belong to (PRE: before f_i runs;
 * POST: after it; END: after f_N). */
enum { OOC_SWAPIN = 0, OOC_ALLOC = 1, OOC_CANCEL = 2, OOC_WAIT_OUT = 3, OOC_SWAPOUT = 4,
       OOC_FREE = 5 };
enum { OOC_PRE = 0, OOC_POST = 1, OOC_END = 2 };

/* Budget or window value meaning "no limit".  A budget of OOC_UNLIMITED
 * selects in-core mode: every PARAM/STATE/INPUT/OUTPUT variable stays on the
 * device for the whole step, TEMPs live from first to last use, and no byte
 * moves over the host link inside ooc_step (ooc_upload / ooc_download move
 * the persistent variables instead). */
#define OOC_UNLIMITED UINT64_MAX

/* Operations a function runs.  Every image tensor is NHWC float32, conv
 * weights [K][R][S][C], dense weights [out][in].  Attributes are int64, in the
 * order listed; variables are listed in the order given (access in
 * brackets).  add_fn checks every variable's byte size against the
 * attributes and rejects any mismatch with OOC_E_INVALID.
 *
 *  NOOP          no kernel (pure scheduling studies).             attrs: -
 *  LINEAR_FWD    Y = X W^T + b        X[R] W[R] b[R] Y[W]          M K N
 *  LINEAR_BWD_W  dW = dY^T X, db = sum_rows dY
 *                                     X[R] dY[R] dW[W] db[W] [part[W]]
 *                                                                  M K N slices
 *                (rows cut into slices; part = slices partial dW copies then
 *                slices partial db copies, present iff slices > 1)
 *  LINEAR_BWD_X  dX = dY W            W[R] dY[R] dX[W]             M K N
 *  RELU_FWD      Y = max(X, 0)        X[R] Y[W]                    n
 *  RELU_BWD      dX = dY [Y > 0]      Y[R] dY[R] dX[W]             n
 *  ADD           Y = A + B            A[R] B[R] Y[W]               n
 *  ACC           A = A + B (in place: the sum of gradient contributions
 *                accumulated into the running one)
 *                                     A[RW] B[R]                   n
 *  SOFTMAX_CE    mean softmax cross-entropy over N rows; loss holds the N
 *                per-row losses then their mean (N + 1 floats), dlogits =
 *                (softmax - onehot) / N; labels int32, an out-of-range label
 *                gives a NaN row loss and a zero gradient row
 *                                     logits[R] labels[R] loss[W] dlogits[W]
 *                                                                  N classes
 *  SGD           per parameter: w -= lr g, or with momentum buffers
 *                v = mu v + g, w -= lr v (lr, mu given to ooc_step)
 *                                     (p[RW] g[R] [v[RW]])...      count has_momentum
 *  CONV_FWD      cross-correlation, zero padding
 *                                     X[R] W[R] Y[W]               N H W C K R S stride pad P Q
 *  CONV_BWD_W    dW                   X[R] dY[R] dW[W] [part[W]]   N H W C K R S stride pad P Q slices
 *                (part = slices partial dW copies, present iff slices > 1)
 *  CONV_BWD_X    dX                   W[R] dY[R] dX[W]             N H W C K R S stride pad P Q
 *  BN_FWD        training-mode batch normalisation over rows = N H W, eps 1e-5;
 *                stats = mean[C] invstd[C] then 2 C floats per row slice
 *                                     X[R] gamma[R] beta[R] Y[W] stats[W]   rows C slices
 *  BN_BWD                             X[R] gamma[R] stats[RW] dY[R] dX[W] dgamma[W] dbeta[W]
 *                                                                  rows C slices
 *  MAXPOOL_FWD   window max, first maximal tap wins, idx = r k + s (uint8)
 *                                     X[R] Y[W] idx[W]             N H W C k stride pad P Q
 *  MAXPOOL_BWD                        idx[R] dY[R] dX[W]           N H W C k stride pad P Q
 *  AVGPOOL_FWD   global average over H W   X[R] Y[W]               N H W C
 *  AVGPOOL_BWD                        dY[R] dX[W]                  N H W C
 *  EMBED_FWD     Y[r] = E[ids[r]] + pos[r mod T] for the B T token rows;
 *                ids int32 (an id outside [0, V) gives a NaN row)
 *                                     ids[R] E[R] pos[R] Y[W]          B T V d
 *  EMBED_BWD     dE[v] = sum of dY rows of tokens with id v (token order),
 *                dpos[t] = sum over b of dY[b T + t]
 *                                     ids[R] dY[R] dE[W] dpos[W]       B T V d
 *  LAYERNORM_FWD per row over d features, biased variance, eps 1e-5;
 *                stats = mean[rows] rstd[rows] then 2 d floats per row slice
 *                                     X[R] gamma[R] beta[R] Y[W] stats[W]   rows d slices
 *  LAYERNORM_BWD                      X[R] gamma[R] stats[RW] dY[R] dX[W] dgamma[W] dbeta[W]
 *                                                                      rows d slices
 *  GELU_FWD      Y = X Phi(X) (exact, normal CDF)    X[R] Y[W]          n
 *  GELU_BWD      dX = dY (Phi(X) + X phi(X))         X[R] dY[R] dX[W]   n
 *  ATTENTION_FWD qkv [B T][3 H dh] holds q, k, v as column thirds, head h in
 *                columns h dh .. (h+1) dh of each; P[b][h] = softmax(q k^T /
 *                sqrt(dh)) with keys after the query masked when causal;
 *                Y [B T][H dh] = P v                qkv[R] P[W] Y[W]    B T H dh causal
 *  ATTENTION_BWD dqkv of the above.  P is not kept from the forward: the
 *                function recomputes it into its own P (bit for bit the
 *                forward's, same kernels); dS is scratch of P's size
 *                                     qkv[R] P[W] dY[R] dqkv[W] dS[W]  B T H dh causal
 *  CONCAT_FWD    channel concatenation of k = 1..64 row-major tensors with
 *                the same rows: Y[r] = [X_1[r] | ... | X_k[r]]
 *                                     X_1[R] .. X_k[R] Y[W]            rows c_1 .. c_k
 *  CONCAT_BWD    dX_j[r] = the c_j columns of dY[r] that X_j filled
 *                                     dY[R] dX_1[W] .. dX_k[W]         rows c_1 .. c_k
 *  UPSAMPLE_FWD  nearest, factor 2: Y[n][2h+i][2w+j] = X[n][h][w]
 *                                     X[R] Y[W]                        N H W C (of X)
 *  UPSAMPLE_BWD  dX[n][h][w] = sum over i, j in {0, 1} of dY[n][2h+i][2w+j],
 *                added in the order (0,0) (0,1) (1,0) (1,1)
 *                                     dY[R] dX[W]                      N H W C (of dX)
 *  MIX           swap-integrity test op on uint32 words (sizes multiple of
 *                4): the last variable y is the only one written (W or RW),
 *                the others are read; y[j] = seed ^ (j * 2654435761) ^ sum
 *                over read variables x (y itself too when RW) of
 *                x[j mod len(x)], sums and products wrapping in uint32
 *                                     x...[R] y[W|RW]              seed
 */
enum {
  OOC_OP_NOOP = 0,
  OOC_OP_LINEAR_FWD = 1,
  OOC_OP_LINEAR_BWD_W = 2,
  OOC_OP_LINEAR_BWD_X = 3,
  OOC_OP_RELU_FWD = 4,
  OOC_OP_RELU_BWD = 5,
  OOC_OP_ADD = 6,
  OOC_OP_SOFTMAX_CE = 7,
  OOC_OP_SGD = 8,
  OOC_OP_CONV_FWD = 9,
  OOC_OP_CONV_BWD_W = 10,
  OOC_OP_CONV_BWD_X = 11,
  OOC_OP_BN_FWD = 12,
  OOC_OP_BN_BWD = 13,
  OOC_OP_MAXPOOL_FWD = 14,
  OOC_OP_MAXPOOL_BWD = 15,
  OOC_OP_AVGPOOL_FWD = 16,
  OOC_OP_AVGPOOL_BWD = 17,
  OOC_OP_MIX = 18,
  OOC_OP_EMBED_FWD = 19,
  OOC_OP_EMBED_BWD = 20,
  OOC_OP_LAYERNORM_FWD = 21,
  OOC_OP_LAYERNORM_BWD = 22,
  OOC_OP_GELU_FWD = 23,
  OOC_OP_GELU_BWD = 24,
  OOC_OP_ATTENTION_FWD = 25,
  OOC_OP_ATTENTION_BWD = 26,
  OOC_OP_CONCAT_FWD = 27,
  OOC_OP_CONCAT_BWD = 28,
  OOC_OP_UPSAMPLE_FWD = 29,
  OOC_OP_UPSAMPLE_BWD = 30,
  OOC_OP_ACC = 31,
  OOC_OP_COUNT = 32
};

/* One schedule op.  fn = N for END ops; held = budget bytes held after it
 * (chunk-rounded sizes). */
typedef struct {
  int32_t fn;
  uint8_t phase;
  uint8_t kind;
  uint16_t reserved;
  int64_t var;
  uint64_t held;
} ooc_op;

/* One residency interval of the chunk plan: a device copy of `var` opened by
 * op `open` (-1: resident for the whole step, in-core mode) and closed by op
 * `close` (-1: never closed), backed by `n_chunks` chunks listed from
 * `first_chunk` in the array ooc_plan_chunks returns. */
typedef struct {
  int64_t var;
  int64_t open;
  int64_t close;
  int64_t first_chunk;
  int64_t n_chunks;
} ooc_interval;

typedef struct {
  uint64_t budget;            /* as set (OOC_UNLIMITED in in-core mode) */
  uint64_t chunk;             /* m_c in use */
  uint64_t peak_accounted;    /* max chunk-rounded bytes held by the schedule */
  uint64_t pool_chunks;       /* physical chunks created (0 with OOC_LAYOUT_BESTFIT) */
  uint64_t pool_bytes;        /* pool_chunks * chunk: the device bytes the pool owns (the
                                 best-fit heap's extent with OOC_LAYOUT_BESTFIT) */
  uint64_t max_chunks_used;   /* most chunks mapped to live intervals at once */
  uint64_t device_bytes_delta;/* hipMemGetInfo used-bytes delta across prepare */
  uint64_t host_bytes;        /* pinned host arena */
  uint64_t sched_h2d_bytes;   /* bytes the schedule swaps in */
  uint64_t sched_d2h_bytes;   /* bytes the schedule swaps out */
  uint64_t h2d_bytes;         /* bytes the last step copied host->device */
  uint64_t d2h_bytes;         /* bytes the last step copied device->host (cancelled and
                                 clean swap-outs need no copy) */
  uint64_t n_intervals;
  uint64_t n_mappings;        /* hipMemMap calls made by prepare */
  double prepare_ms;
  double step_ms;             /* last step, host wall clock */
  double step_gpu_ms;         /* last step, first to last event on the compute stream */
  double h2d_busy_ms;         /* sum of host->device copy durations, last step */
  double d2h_busy_ms;         /* sum of device->host copy durations, last step */
  double compute_busy_ms;     /* sum of kernel-phase durations, last step */
  int32_t incore;
  int32_t policy;
  uint64_t spill_bytes;       /* pageable host homes of TEMPs beyond the host limit */
  uint64_t staged_h2d_bytes;  /* of h2d_bytes: copied through the staging slots */
  uint64_t staged_d2h_bytes;  /* of d2h_bytes: copied through the staging slots */
} ooc_stats;

/* Creates a context bound to HIP device `hip_device`, or a host-only
 * context for `hip_device` = -1 (registration, schedule and plan queries
 * only; prepare returns OOC_E_UNSUPPORTED).  *out receives the context. */
ooc_status ooc_create(int32_t hip_device, ooc_ctx **out);

/* Frees the pool, pinned arena, streams and events.  NULL is accepted. */
void ooc_destroy(ooc_ctx *ctx);

/* Message of the last failing call on ctx (or of the last failing
 * ooc_create when ctx is NULL); owned by the library, valid until the next
 * call on ctx. */
const char *ooc_last_error(const ooc_ctx *ctx);

/* Registers a variable of `bytes` (> 0) bytes and kind OOC_INPUT..OOC_TEMP
 * (Section 3: variable set V with sizes b_v). */
ooc_status ooc_add_var(ooc_ctx *ctx, uint64_t bytes, int32_t kind, int64_t *out_id);

/* Appends f_i to the function sequence (Section 2: topological order is the
 * caller's): operation `op`, its `n` variables with their access flags in
 * the operation's order, and `n_attrs` attributes (copied).  A variable
 * listed twice is merged (first position, accesses or-ed).  Returns
 * OOC_E_INVALID if the sequence breaks a rule: an INPUT written, a TEMP or
 * OUTPUT read before it is written, sizes that do not match the attributes. */
ooc_status ooc_add_fn(ooc_ctx *ctx, int32_t op, const int64_t *vars, const uint8_t *access,
                      int32_t n, const int64_t *attrs, int32_t n_attrs, int64_t *out_id);

/* Physical device-memory budget in bytes (Section 3; Fig. 3 "budget"), or
 * OOC_UNLIMITED for in-core mode.  Default OOC_UNLIMITED. */
ooc_status ooc_set_budget(ooc_ctx *ctx, uint64_t bytes);

/* schedule-window W in bytes (Section 3), OOC_UNLIMITED allowed.  Default:
 * half the budget. */
ooc_status ooc_set_window(ooc_ctx *ctx, uint64_t bytes);

/* Physical chunk size m_c (Section 4).  Must be a multiple of the device's
 * allocation granularity once prepared; default 2 MiB. */
ooc_status ooc_set_chunk(ooc_ctx *ctx, uint64_t bytes);

/* Fixed-distance scheduling rule of LMS as Section 2 describes it, in place
 * of the byte window: a variable is swapped in when it comes within
 * `swapin_ahead` functions of its next use, and after a use it is kept on the
 * device when its next use is at most `swapout_threshold` functions away,
 * otherwise swapped out (the text prints this test as "<= threshold"; it is
 * read as "> threshold", which keeps the variables needed soon).  Budget waits
 * and policies are those of the adaptive scheduler.  Variables kept by the
 * threshold are not waited for, so a tight budget can be infeasible, as with
 * LMS.  Both -1 (default) selects the schedule-window rule; otherwise both
 * must be >= 0.  Baseline for comparisons. */
ooc_status ooc_set_fixed_distance(ooc_ctx *ctx, int64_t swapin_ahead, int64_t swapout_threshold);

/* OOC_POLICY_CANCEL (default) or OOC_POLICY_LITERAL. */
ooc_status ooc_set_policy(ooc_ctx *ctx, int32_t policy);

/* Which pending swap-out a budget wait completes (step (b) of Section 3).
 * OOC_WAIT_OLDEST (default): the oldest, as the paper's Fig. 2 does.
 * OOC_WAIT_FURTHEST: the one whose variable is used again furthest ahead in
 * the variable-sequence (write-backs of variables never used again first,
 * ties to the oldest), so that swap-outs of variables needed sooner stay
 * pending and can still be cancelled when the window reaches them.  The
 * paper leaves the order of swap-outs as future work (Section 6); this is one
 * answer to it.  The waits at the end of the step stay oldest first.
 * Registering stage only; OOC_E_INVALID for another value. */
ooc_status ooc_set_wait_order(ooc_ctx *ctx, int32_t order);

/* Device-memory layout.  OOC_LAYOUT_POOL (default): the chunk pool of
 * Section 4, each residency interval in its own virtual range backed by
 * chunks of m_c bytes.  OOC_LAYOUT_BESTFIT: the allocator the pool is
 * compared with (Section 4, Fig. 3): one device allocation, each interval at
 * the offset a contiguous best-fit heap gives it (requests rounded up to 256
 * bytes, as ooc_bestfit_extent replays them).  The schedule, the copies and
 * the results are the same; only the device bytes the layout needs differ
 * (ooc_stats.pool_bytes: the heap's extent).  With this layout
 * ooc_plan_intervals / ooc_plan_chunks list, instead of chunks, the heap
 * segments each interval covers (the heap cut at every interval's first and
 * last byte).  Registering stage only; OOC_E_INVALID for another value. */
enum { OOC_LAYOUT_POOL = 0, OOC_LAYOUT_BESTFIT = 1 };
ooc_status ooc_set_layout(ooc_ctx *ctx, int32_t layout);

/* Most swap-outs in flight on the device-to-host stream during a step: before
 * issuing another one, the host waits for the oldest.  0 = no bound; default
 * 4.  With dozens of device-to-host copies queued behind their event waits,
 * the HIP runtime on MI355X moves them at 7-14 GB/s instead of the link's
 * 57 GB/s; a short queue keeps the full rate.  Any stage; takes effect at the
 * next step. */
ooc_status ooc_set_swapout_depth(ooc_ctx *ctx, int64_t depth);

/* Most bytes of pinned host memory the host arena may take (the CPU-memory
 * cache of Section 1; pinning is what lets the copies run asynchronously at
 * the link's rate).  Persistent slots (INPUT, PARAM, STATE, OUTPUT) are
 * always pinned.  TEMP slots are pinned while they fit under the limit less
 * 2 GiB of staging slots; the others get homes in pageable memory, and their
 * copies move in 32 MiB pieces through the staging slots, host threads
 * copying each piece between slot and home.  Results are identical; only the
 * transfer rate of the staged bytes changes.  For hosts that pin less memory
 * than a tight budget leaves on the host.  Default OOC_UNLIMITED (everything
 * pinned).  OOC_E_INVALID for 0, OOC_E_STATE after ooc_prepare; ooc_prepare
 * returns OOC_E_HOST_OOM when the persistent slots and the staging slots alone
 * exceed the limit. */
ooc_status ooc_set_host_limit(ooc_ctx *ctx, uint64_t bytes);

/* Runs the scheduler of Section 3 (host only).  OOC_E_INFEASIBLE if one
 * function's variables do not fit in the budget. */
ooc_status ooc_build_schedule(ooc_ctx *ctx);

/* The schedule of Section 3 (Fig. 2, steps (a)-(d)) as an op list, in
 * emission order: per function its PRE ops (swap-ins, allocations,
 * cancelled swap-outs, budget waits), then its POST ops (frees and
 * swap-outs), then the END waits.  Copies up to `cap` ops into `buf`
 * (caller-owned; may be NULL when cap is 0); *n receives the total count.
 * OOC_E_STATE before ooc_build_schedule. */
ooc_status ooc_schedule_get(const ooc_ctx *ctx, ooc_op *buf, uint64_t cap, uint64_t *n);

/* Window end r_i (0-based position of the variable-sequence, Section 3) per
 * function.  OOC_E_STATE before ooc_build_schedule. */
ooc_status ooc_schedule_windows(const ooc_ctx *ctx, int64_t *buf, uint64_t cap, uint64_t *n);

/* P_incore: most chunk-rounded bytes live at one function in the in-core
 * plan, the memory an ordinary step needs (the "in-core" baseline the
 * budgets and speeds of Section 5 are measured against); INPUT, PARAM,
 * STATE and OUTPUT count for the whole step, a TEMP from its first to its
 * last use.  WS_max: largest chunk-rounded footprint of one function (no
 * budget below it is feasible, Section 3).  Valid after registration (the
 * chunk size in effect is used). */
ooc_status ooc_incore_peak(const ooc_ctx *ctx, uint64_t *bytes);
ooc_status ooc_working_set_max(const ooc_ctx *ctx, uint64_t *bytes);

/* Chunk plan (Section 4): residency intervals in opening order and the
 * concatenated chunk ids they map (freed chunks reused in the order they were
 * freed, a new chunk id only when none is free).  Valid
 * after build_schedule; host only. */
ooc_status ooc_plan_intervals(const ooc_ctx *ctx, ooc_interval *buf, uint64_t cap, uint64_t *n);

/* The comparison of Section 4 (host only, after build_schedule): the same
 * residency intervals served by one contiguous best-fit heap instead of the
 * chunk pool.  Each request is the variable's size rounded up to `align` (a
 * power of two); it takes the smallest free hole that holds it (lowest
 * address on ties), else the end of the heap, starting in the free tail.
 * *extent receives the highest address used (the device bytes such a heap
 * needs), *peak_live the most bytes live at once; extent - peak_live is the
 * external fragmentation the chunk pool avoids.  OOC_E_STATE before
 * build_schedule, OOC_E_INVALID for a bad alignment. */
ooc_status ooc_bestfit_extent(const ooc_ctx *ctx, uint64_t align, uint64_t *extent,
                              uint64_t *peak_live);
ooc_status ooc_plan_chunks(const ooc_ctx *ctx, int32_t *buf, uint64_t cap, uint64_t *n);

/* Sets up the memory of Section 4: creates the physical chunks (at most
 * budget / m_c of them), maps every residency interval's chunks into its own
 * contiguous virtual range (eq. 1: at most one partly used chunk per
 * interval), and allocates the pinned host arena of Section 1, the streams
 * and the events.  All mapping happens here, once; a step maps nothing.
 * Each chunk and each mapping of a chunk takes one entry of the process's
 * memory-map table (vm.max_map_count, typically 65530): a plan needing more
 * than the entries left returns OOC_E_UNSUPPORTED (choose a larger chunk).
 * Out of core it also makes one 8 MiB copy each way on every copy stream, in
 * a temporary device and pinned buffer freed before it returns (skipped when
 * they cannot be allocated): the runtime sets a stream up for the DMA engines
 * at its first large copy, which blocks the caller for several milliseconds. */
ooc_status ooc_prepare(ooc_ctx *ctx);

/* Pinned host slot of a host-backed variable (INPUT, PARAM, STATE, OUTPUT;
 * a TEMP has none: OOC_E_INVALID) in the CPU memory that serves as the
 * swap target of Section 1.  The caller writes INPUT/PARAM/STATE
 * slots before a step and reads PARAM/STATE/OUTPUT slots after it; the
 * slot stays owned by the library and valid until ooc_destroy. */
ooc_status ooc_host_ptr(ooc_ctx *ctx, int64_t var, void **p);

/* In-core mode: copy every persistent variable host slot -> device
 * (upload) or PARAM/STATE/OUTPUT device -> host slot (download), blocking.
 * Out-of-core mode: the host slots are the variables' home; both are
 * no-ops. */
ooc_status ooc_upload(ooc_ctx *ctx);
ooc_status ooc_download(ooc_ctx *ctx);

/* One blocking training step (the iteration whose time Section 5 reports):
 * all functions in order on the compute stream, the swaps of the Section 3
 * schedule (Fig. 2) on the copy streams, each function started only once
 * its variables are resident and each chunk reused only once its previous
 * occupant's kernels and copies are done.  lr and momentum feed
 * the SGD functions; *loss_out (may be NULL) receives the mean loss of the
 * last SOFTMAX_CE function (NaN if none). */
ooc_status ooc_step(ooc_ctx *ctx, float lr, float momentum, float *loss_out);

/* Statistics of the schedule, the pool and the last step: the quantities
 * Section 5 reports (budget, actual device usage against it as in Fig. 3,
 * bytes swapped, step time).  OOC_E_STATE before ooc_build_schedule. */
ooc_status ooc_get_stats(const ooc_ctx *ctx, ooc_stats *out);

/* Measures the host link the swaps use (the CPU-memory cache of Section 1
 * sits behind it): copies `bytes` between a pinned host buffer and device
 * memory of HIP device `hip_device`, host-to-device, device-to-host and both
 * at once on two streams, `reps` times each, and returns the best rates in
 * GB/s (1e9 bytes/s; *both_gbs counts the bytes of both directions).
 * Allocates and frees its own buffers. */
ooc_status ooc_link_probe(int32_t hip_device, uint64_t bytes, int32_t reps, double *h2d_gbs,
                          double *d2h_gbs, double *both_gbs);

/* Split-K slice count the library's weight-gradient kernels run best with
 * for one function, for the caller to size its partial-sum variable and to
 * pass as the function's `slices` attribute (Section 3: every byte a
 * function touches is one of its variables, so the budget accounts for the
 * partial sums).  `op` is OOC_OP_CONV_BWD_W with the 11 attributes
 * N H W C K R S stride pad P Q, or OOC_OP_LINEAR_BWD_W with M K N (a
 * trailing slices attribute is ignored).  Any count >= 1 gives the same
 * gradient up to the order of its sums; this one fills whole rounds of
 * resident workgroups on the device.  Host only; no context.  OOC_E_INVALID
 * for another op, too few or negative attributes, or an empty shape
 * (message on ooc_last_error(NULL)). */
ooc_status ooc_wgrad_slices(int32_t op, const int64_t *attrs, int32_t n_attrs, int64_t *slices);

/* Duration in milliseconds of each function's kernels in the last step,
 * measured with events on the compute stream right before and after its
 * launches (waits for swap-ins excluded).  buf caller-owned (cap entries);
 * *n receives the function count.  OOC_E_STATE before the first step. */
ooc_status ooc_fn_times(const ooc_ctx *ctx, double *buf, uint64_t cap, uint64_t *n);

/* One entry of the last step's timeline: a function's kernels (kind 0, var
 * -1, bytes 0), a swap-in (kind 1) or a swap-out (kind 2) of variable var
 * issued for function fn.  start_ms is measured from the step's first event
 * on the compute stream, ms is the duration, both from the events recorded
 * around the launches and copies (a swap's wait for its predecessors is not
 * part of it). */
typedef struct {
  int32_t kind;
  int32_t fn;
  int64_t var;
  uint64_t bytes;
  double start_ms;
  double ms;
} ooc_span;

/* Timeline of the last step: every function, then every copy, in issue
 * order.  buf caller-owned (cap entries); *n receives the entry count.
 * OOC_E_STATE before the first step. */
ooc_status ooc_timeline(ooc_ctx *ctx, ooc_span *buf, uint64_t cap, uint64_t *n);

#ifdef __cplusplus
}
#endif

#endif /* OOC_H */
