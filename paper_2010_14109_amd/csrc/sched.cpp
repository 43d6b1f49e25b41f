// Adaptive-window swap scheduler (Section 3, Fig. 2), in-core plan and the
// chunk plan of the virtual-address pool (Section 4).
//
// The variable-sequence v = flatten([V_1..V_N]) is kept as position arrays;
// next[p] is the next position holding the same variable.  Per function f_i
// (first position l, last e):
//   window  r = largest index with sum(b_v[p], p = l..r) <= W (two pointers
//           over prefix sums), then r = max(r, e, r_prev);
//   (a)+(b) admit positions r_prev+1..r: a variable on the host is swapped
//           in, one never produced is allocated, a pending swap-out is
//           cancelled (policy CANCEL); before each admission the oldest
//           pending swap-outs are waited for until it fits in the budget; if
//           nothing is left to wait for, the window ends before it (an error
//           only when the variable belongs to f_i itself);
//   (c)+(d) after f_i: a variable never used again is freed (INPUT, TEMP) or
//           written back (PARAM, STATE, OUTPUT); one used again inside the
//           window is kept; any other is swapped out.
// Which pending swap-out a budget wait completes: the oldest (Fig. 2), or
// with OOC_WAIT_FURTHEST the one whose variable is used again furthest ahead
// (write-backs first, ties to the oldest), so that swap-outs of variables
// needed sooner stay pending and can still be cancelled.
// Budget accounting uses chunk-rounded sizes a_v = ceil(b_v / m_c) m_c
// (eq. 1), so the chunks the pool maps never exceed the budget.
#include <algorithm>
#include <deque>
#include <functional>
#include <map>
#include <queue>
#include <set>

#include "internal.h"

namespace ooc {

static bool persistent(int32_t kind) {
  return kind == OOC_INPUT || kind == OOC_PARAM || kind == OOC_STATE;
}

ooc_status build_schedule(const std::vector<Var>& vars, const std::vector<Fn>& fns,
                          uint64_t budget, uint64_t window, uint64_t chunk, int policy,
                          Schedule* out, std::string* err, int64_t ahead, int64_t threshold,
                          int wait_order) {
  const bool fixed = ahead >= 0;
  const int64_t N = (int64_t)fns.size();
  const int64_t nv = (int64_t)vars.size();
  std::vector<uint64_t> a(nv);
  for (int64_t v = 0; v < nv; ++v) a[v] = round_up(vars[v].bytes, chunk);

  std::vector<int64_t> seq, first(N), last(N), fn_of;
  for (int64_t i = 0; i < N; ++i) {
    first[i] = (int64_t)seq.size();
    for (const FnVar& fv : fns[i].vars) {
      seq.push_back(fv.var);
      fn_of.push_back(i);
    }
    last[i] = (int64_t)seq.size() - 1;
  }
  const int64_t M = (int64_t)seq.size();
  std::vector<int64_t> next(M, -1), seen(nv, -1);
  for (int64_t p = M - 1; p >= 0; --p) {
    next[p] = seen[seq[p]];
    seen[seq[p]] = p;
  }
  std::vector<uint64_t> pre(M + 1, 0);
  for (int64_t p = 0; p < M; ++p) pre[p + 1] = pre[p] + vars[seq[p]].bytes;

  std::vector<uint8_t> state(nv);
  for (int64_t v = 0; v < nv; ++v) state[v] = persistent(vars[v].kind) ? HOST : UNMAT;

  // pending swap-outs, oldest first; cancelled entries are skipped lazily
  struct Entry {
    int64_t var;
    bool alive;
    int64_t next;   // position of the variable's next use, INT64_MAX for none
  };
  std::vector<Entry> fifo;
  size_t head = 0, alive = 0;
  std::vector<int64_t> entry_of(nv, -1);   // CANCEL policy: the variable's pending entry
  std::vector<int32_t> queued(nv, 0);      // live entries per variable

  Schedule s;
  uint64_t held = 0;
  auto emit = [&](int32_t i, uint8_t phase, uint8_t kind, int64_t v) {
    s.ops.push_back(Op{i, phase, kind, v, held});
  };
  auto pop = [&](int32_t i, uint8_t phase, bool furthest) {
    while (!fifo[head].alive) ++head;
    size_t pick = head;
    if (furthest)
      for (size_t q = head + 1; q < fifo.size(); ++q)
        if (fifo[q].alive && fifo[q].next > fifo[pick].next) pick = q;
    const int64_t w = fifo[pick].var;
    fifo[pick].alive = false;
    if (pick == head) ++head;
    --alive;
    --queued[w];
    entry_of[w] = -1;
    held -= a[w];
    // the state follows the newest copy: HOST only when no newer copy exists
    if (state[w] == PEND && queued[w] == 0) state[w] = HOST;
    emit(i, phase, OOC_WAIT_OUT, w);
  };

  int64_t r_prev = -1, r_hat = -1;
  for (int64_t i = 0; i < N; ++i) {
    const int64_t l = first[i], e = last[i];
    if (fixed) {
      r_hat = last[std::min(i + ahead, N - 1)];
    } else {
      if (r_hat < l - 1) r_hat = l - 1;
      while (r_hat + 1 < M && pre[r_hat + 2] - pre[l] <= window) ++r_hat;
    }
    int64_t r = std::max(std::max(r_hat, e), r_prev);

    for (int64_t p = r_prev + 1; p <= r; ++p) {
      const int64_t u = seq[p];
      if (state[u] == DEV) continue;
      if (state[u] == PEND && policy == OOC_POLICY_CANCEL) {
        fifo[entry_of[u]].alive = false;
        entry_of[u] = -1;
        --alive;
        --queued[u];
        state[u] = DEV;
        emit((int32_t)i, OOC_PRE, OOC_CANCEL, u);
        continue;
      }
      const uint64_t need = a[u];
      while (held + need > budget && alive > 0)
        pop((int32_t)i, OOC_PRE, wait_order == OOC_WAIT_FURTHEST);
      if (held + need <= budget) {
        uint8_t kind = OOC_ALLOC;
        if (state[u] != UNMAT) {
          kind = OOC_SWAPIN;
          s.h2d += vars[u].bytes;
        }
        state[u] = DEV;
        held += need;
        emit((int32_t)i, OOC_PRE, kind, u);
      } else if (p <= e) {
        *err = "function " + std::to_string(i) + " needs more than the budget of " +
               std::to_string(budget) + " bytes";
        return OOC_E_INFEASIBLE;
      } else {
        r = p - 1;
        break;
      }
    }
    s.windows.push_back(r);

    for (size_t j = 0; j < fns[i].vars.size(); ++j) {
      const int64_t u = fns[i].vars[j].var;
      const int64_t n = next[l + (int64_t)j];
      const int32_t kind = vars[u].kind;
      if (n < 0 && (kind == OOC_INPUT || kind == OOC_TEMP)) {
        state[u] = UNMAT;
        held -= a[u];
        emit((int32_t)i, OOC_POST, OOC_FREE, u);
      } else if (n >= 0 && (n <= r || (fixed && fn_of[n] - i <= threshold))) {
        // already reserved inside the window (or close enough): keep it on the device
      } else {
        state[u] = PEND;
        entry_of[u] = (int64_t)fifo.size();
        fifo.push_back(Entry{u, true, n >= 0 ? n : INT64_MAX});
        ++alive;
        ++queued[u];
        s.d2h += vars[u].bytes;
        emit((int32_t)i, OOC_POST, OOC_SWAPOUT, u);
      }
    }
    r_prev = r;
  }
  while (alive > 0) pop((int32_t)N, OOC_END, false);
  for (const Op& o : s.ops) s.peak = std::max(s.peak, o.held);
  *out = std::move(s);
  return OOC_OK;
}

static void first_last_use(const std::vector<Var>& vars, const std::vector<Fn>& fns,
                           std::vector<int64_t>* fu, std::vector<int64_t>* lu) {
  fu->assign(vars.size(), -1);
  lu->assign(vars.size(), -1);
  for (int64_t i = 0; i < (int64_t)fns.size(); ++i)
    for (const FnVar& fv : fns[i].vars) {
      if ((*fu)[fv.var] < 0) (*fu)[fv.var] = i;
      (*lu)[fv.var] = i;
    }
}

void build_incore(const std::vector<Var>& vars, const std::vector<Fn>& fns, uint64_t chunk,
                  Schedule* out) {
  std::vector<int64_t> fu, lu;
  first_last_use(vars, fns, &fu, &lu);
  Schedule s;
  uint64_t held = 0;
  for (const Var& v : vars)
    if (v.kind != OOC_TEMP) held += round_up(v.bytes, chunk);
  s.peak = held;
  for (int64_t i = 0; i < (int64_t)fns.size(); ++i) {
    for (const FnVar& fv : fns[i].vars)
      if (vars[fv.var].kind == OOC_TEMP && fu[fv.var] == i) {
        held += round_up(vars[fv.var].bytes, chunk);
        s.ops.push_back(Op{(int32_t)i, OOC_PRE, OOC_ALLOC, fv.var, held});
        s.peak = std::max(s.peak, held);
      }
    for (const FnVar& fv : fns[i].vars)
      if (vars[fv.var].kind == OOC_TEMP && lu[fv.var] == i) {
        held -= round_up(vars[fv.var].bytes, chunk);
        s.ops.push_back(Op{(int32_t)i, OOC_POST, OOC_FREE, fv.var, held});
      }
  }
  *out = std::move(s);
}

uint64_t incore_peak(const std::vector<Var>& vars, const std::vector<Fn>& fns, uint64_t chunk) {
  Schedule s;
  build_incore(vars, fns, chunk, &s);
  return s.peak;
}

uint64_t working_set_max(const std::vector<Var>& vars, const std::vector<Fn>& fns,
                         uint64_t chunk) {
  uint64_t best = 0;
  for (const Fn& f : fns) {
    uint64_t sum = 0;
    for (const FnVar& fv : f.vars) sum += round_up(vars[fv.var].bytes, chunk);
    best = std::max(best, sum);
  }
  return best;
}

// Chunk cache handing out freed chunks in the order they were freed (least
// recently freed first), and a chunk never used before only when none is
// free.  A swap-in thus lands, where the budget leaves a choice, in memory
// whose previous occupant was released longest ago, so its copy rarely waits
// for the kernel running at the time.  Fresh ids are handed out only while the
// queue is empty, so the ids in use stay below the most chunks ever in use at
// once: the pool needs exactly that many.
namespace {
struct ChunkCache {
  std::deque<int32_t> freed;
  int32_t fresh = 0;
  uint64_t in_use = 0, max_in_use = 0;
  void take(uint64_t k, std::vector<int32_t>* out) {
    for (uint64_t j = 0; j < k; ++j) {
      if (!freed.empty()) {
        out->push_back(freed.front());
        freed.pop_front();
      } else {
        out->push_back(fresh++);
      }
    }
    in_use += k;
    max_in_use = std::max(max_in_use, in_use);
  }
  void give(const std::vector<int32_t>& cs) {
    for (int32_t c : cs) freed.push_back(c);
    in_use -= cs.size();
  }
};
}  // namespace

void build_plan(const std::vector<Var>& vars, const Schedule& s, bool incore, uint64_t chunk,
                Plan* out) {
  Plan plan;
  ChunkCache cache;
  std::vector<int64_t> working(vars.size(), -1);
  std::vector<int64_t> pending;   // interval ids with an issued swap-out, oldest first
  size_t head = 0;
  auto open = [&](int64_t v, int64_t op) {
    Interval iv{v, op, -1, {}};
    cache.take(round_up(vars[v].bytes, chunk) / chunk, &iv.chunks);
    plan.intervals.push_back(std::move(iv));
    working[v] = (int64_t)plan.intervals.size() - 1;
    return working[v];
  };
  auto close = [&](int64_t id, int64_t op) {
    plan.intervals[id].close = op;
    cache.give(plan.intervals[id].chunks);
  };
  if (incore)
    for (int64_t v = 0; v < (int64_t)vars.size(); ++v)
      if (vars[v].kind != OOC_TEMP) open(v, -1);
  plan.op_interval.assign(s.ops.size(), -1);
  for (int64_t k = 0; k < (int64_t)s.ops.size(); ++k) {
    const Op& o = s.ops[k];
    int64_t id = -1;
    switch (o.kind) {
      case OOC_SWAPIN:
      case OOC_ALLOC:
        id = open(o.var, k);
        break;
      case OOC_SWAPOUT:
        id = working[o.var];
        pending.push_back(id);
        working[o.var] = -1;
        break;
      case OOC_CANCEL:
      case OOC_WAIT_OUT:
        // the variable's oldest pending copy (a budget wait need not complete
        // the oldest swap-out overall, see ooc_set_wait_order)
        for (size_t j = head; j < pending.size(); ++j)
          if (pending[j] >= 0 && plan.intervals[pending[j]].var == o.var) {
            id = pending[j];
            pending[j] = -1;
            break;
          }
        while (head < pending.size() && pending[head] < 0) ++head;
        if (o.kind == OOC_CANCEL)
          working[o.var] = id;
        else
          close(id, k);
        break;
      case OOC_FREE:
        id = working[o.var];
        working[o.var] = -1;
        close(id, k);
        break;
    }
    plan.op_interval[k] = id;
  }
  plan.max_chunks_used = cache.max_in_use;
  plan.n_chunks = cache.max_in_use;
  *out = std::move(plan);
}

// The comparison point of Section 4: the plan's residency intervals served by
// one contiguous best-fit heap instead of the chunk pool.  A request (size
// rounded up to `align`) takes the smallest free hole that holds it, lowest
// address on ties; when none does it goes to the end of the heap, starting in
// the free tail if there is one.  Returns the highest address used and the
// most bytes live at once.
void bestfit_extent(const std::vector<Var>& vars, const Plan& plan, uint64_t align,
                    uint64_t* extent, uint64_t* peak_live, std::vector<uint64_t>* offsets) {
  std::map<uint64_t, uint64_t> by_off;             // hole offset -> size
  std::set<std::pair<uint64_t, uint64_t>> by_size; // (size, offset)
  uint64_t end = 0, live = 0, peak = 0;
  std::vector<uint64_t> off(plan.intervals.size(), 0), size(plan.intervals.size(), 0);
  auto erase_hole = [&](std::map<uint64_t, uint64_t>::iterator it) {
    by_size.erase({it->second, it->first});
    return by_off.erase(it);
  };
  auto alloc = [&](int64_t id) {
    const uint64_t sz = round_up(vars[plan.intervals[id].var].bytes, align);
    auto f = by_size.lower_bound({sz, 0});
    uint64_t o;
    if (f != by_size.end()) {
      o = f->second;
      const uint64_t hs = f->first;
      erase_hole(by_off.find(o));
      if (hs > sz) {
        by_off[o + sz] = hs - sz;
        by_size.insert({hs - sz, o + sz});
      }
    } else {
      auto last = by_off.empty() ? by_off.end() : std::prev(by_off.end());
      if (last != by_off.end() && last->first + last->second == end) {
        o = last->first;
        erase_hole(last);
      } else {
        o = end;
      }
      end = o + sz;
    }
    off[id] = o;
    size[id] = sz;
    live += sz;
    peak = std::max(peak, live);
  };
  auto release = [&](int64_t id) {
    uint64_t o = off[id], sz = size[id];
    live -= sz;
    auto nx = by_off.lower_bound(o);
    if (nx != by_off.end() && o + sz == nx->first) {
      sz += nx->second;
      nx = erase_hole(nx);
    }
    if (nx != by_off.begin()) {
      auto pv = std::prev(nx);
      if (pv->first + pv->second == o) {
        o = pv->first;
        sz += pv->second;
        erase_hole(pv);
      }
    }
    by_off[o] = sz;
    by_size.insert({sz, o});
  };
  for (int64_t id = 0; id < (int64_t)plan.intervals.size(); ++id)
    if (plan.intervals[id].open < 0) alloc(id);
  for (int64_t k = 0; k < (int64_t)plan.op_interval.size(); ++k) {
    const int64_t id = plan.op_interval[k];
    if (id < 0) continue;
    if (plan.intervals[id].open == k) alloc(id);
    else if (plan.intervals[id].close == k) release(id);
  }
  *extent = end;
  *peak_live = peak;
  if (offsets) *offsets = std::move(off);
}

// Device layout of the best-fit heap: every interval at its replayed offset.
// The heap is cut at every interval's first and last byte into segments; an
// interval's "chunks" become the segments it covers, so the executor's rule
// (the first writer of memory waits for everyone who used it before) applies
// unchanged.
void bestfit_layout(const std::vector<Var>& vars, uint64_t align, Plan* plan,
                    std::vector<uint64_t>* offsets, uint64_t* extent) {
  uint64_t peak = 0;
  bestfit_extent(vars, *plan, align, extent, &peak, offsets);
  std::vector<uint64_t> cuts;
  for (size_t J = 0; J < plan->intervals.size(); ++J) {
    cuts.push_back((*offsets)[J]);
    cuts.push_back((*offsets)[J] + round_up(vars[plan->intervals[J].var].bytes, align));
  }
  std::sort(cuts.begin(), cuts.end());
  cuts.erase(std::unique(cuts.begin(), cuts.end()), cuts.end());
  for (size_t J = 0; J < plan->intervals.size(); ++J) {
    const uint64_t a = (*offsets)[J], b = a + round_up(vars[plan->intervals[J].var].bytes, align);
    auto& cs = plan->intervals[J].chunks;
    cs.clear();
    for (size_t g = std::lower_bound(cuts.begin(), cuts.end(), a) - cuts.begin();
         g + 1 < cuts.size() && cuts[g] < b; ++g)
      cs.push_back((int32_t)g);
  }
  plan->n_chunks = cuts.empty() ? 0 : cuts.size() - 1;
}

}  // namespace ooc
