"""Device memory needed by a schedule: the chunk pool against a contiguous best-fit heap.

Section 4 builds device memory from equal physical chunks mapped into
per-allocation virtual ranges, so that only internal fragmentation (under one
chunk per allocation, eq. 1 and 2) remains.  This host-only experiment runs
the library's scheduler and reports, per workload and budget B:

* the chunk pool's device bytes (most chunks in use x m_c, never above B);
* the bytes live at the peak (sizes rounded to 256 B, as a device allocator
  would) and the address range a best-fit heap serving the same allocations
  needs (its extent): the excess is external fragmentation;
* the largest budget whose schedule a best-fit heap could serve inside B
  bytes of device memory;
* per chunk size m_c: the pool's internal fragmentation at the peak, the
  memory-map entries its plan needs, and the bytes the schedule swaps.

``python -m paper_2010_14109_amd.fragmentation [--workload NAME ...]`` prints
markdown tables; nothing runs on the GPU.
"""

from __future__ import annotations

import argparse

from . import netdef, ooc, synth

MiB = 1 << 20
ALIGN = 256


def _context(net, budget, window, chunk):
    ctx = ooc.Context(-1)
    net.register(ctx)
    ctx.set_chunk(chunk)
    ctx.set_budget(budget)
    if window is not None:
        ctx.set_window(window)
    return ctx


def measure(net, budget, chunk, window_frac=0.5):
    """Pool bytes, best-fit extent and live peak of the schedule for ``budget``."""
    ctx = _context(net, budget, int(budget * window_frac), chunk)
    try:
        ctx.build_schedule()
        st = ctx.stats()
        extent, peak_live = ctx.bestfit_extent(ALIGN)
        return {"budget": budget, "pool": st["max_chunks_used"] * chunk,
                "accounted": st["peak_accounted"], "extent": extent, "peak_live": peak_live,
                "h2d": st["sched_h2d_bytes"], "d2h": st["sched_d2h_bytes"],
                "map_entries": sum(ctx.plan_counts())}
    finally:
        ctx.close()


def largest_bestfit_budget(net, limit, chunk, ws_max, window_frac=0.5):
    """Largest budget (a multiple of m_c, at least WS_max) whose schedule a best-fit heap serves
    within ``limit`` bytes, or None when even WS_max does not fit."""
    lo, hi = ws_max // chunk, limit // chunk
    if measure(net, lo * chunk, chunk, window_frac)["extent"] > limit:
        return None
    while lo < hi:
        mid = (lo + hi + 1) // 2
        if measure(net, mid * chunk, chunk, window_frac)["extent"] <= limit:
            lo = mid
        else:
            hi = mid - 1
    return lo * chunk


def peaks(net, chunk):
    ctx = ooc.Context(-1)
    try:
        net.register(ctx)
        ctx.set_chunk(chunk)
        return ctx.incore_peak(), ctx.working_set_max()
    finally:
        ctx.close()


def report(name, batch=0, fracs=(0.5, 0.25, 1 / 7.5), chunk=2 * MiB, chunks=(2, 8, 32, 128)):
    spec = synth.workload(name, **({"batch": batch} if batch else {}))
    net = netdef.Net(spec)
    p_incore, ws = peaks(net, chunk)
    gib = 1 << 30
    print(f"\n### {spec['name']} (P_incore {p_incore / gib:.2f} GiB at m_c = {chunk // MiB} MiB, "
          f"WS_max {ws / gib:.2f} GiB)\n")
    print("| B / P | B GiB | pool GiB | live at peak GiB | best-fit extent GiB | extent / B "
          "| largest best-fit budget in B bytes |")
    print("|---|---|---|---|---|---|---|")
    for frac in fracs:
        budget = max(int(p_incore * frac) // chunk * chunk, ws)
        m = measure(net, budget, chunk)
        lb = largest_bestfit_budget(net, budget, chunk, ws)
        lbs = "infeasible" if lb is None else f"{lb / gib:.2f} GiB ({lb / budget:.3f} B)"
        print(f"| {frac:.3f} | {budget / gib:.2f} | {m['pool'] / gib:.2f} | {m['peak_live'] / gib:.2f}"
              f" | {m['extent'] / gib:.2f} | {m['extent'] / budget:.3f} | {lbs} |")
    budget = max(int(p_incore * fracs[-1]) // chunk * chunk, ws)
    print(f"\nChunk size at B = {budget / gib:.2f} GiB ({fracs[-1]:.3f} P):\n")
    print("| m_c MiB | pool GiB | internal fragmentation at the peak | map entries "
          "| swapped in / out GiB |")
    print("|---|---|---|---|---|")
    for c in chunks:
        cb = c * MiB
        b = max(budget // cb * cb, peaks(net, cb)[1])
        try:
            m = measure(net, b, cb)
        except ooc.OocError as e:
            print(f"| {c} | - | infeasible ({e.status}) | - | - |")
            continue
        frag = (m["accounted"] - m["peak_live"]) / m["accounted"]
        print(f"| {c} | {m['pool'] / gib:.2f} | {100 * frag:.1f} % | {m['map_entries']} | "
              f"{m['h2d'] / gib:.1f} / {m['d2h'] / gib:.1f} |")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", nargs="*", default=["cnn", "resnet50_b256", "transformer"])
    ap.add_argument("--batch", type=int, default=0)
    args = ap.parse_args()
    for w in args.workload:
        report(w, args.batch if args.batch else (24 if w == "transformer" else 0))


if __name__ == "__main__":
    main()
