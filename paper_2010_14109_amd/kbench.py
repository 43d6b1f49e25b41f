"""Single-function harness for kernel profiling.

``python -m paper_2010_14109_amd.kbench CASE [REPS]`` registers one function
with seeded inputs, runs it in-core REPS times through the library and prints
its event-timed duration; under ``rocprofv3`` it gives clean per-kernel
statistics and counters.  CASE is ``op:n1,n2,...``:

* ``conv_fwd | conv_bwd_x | conv_bwd_w : N,H,W,C,K,k,stride,pad[,slices]``
* ``linear_fwd | linear_bwd_x : M,K,N``, ``linear_bwd_w : M,K,N[,slices]``
* ``relu_fwd : n``  (reads 4 n bytes, writes 4 n bytes: the calibration kernel)
* ``bn_fwd | bn_bwd : rows,C``  (training-mode batch normalisation over ``rows`` NHWC pixels)

``python -m paper_2010_14109_amd.kbench --traffic FETCH_DIR WRITE_DIR CAL_DIR [CALLS]``
turns ``rocprofv3 --pmc FETCH_SIZE`` / ``--pmc WRITE_SIZE`` output of a case
(FETCH_DIR, WRITE_DIR) into bytes per call, scaling each counter by what it
reads for ``relu_fwd:268435456`` (CAL_DIR holds both counters of that run).
CALLS is how many calls the profiled run made (REPS + 1: one warm-up); a
function may launch one kernel several times per call (one GEMM per stride
class of an input gradient), so the bytes of all its dispatches are added and
divided by CALLS.  Without CALLS every kernel counts once per call.  The
counters see what the L2 caches fetch and write back: reads served by the
256 MB last-level cache count too.
"""

from __future__ import annotations

import csv
import glob
import os
import sys
import time
from collections import defaultdict

import numpy as np

from . import netdef, ooc, synth

CAL_N = 268435456   # floats of the calibration ReLU: 1 GiB read, 1 GiB written


def _conv_attrs(N, H, W, C, K, k, st, pd):
    P = (H + 2 * pd - k) // st + 1
    Q = (W + 2 * pd - k) // st + 1
    return [N, H, W, C, K, k, k, st, pd, P, Q], P, Q


def case(spec):
    """(op, [(bytes, kind, access)], attrs) of a case string."""
    op, nums = spec.split(":")
    v = [int(x) for x in nums.split(",")]
    I, O, R, Wr = ooc.INPUT, ooc.OUTPUT, ooc.R, ooc.W
    if op == "relu_fwd":
        return op, [(v[0] * 4, I, R), (v[0] * 4, O, Wr)], [v[0]]
    if op in ("bn_fwd", "bn_bwd"):
        rows, C = v
        s = netdef.bn_row_slices(rows)
        xb, cb, sb = rows * C * 4, C * 4, (2 + 2 * s) * C * 4
        if op == "bn_fwd":
            return op, [(xb, I, R), (cb, I, R), (cb, I, R), (xb, O, Wr), (sb, O, Wr)], [rows, C, s]
        return op, [(xb, I, R), (cb, I, R), (sb, ooc.STATE, ooc.RW), (xb, I, R), (xb, O, Wr),
                    (cb, O, Wr), (cb, O, Wr)], [rows, C, s]
    if op.startswith("conv"):
        N, H, W, C, K, k, st, pd = v[:8]
        a, P, Q = _conv_attrs(N, H, W, C, K, k, st, pd)
        xb, wb, yb = N * H * W * C * 4, K * k * k * C * 4, N * P * Q * K * 4
        if op == "conv_fwd":
            return op, [(xb, I, R), (wb, I, R), (yb, O, Wr)], a
        if op == "conv_bwd_x":
            return op, [(wb, I, R), (yb, I, R), (xb, O, Wr)], a
        s = v[8] if len(v) > 8 else ooc.wgrad_slices(op, a)
        vs = [(xb, I, R), (yb, I, R), (wb, O, Wr)] + ([(s * wb, O, Wr)] if s > 1 else [])
        return op, vs, a + [s]
    M, K, N = v[:3]
    if op == "linear_fwd":
        return op, [(M * K * 4, I, R), (N * K * 4, I, R), (N * 4, I, R), (M * N * 4, O, Wr)], v
    if op == "linear_bwd_x":
        return op, [(N * K * 4, I, R), (M * N * 4, I, R), (M * K * 4, O, Wr)], v
    s = v[3] if len(v) > 3 else ooc.wgrad_slices(op, v[:3])
    vs = [(M * K * 4, I, R), (M * N * 4, I, R), (N * K * 4, O, Wr), (N * 4, O, Wr)]
    if s > 1:
        vs.append((s * (N * K + N) * 4, O, Wr))
    return op, vs, [M, K, N, s]


def run(spec, reps=20):
    op, vs, attrs = case(spec)
    ctx = ooc.Context(0)
    try:
        ids = [ctx.add_var(b, k) for b, k, _ in vs]
        ctx.add_fn(op, ids, [a for _, _, a in vs], attrs)
        ctx.set_chunk(2 << 20)
        ctx.build_schedule()
        ctx.prepare()
        need = sum(b // 4 for b, k, _ in vs if k in (ooc.INPUT, ooc.STATE))
        pool = synth.normal_pool(max(need, 1), seed=0)
        at = 0
        for (b, k, _), v in zip(vs, ids):
            if k in (ooc.INPUT, ooc.STATE):
                w = pool[at:at + b // 4]
                at += b // 4
                # |N(0,1)| keeps a batch-norm inverse deviation positive
                ctx.host_view(v, np.float32)[...] = np.abs(w) if k == ooc.STATE else w
        ctx.upload()
        ctx.step(0.0, 0.0)
        t0 = time.perf_counter()
        for _ in range(reps):
            ctx.step(0.0, 0.0)
        wall = (time.perf_counter() - t0) / reps * 1e3
        return ctx.fn_times()[0], wall
    finally:
        ctx.close()


def _counters(d, calls=None):
    """{kernel: {counter: value per call}} of the rocprofv3 csv files under d: the sum over
    the kernel's dispatches / calls, or the mean per dispatch when calls is None."""
    acc = defaultdict(lambda: defaultdict(list))
    for f in glob.glob(os.path.join(d, "**", "*_counter_collection.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                name = r["Kernel_Name"].replace("ooc::(anonymous namespace)::", "")
                name = name.replace("void ", "").split("(")[0]
                acc[name][r["Counter_Name"]].append(float(r["Counter_Value"]))
    return {k: {c: sum(x) / (calls or len(x)) for c, x in v.items()} for k, v in acc.items()}


def traffic(fetch_dir, write_dir, cal_dir, calls=None):
    """Calibrated bytes per call: {kernel: (fetch_bytes, write_bytes)} and the scales."""
    cal = _counters(cal_dir)
    ew = [v for k, v in cal.items() if k.startswith("ew_kernel")]
    if len(ew) != 1:
        raise SystemExit(f"calibration run {cal_dir} must hold exactly one ReLU kernel")
    ref = CAL_N * 4
    fs, ws = ref / (ew[0]["FETCH_SIZE"] * 1024), ref / (ew[0]["WRITE_SIZE"] * 1024)
    f, w = _counters(fetch_dir, calls), _counters(write_dir, calls)
    out = {k: (f[k]["FETCH_SIZE"] * 1024 * fs, w.get(k, {}).get("WRITE_SIZE", 0.0) * 1024 * ws)
           for k in f}
    return out, fs, ws


def main(argv):
    if argv and argv[0] == "--traffic":
        calls = int(argv[4]) if len(argv) > 4 else None
        res, fs, ws = traffic(*argv[1:4], calls=calls)
        print(f"scales: FETCH_SIZE x {fs:.4f}, WRITE_SIZE x {ws:.4f}")
        total = 0.0
        for k, (fb, wb) in res.items():
            print(f"{k}: fetch {fb / 1e6:.2f} MB, write {wb / 1e6:.2f} MB")
            total += fb + wb
        print(f"total bytes per call: {int(total)}")
        return 0
    spec = argv[0]
    reps = int(argv[1]) if len(argv) > 1 else 20
    ev, wall = run(spec, reps)
    print(f"{spec}: {ev:.4f} ms per call (events), {wall:.3f} ms wall", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
