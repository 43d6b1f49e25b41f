"""Host-side checks of the single-function harness and of the library's split-K slice rule
(no GPU)."""

import math
import os
import random

import pytest

from paper_2010_14109_amd import kbench, ooc

CASES = ["conv_fwd:4,9,9,8,12,3,1,1", "conv_bwd_x:4,9,9,8,12,3,2,1", "conv_bwd_w:4,9,9,8,12,3,1,1",
         "conv_bwd_w:4,9,9,64,64,3,1,1,7", "linear_fwd:64,32,48", "linear_bwd_x:64,32,48",
         "linear_bwd_w:64,32,48", "linear_bwd_w:1024,32,48,3", "relu_fwd:1000", "bn_fwd:300,12",
         "bn_bwd:300,12"]


@pytest.mark.parametrize("spec", CASES)
def test_case_registers_and_schedules(spec):
    op, vs, attrs = kbench.case(spec)
    ctx = ooc.Context(-1)
    try:
        ids = [ctx.add_var(b, k) for b, k, _ in vs]
        ctx.add_fn(op, ids, [a for _, _, a in vs], attrs)
        ctx.set_chunk(2 << 20)
        ctx.build_schedule()
        assert ctx.stats()["peak_accounted"] > 0
    finally:
        ctx.close()


def conv_attrs(N, H, W, C, K, k, st, pd):
    P, Q = (H + 2 * pd - k) // st + 1, (W + 2 * pd - k) // st + 1
    return [N, H, W, C, K, k, k, st, pd, P, Q]


def test_slice_rule_bounds():
    """The library's split-K count lies in [1, ceil(reduced rows / 256)] for random shapes (at
    least 256 rows a slice), for convolutions and dense layers alike."""
    rng = random.Random(7)
    for _ in range(400):
        N, hw, C = rng.randint(1, 64), rng.choice([1, 7, 14, 56, 112]), rng.choice([3, 4, 64, 256])
        K, k = rng.choice([8, 32, 64, 96, 1024]), rng.choice([1, 3, 7])
        a = conv_attrs(N, hw, hw, C, K, k, 1, k // 2)
        s = ooc.wgrad_slices("conv_bwd_w", a)
        assert 1 <= s <= max(1, math.ceil(N * a[9] * a[10] / 256))
        M = rng.randrange(1, 100_000)
        s = ooc.wgrad_slices("linear_bwd_w", [M, rng.randint(1, 4096), rng.randint(1, 4096)])
        assert 1 <= s <= max(1, math.ceil(M / 256))


def test_slice_rule_known_shapes():
    # plain CNN 3 x 3 64 -> 64 at batch 128: 3 tiles of 64 x 192, 2 per CU, 169 slices fill
    # one round of 512 slots to 507; the transformer's QKV weight gradient (3072 x 1024, 12288
    # rows): 192 tiles of 128 x 128 at 8 slices are three rounds of 512; a dense layer with 256
    # rows is one slice
    assert ooc.wgrad_slices("conv_bwd_w", conv_attrs(128, 32, 32, 64, 64, 3, 1, 1)) == 169
    assert ooc.wgrad_slices("linear_bwd_w", [12288, 1024, 3072]) == 8
    assert ooc.wgrad_slices("linear_bwd_w", [256, 1024, 1024]) == 1
    # a trailing slices attribute is ignored
    a = conv_attrs(128, 32, 32, 64, 64, 3, 1, 1)
    assert ooc.wgrad_slices("conv_bwd_w", a + [5]) == 169


def test_slice_rule_rejects_bad_requests():
    for op, attrs in (("conv_fwd", conv_attrs(2, 8, 8, 4, 4, 3, 1, 1)),
                      ("conv_bwd_w", [2, 8, 8, 4]),
                      ("conv_bwd_w", conv_attrs(0, 8, 8, 4, 4, 3, 1, 1)),
                      ("linear_bwd_w", [0, 4, 4]),
                      ("linear_bwd_w", [4, -1, 4])):
        with pytest.raises(ooc.OocError) as e:
            ooc.wgrad_slices(op, attrs)
        assert e.value.status == ooc.E_INVALID and "ooc_wgrad_slices" in e.value.message


def _counter_csv(path, rows):
    """A rocprofv3 counter-collection file: rows of (dispatch id, kernel name, counter, value)."""
    import csv
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "p_counter_collection.csv"), "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for r in rows:
            w.writerow(r)


def test_traffic_adds_every_dispatch_of_a_call(tmp_path):
    """A function that launches one kernel several times per call (the stride classes of an
    input gradient) must count all of them: bytes per call = all dispatches / calls.  The
    calibration ReLU moves 1 GiB each way; its counters here read half of it (scale 2)."""
    gib_kib = (kbench.CAL_N * 4) // 1024
    cal = tmp_path / "cal"
    _counter_csv(str(cal / "fetch"), [(1, "void ooc::(anonymous namespace)::ew_kernel<0>(x)",
                                       "FETCH_SIZE", gib_kib / 2)])
    _counter_csv(str(cal / "write"), [(1, "void ooc::(anonymous namespace)::ew_kernel<0>(x)",
                                       "WRITE_SIZE", gib_kib)])
    calls, per_call = 3, 4
    rows_f, rows_w = [], []
    for d in range(calls * per_call):
        rows_f.append((d, "void ooc::(anonymous namespace)::gemm_kernel<1>(x)", "FETCH_SIZE", 100.0))
        rows_w.append((d, "void ooc::(anonymous namespace)::gemm_kernel<1>(x)", "WRITE_SIZE", 10.0))
    for d in range(calls):
        rows_f.append((100 + d, "ooc::(anonymous namespace)::class_zero_kernel(y)", "FETCH_SIZE", 0.0))
        rows_w.append((100 + d, "ooc::(anonymous namespace)::class_zero_kernel(y)", "WRITE_SIZE", 7.0))
    _counter_csv(str(tmp_path / "f"), rows_f)
    _counter_csv(str(tmp_path / "w"), rows_w)
    res, fs, ws = kbench.traffic(str(tmp_path / "f"), str(tmp_path / "w"), str(cal), calls=calls)
    assert fs == pytest.approx(2.0) and ws == pytest.approx(1.0)
    gemm, fill = res["gemm_kernel<1>"], res["class_zero_kernel"]
    assert gemm == pytest.approx((per_call * 100 * 1024 * 2.0, per_call * 10 * 1024 * 1.0))
    assert fill == pytest.approx((0.0, 7 * 1024 * 1.0))
    # without the call count every kernel counts once per call (the mean per dispatch)
    res1, _, _ = kbench.traffic(str(tmp_path / "f"), str(tmp_path / "w"), str(cal))
    assert res1["gemm_kernel<1>"] == pytest.approx((100 * 1024 * 2.0, 10 * 1024 * 1.0))
