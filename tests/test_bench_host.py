"""Host-side logic of ``bench.py`` (no GPU): the work counts behind the roofline, the traffic
records it reads, the budget / window / chunk it derives for a workload, and its refusal of more
than one GPU."""

import hashlib
import os
import subprocess
import sys

import pytest

import bench
from paper_2010_14109_amd import netdef, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def r1440():
    return netdef.Net(synth.workload("resnet50_b1440"))


def test_work_counts():
    assert bench.fn_work("linear_fwd", [7, 5, 3]) == ("flop", 2 * 7 * 5 * 3)
    # conv: 2 N P Q K R S C, whatever the stride (P, Q are the output size)
    assert bench.fn_work("conv_bwd_x", [2, 9, 9, 4, 8, 3, 3, 2, 1, 5, 5]) == \
        ("flop", 2 * 2 * 5 * 5 * 8 * 3 * 3 * 4)
    assert bench.fn_work("relu_fwd", [10]) == ("byte", 80)
    assert bench.fn_work("bn_bwd", [10, 4, 1]) == ("byte", 12 * 40)
    # causal attention counts the T (T + 1) / 2 entries on and below the diagonal: two products
    # forward, five backward (q k^T again, since the probabilities are recomputed)
    B, T, H, dh = 2, 8, 3, 4
    pairs = T * (T + 1) // 2
    assert bench.fn_work("attention_fwd", [B, T, H, dh, 1]) == ("flop", 2 * 2 * B * H * pairs * dh)
    assert bench.fn_work("attention_bwd", [B, T, H, dh, 1]) == ("flop", 5 * 2 * B * H * pairs * dh)
    assert bench.fn_work("attention_bwd", [B, T, H, dh, 0]) == ("flop", 5 * 2 * B * H * T * T * dh)


def test_algorithmic_bytes_of_the_default_line(r1440):
    """The default line's dominant function: filter and output gradient read once, input
    gradient written once, averaged over its 52 launches (the figure of its traffic record)."""
    assert bench.algorithmic_bytes(r1440, "conv_bwd_x") == 2_308_355_623
    assert bench.algorithmic_bytes(r1440, "no_such_op") is None


def test_split_partials_are_not_algorithmic():
    """The plain CNN's filter gradients carry split-K partial sums; only X, dY and dW count:
    9 launches of 33.55 + 33.55 + 0.15 MB and the 3-channel one, averaged."""
    net = netdef.Net(synth.workload("cnn"))
    assert any(net.names[v].endswith(".part") for v, _ in net.fn_vars[net.fn_ops.index("conv_bwd_w")])
    x64 = 128 * 32 * 32 * 64 * 4
    per_64 = 2 * x64 + 64 * 9 * 64 * 4
    per_3 = 128 * 32 * 32 * 3 * 4 + x64 + 64 * 9 * 3 * 4
    assert bench.algorithmic_bytes(net, "conv_bwd_w") == round((9 * per_64 + per_3) / 10)


def test_traffic_records_are_read_while_their_source_is_unchanged(r1440, monkeypatch):
    import glob
    src = open(os.path.join(ROOT, "paper_2010_14109_amd", "csrc", "gemm.hip"), "rb").read()
    current = hashlib.sha256(src).hexdigest()
    lines = [ln for f in glob.glob(os.path.join(ROOT, "profiles", "traffic_*.md"))
             for ln in open(f) if ln.startswith("traffic: op=conv_bwd_x ")]
    got = bench.measured_traffic(r1440, "conv_bwd_x")
    if any(("sha256=" + current) in ln for ln in lines):
        # every launch of the default line has a record taken on this source
        assert got is not None and 2_000_000_000 < got < 5_000_000_000
    else:
        assert got is None
    assert bench.measured_traffic(r1440, "conv_fwd") is None      # no record for it
    real = hashlib.sha256

    class Other:
        def __init__(self, data=b""):
            self.h = real(data + b"changed")

        def hexdigest(self):
            return self.h.hexdigest()

    monkeypatch.setattr(hashlib, "sha256", Other)
    assert bench.measured_traffic(r1440, "conv_bwd_x") is None     # kernel source changed


def test_window_fraction():
    assert bench.window_fraction("mlp") == 0.5
    for w in ("cnn", "resnet50_b256", "resnet50_b1440", "transformer", "densenet", "unet"):
        assert bench.window_fraction(w) == bench.DEFAULT_WINDOW_FRAC == 0.25


def test_default_plan_is_the_table_1_setting(r1440):
    """ResNet-50 b1440 at P_incore / 7.5: the smallest chunk whose plans fit the map table is
    16 MiB, the budget is P / 7.5 rounded down to whole chunks, the window a quarter of it."""
    chunk, plan = bench.choose_chunk(r1440, synth.budget_fraction("resnet50_b1440"),
                                     bench.window_fraction("resnet50_b1440"))
    assert chunk == 16 << 20
    assert plan["map_entries"] <= bench.MAP_ENTRY_LIMIT
    assert plan["budget"] % chunk == 0
    assert plan["budget"] <= plan["p_incore"] / 7.5 < plan["budget"] + chunk
    assert plan["window"] == int(plan["budget"] * 0.25)
    assert plan["budget"] >= plan["ws_max"]


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stdout


def test_paper_figure_only_for_the_exact_table_1_setting():
    """vs_baseline divides by the paper's 321 images/s (Table 1, Schedule + VA, batch 1440) only
    when the run is that setting: the default workload, batch and budget, the adaptive scheduler,
    the chunk pool and the paper's oldest-first waits."""
    f = synth.budget_fraction("resnet50_b1440")
    assert bench.paper_figure("resnet50_b1440", 1440, f, "adaptive", "pool", "oldest") == 321.0
    assert bench.paper_figure("resnet50_b1440", 800, f, "adaptive", "pool", "oldest") is None
    assert bench.paper_figure("resnet50_b1440", 1440, 0.25, "adaptive", "pool", "oldest") is None
    assert bench.paper_figure("resnet50_b1440", 1440, f, "naive", "pool", "oldest") is None
    assert bench.paper_figure("resnet50_b1440", 1440, f, "adaptive", "bestfit", "oldest") is None
    assert bench.paper_figure("resnet50_b1440", 1440, f, "adaptive", "pool", "furthest") is None
    assert bench.paper_figure("resnet50_b256", 256, 0.25, "adaptive", "pool", "oldest") is None
