"""Host-side checks of the single-function harness and of the split-K slice rule (no GPU)."""

import math
import random

import pytest

from oracle import lower as oracle_lower
from paper_2010_14109_amd import kbench, netdef, ooc

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


def _cost(tiles, per_cu, s):
    slots = 256 * per_cu
    return math.ceil(tiles * s / slots) / s


def test_slice_rule_agrees_with_oracle_and_fills_rounds():
    """Both lowerings choose the same count; it lies in [1, smax] and its rounds-per-slice cost is
    within 1 % of the best count in that range (brute force), none smaller being that good."""
    rng = random.Random(7)
    for _ in range(400):
        k_out = rng.choice([8, 32, 64, 96, 128, 256, 1024, 3072, 4096])
        c = rng.choice([3, 4, 16, 60, 64, 128, 256])
        rsc = rng.choice([1, 3, 7]) ** 2 * c
        pixels = rng.randrange(1, 3_000_000)
        for ch in (None, c):
            s = netdef.wgrad_pixel_slices(k_out, rsc, pixels, ch)
            assert s == oracle_lower.conv_wgrad_slices(k_out, rsc, pixels, ch)
            tile = netdef.wgrad_tile(k_out, rsc, ch) if ch is not None else None
            if tile is not None:
                tiles, per_cu = math.ceil(rsc / tile[1]), tile[2]
            elif k_out <= 64:
                tiles, per_cu = math.ceil(rsc / 128), 3
            elif rsc <= 64:
                tiles, per_cu = math.ceil(k_out / 128), 3
            else:
                tiles, per_cu = math.ceil(k_out / 128) * math.ceil(rsc / 128), 2
            smax = max(1, min(4 * 256 * per_cu // tiles, math.ceil(pixels / 256)))
            assert 1 <= s <= smax
            best = min(_cost(tiles, per_cu, t) for t in range(1, smax + 1))
            assert _cost(tiles, per_cu, s) <= best * 1.01
            assert all(_cost(tiles, per_cu, t) > best * 1.01 for t in range(1, s))


def test_slice_rule_known_shapes():
    # one round: 5 tiles x 152 = 760 of 768 slots (64 x 128 tiles, within 1 % of 765); three rounds of 512
    # for 192 tiles at 8 slices; the 3 x 3 x 64 filter gradient on 64 x 192 tiles
    assert netdef.wgrad_pixel_slices(64, 576, 131072) == 152
    assert netdef.wgrad_pixel_slices(3072, 1024, 12288) == 8
    assert netdef.wgrad_tile(64, 576, 64) == (64, 192, 2)
    assert netdef.wgrad_tile(64, 1152, 128) is None
    assert netdef.wgrad_tile(32, 1152, 128) == (32, 256, 2)
    assert netdef.wgrad_tile(64, 27, 3) == (64, 64, 4) and netdef.wgrad_tile(64, 64, 64) == (64, 64, 5)
    assert netdef.wgrad_tile(6, 27, 3) is None
    assert netdef.wgrad_pixel_slices(64, 576, 131072, 64) == 169
    assert netdef.wgrad_pixel_slices(1024, 1024, 256) == 1
