"""Host replay of the kernels' index ranges (no GPU needed, nothing launched).

dr_check_ranges runs, on the CPU, the same range arithmetic the kernels use
(ranges.hpp: the Bloom insert's chunk windows and partial slices, the probe
pass's block tile ranges, the value sort's tiles) over every chunk, slice,
block and tile a configuration plans, and counts ranges that would leave
their buffers.  Every kernel-indexing change is checked here before it runs
on a GPU.

The shapes cover empty tensors, one element, exactly one tile, ragged
tails, tensors with more insert chunks than tiles (a 9-tile tensor gets 64
chunks), many small tensors, the support of a 60%-dense gradient (the
bucketed insert) and the full-size workloads' plans.
"""
import os

import pytest

from paper_2102_03112_amd import binding as B
from paper_2102_03112_amd import workloads as W


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(B.LIB_PATH):
        from paper_2102_03112_amd import build

        build.build()
    return B.lib()


SHAPES = {
    "empty": [0, 0],
    "one": [0, 1],
    "one_tile": [0, 4096],
    "tile_plus_one": [0, 4097],
    "resnet20_conv_37k": [0, 36864],  # 9 tiles, 64 insert chunks
    "two_tiles_ragged": [0, 2 * 4096 + 5],
    "zero_inside": [0, 100, 100, 5000, 5000, 5001],
    "many_small": [0] + [7 * (i + 1) * (i + 3) for i in range(40)],
    "ragged_big": [0, 1_000_003, 1_000_003 + 4096 * 37 + 1],
}


@pytest.mark.parametrize("name", list(SHAPES))
@pytest.mark.parametrize("ratio", [(1, 100), (1, 1000), (1, 1), (0, 1), None])
def test_ranges_small_shapes(L, name, ratio):
    offs = SHAPES[name]
    # make the offsets cumulative where they are given as sizes
    if name == "many_small":
        acc = [0]
        for x in offs[1:]:
            acc.append(acc[-1] + x)
        offs = acc
    cfg = B.Config(offs, ratio, 1e-3, 5, 8)
    bad, msg = B.check_ranges(cfg)
    assert bad == 0, msg


@pytest.mark.parametrize("fpr", [1e-2, 1e-4, 0.5])
def test_ranges_other_rates(L, fpr):
    for offs in (SHAPES["resnet20_conv_37k"], SHAPES["zero_inside"], SHAPES["ragged_big"]):
        bad, msg = B.check_ranges(B.Config(offs, (1, 100), fpr, 3, 16))
        assert bad == 0, msg


@pytest.mark.parametrize("name", W.ORDER)
def test_ranges_workloads(L, name):
    cfg = B.Config.from_workload(W.WORKLOADS[name])
    bad, msg = B.check_ranges(cfg)
    assert bad == 0, msg


def test_the_unclamped_chunk_window_would_wrap():
    """The bitmap chunk window of the direct insert for a 9-tile tensor with
    64 chunks of one tile each: chunks 10..63 start past the tensor's end.
    Without the clamp of the window's start, the word count wb - wa of such a
    chunk wraps in 32-bit arithmetic to nearly 2^32, and the chunk's loop
    reads that far past the selection bitmap.  The clamped window (the
    kernel's, replayed by dr_check_ranges above) is empty instead."""
    ntiles, per, words = 9, 1, 128
    for c in range(64):
        wb = min(ntiles, (c + 1) * per) * words
        wa_unclamped = c * per * words
        wa = min(wa_unclamped, wb)
        assert 0 <= wb - wa <= per * words
        if c >= 10:
            assert (wb - wa_unclamped) % (1 << 32) > (1 << 31)


def test_ranges_reject_bad_config(L):
    with pytest.raises(B.DeepReduceError):
        B.check_ranges(B.Config([5, 10], (1, 100), 1e-3, 5, 8))
