"""A CPU model of the probe pass's tile scan (the decoupled look-back over
the blocks' contiguous tile ranges, segmented at tensor starts), run under
random interleavings, against a direct per-tensor exclusive scan.

The probe pass gives each block a contiguous range of tiles (ranges in
block order) and must produce, for every tile, the count of positives in
the earlier tiles of its tensor, and each tensor's total.  A block:
  1. publishes the sum of its trailing segment (its tiles of its last
     tile's tensor): as inclusive if that segment starts at the tensor's
     first tile, else as an aggregate;
  2. if its first tile continues a tensor that began in an earlier block,
     walks back over the preceding blocks' entries in windows of 64 (each
     entry read on its own, so entries may change between the reads of one
     window), adding aggregates until an inclusive entry; a block whose
     range lies inside one tensor then publishes its inclusive prefix;
  3. scans its tiles, segmented at tensor starts: a lane-level emulation of
     the kernel's wave scans (shuffles up by 1, 2, ..., 32) and the
     combination of the 16 waves' results through shared memory.
Blocks start in index order and at most `resident` of them run at once; a
block waits only for blocks with smaller indices, so every wait must end.
"""
import random

import numpy as np
import pytest

PB_THREADS = 1024
WAVES = PB_THREADS // 64
AGG, INC = 1, 2


def block_ranges(ntiles, grid):
    per = (ntiles + grid - 1) // grid
    out = []
    for b in range(grid):
        lo = min(ntiles, b * per)
        out.append((lo, min(ntiles, lo + per)))
    return out


def segmented_scan_block(tcnt, t_begin, t_end, tile_tensor, tile0, ntiles_of, carry):
    """Step 3 for one block, lane by lane as the kernel runs it."""
    toff, totals = {}, {}
    for c0 in range(t_begin, t_end, PB_THREADS):
        t = c0 + np.arange(PB_THREADS)
        inn = t < t_end
        tt = np.where(inn, tile_tensor[np.minimum(t, len(tile_tensor) - 1)], 0)
        v = np.where(inn, tcnt[np.minimum(t, len(tcnt) - 1)], 0).astype(np.int64)
        f = inn & (t == tile0[tt])
        last = inn & (t + 1 == tile0[tt] + ntiles_of[tt])
        sv, sf = v.copy().reshape(WAVES, 64), f.copy().reshape(WAVES, 64)
        lane = np.arange(64)
        d = 1
        while d < 64:
            pv = np.concatenate([sv[:, :d], sv[:, :-d]], axis=1)  # shfl_up: lanes < d keep their own
            pf = np.concatenate([sf[:, :d], sf[:, :-d]], axis=1)
            act = lane >= d
            sv = np.where(act & ~sf, sv + pv, sv)
            sf = np.where(act, sf | pf, sf)
            d <<= 1
        wsum, wflag = sv[:, 63].copy(), sf[:, 63].copy()
        for wv in range(WAVES):
            pre = carry
            for q in range(wv):
                pre = wsum[q] if wflag[q] else pre + wsum[q]
            incl = np.where(sf[wv], sv[wv], pre + sv[wv])
            for ln in range(64):
                x = wv * 64 + ln
                if inn[x]:
                    toff[int(t[x])] = int(incl[ln] - v[x])
                    if last[x]:
                        totals[int(tt[x])] = int(incl[ln])
        for q in range(WAVES):
            carry = wsum[q] if wflag[q] else carry + wsum[q]
    return toff, totals


def block_program(b, lo, hi, st, tcnt, tile_tensor, tile0, ntiles_of, out):
    """The look-back of block b as a generator: each yield is a point where
    another block may run."""
    if hi <= lo:
        return
    t_first, t_last = tile_tensor[lo], tile_tensor[hi - 1]
    trail0 = max(lo, tile0[t_last])
    cont = lo > tile0[t_first]
    s = int(tcnt[trail0:hi].sum())
    trail_inc = trail0 > lo or not cont
    st[b] = (INC if trail_inc else AGG, s)
    yield
    excl = 0
    if cont:
        j = b
        while True:
            nwin = min(64, j)
            vals = []
            for lane in range(nwin):  # one read per lane; others may publish in between
                vals.append(st[j - 1 - lane])
                yield
            first_unpub = next((x for x, e in enumerate(vals) if e[0] == 0), 64)
            first_inc = next((x for x, e in enumerate(vals) if e[0] == INC), 64)
            if first_inc < first_unpub:
                excl += sum(e[1] for e in vals[: first_inc + 1])
                break
            upto = min(first_unpub, nwin)
            excl += sum(e[1] for e in vals[:upto])
            j -= upto
            assert j > 0, "walked past block 0"
            if upto == 0:
                yield  # spin
        if t_first == t_last:
            st[b] = (INC, excl + s)
            yield
    toff, totals = segmented_scan_block(tcnt, lo, hi, tile_tensor, tile0, ntiles_of, excl if cont else 0)
    out.append((toff, totals))


def run_model(tensor_tiles, grid, resident, seed):
    rng = random.Random(seed)
    nt = len(tensor_tiles)
    tile0 = np.concatenate([[0], np.cumsum(tensor_tiles)[:-1]]).astype(np.int64)
    ntiles_of = np.asarray(tensor_tiles, np.int64)
    ntiles = int(ntiles_of.sum())
    tile_tensor = np.repeat(np.arange(nt), tensor_tiles)
    tcnt = np.asarray([rng.randrange(0, 4097) for _ in range(ntiles)], np.int64)
    st = [(0, 0)] * grid
    out = []
    ranges = block_ranges(ntiles, grid)
    progs = [block_program(b, lo, hi, st, tcnt, tile_tensor, tile0, ntiles_of, out) for b, (lo, hi) in
             enumerate(ranges)]
    running, nxt, steps = [], 0, 0
    while nxt < grid or running:
        while nxt < grid and len(running) < resident:  # dispatch in block order
            running.append(progs[nxt])
            nxt += 1
        p = rng.choice(running)
        try:
            next(p)
        except StopIteration:
            running.remove(p)
        steps += 1
        assert steps < 10_000_000, "a wait did not end"
    toff, totals = {}, {}
    for a, b in out:
        toff.update(a)
        totals.update(b)
    # direct scan
    for t in range(nt):
        c = tcnt[tile0[t]: tile0[t] + ntiles_of[t]]
        ex = np.concatenate([[0], np.cumsum(c)[:-1]])
        for x in range(ntiles_of[t]):
            assert toff[int(tile0[t] + x)] == ex[x], (t, x)
        assert totals[t] == int(c.sum()), t
    assert len(toff) == ntiles


@pytest.mark.parametrize("seed", range(6))
def test_lookback_random_layouts(seed):
    rng = random.Random(1000 + seed)
    nt = rng.randrange(1, 40)
    tiles = [rng.choice([1, 1, 2, 3, 5, 8, 40, 200, 1300]) for _ in range(nt)]
    grid = rng.choice([1, 2, 3, 7, 16, 64, 70, 130, 256])
    resident = rng.choice([1, 2, 3, grid])
    run_model(tiles, grid, resident, seed)


def test_lookback_one_tensor_many_blocks():
    # 6,240 tiles over 256 blocks (a 25.6 M-element tensor): windows of 64
    run_model([6240], 256, 256, 7)
    run_model([6240], 256, 3, 8)


def test_lookback_tensor_boundaries_inside_blocks():
    # many small tensors per block, and tensors longer than a window of blocks
    run_model([1] * 300 + [700] + [2] * 50 + [5000], 224, 224, 9)
