"""A CPU model of the bucketed query's index arithmetic (the kernels
k_qb_count, k_qb_scan, k_qb_scatter, k_qb_test and k_qb_fill), replayed with
numpy over the same constants, table layout and buffer sizes the host plans,
checking that every load and store stays inside its buffer, that each
round's scatter fills its bucket array exactly once, and that the bitmap it
ends with is the direct query's (Section 4, policy P0: every index whose k
bits are all set).

The path, for a tensor of d indices and an m-bit filter with k hashes:
  round j < k: the live list (round 0: the indices 0..d-1) is cut into
    chunks (round 0: QB_CH indices each; later rounds: chunk s is the part
    of the list test block s of the previous round wrote); chunk c's
    entries are counted by bin (the 2^QB_SL-bit slice of hash j's bit) into
    column c of a bins x ncol table (round 0 by a count pass, later rounds
    by the previous round's test blocks); one block per bin turns its row
    into exclusive offsets and writes the bin's total; a chunk's entries
    then go to bucket start + its row offset + their rank among the chunk's
    entries of that bin; one block per slice tests its bucket, writes each
    index, or a dead marker, back to the same position of the list, and
    counts its survivors by their next bin;
  round k: the same with the index region (2^QB_RL indices) as the bin, and
    one block per region writes the region's words of the positives bitmap.
Positions come from the oracle's hash (the model checks the plumbing, not
the hash)."""
import numpy as np
import pytest

import oracle

QB_SL, QB_RL = 19, 19
QB_CH = 4 * 1024 * 9  # 4 batches of 1024 threads x 9 entries
QB_MAX_BINS = 2048
TILE = 4096
TILE_WORDS = TILE // 32
DEAD = 0xFFFFFFFF


def cdiv(a, b):
    return -(-a // b)


def bucketed_query(words, m, k, d, layout, m_cap):
    """The kernels' arithmetic; returns the tensor's bitmap words."""
    nsl_cap = cdiv(m_cap, 1 << QB_SL)
    nch_cap = cdiv(d, QB_CH)
    nreg = cdiv(d, 1 << QB_RL)
    assert nsl_cap <= QB_MAX_BINS and nreg <= QB_MAX_BINS
    ncol = max(nch_cap, nsl_cap)
    qcap = cdiv(d, 64) * 64
    tab_words = max(nsl_cap, nreg) * ncol
    rows_words = (k + 1) * QB_MAX_BINS
    qlist = np.full(qcap, 0xA5A5A5A5, dtype=np.uint64)
    qbkt = np.full(qcap, 0xA5A5A5A5, dtype=np.uint64)
    qtab = np.zeros(tab_words, dtype=np.int64)
    qrow = np.zeros(rows_words, dtype=np.int64)
    nsl = cdiv(m, 1 << QB_SL)
    assert nsl <= nsl_cap  # the kernels' check of the actual filter against the plan
    ntiles = max(1, cdiv(d, TILE))

    def key_of(el, j):
        if j == k:
            return (el >> QB_RL).astype(np.int64)
        return (oracle.bloom_pos(el.astype(np.uint32), j, m, k, layout) >> QB_SL).astype(np.int64)

    def write_column(c, keys, nb):
        cnt = np.bincount(keys, minlength=nb)
        assert cnt.size == nb, "a key past the round's bins"
        idx = np.arange(nb) * ncol + c
        assert idx.size == 0 or idx.max() < tab_words
        qtab[idx] = cnt

    # round 0's count pass: chunk c is indices [c QB_CH, (c + 1) QB_CH)
    for c in range(nch_cap):
        el = np.arange(c * QB_CH, min(d, (c + 1) * QB_CH), dtype=np.uint64)
        write_column(c, key_of(el, 0), nsl)
    for j in range(k + 1):
        fin = j == k
        nb = nreg if fin else nsl
        # the round's chunks: places [lo_c, hi_c) of the list
        if j == 0:
            nch = nch_cap
            lo = np.arange(nch) * QB_CH
            hi = np.minimum(lo + QB_CH, d)
        else:
            nch = nsl
            prev = qrow[(j - 1) * QB_MAX_BINS:(j - 1) * QB_MAX_BINS + nsl]
            lo = np.cumsum(prev) - prev
            hi = lo + prev
        assert nch <= ncol
        # k_qb_scan: each row to exclusive offsets, the row total to qrow
        for b in range(nb):
            row = qtab[b * ncol:b * ncol + nch].copy()
            qtab[b * ncol:b * ncol + nch] = np.cumsum(row) - row
            assert j * QB_MAX_BINS + b < rows_words
            qrow[j * QB_MAX_BINS + b] = row.sum()
        tot = qrow[j * QB_MAX_BINS:j * QB_MAX_BINS + nb]
        bstart = np.cumsum(tot) - tot
        n_out = int(tot.sum())
        # k_qb_scatter: bucket start + the chunk's row offset + rank within
        # (chunk, bin); the rank order inside a chunk is the LDS atomics'
        # (any order): shuffle it
        ex_l, el_l, ch_l = [], [], []
        for c in range(nch):
            x = np.arange(lo[c], hi[c], dtype=np.int64)
            if j == 0:
                e = x.astype(np.uint64)
            else:
                assert x.size == 0 or x.max() < qcap
                e = qlist[x].copy()
            live = e != DEAD
            ex_l.append(x[live])
            el_l.append(e[live])
            ch_l.append(np.full(int(live.sum()), c, dtype=np.int64))
        ex, el, chunk = np.concatenate(ex_l), np.concatenate(el_l).astype(np.uint64), np.concatenate(ch_l)
        key = key_of(el, j)
        assert (key < nb).all()
        assert n_out == ex.size, "the counts cover exactly the live entries"
        order = np.lexsort((np.random.default_rng(j).permutation(ex.size), key, chunk))
        kk, cc, ee = key[order], chunk[order], el[order]
        grp = kk * (nch + 1) + cc
        first = np.r_[True, grp[1:] != grp[:-1]]
        starts = np.maximum.accumulate(np.where(first, np.arange(grp.size), 0))
        rank = np.arange(grp.size) - starts
        dst = bstart[kk] + qtab[kk * ncol + cc] + rank
        assert dst.size == 0 or (dst.min() >= 0 and dst.max() < qcap)
        written = np.zeros(n_out, dtype=np.int64)
        np.add.at(written, dst, 1)
        assert (written == 1).all(), "the scatter must fill its bucket array exactly once"
        qbkt[dst] = ee
        if fin:
            break
        # k_qb_test: block s loads its slice and tests its bucket, then
        # counts its survivors by their bin in round j + 1 (column s)
        m_words = m // 32
        nb_next = nreg if j + 1 == k else nsl
        for s in range(nsl):
            a, b_ = int(bstart[s]), int(bstart[s] + tot[s])
            w0 = s << (QB_SL - 5)
            nw = min(1 << (QB_SL - 5), m_words - w0)
            assert nw > 0 and w0 + nw <= m_words
            sl = words[w0:w0 + nw]
            idx = qbkt[a:b_]
            p = (oracle.bloom_pos(idx.astype(np.uint32), j, m, k, layout).astype(np.int64) - (s << QB_SL)) % (1 << 32)
            inside = p < nw * 32
            assert inside.all(), "a bucket holds only its slice's bits"
            alive = ((sl[(p >> 5).clip(0, nw - 1)] >> (p & 31).astype(np.uint32)) & 1).astype(bool)
            assert b_ <= qcap
            qlist[a:b_] = np.where(alive, idx, DEAD)
            assert s < ncol
            write_column(s, key_of(idx[alive], j + 1), nb_next)
    # k_qb_fill: block r sets its region's bits and writes its words
    bits = np.zeros(ntiles * TILE_WORDS, dtype=np.uint32)
    tot = qrow[k * QB_MAX_BINS:k * QB_MAX_BINS + nreg]
    bstart = np.cumsum(tot) - tot
    for r in range(nreg):
        w0 = r * (1 << (QB_RL - 5))
        nw = min(1 << (QB_RL - 5), ntiles * TILE_WORDS - w0)
        assert nw > 0
        bm = np.zeros(1 << (QB_RL - 5), dtype=np.uint32)
        li = qbkt[int(bstart[r]):int(bstart[r] + tot[r])].astype(np.int64) - (r << QB_RL)
        assert ((li >= 0) & (li < (1 << QB_RL))).all()
        np.bitwise_or.at(bm, li >> 5, (np.uint32(1) << (li & 31).astype(np.uint32)))
        bits[w0:w0 + nw] = bm[:nw]
    return bits


def bitmap_of(idx, d):
    ntiles = max(1, cdiv(d, TILE))
    out = np.zeros(ntiles * TILE_WORDS, dtype=np.uint32)
    idx = np.asarray(idx, dtype=np.int64)
    np.bitwise_or.at(out, idx >> 5, (np.uint32(1) << (idx & 31).astype(np.uint32)))
    return out


CASES = [
    # name, d, n items, m (bits), k, layout, planned m_cap
    ("slices_6_regions_4", 3 * (1 << 19) + 12345, 20000, 5 * (1 << 19) + 96, 5, oracle.LAYOUT_STANDARD, None),
    ("one_chunk_one_slice", 5000, 300, 1 << 14, 3, oracle.LAYOUT_STANDARD, None),
    ("partitioned", (1 << 19) + 7, 9000, 3 * (1 << 19) + 32 * 77, 4, oracle.LAYOUT_PARTITIONED, None),
    ("planned_larger_than_actual", 200_000, 5000, (1 << 19) + 64, 2, oracle.LAYOUT_STANDARD, 9 * (1 << 19)),
    ("k1", 70_000, 2000, 1 << 20, 1, oracle.LAYOUT_STANDARD, None),
    ("more_slices_than_chunks", 50_000, 20_000, 5 * (1 << 19) + 3200, 3, oracle.LAYOUT_STANDARD, None),
]


@pytest.mark.parametrize("name,d,n,m,k,layout,m_cap", CASES, ids=[c[0] for c in CASES])
def test_bucketed_query_model(name, d, n, m, k, layout, m_cap):
    rng = np.random.default_rng(len(name) * 7 + k)
    S = np.sort(rng.choice(d, size=n, replace=False)).astype(np.uint32)
    words = oracle.bloom_encode(S, m, k, layout)
    got = bucketed_query(words, m, k, d, layout, m_cap or m)
    want = bitmap_of(oracle.bloom_query(words, m, k, d, layout), d)
    assert np.array_equal(got, want)
