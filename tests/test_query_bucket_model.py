"""A CPU model of the bucketed query's index arithmetic (the kernels
k_qb_count, k_qb_scan, k_qb_scatter, k_qb_test and k_qb_fill), replayed with
numpy over the same constants, table layout and buffer sizes the host plans,
checking that every load and store stays inside its buffer, that each
round's scatter fills its bucket array exactly once, and that the bitmap it
ends with is the direct query's (Section 4, policy P0: every index whose k
bits are all set).

The path, for a tensor of d indices and an m-bit filter with k hashes:
  round j < k: the live list (round 0: the indices 0..d-1) is cut into
    chunks of QB_CH entries; chunk c's
    entries are counted by bin (the 2^QB_SL-bit slice of hash j's bit) into
    column c of a bins x nch_cap table; one block per bin turns its row into
    exclusive offsets and writes the bin's total; a chunk's entries then go
    to bucket start + its row offset + their rank among the chunk's entries
    of that bin; one block per slice tests its bucket and writes each index,
    or a dead marker, back to the same position of the list;
  round k: the same with the index region (2^QB_RL indices) as the bin, and
    one block per region writes the region's words of the positives bitmap.
Positions come from the oracle's hash (the model checks the plumbing, not
the hash)."""
import numpy as np
import pytest

import oracle

QB_SL, QB_RL = 19, 19
QB_CH = 2 * 1024 * 16
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
    qcap = cdiv(d, 64) * 64
    tab_words = max(nsl_cap, nreg) * nch_cap
    rows_words = (k + 1) * QB_MAX_BINS
    qlist = np.full(qcap, 0xA5A5A5A5, dtype=np.uint64)
    qbkt = np.full(qcap, 0xA5A5A5A5, dtype=np.uint64)
    qtab = np.zeros(tab_words, dtype=np.int64)
    qrow = np.zeros(rows_words, dtype=np.int64)
    nsl = cdiv(m, 1 << QB_SL)
    assert nsl <= nsl_cap  # the kernels' check of the actual filter against the plan
    ntiles = max(1, cdiv(d, TILE))
    for j in range(k + 1):
        fin = j == k
        nb = nreg if fin else nsl
        n_in = d if j == 0 else int(qrow[(j - 1) * QB_MAX_BINS:(j - 1) * QB_MAX_BINS + nsl].sum())
        nch = cdiv(n_in, QB_CH)
        assert nch <= nch_cap
        x = np.arange(n_in, dtype=np.int64)
        if j == 0:
            e = x.astype(np.uint64)
        else:
            assert n_in <= qcap
            e = qlist[:n_in].copy()
        live = e != DEAD
        ex, el = x[live], e[live].astype(np.uint64)
        if fin:
            key = (el >> QB_RL).astype(np.int64)
        else:
            key = (oracle.bloom_pos(el.astype(np.uint32), j, m, k, layout) >> QB_SL).astype(np.int64)
        assert (key < nb).all()
        chunk = ex // QB_CH
        # k_qb_count: column c of the table
        cnt = np.zeros((nb, nch), dtype=np.int64)
        np.add.at(cnt, (key, chunk), 1)
        tix = np.arange(nb)[:, None] * nch_cap + np.arange(nch)[None, :]
        assert tix.size == 0 or tix.max() < tab_words
        qtab[tix] = cnt
        # k_qb_scan: each row to exclusive offsets, the row total to qrow
        for b in range(nb):
            row = qtab[b * nch_cap:b * nch_cap + nch].copy()
            qtab[b * nch_cap:b * nch_cap + nch] = np.cumsum(row) - row
            assert j * QB_MAX_BINS + b < rows_words
            qrow[j * QB_MAX_BINS + b] = row.sum()
        tot = qrow[j * QB_MAX_BINS:j * QB_MAX_BINS + nb]
        bstart = np.cumsum(tot) - tot
        n_out = int(tot.sum())
        assert n_out == ex.size
        # k_qb_scatter: bucket start + the chunk's row offset + rank within
        # (chunk, bin); the rank order inside a chunk is the LDS atomics'
        # (any order): shuffle it
        order = np.lexsort((np.random.default_rng(j).permutation(ex.size), key, chunk))
        kk, cc, ee = key[order], chunk[order], el[order]
        grp = kk * (nch + 1) + cc
        first = np.r_[True, grp[1:] != grp[:-1]]
        starts = np.maximum.accumulate(np.where(first, np.arange(grp.size), 0))
        rank = np.arange(grp.size) - starts
        dst = bstart[kk] + qtab[kk * nch_cap + cc] + rank
        assert dst.size == 0 or (dst.min() >= 0 and dst.max() < qcap)
        written = np.zeros(n_out, dtype=np.int64)
        np.add.at(written, dst, 1)
        assert (written == 1).all(), "the scatter must fill its bucket array exactly once"
        qbkt[dst] = ee
        if fin:
            break
        # k_qb_test: block s loads its slice and tests its bucket
        m_words = m // 32
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
]


@pytest.mark.parametrize("name,d,n,m,k,layout,m_cap", CASES, ids=[c[0] for c in CASES])
def test_bucketed_query_model(name, d, n, m, k, layout, m_cap):
    rng = np.random.default_rng(len(name) * 7 + k)
    S = np.sort(rng.choice(d, size=n, replace=False)).astype(np.uint32)
    words = oracle.bloom_encode(S, m, k, layout)
    got = bucketed_query(words, m, k, d, layout, m_cap or m)
    want = bitmap_of(oracle.bloom_query(words, m, k, d, layout), d)
    assert np.array_equal(got, want)
