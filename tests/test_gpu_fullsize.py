"""GPU parity at the workloads' full sizes, in the configuration bench.py
times (one dr_roundtrip over the whole gradient, workspace from
dr_workspace_bytes).

ResNet-50-, NCF- and VGG-16-sized gradients are checked element by element
against the full oracle (tens of seconds of CPU each).  The 350M-parameter
transformer split into 24 tensors is coded in one GPU round trip (a
module-scoped fixture); each of its 24 tensors is then compared element by
element against the oracle's round trip of that tensor (about two seconds
of CPU each, one test per tensor), and every tensor is also checked against
properties that hold at any size.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2102_03112_amd import binding as B
from paper_2102_03112_amd import workloads as W
from _gpu_util import check_roundtrip, log, release_workspace, run_roundtrip, unpack_sigma

pytestmark = pytest.mark.gpu


def _full(name, policy=oracle.POLICY_P0, seed=0):
    w = W.WORKLOADS[name]
    log(f"full-size {name} policy={policy}: generating d={w.d}")
    g = W.generate(w)
    cfg = B.Config.from_workload(w, policy, seed)
    log(f"full-size {name}: GPU round trip")
    out = run_roundtrip(g, cfg)
    log(f"full-size {name}: oracle")
    refs = oracle.roundtrip(g, w.offsets(), w.ratio, w.fpr, w.degree, w.n_seg, policy=policy, seed=seed)
    log(f"full-size {name}: compare")
    check_roundtrip(g, cfg, out, refs)
    release_workspace()


def test_resnet50_25m_full():
    _full("resnet50_25m")


def test_resnet50_25m_random_policy_full():
    _full("resnet50_25m", oracle.POLICY_RANDOM, 20210205)


def _full_partitioned(name):
    w = W.WORKLOADS[name]
    log(f"full-size {w.name} layout=partitioned: generating d={w.d}")
    g = W.generate(w)
    cfg = B.Config.from_workload(w, filter_layout=B.FILTER_PARTITIONED)
    out = run_roundtrip(g, cfg)
    log(f"full-size {w.name} layout=partitioned: oracle")
    refs = oracle.roundtrip(g, w.offsets(), w.ratio, w.fpr, w.degree, w.n_seg, layout=oracle.LAYOUT_PARTITIONED)
    check_roundtrip(g, cfg, out, refs)
    release_workspace()


def test_resnet50_25m_partitioned_layout_full():
    _full_partitioned("resnet50_25m")


@pytest.mark.skip(reason="partitioned filter of 3.7e8 bits: a smaller one (4e7 bits) went silent on the GPU with a "
                         "build that probed such filters in rounds (cause not found); kept off the GPU")
def test_ncf_32m_partitioned_layout_full():
    """The 44.7 MiB partitioned filter of the NCF support."""
    _full_partitioned("ncf_32m")


def test_ncf_32m_support_full():
    _full("ncf_32m")


def test_vgg16_138m_full():
    _full("vgg16_138m")


def _properties(g, w, t, rec, counts, idx, val, dense):
    """What must hold for any tensor, without running the oracle on it."""
    d = g.size
    r = oracle.ratio_count(d, *w.ratio)
    n_sel, nv, nv_dec, flags = [int(x) for x in counts]
    assert (n_sel, flags) == (r, 0)
    assert nv == nv_dec == rec.n_positives == rec.n_values and rec.n_selected == r
    m, k = oracle.bloom_params(r, w.fpr)
    assert (rec.m_bits, rec.k, rec.hash_id, rec.d) == (m, k, 1, d)
    # reorder-map width and fit shape for the reported count (sizes only)
    assert rec.sigma_b == max(1, (nv - 1).bit_length())
    assert (rec.seg_eff, rec.deg_eff) == (min(w.n_seg, max(1, nv // (w.degree + 1))), w.degree)
    P = idx[:nv].astype(np.int64)
    assert np.all(np.diff(P) > 0) and P[0] >= 0 and P[-1] < d
    # the r largest magnitudes are all positives (no false negatives)
    kth = np.partition(np.abs(g), d - r)[d - r]
    big = np.flatnonzero(np.abs(g) > kth)
    assert np.isin(big, P).all()
    # false positives: binomial around fill^k over the non-members
    fill = np.unpackbits(rec.bits.view(np.uint8)).mean()
    q = fill**k
    fp = nv - r
    assert abs(fp - q * (d - r)) < 6 * math.sqrt((d - r) * q) + 10
    # the reorder map is a permutation of the ranks
    ranks = unpack_sigma(rec.sigma, nv, rec.sigma_b)
    assert np.array_equal(np.bincount(ranks.astype(np.int64), minlength=nv), np.ones(nv, np.int64))
    # dense is the values at P and zero elsewhere
    np.testing.assert_array_equal(dense[P], val[:nv])
    off = np.ones(d, bool)
    off[P] = False
    assert np.all(dense[off] == 0)
    # the fitted values follow the sorted curve: relative L2 error of the fit
    V = g[P]
    order = np.argsort(-V.astype(np.float64), kind="stable")
    err = np.linalg.norm(val[:nv][order] - V[order]) / np.linalg.norm(V)
    assert err < 0.5


@pytest.fixture(scope="module")
def transformer_run():
    w = W.WORKLOADS["transformer_355m_x24"]
    log(f"full-size {w.name}: generating d={w.d}")
    g = W.generate(w)
    cfg = B.Config.from_workload(w)
    log(f"full-size {w.name}: GPU round trip")
    out = run_roundtrip(g, cfg)
    release_workspace()
    yield w, g, out
    del g, out


def test_transformer_355m_x24_properties(transformer_run):
    w, g, out = transformer_run
    off = w.offsets()
    for t in range(w.n_tensors):
        a, b = off[t], off[t + 1]
        rec = B.parse_record(out["payload"], out["rec_off"][t])
        _properties(g[a:b], w, t, rec, out["counts"][t], out["idx"][a:b], out["val"][a:b], out["dense"][a:b])
    log(f"full-size {w.name}: properties hold on all {w.n_tensors} tensors")


# 16 tensors of 14,784,299 elements, then 8 of 14,784,298 (array_split order)
@pytest.mark.parametrize("t", range(24))
def test_transformer_355m_x24_tensor(transformer_run, t):
    w, g, out = transformer_run
    off = w.offsets()
    a, b = off[t], off[t + 1]
    log(f"full-size {w.name}: oracle on tensor {t} ({b - a} elements)")
    ref = oracle.roundtrip_tensor(g[a:b], oracle.ratio_count(b - a, *w.ratio), w.fpr, w.degree, w.n_seg)
    sub = B.Config([0, b - a], w.ratio, w.fpr, w.degree, w.n_seg)
    one = {
        "payload": out["payload"][out["rec_off"][t]:out["rec_off"][t + 1]],
        "rec_off": [0, out["rec_off"][t + 1] - out["rec_off"][t]],
        "counts": out["counts"][t:t + 1],
        "idx": out["idx"][a:b], "val": out["val"][a:b], "dense": out["dense"][a:b],
    }
    check_roundtrip(g[a:b], sub, one, [ref])
