"""Non-finite gradient values (the paper is silent; outside the codec's
contract).  The library promises only that every kernel terminates and
that the sender reports DR_FLAG_NONFINITE for the tensor: these tests feed
NaN and +-Inf through every selection mode, segmentation and value model
and check exactly that, plus that finite tensors of the same batch are
coded as the oracle codes them alone.
"""
import numpy as np
import pytest

import oracle
from paper_2102_03112_amd import binding as B
from paper_2102_03112_amd import workloads as W
from _gpu_util import check_roundtrip, log, run_roundtrip

pytestmark = pytest.mark.gpu


def _poisoned(d, seed, zero_frac=0.0):
    g = W.sparse_normal(d, seed, zero_frac) if zero_frac else W.normal(d, seed)
    rng = np.random.default_rng(seed + 1)
    at = rng.choice(d, 6, replace=False)
    g[at[:2]] = np.nan
    g[at[2:4]] = np.inf
    g[at[4:]] = -np.inf
    return g


CASES = {
    # name: (ratio, fpr, degree, n_seg, segmentation, fit_model, zero_frac)
    "topr_poly": ((1, 100), 1e-3, 5, 8, oracle.SEG_EQUAL, oracle.FIT_POLY, 0.0),
    "support_poly": (None, 1e-4, 3, 16, oracle.SEG_EQUAL, oracle.FIT_POLY, 0.4),
    "topr_chord": ((1, 100), 1e-3, 5, 8, oracle.SEG_CHORD, oracle.FIT_POLY, 0.0),
    "topr_heuristic": ((1, 100), 1e-3, 1, 0, oracle.SEG_EQUAL, oracle.FIT_POLY, 0.0),
    "topr_dexp": ((1, 100), 1e-3, 3, 4, oracle.SEG_EQUAL, oracle.FIT_DEXP, 0.0),
}


@pytest.mark.parametrize("name", list(CASES))
def test_nonfinite_input_terminates_and_is_flagged(name):
    ratio, fpr, D, S, seg, model, zf = CASES[name]
    # tensor 0 is poisoned, tensor 1 is finite
    d0, d1 = 40_000, 30_001
    g = np.concatenate([_poisoned(d0, 5, zf), W.sparse_normal(d1, 6, zf) if zf else W.normal(d1, 6)])
    off = [0, d0, d0 + d1]
    log(f"nonfinite {name}")
    cfg = B.Config(off, ratio, fpr, D, S, segmentation=seg, fit_model=model)
    out = run_roundtrip(g, cfg)
    flags = out["counts"][:, 3].astype(np.int64)
    assert flags[0] & B.FLAG_NONFINITE
    assert not flags[0] & B.FLAG_STALLED
    assert flags[1] == 0
    # the finite tensor is coded as the oracle codes it alone
    ref = oracle.roundtrip(g[d0:], [0, d1], ratio, fpr, D, S, seg_mode=seg, model=model)
    sub = B.Config([0, d1], ratio, fpr, D, S, segmentation=seg, fit_model=model)
    one = {
        "payload": out["payload"][out["rec_off"][1]:out["rec_off"][2]],
        "rec_off": [0, out["rec_off"][2] - out["rec_off"][1]],
        "counts": out["counts"][1:2],
        "idx": out["idx"][d0:], "val": out["val"][d0:], "dense": out["dense"][d0:],
    }
    check_roundtrip(g[d0:], sub, one, ref)
