"""dr_roundtrip_static, the round trip for callers that cannot allocate, against
dr_roundtrip with a caller workspace: the same payload bytes, positives,
values, dense gradient and counts, on calls in a row through the C ABI (the
second with a smaller input, so that it runs over the first one's leftovers
in the shared static scratch), and a clear DR_ECAPACITY for a gradient whose
scratch would not fit.
"""
import numpy as np
import pytest

from paper_2102_03112_amd import binding as B
from paper_2102_03112_amd import workloads as W
from _gpu_util import dev_tensor, host, log, run_roundtrip, sync

pytestmark = pytest.mark.gpu


def _run_static(g, cfg):
    import torch

    total, rec_off = B.payload_layout(cfg)
    d = cfg.d
    gd = dev_tensor(g) if d else torch.zeros(1, dtype=torch.float32, device="cuda")
    payload = torch.zeros(total, dtype=torch.uint8, device="cuda")
    dense = torch.full((max(d, 1),), 9.0, dtype=torch.float32, device="cuda")
    idx = torch.full((max(d, 1),), -1, dtype=torch.int32, device="cuda")
    val = torch.zeros(max(d, 1), dtype=torch.float32, device="cuda")
    counts = torch.zeros(4 * cfg.n_tensors, dtype=torch.int64, device="cuda")
    B.roundtrip_static(gd, cfg, payload, dense, idx, val, counts)
    sync()
    return dict(payload=host(payload), rec_off=rec_off, dense=host(dense)[:d], idx=host(idx)[:d].view(np.uint32),
                val=host(val)[:d], counts=host(counts).reshape(cfg.n_tensors, 4))


CALLS = [
    # one 1 M-element tensor, then a smaller ragged batch, then a small tensor
    ("normal_1m", W.normal(1_048_576, 41), [0, 1_048_576], (1, 100), 1e-3, 5, 8),
    ("ragged", W.normal(300_001, 42), [0, 0, 1, 4097, 150_000, 300_001], (1, 100), 1e-3, 5, 8),
    ("small", W.normal(36_864, 43), [0, 36_864], (1, 100), 1e-2, 3, 4),
]


def test_static_scratch_round_trips_match_the_workspace_round_trip():
    for name, g, off, ratio, fpr, D, S in CALLS:
        log(f"static round trip {name} d={g.size}")
        cfg = B.Config(off, ratio, fpr, D, S)
        a = _run_static(g, cfg)
        b = run_roundtrip(g, cfg)
        np.testing.assert_array_equal(a["counts"], b["counts"])
        assert np.all(a["counts"][:, 3] == 0)
        np.testing.assert_array_equal(a["payload"], b["payload"])
        np.testing.assert_array_equal(a["idx"], b["idx"])
        np.testing.assert_array_equal(a["val"].view(np.uint32), b["val"].view(np.uint32))
        np.testing.assert_array_equal(a["dense"].view(np.uint32), b["dense"].view(np.uint32))


def test_static_scratch_rejects_a_gradient_too_large():
    import torch

    d = 8 << 20  # needs several hundred MiB of scratch
    cfg = B.Config([0, d], (1, 100), 1e-3, 5, 8)
    total, _ = B.payload_layout(cfg)
    g = torch.zeros(d, dtype=torch.float32, device="cuda")
    payload = torch.zeros(total, dtype=torch.uint8, device="cuda")
    dense = torch.zeros(d, dtype=torch.float32, device="cuda")
    with pytest.raises(B.DeepReduceError) as e:
        B.roundtrip_static(g, cfg, payload, dense, None, None, None)
    assert e.value.status == B.DR_ECAPACITY
    assert "static scratch" in B.last_error()
