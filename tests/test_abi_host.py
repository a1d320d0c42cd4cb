"""Host-side checks of the C ABI (no GPU needed, nothing is launched).

The library must load on a machine without a GPU and export every function
include/deepreduce.h declares; its host-only helpers must agree with the
oracle; and every invalid argument must be rejected with DR_EINVAL before
anything reaches the device.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2102_03112_amd import binding as B
from paper_2102_03112_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "deepreduce.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(B.LIB_PATH):
        from paper_2102_03112_amd import build

        build.build()
    return B.lib()


def declared_functions():
    text = open(HEADER).read()
    return re.findall(r"DR_EXPORT\s+[\w\s\*]+?\b(dr_\w+)\s*\(", text)


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) == len(set(names)) == 18
    assert sorted(names) == sorted(B.EXPORTS)
    for n in names:
        assert hasattr(L, n), n


@pytest.mark.parametrize("n,fpr", [(0, 1e-3), (1, 1e-3), (369, 1e-3), (10_486, 1e-3), (255_571, 1e-3),
                                   (19_099_546, 1e-4), (147_843, 1e-3), (1000, 0.5), (77, 1e-9)])
def test_bloom_params_match_oracle(L, n, fpr):
    assert B.bloom_params(n, fpr) == oracle.bloom_params(n, fpr)


@pytest.mark.parametrize("fpr", [0.0, 1.0, -1.0, 2.0, float("nan")])
def test_bloom_params_reject_bad_rate(L, fpr):
    with pytest.raises(B.DeepReduceError):
        B.bloom_params(100, fpr)


def test_sigma_bits_match_oracle(L):
    for n in list(range(0, 70)) + [1023, 1024, 1025, 280_873, 1 << 31, (1 << 31) + 1]:
        assert B.sigma_bits(n) == oracle.sigma_bits(n)


def test_payload_layout_is_aligned_and_covers_the_oracle_payload(L):
    w = W.WORKLOADS["normal_1m"]
    cfg = B.Config.from_workload(w)
    total, off = B.payload_layout(cfg)
    assert off[0] == 0 and off[-1] == total and all(o % 256 == 0 for o in off)
    g = W.generate(w)
    (res,) = oracle.roundtrip(g, w.offsets(), w.ratio, w.fpr, w.degree, w.n_seg, want_dense=False)
    bits = res.payload_bits()
    used = 64 + (bits["index"] + bits["values"] + 32 * oracle.sigma_words(res.P.size)) // 8
    assert used <= total
    for name in W.ORDER:
        wl = W.WORKLOADS[name]
        t, o = B.payload_layout(B.Config.from_workload(wl))
        assert len(o) == wl.n_tensors + 1 and t > 0


def test_workspace_bound_grows_with_size(L):
    a = B.workspace_bytes(1 << 20, 1)
    b = B.workspace_bytes(1 << 24, 1)
    c = B.workspace_bytes(1 << 24, 24)
    assert 0 < a < b < c
    assert b < 80 * (1 << 24)  # a few tens of bytes per element


# ---------------------------------------------------------------------------
# argument validation: each call returns DR_EINVAL before any device work.
# Pointers below are never dereferenced because validation fails first.
# ---------------------------------------------------------------------------
FAKE = ctypes.c_void_p(1 << 20)


def _cfg(offsets=(0, 1000), ratio=(1, 100), fpr=1e-3, degree=5, n_seg=8, policy=0, segmentation=0):
    return B.Config(list(offsets), ratio, fpr, degree, n_seg, policy, 0, segmentation)


@pytest.mark.parametrize("bad", [
    dict(fpr=0.0), dict(fpr=1.0), dict(degree=8), dict(n_seg=5000), dict(segmentation=2),
    dict(ratio=(2, 1)), dict(ratio=(1, 0)), dict(offsets=(0, 10, 5)), dict(offsets=(1, 10)),
    dict(offsets=(0, 1 << 32)), dict(policy=5),
])
def test_config_rejected(L, bad):
    cfg = _cfg(**bad)
    assert L.dr_payload_layout(ctypes.byref(cfg.c), None) == 0
    st = L.dr_roundtrip(FAKE, ctypes.byref(cfg.c), FAKE, 1 << 30, FAKE, None, None, None, FAKE, 1 << 40, None)
    assert st == B.DR_EINVAL


def test_decode_sum_rejects_bad_arguments(L):
    cfg = _cfg()
    big = 1 << 40
    one = (ctypes.c_void_p * 65)(*([FAKE.value] * 65))
    nul = (ctypes.c_void_p * 2)(FAKE.value, None)
    f = L.dr_payload_decode_sum
    assert f(one, 0, ctypes.byref(cfg.c), 1.0, FAKE, None, FAKE, big, None) == B.DR_EINVAL
    assert f(one, 65, ctypes.byref(cfg.c), 1.0, FAKE, None, FAKE, big, None) == B.DR_EINVAL
    assert f(None, 1, ctypes.byref(cfg.c), 1.0, FAKE, None, FAKE, big, None) == B.DR_EINVAL
    assert f(nul, 2, ctypes.byref(cfg.c), 1.0, FAKE, None, FAKE, big, None) == B.DR_EINVAL
    assert f(one, 2, ctypes.byref(cfg.c), 1.0, None, None, FAKE, big, None) == B.DR_EINVAL
    assert f(one, 2, ctypes.byref(cfg.c), float("nan"), FAKE, None, FAKE, big, None) == B.DR_EINVAL
    assert f(one, 2, ctypes.byref(cfg.c), float("inf"), FAKE, None, FAKE, big, None) == B.DR_EINVAL
    assert f(one, 2, ctypes.byref(cfg.c), 1.0, FAKE, None, FAKE, 1000, None) == B.DR_EINVAL
    assert f(one, 2, None, 1.0, FAKE, None, FAKE, big, None) == B.DR_EINVAL
    bad = _cfg(policy=9)
    assert f(one, 2, ctypes.byref(bad.c), 1.0, FAKE, None, FAKE, big, None) == B.DR_EINVAL


def test_null_config_and_zero_tensors(L):
    assert L.dr_payload_layout(None, None) == 0
    cfg = _cfg()
    cfg.c.n_tensors = 0
    assert L.dr_payload_layout(ctypes.byref(cfg.c), None) == 0


def test_encode_decode_reject_bad_buffers(L):
    cfg = _cfg()
    total, _ = B.payload_layout(cfg)
    big = 1 << 40
    # payload too small
    assert L.dr_payload_encode(FAKE, ctypes.byref(cfg.c), FAKE, total - 1, None, FAKE, big, None) == B.DR_EINVAL
    # null gradient / payload / dense output
    assert L.dr_payload_encode(None, ctypes.byref(cfg.c), FAKE, total, None, FAKE, big, None) == B.DR_EINVAL
    assert L.dr_payload_decode(None, ctypes.byref(cfg.c), FAKE, None, None, None, FAKE, big, None) == B.DR_EINVAL
    assert L.dr_payload_decode(FAKE, ctypes.byref(cfg.c), None, None, None, None, FAKE, big, None) == B.DR_EINVAL
    # workspace too small, missing, or not 256-byte aligned
    assert L.dr_payload_encode(FAKE, ctypes.byref(cfg.c), FAKE, total, None, FAKE, 1000, None) == B.DR_EINVAL
    assert L.dr_payload_encode(FAKE, ctypes.byref(cfg.c), FAKE, total, None, None, big, None) == B.DR_EINVAL
    odd = ctypes.c_void_p((1 << 20) + 4)
    assert L.dr_payload_encode(FAKE, ctypes.byref(cfg.c), FAKE, total, None, odd, big, None) == B.DR_EINVAL
    assert "workspace" in B.last_error()


def test_standalone_calls_reject_bad_arguments(L):
    big = 1 << 40
    # top-r: r > d, d >= 2^32, null outputs
    assert L.dr_sparsify_topr(FAKE, 10, 11, FAKE, None, FAKE, FAKE, big, None) == B.DR_EINVAL
    assert L.dr_sparsify_topr(FAKE, 1 << 32, 1, FAKE, None, FAKE, FAKE, big, None) == B.DR_EINVAL
    assert L.dr_sparsify_topr(FAKE, 10, 5, None, None, FAKE, FAKE, big, None) == B.DR_EINVAL
    assert L.dr_sparsify_topr(FAKE, 10, 5, FAKE, None, None, FAKE, big, None) == B.DR_EINVAL
    assert L.dr_sparsify_topr(FAKE, 10, 5, FAKE, None, FAKE, FAKE, 10, None) == B.DR_EINVAL
    # Bloom: m not a positive multiple of 32, k out of range
    for m, k in [(0, 3), (33, 3), (1 << 32, 3), (64, 0), (64, 33)]:
        assert L.dr_bloom_encode(FAKE, FAKE, 10, m, k, FAKE, None, FAKE, big, None) == B.DR_EINVAL
        assert L.dr_bloom_decode(FAKE, m, k, 100, FAKE, 100, FAKE, FAKE, big, None) == B.DR_EINVAL
    assert L.dr_bloom_encode(FAKE, None, 10, 64, 3, FAKE, None, FAKE, big, None) == B.DR_EINVAL
    assert L.dr_bloom_decode(FAKE, 64, 3, 1 << 32, FAKE, 100, FAKE, FAKE, big, None) == B.DR_EINVAL
    # curve fit: degree, segments, sizes
    assert L.dr_curvefit_encode(FAKE, FAKE, 10, 8, 1, FAKE, FAKE, None, FAKE, big, None) == B.DR_EINVAL
    assert L.dr_curvefit_encode(FAKE, FAKE, 10, 5, 0, FAKE, FAKE, None, FAKE, big, None) == B.DR_EINVAL
    assert L.dr_curvefit_encode(FAKE, FAKE, 1 << 32, 5, 8, FAKE, FAKE, None, FAKE, big, None) == B.DR_EINVAL
    assert L.dr_curvefit_decode(FAKE, FAKE, FAKE, 10, 8, 1, FAKE, None, FAKE, big, None) == B.DR_EINVAL
    assert L.dr_curvefit_decode(FAKE, FAKE, None, 10, 5, 1, FAKE, None, FAKE, big, None) == B.DR_EINVAL


def test_trace_end_without_begin_is_rejected(L):
    assert L.dr_trace_end(None, 0) == B.DR_EINVAL


def test_parse_record_roundtrips_a_synthetic_header():
    # header layout of include/deepreduce.h, built independently with numpy
    d, n_sel, n_pos, n_v, m, k, pol, seed, de, se, b = 1000, 10, 14, 12, 64, 3, 1, 99, 1, 2, 4
    words = (n_v * b + 31) // 32
    rb = 64 + m // 8 + 4 * se * (de + 1) + 4 * words
    hdr = np.array([0x31435244, 64, d, n_sel, n_pos, n_v, m, k, 1, pol, seed, de, se, b, rb, 0], dtype="<u4")
    body = np.concatenate([np.arange(m // 32, dtype="<u4"), np.arange(se * (de + 1), dtype="<f4").view("<u4"),
                           np.full(words, 7, dtype="<u4")])
    buf = np.concatenate([hdr, body]).view(np.uint8)
    rec = B.parse_record(buf, 0)
    assert (rec.d, rec.n_selected, rec.n_positives, rec.n_values, rec.m_bits, rec.k, rec.hash_id, rec.policy,
            rec.seed, rec.deg_eff, rec.seg_eff, rec.sigma_b, rec.rec_bytes) == (d, n_sel, n_pos, n_v, m, k, 1, pol,
                                                                                 seed, de, se, b, rb)
    np.testing.assert_array_equal(rec.bits, [0, 1])
    np.testing.assert_array_equal(rec.sigma, [7, 7])
