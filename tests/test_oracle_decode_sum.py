"""Pins of the oracle's summing receiver (Section 2, the aggregated gradient;
Section 6.4, payloads exchanged by all-gather)."""
import numpy as np

import oracle
from paper_2102_03112_amd import workloads as W

OFF = [0, 700, 700, 2600]
D = OFF[-1]


def _payloads(n, fpr=1e-2, policy=oracle.POLICY_P0):
    return [oracle.roundtrip(W.normal(D, 40 + p, scale=1e-3), OFF, (3, 100), fpr, 3, 4, policy=policy, seed=p)
            for p in range(n)]


def test_one_payload_at_scale_one_is_the_plain_receiver():
    (res,) = _payloads(1)
    out = oracle.decode_sum([res], D, OFF, 1.0)
    want = np.concatenate([r.dense for r in res])
    np.testing.assert_array_equal(out, want)


def test_brute_force_over_index_value_pairs():
    # each payload as a dictionary {global index: received value}, summed
    # element by element in payload order
    pays = _payloads(5, policy=oracle.POLICY_RANDOM)
    scale = 1.0 / 5
    out = oracle.decode_sum(pays, D, OFF, scale)
    terms = [dict() for _ in range(D)]
    for p, res in enumerate(pays):
        for t, r in enumerate(res):
            for i, v in zip(r.P_dec.tolist(), r.vals.tolist()):
                terms[OFF[t] + i][p] = v
    for i in range(D):
        s = np.float32(0.0)
        for p in sorted(terms[i]):
            s = np.float32(s + np.float32(terms[i][p]))
        assert out[i] == np.float32(np.float32(scale) * s), i
    # the supports overlap somewhere, so the test exercises real sums
    assert max(len(t) for t in terms) >= 2


def test_a_payload_repeated_n_times_averages_to_itself():
    (res,) = _payloads(1)
    single = np.concatenate([r.dense for r in res])
    # y + y and a halving are exact in fp32
    np.testing.assert_array_equal(oracle.decode_sum([res] * 2, D, OFF, 0.5), single)
    # longer sums round once per term: within a few units in the last place
    for n in (3, 4, 7):
        out = oracle.decode_sum([res] * n, D, OFF, 1.0 / n)
        np.testing.assert_allclose(out, single, rtol=4 * n * np.finfo(np.float32).eps, atol=0)


def test_sum_is_zero_off_every_support():
    pays = _payloads(3)
    out = oracle.decode_sum(pays, D, OFF, 0.5)
    on = np.zeros(D, bool)
    for res in pays:
        for t, r in enumerate(res):
            on[OFF[t] + r.P_dec.astype(np.int64)] = True
    assert np.all(out[~on] == 0)
    assert np.count_nonzero(out[on]) > 0
