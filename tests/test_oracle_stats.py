"""Pins of the confidence-statistics oracle (the Step Predictor's confidence and
progress features): a hand-worked example, numpy's own quantile/mean/min/max
routines, and invariants that a dropped term or a wrong index would break."""
import numpy as np
import pytest

from oracle import stats as ost

rng = np.random.default_rng(77)


def test_hand_worked_example():
    # prompt of 3, output of 7: unmasked output confidences 0.9, 0.2, 0.5, 0.7
    tok_conf = np.array([9, 9, 9, 0.9, 0.0, 0.2, 0.5, 0.0, 0.7, 0.0])
    mask = np.array([0, 0, 0, 0, 1, 0, 0, 1, 0, 1], dtype=np.uint8)
    s = ost.confidence_stats(tok_conf, mask, prompt_len=3, block_start=7, block_len=3)
    # sorted: 0.2 0.5 0.7 0.9; h(0.25) = 0.75 -> 0.2 + 0.75*0.3 = 0.425;
    # median h = 1.5 -> 0.6; h(0.75) = 2.25 -> 0.7 + 0.25*0.2 = 0.75; mean 0.575
    want = [4, 0.2, 0.425, 0.6, 0.575, 0.75, 0.9, 1]
    np.testing.assert_allclose(s, want, rtol=0, atol=1e-15)


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 17, 256, 1000])
def test_matches_numpy_routines(n):
    P, G = 11, n + 40
    tok_conf = rng.random(P + G)
    mask = np.ones(P + G, dtype=np.uint8)
    mask[:P] = 0
    pos = rng.choice(np.arange(P, P + G), size=n, replace=False)
    mask[pos] = 0
    s = ost.confidence_stats(tok_conf, mask, P, P, 32)
    v = tok_conf[pos]
    want = [n, v.min(), np.quantile(v, 0.25), np.median(v), v.mean(), np.quantile(v, 0.75),
            v.max()]
    np.testing.assert_allclose(s[:7], want, rtol=1e-13, atol=1e-15)
    assert s[7] == np.sum(mask[P:P + 32] == 0)


def test_prompt_and_masked_positions_are_excluded():
    P, G = 20, 30
    tok_conf = rng.random(P + G)
    mask = np.zeros(P + G, dtype=np.uint8)
    mask[P + 10:] = 1
    s1 = ost.confidence_stats(tok_conf, mask, P, P, 32)
    t2 = tok_conf.copy()
    t2[:P] = 5.0                    # prompt values never enter
    t2[P + 10:] = -3.0              # still-masked values never enter
    s2 = ost.confidence_stats(t2, mask, P, P, 32)
    np.testing.assert_array_equal(s1, s2)
    assert s1[0] == 10


def test_empty_output_gives_zeros():
    mask = np.array([0, 0, 1, 1, 1], dtype=np.uint8)
    s = ost.confidence_stats(np.full(5, 0.3), mask, 2, 2, 3)
    np.testing.assert_array_equal(s, np.zeros(ost.N_STATS))


def test_order_and_permutation_invariance():
    P, G = 5, 300
    tok_conf = rng.random(P + G) ** 3
    mask = (rng.random(P + G) < 0.4).astype(np.uint8)
    mask[:P] = 0
    s = ost.confidence_stats(tok_conf, mask, P, P + 64, 64)
    assert s[1] <= s[2] <= s[3] <= s[5] <= s[6]
    assert s[1] <= s[4] <= s[6]
    perm = P + rng.permutation(G)
    t2, m2 = tok_conf.copy(), mask.copy()
    t2[P:], m2[P:] = tok_conf[perm], mask[perm]
    s2 = ost.confidence_stats(t2, m2, P, P + 64, 64)
    np.testing.assert_allclose(s2[:7], s[:7], rtol=1e-14)


def test_constant_values_and_single_value():
    mask = np.array([0, 0, 0, 0], dtype=np.uint8)
    s = ost.confidence_stats(np.array([0.0, 0.25, 0.25, 0.25]), mask, 1, 1, 3)
    np.testing.assert_allclose(s, [3, 0.25, 0.25, 0.25, 0.25, 0.25, 0.25, 3], atol=0)
    s = ost.confidence_stats(np.array([0.0, 0.6]), np.array([0, 0], np.uint8), 1, 1, 1)
    np.testing.assert_allclose(s, [1, 0.6, 0.6, 0.6, 0.6, 0.6, 0.6, 1], atol=0)


def test_predictor_features():
    s = np.array([4, 0.2, 0.425, 0.6, 0.575, 0.75, 0.9, 1])
    f = ost.predictor_features(0.9, 256, 10, 2, 8, 32, s)
    assert len(f) == 11
    assert f["full_progress"] == 10 / 256 and f["full_unmask_progress"] == 4 / 256
    assert f["block_progress"] == 0.25 and f["block_unmask_progress"] == 1 / 32
    assert f["output_median_confidence"] == 0.6
