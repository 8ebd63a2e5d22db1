"""Pins of the threshold-controller oracle (Algorithms 1, 2, 5 and 6) against
hand-worked scenarios and invariants stated by the algorithms' text: the
highest allowed threshold that fits the budget is chosen, else the lowest; the
worst-case committed load stays within capacity unless only the lowest
threshold is left; unlimited capacity keeps every threshold."""
import numpy as np
import pytest

from oracle import controller as oc

rng = np.random.default_rng(5)


def test_latency_interpolation():
    c = oc.Curve([100, 200, 400], [1.0, 2.0, 3.0])
    assert oc.latency(c, 50) == 1.0
    assert oc.latency(c, 100) == 1.0
    assert oc.latency(c, 150) == 1.5
    assert oc.latency(c, 300) == 2.5
    assert oc.latency(c, 600) == 4.0          # along the last segment
    assert oc.latency(oc.Curve([64], [0.7]), 1e6) == 0.7


def _inst(tokens=200, reqs=1):
    prof = oc.Profile(oc.Curve([100, 200, 400], [1.0, 2.0, 3.0]),
                      oc.Curve([32, 128, 256], [0.1, 0.2, 0.4]))
    return oc.Instance(prof, tokens, reqs)


def test_alg1_picks_highest_threshold_within_budget():
    p = oc.Params([0.5, 0.7, 0.9])
    inst = _inst(200)                          # 2 s per step
    r = oc.Req(100, [10, 20, 40], allowed=[0, 1, 2])
    for slo, want in [(50, 1), (80, 2), (100, 2), (40, 1), (39.9, 0), (10, 0)]:
        r.slo_left_s = slo
        assert oc.update_conf_threshold(p, inst, r) == want, slo
        assert np.isclose(oc.predicted_time_left(p, inst, r, 2), 80.0)
    r.allowed = [0, 1]
    r.slo_left_s = 1000
    assert oc.update_conf_threshold(p, inst, r) == 1


def test_alg6_prices_cache_and_recompute_steps_separately():
    p = oc.Params([0.5, 0.9], cache_block=32)
    inst = _inst(tokens=300, reqs=4)           # cache batch 128 tokens -> 0.2 s
    r = oc.Req(300, [12, 40], recomp_steps_left=5)
    # 35 cache steps x 0.2 s + 5 recompute steps x latency(300) = 2.5 s
    assert np.isclose(oc.predicted_time_left(p, inst, r, 1), 35 * 0.2 + 5 * 2.5)
    assert np.isclose(oc.predicted_time_left(p, inst, r, 0), 7 * 0.2 + 5 * 2.5)
    # no cache-step curve: the single curve is used for both
    inst2 = oc.Instance(oc.Profile(inst.profile.recompute), 300, 4)
    # cache batch of 128 tokens on the recompute curve: 1.0 + 28/100
    assert np.isclose(oc.predicted_time_left(p, inst2, r, 1), 35 * 1.28 + 5 * 2.5)


def test_loads_alg2_and_alg5():
    r = oc.Req(100, [10, 30], recomp_steps_left=2)
    assert oc.req_load(oc.Params([0.5, 0.9]), r, 1) == 3000
    # with caching: (30 - 2) cache steps of 32 tokens + 2 recomputes of 100
    assert oc.req_load(oc.Params([0.5, 0.9], cache_block=32), r, 1) == 28 * 32 + 200


def test_capacity_alg2_and_alg5():
    prof = oc.Profile(oc.Curve([256, 512, 1024], [0.01, 0.015, 0.03]),
                      oc.Curve([64, 256], [0.004, 0.008]))
    p = oc.Params([0.5], slo_s=10.0)
    assert np.isclose(oc.cluster_capacity(p, [prof], 0), 1024 / 0.03 * 10)
    assert np.isclose(oc.cluster_capacity(p, [prof, prof], 0), 2 * 1024 / 0.03 * 10)
    pc = oc.Params([0.5], cache_block=32, max_seqs_per_batch=8, slo_s=10.0)
    # block of 31 cache steps of 256 tokens (0.008 s) + one recompute of 512 (0.015 s)
    want = (256 * 31 + 512) / (0.008 * 31 + 0.015) * 10
    assert np.isclose(oc.cluster_capacity(pc, [prof], 512), want)


def test_alg2_hand_worked():
    p = oc.Params([0.5, 0.9])
    reqs = [oc.Req(100, [10, 30]) for _ in range(3)]   # loads 1000 / 3000 each
    oc.update_allowed(p, reqs, 5000)
    assert [r.allowed for r in reqs] == [[0, 1], [0], [0]]
    oc.update_allowed(p, reqs, 7000)
    assert [r.allowed for r in reqs] == [[0, 1], [0, 1], [0]]
    oc.update_allowed(p, reqs, 9000)
    assert [r.allowed for r in reqs] == [[0, 1], [0, 1], [0, 1]]
    oc.update_allowed(p, reqs, 0)
    assert [r.allowed for r in reqs] == [[0], [0], [0]]


def _random_reqs(n, ng):
    reqs = []
    for _ in range(n):
        steps = np.sort(rng.integers(1, 200, ng))     # higher threshold, more steps
        reqs.append(oc.Req(float(rng.integers(64, 4096)), [float(s) for s in steps],
                           slo_left_s=float(rng.random() * 20),
                           recomp_steps_left=float(rng.integers(0, 4))))
    return reqs


@pytest.mark.parametrize("cache", [0, 32])
def test_alg2_invariants(cache):
    gam = [0.5, 0.6, 0.7, 0.8, 0.9]
    p = oc.Params(gam, cache_block=cache, max_seqs_per_batch=16, slo_s=5.0)
    for trial in range(50):
        reqs = _random_reqs(int(rng.integers(1, 12)), len(gam))
        for r in reqs:
            r.recomp_steps_left = min(r.recomp_steps_left, r.pred_steps_left[0])
        cap = float(rng.random() * 2e6)
        oc.update_allowed(p, reqs, cap)
        used, forced = 0.0, False
        for r in reqs:
            assert r.allowed == list(range(max(r.allowed) + 1))   # a prefix of the candidates
            top = max(r.allowed)
            used += oc.req_load(p, r, top)
            forced |= top == 0
        minimum = sum(oc.req_load(p, r, 0) for r in reqs)
        if minimum <= cap:
            assert used <= cap * (1 + 1e-12) or forced
        oc.update_allowed(p, reqs, float("inf"))
        assert all(r.allowed == list(range(len(gam))) for r in reqs)


def test_alg1_monotone_in_budget():
    p = oc.Params([0.5, 0.6, 0.7, 0.8, 0.9])
    inst = _inst(350)
    for r in _random_reqs(30, 5):
        r.allowed = list(range(5))
        prev = -1
        for slo in np.linspace(0, 2000, 41):
            r.slo_left_s = slo
            g = oc.update_conf_threshold(p, inst, r)
            assert g >= prev
            prev = g


def test_alg2_brute_force_lexicographic_maximum():
    """Load control against an exhaustive search on tiny batches with integer
    loads (exact sums): the maxima given in arrival order are the
    lexicographically largest assignment in which every request above the
    lowest threshold has a worst case (earlier requests at their maxima, this
    one at its maximum, later ones at the lowest threshold) within capacity."""
    import itertools
    for trial in range(400):
        G, n = int(rng.integers(1, 4)), int(rng.integers(1, 5))
        p = oc.Params(list(np.linspace(0.5, 0.9, G)))
        reqs = [oc.Req(float(rng.integers(1, 20)),
                       [float(x) for x in np.sort(rng.integers(1, 10, G))]) for _ in range(n)]
        L = [[r.num_tokens * r.pred_steps_left[g] for g in range(G)] for r in reqs]
        cap = float(rng.integers(0, int(sum(max(l) for l in L)) + 10))

        def feasible(a):
            for i in range(n):
                worst = sum(L[j][a[j]] for j in range(i + 1)) + sum(L[j][0] for j in range(i + 1, n))
                if a[i] > 0 and worst > cap:
                    return False
            return True

        best = max(a for a in itertools.product(range(G), repeat=n) if feasible(a))
        oc.update_allowed(p, reqs, cap)
        assert [max(r.allowed) for r in reqs] == list(best), (trial, L, cap)
        assert all(r.allowed == list(range(max(r.allowed) + 1)) for r in reqs)


def test_alg1_brute_force_over_candidates():
    """The threshold choice against every allowed candidate: the chosen one
    fits the budget and no higher allowed one does, or none fits and it is the
    lowest allowed."""
    p = oc.Params([0.5, 0.6, 0.7, 0.8, 0.9], cache_block=32, max_seqs_per_batch=8)
    inst = oc.Instance(oc.Profile(oc.Curve([256, 4096], [0.01, 0.08]),
                                  oc.Curve([32, 256], [0.004, 0.01])), 3000.0, 5)
    for r in _random_reqs(200, 5):
        r.recomp_steps_left = min(r.recomp_steps_left, r.pred_steps_left[0])
        r.allowed = sorted(set(int(x) for x in rng.integers(0, 5, int(rng.integers(1, 6)))))
        g = oc.update_conf_threshold(p, inst, r)
        t = {a: oc.predicted_time_left(p, inst, r, a) for a in r.allowed}
        fitting = [a for a in r.allowed if t[a] <= r.slo_left_s]
        if fitting:
            assert t[g] <= r.slo_left_s and all(a <= g for a in fitting)
        else:
            assert g == min(r.allowed)
