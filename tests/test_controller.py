"""The threshold-controller library (libdlmctl.so, host code) against the
controller oracle on random scenarios - same decisions, same loads and times
up to rounding - plus its ABI (exports == header declarations) and argument
validation. No GPU."""
import os
import re

import numpy as np
import pytest

from oracle import controller as oc
from paper_2606_29094_amd import controller as ctl
from paper_2606_29094_amd import dlm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
rng = np.random.default_rng(2024)


@pytest.fixture(scope="module", autouse=True)
def built():
    if not os.path.exists(ctl.LIB_PATH):
        pytest.skip("libdlmctl.so not built")


def test_header_declarations_are_exported():
    src = open(os.path.join(ROOT, "include", "dlm_ctl.h")).read()
    declared = set(re.findall(r"\b(dlm_ctl_[a-z_]+)\s*\(", src))
    assert declared == set(ctl.EXPORTS), declared ^ set(ctl.EXPORTS)
    L = ctl.lib()
    for name in declared:
        assert hasattr(L, name), name


def _rand_curve(n):
    t = np.cumsum(rng.integers(1, 500, n)).astype(float)
    l = np.cumsum(rng.random(n) * 0.01 + 1e-4)
    return t, l


def _both_profiles():
    rt, rl = _rand_curve(int(rng.integers(1, 8)))
    with_cache = rng.random() < 0.7
    ct, cl = _rand_curve(int(rng.integers(1, 6))) if with_cache else (None, None)
    po = oc.Profile(oc.Curve(list(rt), list(rl)), oc.Curve(list(ct), list(cl)) if with_cache else None)
    pl = ctl.make_profile((rt, rl), (ct, cl) if with_cache else None)
    return po, pl


def test_latency_matches_oracle():
    for _ in range(300):
        t, l = _rand_curve(int(rng.integers(1, 9)))
        c = ctl.make_curve(t, l)
        co = oc.Curve(list(t), list(l))
        for x in list(rng.random(5) * t[-1] * 1.5) + list(t):
            assert ctl.latency(c, x) == pytest.approx(oc.latency(co, x), rel=1e-14, abs=0)


def _scenario(cache):
    ng = int(rng.integers(1, 7))
    gam = np.sort(rng.choice(np.linspace(0.3, 0.99, 30), ng, replace=False))
    po, pl = _both_profiles()
    blk = 32 if cache else 0
    ms = int(rng.integers(1, 64))
    slo = float(rng.random() * 30 + 0.1)
    Po = oc.Params(list(gam), blk, ms, slo)
    Pl = ctl.make_params(gam, blk, ms, slo)
    return ng, po, pl, Po, Pl


def _rand_req(ng):
    steps = np.sort(rng.integers(0, 300, ng)).astype(float)
    tokens = float(rng.integers(32, 5000))
    recomp = float(min(rng.integers(0, 9), steps[0]))
    slo_left = float(rng.random() * 40)
    return tokens, steps, recomp, slo_left


@pytest.mark.parametrize("cache", [False, True])
def test_threshold_choice_matches_oracle(cache):
    for _ in range(400):
        ng, po, pl, Po, Pl = _scenario(cache)
        tokens, steps, recomp, slo_left = _rand_req(ng)
        allowed = int(rng.integers(1, 1 << ng))
        inst_tokens, inst_reqs = float(rng.integers(32, 20000)), int(rng.integers(1, 64))
        ro = oc.Req(tokens, list(steps), slo_left, recomp,
                    allowed=[i for i in range(ng) if (allowed >> i) & 1])
        rl = ctl.make_req(tokens, steps, slo_left, recomp, allowed)
        io = oc.Instance(po, inst_tokens, inst_reqs)
        il = ctl.make_instance(pl, inst_tokens, inst_reqs)
        for gi in range(ng):
            assert ctl.predicted_time_left(Pl, il, rl, gi) == pytest.approx(
                oc.predicted_time_left(Po, io, ro, gi), rel=1e-12, abs=1e-300)
            assert ctl.req_load(Pl, rl, gi) == pytest.approx(oc.req_load(Po, ro, gi), rel=1e-12)
        assert ctl.update_threshold(Pl, il, rl) == oc.update_conf_threshold(Po, io, ro)


@pytest.mark.parametrize("cache", [False, True])
def test_load_control_matches_oracle(cache):
    for _ in range(300):
        ng, po, pl, Po, Pl = _scenario(cache)
        n = int(rng.integers(0, 40))
        raw = [_rand_req(ng) for _ in range(n)]
        ro = [oc.Req(t, list(s), sl, rc) for t, s, rc, sl in raw]
        rl = [ctl.make_req(t, s, sl, rc) for t, s, rc, sl in raw]
        tpr = float(rng.integers(64, 4000))
        cap_o = oc.cluster_capacity(Po, [po] * int(rng.integers(1, 3)), tpr)
        k = int(round(cap_o / oc.cluster_capacity(Po, [po], tpr)))
        cap_l = ctl.capacity(Pl, [pl] * k, tpr)
        assert cap_l == pytest.approx(cap_o, rel=1e-12)
        cap = cap_o * float(rng.choice([0.0, 0.001, 0.01, 0.1, 1.0, 10.0]))
        oc.update_allowed(Po, ro, cap)
        masks = ctl.update_allowed(Pl, rl, cap)
        for r, m in zip(ro, masks):
            assert ctl.mask_to_list(m, ng) == r.allowed


def test_validation():
    P = ctl.make_params([0.5, 0.9])
    prof = ctl.make_profile(([100, 200], [0.01, 0.02]))
    inst = ctl.make_instance(prof, 100, 1)
    r = ctl.make_req(100, [5, 9], 1.0, allowed=0)
    with pytest.raises(dlm.DlmError, match="no allowed"):
        ctl.update_threshold(P, inst, r)
    with pytest.raises(dlm.DlmError, match="ascending"):
        ctl.update_threshold(ctl.make_params([0.9, 0.5]), inst, ctl.make_req(1, [1, 2]))
    with pytest.raises(dlm.DlmError, match="n_gamma"):
        ctl.update_allowed(ctl.make_params([]), [], 1.0)
    with pytest.raises(dlm.DlmError, match="n_gamma"):
        ctl.update_allowed(ctl.make_params(list(np.linspace(0.1, 0.99, 33))), [], 1.0)
    with pytest.raises(dlm.DlmError, match="ascending"):
        ctl.latency(ctl.make_curve([200, 100], [0.01, 0.02]), 50)
    with pytest.raises(dlm.DlmError, match="latency"):
        ctl.latency(ctl.make_curve([100], [0.0]), 50)
    with pytest.raises(dlm.DlmError, match="NaN"):
        ctl.update_allowed(P, [ctl.make_req(1, [1, 2])], float("nan"))
    with pytest.raises(dlm.DlmError, match="out of range"):
        ctl.req_load(P, ctl.make_req(1, [1, 2]), 2)
    with pytest.raises(dlm.DlmError, match="predicted steps"):
        ctl.req_load(P, ctl.make_req(1, [1, float("nan")]), 0)
    # 32 candidates: the full mask is representable
    g32 = list(np.linspace(0.1, 0.99, 32))
    m = ctl.update_allowed(ctl.make_params(g32), [ctl.make_req(1, list(range(32)))], 1e30)
    assert m == [0xFFFFFFFF]
