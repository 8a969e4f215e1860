"""CPU pins of the MISA-T controller replay (misa_t/): the equations of Sec. 3-4 against hand-derived
values and the identities they imply, the Admit rule case by case, and invariants of a replay driving the
library's host validator with synthetic class mixes."""
import math

import numpy as np
import pytest

from misa_t import controller as M
from misa_t.replay import Replay, ReplayConfig


def test_prefill_cost_and_hold_rule_by_hand():
    # Eq. prefill-cost: 0.2 s backlog + (12000 - 8000) tokens at 20000 tokens/s
    assert M.prefill_cost(0.2, 12000, 8000, 20000) == pytest.approx(0.4)
    assert M.prefill_cost(0.0, 500, 500, 1e4) == 0.0
    # Eq. hold-condition: holding 0.1 s for an 8000-token prefix at 20000 tok/s (0.4 s of prefill) pays off
    assert M.hold_preferable(0.1, 0.05, 0.0, 8000, 20000)
    assert not M.hold_preferable(0.5, 0.05, 0.0, 8000, 20000)
    assert not M.hold_preferable(0.0, 0.0, 0.0, 0, 20000)  # nothing cached: never hold


def test_base_cap_and_hit_degradation():
    assert M.base_cap(1000, 64) == 15 and M.base_cap(1024, 64) == 16 and M.base_cap(63, 64) == 0
    assert M.hit_degradation(0.95, 0.80) == pytest.approx(0.15)
    assert M.hit_degradation(0.80, 0.95) == 0.0


def test_space_caps_by_hand():
    """Eq. spatial-demand and Eq. workloadcap on a worked example: C = 1000 blocks; demands 10 x 20,
    4 x 100 and 2 x 200 blocks: S = 200, 400, 400, so M = 200, 400, 400 and K = 10, 4, 2."""
    N = {"rlvr": 10, "rlhf": 4, "agentic": 2}
    kbar = {"rlvr": 20, "rlhf": 100, "agentic": 200}
    assert M.spatial_demand(N, kbar) == {"rlvr": 200, "rlhf": 400, "agentic": 400}
    Mq, K = M.space_caps(1000, N, kbar)
    assert Mq == pytest.approx({"rlvr": 200, "rlhf": 400, "agentic": 400})
    assert K == {"rlvr": 10, "rlhf": 4, "agentic": 2}
    # quotas partition the budget; a class with a tiny share still gets one session
    Mq, K = M.space_caps(1000, {"rlvr": 1, "rlhf": 0, "agentic": 100}, kbar)
    assert sum(Mq.values()) == pytest.approx(1000)
    assert K["rlhf"] == 1 and K["rlvr"] == 1 and K["agentic"] == math.floor(1000 * 20000 / 20020 / 200)


def test_time_caps_by_hand_and_reductions():
    """Eq. block-time-demand and Eq. residency-quota: with equal residency times they reduce to the
    spatial caps; doubling one class's residency doubles its demand weight."""
    N = {"rlvr": 10, "rlhf": 4, "agentic": 2}
    kbar = {"rlvr": 20, "rlhf": 100, "agentic": 200}
    same = {b: 7.0 for b in N}
    assert M.time_caps(1000, N, kbar, same) == M.space_caps(1000, N, kbar)
    T = {"rlvr": 1.0, "rlhf": 1.0, "agentic": 2.0}
    assert M.block_time_demand(N, kbar, T) == {"rlvr": 200, "rlhf": 400, "agentic": 800}
    Mq, K = M.time_caps(1000, N, kbar, T)
    assert Mq == pytest.approx({"rlvr": 1000 * 200 / 1400, "rlhf": 1000 * 400 / 1400, "agentic": 1000 * 800 / 1400})
    assert K == {"rlvr": 7, "rlhf": 2, "agentic": 2}


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_residency_quota_balances_drain_times(seed):
    """Eq. backlog-drain-time under the quotas of Eq. residency-quota: every class with demand drains in
    the same estimated time, sum_b R_b / C (the property the allocation is chosen for)."""
    rng = np.random.default_rng(seed)
    N = {b: int(rng.integers(1, 50)) for b in M.CLASSES}
    kbar = {b: float(rng.uniform(5, 500)) for b in M.CLASSES}
    T = {b: float(rng.uniform(1, 100)) for b in M.CLASSES}
    C = 5000.0
    Mq, _ = M.time_caps(C, N, kbar, T)
    tau = M.drain_times(N, kbar, T, Mq)
    R = M.block_time_demand(N, kbar, T)
    for b in M.CLASSES:
        assert tau[b] == pytest.approx(sum(R.values()) / C)
    # the spatial quotas do not balance them when residency differs
    Ms, _ = M.space_caps(C, N, kbar)
    taus = M.drain_times(N, kbar, T, Ms)
    assert max(taus.values()) > 1.01 * min(taus.values())


def test_no_demand_gives_unit_caps():
    N = {b: 0 for b in M.CLASSES}
    kbar = {b: 10.0 for b in M.CLASSES}
    assert M.space_caps(100, N, kbar)[1] == {b: 1 for b in M.CLASSES}
    assert M.time_caps(100, N, kbar, {b: 1.0 for b in M.CLASSES})[1] == {b: 1 for b in M.CLASSES}


def _ctl(policy, C=1000, kbar=None):
    est = M.ClassEstimator(kbar or {"rlvr": 100, "rlhf": 100, "agentic": 100}, T_prior=10.0)
    c = M.Controller(C, est, policy)
    return c


def test_admit_rule_cases():
    """Admit(r, w): continuations always pass; a new session needs |O| + |P| < K; pending sessions count
    against the cap until a snapshot makes them active."""
    c = _ctl("global")
    c.update_caps({"rlvr": 1})
    assert c.K == 10
    for s in range(10):
        assert c.admit(s, "rlvr")
    assert not c.admit(10, "rlvr")                 # cap reached with pending sessions
    assert c.admit(3, "rlvr")                      # continuation of a pending session
    c.snapshot(finished=[0, 1])
    assert set(c.O) == set(range(2, 10)) and not c.P
    assert c.admit(7, "rlvr")                      # continuation of an active session
    assert c.admit(10, "rlvr") and c.admit(11, "rlvr")
    assert not c.admit(12, "rlvr")


def test_admit_with_class_caps():
    """With class caps a new session also needs headroom in its own class."""
    c = _ctl("space", C=1000, kbar={"rlvr": 50, "rlhf": 100, "agentic": 250})
    c.update_caps({"rlvr": 10, "rlhf": 5, "agentic": 2})
    # S = 500, 500, 500 -> M = 333.3 each -> K = 6, 3, 1
    assert c.class_caps == {"rlvr": 6, "rlhf": 3, "agentic": 1}
    assert c.admit("a0", "agentic") and not c.admit("a1", "agentic")
    assert all(c.admit(f"h{i}", "rlhf") for i in range(3)) and not c.admit("h3", "rlhf")
    assert c.admit("r0", "rlvr")
    assert c.admit("a0", "agentic")                # continuation: no class headroom needed


def test_overload_pressure_contracts_and_recovers():
    c = _ctl("global")
    c.update_caps({"rlvr": 1}, hit_rate=0.9)
    k0 = c.K
    for _ in range(3):                             # a confirmed drop of the hit rate
        c.update_caps({"rlvr": 1}, hit_rate=0.5)
    assert c.K == max(1, int(k0 * 0.8))
    for _ in range(20):
        c.update_caps({"rlvr": 1}, hit_rate=0.9)
    assert c.K == k0


@pytest.mark.parametrize("policy", ["global", "space", "time"])
def test_replay_invariants(policy):
    """A replay whose every batch passes the library's host table validator (kvp_check_tables); pages are
    never double-used; admissions never push |O| + |P| past the cap; the completed mix tracks rho."""
    r = Replay(ReplayConfig(steps=300, pool_pages=3072, seed=3), policy=policy)
    for _ in range(300):
        before = len(r.ctl.O) + len(r.ctl.P)
        r.step()
        assert len(r.ctl.O) + len(r.ctl.P) <= max(before, r.ctl.K) or r.ctl.K == 0
        used = [p for s in r.sessions.values() for p in s.pages] + [p for g in r.group_pages.values() for p in g]
        refs = np.bincount(np.asarray(used, np.int64), minlength=r.cfg.pool_pages) if used else 0
        assert np.array_equal(refs, r.page_refs)   # reference counts match the tables and group pages
        assert len(r.free) + int(np.count_nonzero(r.page_refs)) == r.cfg.pool_pages
    m = r.history[-1]
    assert sum(m["completed"].values()) > 100
    assert m["tv_distance"] < 0.1
    assert 0.0 < m["hit_rate"] < 1.0


def test_replay_is_deterministic():
    a = Replay(ReplayConfig(steps=120, seed=5)).run()
    b = Replay(ReplayConfig(steps=120, seed=5)).run()
    assert a == b
