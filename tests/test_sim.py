"""The event-driven rescheduling simulation (host logic, oracle planner).

The planner here is the CPU oracle's Algorithm 1, so nothing in this file
needs a GPU.  The GPU test of the same simulation runs the library's planner
and must reproduce these runs event for event.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2510_13668_amd import sim


def oracle_planner(cur, rem, inst, beta, *, n_inst, bucket, n_buckets, theta, min_rem, mem_cap,
                   max_moves):
    out = oracle.plan(cur, rem, inst, beta, n_inst=n_inst, bucket=bucket, n_buckets=n_buckets,
                      theta=theta, min_rem=min_rem, mem_cap=mem_cap, max_moves=max_moves)
    return out["moves"]


SMALL = sim.SimConfig(n_inst=4, rate_per_8=1.6, duration_s=240.0, n_buckets=64, bucket=512,
                      interval_s=2.0, max_moves=3, seed=3)


@pytest.mark.parametrize("policy", sim.POLICIES)
def test_runs_are_deterministic_and_consistent(policy):
    a = sim.simulate(SMALL, policy, oracle_planner)
    b = sim.simulate(SMALL, policy, oracle_planner)
    assert a == b
    assert a.finished > 20 and a.ticks == 119
    if policy == "none":
        assert a.migrations == 0 and a.moves == []
    assert a.migrations == len(a.moves) <= a.ticks * SMALL.max_moves
    assert 0 < a.mean_tpot_ms <= a.p99_tpot_ms


def test_policies_see_the_same_requests():
    """Without migrations the placement is fixed by arrival order, so a
    policy whose planner never moves anything reproduces "none" exactly."""
    never = lambda *args, **kw: []
    a = sim.simulate(SMALL, "none", None)
    b = sim.simulate(SMALL, "oracle", never)
    assert (a.exec_var_ms2, a.p99_tpot_ms, a.finished) != (0, 0, 0)
    assert a.p99_tpot_ms == b.p99_tpot_ms and a.finished == b.finished
    assert a.mean_tpot_ms == b.mean_tpot_ms


def test_rescheduling_reduces_imbalance():
    """A loaded cluster with heavy-tailed outputs: planning with the true
    remaining lengths lowers the time-averaged variance of the iteration time
    below no rescheduling."""
    cfg = dataclasses.replace(SMALL, n_inst=8, rate_per_8=0.6, duration_s=300.0, max_moves=4,
                              seed=11)
    none = sim.simulate(cfg, "none", None)
    orc = sim.simulate(cfg, "oracle", oracle_planner)
    assert orc.migrations > 0
    assert orc.exec_var_ms2 < none.exec_var_ms2


def test_planner_moves_are_checked():
    def wrong(cur, rem, inst, beta, **kw):
        return [(0, int(inst[0]) ^ 1, 0)] if len(cur) else []
    with pytest.raises(RuntimeError):
        sim.simulate(SMALL, "oracle", wrong)
