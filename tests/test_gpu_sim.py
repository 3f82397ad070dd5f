"""The event-driven rescheduling simulation driven by the library.

Every tick the library projects the loads and plans the migrations on the
GPU.  The whole run (every move at every tick, and the metrics) must equal
the same run planned by the CPU oracle.
"""
import dataclasses

import pytest

from paper_2510_13668_amd import sim
from test_sim import SMALL, oracle_planner

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("policy", ["current", "predicted", "oracle"])
@pytest.mark.parametrize("n_inst", [4, 16])
def test_library_run_equals_oracle_run(policy, n_inst):
    cfg = dataclasses.replace(SMALL, n_inst=n_inst, duration_s=120.0 if n_inst > 8 else 240.0,
                              max_moves=4)
    print(f"simulation n_inst={n_inst} policy={policy}", flush=True)
    lib = sim.LibraryPlanner()
    a = sim.simulate(cfg, policy, lib)
    b = sim.simulate(cfg, policy, oracle_planner)
    assert lib.calls == a.ticks > 0
    assert a.moves == b.moves
    assert a == b
    assert a.migrations > 0
