"""The training planner's launch shapes for the five workloads.

Not a parity test: every shape is checked against the oracle elsewhere.
This pins the plans that measured fastest on MI355X (grid sweeps, block
lengths, sweeper counts at each workload).  The planner computes them on
the host from a fitted cost model and the occupancy API, so a change to the
model, or to what the runtime reports, that moves a workload to a slower
plan shows up here.  A four-sweeper plan displacing the 20 x 20 map's
LDS-resident one (1.74 against 1.29 us per step) was caught this way.
"""
import pytest

import paper_1905_09598_amd as som
import workloads
from gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("ci,variant,grid,block_steps,block", [
    (0, 3, 8, 4, 256),      # 10x10, d = 500: pipelined, LDS rows
    (1, 3, 64, 4, 256),     # 20x20, d = 2000
    (2, 3, 256, 2, 256),    # 30x30, d = 5000
    (3, 4, 256, 8, 256),    # 50x50, d = 10000: pipelined, column walk over streamed rows
    (4, 2, 256, 5, 320),    # 100x100, d = 2048: pipelined, streamed rows, four sweepers
])
def test_workload_launch_shapes(ci, variant, grid, block_steps, block, monkeypatch):
    for var in ("SOM_TRAIN_VARIANT", "SOM_TRAIN_GRID", "SOM_TRAIN_BLOCK_M", "SOM_TRAIN_LDS_ROWS",
                "SOM_TRAIN_SWEEPERS"):
        monkeypatch.delenv(var, raising=False)
    cfg = workloads.WORKLOADS[ci]
    m = som.Map(cfg.rows, cfg.cols, cfg.d, seed=0)
    plan = m.plan()
    say("workload", cfg.name, "plan", plan)
    m.close()
    assert (plan["variant"], plan["grid"], plan["block_steps"], plan["block"]) == \
        (variant, grid, block_steps, block)
