"""The planner's choice (wino_plan_r, host-only) against measured per-layer
times: profiles/planner_table.txt holds, for the single 3x3 layers, the ResNet
stage layer and the VGG-16 layers at N=1 and N=32, the time of one
wino_conv2d call with every algorithm the library accepts (bench.py
--planner-table on one MI355X).  AUTO must pick an algorithm within 10% of the
fastest measured one on every layer (closer ones are run-to-run noise)."""
import os

import pytest

import bench
from paper_1903_01521_amd import binding as B

ROWS = bench.read_planner_table()


def test_table_covers_the_planner_layers():
    assert sorted(r["shape"] for r in ROWS) == sorted(bench.planner_layers())


@pytest.mark.parametrize("row", ROWS, ids=lambda r: "n{}_c{}_{}x{}_k{}_p{}_m{}".format(*r["shape"]))
def test_auto_choice_is_near_the_fastest(row):
    N, C, H, W, K, pad, m = row["shape"]
    st, algo, nsl = B.wino_plan_r(N, C, H, W, K, pad, m, 3, 0)
    assert st == B.WINO_OK
    pick = bench.planner_candidate_name(algo, nsl)
    times = row["times"]
    assert pick in times, (pick, times)
    best = min(times.values())
    assert times[pick] <= 1.10 * best, (pick, times)
