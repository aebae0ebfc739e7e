"""CPU tests of the stage performance model (paper: System Design, Hybrid-
Strategy Instance Scheduling) against the paper's own numbers: its table of
per-stage times and the throughputs it measured for two static allocations on
8 GPUs (fixture tests/golden/stage_times_wan22.json, citations inside)."""
import json
import math
import os

import pytest

from paper_2605_25550_amd import stage_model as SM

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "stage_times_wan22.json")))


def alloc(r):
    e, t, d = (int(v) for v in r.split(":"))
    return {"E": e, "T": t, "D": d}


@pytest.mark.parametrize("workload", ["4-steps", "1-step"])
def test_model_reproduces_measured_throughput(workload):
    """QPS = min(g/T) with the table's stage times gives the measured QPM of
    both static allocations to the paper's rounding (0.1 QPM)."""
    times = GOLDEN["stage_seconds"][workload]
    for r, measured in GOLDEN["measured_qpm"][workload].items():
        model = SM.per_minute(SM.qps(alloc(r), times))
        assert abs(model - measured) <= 0.05 + 1e-9, (workload, r, model, measured)


@pytest.mark.parametrize("workload", ["4-steps", "1-step"])
def test_model_bottlenecks_match_paper(workload):
    times = GOLDEN["stage_seconds"][workload]
    for r, stage in GOLDEN["reported_bottleneck"][workload].items():
        assert SM.bottleneck(alloc(r), times) == stage, (workload, r)


def test_best_static_configuration_matches_paper():
    for workload, best in GOLDEN["reported_best_static"].items():
        times = GOLDEN["stage_seconds"][workload]
        cands = [alloc(r) for r in GOLDEN["measured_qpm"][workload]]
        a, _ = SM.best_allocation(GOLDEN["gpus"], times, candidates=cands)
        assert SM.ratios(a) == best, workload


def test_exhaustive_search_4_steps_is_1_6_1():
    """Over every allocation of 8 GPUs the DiT-bound 4-step workload is best
    served by 1:6:1, the allocation the paper's scheduler settles on."""
    a, q = SM.best_allocation(8, GOLDEN["stage_seconds"]["4-steps"])
    assert SM.ratios(a) == "1:6:1"
    assert math.isclose(q, 6 / 74.1)


def test_exhaustive_search_balances_rates():
    """The optimum's service rates are within one GPU's worth of each other:
    moving one GPU from any stage to the bottleneck cannot raise QPS."""
    for times in GOLDEN["stage_seconds"].values():
        a, q = SM.best_allocation(8, times)
        for src in SM.STAGES:
            for dst in SM.STAGES:
                if src == dst or a[src] <= 1:
                    continue
                b = dict(a)
                b[src] -= 1
                b[dst] += 1
                assert SM.qps(b, times) <= q + 1e-15


def test_stage_time_equation_and_memory_constraint():
    # 2 GB of activations at 1000 FLOPs/byte on 500 TFLOP/s, two 1 GB transfers at 10 and 50 GB/s
    c = SM.StageCost(act_bytes=2e9, intensity=1e3, perf=5e14, comm=((1e9, 1e10), (1e9, 5e10)), model_bytes=28e9)
    assert math.isclose(c.time(), 2e12 / 5e14 + 0.1 + 0.02)
    assert math.isclose(SM.StageCost(2e9, 1e3, 5e14).time(), 4e-3)   # no transfers: compute only
    assert c.fits(40e9) and not c.fits(30e9)                          # S_M + S_A < C
    assert not SM.StageCost(2e9, 1e3, 5e14, model_bytes=28e9).fits(30e9)


def test_transformer_time_calibration_and_sweep():
    t = SM.transformer_time(50, 0.0043, act_in=(4e6, 2e10), act_out=(4e6, 2e10))
    assert math.isclose(t, 50 * 0.0043 + 4e-4)
    res = SM.sweep(8, GOLDEN["stage_seconds"])
    assert res["4-steps"][0] == "1:6:1" and res["4-steps"][2] == "T"
    assert res["50-steps"][2] == "T"
    assert SM.qps({"E": 1, "T": 0, "D": 1}, GOLDEN["stage_seconds"]["1-step"]) == 0.0
