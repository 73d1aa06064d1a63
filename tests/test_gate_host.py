"""Host-side tests of the model-level performance gate (Eq. 5): the gate's
decision rule, the benchmark plan, and that the PyTorch eager baseline block
computes the same function as the float64 block oracle (run on the CPU in
float32, so the baseline model is pinned without a GPU)."""
import math

import numpy as np
import pytest
import torch

import fusedsub_data as fd
import oracle
from paper_2609_30059_amd import gate
from paper_2609_30059_amd.block import PARAM_NAMES


def test_gate_rule_and_margin():
    assert gate.GAMMA == 1.03
    assert gate.perf_gate(1.0, 1.0)
    assert gate.perf_gate(0.5, 1.0)
    assert gate.perf_gate(103.0, 100.0)               # exactly at the 3 % margin
    assert not gate.perf_gate(103.01, 100.0)
    assert not gate.perf_gate(2.0, 1.0)
    assert gate.perf_gate(1.2, 1.0, gamma=1.25)
    for bad in (0.0, -1.0, float("nan"), float("inf")):
        with pytest.raises(ValueError):
            gate.perf_gate(bad, 1.0)
        with pytest.raises(ValueError):
            gate.perf_gate(1.0, bad)


def test_bench_plan_fills_budgets():
    assert gate.bench_plan(1.0) == (25, 100)           # 25 ms warm-up, 100 ms of reps
    assert gate.bench_plan(0.4) == (62, 250)
    assert gate.bench_plan(500.0) == (1, 1)            # never zero calls
    with pytest.raises(ValueError):
        gate.bench_plan(0.0)


def test_report_uses_the_baseline_model():
    res = {"fused": {"median_ms": 2.0}, "eager_subkernels": {"median_ms": 3.0},
           "eager": {"median_ms": 4.0}}
    r = gate.report(res)
    assert r["pass"] and math.isclose(r["speedup"], 1.5)
    assert math.isclose(r["speedup_vs_eager"], 2.0)
    r = gate.report({"fused": {"median_ms": 3.2}, "eager_subkernels": {"median_ms": 3.0}})
    assert not r["pass"]
    assert "graph_replay_speedup" not in r
    # the graph replay is context: it never enters the verdict
    r = gate.report({"fused": {"median_ms": 2.0}, "fused_graph": {"median_ms": 1.6},
                     "eager_subkernels": {"median_ms": 2.1}})
    assert r["pass"] and math.isclose(r["speedup"], 1.05)
    assert math.isclose(r["graph_replay_speedup"], 1.25)


@pytest.mark.parametrize("seed", [0, 1])
def test_eager_baseline_block_matches_oracle(seed):
    d = fd.block_inputs(seed, batch=2, seq=16, hidden=64, heads=4, mlp=256)
    p32 = {k: torch.from_numpy(d[k].f64().astype(np.float32)) for k in PARAM_NAMES}
    x32 = torch.from_numpy(d["x"].f64().astype(np.float32))
    got = gate.eager_block(p32, x32, d["heads"], d["eps"]).double().numpy().reshape(2, 16, 64)
    ref = oracle.block_forward(d["x"].f64(), {k: d[k].f64() for k in PARAM_NAMES}, d["heads"],
                               d["eps"])["out"]
    np.testing.assert_allclose(got, ref, rtol=1e-4, atol=1e-4)
