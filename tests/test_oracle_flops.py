"""The FP64 operation counts behind the roofline's algorithmic unit (counting build of the
oracle): a configuration evaluated on its own costs at least what the shared-level loops spend per
configuration, counts add over disjoint id sets, and the stored per-workload figures agree."""
import json
import os

import numpy as np

from oracle import oracle as O
from paper_2503_19050_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_single_configuration_counts_add_up():
    o = O.Oracle(W.workload("tiny"))
    rng = np.random.default_rng(8)
    a = rng.integers(0, o.n_configs, size=300, dtype=np.uint64)
    b = rng.integers(0, o.n_configs, size=200, dtype=np.uint64)
    assert o.count_flops_ids(a) + o.count_flops_ids(b) == o.count_flops_ids(np.concatenate([a, b]))
    assert o.count_flops_ids(a[:1]) > 0


def test_single_configuration_costs_at_least_the_shared_loops():
    """Per group: evaluating every configuration on its own performs every operation of the
    shared-level walk and repeats the shared levels, so its total is larger."""
    o = O.Oracle(W.workload("tiny"))
    for g in range(0, o.n_groups, max(1, o.n_groups // 12)):
        k = o.group_keys(g, 1)[0]
        ids = np.arange(k["base"], k["base"] + k["size"], dtype=np.uint64)
        shared, n = o.count_flops(g, g + 1)
        assert n == len(ids)
        assert o.count_flops_ids(ids) > shared


def test_stored_counts():
    with open(os.path.join(GOLDEN, "flops_per_config.json")) as f:
        d = json.load(f)["workloads"]
    for name in W.WORKLOADS:
        w = d[name]
        assert w["flops_per_config"] > w["flops_per_config_shared_levels"] > 0
    o = O.Oracle(W.workload("gpt1.3b-d8"))
    assert d["gpt1.3b-d8"]["configs_sampled"] == o.n_configs    # gpt1.3b-d8: every configuration
