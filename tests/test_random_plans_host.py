"""Host-side checks over the seeded random small plans of the GPU sweep:
the library and the oracle accept and refuse the same plans, build the same
route options, and plans with many remaining-cost levels are accepted."""
import numpy as np

from oracle import OraclePlan
from paper_2111_04867_amd import binding as B
from workloads import ALLTOALL, random_workload


def test_library_and_oracle_accept_the_same_plans():
    accepted = 0
    for seed in range(1000, 1400):
        w = random_workload(seed)
        try:
            ref = OraclePlan.from_workload(w)
        except Exception:
            ref = None
        try:
            plan = B.Plan.from_workload(w)
        except B.TacclError as e:
            assert ref is None, (seed, str(e))
            assert e.status == B.ERR_UNSUPPORTED, (seed, str(e))
            continue
        assert ref is not None, seed
        assert (plan.route_options() == ref.route_options()).all(), seed
        assert plan.prio_stride == ref.prio_stride, seed
        accepted += 1
    assert accepted >= 300


def test_many_remaining_cost_levels():
    """Random link costs give Alltoall plans hundreds of distinct remaining
    path costs; the general kernel walks any number of them."""
    most = 0
    for seed in range(1000, 1100):
        w = random_workload(seed)
        if w.kind != ALLTOALL:
            continue
        try:
            plan = B.Plan.from_workload(w)
        except B.TacclError:
            continue
        most = max(most, plan.info["num_levels"])
    assert most > 127


def test_library_and_oracle_agree_on_larger_plans():
    """The larger random plans: the same acceptance (apart from the switch
    port model's documented limit, which only the library has) and the same
    route options."""
    from workloads import random_workload_large
    accepted = 0
    for seed in range(300):
        w = random_workload_large(seed)
        try:
            ref = OraclePlan.from_workload(w)
        except Exception:
            ref = None
        try:
            plan = B.Plan.from_workload(w)
        except B.TacclError as e:
            assert ref is None or (w.switch_ports and "port" in str(e)), (seed, str(e))
            continue
        assert ref is not None, seed
        assert (plan.route_options() == ref.route_options()).all(), seed
        accepted += 1
    assert accepted >= 200
