"""GPU parity on many seeded random small plans (random topologies with
optional switch vertex and two nodes, every collective kind, every route
mode, static or greedy orders, contiguity, switch ports), each evaluated on
48 candidates with some unrouted pairs and many equal priorities, bit for
bit against the oracle through the C ABI. Plans the route search refuses on
both sides are skipped (the host test checks that both sides agree on
which), and so are plans outside the documented limits of the kernel an
option needs (Alltoall greedy orders hold at most 1024 send slots); the test
counts both. Needs an MI355X."""
import numpy as np
import pytest

from oracle import OraclePlan
from workloads import generate, random_workload

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SEEDS = range(1000, 1400)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2111_04867_amd import binding
    binding.lib()
    torch.cuda.set_device(0)
    yield


@pytest.mark.parametrize("block", range(4))
def test_random_plans(block):
    from paper_2111_04867_amd.binding import ERR_UNSUPPORTED, Plan, TacclError
    checked, refused = 0, 0
    for seed in SEEDS[block::4]:
        w = random_workload(seed)
        try:
            ref = OraclePlan.from_workload(w)
        except Exception:
            continue  # a relay route through one link twice: refused on both sides
        plan = Plan.from_workload(w)
        opts = plan.route_options()
        assert (opts == ref.route_options()).all(), seed
        routes, prio = generate(seed, 0, 48, opts, plan.prio_stride)
        rng = np.random.default_rng(seed)
        routes[rng.random(routes.shape) < 0.02] = 0xFF
        prio[rng.random(prio.shape) < 0.3] = 5
        print(f"[gpu] random plan {seed}: kind={w.kind} P={w.P} V={w.V} mode={w.route_mode} "
              f"k={w.k} cpr={w.chunks_per_rank} contig={w.contiguity} greedy={w.order} "
              f"ports={w.switch_ports}", flush=True)
        try:
            mk, ok = plan.eval(routes, prio)
        except TacclError as e:
            assert e.status == ERR_UNSUPPORTED, (seed, str(e))
            print(f"[gpu]   refused: {e}", flush=True)
            refused += 1
            continue
        rmk, rok = ref.eval(routes, prio)
        bad = np.nonzero((mk != rmk) | (ok != rok))[0]
        assert bad.size == 0, (f"random plan {seed}: {bad.size} mismatches, first at "
                               f"{bad[:5].tolist()}: gpu {mk[bad[:5]].tolist()} "
                               f"{ok[bad[:5]].tolist()} oracle {rmk[bad[:5]].tolist()} "
                               f"{rok[bad[:5]].tolist()}")
        checked += 1
    print(f"[gpu] block {block}: {checked} plans checked, {refused} refused", flush=True)
    assert checked >= 75


def test_random_larger_plans():
    """300 larger seeded plans (up to 24 ranks, two switches, three nodes,
    six options per pair, three chunks per rank), 32 candidates each. Plans
    whose switch links would be both send and receive ports are refused at
    plan time (a documented limit of the port model) and skipped."""
    from paper_2111_04867_amd.binding import ERR_UNSUPPORTED, Plan, TacclError
    from workloads import random_workload_large
    checked = 0
    for seed in range(300):
        w = random_workload_large(seed)
        try:
            ref = OraclePlan.from_workload(w)
        except Exception:
            continue
        try:
            plan = Plan.from_workload(w)
        except TacclError as e:
            assert e.status == ERR_UNSUPPORTED and w.switch_ports, (seed, str(e))
            continue
        routes, prio = generate(seed, 0, 32, plan.route_options(), plan.prio_stride)
        rng = np.random.default_rng(seed)
        routes[rng.random(routes.shape) < 0.02] = 0xFF
        prio[rng.random(prio.shape) < 0.3] = 5
        print(f"[gpu] larger random plan {seed}: kind={w.kind} P={w.P} V={w.V} "
              f"mode={w.route_mode} k={w.k} cpr={w.chunks_per_rank} contig={w.contiguity} "
              f"greedy={w.order} ports={w.switch_ports}", flush=True)
        mk, ok = plan.eval(routes, prio)
        rmk, rok = ref.eval(routes, prio)
        bad = np.nonzero((mk != rmk) | (ok != rok))[0]
        assert bad.size == 0, (f"larger random plan {seed}: {bad.size} mismatches, first at "
                               f"{bad[:5].tolist()}: gpu {mk[bad[:5]].tolist()} "
                               f"oracle {rmk[bad[:5]].tolist()}")
        checked += 1
    assert checked >= 200
