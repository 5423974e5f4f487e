"""GPU parity at the size limits of the kernels: the largest plans that
still fit one block's LDS run bit-exact against the oracle, the next size up
is refused with UNSUPPORTED (never approximated), and Alltoall plans beyond
the register-resident kernel's chunk limit take the LDS-record kernel.
Needs an MI355X."""
from dataclasses import replace

import numpy as np
import pytest

from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

LDS_PER_BLOCK = 160 * 1024  # gfx950


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2111_04867_amd import binding
    binding.lib()
    torch.cuda.set_device(0)
    yield


def full_mesh_a2a(P, cpr=1):
    """P fully connected ranks, Alltoall on the direct links only."""
    edges = [(u, v, 700, 8) for u in range(P) for v in range(P) if u != v]
    row_ptr, col, a, b = cf.csr_from_edges(P, edges)
    return cf.Workload(f"mesh{P}_a2a", P, P, row_ptr, col, a, b, None, cf.ALLTOALL, cpr, 4096,
                       cf.SHORTEST_ONLY)


def check(w, n, seed):
    from paper_2111_04867_amd.binding import Plan
    plan, ref = Plan.from_workload(w), OraclePlan.from_workload(w)
    opts = plan.route_options()
    assert (opts == ref.route_options()).all()
    routes, prio = generate(seed, 0, n, opts, plan.prio_stride)
    prio[::2, ::3] = 1
    print(f"[gpu] limits {w.name}: {n} candidates, {plan.info['lds_bytes']} B of LDS", flush=True)
    mk, ok = plan.eval(routes, prio)
    rmk, rok = ref.eval_threads(routes, prio)
    assert (mk == rmk).all() and (ok == rok).all()
    return plan


def refused(w):
    from paper_2111_04867_amd.binding import ERR_UNSUPPORTED, Plan, TacclError
    plan = Plan.from_workload(w)
    assert plan.info["lds_bytes"] > LDS_PER_BLOCK
    routes, prio = generate(1, 0, 2, plan.route_options(), plan.prio_stride)
    with pytest.raises(TacclError) as e:
        plan.eval(routes, prio)
    assert e.value.status == ERR_UNSUPPORTED


@pytest.mark.parametrize("kind", [cf.ALLGATHER, cf.REDUCESCATTER, cf.ALLREDUCE])
def test_multicast_largest_block(kind):
    """64 ranks in a ring (one-way for Allgather), chunks per rank raised
    until a block's LDS is exceeded: the largest plan that fits (8192 send
    slots for Allgather on the general kernel) matches the oracle, the next
    one is refused."""
    from paper_2111_04867_amd.binding import Plan
    if kind == cf.ALLGATHER:
        base = cf.uni_ring_ag(64, chunk_bytes=65536)
    else:  # reductions need the reverse links
        row_ptr, col, a, b = cf.csr_from_edges(64, cf.ring_edges(list(range(64)), 700, 46))
        base = cf.Workload("ring64", 64, 64, row_ptr, col, a, b, None, kind, 1, 65536,
                           cf.KSHORTEST, k=1)
    sizes = [Plan.from_workload(replace(base, chunks_per_rank=c)).info["lds_bytes"]
             for c in (1, 2, 3, 4)]
    fits = [c for c, b in zip((1, 2, 3, 4), sizes) if b <= LDS_PER_BLOCK]
    assert fits and max(fits) < 4, sizes
    check(replace(base, chunks_per_rank=max(fits)), 24, 3)
    refused(replace(base, chunks_per_rank=max(fits) + 1))


def test_alltoall_past_the_register_kernel():
    """4900 chunks (more than the register-resident kernel's 4096): the
    LDS-record kernel."""
    plan = check(full_mesh_a2a(70), 32, 4)
    assert plan.info["num_chunks"] > 4096


def test_alltoall_too_large_for_a_block():
    refused(full_mesh_a2a(64, cpr=2))


def test_alltoall_many_remaining_cost_levels():
    """Random link costs: hundreds of distinct remaining path costs."""
    from workloads import random_workload
    for seed in range(1000, 1100):
        w = random_workload(seed)
        if w.kind != cf.ALLTOALL or w.order or w.switch_ports:
            continue
        try:
            ref = OraclePlan.from_workload(w)
        except Exception:
            continue
        from paper_2111_04867_amd.binding import Plan
        if Plan.from_workload(w).info["num_levels"] > 127:
            del ref
            check(w, 64, seed)
            return
    pytest.fail("no plan with more than 127 levels among the seeds")
