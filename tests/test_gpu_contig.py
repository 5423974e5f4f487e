"""GPU parity of contiguous transfers on links between nodes (Sec. 4.1;
Step 3 of Sec. 5.1; the is_together constraints of App. B.3), bit for bit
against the oracle, through the C ABI. Needs an MI355X."""
import numpy as np
import pytest

from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

NV_A, NV_B = 700, 46
IB_A, IB_B = 1700, 106


def say(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2111_04867_amd import binding
    binding.lib()
    torch.cuda.set_device(0)
    yield


def plans(w):
    from paper_2111_04867_amd.binding import Plan
    plan, ref = Plan.from_workload(w), OraclePlan.from_workload(w)
    assert ref.contiguity == w.contiguity
    opts = plan.route_options()
    assert (opts == ref.route_options()).all()
    return plan, ref, opts


def check(plan, ref, routes, prio, label):
    say(f"[gpu] {label}: {routes.shape[0]} candidates")
    mk, ok = plan.eval(routes, prio)
    rmk, rok = ref.eval_threads(routes, prio)
    bad = np.nonzero((mk != rmk) | (ok != rok))[0]
    assert bad.size == 0, (f"{label}: {bad.size} mismatches, first at {bad[:5].tolist()}: "
                           f"gpu {mk[bad[:5]].tolist()} oracle {rmk[bad[:5]].tolist()}")
    return mk, ok


@pytest.mark.parametrize("name", cf.CONTIG_ORDER)
def test_full_size_parity(name):
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed, 0, w.n_candidates, opts, plan.prio_stride)
    mk, ok = check(plan, ref, routes, prio, f"{name} full N={w.n_candidates}")
    assert ok.all()
    # contiguity changes the schedule of these workloads
    base = cf.named(name.replace("_contig", ""))
    bplan, _, _ = plans(base)
    bmk, _ = bplan.eval(routes[:2048], prio[:2048])
    assert (bmk != mk[:2048]).any()


@pytest.mark.parametrize("name", cf.CONTIG_ORDER)
@pytest.mark.parametrize("n", [1, 65, 257])
def test_ragged_batches(name, n):
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 100, 3, n, opts, plan.prio_stride)
    check(plan, ref, routes, prio, f"{name} n={n}")


@pytest.mark.parametrize("name", cf.CONTIG_ORDER)
@pytest.mark.parametrize("value", [0, 0xFFFFFFFF])
def test_equal_priorities(name, value):
    """Equal priorities leave the chunk id to break ties: many equal keys."""
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 7, 0, 96, opts, plan.prio_stride)
    prio[:] = value
    check(plan, ref, routes, prio, f"{name} prio={value:#x}")


@pytest.mark.parametrize("P_per,kind,cpr", [(2, cf.ALLGATHER, 1), (2, cf.ALLGATHER, 4),
                                            (4, cf.ALLGATHER, 2), (2, cf.ALLTOALL, 1),
                                            (4, cf.ALLTOALL, 2), (8, cf.ALLTOALL, 1)])
def test_small_two_node(P_per, kind, cpr):
    w = cf.two_node_full(P_per, kind, chunks_per_rank=cpr)
    plan, ref, opts = plans(w)
    routes, prio = generate(31 + P_per, 0, 500, opts, plan.prio_stride)
    check(plan, ref, routes, prio, f"{w.name} cpr={cpr}")


@pytest.mark.parametrize("P_per", [4, 5, 6])
def test_ring_nodes_alltoall(P_per):
    """Long paths: P_per = 5, 6 exceed the register-resident kernel's level
    and hop limits, so the LDS-record kernel is checked too."""
    w = cf.two_node_rings_a2a(P_per)
    plan, ref, opts = plans(w)
    routes, prio = generate(41 + P_per, 0, 300, opts, plan.prio_stride)
    check(plan, ref, routes, prio, f"{w.name}")


def explicit(V, edges, node_of, owner, posts, chunk_bytes):
    row_ptr, col, a, b = cf.csr_from_edges(V, edges)
    base = cf.Workload("custom", V, V, row_ptr, col, a, b, np.asarray(node_of, dtype=np.int32),
                       cf.ALLGATHER, 1, chunk_bytes, cf.KSHORTEST, k=4)
    w = cf.explicit_multicast(base, owner, posts)
    w.contiguity = 1
    return w


def cost(alpha, beta, nbytes):
    return alpha + (beta * nbytes + 999) // 1000


@pytest.mark.parametrize("m", [1, 2, 3, 8])
def test_closed_forms(m):
    """m chunks over IB then NVLink: one IB transfer, then one by one."""
    S = 65536
    # a fourth rank (inside the second node) keeps the rank count a multiple
    # of 4, which the layered multicast kernel needs
    edges = [(0, 1, IB_A, IB_B), (1, 0, IB_A, IB_B), (1, 2, NV_A, NV_B), (2, 1, NV_A, NV_B),
             (2, 3, NV_A, NV_B), (3, 2, NV_A, NV_B)]
    w = explicit(4, edges, [0, 1, 1, 1], [0] * m, [[2]] * m, S)
    plan, ref, opts = plans(w)
    routes = np.zeros((4, plan.route_stride), dtype=np.uint8)
    prio = np.arange(4 * plan.prio_stride, dtype=np.uint32).reshape(4, -1)
    mk, ok = check(plan, ref, routes, prio, f"chain m={m}")
    assert ok.all() and (mk == cost(IB_A, IB_B, m * S) + m * cost(NV_A, NV_B, S)).all()


def test_large_plan_on_the_general_kernel():
    """A multicast plan too large for the layered kernel (C*V > 1024) runs on
    the general kernel's variant, contiguous transfers included."""
    w = cf.uni_ring_ag(40, chunk_bytes=65536)
    w.node_of = np.array([r // 20 for r in range(40)], dtype=np.int32)
    w.contiguity = 1
    plan, ref, opts = plans(w)
    routes, prio = generate(1, 0, 24, opts, plan.prio_stride)
    prio[:, ::3] = 9
    mk, ok = check(plan, ref, routes, prio, "uniring40 contig")
    assert ok.all()
