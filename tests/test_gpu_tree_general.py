"""GPU parity of the general multicast kernel's variant for plans outside
the layered kernel's limits (rank counts that are not 4, 8, 16 or 32, routes
longer than 4 links, wide link-cost ratios): ReduceScatter and Allreduce
(Sec. 5.2), contiguous transfers (Sec. 5.1, Step 3) and time-aware greedy
orders (App. B.2), bit for bit against the oracle through the C ABI, with
unrouted pairs and many equal priorities. Needs an MI355X."""
from dataclasses import replace

import numpy as np
import pytest

from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

KINDS = [cf.ALLGATHER, cf.REDUCESCATTER, cf.ALLREDUCE]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2111_04867_amd import binding
    binding.lib()
    torch.cuda.set_device(0)
    yield


def ring(P, kind, k=2, cpr=1):
    """Bidirectional ring of P ranks: P % 4 != 0 keeps it off the layered kernel."""
    row_ptr, col, a, b = cf.csr_from_edges(P, cf.ring_edges(list(range(P)), 700, 46))
    return cf.Workload(f"ring{P}", P, P, row_ptr, col, a, b, None, kind, cpr, 65536,
                       cf.KSHORTEST, k=k)


def long_ring(P, kind):
    """Ring of P ranks with shortest routes only: routes up to P/2 links."""
    row_ptr, col, a, b = cf.csr_from_edges(P, cf.ring_edges(list(range(P)), 700, 46))
    return cf.Workload(f"longring{P}", P, P, row_ptr, col, a, b, None, kind, 1, 65536,
                       cf.SHORTEST_ONLY, k=1)


def skewed(P, kind):
    """Full mesh whose link costs differ by up to 40x: too many layers."""
    rng = np.random.default_rng(P)
    edges = [(u, v, int(rng.integers(100, 4000)), int(rng.integers(1, 60)))
             for u in range(P) for v in range(P) if u != v]
    row_ptr, col, a, b = cf.csr_from_edges(P, edges)
    return cf.Workload(f"skewed{P}", P, P, row_ptr, col, a, b, None, kind, 1, 65536,
                       cf.KSHORTEST, k=3)


def two_nodes(per, kind, cpr=1):
    """Two nodes of `per` fully connected ranks, IB between rank i of each."""
    w = cf.two_node_full(per, cf.ALLGATHER, chunks_per_rank=cpr, k=3)
    return replace(w, name=f"twonode{2 * per}", kind=kind, contiguity=0)


def check(w, n=256, seed=5):
    from paper_2111_04867_amd.binding import Plan
    plan, ref = Plan.from_workload(w), OraclePlan.from_workload(w)
    opts = plan.route_options()
    assert (opts == ref.route_options()).all()
    routes, prio = generate(seed, 0, n, opts, plan.prio_stride)
    rng = np.random.default_rng(seed)
    routes[rng.random(routes.shape) < 0.01] = 0xFF
    prio[rng.random(prio.shape) < 0.3] = 7
    print(f"[gpu] general multicast {w.name} kind={w.kind} contig={w.contiguity} "
          f"greedy={w.order}: {n} candidates", flush=True)
    mk, ok = plan.eval(routes, prio)
    rmk, rok = ref.eval(routes, prio)
    bad = np.nonzero((mk != rmk) | (ok != rok))[0]
    assert bad.size == 0, (f"{w.name}: {bad.size} mismatches, first at {bad[:5].tolist()}: "
                           f"gpu {mk[bad[:5]].tolist()} oracle {rmk[bad[:5]].tolist()}")
    assert ok.any()


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("P,cpr", [(3, 1), (6, 2), (10, 1)])
def test_static_orders(kind, P, cpr):
    check(ring(P, kind, cpr=cpr))


@pytest.mark.parametrize("kind", KINDS)
def test_long_routes(kind):
    check(long_ring(12, kind))


@pytest.mark.parametrize("kind", KINDS)
def test_wide_cost_ratio(kind):
    check(skewed(6, kind))


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("per,cpr", [(3, 1), (3, 2), (5, 1)])
def test_contiguity(kind, per, cpr):
    check(cf.with_contiguity(two_nodes(per, kind, cpr)))


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("make", [lambda k: ring(6, k, cpr=2), lambda k: long_ring(10, k),
                                  lambda k: skewed(5, k), lambda k: two_nodes(3, k)])
def test_greedy(kind, make):
    check(cf.with_greedy(make(kind)), n=128)


def test_explicit_greedy_and_contiguity():
    base = two_nodes(3, cf.ALLGATHER)
    owner = [0, 1, 4, 5, 2]
    posts = [[1, 3, 4], [0, 2, 3, 5], [0, 1], [5, 2], [0, 1, 2, 3, 4, 5]]
    w = cf.explicit_multicast(base, owner, posts)
    check(cf.with_greedy(w), n=128)
    check(cf.with_contiguity(w))


@pytest.mark.parametrize("kind", KINDS)
def test_reverse_greedy_general_shapes(kind):
    """Reverse path order on the general variant's shapes (long routes,
    wide cost ratios, two nodes)."""
    for make in (lambda k: long_ring(10, k), lambda k: skewed(5, k), lambda k: two_nodes(3, k),
                 lambda k: ring(6, k, cpr=2)):
        check(cf.with_reverse_greedy(make(kind)), n=96)


@pytest.mark.parametrize("option", ["static", "greedy", "rgreedy", "contig"])
@pytest.mark.parametrize("base", ["cubemesh8", "twonode6"])
def test_degenerate_explicit(base, option):
    """Postconditions that need no send (every chunk only at its owner): no
    sends, makespan 0, valid; then a single chunk with one destination."""
    from paper_2111_04867_amd.binding import Plan
    b = cf.cubemesh8_ag() if base == "cubemesh8" else two_nodes(3, cf.ALLGATHER)
    for owner, posts in (([0, 3, 5], [[0], [3], [5]]), ([2], [[b.P - 1]])):
        w = cf.explicit_multicast(b, owner, posts)
        if option == "greedy":
            w = cf.with_greedy(w)
        elif option == "rgreedy":
            w = cf.with_reverse_greedy(w)
        elif option == "contig":
            if w.node_of is None:
                continue
            w = cf.with_contiguity(w)
        plan, ref = Plan.from_workload(w), OraclePlan.from_workload(w)
        routes, prio = generate(3, 0, 64, plan.route_options(), plan.prio_stride)
        mk, ok = plan.eval(routes, prio)
        rmk, rok = ref.eval(routes, prio)
        assert (mk == rmk).all() and (ok == rok).all()
        if len(owner) == 3:
            assert (mk == 0).all() and ok.all()
        else:
            assert (mk > 0).all() and ok.all()


def quads(P, kind, k=3):
    """P ranks in fully connected groups of four, rank i linked to i + 4:
    a cube-mesh-like graph that 12 and 24 ranks keep within the layered
    kernel's limits (route words of 3 and 6 per chunk)."""
    edges = set()
    for g in range(0, P, 4):
        edges |= {(u, v) for u in range(g, g + 4) for v in range(g, g + 4) if u != v}
    for i in range(P):
        edges |= {(i, (i + 4) % P), ((i + 4) % P, i)}
    row_ptr, col, a, b = cf.csr_from_edges(P, [(u, v, 700, 46) for u, v in sorted(edges)])
    return cf.Workload(f"quads{P}", P, P, row_ptr, col, a, b, None, kind, 1, 65536,
                       cf.KSHORTEST, k=k)


@pytest.mark.parametrize("option", ["static", "greedy", "rgreedy"])
@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("P,k", [(12, 3), (24, 2)])
def test_twelve_and_twenty_four_ranks(P, k, kind, option):
    w = quads(P, kind, k)
    w = {"static": w, "greedy": cf.with_greedy(w), "rgreedy": cf.with_reverse_greedy(w)}[option]
    check(w, n=128)
