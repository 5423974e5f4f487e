"""GPU parity of the switch-port model for Alltoall (App. B.3 switch
constraints; App. B.2 switch send and receive orders), bit for bit against
the oracle, through the C ABI. Needs an MI355X."""
import numpy as np
import pytest

from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


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
    assert ref.switch_ports == w.switch_ports == 1
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


def star(P, relays=True, cpr=1, chunk_bytes=256 * 1024):
    """P ranks on one switch (vertex P): direct sends, or direct and through
    one relay rank."""
    row_ptr, col, a, b = cf.csr_from_edges(P + 1, cf.switch_edges(range(P), P, 700, 8))
    mode = cf.RELAY1 if relays else cf.KSHORTEST
    return cf.Workload(f"star{P}", P + 1, P, row_ptr, col, a, b, None, cf.ALLTOALL, cpr,
                       chunk_bytes, mode, k=1, switch_ports=1)


def two_switches(per=3):
    """Two switch nodes of `per` ranks each; rank i of one node has an IB
    link to rank i of the other."""
    P = 2 * per
    edges = cf.switch_edges(range(per), P, 700, 8) + cf.switch_edges(range(per, P), P + 1, 700, 8)
    for i in range(per):
        edges += [(i, per + i, 1700, 106), (per + i, i, 1700, 106)]
    row_ptr, col, a, b = cf.csr_from_edges(P + 2, edges)
    node_of = np.array([0] * per + [1] * per + [0, 1], dtype=np.int32)
    relay = np.array([1] * P + [0, 0], dtype=np.uint8)
    return cf.Workload(f"twoswitch{per}", P + 2, P, row_ptr, col, a, b, node_of, cf.ALLTOALL,
                       1, 65536, cf.HIER_RELAY, max_cross=1, relay=relay, switch_ports=1)


@pytest.mark.parametrize("name", cf.PORTS_ORDER)
def test_full_size_parity(name):
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed, 0, w.n_candidates, opts, plan.prio_stride)
    mk, ok = check(plan, ref, routes, prio, f"{name} full N={w.n_candidates}")
    assert ok.all()
    # the port model changes these schedules
    base = cf.named(name.replace("_ports", ""))
    from paper_2111_04867_amd.binding import Plan
    bmk, _ = Plan.from_workload(base).eval(routes[:1024], prio[:1024])
    assert (bmk != mk[:1024]).any()


@pytest.mark.parametrize("name", cf.PORTS_ORDER)
@pytest.mark.parametrize("n", [1, 65, 257])
def test_ragged_batches(name, n):
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 100, 3, n, opts, plan.prio_stride)
    check(plan, ref, routes, prio, f"{name} n={n}")


@pytest.mark.parametrize("name", cf.PORTS_ORDER)
@pytest.mark.parametrize("value", [0, 0xFFFFFFFF])
def test_equal_priorities(name, value):
    """Equal priorities leave the chunk id to break ties on both ports."""
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 7, 0, 64, opts, plan.prio_stride)
    prio[:] = value
    check(plan, ref, routes, prio, f"{name} prio={value:#x}")


def test_two_ranks_closed_form():
    w = star(2, relays=False)
    plan, ref, opts = plans(w)
    routes, prio = generate(1, 0, 8, opts, plan.prio_stride)
    mk, ok = check(plan, ref, routes, prio, "star2")
    assert ok.all() and (mk == 700 + (8 * 256 * 1024 + 999) // 1000).all()


@pytest.mark.parametrize("P,relays,cpr", [(3, True, 1), (4, True, 2), (5, False, 3),
                                          (6, True, 1), (8, True, 4)])
def test_stars(P, relays, cpr):
    """Relayed routes put a rank's second switched send at a later level;
    several chunks per pair load one port with many sends of one level."""
    w = star(P, relays, cpr)
    plan, ref, opts = plans(w)
    routes, prio = generate(50 + P, 0, 400, opts, plan.prio_stride)
    check(plan, ref, routes, prio, f"{w.name} cpr={cpr}")


@pytest.mark.parametrize("per", [2, 3, 4])
def test_two_switches(per):
    """Switched sends inside a node, store-and-forward IB links between."""
    w = two_switches(per)
    plan, ref, opts = plans(w)
    routes, prio = generate(60 + per, 0, 400, opts, plan.prio_stride)
    check(plan, ref, routes, prio, w.name)


@pytest.mark.parametrize("P,cpr,relays", [(48, 2, True), (36, 3, False)])
def test_large_levels(P, cpr, relays):
    """Levels of thousands of switched sends in 1024-thread blocks: up to
    four positions per thread are kept in registers through the port passes
    (36 ranks, 3 chunks per pair: 3780 sends in one level), more are looped
    over (48 ranks with relays: up to 4512 sends in the last level)."""
    w = star(P, relays=relays, cpr=cpr, chunk_bytes=64 * 1024)
    plan, ref, opts = plans(w)
    routes, prio = generate(70 + P, 0, 24, opts, plan.prio_stride)
    check(plan, ref, routes, prio, f"{w.name} cpr={cpr}")
