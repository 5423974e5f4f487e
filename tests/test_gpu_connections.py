"""GPU parity of the switch-hyperedge connection count (the is_util count of
App. B.3 that the uc-max / uc-min policies of Sec. 5.1 weigh), bit for bit
against the oracle, through the C ABI. Needs an MI355X."""
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


def star(P, kind, relays=True, cpr=1):
    row_ptr, col, a, b = cf.csr_from_edges(P + 1, cf.switch_edges(range(P), P, 700, 8))
    mode = cf.RELAY1 if relays else cf.KSHORTEST
    return cf.Workload(f"star{P}", P + 1, P, row_ptr, col, a, b, None, kind, cpr, 65536, mode,
                       k=1)


def two_switches(per, kind):
    P = 2 * per
    edges = cf.switch_edges(range(per), P, 700, 8) + cf.switch_edges(range(per, P), P + 1, 700, 8)
    for i in range(per):
        edges += [(i, per + i, 1700, 106), (per + i, i, 1700, 106)]
    row_ptr, col, a, b = cf.csr_from_edges(P + 2, edges)
    node_of = np.array([0] * per + [1] * per + [0, 1], dtype=np.int32)
    relay = np.array([1] * P + [0, 0], dtype=np.uint8)
    return cf.Workload(f"twoswitch{per}", P + 2, P, row_ptr, col, a, b, node_of, kind, 1, 65536,
                       cf.HIER_RELAY, k=2, max_cross=1, relay=relay)


def hybrid(P, kind):
    """P ranks on one switch plus a bidirectional ring of direct links: some
    routes use the switch and some do not, so the count varies."""
    edges = cf.switch_edges(range(P), P, 700, 8) + cf.ring_edges(range(P), 1500, 8)
    row_ptr, col, a, b = cf.csr_from_edges(P + 1, edges)
    return cf.Workload(f"hybrid{P}", P + 1, P, row_ptr, col, a, b, None, kind, 1, 65536,
                       cf.KSHORTEST, k=4)


def check(w, n, seed, unrouted=0.0):
    from paper_2111_04867_amd.binding import Plan
    plan, ref = Plan.from_workload(w), OraclePlan.from_workload(w)
    opts = plan.route_options()
    assert (opts == ref.route_options()).all()
    routes, _ = generate(seed, 0, n, opts, plan.prio_stride)
    if unrouted:
        rng = np.random.default_rng(seed)
        routes[rng.random(routes.shape) < unrouted] = 0xFF
    say(f"[gpu] connections {w.name} kind={w.kind}: {n} candidates, seed {seed}")
    got = plan.connections(routes)
    want = ref.connections(routes)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, (f"{w.name}: {bad.size} mismatches, first at {bad[:5].tolist()}: "
                           f"gpu {got[bad[:5]].tolist()} oracle {want[bad[:5]].tolist()}")
    return got


@pytest.mark.parametrize("name", ["switch16_a2a", "fournode64_a2a", "twonode16_ag",
                                  "cubemesh8_ag"])
def test_named_workloads(name):
    w = cf.named(name)
    n = min(w.n_candidates, 512)
    got = check(w, n, w.seed)
    if name == "fournode64_a2a":
        assert (got == 4 * 16 * 15).all()  # every on-node pair goes direct via the switch
    if name in ("twonode16_ag", "cubemesh8_ag"):
        assert (got == 0).all()  # no switch vertex


@pytest.mark.parametrize("kind", [cf.ALLTOALL, cf.ALLGATHER, cf.REDUCESCATTER, cf.ALLREDUCE])
@pytest.mark.parametrize("P,cpr", [(3, 1), (5, 2), (16, 1), (33, 1)])
def test_star(kind, P, cpr):
    check(star(P, kind, cpr=cpr), 300, 100 + P, unrouted=0.05)


@pytest.mark.parametrize("kind", [cf.ALLTOALL, cf.ALLGATHER, cf.REDUCESCATTER, cf.ALLREDUCE])
@pytest.mark.parametrize("P", [5, 8, 24])
def test_switch_plus_ring(kind, P):
    got = check(hybrid(P, kind), 400, 11 + P, unrouted=0.02)
    assert len(set(got.tolist())) > 1


@pytest.mark.parametrize("kind", [cf.ALLTOALL, cf.ALLGATHER, cf.ALLREDUCE])
def test_two_switch_nodes(kind):
    check(two_switches(4, kind), 400, 7)


def test_batch_split_and_empty():
    from paper_2111_04867_amd.binding import Plan
    w = cf.switch16_a2a(n_candidates=1000)
    plan = Plan.from_workload(w)
    routes, _ = generate(w.seed, 0, 1000, plan.route_options(), plan.prio_stride)
    whole = plan.connections(routes)
    parts = np.concatenate([plan.connections(routes[:333]), plan.connections(routes[333:])])
    assert np.array_equal(whole, parts)
    d_r = torch.empty((0, plan.route_stride), dtype=torch.uint8, device="cuda")
    d_c = torch.empty(1, dtype=torch.int32, device="cuda")
    plan.connections_tensors(d_r, d_c)  # n == 0 is a no-op
    torch.cuda.synchronize()
