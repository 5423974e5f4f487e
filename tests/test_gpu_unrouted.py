"""GPU parity of unrouted pairs whose choice lies just past the option count.

A route choice at or beyond its entry's option count leaves the pair
unrouted (the candidate may then fail its postcondition). The kernels
decode choices below 8 and from 8 up on different paths, so every kernel
family is fed choices drawn from [options, 8), exactly options, and the
values 8 and 255, and compared with the oracle bit for bit. Needs an MI355X.
"""
import numpy as np
import pytest

from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2111_04867_amd import binding
    binding.lib()
    torch.cuda.set_device(0)
    yield


# (label, workload, candidates): one per kernel family
CASES = [
    ("layered ring4", lambda: cf.named("ring4_ag"), 200),
    ("layered cubemesh8", lambda: cf.named("cubemesh8_ag"), 200),
    ("layered twonode16", lambda: cf.named("twonode16_ag"), 300),
    ("layered twonode16 rs", lambda: cf.named("twonode16_rs"), 200),
    ("layered cubemesh8 ar", lambda: cf.named("cubemesh8_ar"), 200),
    ("layered contig", lambda: cf.named("twonode16_ag_contig"), 200),
    ("general ring6", lambda: cf.uni_ring_ag(6), 200),
    ("general full5", lambda: cf.full_ag(5, k=3), 200),
    ("general rgreedy ring6", lambda: cf.with_reverse_greedy(cf.uni_ring_ag(6)), 200),
    ("tree rgreedy twonode16", lambda: cf.named("twonode16_ag_rgreedy"), 100),
    ("tree greedy", lambda: cf.named("cubemesh8_ag_greedy"), 200),
    ("fast a2a switch16", lambda: cf.named("switch16_a2a"), 200),
    ("fast a2a fournode64", lambda: cf.named("fournode64_a2a"), 24),
    ("fast a2a contig", lambda: cf.named("fournode64_a2a_contig"), 16),
    ("path greedy switch16", lambda: cf.named("switch16_a2a_greedy"), 100),
    ("block greedy fournode64", lambda: cf.named("fournode64_a2a_greedy"), 6),
    ("ports switch16", lambda: cf.named("switch16_a2a_ports"), 100),
    ("relay a2a full5", lambda: cf.full_a2a(5), 200),
]


def near_miss_routes(routes, opts, seed):
    """Per candidate, a few used entries get a choice from [options, 8) or
    exactly options, one candidate gets exactly options on every entry, one
    gets 8 (the first value the one-hot decoding of the multicast kernels
    drops; options where an entry has more) and one gets 255 on half of
    them."""
    rng = np.random.default_rng(seed)
    used = np.nonzero(opts > 0)[0]
    n = routes.shape[0]
    for i in range(3, n):
        k = int(rng.integers(0, 5))
        if k == 0:
            continue
        cols = rng.choice(used, size=min(k, used.size), replace=False)
        for e in cols:
            o = int(opts[e])
            routes[i, e] = o if (o >= 8 or rng.random() < 0.3) else int(rng.integers(o, 8))
    routes[0, used] = opts[used]
    if n > 1:
        routes[1, used] = np.maximum(opts[used], 8)
    if n > 2:
        routes[2, used[: max(1, used.size // 2)]] = 255
    return routes


@pytest.mark.parametrize("label,make,n", CASES, ids=[c[0] for c in CASES])
def test_choices_just_past_the_options(label, make, n):
    from paper_2111_04867_amd.binding import Plan
    w = make()
    plan, ref = Plan.from_workload(w), OraclePlan.from_workload(w)
    opts = plan.route_options()
    assert (opts == ref.route_options()).all()
    routes, prio = generate(w.seed + 31, 0, n, opts, plan.prio_stride)
    routes = near_miss_routes(routes, opts, 7)
    print(f"[gpu] unrouted near miss {label}: {n} candidates", flush=True)
    mk, ok = plan.eval(routes, prio)
    rmk, rok = ref.eval_threads(routes, prio)
    bad = np.nonzero((mk != rmk) | (ok != rok))[0]
    assert bad.size == 0, (f"{label}: {bad.size} mismatches, first at {bad[:5].tolist()}: "
                           f"gpu {mk[bad[:5]].tolist()} {ok[bad[:5]].tolist()} "
                           f"oracle {rmk[bad[:5]].tolist()} {rok[bad[:5]].tolist()}")
    assert ok[0] == 0 and ok[1] == 0  # nothing routed
    assert (mk != 0xFFFFFFFF).all()


@pytest.mark.parametrize("name", ["switch16_a2a", "fournode64_a2a", "cubemesh8_ag", "twonode16_ar"])
def test_connections_just_past_the_options(name):
    from paper_2111_04867_amd.binding import Plan
    w = cf.named(name)
    plan, ref = Plan.from_workload(w), OraclePlan.from_workload(w)
    opts = plan.route_options()
    routes, _ = generate(w.seed + 33, 0, 120, opts, plan.prio_stride)
    routes = near_miss_routes(routes, opts, 9)
    print(f"[gpu] connections near miss {name}", flush=True)
    got = plan.connections(routes)
    want = ref.connections(routes)
    assert (got == want).all()
