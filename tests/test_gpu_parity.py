"""GPU parity: the HIP evaluator against the CPU oracle, bit for bit.

Every test calls the library through its C ABI (via the ctypes binding) on
seeded synthetic inputs and compares makespan and valid flag of every
candidate with the oracle's. Needs an MI355X.
"""
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
    binding.lib()  # fails loudly if the HIP library is missing
    torch.cuda.set_device(0)
    yield


def plans(w):
    from paper_2111_04867_amd.binding import Plan
    plan, ref = Plan.from_workload(w), OraclePlan.from_workload(w)
    opts = plan.route_options()
    assert (opts == ref.route_options()).all()
    return plan, ref, opts


def check(plan, ref, routes, prio, label):
    say(f"[gpu] {label}: {routes.shape[0]} candidates")
    mk, ok = plan.eval(routes, prio)
    rmk, rok = ref.eval_threads(routes, prio)
    bad = np.nonzero((mk != rmk) | (ok != rok))[0]
    assert bad.size == 0, (f"{label}: {bad.size} mismatches, first at {bad[:5].tolist()}: "
                           f"gpu {mk[bad[:5]].tolist()} {ok[bad[:5]].tolist()} "
                           f"oracle {rmk[bad[:5]].tolist()} {rok[bad[:5]].tolist()}")
    return mk, ok


# ----------------------------------------------------------------------------
# the five workloads at full size, in the launch configuration the benchmark
# times (one call over all candidates)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("name", cf.ORDER)
def test_full_size_parity(name):
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed, 0, w.n_candidates, opts, plan.prio_stride)
    mk, ok = check(plan, ref, routes, prio, f"{name} full N={w.n_candidates}")
    assert ok.all()
    from paper_2111_04867_amd.binding import count_faults
    assert count_faults(mk) == 0
    if name == "ring4_ag":
        assert (mk == 97870).all()


@pytest.mark.parametrize("name", cf.ORDER)
@pytest.mark.parametrize("n", [1, 2, 63, 65, 257])
def test_ragged_batches(name, n):
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 100, 5, n, opts, plan.prio_stride)
    check(plan, ref, routes, prio, f"{name} n={n}")


def test_empty_batch_is_a_noop():
    w = cf.ring4_ag()
    plan, _, _ = plans(w)
    mk = torch.full((4,), 7, dtype=torch.int32, device="cuda")
    ok = torch.full((4,), 7, dtype=torch.uint8, device="cuda")
    r = torch.zeros((0, plan.route_stride), dtype=torch.uint8, device="cuda")
    p = torch.zeros((0, plan.prio_stride), dtype=torch.int32, device="cuda")
    plan.eval_tensors(r, p, mk, ok)
    torch.cuda.synchronize()
    assert (mk.cpu() == 7).all() and (ok.cpu() == 7).all()


# ----------------------------------------------------------------------------
# degenerate and adversarial inputs
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("name", cf.ORDER)
def test_unrouted_pairs(name):
    """Choices at or beyond a pair's option count leave it unrouted."""
    w = cf.named(name)
    plan, ref, opts = plans(w)
    n = 300
    routes, prio = generate(w.seed + 7, 0, n, opts, plan.prio_stride)
    rng = np.random.default_rng(5)
    used = np.nonzero(opts > 0)[0]
    for i in range(n):
        k = rng.integers(0, 4)
        if k:
            cols = rng.choice(used, size=min(k, used.size), replace=False)
            routes[i, cols] = rng.choice([255, 254, 200, 17])
    routes[0, used] = 255  # nothing routed at all
    mk, ok = check(plan, ref, routes, prio, f"{name} unrouted")
    assert mk[0] == 0 and ok[0] == 0


@pytest.mark.parametrize("name", cf.ORDER)
@pytest.mark.parametrize("value", [0, 0xFFFFFFFF])
def test_equal_priorities(name, value):
    """All priorities equal: the chunk id breaks every remaining tie."""
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 9, 0, 64, opts, plan.prio_stride)
    prio[:] = value
    check(plan, ref, routes, prio, f"{name} prio={value:#x}")


@pytest.mark.parametrize("name", cf.ORDER)
def test_few_distinct_priorities(name):
    """Priorities from {0, 1, 2}: many ties on (rem, trav, prio)."""
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 11, 0, 64, opts, plan.prio_stride)
    prio %= 3
    check(plan, ref, routes, prio, f"{name} prio%3")


@pytest.mark.parametrize("P", [2, 3, 5, 16, 33, 64])
def test_unidirectional_ring_closed_form(P):
    w = cf.uni_ring_ag(P)
    plan, ref, opts = plans(w)
    routes, prio = generate(P, 0, 40, opts, plan.prio_stride)
    mk, ok = check(plan, ref, routes, prio, f"uniring{P}")
    assert (mk == (P - 1) * int(plan.link_costs()[0])).all() and ok.all()


@pytest.mark.parametrize("make", [lambda: cf.full_a2a(4), lambda: cf.full_a2a(9),
                                  lambda: cf.full_ag(5, k=3, chunks_per_rank=3),
                                  lambda: cf.full_ag(12, k=6),
                                  lambda: cf.explicit_multicast(
                                      cf.full_ag(6, k=4), [0, 1, 2, 3, 4, 5, 0, 3],
                                      [[1, 3], [0, 2, 4, 5], [2], [0, 1, 2, 4], [1, 2, 3, 5],
                                       [0], [1, 2, 3, 4, 5], []])])
def test_small_topologies(make):
    w = make()
    plan, ref, opts = plans(w)
    routes, prio = generate(3, 0, 500, opts, plan.prio_stride)
    check(plan, ref, routes, prio, w.name)


def test_alltoall_with_two_chunks_per_pair():
    P = 6
    row_ptr, col, a, b = cf.csr_from_edges(P + 1, cf.switch_edges(range(P), P, 700, 8))
    w = cf.Workload("star6x2", P + 1, P, row_ptr, col, a, b, None, cf.ALLTOALL, 2, 1 << 18,
                    cf.RELAY1)
    plan, ref, opts = plans(w)
    routes, prio = generate(4, 0, 300, opts, plan.prio_stride)
    check(plan, ref, routes, prio, w.name)


# ----------------------------------------------------------------------------
# determinism, batch splits, streams
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["twonode16_ag", "fournode64_a2a"])
def test_repeatable_and_split_invariant(name):
    """Three launches give the same bits, and two half launches equal one."""
    w = cf.named(name)
    plan, _, opts = plans(w)
    n = 1000 if name == "fournode64_a2a" else 4000
    routes, prio = generate(w.seed, 0, n, opts, plan.prio_stride)
    say(f"[gpu] {name} repeat/split n={n}")
    d_r = torch.from_numpy(routes).cuda()
    d_p = torch.from_numpy(prio.view(np.int32)).cuda()
    outs = []
    for _ in range(3):
        mk = torch.empty(n, dtype=torch.int32, device="cuda")
        ok = torch.empty(n, dtype=torch.uint8, device="cuda")
        plan.eval_tensors(d_r, d_p, mk, ok)
        outs.append((mk.cpu(), ok.cpu()))
    for mk, ok in outs[1:]:
        assert torch.equal(mk, outs[0][0]) and torch.equal(ok, outs[0][1])
    h = 377
    mk = torch.empty(n, dtype=torch.int32, device="cuda")
    ok = torch.empty(n, dtype=torch.uint8, device="cuda")
    plan.eval_tensors(d_r[:h], d_p[:h], mk[:h], ok[:h])
    plan.eval_tensors(d_r[h:], d_p[h:], mk[h:], ok[h:])
    torch.cuda.synchronize()
    assert torch.equal(mk.cpu(), outs[0][0]) and torch.equal(ok.cpu(), outs[0][1])


def test_runs_on_a_side_stream():
    w = cf.switch16_a2a()
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed, 0, 512, opts, plan.prio_stride)
    say("[gpu] switch16_a2a on a side stream")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        d_r = torch.from_numpy(routes).cuda()
        d_p = torch.from_numpy(prio.view(np.int32)).cuda()
        mk = torch.empty(512, dtype=torch.int32, device="cuda")
        ok = torch.empty(512, dtype=torch.uint8, device="cuda")
        plan.eval_tensors(d_r, d_p, mk, ok, stream=s)
    s.synchronize()
    rmk, rok = ref.eval(routes, prio)
    assert (mk.cpu().numpy().view(np.uint32) == rmk).all() and (ok.cpu().numpy() == rok).all()


def hybrid_multicast(P, kind, cpr, k=4):
    """P ranks on one switch (vertex P) plus a bidirectional ring of direct
    links. V = P + 1 does not divide 64, so a chunk's vertex slots straddle
    the kernel's 64-slot groups and a parent can sit in an earlier group than
    its child; trees mix direct and switched hops and run several levels deep."""
    edges = cf.switch_edges(range(P), P, 700, 8) + cf.ring_edges(range(P), 1500, 8)
    row_ptr, col, a, b = cf.csr_from_edges(P + 1, edges)
    return cf.Workload(f"hybrid{P}_{kind}_{cpr}", P + 1, P, row_ptr, col, a, b, None, kind, cpr,
                       65536, cf.KSHORTEST, k=k)


@pytest.mark.parametrize("greedy", [0, 1])
@pytest.mark.parametrize("kind", [cf.ALLGATHER, cf.REDUCESCATTER, cf.ALLREDUCE])
@pytest.mark.parametrize("P,cpr", [(8, 1), (8, 2), (16, 1), (16, 2)])
def test_multicast_slots_straddling_groups(kind, P, cpr, greedy):
    from paper_2111_04867_amd.binding import Plan
    w = hybrid_multicast(P, kind, cpr)
    if greedy:
        w = cf.with_greedy(w)
    plan, ref = Plan.from_workload(w), OraclePlan.from_workload(w)
    opts = plan.route_options()
    assert (opts == ref.route_options()).all()
    routes, prio = generate(31 + P + cpr, 0, 600, opts, plan.prio_stride)
    say(f"[gpu] {w.name}: 600 candidates")
    mk, ok = plan.eval(routes, prio)
    rmk, rok = ref.eval_threads(routes, prio)
    bad = np.nonzero((mk != rmk) | (ok != rok))[0]
    assert bad.size == 0, f"{w.name}: {bad.size} mismatches, first at {bad[:5].tolist()}"


@pytest.mark.parametrize("option", ["static", "contig", "greedy", "rgreedy"])
def test_alltoall_pairs_without_any_route(option):
    """Pairs the sketch leaves without any route option can never be
    delivered: every candidate is invalid (regression: the register-resident
    kernel once skipped such pairs and reported valid)."""
    edges = [(0, 1, 700, 46), (1, 0, 700, 46), (2, 3, 700, 46), (3, 2, 700, 46),
             (1, 3, 1700, 106), (3, 1, 1700, 106)]
    row_ptr, col, a, b = cf.csr_from_edges(4, edges)
    node_of = np.array([0, 0, 1, 1], dtype=np.int32)
    relay = np.array([1, 0, 1, 0], dtype=np.uint8)  # the IB link joins two non-relays
    w = cf.Workload("split4_a2a", 4, 4, row_ptr, col, a, b, node_of, cf.ALLTOALL, 2, 65536,
                    cf.KSHORTEST, k=2, max_cross=1, relay=relay)
    w = {"static": w, "contig": cf.with_contiguity(w), "greedy": cf.with_greedy(w),
         "rgreedy": cf.with_reverse_greedy(w)}[option]
    plan, ref, opts = plans(w)
    assert (opts == 0).any() and (opts > 0).any()
    routes, prio = generate(3, 0, 64, opts, plan.prio_stride)
    mk, ok = check(plan, ref, routes, prio, f"split4 {option}")
    assert not ok.any() and (mk > 0).all()
