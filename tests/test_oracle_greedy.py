"""Pins of the oracle's time-aware greedy link orders (App. B.2).

Reading: round by round, among the sends whose chunk has arrived at their
source, the one that can start earliest -- max(its link's time, its chunk's
time) -- is scheduled next; ties go to the Step-2 heuristics (longer
remaining path, then shorter travelled path), then priority, then chunk id;
the link's and the chunk's times advance by the link latency.

The pins: closed forms where every order is forced, a hand-worked case where
the greedy avoids the idle link that the static order causes, the greedy's
defining choice property on every link of the named workloads, and the
optimum over all link orders as a lower bound on tiny inputs.
"""
import numpy as np
import pytest

import bruteforce as bf
from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate

C1 = 48935  # 1 MiB at 700 ns + 46 ps/B


def greedy(w):
    plan = OraclePlan.from_workload(w)
    plan.set_order(1)
    return plan


def test_ring4_every_candidate_two_costs():
    w = cf.ring4_ag()
    plan = greedy(w)
    routes, prio = generate(w.seed, 0, 256, plan.route_options(), plan.prio_stride)
    mk, ok = plan.eval(routes, prio)
    assert ok.all() and (mk == 2 * C1).all()


@pytest.mark.parametrize("P", [2, 3, 5, 8])
def test_unidirectional_ring(P):
    w = cf.uni_ring_ag(P)
    plan = greedy(w)
    routes, prio = generate(1, 0, 8, plan.route_options(), plan.prio_stride)
    mk, ok = plan.eval(routes, prio)
    assert ok.all() and (mk == (P - 1) * C1).all()


def chain4():
    """0 -> 1 -> 2 -> 3 (one way), explicit chunks: A from 0 to 3, B1 and B2
    from 1 to 2."""
    edges = [(0, 1, 700, 46), (1, 2, 700, 46), (2, 3, 700, 46)]
    row_ptr, col, a, b = cf.csr_from_edges(4, edges)
    base = cf.Workload("chain4", 4, 4, row_ptr, col, a, b, None, cf.ALLGATHER, 1, 1 << 20,
                       cf.KSHORTEST, k=1)
    return cf.explicit_multicast(base, [0, 1, 1], [[3], [2], [2]])


def test_greedy_fills_the_idle_link():
    """Static order puts A (remaining 2c) first on 1 -> 2 although it only
    arrives at c: B1 and B2 wait, 4c in all. The greedy sends B1 at 0, then A
    at c (it ties B2 and has the longer remaining path), then B2: 3c."""
    w = chain4()
    static = OraclePlan.from_workload(w)
    g = greedy(w)
    routes = np.zeros((1, static.route_stride), dtype=np.uint8)
    prio = np.zeros((1, static.prio_stride), dtype=np.uint32)
    assert int(static.eval(routes, prio)[0][0]) == 4 * C1
    mk, ok, s = g.eval_detail(routes[0], prio[0])
    assert ok and mk == 3 * C1
    on12 = sorted((int(p), int(c), int(st)) for c, l, p, st in
                  zip(s["chunk"], s["link"], s["pos"], s["start"]) if l == 1)
    assert on12 == [(0, 1, 0), (1, 0, C1), (2, 2, 2 * C1)]


@pytest.mark.parametrize("name", ["cubemesh8_ag", "twonode16_ag", "switch16_a2a"])
def test_choice_property(name):
    """On every link, for consecutive sends x then y: x started at the
    earliest time available to it, and no later send y could have started
    earlier than x, nor at the same time with a smaller key."""
    w = cf.named(name)
    plan = greedy(w)
    n = 6 if w.kind == cf.ALLGATHER else 2
    routes, prio = generate(w.seed, 0, n, plan.route_options(), plan.prio_stride)
    for r, p in zip(routes, prio):
        mk, ok, s = plan.eval_detail(r, p)
        m = len(s["chunk"])
        if w.kind == cf.ALLTOALL:
            arrive = {(int(c), int(h) + 1): int(f) for c, h, f in
                      zip(s["chunk"], s["hop"], s["finish"])}
            ready = [arrive.get((int(s["chunk"][i]), int(s["hop"][i])), 0) for i in range(m)]
        else:
            arrive = {(int(c), int(t)): int(f) for c, t, f in
                      zip(s["chunk"], s["to"], s["finish"])}
            ready = [arrive.get((int(s["chunk"][i]), int(s["from"][i])), 0) for i in range(m)]
        key = [(-int(s["rem"][i]), int(s["trav"][i]), int(s["prio"][i]), int(s["chunk"][i]))
               for i in range(m)]
        by_link = {}
        for i in range(m):
            by_link.setdefault(int(s["link"][i]), []).append(i)
        for l, idx in by_link.items():
            idx.sort(key=lambda i: int(s["pos"][i]))
            free = 0
            for q, x in enumerate(idx):
                assert int(s["start"][x]) == max(free, ready[x])
                for y in idx[q + 1:]:
                    alt = max(free, ready[y])
                    assert alt >= int(s["start"][x])
                    if alt == int(s["start"][x]):
                        assert key[x] < key[y]
                free = int(s["finish"][x])
        assert mk == max(int(f) for f in s["finish"])


def test_no_better_than_the_best_order():
    """Tiny inputs: the greedy's makespan is at least the optimum over every
    permutation of every link's sends (the greedy is one of them)."""
    w = cf.ring4_ag()
    plan = greedy(w)
    table = {(s, d): [plan.path(s, d, i) for i in range(plan.npaths(s, d))]
             for s in range(4) for d in range(4) if s != d}
    routes, prio = generate(9, 0, 4, plan.route_options(), plan.prio_stride)
    for r, p in zip(routes, prio):
        _, _, sends, _, _, _ = bf.evaluate(w, table, r, p)
        assert bf.optimum_over_orders(w, sends) <= int(plan.eval(r[None], p[None])[0][0])


def test_greedy_and_contiguity_are_not_combined():
    w = cf.with_contiguity(cf.twonode16_ag(n_candidates=2))
    plan = OraclePlan.from_workload(w)
    plan.set_order(1)
    routes, prio = generate(1, 0, 1, plan.route_options(), plan.prio_stride)
    with pytest.raises(Exception):
        plan.eval(routes, prio)


# ---- reverse path order ----------------------------------------------------
# Reading: App. B.2 lets the greedy start from the last link of every path
# instead of the first. The oracle runs the same greedy on the mirrored
# schedule (dependencies reversed, remaining and travelled lengths measured
# from the other end), reverses each link's service order and times those
# orders by the App. B.3 rule. The pins below check it against a separate
# event-loop formulation in `bruteforce` (mirrored dependency lists built by
# search, not by the oracle's successor counts), against the forced orders
# of single-hop plans, and against the defining property that the result is
# the least schedule of its own orders.

def ordered(w, mode):
    plan = OraclePlan.from_workload(w)
    plan.set_order(mode)
    return plan


def path_table(plan, P):
    return {(s, d): [plan.path(s, d, i) for i in range(plan.npaths(s, d))]
            for s in range(P) for d in range(P) if s != d}


def brute_greedy(w, table, r, p, H, reverse):
    """(makespan, {link: [(chunk, position)]}) of the greedy by brute force."""
    cost = bf.costs_of(w)
    if w.kind in (cf.REDUCESCATTER, cf.ALLREDUCE):
        C = w.P * w.chunks_per_rank
        owner = [c // w.chunks_per_rank for c in range(C)]
        posts = [list(range(w.P)) for _ in range(C)]
        CV = C * w.V
        ag, _ = bf.tree_sends(w, cost, table, r, p[:CV], owner, posts)
        rs = bf.reduce_sends(w, cost, ag, owner)
        orders = bf.greedy_link_orders(rs, cost, bf.reduce_deps(rs), reverse)
        _, fin = bf.reduce_least_schedule(rs, cost, orders)
        mk = max(fin, default=0)
        got = {(l, rs[i]["chunk"]): q for l, o in orders.items() for q, i in enumerate(o)}
        if w.kind == cf.REDUCESCATTER:
            return mk, got
        ag2, _ = bf.tree_sends(w, cost, table, r, p[CV:], owner, posts)
        deps = [[x] if x is not None else [] for x in bf.chunk_pred(ag2)]
        orders2 = bf.greedy_link_orders(ag2, cost, deps, reverse)
        _, fin2 = bf.least_schedule(ag2, cost, orders2)
        return mk + max(fin2, default=0), None
    _, _, sends, _, _, _ = bf.evaluate(w, table, r, p, H)
    deps = [[x] if x is not None else [] for x in bf.chunk_pred(sends)]
    orders = bf.greedy_link_orders(sends, cost, deps, reverse)
    _, fin = bf.least_schedule(sends, cost, orders)
    got = {(l, sends[i]["chunk"]): q for l, o in orders.items() for q, i in enumerate(o)}
    return max(fin, default=0), got


TINY = {
    "ring4_ag": lambda: cf.ring4_ag(),
    "uniring5_ag": lambda: cf.uni_ring_ag(5, chunk_bytes=4096),
    "chain4": chain4,
    "full4_a2a": lambda: cf.full_a2a(4, chunk_bytes=65536),
    "cubemesh8_ag": lambda: cf.cubemesh8_ag(),
    "ring4_rs": lambda: cf.as_reduction(cf.ring4_ag(), cf.REDUCESCATTER),
    "ring4_ar": lambda: cf.as_reduction(cf.ring4_ag(), cf.ALLREDUCE),
    "full4_rs": lambda: cf.as_reduction(cf.full_ag(4, chunk_bytes=65536, k=2),
                                        cf.REDUCESCATTER),
}


@pytest.mark.parametrize("mode", [1, 2])
@pytest.mark.parametrize("name", sorted(TINY))
def test_greedy_matches_event_loop(name, mode):
    """Both greedy directions equal the brute-force event loop followed by
    the brute-force least schedule: makespan and every link's order."""
    w = TINY[name]()
    plan = ordered(w, mode)
    table = path_table(plan, w.P)
    routes, prio = generate(17, 0, 6, plan.route_options(), plan.prio_stride)
    prio[1::2, ::2] = 3  # equal priorities
    for r, p in zip(routes, prio):
        want_mk, want_pos = brute_greedy(w, table, r, p, plan.max_hops, reverse=mode == 2)
        mk, ok, s = plan.eval_detail(r, p)
        assert mk == want_mk
        if want_pos is not None:
            got = {(int(l), int(c)): int(q) for l, c, q in zip(s["link"], s["chunk"], s["pos"])}
            assert got == want_pos


def test_reverse_order_single_hop_reverses_the_static_order():
    """Direct routes only: every send is ready at once in both directions and
    every link's sends tie on the Step-2 key, so the static order is
    (priority, chunk) ascending and the mirrored greedy serves the links in
    that order too; the reverse path order is therefore its exact reverse,
    and with no chunk dependencies the makespan (the busiest link) is the
    same."""
    w = cf.full_a2a(5, chunk_bytes=65536)
    static, rev = ordered(w, 0), ordered(w, 2)
    routes = np.zeros((4, static.route_stride), dtype=np.uint8)  # option 0: direct
    _, prio = generate(3, 0, 4, static.route_options(), static.prio_stride)
    prio[2] = 0  # all equal: chunk order decides
    for r, p in zip(routes, prio):
        m0, _, s0 = static.eval_detail(r, p)
        m2, _, s2 = rev.eval_detail(r, p)
        assert m0 == m2
        n_on = {}
        for l in s0["link"]:
            n_on[int(l)] = n_on.get(int(l), 0) + 1
        pos0 = {(int(l), int(c)): int(q) for l, c, q in zip(s0["link"], s0["chunk"], s0["pos"])}
        pos2 = {(int(l), int(c)): int(q) for l, c, q in zip(s2["link"], s2["chunk"], s2["pos"])}
        assert pos2 == {k: n_on[k[0]] - 1 - q for k, q in pos0.items()}


@pytest.mark.parametrize("name", ["cubemesh8_ag", "twonode16_ag", "switch16_a2a"])
def test_reverse_order_is_the_least_schedule_of_its_orders(name):
    """On the named workloads every send starts at the later of its chunk's
    arrival and the end of the send before it on its link."""
    w = cf.named(name)
    plan = ordered(w, 2)
    routes, prio = generate(w.seed, 0, 2, plan.route_options(), plan.prio_stride)
    for r, p in zip(routes, prio):
        mk, ok, s = plan.eval_detail(r, p)
        m = len(s["chunk"])
        if w.kind == cf.ALLTOALL:
            arrive = {(int(c), int(h) + 1): int(f) for c, h, f in
                      zip(s["chunk"], s["hop"], s["finish"])}
            ready = [arrive.get((int(s["chunk"][i]), int(s["hop"][i])), 0) for i in range(m)]
        else:
            arrive = {(int(c), int(t)): int(f) for c, t, f in
                      zip(s["chunk"], s["to"], s["finish"])}
            ready = [arrive.get((int(s["chunk"][i]), int(s["from"][i])), 0) for i in range(m)]
        prev = {}
        for i in sorted(range(m), key=lambda i: (int(s["link"][i]), int(s["pos"][i]))):
            l = int(s["link"][i])
            assert int(s["pos"][i]) == (prev[l][0] + 1 if l in prev else 0)
            free = prev[l][1] if l in prev else 0
            assert int(s["start"][i]) == max(free, ready[i])
            prev[l] = (int(s["pos"][i]), int(s["finish"][i]))
        assert ok and mk == max(int(f) for f in s["finish"])
