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
