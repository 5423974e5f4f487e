"""Pins of the oracle's ReduceScatter and Allreduce.

Reading (TACCL builds both from an Allgather algorithm, Sec. 5.2):
ReduceScatter runs every chunk's Allgather tree backwards; the send from v to
its parent carries v's partial reduction and waits for every send into v;
Step 2 measures lengths on the reversed tree. Allreduce is ReduceScatter
then Allgather on the same trees, timed back to back, each phase with its
own row of priorities.

The pins: closed forms on the 4-ring and on two ranks, an independent
brute-force evaluation (tests/bruteforce.py: reversed trees by explicit
walks, fixed-point least schedule with all-children readiness), the
composition of Allreduce from separately evaluated phases, and schedule
invariants on the named workloads.
"""
import numpy as np
import pytest

import bruteforce as bf
from oracle import OraclePlan
from oracle.oracle import OracleError
from workloads import configs as cf
from workloads import generate

RING_COST = 48935  # 1 MiB at 700 ns + 46 ps/B


def reduction(w, kind):
    return cf.as_reduction(w, kind)


def table_of(plan, w):
    return {(s, d): [plan.path(s, d, i) for i in range(plan.npaths(s, d))]
            for s in range(w.P) for d in range(w.P) if s != d}


@pytest.mark.parametrize("kind,want", [(cf.REDUCESCATTER, 2 * RING_COST),
                                       (cf.ALLREDUCE, 4 * RING_COST)])
def test_ring4_every_routing(kind, want):
    """4-ring: every routing and priority draw reduces in two link costs (the
    distance bound), and Allreduce takes one such phase twice."""
    w = reduction(cf.ring4_ag(), kind)
    plan = OraclePlan.from_workload(w)
    opts = plan.route_options()
    multi = [e for e in range(len(opts)) if opts[e] == 2]
    _, prio = generate(3, 0, 4, opts, plan.prio_stride)
    for bits in range(1 << len(multi)):
        routes = np.zeros(plan.route_stride, dtype=np.uint8)
        for j, e in enumerate(multi):
            routes[e] = (bits >> j) & 1
        mk, ok = plan.eval(np.repeat(routes[None], len(prio), 0), prio)
        assert ok.all() and (mk == want).all()


def test_two_ranks():
    row_ptr, col, a, b = cf.csr_from_edges(2, [(0, 1, 700, 46), (1, 0, 700, 46)])
    base = cf.Workload("pair", 2, 2, row_ptr, col, a, b, None, cf.ALLGATHER, 3, 1 << 20,
                       cf.KSHORTEST, k=1)
    for kind, phases in [(cf.REDUCESCATTER, 1), (cf.ALLREDUCE, 2)]:
        plan = OraclePlan.from_workload(reduction(base, kind))
        routes, prio = generate(5, 0, 16, plan.route_options(), plan.prio_stride)
        mk, ok = plan.eval(routes, prio)
        # three chunks per rank cross each direction one after the other
        assert ok.all() and (mk == phases * 3 * RING_COST).all()


@pytest.mark.parametrize("kind", [cf.REDUCESCATTER, cf.ALLREDUCE])
@pytest.mark.parametrize("cpr", [1, 2])
def test_bruteforce_full4(kind, cpr):
    w = reduction(cf.full_ag(4, k=3, chunks_per_rank=cpr), kind)
    plan = OraclePlan.from_workload(w)
    table = table_of(plan, w)
    routes, prio = generate(17 + cpr, 0, 40, plan.route_options(), plan.prio_stride)
    for r, p in zip(routes, prio):
        mk, ok, s = plan.eval_detail(r, p)
        bmk, bok, bsends, bstart, bfinish, _ = bf.evaluate(w, table, r, p)
        assert (mk, ok) == (bmk, bok)
        assert len(s["chunk"]) == len(bsends)
        got = sorted(zip(s["chunk"].tolist(), s["link"].tolist(), s["rem"].tolist(),
                         s["trav"].tolist(), s["start"].tolist(), s["finish"].tolist()))
        want = sorted((b["chunk"], b["link"], b["rem"], b["trav"], st, fi)
                      for b, st, fi in zip(bsends, bstart, bfinish))
        assert got == want


def test_bruteforce_cubemesh8_reducescatter():
    w = reduction(cf.cubemesh8_ag(), cf.REDUCESCATTER)
    plan = OraclePlan.from_workload(w)
    table = table_of(plan, w)
    routes, prio = generate(23, 0, 6, plan.route_options(), plan.prio_stride)
    for r, p in zip(routes, prio):
        mk, ok, _ = plan.eval_detail(r, p)
        bmk, bok, _, _, _, _ = bf.evaluate(w, table, r, p)
        assert (mk, ok) == (bmk, bok)


@pytest.mark.parametrize("name", ["cubemesh8_ag", "twonode16_ag"])
def test_allreduce_is_reducescatter_then_allgather(name):
    """Allreduce = ReduceScatter on the first priority row + Allgather on the
    second, evaluated by separate plans."""
    ag = cf.named(name)
    ar = OraclePlan.from_workload(reduction(ag, cf.ALLREDUCE))
    rs = OraclePlan.from_workload(reduction(ag, cf.REDUCESCATTER))
    agp = OraclePlan.from_workload(ag)
    routes, prio = generate(ag.seed, 0, 16, ar.route_options(), ar.prio_stride)
    half = rs.prio_stride
    m1, v1 = rs.eval(routes, np.ascontiguousarray(prio[:, :half]))
    m2, v2 = agp.eval(routes, np.ascontiguousarray(prio[:, half:]))
    m, v = ar.eval(routes, prio)
    assert (m == m1 + m2).all() and (v == (v1 & v2)).all()


@pytest.mark.parametrize("name", ["cubemesh8_ag", "twonode16_ag"])
def test_reducescatter_schedule_invariants(name):
    """Every send out of v starts after every send into v (same chunk) has
    ended; sends on one link do not overlap and follow the Step-2 order;
    remaining length falls by the link's cost along the reversed tree."""
    w = reduction(cf.named(name), cf.REDUCESCATTER)
    plan = OraclePlan.from_workload(w)
    cost = plan.link_costs()
    routes, prio = generate(w.seed, 0, 8, plan.route_options(), plan.prio_stride)
    for r, p in zip(routes, prio):
        mk, ok, s = plan.eval_detail(r, p)
        n = len(s["chunk"])
        into = {}
        out_of = {}
        for i in range(n):
            into.setdefault((int(s["chunk"][i]), int(s["to"][i])), []).append(i)
            out_of[(int(s["chunk"][i]), int(s["from"][i]))] = i
        for i in range(n):
            c, v = int(s["chunk"][i]), int(s["from"][i])
            for j in into.get((c, v), []):
                assert s["start"][i] >= s["finish"][j]
            u = int(s["to"][i])
            if (c, u) in out_of:
                k = out_of[(c, u)]
                assert int(s["rem"][i]) == int(s["rem"][k]) + int(cost[s["link"][i]])
        by_link = {}
        for i in range(n):
            by_link.setdefault(int(s["link"][i]), []).append(i)
        for l, idx in by_link.items():
            idx.sort(key=lambda i: int(s["pos"][i]))
            for a_, b_ in zip(idx, idx[1:]):
                assert s["start"][b_] >= s["finish"][a_]
                ka = (-int(s["rem"][a_]), int(s["trav"][a_]), int(s["prio"][a_]))
                kb = (-int(s["rem"][b_]), int(s["trav"][b_]), int(s["prio"][b_]))
                assert ka <= kb
        assert mk == max(int(x) for x in s["finish"])


def test_reduction_needs_reverse_links():
    with pytest.raises(OracleError):
        OraclePlan.from_workload(reduction(cf.uni_ring_ag(4), cf.REDUCESCATTER))
