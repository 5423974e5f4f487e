"""Pins of the oracle's switch-hyperedge connection count (the is_util count
that the uc-max / uc-min policies weigh: Sec. 5.1 switch-hyperedge policy,
App. B.3).

Reading: a connection is an ordered rank pair (a, b) that carries some chunk
through switch vertices only. Alltoall: two ranks of a routed path with only
switch vertices between them. Multicast: a rank whose tree parent is a
switch, paired with the nearest rank above it. ReduceScatter reverses each
pair; Allreduce has both directions.

The pins: closed forms on a star and on the four-node topology, zero where
there is no switch, and an independent count from explicit path walks and
brute-force trees (tests/bruteforce.py) on small switched topologies.
"""
import numpy as np
import pytest

import bruteforce as bf
from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate


def star(P, kind, relays=True, cpr=1):
    row_ptr, col, a, b = cf.csr_from_edges(P + 1, cf.switch_edges(range(P), P, 700, 8))
    mode = cf.RELAY1 if relays else cf.KSHORTEST
    return cf.Workload(f"star{P}", P + 1, P, row_ptr, col, a, b, None, kind, cpr, 65536, mode,
                       k=1)


def table_of(plan, w):
    return {(s, d): [plan.path(s, d, i) for i in range(plan.npaths(s, d))]
            for s in range(w.P) for d in range(w.P) if s != d}


def pairs_alltoall(w, table, routes):
    P, cpr = w.P, w.chunks_per_rank
    out = set()
    for c in range(P * P * cpr):
        s, d = divmod(c // cpr, P)
        if s == d or routes[c] >= len(table[(s, d)]):
            continue
        verts = bf.path_vertices(w, table[(s, d)][routes[c]], s)
        ranks = [i for i, v in enumerate(verts) if v < P]
        for i, j in zip(ranks, ranks[1:]):
            if j - i > 1:
                out.add((verts[i], verts[j]))
    return out


def pairs_multicast(w, table, routes):
    P, cpr = w.P, w.chunks_per_rank
    C = P * cpr
    owner = [c // cpr for c in range(C)]
    posts = [list(range(P)) for _ in range(C)]
    prio = np.zeros(C * w.V, dtype=np.uint32)
    sends, _ = bf.tree_sends(w, bf.costs_of(w), table, routes, prio, owner, posts)
    out = set()
    for c in range(C):
        parent = {s["to"]: s["frm"] for s in sends if s["chunk"] == c}
        for b, u in parent.items():
            if b < P and u >= P:
                x = u
                while x >= P:
                    x = parent[x]
                out.add((x, b))
    return out


def test_star_direct_every_pair():
    for kind in (cf.ALLTOALL, cf.ALLGATHER):
        w = star(5, kind, relays=False)
        plan = OraclePlan.from_workload(w)
        routes, _ = generate(1, 0, 4, plan.route_options(), plan.prio_stride)
        assert (plan.connections(routes) == 5 * 4).all()


def test_fournode_closed_form():
    """Every route of the four-node topology enters and leaves a switch only
    between ranks of one node, and every on-node pair is routed directly:
    4 nodes x 16 x 15 connections for every candidate."""
    w = cf.fournode64_a2a(n_candidates=4)
    plan = OraclePlan.from_workload(w)
    routes, _ = generate(w.seed, 0, 4, plan.route_options(), plan.prio_stride)
    assert (plan.connections(routes) == 4 * 16 * 15).all()


@pytest.mark.parametrize("name", ["ring4_ag", "cubemesh8_ag", "twonode16_ag"])
def test_no_switch_no_connection(name):
    w = cf.named(name)
    plan = OraclePlan.from_workload(w)
    routes, _ = generate(w.seed, 0, 16, plan.route_options(), plan.prio_stride)
    assert (plan.connections(routes) == 0).all()


@pytest.mark.parametrize("P", [3, 4, 6])
def test_bruteforce_alltoall_star(P):
    w = star(P, cf.ALLTOALL)
    plan = OraclePlan.from_workload(w)
    table = table_of(plan, w)
    routes, _ = generate(70 + P, 0, 40, plan.route_options(), plan.prio_stride)
    got = plan.connections(routes)
    want = [len(pairs_alltoall(w, table, r)) for r in routes]
    assert got.tolist() == want
    assert len(set(want)) > 1  # relays change the count


@pytest.mark.parametrize("P,cpr", [(3, 1), (4, 2), (5, 1)])
def test_bruteforce_multicast_and_reductions(P, cpr):
    w = star(P, cf.ALLGATHER, cpr=cpr)
    plan = OraclePlan.from_workload(w)
    table = table_of(plan, w)
    routes, _ = generate(80 + P, 0, 40, plan.route_options(), plan.prio_stride)
    rs = OraclePlan.from_workload(cf.as_reduction(w, cf.REDUCESCATTER))
    ar = OraclePlan.from_workload(cf.as_reduction(w, cf.ALLREDUCE))
    g, grs, gar = plan.connections(routes), rs.connections(routes), ar.connections(routes)
    for i, r in enumerate(routes):
        pairs = pairs_multicast(w, table, r)
        assert g[i] == len(pairs)
        assert grs[i] == len({(b, a) for a, b in pairs})
        assert gar[i] == len(pairs | {(b, a) for a, b in pairs})


def test_two_switches_bruteforce():
    """Switch nodes joined by IB between ranks: connections only inside a
    node, never across the IB links."""
    per = 3
    P = 2 * per
    edges = cf.switch_edges(range(per), P, 700, 8) + cf.switch_edges(range(per, P), P + 1, 700, 8)
    for i in range(per):
        edges += [(i, per + i, 1700, 106), (per + i, i, 1700, 106)]
    row_ptr, col, a, b = cf.csr_from_edges(P + 2, edges)
    node_of = np.array([0] * per + [1] * per + [0, 1], dtype=np.int32)
    relay = np.array([1] * P + [0, 0], dtype=np.uint8)
    w = cf.Workload("twoswitch", P + 2, P, row_ptr, col, a, b, node_of, cf.ALLTOALL, 1, 65536,
                    cf.HIER_RELAY, max_cross=1, relay=relay)
    plan = OraclePlan.from_workload(w)
    table = table_of(plan, w)
    routes, _ = generate(91, 0, 40, plan.route_options(), plan.prio_stride)
    got = plan.connections(routes)
    for i, r in enumerate(routes):
        pairs = pairs_alltoall(w, table, r)
        assert all(int(node_of[x]) == int(node_of[y]) for x, y in pairs)
        assert got[i] == len(pairs)


def switch_plus_directed_ring(P, kind, cpr=1):
    """Ranks on one switch plus a ring that is cheap one way (r -> r+1) and
    dear the other way (every link has its reverse, as reductions need): a
    chunk reaches some ranks over the ring and others through the switch, so
    the pairs of a candidate are not closed under reversal."""
    edges = cf.switch_edges(range(P), P, 700, 8)
    for r in range(P):
        edges += [(r, (r + 1) % P, 300, 8), ((r + 1) % P, r, 3000, 8)]
    row_ptr, col, a, b = cf.csr_from_edges(P + 1, edges)
    return cf.Workload(f"swring{P}", P + 1, P, row_ptr, col, a, b, None, kind, cpr, 65536,
                       cf.KSHORTEST, k=3)


@pytest.mark.parametrize("P,cpr", [(4, 1), (5, 2), (7, 1)])
def test_bruteforce_reductions_asymmetric(P, cpr):
    """ReduceScatter counts the reverse of every Allgather pair and Allreduce
    the union of both directions (App. B.3 is_util over the links each phase
    uses); on a topology whose pairs are asymmetric the three counts differ,
    so dropping either direction of the Allreduce union fails here."""
    w = switch_plus_directed_ring(P, cf.ALLGATHER, cpr=cpr)
    plan = OraclePlan.from_workload(w)
    table = table_of(plan, w)
    routes, _ = generate(120 + P, 0, 48, plan.route_options(), plan.prio_stride)
    rs = OraclePlan.from_workload(cf.as_reduction(w, cf.REDUCESCATTER))
    ar = OraclePlan.from_workload(cf.as_reduction(w, cf.ALLREDUCE))
    g, grs, gar = plan.connections(routes), rs.connections(routes), ar.connections(routes)
    asym = 0
    for i, r in enumerate(routes):
        pairs = pairs_multicast(w, table, r)
        rev = {(b, a) for a, b in pairs}
        assert g[i] == len(pairs)
        assert grs[i] == len(rev)
        assert gar[i] == len(pairs | rev)
        asym += gar[i] > g[i]
    assert asym > len(routes) // 2  # the union is larger than one direction
