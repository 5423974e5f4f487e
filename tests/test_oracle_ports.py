"""Pins of the oracle's switch-port model (App. B.3 switch constraints,
App. B.2 switch_send_order / switch_recv_order).

Reading: in an Alltoall, a hop into a switch vertex and the hop out of it
(rank -> switch -> rank) are one switched send that costs one latency (the
uplink's alpha and beta) and holds the sender's send port (its uplink) and
the receiver's receive port (its downlink) for its whole duration; each port
serves its sends in Step-2 order. Other links are unchanged.

The pins: one switched send on two ranks, port-load lower bounds and port
exclusivity on the named switch workloads, identity with the store-and-
forward model where there is no switch, and an independent brute force
(tests/bruteforce.py: units built from the path table, fixed-point least
schedule over both ports) on small switched topologies.
"""
import numpy as np
import pytest

import bruteforce as bf
from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate


def star(P, relays=True, chunk_bytes=256 * 1024):
    """P ranks on one switch (vertex P), Alltoall; direct, or direct and one
    relay rank."""
    row_ptr, col, a, b = cf.csr_from_edges(P + 1, cf.switch_edges(range(P), P, 700, 8))
    mode = cf.RELAY1 if relays else cf.KSHORTEST
    return cf.Workload(f"star{P}", P + 1, P, row_ptr, col, a, b, None, cf.ALLTOALL, 1,
                       chunk_bytes, mode, k=1, switch_ports=1)


def cost(alpha, beta, nbytes):
    return alpha + (beta * nbytes + 999) // 1000


def test_two_ranks_one_switched_send_each():
    w = star(2, relays=False)
    plan = OraclePlan.from_workload(w)
    routes, prio = generate(1, 0, 8, plan.route_options(), plan.prio_stride)
    mk, ok = plan.eval(routes, prio)
    c = cost(700, 8, 256 * 1024)
    assert ok.all() and (mk == c).all()
    plan.set_switch_ports(0)  # store and forward: uplink then downlink
    mk0, _ = plan.eval(routes, prio)
    assert (mk0 == 2 * c).all()


@pytest.mark.parametrize("P", [3, 4])
def test_bruteforce_star(P):
    w = star(P)
    plan = OraclePlan.from_workload(w)
    table = {(s, d): [plan.path(s, d, i) for i in range(plan.npaths(s, d))]
             for s in range(P) for d in range(P) if s != d}
    routes, prio = generate(30 + P, 0, 30, plan.route_options(), plan.prio_stride)
    for r, p in zip(routes, prio):
        mk, ok, s = plan.eval_detail(r, p)
        bmk, bok, units, bstart, bfinish, _ = bf.evaluate(w, table, r, p, H=plan.max_hops)
        assert (mk, ok) == (bmk, bok)
        got = sorted(zip(s["chunk"].tolist(), s["hop"].tolist(), s["start"].tolist(),
                         s["finish"].tolist()))
        want = sorted((u["chunk"], u["hop"], st, fi) for u, st, fi in zip(units, bstart, bfinish))
        assert got == want


def test_bruteforce_two_switches():
    """Two switch nodes of 3 ranks, IB between rank i of each node: switched
    sends inside a node, ordinary links between nodes."""
    edges = cf.switch_edges(range(3), 6, 700, 8) + cf.switch_edges(range(3, 6), 7, 700, 8)
    for i in range(3):
        edges += [(i, 3 + i, 1700, 106), (3 + i, i, 1700, 106)]
    row_ptr, col, a, b = cf.csr_from_edges(8, edges)
    node_of = np.array([0, 0, 0, 1, 1, 1, 0, 1], dtype=np.int32)
    relay = np.array([1] * 6 + [0, 0], dtype=np.uint8)
    w = cf.Workload("twoswitch", 8, 6, row_ptr, col, a, b, node_of, cf.ALLTOALL, 1, 65536,
                    cf.HIER_RELAY, max_cross=1, relay=relay, switch_ports=1)
    plan = OraclePlan.from_workload(w)
    table = {(s, d): [plan.path(s, d, i) for i in range(plan.npaths(s, d))]
             for s in range(6) for d in range(6) if s != d}
    routes, prio = generate(44, 0, 25, plan.route_options(), plan.prio_stride)
    for r, p in zip(routes, prio):
        mk, ok = plan.eval(r[None], p[None])
        bmk, bok, _, _, _, _ = bf.evaluate(w, table, r, p, H=plan.max_hops)
        assert (int(mk[0]), int(ok[0])) == (bmk, bok)


@pytest.mark.parametrize("name", ["switch16_a2a", "fournode64_a2a"])
def test_ports_are_exclusive_and_bound_the_makespan(name):
    """Sends into one rank through its switch never overlap (its receive
    port), sends out of one rank through its switch never overlap (its send
    port), and the busiest port bounds the makespan from below."""
    w = cf.with_switch_ports(cf.named(name))
    plan = OraclePlan.from_workload(w)
    routes, prio = generate(w.seed, 0, 3, plan.route_options(), plan.prio_stride)
    for r, p in zip(routes, prio):
        mk, ok, s = plan.eval_detail(r, p)
        assert ok
        sw_out, sw_in = {}, {}
        for i in range(len(s["chunk"])):
            src, dst = w.edges()[int(s["link"][i])]
            if dst >= w.P:  # a switched send: uplink of its source
                sw_out.setdefault(int(s["from"][i]), []).append(i)
                sw_in.setdefault(int(s["to"][i]), []).append(i)
        for groups in (sw_out, sw_in):
            for idx in groups.values():
                spans = sorted((int(s["start"][i]), int(s["finish"][i])) for i in idx)
                for (a0, a1), (b0, _) in zip(spans, spans[1:]):
                    assert b0 >= a1
                busy = sum(b - a for a, b in spans)
                assert mk >= busy


def test_no_switch_means_no_change():
    w = cf.cubemesh8_ag()
    w2 = cf.full_a2a(5)
    for base in (w, w2):
        plan = OraclePlan.from_workload(base)
        routes, prio = generate(3, 0, 32, plan.route_options(), plan.prio_stride)
        m0 = plan.eval(routes, prio)
        plan.set_switch_ports(1)
        m1 = plan.eval(routes, prio)
        assert np.array_equal(m0[0], m1[0]) and np.array_equal(m0[1], m1[1])
