"""Pins of the oracle's algorithmic operation count (orc_eval_ops).

The count prices one candidate's evaluation against the chip's integer
issue rate. Its model: one operation per link of every routed path walked
to build the send set, three per send for the Step-2 keys (Sec. 5.1),
n_l * ceil(log2 n_l) comparisons to order the n_l sends of each link
(App. B.2), four per send for the timing sweep (App. B.3), two per word of
the presence bitmasks the postcondition reads (App. B).

The pins: closed forms on the unidirectional ring (P = 2..64) and the
direct star Alltoall, the constant of the 4-ring, the empty candidate, and
an independent recount from the brute-force send sets of tests/bruteforce.py
on small random plans.
"""
import math

import numpy as np
import pytest

import bruteforce as bf
from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate


def clog2(n):
    return 0 if n <= 1 else math.ceil(math.log2(n))


def words(n_bits):
    return (n_bits + 31) // 32


@pytest.mark.parametrize("P", [2, 3, 4, 5, 8, 13, 16, 31, 32, 33, 64])
def test_unidirectional_ring_closed_form(P):
    """Chunk of rank r walks 1 + 2 + ... + (P-1) links to reach everyone;
    P(P-1) sends; each of the P links carries P-1 of them; every vertex
    keeps ceil(P/32) presence words."""
    w = cf.uni_ring_ag(P)
    plan = OraclePlan.from_workload(w)
    routes, prio = generate(P, 0, 3, plan.route_options(), plan.prio_stride)
    _, _, ops = plan.eval_ops(routes, prio)
    sends = P * (P - 1)
    want = P * P * (P - 1) // 2 + 7 * sends + P * (P - 1) * clog2(P - 1) + 2 * P * words(P)
    assert ops.tolist() == [want] * 3


@pytest.mark.parametrize("P", [2, 3, 5, 9, 16, 40])
def test_star_alltoall_closed_form(P):
    """Direct routes through one switch: every off-diagonal chunk takes an
    uplink and a downlink (2 visits, 2 sends); every uplink and downlink
    carries P-1 sends; every rank keeps ceil(P/32) presence words."""
    row_ptr, col, a, b = cf.csr_from_edges(P + 1, cf.switch_edges(range(P), P, 700, 8))
    w = cf.Workload(f"star{P}", P + 1, P, row_ptr, col, a, b, None, cf.ALLTOALL, 1, 65536,
                    cf.KSHORTEST, k=1)
    plan = OraclePlan.from_workload(w)
    routes, prio = generate(P, 0, 2, plan.route_options(), plan.prio_stride)
    _, _, ops = plan.eval_ops(routes, prio)
    sends = 2 * P * (P - 1)
    want = sends + 7 * sends + 2 * P * (P - 1) * clog2(P - 1) + 2 * P * words(P)
    assert ops.tolist() == [want] * 2


def test_ring4_constant():
    """The 4-ring of 1 MiB chunks: 4 chunks x (1 + 1 + 2) visits, 12 sends,
    four links with two sends and four with one, 4 presence words: 116."""
    w = cf.ring4_ag(n_candidates=256)
    plan = OraclePlan.from_workload(w)
    routes, prio = generate(w.seed, 0, 256, plan.route_options(), plan.prio_stride)
    _, _, ops = plan.eval_ops(routes, prio)
    assert (ops == 16 + 36 + 8 + 48 + 8).all()


@pytest.mark.parametrize("name", ["cubemesh8_ag", "switch16_a2a"])
def test_nothing_routed(name):
    """Every pair unrouted: no visits and no sends, only the postcondition's
    words are read."""
    w = cf.named(name)
    plan = OraclePlan.from_workload(w)
    routes = np.full((2, plan.route_stride), 255, dtype=np.uint8)
    prio = np.zeros((2, plan.prio_stride), dtype=np.uint32)
    mk, ok, ops = plan.eval_ops(routes, prio)
    if w.kind == cf.ALLTOALL:
        expect = 2 * w.P * words(w.P * w.chunks_per_rank)
    else:
        expect = 2 * w.V * words(w.P * w.chunks_per_rank)
    assert ops.tolist() == [expect] * 2 and mk.tolist() == [0, 0] and ok.tolist() == [0, 0]


def recount(w, plan, routes, prio):
    """The op model recomputed from the brute force's own send sets."""
    table = {(s, d): [plan.path(s, d, i) for i in range(plan.npaths(s, d))]
             for s in range(w.P) for d in range(w.P) if s != d}
    P, cpr = w.P, w.chunks_per_rank
    if w.kind == cf.ALLTOALL:
        C = P * P * cpr
        visits = sum(len(table[(c // cpr // P, c // cpr % P)][routes[c]])
                     for c in range(C) if c // cpr // P != c // cpr % P
                     and routes[c] < len(table[(c // cpr // P, c // cpr % P)]))
        post_words = P * words(P * cpr)
    else:
        C = P * cpr
        visits = sum(len(table[(c // cpr, d)][routes[c * P + d]])
                     for c in range(C) for d in range(P) if d != c // cpr
                     and routes[c * P + d] < len(table[(c // cpr, d)]))
        post_words = w.V * words(C)
    _, _, sends, _, _, _ = bf.evaluate(w, table, routes, prio, H=plan.max_hops)

    def phase(ss):
        per = {}
        for s in ss:
            per[s["link"]] = per.get(s["link"], 0) + 1
        return visits + 7 * len(ss) + sum(n * clog2(n) for n in per.values()) + 2 * post_words

    if w.kind == cf.ALLREDUCE:  # both phases walk the same trees
        half = len(sends) // 2
        return phase(sends[:half]) + phase(sends[half:])
    return phase(sends)


@pytest.mark.parametrize("kind", [cf.ALLGATHER, cf.ALLTOALL, cf.REDUCESCATTER, cf.ALLREDUCE])
def test_bruteforce_recount(kind):
    """Small bidirectional rings with chords and a switch, every kind: the
    count equals the model applied to the brute force's sends."""
    checked = 0
    for seed in range(400):
        if checked == 4:
            break
        w = cf.random_workload(1000 + seed)
        if w.kind != kind or w.contiguity or w.order or w.switch_ports or w.P > 6:
            continue
        try:
            plan = OraclePlan.from_workload(w)
        except Exception:
            continue  # a draw the route search refuses
        routes, prio = generate(seed, 0, 6, plan.route_options(), plan.prio_stride)
        routes[0, ::3] = 200  # some pairs unrouted
        _, _, ops = plan.eval_ops(routes, prio)
        assert ops.tolist() == [recount(w, plan, routes[i], prio[i]) for i in range(6)]
        checked += 1
    assert checked == 4


def test_headline_estimates():
    """The two headline plans land on the op model's planning estimates:
    about 6.0 K operations per two-node Allgather candidate and about 247 K
    per four-node Alltoall candidate (sampled)."""
    for name, est, n in (("twonode16_ag", 6.0e3, 64), ("fournode64_a2a", 2.47e5, 4)):
        w = cf.named(name)
        plan = OraclePlan.from_workload(w)
        routes, prio = generate(w.seed, 0, n, plan.route_options(), plan.prio_stride)
        _, _, ops = plan.eval_ops(routes, prio)
        assert abs(ops.mean() / est - 1) < 0.15, (name, ops.mean())
