"""Pins of the oracle's contiguous transfers (Sec. 4.1; Step 3 of Sec. 5.1;
the is_together constraints of App. B.3).

Reading: on a link whose endpoints lie in different nodes, a transfer
carries the next send of the link's Step-2 order plus every following send
of that order with the same remaining length whose chunk is already at the
link's source when the transfer starts; m chunks of S bytes cost
alpha + ceil(beta * m * S / 1000) ns and all arrive when the transfer ends.
Links inside a node never merge.

The pins: the paper's 17% example, closed forms on small chains, the cases
that must not merge, identity with the uncontiguous schedule where nothing
can merge, and an independent time-ordered simulation (tests/bruteforce.py)
on small two-node topologies.
"""
import json
import os

import numpy as np
import pytest

import bruteforce as bf
from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

NV_A, NV_B = 700, 46      # NDv2 NVLink alpha (ns) and beta (ps/B), Table 1
IB_A, IB_B = 1700, 106    # NDv2 InfiniBand


def cost(alpha, beta, nbytes):
    return alpha + (beta * nbytes + 999) // 1000


def explicit(V, edges, node_of, owner, posts, chunk_bytes, contiguity=1, k=4):
    """Explicit multicast on a custom topology (each edge listed once per
    direction)."""
    row_ptr, col, a, b = cf.csr_from_edges(V, edges)
    base = cf.Workload("custom", V, V, row_ptr, col, a, b, np.asarray(node_of, dtype=np.int32),
                       cf.ALLGATHER, 1, chunk_bytes, cf.KSHORTEST, k=k)
    w = cf.explicit_multicast(base, owner, posts)
    w.contiguity = contiguity
    return w


def run(w, routes=None, prio=None):
    plan = OraclePlan.from_workload(w)
    if routes is None:
        routes = np.zeros((1, plan.route_stride), dtype=np.uint8)
    if prio is None:
        prio = np.arange(plan.prio_stride, dtype=np.uint32)[None, :]
    mk, ok = plan.eval(routes, prio)
    return int(mk[0]), int(ok[0]), plan


def test_sec41_two_chunks_together_17_percent():
    """Two 32 KB chunks over one IB link: together one alpha, apart two."""
    g = json.load(open(os.path.join(GOLDEN, "alpha_beta_example.json")))
    S = g["chunk_bytes"]
    edges = [(0, 1, g["alpha_ns"], g["beta_ps_per_byte"]), (1, 0, g["alpha_ns"], g["beta_ps_per_byte"])]
    together, ok, _ = run(explicit(2, edges, [0, 1], [0, 0], [[1], [1]], S, contiguity=1))
    apart, ok2, _ = run(explicit(2, edges, [0, 1], [0, 0], [[1], [1]], S, contiguity=0))
    assert ok and ok2
    assert together == cost(g["alpha_ns"], g["beta_ps_per_byte"], 2 * S)
    assert apart == 2 * cost(g["alpha_ns"], g["beta_ps_per_byte"], S)
    assert abs((1 - together / apart) - g["stated_saving"]) < g["tolerance"]


@pytest.mark.parametrize("m", [1, 2, 3, 5, 8])
def test_m_chunks_one_transfer(m):
    """m chunks ready at the source of one IB link leave in one transfer."""
    S = 65536
    edges = [(0, 1, IB_A, IB_B), (1, 0, IB_A, IB_B)]
    mk, ok, _ = run(explicit(2, edges, [0, 1], [0] * m, [[1]] * m, S))
    assert ok and mk == cost(IB_A, IB_B, m * S)


def test_same_link_inside_a_node_never_merges():
    S = 65536
    edges = [(0, 1, IB_A, IB_B), (1, 0, IB_A, IB_B)]
    mk, ok, _ = run(explicit(2, edges, [0, 0], [0] * 3, [[1]] * 3, S))
    assert ok and mk == 3 * cost(IB_A, IB_B, S)


@pytest.mark.parametrize("m", [1, 2, 4])
def test_merged_chunks_are_forwarded_after_the_last_arrives(m):
    """0 -(IB)-> 1 -(NVLink)-> 2: the m chunks cross the IB link together,
    then leave rank 1 one after the other."""
    S = 65536
    edges = [(0, 1, IB_A, IB_B), (1, 0, IB_A, IB_B), (1, 2, NV_A, NV_B), (2, 1, NV_A, NV_B)]
    mk, ok, _ = run(explicit(3, edges, [0, 1, 1], [0] * m, [[2]] * m, S))
    ib = cost(IB_A, IB_B, m * S)
    assert ok and mk == ib + m * cost(NV_A, NV_B, S)


def test_different_remaining_lengths_do_not_merge():
    """Chunk 0 continues past rank 1, chunk 1 stops there: different remaining
    lengths, so they cross the IB link separately, the longer one first."""
    S = 65536
    edges = [(0, 1, IB_A, IB_B), (1, 0, IB_A, IB_B), (1, 2, NV_A, NV_B), (2, 1, NV_A, NV_B)]
    ib, nv = cost(IB_A, IB_B, S), cost(NV_A, NV_B, S)
    mk, ok, _ = run(explicit(3, edges, [0, 1, 1], [0, 0], [[2], [1]], S))
    assert ok and mk == max(ib + nv, 2 * ib)


def test_a_chunk_that_arrives_later_does_not_join():
    """Chunk 1 reaches rank 1 (over NVLink) only after chunk 0 starts on the
    IB link 1 -> 2, so it waits for the next transfer."""
    S = 65536
    edges = [(0, 1, NV_A, NV_B), (1, 0, NV_A, NV_B), (1, 2, IB_A, IB_B), (2, 1, IB_A, IB_B)]
    ib, nv = cost(IB_A, IB_B, S), cost(NV_A, NV_B, S)
    mk, ok, _ = run(explicit(3, edges, [0, 0, 1], [1, 0], [[2], [2]], S))
    assert ok and mk == max(ib, nv) + ib


@pytest.mark.parametrize("name", ["cubemesh8_ag", "switch16_a2a"])
def test_no_inter_node_link_means_no_change(name):
    """With every link inside one node the contiguous schedule is the
    uncontiguous one, candidate by candidate."""
    w = cf.named(name)
    plan = OraclePlan.from_workload(w)
    routes, prio = generate(w.seed, 0, 64, plan.route_options(), plan.prio_stride)
    base = plan.eval(routes, prio)
    plan.set_contiguity(1)
    contig = plan.eval(routes, prio)
    assert np.array_equal(base[0], contig[0]) and np.array_equal(base[1], contig[1])


def two_node_ag(P_per, chunks_per_rank, k=3):
    return cf.two_node_full(P_per, cf.ALLGATHER, chunks_per_rank=chunks_per_rank, k=k)


def two_node_a2a(P_per):
    return cf.two_node_full(P_per, cf.ALLTOALL)


def bf_table(w, hop_limit):
    return {(s, d): bf.sorted_paths(w, s, d, hop_limit) for s in range(w.P) for d in range(w.P)
            if s != d}


@pytest.mark.parametrize("cpr", [1, 2])
def test_time_ordered_simulation_allgather(cpr):
    """An independent simulation in time order agrees on every send."""
    w = two_node_ag(2, cpr)
    plan = OraclePlan.from_workload(w)
    table = {(s, d): [plan.path(s, d, i) for i in range(plan.npaths(s, d))]
             for s in range(w.P) for d in range(w.P) if s != d}
    routes, prio = generate(21, 0, 60, plan.route_options(), plan.prio_stride)
    merged = 0
    for r, p in zip(routes, prio):
        mk, ok, s = plan.eval_detail(r, p)
        bmk, bok, bsends, bstart, bfinish, _ = bf.evaluate(w, table, r, p)
        assert (mk, ok) == (bmk, bok)
        got = {(int(c), int(l)): (int(st), int(fi)) for c, l, st, fi in
               zip(s["chunk"], s["link"], s["start"], s["finish"])}
        for i, b in enumerate(bsends):
            assert got[(b["chunk"], b["link"])] == (bstart[i], bfinish[i])
        merged += len(bstart) - len(set(zip(bstart, bfinish, [b["link"] for b in bsends])))
    assert merged > 0  # the sample exercises merging


def test_time_ordered_simulation_alltoall():
    w = two_node_a2a(2)
    plan = OraclePlan.from_workload(w)
    table = {(s, d): [plan.path(s, d, i) for i in range(plan.npaths(s, d))]
             for s in range(w.P) for d in range(w.P) if s != d}
    routes, prio = generate(22, 0, 60, plan.route_options(), plan.prio_stride)
    merged = 0
    for r, p in zip(routes, prio):
        mk, ok, s = plan.eval_detail(r, p)
        bmk, bok, bsends, bstart, bfinish, _ = bf.evaluate(w, table, r, p, H=plan.max_hops)
        assert (mk, ok) == (bmk, bok)
        got = {(int(c), int(l)): (int(st), int(fi)) for c, l, st, fi in
               zip(s["chunk"], s["link"], s["start"], s["finish"])}
        for i, b in enumerate(bsends):
            assert got[(b["chunk"], b["link"])] == (bstart[i], bfinish[i])
        merged += len(bstart) - len(set(zip(bstart, bfinish, [b["link"] for b in bsends])))
    assert merged > 0


@pytest.mark.parametrize("name", ["twonode16_ag_contig", "fournode64_a2a_contig"])
def test_transfer_invariants(name):
    """On the named two- and four-node workloads: transfers on one link never
    overlap, a transfer's sends share its start and end, were ready at its
    start, have one remaining length, and the transfer costs
    alpha + ceil(beta * m * S / 1000); links inside a node carry one chunk
    per transfer."""
    w = cf.named(name)
    plan = OraclePlan.from_workload(w)
    n = 24 if w.kind == cf.ALLGATHER else 2
    routes, prio = generate(w.seed, 0, n, plan.route_options(), plan.prio_stride)
    S = w.chunk_bytes
    merged = 0
    for r, p in zip(routes, prio):
        mk, ok, s = plan.eval_detail(r, p)
        fin_into = {}
        for c, t, h, fi in zip(s["chunk"], s["to"], s["hop"], s["finish"]):
            fin_into[(int(c), int(t) if w.kind != cf.ALLTOALL else int(h) + 1)] = int(fi)
        by_link = {}
        for i in range(len(s["chunk"])):
            by_link.setdefault(int(s["link"][i]), []).append(i)
        for l, idx in by_link.items():
            idx.sort(key=lambda i: int(s["pos"][i]))
            src, dst = w.edges()[l]
            between = int(w.node_of[src]) != int(w.node_of[dst])
            groups = []
            for i in idx:
                key = (int(s["start"][i]), int(s["finish"][i]))
                if groups and groups[-1][0] == key:
                    groups[-1][1].append(i)
                else:
                    groups.append((key, [i]))
            prev_end = 0
            for (st, fi), members in groups:
                m = len(members)
                assert between or m == 1
                assert st >= prev_end
                prev_end = fi
                assert fi - st == cost(int(w.alpha_ns[l]), int(w.beta_ps_per_byte[l]), m * S)
                assert len({int(s["rem"][i]) for i in members}) == 1
                for i in members:
                    c = int(s["chunk"][i])
                    key = (c, int(s["from"][i])) if w.kind != cf.ALLTOALL else (c, int(s["hop"][i]))
                    ready = fin_into.get(key, 0)
                    assert ready <= st
                merged += m - 1
        assert mk == max(int(x) for x in s["finish"])
    assert merged > 0
