"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these tests needs a GPU. They check the oracle against values worked
out from the paper's constants, closed forms, brute force on tiny inputs and
invariants that hold for any candidate, so that a plausible mistake anywhere
in the oracle fails at least one of them.
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


def golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def two_rank(alpha, beta, chunk_bytes):
    row_ptr, col, a, b = cf.csr_from_edges(2, [(0, 1, alpha, beta), (1, 0, alpha, beta)])
    return cf.Workload("pair", 2, 2, row_ptr, col, a, b, None, cf.ALLGATHER, 1, chunk_bytes,
                       cf.KSHORTEST, k=1)


def gen_for(plan, w, first, count, seed=None):
    return generate(w.seed if seed is None else seed, first, count, plan.route_options(),
                    plan.prio_stride)


# ----------------------------------------------------------------------------
# alpha-beta cost (Sec. 4.1, Table 1)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("case", golden("link_costs.json")["cases"])
def test_link_cost_matches_table1_worked_values(case):
    plan = OraclePlan.from_workload(two_rank(case["alpha_ns"], case["beta_ps_per_byte"],
                                             case["chunk_bytes"]))
    assert plan.link_cost(0) == case["cost_ns"]
    assert plan.link_cost(1) == case["cost_ns"]


@pytest.mark.parametrize("name", cf.ORDER)
def test_named_workload_link_costs(name):
    want = golden("link_costs.json")["per_workload"][name]
    plan = OraclePlan.from_workload(cf.named(name))
    assert sorted(set(plan.link_costs().tolist())) == want


def test_sec41_coalescing_example():
    """Two 32 KB IB chunks sent as one 64 KB transfer save ~17% (Sec. 4.1)."""
    g = golden("alpha_beta_example.json")
    one = OraclePlan.from_workload(two_rank(g["alpha_ns"], g["beta_ps_per_byte"],
                                            g["chunk_bytes"])).link_cost(0)
    both = OraclePlan.from_workload(two_rank(g["alpha_ns"], g["beta_ps_per_byte"],
                                             2 * g["chunk_bytes"])).link_cost(0)
    saving = 1.0 - both / (2.0 * one)
    assert abs(saving - g["stated_saving"]) <= g["tolerance"]


# ----------------------------------------------------------------------------
# path tables
# ----------------------------------------------------------------------------

def oracle_table(plan, P):
    return {(s, d): plan.paths(s, d) for s in range(P) for d in range(P) if s != d}


@pytest.mark.parametrize("name,hop_limit", [("ring4_ag", 3), ("cubemesh8_ag", 7),
                                            ("twonode16_ag", 6)])
def test_kshortest_tables_equal_exhaustive_enumeration(name, hop_limit):
    w = cf.named(name)
    plan = OraclePlan.from_workload(w)
    cost = bf.costs_of(w)
    min_cost = min(cost)
    for s in range(w.P):
        for d in range(w.P):
            if s == d:
                continue
            ps, _ = bf.sorted_paths(w, s, d, hop_limit)
            if w.route_mode == cf.SHORTEST_ONLY:
                best = sum(cost[e] for e in ps[0][1])
                want = [links for _, links in ps if sum(cost[e] for e in links) == best][:w.k]
            else:
                want = [links for _, links in ps][:w.k]
            got = plan.paths(s, d)
            assert got == want, (s, d)
            # the hop limit cannot have cut a better path off
            kth = sum(cost[e] for e in got[-1])
            assert (hop_limit + 1) * min_cost > kth


def test_ring4_path_counts():
    """Neighbours on a 4-ring have one shortest path, opposite ranks two."""
    w = cf.ring4_ag()
    plan = OraclePlan.from_workload(w)
    for s in range(4):
        for d in range(4):
            if s != d:
                assert plan.npaths(s, d) == (2 if (s - d) % 4 == 2 else 1)


def test_relay1_table_structure():
    """switch16: option 0 is s->SW->d, then s->SW->m->SW->d for m ascending."""
    w = cf.switch16_a2a()
    plan = OraclePlan.from_workload(w)
    SW = w.P
    up = {r: w.link_id(r, SW) for r in range(w.P)}
    down = {r: w.link_id(SW, r) for r in range(w.P)}
    for s in range(w.P):
        for d in range(w.P):
            if s == d:
                continue
            want = [[up[s], down[d]]]
            want += [[up[s], down[m], up[m], down[d]] for m in range(w.P) if m not in (s, d)]
            assert plan.paths(s, d) == want


def test_hier_relay_table_structure():
    """fournode64: on-node chunks go through the switch; off-node chunk via
    relay index i goes s->SW->R_i, R_i->R'_i over IB, R'_i->SW'->d, skipping
    the local legs when s or d is the relay itself."""
    w = cf.fournode64_a2a()
    plan = OraclePlan.from_workload(w)
    per, P = 16, w.P

    def sw(r):
        return P + r // per

    def leg(a, b):
        if a == b:
            return []
        return [w.link_id(a, sw(a)), w.link_id(sw(a), b)]

    for s in range(P):
        for d in range(P):
            if s == d:
                continue
            if s // per == d // per:
                want = [leg(s, d)]
            else:
                want = []
                for i in range(8):
                    R, R2 = (s // per) * per + i, (d // per) * per + i
                    want.append(leg(s, R) + [w.link_id(R, R2)] + leg(R2, d))
            assert plan.paths(s, d) == want, (s, d)


# ----------------------------------------------------------------------------
# closed forms
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("P", [2, 3, 4, 5, 8, 13, 16, 32, 64])
def test_unidirectional_ring_allgather_closed_form(P):
    """A ring Allgather needs P-1 link steps per chunk (Sec. 2); with every
    link busy at every step the makespan is (P-1)(alpha + beta*S)."""
    w = cf.uni_ring_ag(P)
    plan = OraclePlan.from_workload(w)
    cost = plan.link_cost(0)
    routes, prio = gen_for(plan, w, 0, 8, seed=P)
    mk, ok = plan.eval(routes, prio)
    assert (mk == (P - 1) * cost).all()
    assert ok.all()
    # chunk c reaches rank c+j at exactly j link costs
    _, _, s = plan.eval_detail(routes[0], prio[0])
    for c, to, fin in zip(s["chunk"], s["to"], s["finish"]):
        assert fin == ((to - c) % P) * cost


def test_unidirectional_ring4_value():
    w = cf.uni_ring_ag(4)
    plan = OraclePlan.from_workload(w)
    routes, prio = gen_for(plan, w, 0, 4)
    mk, ok = plan.eval(routes, prio)
    assert (mk == 146805).all() and ok.all()


def test_ring4_every_candidate_is_two_link_costs():
    """On the 4-ring with minimal routes each directed link carries its own
    chunk plus at most one relayed chunk; the own chunk wins (longer
    remaining path, or shorter travelled one) so every candidate finishes
    in exactly two link costs, which is also the distance lower bound."""
    w = cf.ring4_ag()
    plan = OraclePlan.from_workload(w)
    routes, prio = gen_for(plan, w, 0, w.n_candidates)
    mk, ok = plan.eval(routes, prio)
    assert (mk == 97870).all() and ok.all()


def test_single_send():
    w = two_rank(700, 46, 1 << 20)
    plan = OraclePlan.from_workload(w)
    routes, prio = gen_for(plan, w, 0, 3)
    mk, ok = plan.eval(routes, prio)
    assert (mk == 48935).all() and ok.all()


def test_star_alltoall_uplink_serialises():
    """Every chunk through one switch: the makespan is at least P link costs
    (P-1 sends queue on each uplink, then one downlink hop) and at most the
    sum of all send costs."""
    P = 6
    row_ptr, col, a, b = cf.csr_from_edges(P + 1, cf.switch_edges(range(P), P, 700, 8))
    w = cf.Workload("star", P + 1, P, row_ptr, col, a, b, None, cf.ALLTOALL, 1, 1 << 16,
                    cf.KSHORTEST, k=1)
    plan = OraclePlan.from_workload(w)
    c = plan.link_cost(0)
    routes, prio = gen_for(plan, w, 0, 32, seed=9)
    mk, ok = plan.eval(routes, prio)
    assert ok.all()
    assert (mk >= P * c).all()
    assert (mk <= 2 * P * (P - 1) * c).all()


# ----------------------------------------------------------------------------
# brute force on tiny inputs
# ----------------------------------------------------------------------------

def bf_table(w, hop_limit):
    table = {}
    cost = bf.costs_of(w)
    for s in range(w.P):
        for d in range(w.P):
            if s == d:
                continue
            if w.route_mode == cf.RELAY1:
                best = bf.sorted_paths(w, s, d, hop_limit)[0][0][1]
                opts = [best]
                for m in range(w.P):
                    if m in (s, d):
                        continue
                    a_ = bf.sorted_paths(w, s, m, hop_limit)[0][0][1]
                    b_ = bf.sorted_paths(w, m, d, hop_limit)[0][0][1]
                    opts.append(a_ + b_)
                table[(s, d)] = opts
            else:
                ps, _ = bf.sorted_paths(w, s, d, hop_limit)
                if w.route_mode == cf.SHORTEST_ONLY:
                    best = sum(cost[e] for e in ps[0][1])
                    ps = [p for p in ps if sum(cost[e] for e in p[1]) == best]
                table[(s, d)] = [links for _, links in ps][:w.k]
    return table


def compare_detail(w, plan, table, routes, prio):
    mk, ok, s = plan.eval_detail(routes, prio)
    bmk, bok, bsends, bstart, bfinish, orders = bf.evaluate(w, table, routes, prio,
                                                            H=plan.max_hops)
    assert (mk, ok) == (bmk, bok)
    assert len(s["chunk"]) == len(bsends)
    got = {(int(c), int(l)): (int(r), int(t), int(st), int(fi), int(po))
           for c, l, r, t, st, fi, po in zip(s["chunk"], s["link"], s["rem"], s["trav"],
                                             s["start"], s["finish"], s["pos"])}
    for i, b in enumerate(bsends):
        pos = orders[b["link"]].index(i)
        assert got[(b["chunk"], b["link"])] == (b["rem"], b["trav"], bstart[i], bfinish[i], pos)
    return mk, ok, bsends


def test_bruteforce_ring4_all_routings():
    """All 16 routings of the 4-ring Allgather, several priority draws each."""
    w = cf.ring4_ag()
    plan = OraclePlan.from_workload(w)
    table = bf_table(w, 3)
    opts = plan.route_options()
    multi = [e for e in range(len(opts)) if opts[e] == 2]
    _, prio = gen_for(plan, w, 0, 4)
    for bits in range(1 << len(multi)):
        routes = np.zeros(plan.route_stride, dtype=np.uint8)
        for j, e in enumerate(multi):
            routes[e] = (bits >> j) & 1
        for p in prio:
            compare_detail(w, plan, table, routes, p)


def test_bruteforce_full4_allgather():
    """Fully connected 4 ranks, Allgather, 3 shortest paths per pair: the
    multicast tree merge is exercised (relayed paths overlap)."""
    w = cf.full_ag(4, k=3, chunks_per_rank=2)
    plan = OraclePlan.from_workload(w)
    table = bf_table(w, 3)
    routes, prio = gen_for(plan, w, 0, 60, seed=11)
    for r, p in zip(routes, prio):
        compare_detail(w, plan, table, r, p)


def test_bruteforce_full4_alltoall_all_routings():
    """Fully connected 4 ranks, Alltoall, direct or one relay: all 3^12
    routings are too many for pure Python, so every routing of the chunks of
    two sources is enumerated with the rest fixed, plus seeded samples."""
    w = cf.full_a2a(4)
    plan = OraclePlan.from_workload(w)
    table = bf_table(w, 3)
    routes, prio = gen_for(plan, w, 0, 40, seed=12)
    for r, p in zip(routes, prio):
        compare_detail(w, plan, table, r, p)
    base = routes[0].copy()
    chunks = [c for c in range(16) if c // 4 in (0, 1) and c // 4 != c % 4]
    for combo in range(3 ** len(chunks)):
        r = base.copy()
        x = combo
        for c in chunks:
            r[c] = x % 3
            x //= 3
        if combo % 7 == 0:  # keep the pure-Python run short
            compare_detail(w, plan, table, r, prio[combo % len(prio)])


def test_bruteforce_explicit_multicast():
    """Explicit pre/postcondition (App. B): chunks reach a subset of ranks."""
    base = cf.full_ag(5, k=3)
    owner = [0, 1, 2, 3, 4, 0]
    posts = [[1, 3], [0, 2, 4], [2], [0, 1, 2, 4], [1, 2, 3], [4]]
    w = cf.explicit_multicast(base, owner, posts)
    plan = OraclePlan.from_workload(w)
    table = bf_table(w, 3)
    routes, prio = gen_for(plan, w, 0, 40, seed=13)
    for r, p in zip(routes, prio):
        compare_detail(w, plan, table, r, p)


def test_heuristic_never_beats_the_exhaustive_optimum():
    """The heuristic order is one of all per-link orders, so its makespan is
    at least the optimum over all of them; on the 4-ring it is optimal."""
    w = cf.ring4_ag()
    plan = OraclePlan.from_workload(w)
    table = bf_table(w, 3)
    routes, prio = gen_for(plan, w, 0, 6)
    for r, p in zip(routes, prio):
        mk, _, sends, _, _, _ = bf.evaluate(w, table, r, p)
        assert bf.optimum_over_orders(w, sends) == mk
    w = cf.full_a2a(3)
    plan = OraclePlan.from_workload(w)
    table = bf_table(w, 2)
    routes, prio = gen_for(plan, w, 0, 6, seed=3)
    for r, p in zip(routes, prio):
        mk, _, sends, _, _, _ = bf.evaluate(w, table, r, p, H=plan.max_hops)
        assert plan.eval(r[None], p[None])[0][0] == mk
        assert bf.optimum_over_orders(w, sends) <= mk


# ----------------------------------------------------------------------------
# unrouted pairs and the postcondition
# ----------------------------------------------------------------------------

def test_unrouted_alltoall_pair_is_invalid():
    w = cf.switch16_a2a()
    plan = OraclePlan.from_workload(w)
    routes, prio = gen_for(plan, w, 0, 2)
    r = routes[0].copy()
    r[1] = 255  # chunk 0 -> 1 left unrouted
    mk, ok = plan.eval(np.stack([routes[0], r]), prio[[0, 0]])
    assert ok.tolist() == [1, 0]


def test_unrouted_allgather_pair_reached_through_another_path():
    """Allgather: a pair without a route still holds if another destination's
    path passes through its rank."""
    w = cf.uni_ring_ag(5)
    plan = OraclePlan.from_workload(w)
    routes, prio = gen_for(plan, w, 0, 1)
    r = routes[0].copy()
    r[0 * 5 + 2] = 255  # chunk 0 to rank 2 unrouted, but 0->1->2->3 reaches it
    mk, ok = plan.eval(r[None], prio)
    assert ok[0] == 1 and mk[0] == 4 * plan.link_cost(0)
    r[0 * 5 + 4] = 255  # now nobody routes chunk 0 to rank 4
    mk, ok = plan.eval(r[None], prio)
    assert ok[0] == 0 and mk[0] == 4 * plan.link_cost(0)


def test_all_unrouted_gives_zero_makespan():
    w = cf.full_a2a(4)
    plan = OraclePlan.from_workload(w)
    r = np.full(plan.route_stride, 255, dtype=np.uint8)
    p = np.zeros(plan.prio_stride, dtype=np.uint32)
    mk, ok = plan.eval(r[None], p[None])
    assert mk[0] == 0 and ok[0] == 0


# ----------------------------------------------------------------------------
# invariants on the named workloads
# ----------------------------------------------------------------------------

CUT_BOUNDS = {
    # 16 chunks must cross 4 IB links per direction: one link carries >= 4
    "twonode16_ag": 4 * 112850,
    # 256 chunks per node pair over 8 IB links: one link carries >= 32
    "fournode64_a2a": 32 * 8647,
    # each uplink carries its rank's 15 chunks
    "switch16_a2a": 15 * 2798,
    # diameter 2: some chunk needs two hops
    "cubemesh8_ag": 2 * 193638,
    "ring4_ag": 2 * 48935,
}


def dijkstra_all(w, cost):
    import heapq
    dist = {}
    for s in range(w.P):
        d = {s: 0}
        pq = [(0, s)]
        while pq:
            t, u = heapq.heappop(pq)
            if t > d.get(u, 1 << 62):
                continue
            for e, v in bf.out_links(w, u):
                nt = t + cost[e]
                if nt < d.get(v, 1 << 62):
                    d[v] = nt
                    heapq.heappush(pq, (nt, v))
        dist[s] = d
    return dist


@pytest.mark.parametrize("name,count", [("ring4_ag", 64), ("cubemesh8_ag", 64),
                                        ("switch16_a2a", 24), ("twonode16_ag", 24),
                                        ("fournode64_a2a", 3)])
def test_invariants_on_named_workloads(name, count):
    w = cf.named(name)
    plan = OraclePlan.from_workload(w)
    cost = bf.costs_of(w)
    dist = dijkstra_all(w, cost)
    routes, prio = gen_for(plan, w, 0, count)
    mk, ok = plan.eval(routes, prio)
    for i in range(count):
        m, v, s = plan.eval_detail(routes[i], prio[i])
        assert (m, v) == (mk[i], ok[i])
        assert v == 1  # the generator only draws valid route choices
        n = len(s["chunk"])
        # exactly-once delivery: one incoming send per (chunk, vertex)
        if w.kind != cf.ALLTOALL:
            assert len(set(zip(s["chunk"].tolist(), s["to"].tolist()))) == n
            if w.V == w.P:
                assert n == plan.num_chunks * (w.P - 1)
        # lower bounds: link load and distance (Step-1 relaxation, App. B.1)
        load = {}
        for l in s["link"].tolist():
            load[l] = load.get(l, 0) + cost[l]
        assert m >= max(load.values())
        assert m >= CUT_BOUNDS[name]
        if w.kind == cf.ALLTOALL:
            for c in set(s["chunk"].tolist()):
                src, dst = (c // w.P), (c % w.P)
                assert m >= dist[src][dst]
        else:
            for c in range(plan.num_chunks):
                o = c // w.chunks_per_rank
                assert m >= max(dist[o][r] for r in range(w.P))
        # upper bound and schedule validity
        assert m <= sum(cost[l] for l in s["link"].tolist())
        assert m == int(s["finish"].max())
        for l in set(s["link"].tolist()):
            idx = np.where(s["link"] == l)[0]
            order = idx[np.argsort(s["pos"][idx])]
            for a_, b_ in zip(order[:-1], order[1:]):
                assert s["start"][b_] >= s["finish"][a_]
                key_a = (-int(s["rem"][a_]), int(s["trav"][a_]), int(s["prio"][a_]),
                         int(s["chunk"][a_]))
                key_b = (-int(s["rem"][b_]), int(s["trav"][b_]), int(s["prio"][b_]),
                         int(s["chunk"][b_]))
                assert key_a < key_b


# ----------------------------------------------------------------------------
# tie-breaks and sketch rules that the named workloads never exercise
# ----------------------------------------------------------------------------

def test_equal_priorities_fall_back_to_chunk_order():
    """With every priority equal, the last tie-break (chunk id) decides."""
    for w, hop in ((cf.full_ag(4, k=3, chunks_per_rank=2), 3), (cf.full_a2a(4), 3)):
        plan = OraclePlan.from_workload(w)
        table = bf_table(w, hop)
        routes, _ = gen_for(plan, w, 0, 30, seed=21)
        for value in (0, 7, 0xFFFFFFFF):
            p = np.full(plan.prio_stride, value, dtype=np.uint32)
            for r in routes:
                compare_detail(w, plan, table, r, p)


def test_path_order_breaks_cost_ties_by_hops_then_vertices():
    """Equal-cost paths with different hop counts: fewer hops first; equal
    cost and hops: lexicographically smaller vertex sequence first."""
    edges = [(0, 1, 100, 0), (1, 2, 100, 0), (0, 2, 200, 0), (0, 3, 50, 0), (3, 2, 150, 0),
             (1, 0, 100, 0), (2, 1, 100, 0), (2, 0, 200, 0), (3, 0, 50, 0), (2, 3, 150, 0)]
    row_ptr, col, a, b = cf.csr_from_edges(4, edges)
    w = cf.Workload("ties", 4, 4, row_ptr, col, a, b, None, cf.ALLGATHER, 1, 1000, cf.KSHORTEST,
                    k=3)
    plan = OraclePlan.from_workload(w)
    got = plan.paths(0, 2)
    assert got == [[w.link_id(0, 2)], [w.link_id(0, 1), w.link_id(1, 2)],
                   [w.link_id(0, 3), w.link_id(3, 2)]]
    for s in range(4):
        for d in range(4):
            if s != d:
                ps, _ = bf.sorted_paths(w, s, d, 3)
                assert plan.paths(s, d) == [links for _, links in ps][:3]


def test_crossings_only_between_relays():
    """A link between nodes that does not join two relays is never used
    (App. A internode relay sketch), even when it would be shorter."""
    base = cf.twonode16_ag()
    edges = [(u, v, int(base.alpha_ns[e]), int(base.beta_ps_per_byte[e]))
             for e, (u, v) in enumerate(base.edges())]
    edges += [(1, 9, 1700, 106), (9, 1, 1700, 106)]
    row_ptr, col, a, b = cf.csr_from_edges(16, edges)
    w = cf.Workload("twonode16_extra", 16, 16, row_ptr, col, a, b, base.node_of, cf.ALLGATHER, 2,
                    base.chunk_bytes, cf.KSHORTEST, k=4, max_cross=1, relay=base.relay)
    plan = OraclePlan.from_workload(w)
    bad = {w.link_id(1, 9), w.link_id(9, 1)}
    for s in range(16):
        for d in range(16):
            if s != d:
                got = plan.paths(s, d)
                assert not any(set(p) & bad for p in got)
                ps, _ = bf.sorted_paths(w, s, d, 6)
                assert got == [links for _, links in ps][:4]
    # without the relay rule the extra link is taken
    w2 = cf.Workload("twonode16_extra_norelay", 16, 16, row_ptr, col, a, b, base.node_of,
                     cf.ALLGATHER, 2, base.chunk_bytes, cf.KSHORTEST, k=4, max_cross=1)
    plan2 = OraclePlan.from_workload(w2)
    assert plan2.paths(1, 9)[0] == [w.link_id(1, 9)]
