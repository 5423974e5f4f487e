"""Synthetic workload descriptors: topologies, collectives and sketches.

Shared input code for the oracle and the GPU evaluator. A descriptor is
plain data (a CSR link list with per-link alpha/beta, the collective, the
sketch knobs, the batch size and seed); it holds none of the evaluation's
arithmetic, which each side implements on its own.

The five named workloads stand in for the paper's sketches (the paper
measured on DGX-2 and NDv2 clusters; none of that hardware is needed here):
  ring4_ag        4-rank bidirectional ring, Allgather (closed-form case)
  cubemesh8_ag    one NDv2-like node: the hybrid cube-mesh NVLink graph of
                  Sec. 4 (two fully connected quads plus i<->i+4), Allgather
  switch16_a2a    one DGX-2-like node: 16 ranks behind one switch, Alltoall
                  with an optional one-hop relay
  twonode16_ag    two cube-mesh nodes joined by IB links between relay GPUs
                  (the ndv2 relay sketch of Sec. 3.1, Example 2), Allgather
  fournode64_a2a  four 16-rank switch nodes, NIC relays per local index
                  (the dgx2 relay sketch of App. A), Alltoall
alpha/beta come from Table 1 (NVLink 0.7 us with 46 or 8 us/MB, IB 1.7 us
with 106 us/MB); us/MB equals ps/B with MB = 10^6 B.
"""
from dataclasses import dataclass, field, replace
from typing import Optional

import numpy as np

ALLGATHER, ALLTOALL, EXPLICIT, REDUCESCATTER, ALLREDUCE = 0, 1, 2, 3, 4
SHORTEST_ONLY, KSHORTEST, RELAY1, HIER_RELAY = 0, 1, 2, 3

KIB = 1024
MIB = 1024 * 1024

# Table 1 (ns, ps/B)
NVLINK_ALPHA = 700
NDV2_NVLINK_BETA = 46
DGX2_NVLINK_BETA = 8
IB_ALPHA = 1700
IB_BETA = 106


@dataclass
class Workload:
    name: str
    V: int
    P: int
    row_ptr: np.ndarray
    col: np.ndarray
    alpha_ns: np.ndarray
    beta_ps_per_byte: np.ndarray
    node_of: Optional[np.ndarray]
    kind: int
    chunks_per_rank: int
    chunk_bytes: int
    route_mode: int
    k: int = 1
    max_cross: int = -1
    allowed: Optional[np.ndarray] = None
    relay: Optional[np.ndarray] = None
    owner: Optional[np.ndarray] = None
    post_ptr: Optional[np.ndarray] = None
    post: Optional[np.ndarray] = None
    n_candidates: int = 1
    seed: int = 0
    description: str = ""
    extra: dict = field(default_factory=dict)
    # 1: merge ready sends of equal remaining length into contiguous
    # transfers on links between nodes
    contiguity: int = 0
    # 0: static Step-2 link orders; 1: time-aware greedy orders
    order: int = 0
    # 1: Alltoall hop pairs through a switch vertex are one send holding the
    # sender's send port and the receiver's receive port
    switch_ports: int = 0

    @property
    def E(self):
        return int(self.row_ptr[-1])

    def edges(self):
        """(src, dst) of every link, in link-id order."""
        src = np.repeat(np.arange(self.V), np.diff(self.row_ptr))
        return list(zip(src.tolist(), self.col.tolist()))

    def link_id(self, u, v):
        for e in range(int(self.row_ptr[u]), int(self.row_ptr[u + 1])):
            if int(self.col[e]) == v:
                return e
        raise KeyError((u, v))


def csr_from_edges(V, edges):
    """edges: iterable of (u, v, alpha_ns, beta_ps_per_byte). Links are
    numbered in (u, v) order; duplicate links are rejected."""
    edges = sorted(edges)
    seen = set()
    for u, v, _, _ in edges:
        if (u, v) in seen:
            raise ValueError(f"duplicate link {u}->{v}")
        if not (0 <= u < V and 0 <= v < V) or u == v:
            raise ValueError(f"bad link {u}->{v}")
        seen.add((u, v))
    row_ptr = np.zeros(V + 1, dtype=np.int32)
    for u, _, _, _ in edges:
        row_ptr[u + 1] += 1
    row_ptr = np.cumsum(row_ptr).astype(np.int32)
    col = np.array([v for _, v, _, _ in edges], dtype=np.int32)
    alpha = np.array([a for _, _, a, _ in edges], dtype=np.uint32)
    beta = np.array([b for _, _, _, b in edges], dtype=np.uint32)
    return row_ptr, col, alpha, beta


# --------------------------------------------------------------------------
# topology pieces
# --------------------------------------------------------------------------

def ring_edges(ranks, alpha, beta, bidirectional=True):
    n = len(ranks)
    out = []
    for i in range(n):
        out.append((ranks[i], ranks[(i + 1) % n], alpha, beta))
        if bidirectional and n > 2:
            out.append((ranks[i], ranks[(i - 1) % n], alpha, beta))
    return out


def cube_mesh_edges(base, alpha, beta):
    """Hybrid cube-mesh of 8 ranks: quads {0..3} and {4..7} fully connected,
    plus i <-> i+4 (the NDv2 / DGX-1 NVLink graph)."""
    out = []
    for quad in ((0, 1, 2, 3), (4, 5, 6, 7)):
        for a in quad:
            for b in quad:
                if a != b:
                    out.append((base + a, base + b, alpha, beta))
    for i in range(4):
        out.append((base + i, base + i + 4, alpha, beta))
        out.append((base + i + 4, base + i, alpha, beta))
    return out


def switch_edges(ranks, sw, alpha, beta):
    """A store-and-forward switch vertex: one uplink and one downlink per rank."""
    out = []
    for r in ranks:
        out.append((r, sw, alpha, beta))
        out.append((sw, r, alpha, beta))
    return out


# --------------------------------------------------------------------------
# the five named workloads
# --------------------------------------------------------------------------

def ring4_ag(n_candidates=256, seed=1):
    V = P = 4
    row_ptr, col, a, b = csr_from_edges(V, ring_edges(list(range(4)), NVLINK_ALPHA,
                                                      NDV2_NVLINK_BETA))
    return Workload("ring4_ag", V, P, row_ptr, col, a, b, None, ALLGATHER, 1, 1 * MIB,
                    SHORTEST_ONLY, k=2, n_candidates=n_candidates, seed=seed,
                    description="4-rank bidirectional ring, Allgather, 1 MiB chunks, "
                                "<=2 minimal-cost paths per pair")


def cubemesh8_ag(n_candidates=4096, seed=2):
    V = P = 8
    row_ptr, col, a, b = csr_from_edges(V, cube_mesh_edges(0, NVLINK_ALPHA, NDV2_NVLINK_BETA))
    return Workload("cubemesh8_ag", V, P, row_ptr, col, a, b, None, ALLGATHER, 1, 4 * MIB,
                    KSHORTEST, k=4, n_candidates=n_candidates, seed=seed,
                    description="8-rank hybrid cube-mesh, Allgather, 4 MiB chunks, "
                                "k=4 shortest paths")


def switch16_a2a(n_candidates=16384, seed=3):
    P = 16
    V = P + 1
    row_ptr, col, a, b = csr_from_edges(V, switch_edges(range(P), P, NVLINK_ALPHA,
                                                        DGX2_NVLINK_BETA))
    return Workload("switch16_a2a", V, P, row_ptr, col, a, b, None, ALLTOALL, 1, 256 * KIB,
                    RELAY1, n_candidates=n_candidates, seed=seed,
                    description="16 ranks behind one switch, Alltoall, 256 KiB chunks, "
                                "direct or one-hop relay")


def twonode16_ag(n_candidates=65536, seed=4):
    P = V = 16
    edges = cube_mesh_edges(0, NVLINK_ALPHA, NDV2_NVLINK_BETA)
    edges += cube_mesh_edges(8, NVLINK_ALPHA, NDV2_NVLINK_BETA)
    for s in (0, 4):
        for d in (8, 12):
            edges.append((s, d, IB_ALPHA, IB_BETA))
            edges.append((d, s, IB_ALPHA, IB_BETA))
    row_ptr, col, a, b = csr_from_edges(V, edges)
    node_of = np.array([r // 8 for r in range(V)], dtype=np.int32)
    relay = np.zeros(V, dtype=np.uint8)
    relay[[0, 4, 8, 12]] = 1
    return Workload("twonode16_ag", V, P, row_ptr, col, a, b, node_of, ALLGATHER, 2, 1 * MIB,
                    KSHORTEST, k=4, max_cross=1, relay=relay, n_candidates=n_candidates,
                    seed=seed,
                    description="2 nodes x 8-rank cube-mesh, IB between relays {0,4} and "
                                "{8,12}, Allgather, 2 x 1 MiB chunks per rank, k=4 "
                                "sketch-valid shortest paths")


def fournode64_a2a(n_candidates=8192, seed=5):
    nodes, per = 4, 16
    P = nodes * per
    V = P + nodes
    edges = []
    for n in range(nodes):
        edges += switch_edges(range(n * per, (n + 1) * per), P + n, NVLINK_ALPHA,
                              DGX2_NVLINK_BETA)
    for A in range(nodes):
        for B in range(nodes):
            if A != B:
                for i in range(8):
                    edges.append((A * per + i, B * per + i, IB_ALPHA, IB_BETA))
    row_ptr, col, a, b = csr_from_edges(V, edges)
    node_of = np.array([r // per for r in range(P)] + list(range(nodes)), dtype=np.int32)
    relay = np.zeros(V, dtype=np.uint8)
    for n in range(nodes):
        relay[n * per:n * per + 8] = 1
    return Workload("fournode64_a2a", V, P, row_ptr, col, a, b, node_of, ALLTOALL, 1, 64 * KIB,
                    HIER_RELAY, max_cross=1, relay=relay, n_candidates=n_candidates, seed=seed,
                    description="4 nodes x 16 ranks behind a switch per node, local relay i "
                                "-> remote relay i over IB, Alltoall, 64 KiB chunks")


NAMED = {
    "ring4_ag": ring4_ag,
    "cubemesh8_ag": cubemesh8_ag,
    "switch16_a2a": switch16_a2a,
    "twonode16_ag": twonode16_ag,
    "fournode64_a2a": fournode64_a2a,
}
ORDER = ["ring4_ag", "cubemesh8_ag", "switch16_a2a", "twonode16_ag", "fournode64_a2a"]


def with_contiguity(w):
    """The same workload with contiguous transfers on links between nodes."""
    return replace(w, name=w.name + "_contig", contiguity=1,
                   description=w.description + "; contiguous transfers on IB links")


NAMED["twonode16_ag_contig"] = lambda **kw: with_contiguity(twonode16_ag(**kw))
NAMED["fournode64_a2a_contig"] = lambda **kw: with_contiguity(fournode64_a2a(**kw))
CONTIG_ORDER = ["twonode16_ag_contig", "fournode64_a2a_contig"]


def as_reduction(w, kind):
    """The same topology, sketch and trees as an Allgather workload, as
    ReduceScatter (the trees run backwards) or Allreduce (ReduceScatter then
    Allgather)."""
    suffix = {REDUCESCATTER: "_rs", ALLREDUCE: "_ar"}[kind]
    base = w.name[:-3] if w.name.endswith("_ag") else w.name
    what = {REDUCESCATTER: "ReduceScatter", ALLREDUCE: "Allreduce"}[kind]
    return replace(w, name=base + suffix, kind=kind,
                   description=w.description.replace("Allgather", what))


NAMED["cubemesh8_ar"] = lambda **kw: as_reduction(cubemesh8_ag(**kw), ALLREDUCE)
NAMED["twonode16_rs"] = lambda **kw: as_reduction(twonode16_ag(**kw), REDUCESCATTER)
NAMED["twonode16_ar"] = lambda **kw: as_reduction(twonode16_ag(**kw), ALLREDUCE)
REDUCE_ORDER = ["cubemesh8_ar", "twonode16_rs", "twonode16_ar"]


def with_greedy(w):
    """The same workload with link orders from the time-aware greedy."""
    return replace(w, name=w.name + "_greedy", order=1,
                   description=w.description + "; time-aware greedy link orders")


def with_reverse_greedy(w):
    """The same workload with time-aware greedy orders in reverse path order."""
    return replace(w, name=w.name + "_rgreedy", order=2,
                   description=w.description + "; time-aware greedy in reverse path order")


NAMED["twonode16_ag_greedy"] = lambda **kw: with_greedy(twonode16_ag(**kw))
NAMED["cubemesh8_ag_greedy"] = lambda **kw: with_greedy(cubemesh8_ag(**kw))
NAMED["switch16_a2a_greedy"] = lambda **kw: with_greedy(switch16_a2a(**kw))
NAMED["fournode64_a2a_greedy"] = lambda **kw: with_greedy(fournode64_a2a(**kw))
NAMED["twonode16_ag_rgreedy"] = lambda **kw: with_reverse_greedy(twonode16_ag(**kw))
GREEDY_ORDER = ["cubemesh8_ag_greedy", "twonode16_ag_greedy", "switch16_a2a_greedy",
                "twonode16_ag_rgreedy"]
# timed by the benchmark; the oracle needs about a second per candidate, so
# parity tests sample them
GREEDY_LARGE_ORDER = ["fournode64_a2a_greedy"]


def with_switch_ports(w):
    """The same workload with the switch-port model."""
    return replace(w, name=w.name + "_ports", switch_ports=1,
                   description=w.description + "; switched sends hold send and receive ports")


NAMED["switch16_a2a_ports"] = lambda **kw: with_switch_ports(switch16_a2a(**kw))
NAMED["fournode64_a2a_ports"] = lambda **kw: with_switch_ports(fournode64_a2a(**kw))
PORTS_ORDER = ["switch16_a2a_ports", "fournode64_a2a_ports"]


def named(name, **kw):
    return NAMED[name](**kw)


# --------------------------------------------------------------------------
# small parametric workloads for tests
# --------------------------------------------------------------------------

def uni_ring_ag(P, chunk_bytes=1 * MIB, alpha=NVLINK_ALPHA, beta=NDV2_NVLINK_BETA,
                n_candidates=1, seed=0):
    """Unidirectional ring r -> r+1: every pair has exactly one path."""
    row_ptr, col, a, b = csr_from_edges(P, ring_edges(list(range(P)), alpha, beta,
                                                      bidirectional=False))
    return Workload(f"uniring{P}_ag", P, P, row_ptr, col, a, b, None, ALLGATHER, 1, chunk_bytes,
                    KSHORTEST, k=1, n_candidates=n_candidates, seed=seed)


def full_a2a(P, chunk_bytes=1 * MIB, alpha=NVLINK_ALPHA, beta=NDV2_NVLINK_BETA, n_candidates=1,
             seed=0):
    """Fully connected P ranks, Alltoall, direct path or one relay rank."""
    edges = [(u, v, alpha, beta) for u in range(P) for v in range(P) if u != v]
    row_ptr, col, a, b = csr_from_edges(P, edges)
    return Workload(f"full{P}_a2a", P, P, row_ptr, col, a, b, None, ALLTOALL, 1, chunk_bytes,
                    RELAY1, n_candidates=n_candidates, seed=seed)


def full_ag(P, chunk_bytes=1 * MIB, alpha=NVLINK_ALPHA, beta=NDV2_NVLINK_BETA, k=3,
            chunks_per_rank=1, n_candidates=1, seed=0):
    """Fully connected P ranks, Allgather, k shortest paths."""
    edges = [(u, v, alpha, beta) for u in range(P) for v in range(P) if u != v]
    row_ptr, col, a, b = csr_from_edges(P, edges)
    return Workload(f"full{P}_ag", P, P, row_ptr, col, a, b, None, ALLGATHER, chunks_per_rank,
                    chunk_bytes, KSHORTEST, k=k, n_candidates=n_candidates, seed=seed)


def explicit_multicast(base, owner, posts, n_candidates=1, seed=0):
    """Same topology and sketch as `base`, explicit pre/postcondition: chunk c
    starts at owner[c] and must reach every rank in posts[c]."""
    post_ptr = np.zeros(len(owner) + 1, dtype=np.int32)
    for c, ps in enumerate(posts):
        post_ptr[c + 1] = post_ptr[c] + len(ps)
    post = np.array([r for ps in posts for r in ps], dtype=np.int32)
    w = Workload(base.name + "_explicit", base.V, base.P, base.row_ptr, base.col, base.alpha_ns,
                 base.beta_ps_per_byte, base.node_of, EXPLICIT, 1, base.chunk_bytes,
                 base.route_mode, k=base.k, max_cross=base.max_cross, allowed=base.allowed,
                 relay=base.relay, owner=np.asarray(owner, dtype=np.int32), post_ptr=post_ptr,
                 post=post, n_candidates=n_candidates, seed=seed)
    return w


def two_node_full(P_per, kind, chunks_per_rank=1, k=3, chunk_bytes=64 * KIB, contiguity=1):
    """Two nodes of P_per fully connected ranks (NVLink inside a node), IB
    between rank i of one node and rank i of the other, both directions.
    Allgather: k shortest paths; Alltoall: hierarchical relays."""
    P = 2 * P_per
    edges = []
    for n in range(2):
        for u in range(P_per):
            for v in range(P_per):
                if u != v:
                    edges.append((n * P_per + u, n * P_per + v, NVLINK_ALPHA, NDV2_NVLINK_BETA))
    for i in range(P_per):
        edges.append((i, P_per + i, IB_ALPHA, IB_BETA))
        edges.append((P_per + i, i, IB_ALPHA, IB_BETA))
    row_ptr, col, a, b = csr_from_edges(P, edges)
    node_of = np.array([r // P_per for r in range(P)], dtype=np.int32)
    if kind == ALLGATHER:
        return Workload(f"twonode{P}_full_ag", P, P, row_ptr, col, a, b, node_of, ALLGATHER,
                        chunks_per_rank, chunk_bytes, KSHORTEST, k=k, contiguity=contiguity)
    relay = np.ones(P, dtype=np.uint8)
    return Workload(f"twonode{P}_full_a2a", P, P, row_ptr, col, a, b, node_of, ALLTOALL,
                    chunks_per_rank, chunk_bytes, HIER_RELAY, max_cross=1, relay=relay,
                    contiguity=contiguity)


def two_node_rings_a2a(P_per, chunk_bytes=64 * KIB, contiguity=1):
    """Two nodes whose ranks form a one-way ring, IB between rank i of one
    node and rank i of the other: Alltoall paths run up to 2*P_per - 1 links."""
    P = 2 * P_per
    edges = []
    for n in range(2):
        for u in range(P_per):
            edges.append((n * P_per + u, n * P_per + (u + 1) % P_per, NVLINK_ALPHA,
                          NDV2_NVLINK_BETA))
    for i in range(P_per):
        edges.append((i, P_per + i, IB_ALPHA, IB_BETA))
        edges.append((P_per + i, i, IB_ALPHA, IB_BETA))
    row_ptr, col, a, b = csr_from_edges(P, edges)
    node_of = np.array([r // P_per for r in range(P)], dtype=np.int32)
    return Workload(f"tworings{P}_a2a", P, P, row_ptr, col, a, b, node_of, ALLTOALL, 1,
                    chunk_bytes, KSHORTEST, k=2, max_cross=1, contiguity=contiguity)


def random_workload(seed):
    """A seeded random small plan for parity sweeps: a bidirectional ring of
    3..16 ranks with random extra link pairs, alpha/beta drawn either from
    Table 1's values or from wide uniform ranges, half the time a switch
    vertex linked to most ranks, sometimes two nodes joined
    only between relay ranks; any collective kind (explicit ones with random
    owners and postconditions), a random route mode and k, and one of static
    orders, greedy orders in path or reverse path order, contiguous transfers
    (two nodes) or switch ports (Alltoall with a switch). Some draws give plans a route search refuses
    (a relay route through one link twice); callers skip those."""
    rng = np.random.default_rng(seed)
    kind = int(rng.choice([ALLGATHER, ALLTOALL, REDUCESCATTER, ALLREDUCE, EXPLICIT]))
    P = int(rng.integers(3, 13)) if rng.random() < 0.5 else int(rng.choice([4, 8, 12, 16]))
    switch = bool(rng.random() < 0.5)
    two_nodes = bool(rng.random() < 0.35) and P >= 4
    V = P + (1 if switch else 0)
    table1 = bool(rng.random() < 0.5)  # only Table 1's link parameters
    links = {}

    def add(u, v):
        if u != v and (u, v) not in links:
            if table1:
                links[(u, v)] = (int(rng.choice([NVLINK_ALPHA, IB_ALPHA])),
                                 int(rng.choice([DGX2_NVLINK_BETA, NDV2_NVLINK_BETA, IB_BETA])))
            else:
                links[(u, v)] = (int(rng.integers(100, 2000)), int(rng.integers(1, 120)))

    for i in range(P):
        add(i, (i + 1) % P)
        add((i + 1) % P, i)
    for _ in range(int(rng.integers(0, 2 * P))):
        u, v = (int(x) for x in rng.integers(0, P, 2))
        add(u, v)
        add(v, u)
    if switch:
        for r in range(P):
            if rng.random() < 0.8:
                add(r, P)
                add(P, r)
    node_of = relay = None
    max_cross = -1
    if two_nodes:
        half = P // 2
        node_of = np.array([0 if r < half else 1 for r in range(P)] + [0] * (V - P),
                           dtype=np.int32)
        relay = np.zeros(V, dtype=np.uint8)
        relay[[0, half - 1, half, P - 1]] = 1
        # links between the nodes only join relay ranks (the ring's crossing
        # links 0 <-> P-1 and half-1 <-> half do); the switch is node 0's
        links = {(u, v): ab for (u, v), ab in links.items()
                 if node_of[u] == node_of[v] or (relay[u] and relay[v] and u < P and v < P)}
        max_cross = 1
    row_ptr, col, a, b = csr_from_edges(V, [(u, v, ab[0], ab[1]) for (u, v), ab in links.items()])
    modes = [SHORTEST_ONLY, KSHORTEST, KSHORTEST, RELAY1] + ([HIER_RELAY] if two_nodes else [])
    mode = int(rng.choice(modes))
    owner = post_ptr = post = None
    if kind == EXPLICIT:
        C = int(rng.integers(1, 2 * P))
        owner = rng.integers(0, P, C).astype(np.int32)
        posts = [sorted(set(int(x) for x in rng.integers(0, P, int(rng.integers(1, P + 1)))))
                 for _ in range(C)]
        post_ptr = np.cumsum([0] + [len(p) for p in posts]).astype(np.int32)
        post = np.array([x for p in posts for x in p], dtype=np.int32)
    w = Workload(f"random{seed}", V, P, row_ptr, col, a, b, node_of, kind,
                 int(rng.integers(1, 3)), int(rng.choice([4096, 65536, 1 << 20])), mode,
                 k=int(rng.integers(1, 5)), max_cross=max_cross, relay=relay, owner=owner,
                 post_ptr=post_ptr, post=post, seed=seed)
    extra = rng.choice(["static", "greedy", "rgreedy", "contig", "ports"])
    if extra == "greedy":
        w = with_greedy(w)
    elif extra == "rgreedy":
        w = with_reverse_greedy(w)
    elif extra == "contig" and two_nodes:
        w = with_contiguity(w)
    elif extra == "ports" and kind == ALLTOALL and switch:
        w = with_switch_ports(w)
    return w


def random_workload_large(seed):
    """A seeded random larger plan for parity sweeps: 2..24 ranks on a
    bidirectional ring plus random link pairs, up to two switch vertices
    (possibly linked to each other), up to three nodes with random relay
    ranks and inter-node links only between relays, any collective kind,
    any route mode, up to 6 options per pair and 3 chunks per rank, and one
    of static orders, greedy orders in path or reverse path order,
    contiguous transfers or switch ports."""
    rng = np.random.default_rng(seed)
    kind = int(rng.choice([ALLGATHER, ALLTOALL, REDUCESCATTER, ALLREDUCE, EXPLICIT]))
    P = int(rng.integers(2, 25))
    nsw = int(rng.choice([0, 0, 1, 2]))
    nn = int(rng.choice([1, 1, 2, 3])) if P >= 3 else 1
    V = P + nsw
    node_of = np.array([min(r * nn // P, nn - 1) for r in range(P)] +
                       [int(rng.integers(0, nn)) for _ in range(nsw)], dtype=np.int32)
    relay = (rng.random(V) < 0.5).astype(np.uint8)
    for n in range(nn):
        ranks = [r for r in range(P) if node_of[r] == n]
        if ranks:
            relay[ranks[0]] = 1
    links = {}

    def add(u, v):
        if u != v and (u, v) not in links:
            links[(u, v)] = (int(rng.choice([700, 1700, 300])), int(rng.choice([8, 46, 106, 3])))

    for i in range(P):
        add(i, (i + 1) % P)
        add((i + 1) % P, i)
    for _ in range(int(rng.integers(0, 3 * P))):
        u, v = (int(x) for x in rng.integers(0, P, 2))
        add(u, v)
        add(v, u)
    for k in range(nsw):
        sw = P + k
        for r in range(P):
            if node_of[r] == node_of[sw] and rng.random() < 0.9:
                add(r, sw)
                add(sw, r)
    if nsw == 2 and rng.random() < 0.5:
        add(P, P + 1)
        add(P + 1, P)
    cross = bool(rng.random() < 0.7) and nn > 1
    if cross:
        links = {(u, v): x for (u, v), x in links.items()
                 if node_of[u] == node_of[v] or (relay[u] and relay[v])}
    row_ptr, col, a, b = csr_from_edges(V, [(u, v, x[0], x[1]) for (u, v), x in links.items()])
    modes = [SHORTEST_ONLY, KSHORTEST, KSHORTEST, RELAY1] + ([HIER_RELAY] if nn > 1 else [])
    mode = int(rng.choice(modes))
    owner = post_ptr = post = None
    if kind == EXPLICIT:
        C = int(rng.integers(1, 3 * P))
        owner = rng.integers(0, P, C).astype(np.int32)
        posts = [sorted(set(int(x) for x in rng.integers(0, P, int(rng.integers(1, P + 1)))))
                 for _ in range(C)]
        post_ptr = np.cumsum([0] + [len(p) for p in posts]).astype(np.int32)
        post = np.array([x for p in posts for x in p], dtype=np.int32)
    w = Workload(f"large{seed}", V, P, row_ptr, col, a, b, node_of if nn > 1 else None, kind,
                 int(rng.integers(1, 4)), int(rng.choice([4096, 65536, 1 << 20])), mode,
                 k=int(rng.integers(1, 7)), max_cross=1 if cross else -1,
                 relay=relay if (cross or mode in (RELAY1, HIER_RELAY)) else None,
                 owner=owner, post_ptr=post_ptr, post=post, seed=seed)
    extra = rng.choice(["static", "greedy", "rgreedy", "contig", "ports"])
    if extra == "greedy":
        w = with_greedy(w)
    elif extra == "rgreedy":
        w = with_reverse_greedy(w)
    elif extra == "contig" and nn > 1:
        w = with_contiguity(w)
    elif extra == "ports" and kind == ALLTOALL and nsw:
        w = with_switch_ports(w)
    return w
