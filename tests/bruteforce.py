"""Pure-Python brute force for tiny inputs, independent of the oracle.

Used only to pin the oracle. Each piece is a different formulation of what
the paper defines, so that a slip in the oracle (a dropped term, a wrong
index, a reversed order) shows up as a disagreement:

* paths: every sketch-valid simple path up to a hop limit, enumerated
  without pruning, then sorted by (cost, hops, vertex sequence);
* multicast tree: the link that first brings chunk c to vertex v is taken
  from the routed path of the smallest destination whose path contains v
  (a closed characterisation of the first-reach merge, no sequential walk);
* keys: the remaining path of a send is the longest root-to-leaf tree path
  below it, found by enumerating those paths explicitly;
* times: the least solution of the difference constraints of App. B.3
  (send >= start at the source, start = send + lat, and for every pair of
  sends on a link, the later one in the order starts no earlier than the
  earlier one finishes), by Bellman-Ford style relaxation to a fixpoint;
* optimum: the best makespan over every permutation of every link's sends.
"""
import itertools


def link_cost(alpha, beta, chunk_bytes):
    return int(alpha) + -(-int(beta) * int(chunk_bytes) // 1000)


def costs_of(w):
    return [link_cost(w.alpha_ns[e], w.beta_ps_per_byte[e], w.chunk_bytes) for e in range(w.E)]


def out_links(w, u):
    return [(e, int(w.col[e])) for e in range(int(w.row_ptr[u]), int(w.row_ptr[u + 1]))]


def node(w, v):
    return 0 if w.node_of is None else int(w.node_of[v])


def all_simple_paths(w, s, d, hop_limit, max_cross=None):
    """Every simple path s -> d with at most hop_limit links that respects the
    sketch (allowed links, crossing limit, relay-only crossings)."""
    mc = w.max_cross if max_cross is None else max_cross
    out = []

    def rec(u, verts, links, cross):
        if u == d:
            out.append((list(verts), list(links)))
            return
        if len(links) == hop_limit:
            return
        for e, v in out_links(w, u):
            if w.allowed is not None and not w.allowed[e]:
                continue
            if v in verts:
                continue
            c2 = cross
            if node(w, u) != node(w, v):
                c2 += 1
                if mc >= 0 and c2 > mc:
                    continue
                if w.relay is not None and not (w.relay[u] and w.relay[v]):
                    continue
            verts.append(v)
            links.append(e)
            rec(v, verts, links, c2)
            verts.pop()
            links.pop()

    rec(s, [s], [], 0)
    return out


def sorted_paths(w, s, d, hop_limit, max_cross=None):
    cost = costs_of(w)
    ps = all_simple_paths(w, s, d, hop_limit, max_cross)
    ps.sort(key=lambda p: (sum(cost[e] for e in p[1]), len(p[1]), p[0]))
    return ps, cost


def path_vertices(w, links, start):
    vs = [start]
    for e in links:
        vs.append(int(w.col[e]))
    return vs


# ----------------------------------------------------------------------------
# sends of one candidate
# ----------------------------------------------------------------------------

def tree_sends(w, cost, table, routes, prio, owner, posts):
    """Multicast chunks. table[(s, d)] = list of link lists."""
    P, V = w.P, w.V
    sends = []
    present = {}
    for c, o in enumerate(owner):
        routed = {}
        for d in sorted(posts[c]):
            if d == o:
                continue
            opts = table.get((o, d), [])
            ch = int(routes[c * P + d])
            if ch < len(opts):
                routed[d] = opts[ch]
        parent = {}
        for v in range(V):
            if v == o:
                continue
            holders = [d for d in sorted(routed) if v in path_vertices(w, routed[d], o)[1:]]
            if holders:
                dstar = holders[0]
                links = routed[dstar]
                vs = path_vertices(w, links, o)
                parent[v] = links[vs.index(v) - 1]
        # tree distances by walking to the root
        src = {v: _src(w, parent[v]) for v in parent}

        def dist(x):
            t = 0
            while x != o:
                t += cost[parent[x]]
                x = src[x]
            return t

        children = {}
        for v in parent:
            children.setdefault(src[v], []).append(v)

        def leaf_paths(x):
            """all downward tree paths from x, as lists of links"""
            res = [[]]
            for ch in children.get(x, []):
                for tail in leaf_paths(ch):
                    res.append([parent[ch]] + tail)
            return res

        for v in sorted(parent):
            l = parent[v]
            u = src[v]
            longest_below = max(sum(cost[e] for e in p) for p in leaf_paths(v))
            sends.append(dict(chunk=c, link=l, frm=u, to=v, rem=cost[l] + longest_below,
                              trav=dist(u), prio=int(prio[c * V + v])))
        present[c] = {o} | set(parent)
    return sends, present


def _src(w, e):
    u = 0
    while not (int(w.row_ptr[u]) <= e < int(w.row_ptr[u + 1])):
        u += 1
    return u


def path_sends(w, cost, table, routes, prio, owner, dest, H):
    sends = []
    present = {}
    for c, (s, d) in enumerate(zip(owner, dest)):
        present[c] = {s}
        if s == d:
            continue
        opts = table.get((s, d), [])
        ch = int(routes[c])
        if ch >= len(opts):
            continue
        links = opts[ch]
        vs = path_vertices(w, links, s)
        for h, l in enumerate(links):
            sends.append(dict(chunk=c, link=l, frm=vs[h], to=vs[h + 1], hop=h,
                              rem=sum(cost[e] for e in links[h:]),
                              trav=sum(cost[e] for e in links[:h]),
                              prio=int(prio[c * H + h])))
        present[c].add(d)
    return sends, present


def port_units(w, cost, table, routes, prio, owner, dest, H):
    """Alltoall sends under the switch-port model: a hop into a switch vertex
    (index >= P) and the hop out of it form one unit holding both links (the
    sender's send port and the receiver's receive port) for the uplink's
    latency; other hops are units of their own."""
    units, present = [], {}
    for c, (s, d) in enumerate(zip(owner, dest)):
        present[c] = {s}
        if s == d:
            continue
        opts = table.get((s, d), [])
        ch = int(routes[c])
        if ch >= len(opts):
            continue
        links = opts[ch]
        vs = path_vertices(w, links, s)
        mine = []
        h = 0
        while h < len(links):
            if vs[h + 1] >= w.P and h + 1 < len(links):
                mine.append(dict(chunk=c, links=[links[h], links[h + 1]], frm=vs[h], to=vs[h + 2],
                                 hop=h, lat=cost[links[h]], prio=int(prio[c * H + h])))
                h += 2
            else:
                mine.append(dict(chunk=c, links=[links[h]], frm=vs[h], to=vs[h + 1], hop=h,
                                 lat=cost[links[h]], prio=int(prio[c * H + h])))
                h += 1
        for q, u in enumerate(mine):
            u["rem"] = sum(x["lat"] for x in mine[q:])
            u["trav"] = sum(x["lat"] for x in mine[:q])
            u["pred"] = len(units) - 1 if q > 0 else None
            units.append(u)
        present[c].add(d)
    return units, present


def port_least_schedule(units):
    """Least start times: after the chunk's previous unit, and on every link
    a unit holds, after the units before it in that link's Step-2 order."""
    orders = {}
    for i, u in enumerate(units):
        for l in u["links"]:
            orders.setdefault(l, []).append(i)
    for l in orders:
        orders[l].sort(key=lambda i: (-units[i]["rem"], units[i]["trav"], units[i]["prio"],
                                      units[i]["chunk"]))
    t = [0] * len(units)
    changed, rounds = True, 0
    while changed:
        changed = False
        rounds += 1
        if rounds > len(units) + 2:
            raise RuntimeError("constraint graph has a positive cycle")
        for i, u in enumerate(units):
            if u["pred"] is not None:
                need = t[u["pred"]] + units[u["pred"]]["lat"]
                if need > t[i]:
                    t[i] = need
                    changed = True
        for order in orders.values():
            for a_pos in range(len(order)):
                for b_pos in range(a_pos + 1, len(order)):
                    a, b = order[a_pos], order[b_pos]
                    if t[a] + units[a]["lat"] > t[b]:
                        t[b] = t[a] + units[a]["lat"]
                        changed = True
    return t, [t[i] + u["lat"] for i, u in enumerate(units)]


def link_orders(sends):
    """chunk_order per link: the Step-2 heuristic (longest remaining path
    first, then shortest travelled path) with priority and chunk id last."""
    by_link = {}
    for i, s in enumerate(sends):
        by_link.setdefault(s["link"], []).append(i)
    for l in by_link:
        by_link[l].sort(key=lambda i: (-sends[i]["rem"], sends[i]["trav"], sends[i]["prio"],
                                       sends[i]["chunk"]))
    return by_link


def chunk_pred(sends):
    """index of the send that delivers the chunk to each send's source."""
    into = {}
    for i, s in enumerate(sends):
        if "hop" in s:
            into[(s["chunk"], s["hop"] + 1)] = i
        else:
            into[(s["chunk"], s["to"])] = i
    pred = []
    for s in sends:
        if "hop" in s:
            pred.append(into.get((s["chunk"], s["hop"])) if s["hop"] > 0 else None)
        else:
            pred.append(into.get((s["chunk"], s["frm"])))
    return pred


def least_schedule(sends, cost, orders):
    """Least send times satisfying the App. B.3 constraints (no contiguity):
    send >= arrival at the source; for any two sends a before b on one link,
    send[b] >= send[a] + lat. Relaxed to a fixpoint."""
    pred = chunk_pred(sends)
    t = [0] * len(sends)
    changed = True
    rounds = 0
    while changed:
        changed = False
        rounds += 1
        if rounds > len(sends) + 2:
            raise RuntimeError("constraint graph has a positive cycle")
        for i, s in enumerate(sends):
            lo = 0
            if pred[i] is not None:
                p = pred[i]
                lo = max(lo, t[p] + cost[sends[p]["link"]])
            if lo > t[i]:
                t[i] = lo
                changed = True
        for l, order in orders.items():
            for a_pos in range(len(order)):
                for b_pos in range(a_pos + 1, len(order)):
                    a, b = order[a_pos], order[b_pos]
                    need = t[a] + cost[l]
                    if need > t[b]:
                        t[b] = need
                        changed = True
    finish = [t[i] + cost[s["link"]] for i, s in enumerate(sends)]
    return t, finish


def contiguous_schedule(w, sends, orders):
    """Schedule with contiguous transfers, by simulation in time order: the
    transfer that can start earliest (a link's next send whose chunk has
    arrived) starts; on a link between two nodes it also carries the
    following sends of the link's order that have the same remaining length
    and whose chunk has already arrived at that moment; m chunks cost
    alpha + ceil(beta * m * S / 1000) and all arrive when the transfer ends.
    A chunk whose delivering send has not started yet cannot have arrived:
    that send ends after the current time."""
    pred = chunk_pred(sends)
    n = len(sends)
    start = [None] * n
    finish = [None] * n
    head = {l: 0 for l in orders}
    free = {l: 0 for l in orders}
    done = 0
    while done < n:
        best = None
        for l, order in orders.items():
            if head[l] == len(order):
                continue
            x = order[head[l]]
            if pred[x] is not None and finish[pred[x]] is None:
                continue
            ready = 0 if pred[x] is None else finish[pred[x]]
            t = max(free[l], ready)
            if best is None or t < best[0]:
                best = (t, l)
        if best is None:
            raise RuntimeError("no transfer can start")
        t, l = best
        order = orders[l]
        x = order[head[l]]
        group = [x]
        u, v = _src(w, l), int(w.col[l])
        if node(w, u) != node(w, v):
            j = head[l] + 1
            while j < len(order):
                y = order[j]
                if sends[y]["rem"] != sends[x]["rem"]:
                    break
                if pred[y] is not None and (finish[pred[y]] is None or finish[pred[y]] > t):
                    break
                group.append(y)
                j += 1
        m = len(group)
        lat = int(w.alpha_ns[l]) + (int(w.beta_ps_per_byte[l]) * m * int(w.chunk_bytes) + 999) // 1000
        for y in group:
            start[y] = t
            finish[y] = t + lat
        free[l] = t + lat
        head[l] += m
        done += m
    return start, finish


def reverse_link(w, e):
    u, v = _src(w, e), int(w.col[e])
    for f, x in out_links(w, v):
        if x == u:
            return f
    raise ValueError(f"link {e} has no reverse")


def reduce_sends(w, cost, ag_sends, owner):
    """ReduceScatter sends: every Allgather tree edge u -> v run backwards,
    v -> u on the reverse link, carrying v's partial. Remaining length: the
    reversed path from v to the owner, walked edge by edge; travelled: the
    longest reversed path from any vertex below v up to v, by enumerating the
    vertices whose walk to the owner passes v."""
    into = {(s["chunk"], s["to"]): s for s in ag_sends}

    def walk(c, y, stop):
        t, x = 0, y
        while x != owner[c] and x != stop:
            p = into[(c, x)]
            t += cost[reverse_link(w, p["link"])]
            x = p["frm"]
        return t, x

    rs = []
    for s in ag_sends:
        c, u, v = s["chunk"], s["frm"], s["to"]
        up, _ = walk(c, v, None)
        below = 0
        for (cc, y) in into:
            if cc == c:
                t, x = walk(c, y, v)
                if x == v:
                    below = max(below, t)
        rs.append(dict(chunk=c, link=reverse_link(w, s["link"]), frm=v, to=u, rem=up,
                       trav=below, prio=s["prio"]))
    return rs


def reduce_least_schedule(sends, cost, orders):
    """Least send times of a reduction: a send from v waits for every send
    into v (same chunk); link order as in App. B.3. Relaxed to a fixpoint."""
    deps = [[j for j, y in enumerate(sends) if y["chunk"] == x["chunk"] and y["to"] == x["frm"]]
            for x in sends]
    t = [0] * len(sends)
    changed, rounds = True, 0
    while changed:
        changed = False
        rounds += 1
        if rounds > len(sends) + 2:
            raise RuntimeError("constraint graph has a positive cycle")
        for i in range(len(sends)):
            lo = max([t[j] + cost[sends[j]["link"]] for j in deps[i]], default=0)
            if lo > t[i]:
                t[i] = lo
                changed = True
        for l, order in orders.items():
            for a_pos in range(len(order)):
                for b_pos in range(a_pos + 1, len(order)):
                    a, b = order[a_pos], order[b_pos]
                    if t[a] + cost[l] > t[b]:
                        t[b] = t[a] + cost[l]
                        changed = True
    return t, [t[i] + cost[s["link"]] for i, s in enumerate(sends)]


def reduce_deps(sends):
    """Chunk predecessors of every ReduceScatter send: the sends into its source."""
    return [[j for j, y in enumerate(sends) if y["chunk"] == x["chunk"] and y["to"] == x["frm"]]
            for x in sends]


def greedy_link_orders(sends, cost, deps, reverse=False):
    """The time-aware greedy of App. B.2 as a plain event loop: at every step
    every unserved send whose dependencies are all served gets the start
    max(its link's time, the latest finish among them); the smallest
    (start, Step-2 key, priority, chunk) is served. deps[i] lists the sends
    that send i waits for. reverse: the mirrored run, in which a send waits
    for the sends that waited for it and the Step-2 lengths are measured
    from the other end (remaining' = travelled + latency, travelled' =
    remaining - latency); each link's order is then the reverse of the order
    it was served in. Returns {link: [send index, ...]} in schedule order."""
    n = len(sends)
    if reverse:
        waits = [[j for j in range(n) if i in deps[j]] for i in range(n)]
    else:
        waits = deps

    def key(i):
        s, c = sends[i], cost[sends[i]["link"]]
        rem, trav = (s["trav"] + c, s["rem"] - c) if reverse else (s["rem"], s["trav"])
        return (-rem, trav, s["prio"], s["chunk"])

    finish = [None] * n
    link_time = {}
    served = {}
    for _ in range(n):
        ready = [i for i in range(n)
                 if finish[i] is None and all(finish[j] is not None for j in waits[i])]

        def start(i):
            return max([link_time.get(sends[i]["link"], 0)] + [finish[j] for j in waits[i]])

        i = min(ready, key=lambda i: (start(i), key(i)))
        t = start(i)
        finish[i] = t + cost[sends[i]["link"]]
        link_time[sends[i]["link"]] = finish[i]
        served.setdefault(sends[i]["link"], []).append(i)
    if reverse:
        served = {l: order[::-1] for l, order in served.items()}
    return served


def evaluate(w, table, routes, prio, H=None):
    """Makespan, valid and per-send detail of one candidate."""
    if w.kind in (3, 4):  # ReduceScatter, Allreduce
        cost = costs_of(w)
        P, V = w.P, w.V
        C = P * w.chunks_per_rank
        owner = [c // w.chunks_per_rank for c in range(C)]
        posts = [list(range(P)) for _ in range(C)]
        CV = C * V
        ag, present = tree_sends(w, cost, table, routes, prio[:CV], owner, posts)
        rs = reduce_sends(w, cost, ag, owner)
        orders = link_orders(rs)
        start, finish = reduce_least_schedule(rs, cost, orders)
        valid = all(r in present[c] for c in range(C) for r in posts[c])
        mk = max(finish) if finish else 0
        if w.kind == 3:
            return mk, int(valid), rs, start, finish, orders
        ag2, _ = tree_sends(w, cost, table, routes, prio[CV:], owner, posts)
        orders2 = link_orders(ag2)
        start2, finish2 = least_schedule(ag2, cost, orders2)
        mk2 = max(finish2) if finish2 else 0
        return (mk + mk2, int(valid), rs + ag2, start + [x + mk for x in start2],
                finish + [x + mk for x in finish2], None)
    cost = costs_of(w)
    P = w.P
    if w.kind == 1 and getattr(w, "switch_ports", 0):  # Alltoall, switch ports
        C = P * P * w.chunks_per_rank
        owner = [(c // w.chunks_per_rank) // P for c in range(C)]
        dest = [(c // w.chunks_per_rank) % P for c in range(C)]
        units, present = port_units(w, cost, table, routes, prio, owner, dest, H)
        start, finish = port_least_schedule(units)
        valid = all(d in present[c] for c, d in enumerate(dest))
        return max(finish) if finish else 0, int(valid), units, start, finish, None
    if w.kind == 1:  # Alltoall
        C = P * P * w.chunks_per_rank
        owner = [(c // w.chunks_per_rank) // P for c in range(C)]
        dest = [(c // w.chunks_per_rank) % P for c in range(C)]
        sends, present = path_sends(w, cost, table, routes, prio, owner, dest, H)
        posts = [[d] for d in dest]
    else:
        if w.kind == 0:
            C = P * w.chunks_per_rank
            owner = [c // w.chunks_per_rank for c in range(C)]
            posts = [list(range(P)) for _ in range(C)]
        else:
            owner = [int(x) for x in w.owner]
            posts = [[int(r) for r in w.post[w.post_ptr[c]:w.post_ptr[c + 1]]]
                     for c in range(len(owner))]
        sends, present = tree_sends(w, cost, table, routes, prio, owner, posts)
    orders = link_orders(sends)
    if getattr(w, "contiguity", 0):
        start, finish = contiguous_schedule(w, sends, orders)
    else:
        start, finish = least_schedule(sends, cost, orders)
    valid = all(r in present[c] for c in range(len(posts)) for r in posts[c])
    makespan = max(finish) if finish else 0
    return makespan, int(valid), sends, start, finish, orders


def optimum_over_orders(w, sends):
    """Smallest makespan over every permutation of every link's sends."""
    cost = costs_of(w)
    by_link = {}
    for i, s in enumerate(sends):
        by_link.setdefault(s["link"], []).append(i)
    links = sorted(by_link)
    best = None
    for perms in itertools.product(*[itertools.permutations(by_link[l]) for l in links]):
        orders = {l: list(p) for l, p in zip(links, perms)}
        try:
            _, finish = least_schedule(sends, cost, orders)
        except RuntimeError:
            continue  # an order that contradicts the chunk dependencies
        m = max(finish) if finish else 0
        best = m if best is None else min(best, m)
    return best
