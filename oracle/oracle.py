"""ctypes wrapper of the C oracle (test infrastructure only).

The oracle evaluates candidate schedules one by one on the CPU; see the
header of taccl_oracle.c for what it computes and which passages of the
paper each step follows.
"""
import ctypes as ct
import os

import numpy as np

from .build import LIB, build_oracle

ALLGATHER, ALLTOALL, EXPLICIT = 0, 1, 2
SHORTEST_ONLY, KSHORTEST, RELAY1, HIER_RELAY = 0, 1, 2, 3

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = os.environ.get("TACCL_ORACLE_LIB", LIB)
    if path == LIB and not os.path.exists(LIB):
        build_oracle()
    lib = ct.CDLL(path)
    P = ct.c_void_p
    lib.orc_create.restype = ct.c_int
    lib.orc_create.argtypes = [ct.c_int, ct.c_int, P, P, P, P, P, ct.c_int, ct.c_int, ct.c_uint64,
                               ct.c_int, P, P, P, P, P, ct.c_int, ct.c_int, ct.c_int,
                               ct.POINTER(ct.c_void_p)]
    lib.orc_destroy.argtypes = [P]
    lib.orc_error.restype = ct.c_char_p
    lib.orc_error.argtypes = [P]
    for name in ("orc_route_stride", "orc_prio_stride", "orc_max_hops", "orc_num_chunks",
                 "orc_max_sends"):
        getattr(lib, name).restype = ct.c_int
        getattr(lib, name).argtypes = [P]
    lib.orc_link_cost.restype = ct.c_uint64
    lib.orc_link_cost.argtypes = [P, ct.c_int]
    lib.orc_npaths.restype = ct.c_int
    lib.orc_npaths.argtypes = [P, ct.c_int, ct.c_int]
    lib.orc_path.restype = ct.c_int
    lib.orc_path.argtypes = [P, ct.c_int, ct.c_int, ct.c_int, P, ct.c_int]
    lib.orc_route_options.restype = ct.c_int
    lib.orc_route_options.argtypes = [P, ct.c_int]
    lib.orc_set_switch_ports.restype = ct.c_int
    lib.orc_set_switch_ports.argtypes = [P, ct.c_int]
    lib.orc_set_order.restype = ct.c_int
    lib.orc_set_order.argtypes = [P, ct.c_int]
    lib.orc_set_contiguity.restype = ct.c_int
    lib.orc_set_contiguity.argtypes = [P, ct.c_int]
    lib.orc_eval.restype = ct.c_int
    lib.orc_eval.argtypes = [P, ct.c_int64, P, P, P, P]
    lib.orc_eval_ops.restype = ct.c_int
    lib.orc_eval_ops.argtypes = [P, ct.c_int64, P, P, P, P, P]
    lib.orc_connections.restype = ct.c_int
    lib.orc_connections.argtypes = [P, ct.c_int64, P, P]
    lib.orc_eval_detail.restype = ct.c_int
    lib.orc_eval_detail.argtypes = [P, P, P, ct.c_int, P] + [P] * 13
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ct.c_void_p)


class OracleError(RuntimeError):
    pass


class OraclePlan:
    """A topology + collective + sketch, as the oracle sees it.

    Arguments mirror the workload descriptors: CSR topology (row_ptr, col,
    alpha_ns, beta_ps_per_byte), node_of (or None), collective kind,
    chunks_per_rank, chunk_bytes, optional explicit pre/postcondition
    (owner, post_ptr, post) and the sketch (allowed, relay, max_cross,
    route_mode, k).
    """

    def __init__(self, V, P, row_ptr, col, alpha_ns, beta_ps_per_byte, node_of, kind,
                 chunks_per_rank, chunk_bytes, allowed=None, relay=None, max_cross=-1,
                 route_mode=KSHORTEST, k=1, owner=None, post_ptr=None, post=None):
        lib = _load()
        i32 = lambda a: None if a is None else np.ascontiguousarray(a, dtype=np.int32)  # noqa: E731
        u32 = lambda a: np.ascontiguousarray(a, dtype=np.uint32)  # noqa: E731
        u8 = lambda a: None if a is None else np.ascontiguousarray(a, dtype=np.uint8)  # noqa: E731
        self._keep = [i32(row_ptr), i32(col), u32(alpha_ns), u32(beta_ps_per_byte), i32(node_of),
                      i32(owner), i32(post_ptr), i32(post), u8(allowed), u8(relay)]
        rp, cl, al, be, nd, ow, pp, po, alw, rl = self._keep
        h = ct.c_void_p()
        rc = lib.orc_create(int(V), int(P), _ptr(rp), _ptr(cl), _ptr(al), _ptr(be), _ptr(nd),
                            int(kind), int(chunks_per_rank), int(chunk_bytes),
                            0 if ow is None else len(ow), _ptr(ow), _ptr(pp), _ptr(po),
                            _ptr(alw), _ptr(rl), int(max_cross), int(route_mode), int(k),
                            ct.byref(h))
        self._h = h
        if rc != 0:
            msg = lib.orc_error(h).decode() if h.value else "allocation failed"
            lib.orc_destroy(h)
            self._h = None
            raise OracleError(f"orc_create failed ({rc}): {msg}")
        self.V, self.P, self.E = int(V), int(P), len(cl)
        self.kind = int(kind)
        self.route_stride = lib.orc_route_stride(h)
        self.prio_stride = lib.orc_prio_stride(h)
        self.max_hops = lib.orc_max_hops(h)
        self.num_chunks = lib.orc_num_chunks(h)
        self.max_sends = lib.orc_max_sends(h)

    @classmethod
    def from_workload(cls, w):
        """Build from a workloads.Workload descriptor."""
        plan = cls(w.V, w.P, w.row_ptr, w.col, w.alpha_ns, w.beta_ps_per_byte, w.node_of,
                   w.kind, w.chunks_per_rank, w.chunk_bytes, allowed=w.allowed, relay=w.relay,
                   max_cross=w.max_cross, route_mode=w.route_mode, k=w.k, owner=w.owner,
                   post_ptr=w.post_ptr, post=w.post)
        plan.set_contiguity(getattr(w, "contiguity", 0))
        plan.set_order(getattr(w, "order", 0))
        plan.set_switch_ports(getattr(w, "switch_ports", 0))
        return plan

    def set_switch_ports(self, mode):
        """0: switch vertices store and forward; 1: a hop pair through a switch
        is one send holding the sender's and the receiver's ports."""
        if _load().orc_set_switch_ports(self._h, int(mode)) != 0:
            raise OracleError(f"bad switch-port mode {mode}")
        self.switch_ports = int(mode)

    def set_order(self, mode):
        """0: static Step-2 orders; 1: time-aware greedy orders (App. B.2) in
        path order; 2: the same greedy in reverse path order."""
        if _load().orc_set_order(self._h, int(mode)) != 0:
            raise OracleError(f"bad order mode {mode}")
        self.order = int(mode)

    def set_contiguity(self, mode):
        """0: one chunk per transfer; 1: contiguous transfers of equal-remaining,
        already-ready sends on links between nodes."""
        if _load().orc_set_contiguity(self._h, int(mode)) != 0:
            raise OracleError(f"bad contiguity mode {mode}")
        self.contiguity = int(mode)

    def __del__(self):
        if getattr(self, "_h", None):
            _load().orc_destroy(self._h)
            self._h = None

    # ---- plan views --------------------------------------------------
    def link_cost(self, e):
        return int(_load().orc_link_cost(self._h, int(e)))

    def link_costs(self):
        return np.array([self.link_cost(e) for e in range(self.E)], dtype=np.uint64)

    def npaths(self, s, d):
        return int(_load().orc_npaths(self._h, int(s), int(d)))

    def path(self, s, d, i):
        buf = np.zeros(max(self.V, 1) * 4, dtype=np.int32)
        n = _load().orc_path(self._h, int(s), int(d), int(i), _ptr(buf), len(buf))
        if n < 0:
            raise IndexError((s, d, i))
        return [int(x) for x in buf[:n]]

    def paths(self, s, d):
        return [self.path(s, d, i) for i in range(self.npaths(s, d))]

    def route_options(self):
        """Number of route choices for every route entry (0 = entry unused)."""
        lib = _load()
        return np.array([lib.orc_route_options(self._h, e) for e in range(self.route_stride)],
                        dtype=np.int32)

    # ---- evaluation ----------------------------------------------------
    def eval(self, routes, prio):
        routes = np.ascontiguousarray(routes, dtype=np.uint8).reshape(-1, self.route_stride)
        prio = np.ascontiguousarray(prio, dtype=np.uint32).reshape(-1, self.prio_stride)
        n = routes.shape[0]
        if prio.shape[0] != n:
            raise ValueError("routes and prio disagree on the candidate count")
        mk = np.zeros(n, dtype=np.uint32)
        ok = np.zeros(n, dtype=np.uint8)
        rc = _load().orc_eval(self._h, n, _ptr(routes), _ptr(prio), _ptr(mk), _ptr(ok))
        if rc != 0:
            raise OracleError(f"orc_eval failed ({rc})")
        return mk, ok

    def eval_ops(self, routes, prio):
        """eval() plus the algorithmic operation count of every candidate (the
        op model of orc_eval_ops); returns (makespan, valid, ops)."""
        routes = np.ascontiguousarray(routes, dtype=np.uint8).reshape(-1, self.route_stride)
        prio = np.ascontiguousarray(prio, dtype=np.uint32).reshape(-1, self.prio_stride)
        n = routes.shape[0]
        if prio.shape[0] != n:
            raise ValueError("routes and prio disagree on the candidate count")
        mk = np.zeros(n, dtype=np.uint32)
        ok = np.zeros(n, dtype=np.uint8)
        ops = np.zeros(n, dtype=np.uint64)
        rc = _load().orc_eval_ops(self._h, n, _ptr(routes), _ptr(prio), _ptr(mk), _ptr(ok),
                                  _ptr(ops))
        if rc != 0:
            raise OracleError(f"orc_eval_ops failed ({rc})")
        return mk, ok, ops

    def eval_threads(self, routes, prio, threads=None):
        """eval() split over threads on disjoint candidate ranges (the C call
        releases the GIL; each call has its own scratch)."""
        from concurrent.futures import ThreadPoolExecutor
        routes = np.ascontiguousarray(routes, dtype=np.uint8).reshape(-1, self.route_stride)
        prio = np.ascontiguousarray(prio, dtype=np.uint32).reshape(-1, self.prio_stride)
        n = routes.shape[0]
        threads = threads or min(16, os.cpu_count() or 1)
        if n < 2 * threads:
            return self.eval(routes, prio)
        bounds = np.linspace(0, n, threads + 1).astype(int)
        with ThreadPoolExecutor(threads) as ex:
            parts = list(ex.map(lambda ab: self.eval(routes[ab[0]:ab[1]], prio[ab[0]:ab[1]]),
                                zip(bounds[:-1], bounds[1:])))
        return np.concatenate([p[0] for p in parts]), np.concatenate([p[1] for p in parts])

    def connections(self, routes):
        """Per candidate, the ordered rank pairs that exchange a chunk through
        switch vertices only (the uc-max / uc-min count)."""
        routes = np.ascontiguousarray(routes, dtype=np.uint8).reshape(-1, self.route_stride)
        out = np.zeros(routes.shape[0], dtype=np.uint32)
        rc = _load().orc_connections(self._h, routes.shape[0], _ptr(routes), _ptr(out))
        if rc != 0:
            raise OracleError(f"orc_connections failed ({rc})")
        return out

    def eval_detail(self, routes, prio):
        """One candidate; returns (makespan, valid, sends) where sends is a
        dict of per-send arrays."""
        routes = np.ascontiguousarray(routes, dtype=np.uint8).reshape(self.route_stride)
        prio = np.ascontiguousarray(prio, dtype=np.uint32).reshape(self.prio_stride)
        cap = max(self.max_sends, 1) * (2 if self.kind == 4 else 1)  # Allreduce: two phases
        out = {k: np.zeros(cap, dtype=np.int32) for k in ("chunk", "link", "from", "to", "hop",
                                                           "pos")}
        out.update({k: np.zeros(cap, dtype=np.uint64) for k in ("rem", "trav", "start",
                                                                 "finish")})
        out["prio"] = np.zeros(cap, dtype=np.uint32)
        ns = ct.c_int()
        mk = ct.c_uint32()
        ok = ct.c_uint8()
        rc = _load().orc_eval_detail(
            self._h, _ptr(routes), _ptr(prio), cap, ct.byref(ns), _ptr(out["chunk"]),
            _ptr(out["link"]), _ptr(out["from"]), _ptr(out["to"]), _ptr(out["hop"]),
            _ptr(out["rem"]), _ptr(out["trav"]), _ptr(out["prio"]), _ptr(out["pos"]),
            _ptr(out["start"]), _ptr(out["finish"]), ct.byref(mk), ct.byref(ok))
        if rc != 0:
            raise OracleError(f"orc_eval_detail failed ({rc})")
        n = ns.value
        return int(mk.value), int(ok.value), {k: v[:n].copy() for k, v in out.items()}
