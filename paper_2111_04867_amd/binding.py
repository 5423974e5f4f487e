"""Thin ctypes binding of libtaccl.so (argument marshalling only).

Every step of the evaluation runs in the library's HIP kernels; this module
only converts Python/numpy/torch arguments into the pointers and sizes of
the C ABI (include/taccl.h). There is no fallback: if the library is
missing the import of this module's functions raises.
"""
import ctypes as ct
import os

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
# TACCL_LIB selects another build of the same sources (the host-sanitizer
# build of tests/sanitize.py); the default is the in-tree library
LIB_PATH = os.environ.get("TACCL_LIB", os.path.join(PKG, "libtaccl.so"))

OK, ERR_INVALID_ARGUMENT, ERR_UNSUPPORTED, ERR_LIMIT, ERR_NO_MEMORY, ERR_HIP = range(6)
ALLGATHER, ALLTOALL, EXPLICIT = 0, 1, 2
SHORTEST_ONLY, KSHORTEST, RELAY1, HIER_RELAY = 0, 1, 2, 3


class TacclError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"taccl error {status}: {msg}")
        self.status = status


class SketchDesc(ct.Structure):
    _fields_ = [("allowed_link", ct.c_void_p), ("is_relay", ct.c_void_p),
                ("max_node_crossings", ct.c_int32), ("route_mode", ct.c_int32),
                ("k", ct.c_int32), ("contiguity", ct.c_int32), ("order", ct.c_int32),
                ("switch_ports", ct.c_int32)]


class PlanInfo(ct.Structure):
    _fields_ = [("num_vertices", ct.c_int32), ("num_ranks", ct.c_int32),
                ("num_links", ct.c_int32), ("num_chunks", ct.c_int32), ("kind", ct.c_int32),
                ("route_stride", ct.c_int32), ("prio_stride", ct.c_int32),
                ("max_hops", ct.c_int32), ("max_paths", ct.c_int32), ("num_pairs", ct.c_int32),
                ("num_levels", ct.c_int32), ("max_sends", ct.c_int64),
                ("bytes_per_candidate", ct.c_uint64), ("num_classes", ct.c_int32),
                ("lds_bytes", ct.c_int32)]


# every symbol include/taccl.h declares
EXPORTS = ["taccl_topology_create", "taccl_topology_destroy", "taccl_collective_create",
           "taccl_collective_create_explicit", "taccl_collective_destroy", "taccl_sketch_apply",
           "taccl_plan_destroy", "taccl_plan_info", "taccl_plan_route_options",
           "taccl_plan_path", "taccl_plan_link_costs", "taccl_plan_upload", "taccl_eval_batch",
           "taccl_connections_batch", "taccl_generate_host", "taccl_count_faults",
           "taccl_last_error",
           "taccl_version"]

_lib = None


def lib():
    """Load libtaccl.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() or "
                          "python paper_2111_04867_amd/build.py")
    # torch carries its own HIP runtime (soname libamdhip64.so.7); loading it
    # first makes the library bind to that same runtime instead of starting
    # a second one that would compete for the device
    import torch  # noqa: F401
    L = ct.CDLL(LIB_PATH)
    P = ct.c_void_p
    st = ct.c_int
    L.taccl_topology_create.restype = st
    L.taccl_topology_create.argtypes = [ct.c_int32, ct.c_int32, P, P, P, P, P, P]
    L.taccl_topology_destroy.argtypes = [P]
    L.taccl_collective_create.restype = st
    L.taccl_collective_create.argtypes = [ct.c_int, ct.c_int32, ct.c_int32, ct.c_uint64, P]
    L.taccl_collective_create_explicit.restype = st
    L.taccl_collective_create_explicit.argtypes = [ct.c_int32, ct.c_int32, ct.c_uint64, P, P, P,
                                                   P]
    L.taccl_collective_destroy.argtypes = [P]
    L.taccl_sketch_apply.restype = st
    L.taccl_sketch_apply.argtypes = [P, P, ct.POINTER(SketchDesc), P]
    L.taccl_plan_destroy.argtypes = [P]
    L.taccl_plan_info.restype = st
    L.taccl_plan_info.argtypes = [P, ct.POINTER(PlanInfo)]
    L.taccl_plan_route_options.restype = st
    L.taccl_plan_route_options.argtypes = [P, P]
    L.taccl_plan_path.restype = st
    L.taccl_plan_path.argtypes = [P, ct.c_int32, ct.c_int32, ct.c_int32, P, ct.c_int32,
                                  ct.POINTER(ct.c_int32)]
    L.taccl_plan_link_costs.restype = st
    L.taccl_plan_link_costs.argtypes = [P, P]
    L.taccl_plan_upload.restype = st
    L.taccl_plan_upload.argtypes = [P]
    L.taccl_eval_batch.restype = st
    L.taccl_eval_batch.argtypes = [P, ct.c_int64, P, P, P, P, P]
    L.taccl_connections_batch.restype = st
    L.taccl_connections_batch.argtypes = [P, ct.c_int64, P, P, P]
    L.taccl_generate_host.restype = st
    L.taccl_generate_host.argtypes = [P, ct.c_uint64, ct.c_int64, ct.c_int64, P, P]
    L.taccl_count_faults.restype = st
    L.taccl_count_faults.argtypes = [ct.c_int64, P, ct.POINTER(ct.c_int64)]
    L.taccl_last_error.restype = ct.c_char_p
    L.taccl_last_error.argtypes = []
    L.taccl_version.restype = ct.c_int32
    _lib = L
    return L


def _check(status):
    if status != OK:
        raise TacclError(status, lib().taccl_last_error().decode())


def _np_ptr(a):
    return None if a is None else a.ctypes.data_as(ct.c_void_p)


MAKESPAN_FAULT = 0xFFFFFFFF  # makespan of a candidate whose evaluation faulted


def count_faults(makespan):
    """Number of host makespans equal to MAKESPAN_FAULT (taccl_count_faults)."""
    m = np.ascontiguousarray(makespan).view(np.uint32).reshape(-1)
    out = ct.c_int64()
    _check(lib().taccl_count_faults(int(m.size), _np_ptr(m), ct.byref(out)))
    return int(out.value)


class Plan:
    """Topology + collective + sketch compiled by the library.

    `keepalive` holds the numpy arrays whose pointers were passed in (the
    library copies them, but they must live through the create calls)."""

    def __init__(self, V, P, row_ptr, col, alpha_ns, beta_ps_per_byte, node_of, kind,
                 chunks_per_rank, chunk_bytes, allowed=None, relay=None, max_cross=-1,
                 route_mode=KSHORTEST, k=1, owner=None, post_ptr=None, post=None, contiguity=0,
                 order=0, switch_ports=0):
        L = lib()
        i32 = lambda a: None if a is None else np.ascontiguousarray(a, dtype=np.int32)  # noqa
        u32 = lambda a: np.ascontiguousarray(a, dtype=np.uint32)  # noqa: E731
        u8 = lambda a: None if a is None else np.ascontiguousarray(a, dtype=np.uint8)  # noqa
        rp, cl, al, be, nd = i32(row_ptr), i32(col), u32(alpha_ns), u32(beta_ps_per_byte), \
            i32(node_of)
        topo, coll, plan = ct.c_void_p(), ct.c_void_p(), ct.c_void_p()
        self._h = None
        try:
            _check(L.taccl_topology_create(int(V), int(P), _np_ptr(rp), _np_ptr(cl), _np_ptr(al),
                                           _np_ptr(be), _np_ptr(nd), ct.byref(topo)))
            if kind == EXPLICIT:
                ow, pp, po = i32(owner), i32(post_ptr), i32(post)
                _check(L.taccl_collective_create_explicit(len(ow), int(P), int(chunk_bytes),
                                                          _np_ptr(ow), _np_ptr(pp), _np_ptr(po),
                                                          ct.byref(coll)))
            else:
                _check(L.taccl_collective_create(int(kind), int(P), int(chunks_per_rank),
                                                 int(chunk_bytes), ct.byref(coll)))
            alw, rl = u8(allowed), u8(relay)
            sk = SketchDesc(_np_ptr(alw), _np_ptr(rl), int(max_cross), int(route_mode), int(k),
                            int(contiguity), int(order), int(switch_ports))
            _check(L.taccl_sketch_apply(topo, coll, ct.byref(sk), ct.byref(plan)))
        finally:
            L.taccl_topology_destroy(topo)
            L.taccl_collective_destroy(coll)
        self._h = plan
        info = PlanInfo()
        _check(L.taccl_plan_info(plan, ct.byref(info)))
        self.info = {name: getattr(info, name) for name, _ in PlanInfo._fields_}
        self.route_stride = info.route_stride
        self.prio_stride = info.prio_stride
        self.max_hops = info.max_hops
        self.num_chunks = info.num_chunks
        self.bytes_per_candidate = info.bytes_per_candidate
        self.V, self.P, self.E = info.num_vertices, info.num_ranks, info.num_links

    @classmethod
    def from_workload(cls, w):
        return cls(w.V, w.P, w.row_ptr, w.col, w.alpha_ns, w.beta_ps_per_byte, w.node_of,
                   w.kind, w.chunks_per_rank, w.chunk_bytes, allowed=w.allowed, relay=w.relay,
                   max_cross=w.max_cross, route_mode=w.route_mode, k=w.k, owner=w.owner,
                   post_ptr=w.post_ptr, post=w.post, contiguity=getattr(w, "contiguity", 0),
                   order=getattr(w, "order", 0), switch_ports=getattr(w, "switch_ports", 0))

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.taccl_plan_destroy(self._h)
            self._h = None

    # ---- host views ------------------------------------------------------
    def route_options(self):
        out = np.zeros(self.route_stride, dtype=np.int32)
        _check(lib().taccl_plan_route_options(self._h, _np_ptr(out)))
        return out

    def generate(self, seed, first, count):
        """Seeded candidates first .. first+count-1 on the host:
        (routes u8 [count, route_stride], prio u32 [count, prio_stride])."""
        routes = np.zeros((count, self.route_stride), dtype=np.uint8)
        prio = np.zeros((count, self.prio_stride), dtype=np.uint32)
        _check(lib().taccl_generate_host(self._h, int(seed), int(first), int(count),
                                         _np_ptr(routes), _np_ptr(prio)))
        return routes, prio

    def link_costs(self):
        out = np.zeros(self.E, dtype=np.uint32)
        _check(lib().taccl_plan_link_costs(self._h, _np_ptr(out)))
        return out

    def path(self, s, d, i):
        buf = np.zeros(max(self.max_hops, 1), dtype=np.int32)
        hops = ct.c_int32()
        _check(lib().taccl_plan_path(self._h, int(s), int(d), int(i), _np_ptr(buf), len(buf),
                                     ct.byref(hops)))
        return [int(x) for x in buf[:hops.value]]

    def paths(self, s, d):
        n = int(self.route_options_for_pair(s, d))
        return [self.path(s, d, i) for i in range(n)]

    def route_options_for_pair(self, s, d):
        """Number of options of pair (s, d), probed through taccl_plan_path."""
        n = 0
        hops = ct.c_int32()
        buf = np.zeros(max(self.max_hops, 1), dtype=np.int32)
        while lib().taccl_plan_path(self._h, int(s), int(d), n, _np_ptr(buf), len(buf),
                                    ct.byref(hops)) == OK:
            n += 1
        return n

    def upload(self):
        _check(lib().taccl_plan_upload(self._h))

    # ---- evaluation -------------------------------------------------------
    def eval_batch(self, n, d_routes, d_prio, d_makespan, d_valid, stream=0):
        """Raw call: device pointers (ints) and a hipStream_t handle (int)."""
        _check(lib().taccl_eval_batch(self._h, int(n), ct.c_void_p(int(d_routes)),
                                      ct.c_void_p(int(d_prio)), ct.c_void_p(int(d_makespan)),
                                      ct.c_void_p(int(d_valid)), ct.c_void_p(int(stream))))

    def eval_tensors(self, routes, prio, makespan, valid, stream=None):
        """torch CUDA tensors: routes uint8 [n, route_stride], prio int32/uint32
        [n, prio_stride], makespan int32/uint32 [n], valid uint8 [n]. Runs on
        `stream` (default: torch's current stream), asynchronously."""
        import torch
        n = routes.shape[0]
        for t, w, nm in ((routes, self.route_stride, "routes"), (prio, self.prio_stride, "prio")):
            if not t.is_cuda or not t.is_contiguous() or t.dim() != 2 or t.shape[1] != w:
                raise ValueError(f"{nm} must be a contiguous CUDA tensor [n, {w}]")
        if prio.shape[0] != n or makespan.numel() < n or valid.numel() < n:
            raise ValueError("tensor sizes disagree on the candidate count")
        if routes.element_size() != 1 or prio.element_size() != 4 or \
                makespan.element_size() != 4 or valid.element_size() != 1:
            raise ValueError("dtypes: routes u8, prio 32-bit, makespan 32-bit, valid u8")
        s = (stream if stream is not None else torch.cuda.current_stream()).cuda_stream
        self.eval_batch(n, routes.data_ptr(), prio.data_ptr(), makespan.data_ptr(),
                        valid.data_ptr(), s)

    def eval(self, routes, prio, device="cuda"):
        """Convenience: host numpy in, host numpy out (copies and syncs)."""
        import torch
        routes = np.ascontiguousarray(routes, dtype=np.uint8).reshape(-1, self.route_stride)
        prio = np.ascontiguousarray(prio, dtype=np.uint32).reshape(-1, self.prio_stride)
        n = routes.shape[0]
        d_r = torch.from_numpy(routes).to(device)
        d_p = torch.from_numpy(prio.view(np.int32)).to(device)
        d_m = torch.empty(max(n, 1), dtype=torch.int32, device=device)
        d_v = torch.empty(max(n, 1), dtype=torch.uint8, device=device)
        self.eval_tensors(d_r, d_p, d_m, d_v)
        torch.cuda.synchronize()
        return d_m[:n].cpu().numpy().view(np.uint32), d_v[:n].cpu().numpy()

    # ---- switch-hyperedge connections --------------------------------------
    def connections_batch(self, n, d_routes, d_connections, stream=0):
        """Raw call: device pointers (ints) and a hipStream_t handle (int)."""
        _check(lib().taccl_connections_batch(self._h, int(n), ct.c_void_p(int(d_routes)),
                                             ct.c_void_p(int(d_connections)),
                                             ct.c_void_p(int(stream))))

    def connections_tensors(self, routes, out, stream=None):
        """torch CUDA tensors: routes uint8 [n, route_stride], out int32/uint32
        [n]. Runs on `stream` (default: torch's current stream)."""
        import torch
        n = routes.shape[0]
        if not routes.is_cuda or not routes.is_contiguous() or routes.dim() != 2 or \
                routes.shape[1] != self.route_stride or routes.element_size() != 1:
            raise ValueError(f"routes must be a contiguous CUDA uint8 tensor [n, "
                             f"{self.route_stride}]")
        if out.numel() < n or out.element_size() != 4:
            raise ValueError("out must hold n 32-bit counts")
        s = (stream if stream is not None else torch.cuda.current_stream()).cuda_stream
        self.connections_batch(n, routes.data_ptr(), out.data_ptr(), s)

    def connections(self, routes, device="cuda"):
        """Convenience: host numpy routes in, host numpy counts out."""
        import torch
        routes = np.ascontiguousarray(routes, dtype=np.uint8).reshape(-1, self.route_stride)
        n = routes.shape[0]
        d_r = torch.from_numpy(routes).to(device)
        d_c = torch.empty(max(n, 1), dtype=torch.int32, device=device)
        self.connections_tensors(d_r, d_c)
        torch.cuda.synchronize()
        return d_c[:n].cpu().numpy().view(np.uint32)
