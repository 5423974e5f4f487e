"""Host-side checks of the C ABI library (no kernel launches, no GPU).

The library loads, exports every symbol include/taccl.h declares, builds
the same route tables as the oracle, and rejects bad arguments with the
documented status codes before touching a device.
"""
import ctypes as ct
import os
import re

import numpy as np
import pytest

from oracle import OraclePlan
from paper_2111_04867_amd import binding as B
from workloads import configs as cf
from workloads import generate

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "taccl.h")).read()
    return sorted(set(re.findall(r"\b(taccl_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = B.lib()
    declared = header_functions()
    assert declared, "no declarations found"
    for name in declared:
        assert hasattr(L, name), name
    assert sorted(B.EXPORTS) == declared
    assert L.taccl_version() >= 100


SMALL = [lambda: cf.uni_ring_ag(7), lambda: cf.full_a2a(5), lambda: cf.full_ag(5, k=3),
         lambda: cf.explicit_multicast(cf.full_ag(5, k=3), [0, 1, 2, 3],
                                       [[1, 3], [0, 2, 4], [2], [0, 1, 2, 4]])]


@pytest.mark.parametrize("make", [lambda n=n: cf.named(n)
                                  for n in cf.ORDER + cf.CONTIG_ORDER + cf.REDUCE_ORDER
                                  + cf.PORTS_ORDER] + SMALL)
def test_plan_tables_equal_oracle(make):
    w = make()
    plan = B.Plan.from_workload(w)
    ref = OraclePlan.from_workload(w)
    assert plan.route_stride == ref.route_stride
    assert plan.prio_stride == ref.prio_stride
    assert plan.max_hops == ref.max_hops
    assert (plan.route_options() == ref.route_options()).all()
    assert (plan.link_costs().astype(np.uint64) == ref.link_costs()).all()
    for s in range(w.P):
        for d in range(w.P):
            if s != d:
                assert plan.paths(s, d) == ref.paths(s, d), (s, d)


def test_bytes_per_candidate():
    """routes + 4 * priorities + 5 output bytes per candidate."""
    want = {"ring4_ag": 85, "cubemesh8_ag": 325, "switch16_a2a": 4357, "twonode16_ag": 2565,
            "fournode64_a2a": 86021}
    for name, b in want.items():
        assert B.Plan.from_workload(cf.named(name)).bytes_per_candidate == b
    # Allreduce reads two priority rows
    assert B.Plan.from_workload(cf.named("twonode16_ar")).bytes_per_candidate == 512 + 8 * 512 + 5


def test_greedy_orders_are_not_combined_with_contiguity():
    w = cf.with_greedy(cf.with_contiguity(cf.twonode16_ag(n_candidates=1)))
    with pytest.raises(B.TacclError) as e:
        B.Plan.from_workload(w)
    assert e.value.status == B.ERR_INVALID_ARGUMENT


def test_reduction_needs_reverse_links():
    w = cf.as_reduction(cf.uni_ring_ag(4), cf.REDUCESCATTER)
    with pytest.raises(B.TacclError) as e:
        B.Plan.from_workload(w)
    assert e.value.status == B.ERR_INVALID_ARGUMENT


def test_switch_ports_limits():
    """Switch ports apply to Alltoall only; a switch-to-switch link would be
    a send port of some switched sends and a receive port of others, which
    the oracle times and the kernel does not: the library refuses it."""
    w = cf.with_switch_ports(cf.cubemesh8_ag(n_candidates=1))
    with pytest.raises(B.TacclError) as e:
        B.Plan.from_workload(w)
    assert e.value.status == B.ERR_UNSUPPORTED
    edges = (cf.switch_edges(range(2), 4, 700, 8) + cf.switch_edges(range(2, 4), 5, 700, 8)
             + [(4, 5, 1000, 10), (5, 4, 1000, 10)])
    row_ptr, col, a, b = cf.csr_from_edges(6, edges)
    w = cf.Workload("twoswitch_linked", 6, 4, row_ptr, col, a, b, None, cf.ALLTOALL, 1, 65536,
                    cf.KSHORTEST, k=1, switch_ports=1)
    ref = OraclePlan.from_workload(w)
    assert ref.max_hops == 3
    with pytest.raises(B.TacclError) as e:
        B.Plan.from_workload(w)
    assert e.value.status == B.ERR_UNSUPPORTED
    assert "send port and a receive port" in str(e.value)


# ----------------------------------------------------------------------------
# error paths
# ----------------------------------------------------------------------------

def status_of(fn):
    with pytest.raises(B.TacclError) as e:
        fn()
    return e.value.status


def test_topology_errors():
    L = B.lib()
    h = ct.c_void_p()
    rp = np.array([0, 1, 2], dtype=np.int32)
    col = np.array([0, 0], dtype=np.int32)  # 0 -> 0 self loop
    a = np.ones(2, dtype=np.uint32)
    assert L.taccl_topology_create(2, 2, rp.ctypes.data, col.ctypes.data, a.ctypes.data,
                                   a.ctypes.data, None, ct.byref(h)) == B.ERR_INVALID_ARGUMENT
    assert b"self loop" in L.taccl_last_error()
    col = np.array([1, 0], dtype=np.int32)
    assert L.taccl_topology_create(2, 3, rp.ctypes.data, col.ctypes.data, a.ctypes.data,
                                   a.ctypes.data, None, ct.byref(h)) == B.ERR_INVALID_ARGUMENT
    rp2 = np.array([0, 2, 2], dtype=np.int32)
    col2 = np.array([1, 1], dtype=np.int32)  # duplicate 0 -> 1
    assert L.taccl_topology_create(2, 2, rp2.ctypes.data, col2.ctypes.data, a.ctypes.data,
                                   a.ctypes.data, None, ct.byref(h)) == B.ERR_INVALID_ARGUMENT
    assert L.taccl_topology_create(2, 2, rp.ctypes.data, col.ctypes.data, a.ctypes.data,
                                   a.ctypes.data, None, None) == B.ERR_INVALID_ARGUMENT


def test_collective_and_sketch_errors():
    L = B.lib()
    h = ct.c_void_p()
    assert L.taccl_collective_create(7, 4, 1, 1024, ct.byref(h)) == B.ERR_INVALID_ARGUMENT
    assert L.taccl_collective_create(0, 4, 0, 1024, ct.byref(h)) == B.ERR_INVALID_ARGUMENT
    assert L.taccl_collective_create(1, 300, 1, 1024, ct.byref(h)) == B.ERR_LIMIT
    w = cf.ring4_ag()
    assert status_of(lambda: B.Plan(w.V, w.P, w.row_ptr, w.col, w.alpha_ns, w.beta_ps_per_byte,
                                    None, cf.ALLGATHER, 1, 1024, route_mode=cf.KSHORTEST,
                                    k=0)) == B.ERR_INVALID_ARGUMENT
    assert status_of(lambda: B.Plan(w.V, w.P, w.row_ptr, w.col, w.alpha_ns, w.beta_ps_per_byte,
                                    None, cf.ALLGATHER, 1, 1024, route_mode=9,
                                    k=1)) == B.ERR_INVALID_ARGUMENT


def test_cost_and_makespan_limits():
    w = cf.uni_ring_ag(4)
    big = np.full(w.E, 0xFFFFFF00, dtype=np.uint32)
    assert status_of(lambda: B.Plan(w.V, w.P, w.row_ptr, w.col, big, np.full(w.E, 1000),
                                    None, cf.ALLGATHER, 1, 1 << 20)) == B.ERR_LIMIT
    # each cost fits, but 12 sends of it may not
    assert status_of(lambda: B.Plan(w.V, w.P, w.row_ptr, w.col, np.full(w.E, 1 << 29), w.beta_ps_per_byte,
                                    None, cf.ALLGATHER, 1, 1 << 20)) == B.ERR_LIMIT


def test_multicast_vertex_limit():
    w = cf.uni_ring_ag(65)
    assert status_of(lambda: B.Plan.from_workload(w)) == B.ERR_UNSUPPORTED


def test_eval_batch_argument_checks_do_not_touch_the_device():
    L = B.lib()
    plan = B.Plan.from_workload(cf.ring4_ag())
    h = plan._h
    assert L.taccl_eval_batch(h, 0, None, None, None, None, None) == B.OK
    assert L.taccl_eval_batch(h, -1, None, None, None, None, None) == B.ERR_INVALID_ARGUMENT
    assert L.taccl_eval_batch(h, 4, None, None, None, None, None) == B.ERR_INVALID_ARGUMENT
    assert L.taccl_eval_batch(h, 4, 16, 18, 32, 48, None) == B.ERR_INVALID_ARGUMENT  # misaligned
    assert L.taccl_eval_batch(None, 4, 16, 16, 32, 48, None) == B.ERR_INVALID_ARGUMENT
    assert b"aligned" in L.taccl_last_error() or b"null" in L.taccl_last_error()


def test_plan_path_errors():
    plan = B.Plan.from_workload(cf.ring4_ag())
    with pytest.raises(B.TacclError):
        plan.path(0, 0, 0)
    with pytest.raises(B.TacclError):
        plan.path(0, 1, 5)
    with pytest.raises(B.TacclError):
        plan.path(0, 9, 0)


def test_connections_argument_checks():
    """taccl_connections_batch rejects bad arguments before touching a device."""
    L = B.lib()
    plan = B.Plan.from_workload(cf.switch16_a2a(n_candidates=1))
    buf = ct.c_void_p(64)  # never dereferenced: every call below fails its checks first
    assert L.taccl_connections_batch(None, 1, buf, buf, None) == B.ERR_INVALID_ARGUMENT
    assert L.taccl_connections_batch(plan._h, -1, buf, buf, None) == B.ERR_INVALID_ARGUMENT
    assert L.taccl_connections_batch(plan._h, 1, None, buf, None) == B.ERR_INVALID_ARGUMENT
    assert L.taccl_connections_batch(plan._h, 1, buf, None, None) == B.ERR_INVALID_ARGUMENT
    assert L.taccl_connections_batch(plan._h, 1, buf, ct.c_void_p(66), None) == \
        B.ERR_INVALID_ARGUMENT
    assert L.taccl_connections_batch(plan._h, 0, None, None, None) == B.OK


def test_generate_host_matches_the_shared_generator():
    """taccl_generate_host draws exactly what the tests' generator draws, for
    any candidate range on its own."""
    for name in ("twonode16_ag", "fournode64_a2a", "switch16_a2a"):
        w = cf.named(name)
        plan = B.Plan.from_workload(w)
        r1, p1 = plan.generate(w.seed, 5, 7)
        r2, p2 = generate(w.seed, 5, 7, plan.route_options(), plan.prio_stride)
        assert np.array_equal(r1, r2) and np.array_equal(p1, p2)
        r3, p3 = plan.generate(w.seed, 0, 12)
        assert np.array_equal(r3[5:], r1) and np.array_equal(p3[5:], p1)
        opts = plan.route_options()
        assert ((r3 < np.maximum(opts, 1)) | (opts == 0)).all()


def test_generate_host_argument_checks():
    plan = B.Plan.from_workload(cf.ring4_ag())
    assert status_of(lambda: plan.generate(1, -1, 2)) == B.ERR_INVALID_ARGUMENT
    assert status_of(lambda: plan.generate(1, (1 << 32) - 1, 2)) == B.ERR_INVALID_ARGUMENT
    assert plan.generate(1, 0, 0)[0].shape == (0, plan.route_stride)


def test_count_faults():
    """The fault sentinel is counted on the host; LIMIT keeps every real
    makespan below it, both phases of an Allreduce included."""
    m = np.array([0, 5, B.MAKESPAN_FAULT, 0xFFFFFFFE, B.MAKESPAN_FAULT], dtype=np.uint32)
    assert B.count_faults(m) == 2
    assert B.count_faults(np.zeros(0, dtype=np.uint32)) == 0
    out = ct.c_int64()
    assert B.lib().taccl_count_faults(-1, None, ct.byref(out)) == B.ERR_INVALID_ARGUMENT
    assert B.lib().taccl_count_faults(3, None, ct.byref(out)) == B.ERR_INVALID_ARGUMENT
    # 12 sends of 2^28 ns fit one phase (3 * 2^30 < 2^32 - 1) but not two
    w = cf.ring4_ag()
    cost = np.full(w.E, 1 << 28, dtype=np.uint32)
    beta = np.zeros(w.E, dtype=np.uint32)
    B.Plan(w.V, w.P, w.row_ptr, w.col, cost, beta, None, cf.ALLGATHER, 1, 1 << 20)
    assert status_of(lambda: B.Plan(w.V, w.P, w.row_ptr, w.col, cost, beta, None,
                                    cf.ALLREDUCE, 1, 1 << 20)) == B.ERR_LIMIT
