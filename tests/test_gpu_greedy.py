"""GPU parity of the time-aware greedy link orders (App. B.2) for multicast
collectives and Alltoall, bit for bit against the oracle, through the C ABI.
Needs an MI355X."""
from dataclasses import replace

import numpy as np
import pytest

from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

C1 = 48935


def say(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2111_04867_amd import binding
    binding.lib()
    torch.cuda.set_device(0)
    yield


def plans(w):
    from paper_2111_04867_amd.binding import Plan
    plan, ref = Plan.from_workload(w), OraclePlan.from_workload(w)
    assert ref.order == w.order and w.order in (1, 2)
    opts = plan.route_options()
    assert (opts == ref.route_options()).all()
    return plan, ref, opts


def check(plan, ref, routes, prio, label):
    say(f"[gpu] {label}: {routes.shape[0]} candidates")
    mk, ok = plan.eval(routes, prio)
    rmk, rok = ref.eval_threads(routes, prio)
    bad = np.nonzero((mk != rmk) | (ok != rok))[0]
    assert bad.size == 0, (f"{label}: {bad.size} mismatches, first at {bad[:5].tolist()}: "
                           f"gpu {mk[bad[:5]].tolist()} oracle {rmk[bad[:5]].tolist()}")
    return mk, ok


@pytest.mark.parametrize("name", cf.GREEDY_ORDER)
def test_full_size_parity(name):
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed, 0, w.n_candidates, opts, plan.prio_stride)
    mk, ok = check(plan, ref, routes, prio, f"{name} full N={w.n_candidates}")
    assert ok.all()


@pytest.mark.parametrize("name", cf.GREEDY_ORDER)
@pytest.mark.parametrize("n", [1, 65, 257])
def test_ragged_batches(name, n):
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 90, 4, n, opts, plan.prio_stride)
    check(plan, ref, routes, prio, f"{name} n={n}")


@pytest.mark.parametrize("value", [0, 0xFFFFFFFF])
def test_equal_priorities(value):
    w = cf.named("twonode16_ag_greedy")
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 6, 0, 200, opts, plan.prio_stride)
    prio[:] = value
    check(plan, ref, routes, prio, f"twonode16_ag_greedy prio={value:#x}")


def test_idle_link_case():
    """0 -> 1 -> 2 -> 3: the greedy fills link 1 -> 2 while the longer chunk
    is still on its way (3 link costs; the static order needs 4)."""
    edges = [(0, 1, 700, 46), (1, 2, 700, 46), (2, 3, 700, 46)]
    row_ptr, col, a, b = cf.csr_from_edges(4, edges)
    base = cf.Workload("chain4", 4, 4, row_ptr, col, a, b, None, cf.ALLGATHER, 1, 1 << 20,
                       cf.KSHORTEST, k=1)
    w = cf.with_greedy(cf.explicit_multicast(base, [0, 1, 1], [[3], [2], [2]]))
    plan, ref, opts = plans(w)
    routes = np.zeros((8, plan.route_stride), dtype=np.uint8)
    prio = np.zeros((8, plan.prio_stride), dtype=np.uint32)
    mk, ok = check(plan, ref, routes, prio, "chain4")
    assert ok.all() and (mk == 3 * C1).all()


@pytest.mark.parametrize("kind", [cf.ALLGATHER, cf.REDUCESCATTER, cf.ALLREDUCE])
@pytest.mark.parametrize("cpr", [1, 3])
def test_full4(kind, cpr):
    w = cf.full_ag(4, k=3, chunks_per_rank=cpr)
    if kind != cf.ALLGATHER:
        w = cf.as_reduction(w, kind)
    w = cf.with_greedy(w)
    plan, ref, opts = plans(w)
    routes, prio = generate(81 + cpr, 0, 600, opts, plan.prio_stride)
    check(plan, ref, routes, prio, f"{w.name} cpr={cpr}")


@pytest.mark.parametrize("kind", [cf.REDUCESCATTER, cf.ALLREDUCE])
def test_twonode_reductions(kind):
    w = cf.with_greedy(cf.as_reduction(cf.twonode16_ag(), kind))
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 8, 0, 1024, opts, plan.prio_stride)
    check(plan, ref, routes, prio, w.name)


@pytest.mark.parametrize("make,n", [
    (lambda: cf.with_greedy(cf.full_a2a(4)), 300),
    (lambda: cf.with_greedy(replace(cf.full_a2a(6), chunks_per_rank=2)), 300),
    (lambda: cf.with_greedy(cf.switch16_a2a()), 512),
    (lambda: cf.with_greedy(cf.two_node_rings_a2a(4, contiguity=0)), 300)])
def test_alltoall(make, n):
    """Alltoall: a chunk's hops are ready one after the other."""
    w = make()
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 11, 0, n, opts, plan.prio_stride)
    check(plan, ref, routes, prio, f"{w.name} alltoall greedy")


def test_alltoall_unrouted_and_equal_priorities():
    w = cf.with_greedy(cf.switch16_a2a())
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 12, 0, 256, opts, plan.prio_stride)
    rng = np.random.default_rng(5)
    routes[rng.random(routes.shape) < 0.01] = 0xFF
    prio[:128] = 7
    mk, ok = check(plan, ref, routes, prio, "switch16 greedy unrouted / equal priorities")
    assert not ok.all()


@pytest.mark.parametrize("order", [1, 2])
@pytest.mark.parametrize("make,n", [
    (lambda: cf.full_a2a(40, chunk_bytes=65536), 64),
    (lambda: cf.two_node_rings_a2a(8, contiguity=0), 64),
    (lambda: replace(cf.full_a2a(24, chunk_bytes=65536), chunks_per_rank=3), 48),
    (lambda: cf.fournode64_a2a(n_candidates=16), 16)])
def test_alltoall_block_kernel(make, n, order):
    """Plans beyond a wavefront's lists (more than 1024 send slots) run one
    block per candidate."""
    w = make()
    w = cf.with_greedy(w) if order == 1 else cf.with_reverse_greedy(w)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 13, 0, n, opts, plan.prio_stride)
    rng = np.random.default_rng(n + order)
    routes[rng.random(routes.shape) < 0.002] = 0xFF
    prio[1::2] = 4
    check(plan, ref, routes, prio, f"{w.name} alltoall greedy, block kernel")


@pytest.mark.parametrize("name", cf.GREEDY_LARGE_ORDER)
def test_full_batch_sampled(name):
    """The whole batch in the benchmark's launch shape; 256 sampled
    candidates (first, last, and a seeded spread over the batch) against
    the oracle, on every host thread."""
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed, 0, w.n_candidates, opts, plan.prio_stride)
    say(f"[gpu] {name}: full batch N={w.n_candidates}")
    mk, ok = plan.eval(routes, prio)
    idx = np.unique(np.r_[0, w.n_candidates - 1,
                          np.random.default_rng(3).choice(np.arange(1, w.n_candidates - 1), 254,
                                                          replace=False)])
    assert idx.size == 256
    say(f"[gpu] {name}: oracle on {idx.size} sampled candidates")
    rmk, rok = ref.eval_threads(routes[idx], prio[idx])
    assert (mk[idx] == rmk).all() and (ok[idx] == rok).all()
    assert ok.all()


@pytest.mark.parametrize("order", [1, 2])
def test_alltoall_block_kernel_two_word_keys(order):
    """The block kernel packs (start - previous window start, key rank,
    priority, chunk) into one word when the relative start (below 2 c_min +
    c_max), the key rank and the chunk fit 32 bits together; 16 MiB chunks
    on 1600 chunks do not fit, so the windows take the two-word minima."""
    w = cf.full_a2a(40, chunk_bytes=16 << 20)
    w = cf.with_greedy(w) if order == 1 else cf.with_reverse_greedy(w)
    plan, ref, opts = plans(w)
    cost = [int(x) for x in plan.link_costs()]
    assert (2 * min(cost) + max(cost)).bit_length() + (plan.num_chunks - 1).bit_length() > 32
    routes, prio = generate(w.seed + 14, 0, 48, opts, plan.prio_stride)
    prio[::3] = 9
    check(plan, ref, routes, prio, f"full40 16 MiB alltoall greedy order={order}")


@pytest.mark.parametrize("order", [1, 2])
def test_alltoall_block_kernel_unstaged_priorities(order):
    """A bidirectional 30-rank ring, shortest routes, four chunks per pair:
    3600 chunks (four per thread of the block kernel, its largest shape) and
    27000 sends, more than the kernel stages in LDS (it stages a candidate's
    priorities while two blocks still fit a CU), so the priorities are read
    hop by hop; keys of up to 15 hops need two words."""
    row_ptr, col, a, b = cf.csr_from_edges(30, cf.ring_edges(list(range(30)), 700, 46))
    w = cf.Workload("ring30_a2a", 30, 30, row_ptr, col, a, b, None, cf.ALLTOALL, 4, 65536,
                    cf.SHORTEST_ONLY, k=1, order=order)
    plan, ref, opts = plans(w)
    assert plan.num_chunks == 3600 and 4 * plan.info["max_sends"] > 80 * 1024
    routes, prio = generate(w.seed + 15, 0, 2, opts, plan.prio_stride)
    prio[:, ::7] = 3
    check(plan, ref, routes, prio, f"ring30 cpr=4 alltoall greedy order={order}")


@pytest.mark.parametrize("make", [
    # more than 4096 chunks (4 per thread of a 1024-thread block)
    lambda: cf.with_greedy(replace(cf.fournode64_a2a(n_candidates=2), chunks_per_rank=2)),
    lambda: cf.with_greedy(replace(cf.full_a2a(24, chunk_bytes=4096), chunks_per_rank=15)),
])
def test_alltoall_too_large_refused(make):
    """Greedy Alltoall plans beyond the block kernel's largest shape: refused,
    not approximated."""
    from paper_2111_04867_amd.binding import Plan, TacclError
    w = make()
    plan = Plan.from_workload(w)
    assert plan.num_chunks > 4096
    routes, prio = generate(1, 0, 2, plan.route_options(), plan.prio_stride)
    with pytest.raises(TacclError) as e:
        plan.eval(routes, prio)
    assert "greedy" in str(e.value)


# ---- greedy in reverse path order --------------------------------------------
# multicast plans run it on the general kernel, Alltoall on the greedy kernel


@pytest.mark.parametrize("make,n", [
    (lambda: cf.cubemesh8_ag(), 512),
    (lambda: cf.twonode16_ag(), 256),
    (lambda: cf.as_reduction(cf.twonode16_ag(), cf.REDUCESCATTER), 256),
    (lambda: cf.as_reduction(cf.twonode16_ag(), cf.ALLREDUCE), 128),
    (lambda: cf.as_reduction(cf.full_ag(4, k=3, chunks_per_rank=3), cf.ALLREDUCE), 400),
    (lambda: cf.full_ag(6, k=3, chunks_per_rank=2), 300),
    (lambda: cf.explicit_multicast(cf.cubemesh8_ag(), [0, 3, 5, 5, 7],
                                   [[1, 2], [0, 4, 6], [1, 3, 7], [2], [0, 1, 2, 3, 4, 5, 6]]),
     400),
    (lambda: cf.full_a2a(4), 300),
    (lambda: replace(cf.full_a2a(6), chunks_per_rank=2), 300),
    (lambda: cf.switch16_a2a(), 512),
    (lambda: cf.two_node_rings_a2a(4, contiguity=0), 300)])
def test_reverse_path_order(make, n):
    w = cf.with_reverse_greedy(make())
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 21, 0, n, opts, plan.prio_stride)
    rng = np.random.default_rng(n)
    routes[rng.random(routes.shape) < 0.01] = 0xFF
    prio[::3] = 11
    check(plan, ref, routes, prio, f"{w.name} reverse path order")


def test_reverse_path_order_differs_from_path_order():
    """The two greedy directions give different orders on twonode16_ag."""
    w = cf.twonode16_ag()
    fwd, rev = plans(cf.with_greedy(w)), plans(cf.with_reverse_greedy(w))
    routes, prio = generate(w.seed, 0, 128, fwd[2], fwd[0].prio_stride)
    m1, _ = check(fwd[0], fwd[1], routes, prio, "twonode16 path order")
    m2, _ = check(rev[0], rev[1], routes, prio, "twonode16 reverse path order")
    assert (m1 != m2).any()
