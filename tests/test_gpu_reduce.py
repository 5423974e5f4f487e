"""GPU parity of ReduceScatter and Allreduce (Allgather trees run backwards,
then forwards; Sec. 5.2) against the oracle, bit for bit, through the C ABI.
Needs an MI355X."""
import numpy as np
import pytest

from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


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
    opts = plan.route_options()
    assert (opts == ref.route_options()).all()
    assert plan.prio_stride == ref.prio_stride
    return plan, ref, opts


def check(plan, ref, routes, prio, label):
    say(f"[gpu] {label}: {routes.shape[0]} candidates")
    mk, ok = plan.eval(routes, prio)
    rmk, rok = ref.eval_threads(routes, prio)
    bad = np.nonzero((mk != rmk) | (ok != rok))[0]
    assert bad.size == 0, (f"{label}: {bad.size} mismatches, first at {bad[:5].tolist()}: "
                           f"gpu {mk[bad[:5]].tolist()} oracle {rmk[bad[:5]].tolist()}")
    return mk, ok


@pytest.mark.parametrize("name", cf.REDUCE_ORDER)
def test_full_size_parity(name):
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed, 0, w.n_candidates, opts, plan.prio_stride)
    mk, ok = check(plan, ref, routes, prio, f"{name} full N={w.n_candidates}")
    assert ok.all()


@pytest.mark.parametrize("name", cf.REDUCE_ORDER)
@pytest.mark.parametrize("n", [1, 63, 257])
def test_ragged_batches(name, n):
    w = cf.named(name)
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 50, 9, n, opts, plan.prio_stride)
    check(plan, ref, routes, prio, f"{name} n={n}")


@pytest.mark.parametrize("kind,want", [(cf.REDUCESCATTER, 2 * 48935), (cf.ALLREDUCE, 4 * 48935)])
def test_ring4_closed_form(kind, want):
    w = cf.as_reduction(cf.ring4_ag(), kind)
    plan, ref, opts = plans(w)
    routes, prio = generate(2, 0, 256, opts, plan.prio_stride)
    mk, ok = check(plan, ref, routes, prio, w.name)
    assert ok.all() and (mk == want).all()


@pytest.mark.parametrize("kind", [cf.REDUCESCATTER, cf.ALLREDUCE])
@pytest.mark.parametrize("cpr", [1, 3])
def test_full4(kind, cpr):
    w = cf.as_reduction(cf.full_ag(4, k=3, chunks_per_rank=cpr), kind)
    plan, ref, opts = plans(w)
    routes, prio = generate(61 + cpr, 0, 1000, opts, plan.prio_stride)
    check(plan, ref, routes, prio, f"{w.name} cpr={cpr}")


@pytest.mark.parametrize("kind", [cf.REDUCESCATTER, cf.ALLREDUCE])
def test_with_contiguous_transfers(kind):
    w = cf.with_contiguity(cf.as_reduction(cf.twonode16_ag(), kind))
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 3, 0, 2048, opts, plan.prio_stride)
    check(plan, ref, routes, prio, w.name)
    w2 = cf.two_node_full(2, cf.ALLGATHER, chunks_per_rank=2)
    w2 = cf.as_reduction(w2, kind)
    w2.contiguity = 1
    plan, ref, opts = plans(w2)
    routes, prio = generate(71, 0, 500, opts, plan.prio_stride)
    check(plan, ref, routes, prio, w2.name + "_contig")


@pytest.mark.parametrize("value", [0, 0xFFFFFFFF])
def test_equal_priorities(value):
    w = cf.named("twonode16_ar")
    plan, ref, opts = plans(w)
    routes, prio = generate(w.seed + 5, 0, 128, opts, plan.prio_stride)
    prio[:] = value
    check(plan, ref, routes, prio, f"twonode16_ar prio={value:#x}")


@pytest.mark.parametrize("kind", [cf.REDUCESCATTER, cf.ALLREDUCE])
def test_plans_outside_the_layered_kernel(kind):
    """Three ranks: not a multiple of 4, so the general kernel's variant."""
    w = cf.as_reduction(cf.full_ag(3, k=2), kind)
    plan, ref, opts = plans(w)
    routes, prio = generate(1, 0, 200, opts, plan.prio_stride)
    prio[::2, ::2] = 3
    check(plan, ref, routes, prio, f"full3 kind={kind}")


@pytest.mark.parametrize("kind", [cf.REDUCESCATTER, cf.ALLREDUCE])
@pytest.mark.parametrize("skew", [0, 30])
def test_reverse_link_costs(kind, skew):
    """Two fully connected quads joined rank by rank. With skew 0 every link's
    reverse costs the same, so the ranked kernel runs the ReduceScatter; with
    a skew the reverse links cost more (reversed path sums leave the set the
    path codes cover) and the layered kernel runs it."""
    edges = []
    for u in range(8):
        for v in range(8):
            if u != v and (u // 4 == v // 4 or u % 4 == v % 4):
                edges.append((u, v, 700, 46 + (skew if u < v else 0)))
    row_ptr, col, a, b = cf.csr_from_edges(8, edges)
    w = cf.Workload(f"quads8_skew{skew}", 8, 8, row_ptr, col, a, b, None, kind, 2, 65536,
                    cf.KSHORTEST, k=3)
    plan, ref, opts = plans(w)
    routes, prio = generate(11 + skew, 0, 512, opts, plan.prio_stride)
    prio[::3, ::5] = 7
    check(plan, ref, routes, prio, f"quads8 skew={skew} kind={kind}")
