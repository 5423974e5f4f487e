"""The windowed time-aware greedy (App. B.2) of the GPU kernels, run on the
host under AddressSanitizer and UndefinedBehaviorSanitizer.

tests/greedy_host/greedy_host.cpp drives the library's own per-lane steps
(paper_2111_04867_amd/csrc/greedy_window.h: scan one link's pending sends
for the best ready one, commit a window's winners) for every lane of a
64-lane wavefront in turn, exactly as the kernels arrange them. Its inputs
are the sends of the oracle's schedule of each candidate, laid out as the
kernels lay them out (per-link record lists: travelled, ~remaining,
priority, slot | the slot of the send the chunk arrives by), and every
send's finish time must equal the oracle's greedy schedule.
"""
import os
import shutil
import struct
import subprocess

import numpy as np
import pytest

from oracle import OraclePlan
from workloads import configs as cf
from workloads import generate

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2111_04867_amd", "csrc")
NONE = 0xFFFFFFFF
NOPRED = 0xFFFF


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    if shutil.which("hipcc") is None:
        pytest.skip("hipcc is not installed")
    exe = str(tmp_path_factory.mktemp("greedy") / "greedy_host")
    san = []
    for flag in ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all",
                 "-fno-omit-frame-pointer"):
        san += ["-Xarch_host", flag]
    subprocess.run(["hipcc", "-x", "hip", "--cuda-host-only", "-O1", "-g", "-std=c++17",
                    "-I" + CSRC] + san + [os.path.join(HERE, "greedy_host", "greedy_host.cpp"),
                                          "-o", exe], check=True)
    return exe


def records(w, ref, sends, multicast, push=False):
    """Per-link record lists as the greedy kernels build them (push: a
    ReduceScatter, whose send out of v carries the partial on to the send
    out of its parent u)."""
    P, V = w.P, w.V
    cpr = w.chunks_per_rank
    H = ref.max_hops
    owner = {}
    recs = [[] for _ in range(w.E)]
    slot_of = {}
    n = len(sends["chunk"])
    for i in range(n):
        c, l, u, v = (int(sends[k][i]) for k in ("chunk", "link", "from", "to"))
        if multicast and push:
            o = c // cpr
            slot = c * V + u
            pred = NOPRED if v == o else c * V + v
        elif multicast:
            o = c // cpr
            slot = c * V + v
            pred = NOPRED if u == o else c * V + u
        else:
            h = int(sends["hop"][i])
            slot = c * H + h
            pred = NOPRED if h == 0 else c * H + h - 1
        slot_of[i] = slot
        rem, trav = int(sends["rem"][i]), int(sends["trav"][i])
        recs[l].append((trav, (~rem) & NONE, int(sends["prio"][i]), slot | (pred << 16)))
    gofs = np.cumsum([0] + [len(r) for r in recs])
    flat = [x for r in recs for x in r]
    nslots = (w.P * cpr * V) if multicast else (ref.num_chunks * H)
    return nslots, gofs, flat, slot_of


def run(harness, w, ref, routes, prio, multicast, push=False):
    mk, ok, sends = ref.eval_detail(routes, prio)
    nslots, gofs, flat, slot_of = records(w, ref, sends, multicast, push)
    cost = [ref.link_cost(e) for e in range(w.E)]
    cmin = min(cost)
    blob = struct.pack(f"<5I{w.E}I{w.E + 1}I", w.E, nslots, cmin, len(flat), int(push), *cost,
                       *gofs)
    blob += b"".join(struct.pack("<4I", *r) for r in flat)
    # the harness carries its own sanitizer runtime: drop a preloaded one
    # (the sanitizer leg of the CPU suite preloads clang's into this process)
    env = {k: v for k, v in os.environ.items() if k != "LD_PRELOAD"}
    env.update(ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    out = subprocess.run([harness], input=blob, capture_output=True, env=env)
    assert out.returncode == 0, out.stderr.decode()[-2000:]
    vals = [int(x) for x in out.stdout.split()]
    assert vals[0] == mk
    fin = vals[1:]
    for i, s in slot_of.items():
        assert fin[s] == int(sends["finish"][i]), (i, s)
    return mk


def rs(w):
    return cf.as_reduction(w, cf.REDUCESCATTER)


@pytest.mark.parametrize("make,n,multicast,push", [
    (lambda: cf.with_greedy(cf.cubemesh8_ag()), 40, True, False),
    (lambda: cf.with_greedy(cf.twonode16_ag()), 6, True, False),
    (lambda: cf.with_greedy(cf.full_ag(6, k=3, chunks_per_rank=2)), 20, True, False),
    (lambda: cf.with_greedy(cf.switch16_a2a()), 4, False, False),
    (lambda: cf.with_greedy(cf.full_a2a(5)), 20, False, False),
    (lambda: cf.with_greedy(rs(cf.cubemesh8_ag())), 40, True, True),
    (lambda: cf.with_greedy(rs(cf.twonode16_ag())), 6, True, True),
    (lambda: cf.with_greedy(rs(cf.full_ag(6, k=3, chunks_per_rank=2))), 20, True, True),
])
def test_window_steps_match_the_oracle(harness, make, n, multicast, push):
    w = make()
    ref = OraclePlan.from_workload(w)
    assert ref.order == 1
    routes, prio = generate(w.seed + 41, 0, n, ref.route_options(), ref.prio_stride)
    prio[1::3] = 7  # equal priorities: the slot breaks the tie
    spans = [run(harness, w, ref, routes[i], prio[i], multicast, push) for i in range(n)]
    assert len(set(spans)) > 1 or n < 4
