"""Seeded synthetic inputs shared by the oracle tests and the GPU path.

Holds workload descriptors (topology, collective, sketch, batch size, seed)
and the counter-based candidate generator; none of the evaluation's
arithmetic lives here.
"""
from .configs import (ALLGATHER, ALLREDUCE, ALLTOALL, CONTIG_ORDER, EXPLICIT,  # noqa: F401
                      GREEDY_LARGE_ORDER, GREEDY_ORDER, HIER_RELAY, KSHORTEST, NAMED, ORDER,
                      PORTS_ORDER, REDUCE_ORDER, REDUCESCATTER, RELAY1, SHORTEST_ONLY, Workload,
                      as_reduction, named, random_workload, random_workload_large,
                      with_contiguity, with_greedy,
                      with_reverse_greedy, with_switch_ports)
from .candgen import build_candgen, generate  # noqa: F401
