"""Seeded synthetic inputs shared by the oracle tests and the GPU path.

Holds workload descriptors (topology, collective, sketch, batch size, seed)
and the counter-based candidate generator; none of the evaluation's
arithmetic lives here.
"""
from .configs import (ALLGATHER, ALLTOALL, CONTIG_ORDER, EXPLICIT, HIER_RELAY, KSHORTEST,  # noqa
                      NAMED, ORDER, RELAY1, SHORTEST_ONLY, Workload, named, with_contiguity)
from .candgen import build_candgen, generate  # noqa: F401
