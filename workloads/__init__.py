"""Seeded synthetic inputs shared by the oracle tests and the GPU path.

Holds workload descriptors (topology, collective, sketch, batch size, seed)
and the counter-based candidate generator; none of the evaluation's
arithmetic lives here.
"""
from .configs import (ALLGATHER, ALLTOALL, EXPLICIT, HIER_RELAY, KSHORTEST, NAMED, ORDER,  # noqa
                      RELAY1, SHORTEST_ONLY, Workload, named)
from .candgen import build_candgen, generate  # noqa: F401
