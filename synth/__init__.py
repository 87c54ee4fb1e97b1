"""Seeded synthetic inputs for NOVA-KV workloads.

This package is shared by the CPU oracle's tests and by the GPU path (tests,
smoke check and benchmark).  It holds no part of the method's arithmetic: only
random draws (Gaussian vectors with seeded SPD covariances, sink logits,
sequence lengths, block tables, code bytes) and their rounding to the storage
dtype the workload names.
"""

from .workloads import *  # noqa: F401,F403
