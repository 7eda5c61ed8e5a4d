"""CPU oracle for ClusterAttention (test infrastructure only).

Only tests/, the smoke check in __graft_entry__ and the bench's CPU-baseline
leg may import this package. The HIP library never calls it.
"""
from . import ref  # noqa: F401
