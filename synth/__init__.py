"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle's callers.

This package builds graphs (stochastic block model, Chung-Lu, batches of small
graphs) and dense feature tensors.  It holds none of the attention, reorder or tiling arithmetic: both the
HIP path and the oracle receive what is produced here as plain arrays.
"""

from .graphs import (  # noqa: F401
    Graph,
    batched_graphs,
    sbm_graph,
    chung_lu_graph,
    csr_from_pairs,
    lognormal_block_sizes,
)
from .tensors import bf16_round, bf16_bits, normal_tensor  # noqa: F401
from .workloads import WORKLOADS, make_workload, Workload  # noqa: F401
