"""Plain fp64 / integer CPU oracle for graph-topology sparse attention.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, links or runs
this package: it is used by ``tests/``, by the smoke check and by the
benchmark's CPU baseline leg, and it shares no code, tables or constants with
the HIP library.  Each function states the passage of the paper (TorchGT,
arXiv 2407.14106) it follows; where the paper is silent the reading taken is
stated in the function's docstring.

Modules:

* ``attention`` - neighbour-restricted softmax attention (§3.2, local
  topology-induced pattern) and full softmax attention (§2.1, Eq. 1), forward
  and backward, written out from their definitions in fp64.
* ``reorder`` - the cluster reordering of §3.3 in the deterministic
  label-propagation reading used instead of METIS.
* ``plan`` - relabelled CSR and the tile classification of §3.4 (cluster
  sparsity, transfer threshold), as plain integer array code.
* ``ecr`` - the paper's lossy reformation of sparse clusters into sub-blocks
  and the Auto Tuner that walks its transfer threshold (§3.4).
* ``interleave`` - the checks of conditions C1-C3 that decide when a dense
  layer is interleaved (§3.2).
"""

from . import attention, ecr, interleave, plan, reorder  # noqa: F401
