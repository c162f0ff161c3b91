"""The named workloads (graph + tensor recipes) and scaled-down variants.

Recipes (seed = 1000 + workload number for the c workloads, 2000 + number for
the b workloads; node order shuffled in every c graph, batch order kept in the
b graphs):

* ``c1``: SBM, 4,096 nodes, 16 equal blocks, average degree 8, 10% of pairs
  across blocks; Q,K,V fp32 [4096, 1, 64]; forward only.
* ``c2``: SBM, 100,000 nodes, 200 equal blocks, degree 16, 15% across;
  Q,K,V,dO bf16 [100000, 8, 64]; forward and backward.
* ``c3``: Chung-Lu, 1,000,000 nodes, exponent 2.1, degree 12, expected degree
  capped at 20,000; bf16 [1M, 4, 32]; forward, backward, reorder, tile build.
* ``c4``: SBM, 1,000,000 nodes, 1,000 log-normal blocks (sigma 0.5), degree
  30, 5% across; bf16 [1M, 8, 32]; 128-wide tiles at densities 1%, 5%, 20%.
* ``c5``: SBM, 65,536 nodes, 256 equal blocks, degree 20, 10% across;
  bf16 [65536, 8, 64]; a sparse layer then a full dense layer.
* ``b1``: graph-level batch of molecule-sized graphs (23 to 26 nodes, degree
  2.2: a spanning tree plus a few ring closures), 40,000 graphs, plus a
  global token attending to and attended by every node; bf16 [N, 8, 32].
* ``b2``: graph-level batch of call-graph-sized graphs (log-normal sizes with
  mean 15,378 nodes, degree 4.57), 64 graphs, plus a global token; bf16
  [N, 8, 32].

``scale`` shrinks the node count (and block count, keeping block sizes) so the
same recipe can run at oracle-friendly sizes.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .graphs import Graph, batched_graphs, chung_lu_graph, lognormal_block_sizes, sbm_graph
from .tensors import normal_tensor


@dataclass
class Workload:
    name: str
    graph: Graph
    heads: int
    dim: int
    dtype: str  # "f32" | "bf16"
    backward: bool
    tile: int
    taus: tuple
    seed: int
    description: str

    def tensors(self, with_grad: bool | None = None):
        """Q, K, V (and dO when the workload has a backward pass) as fp32 numpy arrays."""
        shape = (self.graph.n, self.heads, self.dim)
        q = normal_tensor(shape, (self.seed, 0), self.dtype)
        k = normal_tensor(shape, (self.seed, 1), self.dtype)
        v = normal_tensor(shape, (self.seed, 2), self.dtype)
        want = self.backward if with_grad is None else with_grad
        do = normal_tensor(shape, (self.seed, 3), self.dtype) if want else None
        return q, k, v, do

    def edge_bias(self) -> np.ndarray:
        """A per-edge, per-head additive bias: fp32 N(0, 1) draws [nnz, heads] in the graph's CSR order."""
        return normal_tensor((self.graph.nnz, self.heads), (self.seed, 4), "f32")


def _equal_blocks(n: int, nb: int) -> np.ndarray:
    base = np.full(nb, n // nb, dtype=np.int64)
    base[: n - int(base.sum())] += 1
    return base


WORKLOADS = {
    "c1": dict(n=4096, kind="sbm", blocks=16, degree=8, cross=0.10, heads=1, dim=64, dtype="f32",
               backward=False, tile=128, taus=(0.01,)),
    "c2": dict(n=100_000, kind="sbm", blocks=200, degree=16, cross=0.15, heads=8, dim=64, dtype="bf16",
               backward=True, tile=128, taus=(0.01,)),
    "c3": dict(n=1_000_000, kind="chung_lu", gamma=2.1, degree=12, cap=20_000, heads=4, dim=32,
               dtype="bf16", backward=True, tile=128, taus=(0.01,)),
    "c4": dict(n=1_000_000, kind="sbm_lognormal", blocks=1000, sigma=0.5, degree=30, cross=0.05, heads=8,
               dim=32, dtype="bf16", backward=True, tile=128, taus=(0.01, 0.05, 0.20)),
    "c5": dict(n=65_536, kind="sbm", blocks=256, degree=20, cross=0.10, heads=8, dim=64, dtype="bf16",
               backward=True, tile=128, taus=(0.01,)),
    "b1": dict(n=1_000_000, kind="batched", graphs=40_000, size_lo=23, size_hi=26, degree=2.2, token=True,
               heads=8, dim=32, dtype="bf16", backward=True, tile=128, taus=(0.01, 0.05)),
    "b2": dict(n=1_000_000, kind="batched_lognormal", graphs=64, size_mean=15_378, sigma=0.8, degree=4.57,
               token=True, heads=8, dim=32, dtype="bf16", backward=True, tile=128, taus=(0.05,)),
}


def make_workload(name: str, scale: float = 1.0) -> Workload:
    """Build workload ``name``; ``scale < 1`` shrinks N (blocks shrink in number, not size)."""
    spec = WORKLOADS[name]
    seed = (1000 if name[0] == "c" else 2000) + int(name[1:])
    n = max(64, int(round(spec["n"] * scale)))
    kind = spec["kind"]
    if kind == "sbm":
        nb = max(1, int(round(spec["blocks"] * n / spec["n"])))
        g = sbm_graph(_equal_blocks(n, nb), spec["degree"], spec["cross"], seed)
        desc = f"SBM n={n} blocks={nb} deg={spec['degree']} cross={spec['cross']}"
    elif kind == "sbm_lognormal":
        nb = max(1, int(round(spec["blocks"] * n / spec["n"])))
        sizes = lognormal_block_sizes(n, nb, spec["sigma"], seed + 1)
        g = sbm_graph(sizes, spec["degree"], spec["cross"], seed)
        desc = f"SBM n={n} lognormal blocks={nb} sigma={spec['sigma']} deg={spec['degree']} cross={spec['cross']}"
    elif kind == "chung_lu":
        cap = min(spec["cap"], max(2, n // 50))
        g = chung_lu_graph(n, spec["gamma"], spec["degree"], cap, seed)
        desc = f"Chung-Lu n={n} gamma={spec['gamma']} deg={spec['degree']} cap={cap}"
    elif kind == "batched":
        rng = np.random.Generator(np.random.PCG64(seed + 1))
        ng = max(1, int(round(spec["graphs"] * scale)))
        sizes = rng.integers(spec["size_lo"], spec["size_hi"] + 1, size=ng)
        g = batched_graphs(sizes, spec["degree"], seed, global_token=spec["token"])
        desc = (f"batch of {ng} graphs of {spec['size_lo']}-{spec['size_hi']} nodes, deg={spec['degree']}"
                f"{', global token' if spec['token'] else ''}")
    elif kind == "batched_lognormal":
        rng = np.random.Generator(np.random.PCG64(seed + 1))
        ng = max(1, int(round(spec["graphs"] * scale)))
        mu = np.log(spec["size_mean"]) - spec["sigma"] ** 2 / 2
        sizes = np.maximum(2, np.round(rng.lognormal(mu, spec["sigma"], size=ng))).astype(np.int64)
        g = batched_graphs(sizes, spec["degree"], seed, global_token=spec["token"])
        desc = (f"batch of {ng} graphs, log-normal sizes mean {spec['size_mean']} sigma {spec['sigma']}, "
                f"deg={spec['degree']}{', global token' if spec['token'] else ''}")
    else:
        raise ValueError(kind)
    return Workload(name=name, graph=g, heads=spec["heads"], dim=spec["dim"], dtype=spec["dtype"],
                    backward=spec["backward"], tile=spec["tile"], taus=tuple(spec["taus"]), seed=seed,
                    description=desc)
