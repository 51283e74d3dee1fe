"""Named synthetic workloads (stand-ins for the paper's OGB inputs, Table 2).

Each preset fixes the graph recipe (Chung-Lu power law, seed 0), the
random-range partitioning, the feature shape, the seed schedule, the
GraphSAGE fanout (hop-first: the first entry is sampled around the seeds) and
the prefetch-buffer parameters (f as integer percent of the halo, decay
gamma, eviction interval delta) of section IV-B.

The paper's datasets (arxiv, products, papers100M) are not available; these
graphs only reproduce their size, mean degree and a power-law degree tail.
"""
from dataclasses import dataclass, field, replace
from typing import Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    n: int                 # nodes of the whole graph
    beta: float            # Chung-Lu degree exponent
    mean_deg: float        # mean degree (mean out-degree when sym)
    sym: bool              # directed draw, then symmetrised
    parts: int             # random-range partitions; partition 0 is local
    d: int                 # feature dimension
    dtype: str             # "f32" | "bf16"
    train_pct: int         # percent of local nodes that are seeds
    batch: int             # seeds per minibatch
    fanout: Tuple[int, ...]  # hop-first fanout
    buffer_pct: int        # f_p^h, integer percent of the halo
    gamma: float           # decay factor
    delta: int             # eviction interval
    steps: int             # minibatches in the stated run
    seed: int = 0          # graph / partition / feature / schedule seed
    philox_seed: int = 0   # sampler key
    note: str = ""

    @property
    def row_bytes(self) -> int:
        return self.d * (4 if self.dtype == "f32" else 2)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    # 10K-node power law, 4 partitions: small enough for brute-force checks.
    "cl10k": Workload("cl10k", 10_000, 2.1, 10.0, False, 4, 64, "f32", 10, 256,
                      (25, 10), 25, 0.95, 8, 50, note="none (CPU-oracle scale)"),
    # arxiv-sized: 170K nodes, ~1.17M directed edges, 8 partitions.
    "cl170k": Workload("cl170k", 170_000, 2.2, 7.0, True, 8, 128, "f32", 50, 1024,
                       (15, 10, 5), 25, 0.95, 16, 200, note="arxiv (Table 2)"),
    # products-sized: 2.45M nodes, ~62M undirected edges, 16 partitions.
    "cl2m45": Workload("cl2m45", 2_450_000, 2.0, 50.0, False, 16, 100, "f32", 8, 2000,
                       (15, 10, 5), 25, 0.95, 32, 7, note="products (Table 2)"),
    # same graph, bf16 rows and a stress eviction setting.
    "cl2m45_bf16": Workload("cl2m45_bf16", 2_450_000, 2.0, 50.0, False, 16, 100, "bf16", 8, 4096,
                            (20, 15, 10), 50, 0.8, 4, 3, note="products (Table 2), stress eviction"),
    # papers-sized share: partition 0 of 64 of a 111M-node, ~1.6B-edge graph.
    "cl111m_p64": Workload("cl111m_p64", 111_000_000, 1.9, 29.0, False, 64, 128, "f32", 1, 1024,
                           (15, 10, 5), 25, 0.95, 32, 17, note="one of 64 partitions of papers (Table 2)"),
}


def get(name: str) -> Workload:
    return WORKLOADS[name]
