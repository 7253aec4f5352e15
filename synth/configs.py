"""The five synthetic workloads the hot path is checked and measured on.

They stand in for the paper's six public interaction datasets (Section VII-A,
dataset table), which are not available here: the shapes mirror them
(bipartite user-item streams, skewed hub-heavy streams, large streams), and no
record of any dataset is reproduced.  Dimensions and batch sizes are fixed by
the workload definitions below; the paper itself states none.
"""

from dataclasses import dataclass


@dataclass(frozen=True)
class Workload:
    cid: int                 # workload id (1..5)
    name: str
    n_nodes: int
    n_events: int
    src_rule: str            # "uniform" | "zipf" | "uniform_src" (bipartite sources)
    dst_rule: str            # "uniform" | "zipf" | "zipf_dst" (bipartite destinations)
    zipf_s: float            # Zipf exponent (ignored for uniform rules)
    n_src: int               # bipartite: sources are [0, n_src), destinations [n_src, n_nodes)
    t_rule: str              # "uniform_sorted": sort(U[0,1e5)); "exp_gaps": cumsum(Exp(mean 15))
    d_edge: int
    d_mem: int
    d_time: int
    d_attn: int
    n_heads: int
    batch: int
    k: int
    dtype: str               # storage dtype of memory/weights/messages: "f32" | "bf16"
    replay_p: float          # P(event is a replayed cache event)
    prune_p: float           # P(replay event is pruned)
    neg_rule: str            # "all": uniform over nodes; "dst": uniform over destinations
    stream_cid: int          # workload whose event stream is reused (5 reuses 3)
    window_b0: int           # first batch index of the mid-stream parity/bench window

    @property
    def d_msg(self) -> int:
        return 2 * self.d_mem + self.d_time + self.d_edge

    @property
    def d_kv(self) -> int:
        return self.d_mem + self.d_edge + self.d_time

    @property
    def d_q(self) -> int:
        return self.d_mem + self.d_time

    @property
    def n_batches(self) -> int:
        return (self.n_events + self.batch - 1) // self.batch


WORKLOADS = {
    1: Workload(1, "tiny-uniform-1k", 1_000, 20_000, "uniform", "uniform", 0.0, 0,
                "uniform_sorted", 16, 32, 32, 32, 1, 200, 5, "f32", 0.0, 0.0, "all", 1, 0),
    2: Workload(2, "bipartite-zipf1.0-9k", 9_000, 160_000, "uniform_src", "zipf_dst", 1.0, 8_000,
                "exp_gaps", 172, 100, 100, 100, 2, 600, 10, "f32", 0.0, 0.0, "dst", 2, 0),
    3: Workload(3, "skewed-zipf1.2-1M", 1_000_000, 10_000_000, "zipf", "zipf", 1.2, 0,
                "uniform_sorted", 0, 100, 100, 100, 2, 4_000, 10, "f32", 0.0, 0.0, "all", 3, 100),
    4: Workload(4, "large-zipf0.8-10M", 10_000_000, 100_000_000, "zipf", "zipf", 0.8, 0,
                "uniform_sorted", 16, 100, 100, 100, 2, 60_000, 20, "f32", 0.0, 0.0, "all", 4, 800),
    5: Workload(5, "partition-share-replay-bf16", 1_000_000, 10_000_000, "zipf", "zipf", 1.2, 0,
                "uniform_sorted", 0, 100, 100, 100, 2, 60_000, 20, "bf16", 0.25, 0.10, "all", 3, 100),
}


def workload(cid: int) -> Workload:
    return WORKLOADS[int(cid)]
