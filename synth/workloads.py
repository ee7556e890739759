"""The synthetic workloads with every integer the method needs written out: the five stated
workloads C1..C5, and X1, short summarization prompts with the paper's small clusters (cluster
size 8 at the coarse level and 4 at the fine level, i.e. fine clusters of 4 tokens, fan-out 2).

Budgets are given as ratios in the workload descriptions; the integers below follow the rounding
readings documented with the oracle (window rows, kept tokens as whole clusters, level-1 keeps
half of the super-clusters when the final ratio is below 0.5, level-2 count in clusters of the
post-eviction cache). ``tests/test_oracle_pins.py`` re-derives each integer from the oracle's
rule functions, so this table cannot drift from them.
"""
from dataclasses import dataclass, replace

SEED_BASE = 0x4D504331  # "MPC1"


@dataclass(frozen=True)
class Workload:
    name: str
    n_layers: int
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str
    T: int                 # prompt tokens in the prefill cache
    window: int            # window query rows used for static scoring
    keep: int              # tokens kept by static eviction (T_s)
    local_keep: int        # most recent tokens always kept
    cluster: int           # tokens per cluster (s)
    fanout: int            # clusters per super-cluster (f)
    k_super: int           # level-1 budget (super-clusters)
    k_clusters: int        # level-2 budget (clusters)
    share_period: int      # layers sharing one selection (1 = no sharing)
    steps: int             # decode steps with fresh queries
    static_ratio: float    # kept fraction, as stated
    dynamic_ratio: float   # selected fraction of the kept cache, as stated
    seed: int
    seq_stride: int = 0    # per-sequence seed offset (independent sequences)
    n_outlier: int = 0
    outlier_scale: float = 1.0
    rope: bool = False
    rope_base: float = 10000.0
    n_sinks: int = 0
    hh_count: int = 0
    hh_span: int = 1
    hh_lo: int = 0
    hh_hi: int = 0
    share_start: int = 2   # the first two layers never share

    @property
    def group(self):
        return self.n_q_heads // self.n_kv_heads

    @property
    def n_clusters(self):
        return -(-self.keep // self.cluster)

    @property
    def n_super(self):
        return -(-self.n_clusters // self.fanout)

    @property
    def elt(self):
        return 4 if self.dtype == "fp32" else 2

    def with_(self, **kw):
        return replace(self, **kw)


WORKLOADS = {
    "C1": Workload(
        name="tiny-1L-12H-d64-T512-fp32", n_layers=1, batch=1, n_q_heads=12, n_kv_heads=12,
        head_dim=64, dtype="fp32", T=512, window=102, keep=256, local_keep=32, cluster=16,
        fanout=4, k_super=4, k_clusters=8, share_period=1, steps=1, static_ratio=0.5,
        dynamic_ratio=0.5, seed=SEED_BASE + 0, n_sinks=4, hh_count=16, hh_span=1, hh_lo=4,
        hh_hi=512 - 32),
    "C2": Workload(
        name="gpt2-12L-12H-d64-T2048-fp16", n_layers=12, batch=1, n_q_heads=12, n_kv_heads=12,
        head_dim=64, dtype="fp16", T=2048, window=409, keep=1024, local_keep=32, cluster=16,
        fanout=4, k_super=8, k_clusters=8, share_period=2, steps=64, static_ratio=0.5,
        dynamic_ratio=0.125, seed=SEED_BASE + 1, n_outlier=4, outlier_scale=8.0),
    "C3": Workload(
        name="llama2-7b-32L-32H-d128-T8192-bf16", n_layers=32, batch=1, n_q_heads=32,
        n_kv_heads=32, head_dim=128, dtype="bf16", T=8192, window=1638, keep=4096, local_keep=32,
        cluster=32, fanout=8, k_super=8, k_clusters=12, share_period=4, steps=128,
        static_ratio=0.5, dynamic_ratio=0.10, seed=SEED_BASE + 2, n_outlier=4, outlier_scale=8.0,
        rope=True),
    "C4": Workload(
        name="llama2-7b-32L-32H-d128-B4-T32768-bf16", n_layers=32, batch=4, n_q_heads=32,
        n_kv_heads=32, head_dim=128, dtype="bf16", T=32768, window=3276, keep=9824,
        local_keep=32, cluster=32, fanout=8, k_super=20, k_clusters=15, share_period=4, steps=64,
        static_ratio=0.30, dynamic_ratio=0.05, seed=SEED_BASE + 3, seq_stride=1000, n_outlier=4,
        outlier_scale=8.0, rope=True),
    "C5": Workload(
        name="gqa-32L-32Hq-8Hkv-d128-T131072-bf16", n_layers=32, batch=1, n_q_heads=32,
        n_kv_heads=8, head_dim=128, dtype="bf16", T=131072, window=13107, keep=32768,
        local_keep=32, cluster=64, fanout=8, k_super=32, k_clusters=10, share_period=4, steps=32,
        static_ratio=0.25, dynamic_ratio=0.02, seed=SEED_BASE + 4, n_outlier=4, outlier_scale=8.0,
        rope=True, n_sinks=8, hh_count=64, hh_span=128, hh_lo=8, hh_hi=131072 - 32),
    # short summarization prompts (the paper's XSUM setting: coarse clusters of 8 tokens over fine
    # clusters of 4, a 10% budget, pairs of layers sharing), 8 independent sequences
    "X1": Workload(
        name="xsum-llama2-7b-32L-32H-d128-B8-T1024-bf16", n_layers=32, batch=8, n_q_heads=32,
        n_kv_heads=32, head_dim=128, dtype="bf16", T=1024, window=204, keep=512, local_keep=32,
        cluster=4, fanout=2, k_super=32, k_clusters=12, share_period=2, steps=64, static_ratio=0.5,
        dynamic_ratio=0.10, seed=SEED_BASE + 5, seq_stride=1000, n_outlier=4, outlier_scale=8.0,
        rope=True),
}


# Level-2 budgets with the dynamic ratio read against the prompt length T instead of the kept cache
# (the Fig. 9 caption speaks of the final budget of the KV cache): floor(eta * T / s) clusters, at most the
# candidates. The tiny workload states its budget (8 clusters) outright, so it keeps it.
K_CLUSTERS_OF_PROMPT = {"C1": 8, "C2": 16, "C3": 25, "C4": 51, "C5": 40, "X1": 25}


def get(name: str) -> Workload:
    """A workload by name; a trailing "-T" selects the reading of the dynamic ratio against the
    prompt length (e.g. "C2-T": 16 clusters per selection instead of 8)."""
    if name.endswith("-T"):
        base = name[:-2]
        w = WORKLOADS[base]
        return w.with_(name=w.name + "-eta-of-prompt", k_clusters=K_CLUSTERS_OF_PROMPT[base])
    return WORKLOADS[name]
