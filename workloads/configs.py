"""The five MoE-block workloads.

Each entry fixes the shape of one expert-parallel rank's share of a FarSkip
MoE block (Section 2.1 gives the MoE layer, Section 3 the FarSkip residual):
tokens routed by this rank, hidden size, experts, top-k, routing function,
expert and shared-expert FFN widths, EP size and the element type.
"""

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class MoEConfig:
    name: str
    n_tokens: int          # N: tokens this rank routes
    hidden: int            # d
    n_experts: int         # E: global routed experts
    top_k: int             # k
    ffn: int               # F: routed expert FFN width
    score: str             # "softmax" | "sigmoid"
    norm_topk: bool        # renormalise the k selected weights
    n_shared: int = 0      # S: always-on shared experts
    ffn_shared: int = 0    # width of each shared expert
    n_groups: int = 1      # G: expert groups for group-limited routing (1 = off)
    topk_groups: int = 1   # groups kept when G > 1
    routed_scale: float = 1.0
    ep_size: int = 1       # R
    ep_rank: int = 0       # r (this GPU)
    dtype: str = "bf16"    # "f32" | "bf16": x, weights, expert outputs, residual
    bias: str = "none"     # selection bias: "none" | "uniform" | "zipf"
    zipf_s: float = 1.2
    zipf_beta: float = 0.0
    seed: int = 0
    next_linear: bool = True   # a dense d x d linear stands in for the next layer
    # "a2a": each rank routes its own tokens and exchanges rows with
    # Dispatch / Combine; "allreduce": every rank holds all n_tokens tokens
    # (replicated activations), runs its own experts and the per-rank
    # partial sums are all-reduced (the inference variant)
    ep_mode: str = "a2a"

    @property
    def n_local(self):
        return self.n_experts // self.ep_size

    @property
    def cap(self):
        """Rows one source rank sends in total (every token sends k rows)."""
        return self.n_tokens * self.top_k

    @property
    def n_global_tokens(self):
        return self.n_tokens if self.ep_mode == "allreduce" else self.n_tokens * self.ep_size

    @property
    def n_sources(self):
        """Token sets this rank sees: its own (replicated) or one per rank."""
        return 1 if self.ep_mode == "allreduce" else self.ep_size

    @property
    def elem_bytes(self):
        return 4 if self.dtype == "f32" else 2

    def scaled(self, **kw):
        return replace(self, **kw)


CONFIGS = {
    # Tiny FarSkip block pair in fp32; the oracle finishes it in seconds.
    "tiny": MoEConfig(
        name="tiny", n_tokens=128, hidden=256, n_experts=8, top_k=2, ffn=512,
        score="softmax", norm_topk=True, dtype="f32", seed=1),
    # DeepSeek-V2-Lite-shaped layer: 64 experts top-6 softmax (no renorm),
    # 2 shared experts of width 1408.
    "dsv2lite": MoEConfig(
        name="dsv2lite", n_tokens=4096, hidden=2048, n_experts=64, top_k=6,
        ffn=1408, score="softmax", norm_topk=False, n_shared=2,
        ffn_shared=1408, dtype="bf16", seed=2),
    # Llama-4-Scout-shaped layer: 16 experts top-1 sigmoid, one shared
    # expert, a uniform(-0.1, 0.1) selection bias for uneven loads.
    "scout": MoEConfig(
        name="scout", n_tokens=8192, hidden=5120, n_experts=16, top_k=1,
        ffn=8192, score="sigmoid", norm_topk=False, n_shared=1,
        ffn_shared=8192, dtype="bf16", bias="uniform", seed=3),
    # DeepSeek-V3-shaped prefill, one rank of EP=8: 4096 own tokens,
    # 256 experts top-8 sigmoid with 8 groups / top-4 groups, one shared.
    "dsv3_prefill": MoEConfig(
        name="dsv3_prefill", n_tokens=4096, hidden=7168, n_experts=256,
        top_k=8, ffn=2048, score="sigmoid", norm_topk=True, n_shared=1,
        ffn_shared=2048, n_groups=8, topk_groups=4, ep_size=8, ep_rank=0,
        dtype="bf16", seed=4),
    # DeepSeek-V3-shaped decode step: 64 tokens per rank x 8 ranks, a
    # Zipf(1.2) popularity bias so some local experts receive 0-2 rows.
    "dsv3_decode": MoEConfig(
        name="dsv3_decode", n_tokens=64, hidden=7168, n_experts=256,
        top_k=8, ffn=2048, score="sigmoid", norm_topk=True, n_shared=1,
        ffn_shared=2048, n_groups=8, topk_groups=4, ep_size=8, ep_rank=0,
        dtype="bf16", bias="zipf", zipf_s=1.2, zipf_beta=0.05, seed=5),
    # Replicated-activation inference (all-reduce variant), one rank of
    # EP = TP = 8: a DeepSeek-V2-shaped layer (160 experts top-6 softmax of
    # 8 groups / top-3, 2 shared experts, routed scale 16) on a prefill of
    # 2 sequences x 2048 tokens held by every rank.
    "dsv2_ar": MoEConfig(
        name="dsv2_ar", n_tokens=4096, hidden=5120, n_experts=160, top_k=6,
        ffn=1536, score="softmax", norm_topk=False, n_shared=2, ffn_shared=1536,
        n_groups=8, topk_groups=3, routed_scale=16.0, ep_size=8, ep_rank=0,
        dtype="bf16", seed=6, ep_mode="allreduce"),
    # The same variant on a Llama-4-Scout-shaped layer: 16 experts top-1
    # sigmoid with a uniform selection bias, one shared expert.
    "scout_ar": MoEConfig(
        name="scout_ar", n_tokens=4096, hidden=5120, n_experts=16, top_k=1,
        ffn=8192, score="sigmoid", norm_topk=False, n_shared=1, ffn_shared=8192,
        ep_size=8, ep_rank=0, dtype="bf16", bias="uniform", seed=7, ep_mode="allreduce"),
}

ORDER = ["tiny", "dsv2lite", "scout", "dsv3_prefill", "dsv3_decode"]


def get_config(name):
    return CONFIGS[name]
