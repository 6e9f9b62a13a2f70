"""Model shapes and verify workloads.

The five full-size workloads are the configurations the verify path is measured
on: a tiny fp32 verifier and Llama-7B/13B/33B-shaped bf16 verifiers.  The paper
itself runs LLaMA-3.1-8B as the cloud verifier (Experiments, "Models"); the
synthetic shapes stand in for it.  ``mini_workloads`` are scaled-down variants
with the same structure (ragged vocab tail, ragged contexts, several tiles per
GEMM, mixed greedy/sampling rows) sized so the CPU oracle finishes in seconds.
"""

from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import List, Optional, Tuple


@dataclass(frozen=True)
class ModelShape:
    """Pre-RMSNorm decoder with RoPE, multi-head (or grouped-query) attention
    and a SwiGLU FFN."""

    name: str
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    weight_dtype: str = "bf16"  # "bf16" or "f32"
    kv_dtype: str = "bf16"  # "bf16" or "f32"
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0
    init_std: float = 0.02
    # Gains of the three RMSNorms.  1.0 everywhere for the full-size shapes;
    # the mini shapes draw them from N(1, gain_std) so a dropped gain shows.
    gain_std: float = 0.0
    # K/V heads; 0 means one per query head (multi-head attention).
    n_kv_heads: int = 0

    @property
    def kv_heads(self) -> int:
        return self.n_kv_heads or self.n_heads

    def weight_bytes(self) -> int:
        elt = 2 if self.weight_dtype == "bf16" else 4
        d, f, v = self.d_model, self.d_ffn, self.vocab
        dkv = self.kv_heads * self.head_dim
        per_layer = (2 * d * d + 2 * d * dkv + 3 * d * f) * elt + 2 * d * 4
        return self.n_layers * per_layer + 2 * v * d * elt + d * 4


@dataclass(frozen=True)
class Workload:
    """One verify call: B requests, gamma drafts each, cached contexts."""

    name: str
    model: ModelShape
    batch: int
    gamma: int
    # Either a fixed cached length for every request or an inclusive range
    # [lo, hi] drawn uniformly per request.
    ctx: Tuple[int, int]
    # "greedy", "sample" or "mixed" (even requests greedy, odd sampling).
    mode: str
    temperature: float = 1.0
    # How draft tokens are chosen: "random" (uniform ids), "chain_half"
    # (first ceil(gamma/2) from the verifier's own argmax chain, rest random),
    # "draft_model" (sampled from q = softmax(verifier logits + N(0,1))),
    # "noise_q" (q = softmax(N(0,1)) per row, drafts sampled from q).
    draft_recipe: str = "random"
    rounds: int = 1
    seed: int = 1000
    description: str = ""

    @property
    def rows(self) -> int:
        return self.batch * (self.gamma + 1)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


TINY = ModelShape("tiny-fp32", n_layers=2, d_model=256, n_heads=4, head_dim=64,
                  d_ffn=1024, vocab=4096, weight_dtype="f32", kv_dtype="f32")
LLAMA_7B = ModelShape("llama-7b-shape", n_layers=32, d_model=4096, n_heads=32,
                      head_dim=128, d_ffn=11008, vocab=32000)
LLAMA_13B = ModelShape("llama-13b-shape", n_layers=40, d_model=5120, n_heads=40,
                       head_dim=128, d_ffn=13824, vocab=32000)
LLAMA_33B = ModelShape("llama-33b-shape", n_layers=60, d_model=6656, n_heads=52,
                       head_dim=128, d_ffn=17920, vocab=32000)
# The paper's cloud verifier's shape (LLaMA-3.1-8B: grouped-query attention
# with 8 K/V heads for 32 query heads, a 128256-token vocabulary, RoPE base
# 500000); random weights as for the other shapes.
LLAMA3_8B = ModelShape("llama3-8b-gqa-shape", n_layers=32, d_model=4096, n_heads=32,
                       head_dim=128, d_ffn=14336, vocab=128256, n_kv_heads=8,
                       rope_theta=500000.0)

WORKLOADS = {
    "c1_tiny_greedy": Workload(
        "c1_tiny_greedy", TINY, batch=1, gamma=4, ctx=(128, 128), mode="greedy",
        draft_recipe="random", seed=1001,
        description="tiny fp32 verifier, 128 cached tokens, gamma=4, greedy"),
    "c1_tiny_sample": Workload(
        "c1_tiny_sample", TINY, batch=1, gamma=4, ctx=(128, 128), mode="sample",
        draft_recipe="noise_q", seed=1011,
        description="tiny fp32 verifier, gamma=4, sampling, q=softmax(N(0,1))"),
    "c2_7b_greedy": Workload(
        "c2_7b_greedy", LLAMA_7B, batch=1, gamma=5, ctx=(1024, 1024), mode="greedy",
        draft_recipe="chain_half", seed=1002,
        description="7B-shaped bf16 verifier, 1024 cached tokens, gamma=5, greedy, "
                    "half the drafts from the verifier's argmax chain"),
    "c3_13b_sample": Workload(
        "c3_13b_sample", LLAMA_13B, batch=1, gamma=8, ctx=(2048, 2048), mode="sample",
        draft_recipe="draft_model", seed=1003,
        description="13B-shaped bf16 verifier, 2048 cached tokens, gamma=8, sampling "
                    "at T=1, q=softmax(verifier logits + N(0,1))"),
    "c4_7b_batched": Workload(
        "c4_7b_batched", LLAMA_7B, batch=16, gamma=8, ctx=(256, 4096), mode="mixed",
        draft_recipe="chain_half", seed=1004,
        description="7B-shaped bf16 verifier, 16 requests, contexts U[256,4096], "
                    "gamma=8, mixed greedy/sampling, ragged KV cache"),
    "c5_33b_commit": Workload(
        "c5_33b_commit", LLAMA_33B, batch=4, gamma=6, ctx=(1536, 1536), mode="greedy",
        draft_recipe="chain_half", rounds=2, seed=1005,
        description="33B-shaped bf16 verifier, 4 requests x 1536 cached tokens, "
                    "gamma=6, greedy, kv_commit then a second verify round"),
    "gqa_8b_greedy": Workload(
        "gqa_8b_greedy", LLAMA3_8B, batch=1, gamma=5, ctx=(1024, 1024), mode="greedy",
        draft_recipe="random", seed=1006,
        description="8B-shaped bf16 verifier with grouped-query attention (8 K/V heads) and a "
                    "128256-token vocabulary, 1024 cached tokens, gamma=5, greedy"),
    "gqa_8b_batched": Workload(
        "gqa_8b_batched", LLAMA3_8B, batch=16, gamma=8, ctx=(256, 4096), mode="mixed",
        draft_recipe="chain_half", seed=1007,
        description="8B-shaped GQA verifier, 16 requests, contexts U[256,4096], gamma=8, "
                    "mixed greedy/sampling (sampling rows: q = softmax(N(0,1)))"),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


# Scaled-down shapes for oracle-vs-GPU parity.  Every GEMM spans several
# 16-row panels and several 256-wide k-blocks; the vocab has a ragged tail
# (not a multiple of 16); gains are random.
MINI_BF16 = ModelShape("mini-bf16", n_layers=2, d_model=512, n_heads=4, head_dim=128,
                       d_ffn=1536, vocab=4001, init_std=0.06, gain_std=0.1)
MINI_BF16_WIDE = ModelShape("mini-bf16-wide", n_layers=3, d_model=1024, n_heads=8,
                            head_dim=128, d_ffn=2816, vocab=8011, init_std=0.05, gain_std=0.1)
MINI_GQA = ModelShape("mini-gqa", n_layers=2, d_model=1024, n_heads=8, head_dim=128,
                      d_ffn=2816, vocab=12007, n_kv_heads=2, rope_theta=500000.0,
                      init_std=0.05, gain_std=0.1)
MINI_F32 = ModelShape("mini-f32", n_layers=2, d_model=256, n_heads=4, head_dim=64,
                      d_ffn=768, vocab=1999, weight_dtype="f32", kv_dtype="f32", init_std=0.06,
                      gain_std=0.1)


def mini_workloads() -> List[Workload]:
    return [
        Workload("mini_f32_greedy", MINI_F32, batch=2, gamma=4, ctx=(37, 130),
                 mode="greedy", draft_recipe="random", seed=2001),
        Workload("mini_bf16_greedy", MINI_BF16, batch=1, gamma=5, ctx=(300, 300),
                 mode="greedy", draft_recipe="chain_half", seed=2002),
        Workload("mini_bf16_sample", MINI_BF16, batch=1, gamma=8, ctx=(257, 257),
                 mode="sample", draft_recipe="noise_q", seed=2003),
        Workload("mini_bf16_mixed", MINI_BF16, batch=4, gamma=3, ctx=(1, 520),
                 mode="mixed", draft_recipe="chain_half", seed=2004),
        Workload("mini_bf16_wide_b5", MINI_BF16_WIDE, batch=5, gamma=6, ctx=(60, 700),
                 mode="mixed", draft_recipe="chain_half", seed=2005),
        Workload("mini_gqa_greedy", MINI_GQA, batch=1, gamma=5, ctx=(300, 300),
                 mode="greedy", draft_recipe="chain_half", seed=2006),
        Workload("mini_gqa_mixed_b5", MINI_GQA, batch=5, gamma=6, ctx=(40, 650),
                 mode="mixed", draft_recipe="chain_half", seed=2007),
    ]
