"""Model shapes and decode workloads used as synthetic stand-ins for the
paper's evaluation (Section 4.1: batch 1, greedy, LayerSkip Llama models).

The paper's checkpoints and datasets (CNN/DM, TOPv2, Alpaca, HumanEval) are
not available, so every workload is a random-init Llama-shaped decoder with
N(0, 0.02) weights and a uniform-random prompt.  Nothing here computes any
part of the decoding method; it only names sizes, seeds and policies.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Tuple

# Seeds of the four independent input streams.
SEED_WEIGHTS = 0
SEED_PROMPT = 1
SEED_SCHEDULE = 2
SEED_QNET = 3
SEED_SAMPLE = 4          # uniforms of speculative sampling
SEED_DQN = 5             # policy-trainer inputs: transitions, mini-batch uniforms, noise
SAMPLE_SLOTS = 16        # per step: draft uniforms [0, 16), acceptance uniforms [16, 32), residual / bonus [32]
SAMPLE_STRIDE = 2 * SAMPLE_SLOTS + 1

WEIGHT_STD = 0.02  # standard deviation of every random weight

PAGE_SIZE = 64  # tokens per KV page


@dataclass(frozen=True)
class ModelConfig:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    dtype: str  # "f32" or "bf16": weights, linear-layer inputs and KV cache
    rope_base: float = 10000.0
    rms_eps: float = 1e-5
    # Q-network that maps a hidden state to a joint (exit layer, draft length)
    # action: d -> qnet_hidden -> len(exits) * len(lengths).
    qnet_hidden: int = 64
    exits: Tuple[int, ...] = (1, 2, 3, 4)
    lengths: Tuple[int, ...] = (1, 2, 3, 4, 5, 6, 7, 8)

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def n_actions(self) -> int:
        return len(self.exits) * len(self.lengths)

    @property
    def wbytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    def layer_weight_bytes(self) -> int:
        d, f = self.d_model, self.ffn_dim
        n = (self.q_dim + 2 * self.kv_dim) * d + d * self.q_dim + 3 * f * d
        return n * self.wbytes + 2 * d * self.wbytes

    def head_weight_bytes(self) -> int:
        return self.vocab * self.d_model * self.wbytes + self.d_model * self.wbytes

    def kv_bytes_per_token_layer(self) -> int:
        return 2 * self.kv_dim * self.wbytes

    def qnet_bytes(self) -> int:
        return 4 * (self.d_model * self.qnet_hidden + self.qnet_hidden * self.n_actions
                    + self.qnet_hidden + self.n_actions)


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelConfig
    prompt_len: int
    n_gen: int  # tokens produced after the prompt, including the prefill's token
    policy: str  # "fixed", "schedule" or "qnet"
    fixed: Tuple[int, int] = (2, 4)
    sched_l: Tuple[int, int] = (1, 1)  # inclusive range of the seeded schedule
    sched_k: Tuple[int, int] = (1, 8)
    qnet_logged: bool = True  # evaluate the Q-net every step even when it is overridden
    sweep_l: Tuple[int, ...] = ()
    sweep_k: Tuple[int, ...] = ()

    @property
    def max_ctx(self) -> int:
        return self.prompt_len + self.n_gen + max(self.model.lengths) + 1


TINY = ModelConfig("tiny", n_layers=4, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
                   ffn_dim=688, vocab=1024, dtype="f32", qnet_hidden=64,
                   exits=(1, 2, 3, 4), lengths=tuple(range(1, 9)))
LLAMA2_7B = ModelConfig("llama2-7b", n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32,
                        head_dim=128, ffn_dim=11008, vocab=32000, dtype="bf16", qnet_hidden=256,
                        exits=(4, 8, 12, 16), lengths=(2, 4, 6, 8))
LLAMA3_8B = ModelConfig("llama3-8b", n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8,
                        head_dim=128, ffn_dim=14336, vocab=128256, dtype="bf16",
                        rope_base=500000.0, qnet_hidden=256,
                        exits=tuple(range(2, 33, 2)), lengths=tuple(range(1, 9)))
LLAMA2_13B = ModelConfig("llama2-13b", n_layers=40, d_model=5120, n_heads=40, n_kv_heads=40,
                         head_dim=128, ffn_dim=13824, vocab=32000, dtype="bf16", qnet_hidden=256,
                         exits=tuple(range(5, 21)), lengths=tuple(range(1, 9)))
LLAMA2_70B = ModelConfig("llama2-70b", n_layers=80, d_model=8192, n_heads=64, n_kv_heads=8,
                         head_dim=128, ffn_dim=28672, vocab=32000, dtype="bf16", qnet_hidden=256,
                         exits=tuple(range(10, 41)), lengths=tuple(range(1, 9)))

WORKLOADS = {
    "tiny": Workload("tiny", TINY, prompt_len=32, n_gen=64, policy="fixed", fixed=(2, 4)),
    "llama2-7b": Workload("llama2-7b", LLAMA2_7B, prompt_len=512, n_gen=256, policy="fixed",
                          fixed=(8, 4), sweep_l=(4, 8, 12, 16), sweep_k=(2, 4, 6, 8)),
    "llama3-8b": Workload("llama3-8b", LLAMA3_8B, prompt_len=1024, n_gen=256, policy="qnet"),
    "llama2-13b": Workload("llama2-13b", LLAMA2_13B, prompt_len=4096, n_gen=512,
                           policy="schedule", sched_l=(5, 20), sched_k=(1, 8)),
    "llama2-70b": Workload("llama2-70b", LLAMA2_70B, prompt_len=2048, n_gen=256,
                           policy="schedule", sched_l=(10, 40), sched_k=(1, 8)),
}


def shrink(model: ModelConfig, **kw) -> ModelConfig:
    """A variant of a model shape (fewer layers, smaller vocab, ...) for tests."""
    return replace(model, **kw)
