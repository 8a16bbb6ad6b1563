"""Model shapes and rollout workloads of the GRPO hot path.

The paper fine-tunes a Llama-family decoder with GRPO (Sec. VI-A, Alg. 1):
for every prompt it samples a group of K completions, scores them, normalises
the rewards inside the group and applies the clipped-ratio + KL loss against a
frozen reference copy.  The paper publishes no shapes for its own training
system, so the workloads below are synthetic Llama-style decoders at five
sizes, from a 2-layer fp32 toy to a 32B-shape model that fills one MI355X.

Nothing here computes anything: these are plain records shared by the bench,
the tests and the input generator.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

DTYPE_F32 = 0
DTYPE_BF16 = 1


@dataclass(frozen=True)
class ModelConfig:
    """Decoder shape (Llama family: RMSNorm, RoPE, GQA, SwiGLU, untied head)."""

    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    rms_eps: float = 1e-6
    rope_theta: float = 10000.0
    dtype: int = DTYPE_BF16

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == DTYPE_F32 else 2

    def n_params(self) -> int:
        d, f, V = self.d_model, self.d_ffn, self.vocab
        per_layer = 2 * d + d * (self.q_dim + 2 * self.kv_dim) + self.q_dim * d + 3 * f * d
        return V * d * 2 + d + self.n_layers * per_layer

    def weight_bytes(self) -> int:
        return self.n_params() * self.elem_bytes

    def kv_bytes_per_token(self) -> int:
        """K and V of one token over all layers."""
        return 2 * self.n_layers * self.kv_dim * self.elem_bytes


@dataclass(frozen=True)
class Workload:
    """One GRPO iteration's worth of rollout, scoring and loss work."""

    name: str
    index: int                 # position in the workload list; picks the master seed
    model: ModelConfig
    n_prompts: int             # P
    group: int                 # G samples per prompt (the paper's K)
    prompt_len: int            # Tp
    new_tokens: int            # Tn sampled tokens per completion
    temperature: float         # 0 means greedy
    top_k: int = 0             # 0 means the full vocabulary
    prompt_kind: str = "uniform"   # "uniform" or "code" (code-like stream + tool spans)
    tool_spans: int = 0        # number of 256-token tool-output spans in a prompt
    score: bool = True         # teacher-forced scoring of policy + reference
    shared_prompt: bool = True  # decode and scoring run each group's shared prompt once
    clip_eps: float = 0.2
    beta: float = 0.04
    adv_eps: float = 1e-6

    @property
    def batch(self) -> int:
        return self.n_prompts * self.group

    @property
    def total_len(self) -> int:
        return self.prompt_len + self.new_tokens

    @property
    def max_len(self) -> int:
        """KV positions a rollout writes: the last sampled token is never fed back."""
        return self.prompt_len + self.new_tokens - 1

    @property
    def master_seed(self) -> int:
        return 20251017 + self.index

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


TINY = ModelConfig(n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
                   d_ffn=1024, vocab=2048, dtype=DTYPE_F32)
SMALL = ModelConfig(n_layers=12, d_model=768, n_heads=12, n_kv_heads=4, head_dim=64,
                    d_ffn=3072, vocab=32000)
M1B = ModelConfig(n_layers=16, d_model=2048, n_heads=32, n_kv_heads=8, head_dim=64,
                  d_ffn=8192, vocab=32000)
M7B = ModelConfig(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                  d_ffn=14336, vocab=32000)
M32B = ModelConfig(n_layers=64, d_model=5120, n_heads=40, n_kv_heads=8, head_dim=128,
                   d_ffn=27648, vocab=152064)

WORKLOADS = {
    "tiny": Workload("tiny", 0, TINY, n_prompts=4, group=4, prompt_len=64, new_tokens=64,
                     temperature=0.0),
    "small": Workload("small", 1, SMALL, n_prompts=8, group=8, prompt_len=512, new_tokens=512,
                      temperature=1.0),
    "1b": Workload("1b", 2, M1B, n_prompts=16, group=8, prompt_len=1024, new_tokens=1024,
                   temperature=0.8, top_k=50, score=False),
    "7b": Workload("7b", 3, M7B, n_prompts=8, group=8, prompt_len=2048, new_tokens=2048,
                   temperature=1.0, prompt_kind="code", tool_spans=3),
    "32b": Workload("32b", 4, M32B, n_prompts=4, group=8, prompt_len=8192, new_tokens=4096,
                    temperature=1.0, prompt_kind="code", tool_spans=12, score=False),
    # the group size the paper settles on (K = 12, Sec. VI-A) at the 7B shape
    "7b-k12": Workload("7b-k12", 5, M7B, n_prompts=8, group=12, prompt_len=2048,
                       new_tokens=2048, temperature=1.0, prompt_kind="code", tool_spans=3),
}


def get(name: str) -> Workload:
    return WORKLOADS[name]


def truncated(w: Workload, n_layers: int, **kw) -> Workload:
    """Same widths, fewer layers: used where the fp64 oracle cannot run full depth."""
    return replace(w, model=replace(w.model, n_layers=n_layers), **kw)
