"""CPU oracle of the GRPO hot path — TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously-correct NumPy (fp64 accumulation) versions of what the
HIP path computes: the Llama-family decoder forward the paper fine-tunes
(Sec. VI-C), counter-based sampling of a group of K rollouts per prompt
(Alg. 1, sampling step), teacher-forced scoring of the sampled completions
(log pi(x|c) in Eq. 1), group-normalised advantages (Alg. 1, normalisation
step), the clipped-ratio + KL token loss (Eq. 1 in the clipped GRPO form the
paper keeps, Sec. VI-A), and the gradient step that closes each iteration
(Alg. 1: the weight gradient of the scored log-probs, AdamW).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It imports nothing from the HIP
package and shares no code with it; both sides consume the same seeded inputs.

Pins (tests/test_oracle_*.py) tie every function to something other than
itself: brute-force loops, closed forms, invariants, library routines and
worked examples.  The composed full-vocabulary Gumbel/top-k sampler is pinned
only through its parts and limits (greedy limit, softmax frequencies); beyond
that it is "parity unpinned": no external reference for the composition exists.
"""
from .numerics import bf16_bits_to_f64, round_bf16, rmsnorm, silu, rope
from .philox import philox4x32_10, philox_uniform24, gumbel_keys
from .sampler import sample_token, topk_set, log_softmax
from .model import OracleModel
from .grpo import advantages, token_loss
from .distill import exact_kl, reward, sft_loss
from .backward import adamw, policy_gradient

__all__ = [
    "bf16_bits_to_f64", "round_bf16", "rmsnorm", "silu", "rope",
    "philox4x32_10", "philox_uniform24", "gumbel_keys",
    "sample_token", "topk_set", "log_softmax",
    "OracleModel", "advantages", "token_loss", "reward", "sft_loss", "exact_kl",
    "policy_gradient", "adamw",
]
