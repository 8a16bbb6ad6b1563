"""The paper's reward, the distillation loss and the exact KL, in fp64 — TEST
INFRASTRUCTURE ONLY (see the package docstring).

Reward (Sec. VI-A, Eq. 2-4): r(x) = r_perf(x) + r_tools(x) with
    r_perf = -2 if the final code is incorrect, -1 if correct but slower than
             the baseline (t > t_base), else min(10, t_base / t - 1);
    r_tools = 0.5 * |unique tools used among the available ones| / |available|.
Distillation (Sec. VI-B): supervised fine-tuning of a small model on the large
model's (prompt, reasoning trace, final code) tuples, tool-call tokens and
arguments kept in the targets: the teacher-forced cross-entropy -log pi over the
target tokens.  Exact KL: the full-vocabulary KL(pi || pi_ref) of one position,
sum_v p(v) (log p(v) - log p_ref(v)) with p = softmax(z / T); Alg. 1 computes a
KL to the frozen reference and the per-token estimator exp(d) - d - 1 of the GRPO
loss is its sampled form.
"""
from __future__ import annotations

import numpy as np

from .sampler import log_softmax


def reward(correct, t_base, t, tools_used, tools_avail, lam: float = 0.5) -> np.ndarray:
    """Eq. 2-4 for arrays of (correct flag, baseline time, time, number of unique
    available tools used, number of available tools)."""
    correct = np.asarray(correct).astype(bool)
    t_base = np.asarray(t_base, np.float64)
    t = np.asarray(t, np.float64)
    used = np.asarray(tools_used, np.float64)
    avail = np.asarray(tools_avail, np.float64)
    slower = t > t_base
    with np.errstate(divide="ignore", invalid="ignore"):
        fast = np.minimum(10.0, t_base / t - 1.0)
    r_perf = np.where(~correct, -2.0, np.where(slower, -1.0, fast))
    r_tools = lam * np.minimum(used, avail) / np.maximum(avail, 1.0)
    return r_perf + r_tools


def sft_loss(logp, mask, agg: int = 1) -> dict:
    """Cross-entropy of the target tokens given their log-probs [N, Tr] (as
    teacher-forced scoring returns them) and target mask.  agg 1: mean over all
    target tokens; agg 0: mean over each sequence's targets, then over sequences
    (a sequence without targets counts 0).  Returns the loss and d loss / d logp."""
    lp = np.asarray(logp, np.float64)
    m = np.asarray(mask).astype(bool)
    N = lp.shape[0]
    cnt = m.sum(axis=1).astype(np.float64)
    if agg == 1:
        w = m / max(1.0, float(cnt.sum()))
    else:
        w = m / (N * np.maximum(1.0, cnt))[:, None]
    loss = -float(np.sum(np.where(m, lp, 0.0) * w))
    return dict(loss=loss, grad=-np.where(m, w, 0.0))


def exact_kl(logits, logits_ref, temperature: float = 1.0) -> np.ndarray:
    """Rows of full-vocabulary KL(softmax(z / T) || softmax(z_ref / T))."""
    T = temperature if temperature > 0 else 1.0
    lp = log_softmax(np.asarray(logits, np.float64) / T)
    lq = log_softmax(np.asarray(logits_ref, np.float64) / T)
    return np.sum(np.exp(lp) * (lp - lq), axis=-1)
