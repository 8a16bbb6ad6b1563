"""GRPO group advantages and the clipped-ratio + KL token loss, in fp64.

Alg. 1 normalises the K rewards of each prompt's group into advantages w(x)
and applies the GRPO objective of Eq. 1 with a KL penalty towards the frozen
reference.  Sec. VI-A keeps "the traditional GRPO policy" (Shao et al.), whose
per-token form is the clipped surrogate used below.  Readings where the paper
is silent: sample standard deviation (divisor G-1) plus eps; a group whose
rewards are all equal gets advantage 0; the KL is the per-token estimator
exp(d) - d - 1 with d = logp_ref - logp; the loss averages each sequence's
masked tokens, then the sequences.
"""
from __future__ import annotations

import numpy as np


def advantages(rewards, P: int, G: int, eps: float = 1e-6) -> np.ndarray:
    """[P*G] rewards -> [P*G] advantages (r - mean_g) / (std_g + eps)."""
    if G < 2:
        raise ValueError("a group needs at least two samples")
    r = np.asarray(rewards, np.float64).reshape(P, G)
    m = r.mean(axis=1, keepdims=True)
    s = np.sqrt(((r - m) ** 2).sum(axis=1, keepdims=True) / (G - 1))
    with np.errstate(invalid="ignore", divide="ignore"):
        a = (r - m) / (s + eps)
    degenerate = (r.max(axis=1) == r.min(axis=1))
    a[degenerate] = 0.0
    return a.reshape(-1)


def token_loss(logp, logp_old, logp_ref, mask, adv, clip_eps: float, beta: float,
               agg: int = 0) -> dict:
    """Per-token GRPO loss, its total, its gradient w.r.t. logp, and statistics.

    rho = exp(logp - logp_old); s = min(rho*A, clip(rho, 1-eps, 1+eps)*A);
    kl = exp(d) - d - 1, d = logp_ref - logp; l = -s + beta*kl.
    agg 0: mean over each sequence's masked tokens, then over sequences.
    agg 1: mean over all masked tokens.
    """
    lp = np.asarray(logp, np.float64)
    lo = np.asarray(logp_old, np.float64)
    lr = np.asarray(logp_ref, np.float64)
    m = np.asarray(mask).astype(bool)
    A = np.asarray(adv, np.float64)[:, None] * np.ones_like(lp)
    N = lp.shape[0]
    rho = np.exp(lp - lo)
    clipped = np.clip(rho, 1.0 - clip_eps, 1.0 + clip_eps)
    unclip_term, clip_term = rho * A, clipped * A
    s = np.minimum(unclip_term, clip_term)
    d = lr - lp
    kl = np.exp(d) - d - 1.0
    ell = -s + beta * kl
    # gradient of s: rho*A where the unclipped term is the minimum, else 0
    # (equal terms count as unclipped)
    unclipped_active = unclip_term <= clip_term
    ds = np.where(unclipped_active, rho * A, 0.0)
    dl = -ds + beta * (1.0 - np.exp(d))
    cnt = m.sum(axis=1).astype(np.float64)
    if agg == 0:
        wgt = m / (N * np.maximum(1.0, cnt))[:, None]
    else:
        wgt = m / max(1.0, float(cnt.sum()))
    loss = float(np.sum(np.where(m, ell, 0.0) * wgt))
    ntok = max(1.0, float(m.sum()))
    clip_hit = m & ~unclipped_active
    return dict(
        loss=loss,
        tok_loss=np.where(m, ell, 0.0),
        grad=np.where(m, dl * wgt, 0.0),
        kl_mean=float(np.sum(np.where(m, kl, 0.0)) / ntok),
        clip_frac=float(clip_hit.sum() / ntok),
        ratio_mean=float(np.sum(np.where(m, rho, 0.0)) / ntok),
        nonfinite=float(np.sum(m & ~np.isfinite(ell))),
    )
