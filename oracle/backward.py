"""Gradient of the teacher-forced policy objective and the optimizer step, in fp64.

Alg. 1 ends each iteration with a gradient step on the GRPO objective (Eq. 1 in
the clipped form of Sec. VI-A).  The objective reaches the policy's weights only
through the per-token log-probabilities log pi(x_t | c, x_<t) of the scored
tokens, so with g_t = dL/dlogp_t (what ``token_loss`` returns) the weight
gradient is the gradient of sum_t g_t logp_t, back through the decoder of
``model.py``:

    logp_t = log_softmax(z_t / T)[x_{t+1}],   z = R5(rmsnorm(x_L) g_f) W_head^T
    dz_t   = g_t / T (onehot(x_{t+1}) - softmax(z_t / T))

and then the chain rule through every layer in reverse (RMSNorm, SwiGLU, the
projections, causal grouped-query attention, RoPE, the embedding gather).
The bf16 rounding points R1..R5 of the forward are passed straight through
(their derivative is taken as 1, the usual rule of mixed-precision training);
the activations the weight gradients multiply are the rounded forward values.

The optimizer (the paper names none) is AdamW with decoupled weight decay and
bias correction, the standard choice for fine-tuning these decoders.
"""
from __future__ import annotations

import numpy as np

from .model import causal_attention
from .numerics import rmsnorm, rope, rope_angles, silu
from .sampler import log_softmax


def rmsnorm_backward(x: np.ndarray, g: np.ndarray, eps: float, dy: np.ndarray):
    """y = x r g with r = (mean(x^2) + eps)^(-1/2) over the last axis.
    Returns (dx, dg) for the upstream gradient dy (rows summed into dg)."""
    d = x.shape[-1]
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    gdy = dy * g
    dx = r * gdy - x * r ** 3 * np.sum(gdy * x, axis=-1, keepdims=True) / d
    dg = np.sum(dy * x * r, axis=0)
    return dx, dg


def rope_backward(dy: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Adjoint of ``rope`` (rotation by the opposite angle) on [T, n, hd]."""
    hd = dy.shape[-1]
    a = rope_angles(pos, hd, theta)[:, None, :]
    c, s = np.cos(a), np.sin(a)
    lo, hi = dy[..., : hd // 2], dy[..., hd // 2:]
    return np.concatenate([lo * c + hi * s, hi * c - lo * s], axis=-1)


def attention_backward(q, k, v, do):
    """Causal grouped-query attention o = softmax(q k^T / sqrt(hd)) v, backward.

    q, do [T, H, hd]; k, v [T, Hkv, hd] -> dq, dk, dv of the same shapes."""
    T, H, hd = q.shape
    Hk = k.shape[1]
    s = 1.0 / np.sqrt(hd)
    causal = np.tril(np.ones((T, T), bool))
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for h in range(H):
        g = h * Hk // H
        S = np.where(causal, q[:, h] @ k[:, g].T * s, -np.inf)
        P = np.exp(S - S.max(axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        dv[:, g] += P.T @ do[:, h]
        dP = do[:, h] @ v[:, g].T
        dS = P * (dP - np.sum(P * dP, axis=1, keepdims=True))
        dq[:, h] = dS @ k[:, g] * s
        dk[:, g] += dS.T @ q[:, h] * s
    return dq, dk, dv


def policy_gradient(om, tokens, score_from: int, temperature: float, dlogp) -> dict:
    """Gradient of sum_j dlogp[j] * logp[j] over one sequence's scored tokens
    j = score_from .. T-1 (logp as ``OracleModel.score``) with respect to every
    weight of ``om`` (dict of fp64 arrays with the weights' names and shapes)."""
    c, R = om.cfg, om.R
    tokens = np.asarray(tokens)
    T = len(tokens)
    H, Hk, hd = c.n_heads, c.n_kv_heads, c.head_dim
    pos = np.arange(T)
    Tt = temperature if temperature > 0 else 1.0
    # ---- forward, keeping what the backward multiplies ----
    x = om.embed(tokens)
    saved = []
    for l in range(c.n_layers):
        p = f"l{l}."
        h = R(rmsnorm(x, om.mat(p + "attn_norm"), c.rms_eps))
        q = R(rope(om.mm(h, p + "wq").reshape(T, H, hd), pos, c.rope_theta))
        k = R(rope(om.mm(h, p + "wk").reshape(T, Hk, hd), pos, c.rope_theta))
        v = R(om.mm(h, p + "wv").reshape(T, Hk, hd))
        o = R(causal_attention(q, k, v).reshape(T, H * hd))
        xa = x + om.mm(o, p + "wo")
        h2 = R(rmsnorm(xa, om.mat(p + "mlp_norm"), c.rms_eps))
        gate, up = om.mm(h2, p + "w_gate"), om.mm(h2, p + "w_up")
        a = R(silu(gate) * up)
        saved.append((x, h, q, k, v, o, xa, h2, gate, up, a))
        x = xa + om.mm(a, p + "w_down")
    hf = R(rmsnorm(x, om.mat("final_norm"), c.rms_eps))
    z = om.mm(hf, "lm_head")
    # ---- head: dz on the scored rows t = score_from - 1 .. T - 2 ----
    grads = {}
    rows = np.arange(score_from - 1, T - 1)
    dz = np.zeros_like(z)
    prob = np.exp(log_softmax(z[rows] / Tt))
    onehot = np.zeros_like(prob)
    onehot[np.arange(len(rows)), tokens[rows + 1]] = 1.0
    dz[rows] = np.asarray(dlogp, np.float64)[:, None] / Tt * (onehot - prob)
    grads["lm_head"] = dz.T @ hf
    dx, grads["final_norm"] = rmsnorm_backward(x, om.mat("final_norm"), c.rms_eps,
                                               dz @ om.mat("lm_head"))
    # ---- layers in reverse ----
    for l in reversed(range(c.n_layers)):
        p = f"l{l}."
        x, h, q, k, v, o, xa, h2, gate, up, a = saved[l]
        grads[p + "w_down"] = dx.T @ a
        da = dx @ om.mat(p + "w_down")
        sg = 1.0 / (1.0 + np.exp(-gate))
        dgate = da * up * sg * (1.0 + gate * (1.0 - sg))
        dup = da * silu(gate)
        grads[p + "w_gate"] = dgate.T @ h2
        grads[p + "w_up"] = dup.T @ h2
        dh2 = dgate @ om.mat(p + "w_gate") + dup @ om.mat(p + "w_up")
        dxa_n, grads[p + "mlp_norm"] = rmsnorm_backward(xa, om.mat(p + "mlp_norm"), c.rms_eps, dh2)
        dxa = dx + dxa_n
        grads[p + "wo"] = dxa.T @ o
        do = (dxa @ om.mat(p + "wo")).reshape(T, H, hd)
        dq, dk, dv = attention_backward(q, k, v, do)
        dq = rope_backward(dq, pos, c.rope_theta).reshape(T, H * hd)
        dk = rope_backward(dk, pos, c.rope_theta).reshape(T, Hk * hd)
        dv = dv.reshape(T, Hk * hd)
        grads[p + "wq"] = dq.T @ h
        grads[p + "wk"] = dk.T @ h
        grads[p + "wv"] = dv.T @ h
        dh = dq @ om.mat(p + "wq") + dk @ om.mat(p + "wk") + dv @ om.mat(p + "wv")
        dx_n, grads[p + "attn_norm"] = rmsnorm_backward(x, om.mat(p + "attn_norm"), c.rms_eps, dh)
        dx = dxa + dx_n
    demb = np.zeros((c.vocab, c.d_model))
    np.add.at(demb, tokens, dx)
    grads["tok_emb"] = demb
    return grads


def adamw(param, grad, m, v, step: int, lr: float, beta1: float, beta2: float, eps: float,
          weight_decay: float):
    """One AdamW update (decoupled weight decay, bias-corrected moments) at step
    number `step` (1 for the first).  Returns (param, m, v), all fp64."""
    m = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * grad
    v = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * grad * grad
    mh = m / (1.0 - beta1 ** step)
    vh = v / (1.0 - beta2 ** step)
    p = np.asarray(param, np.float64)
    p = p - lr * weight_decay * p - lr * mh / (np.sqrt(vh) + eps)
    return p, m, v
