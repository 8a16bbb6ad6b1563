"""An fp32 emulation of one decoder layer under the precision contract, for CPU
tests of the rounding-point-local checker (not collected: no test_ prefix).

It follows the arithmetic model of tests/bounds.py: each 32-wide matrix-core
step adds the exact sum of its products to an fp32 accumulator with one
rounding, vector operations round to fp32 after each step, bf16 rounding points
where the contract has them.  `mutate` plants one mistake of the kind a kernel
could make, which the checker must reject."""
from __future__ import annotations

import numpy as np

import oracle

f32 = np.float32


def gemm32(a, W, kc=32):
    """a [R, K] @ W[N, K]^T: one chain of kc-wide steps, exact step sums rounded into
    an fp32 accumulator."""
    a = np.asarray(a, np.float64)
    W = np.asarray(W, np.float64)
    acc = np.zeros((a.shape[0], W.shape[0]), f32)
    for k0 in range(0, a.shape[1], kc):
        acc = (acc.astype(np.float64) + a[:, k0:k0 + kc] @ W[:, k0:k0 + kc].T).astype(f32)
    return acc


def rms32(x, g, eps):
    x = np.asarray(x, f32)
    ss = np.sum(x.astype(np.float64) ** 2, -1, keepdims=True).astype(f32)   # one rounding
    r = f32(1) / np.sqrt(ss / f32(x.shape[-1]) + f32(eps))
    return (x * r) * np.asarray(g, f32)


def rope32(v, pos, theta):
    hd = v.shape[-1]
    ang = oracle.numerics.rope_angles(pos, hd, theta)[:, None, :]
    c, s = np.cos(ang).astype(f32), np.sin(ang).astype(f32)
    lo, hi = v[..., :hd // 2].astype(f32), v[..., hd // 2:].astype(f32)
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], -1)


def attn32(q, K, V, scale, mutate=None):
    """q [hd]; K, V [ctx, hd]: flash-like fp32: scores by 32-wide steps, exp, P.V by
    32-key steps rounded into fp32."""
    s = gemm32(K, q[None, :])[:, 0] * f32(scale)
    if mutate == "scale":
        s = s * f32(1.0001)
    p = np.exp((s - s.max()).astype(f32)).astype(f32)
    L = np.sum(p.astype(np.float64)).astype(f32)
    Vv = V[::-1] if mutate == "reversed_v" else V   # values paired with the wrong keys
    acc = gemm32(p[None, :], Vv.T)[0]
    return acc / L


def emulate_layer(cfg, om, l, x, pos, Kc, Vc, mutate=None):
    """One decode layer for rows x [R, d] at positions pos, cache Kc/Vc
    [R, n_kv, ctx_max, hd] (positions below pos[r] filled).  Returns the trace
    entries of that layer (bf16 values as float64)."""
    R = oracle.round_bf16
    H, Hk, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    p = f"l{l}."
    x = np.asarray(x, f32)
    h = R(rms32(x, om.mat(p + "attn_norm"), cfg.rms_eps))
    W = np.concatenate([om.mat(p + "wq"), om.mat(p + "wk"), om.mat(p + "wv")], 0)
    if mutate == "drop_term":
        W = W.copy()
        W[:, 7] = 0
    qkv = gemm32(h, W)
    qd, kvd = cfg.q_dim, cfg.kv_dim
    n = x.shape[0]
    q = rope32(qkv[:, :qd].reshape(n, H, hd), pos, cfg.rope_theta)
    k = rope32(qkv[:, qd:qd + kvd].reshape(n, Hk, hd), pos, cfg.rope_theta)
    if mutate == "rope_sign":
        k = rope32(qkv[:, qd:qd + kvd].reshape(n, Hk, hd), -np.asarray(pos), cfg.rope_theta)
    q, k, v = R(q), R(k), R(qkv[:, qd + kvd:].reshape(n, Hk, hd))
    o = np.zeros((n, H, hd))
    for b in range(n):
        Kc[b, :, pos[b]] = k[b]
        Vc[b, :, pos[b]] = v[b]
        for hh in range(H):
            g = hh * Hk // H
            o[b, hh] = attn32(q[b, hh].astype(np.float64), Kc[b, g, :pos[b] + 1],
                              Vc[b, g, :pos[b] + 1], 1.0 / np.sqrt(hd), mutate)
    o = R(o.reshape(n, qd))
    xa = (x.astype(np.float64) + gemm32(o, om.mat(p + "wo"))).astype(f32)
    if mutate == "no_resid":
        xa = gemm32(o, om.mat(p + "wo"))
    h2 = R(rms32(xa, om.mat(p + "mlp_norm"), cfg.rms_eps))
    gt, up = gemm32(h2, om.mat(p + "w_gate")), gemm32(h2, om.mat(p + "w_up"))
    a = R((gt / (f32(1) + np.exp(-gt))) * up)
    xo = (xa.astype(np.float64) + gemm32(a, om.mat(p + "w_down"))).astype(f32)
    return dict(x=x, h_attn=h, q=q.reshape(n, qd), k=k.reshape(n, kvd), v=v.reshape(n, kvd),
                o=o, x_attn=xa, h_mlp=h2, act=a, x_out=xo)
