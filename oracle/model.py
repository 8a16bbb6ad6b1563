"""Llama-family decoder, rollout and teacher-forced scoring, in fp64.

The paper's policy and its frozen reference are Llama3 decoders (Sec. VI-C);
GRPO samples K completions per prompt from the policy (Alg. 1, sampling step)
and needs log pi(x|c) of each sampled token under the policy and the reference
(Eq. 1 and the KL term).  The decoder here is the family's standard
definition, per layer:

    h = R1(rmsnorm(x) * g_attn)
    q, k, v = h Wq^T, h Wk^T, h Wv^T         (q, k rotated by RoPE, then R2)
    o_h = softmax_j(q_h . k_{kv(h), j} / sqrt(hd)) v_{kv(h), j}   over j <= i
    x += R3(o) Wo^T
    h = R1(rmsnorm(x) * g_mlp)
    x += R4(silu(h Wg^T) * (h Wu^T)) Wd^T

and logits = R5(rmsnorm(x) * g_final) W_head^T.  kv(h) = floor(h * H_kv / H)
(grouped-query attention).  R1..R5 are bf16 round-to-nearest-even applied only
for bf16 models (weights stored in bf16); fp32 models have no rounding points.
Everything else is fp64.

``forward`` is the plain full-sequence definition.  ``decode_layer`` is the
same layer for one new token per sequence against a KV cache; the test suite
pins it to ``forward`` (cached decode equals full recompute).
"""
from __future__ import annotations

import numpy as np

from .numerics import bf16_bits_to_f64, rmsnorm, round_bf16, rope, silu
from .sampler import log_softmax, sample_token


def _ident(x):
    return x


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """q [T, H, hd], k/v [T, Hkv, hd] -> o [T, H, hd]; query i sees keys j <= i.

    Query head h reads key/value head floor(h * Hkv / H) (grouped-query attention).
    """
    T, H, hd = q.shape
    Hk = k.shape[1]
    causal = np.tril(np.ones((T, T), bool))
    o = np.empty((T, H, hd), q.dtype)
    for hh in range(H):
        g = hh * Hk // H
        s = (q[:, hh, :] @ k[:, g, :].T) / float(np.sqrt(hd))
        s = np.where(causal, s, -np.inf)
        pr = np.exp(s - s.max(axis=1, keepdims=True))
        pr /= pr.sum(axis=1, keepdims=True)
        o[:, hh, :] = pr @ v[:, g, :]
    return o


class OracleModel:
    """cfg: any object with the decoder shape attributes (n_layers, d_model, ...).

    Everything is evaluated in fp64; for bf16 models (weights stored as bf16 bit
    patterns) the rounding points R1..R5 are applied unless round_points is
    False."""

    def __init__(self, cfg, weights: dict, round_points: bool = True):
        self.cfg = cfg
        self.w = weights
        self.bf16 = np.asarray(weights["tok_emb"]).dtype == np.uint16
        self.dt = np.float64
        self.R = round_bf16 if (self.bf16 and round_points) else _ident
        self._f64 = {}

    # -- weights --------------------------------------------------------------
    def mat(self, name: str) -> np.ndarray:
        if name not in self._f64:
            a = np.asarray(self.w[name])
            f = bf16_bits_to_f64(a) if a.dtype == np.uint16 else a.astype(np.float64)
            self._f64[name] = f.astype(self.dt, copy=False)
        return self._f64[name]

    def drop_cache(self):
        self._f64.clear()

    def mm(self, h: np.ndarray, name: str) -> np.ndarray:
        """h @ W^T for the weight matrix `name` ([out, in])."""
        return h @ self.mat(name).T

    def embed(self, tokens) -> np.ndarray:
        a = np.asarray(self.w["tok_emb"])[np.asarray(tokens)]
        f = bf16_bits_to_f64(a) if a.dtype == np.uint16 else a.astype(np.float64)
        return f.astype(self.dt, copy=False)

    # -- full-sequence forward (the definition) -------------------------------
    def forward(self, tokens, return_hidden: bool = False):
        """tokens [T] of one sequence -> logits [T, V], per-layer (k, v) [Hkv, T, hd]."""
        c = self.cfg
        x = self.embed(tokens)
        kv, hidden = [], [x.copy()]
        for l in range(c.n_layers):
            x, k, v = self.layer(l, x)
            kv.append((k, v))
            hidden.append(x.copy())
        logits = self.head(x)
        if return_hidden:
            return logits, kv, hidden
        return logits, kv

    def layer(self, l: int, x: np.ndarray):
        """Layer l over one full sequence x [T, d] (positions 0..T-1, causal).

        Returns the new residual and the layer's K, V as [Hkv, T, hd].
        """
        c, R = self.cfg, self.R
        x = np.asarray(x).astype(self.dt, copy=False)
        T = x.shape[0]
        H, Hk, hd = c.n_heads, c.n_kv_heads, c.head_dim
        pos = np.arange(T)
        p = f"l{l}."
        h = R(rmsnorm(x, self.mat(p + "attn_norm"), c.rms_eps))
        q = self.mm(h, p + "wq").reshape(T, H, hd)
        k = self.mm(h, p + "wk").reshape(T, Hk, hd)
        v = self.mm(h, p + "wv").reshape(T, Hk, hd)
        q = R(rope(q, pos, c.rope_theta))
        k = R(rope(k, pos, c.rope_theta))
        v = R(v)
        o = causal_attention(q, k, v)
        x = x + self.mm(R(o.reshape(T, H * hd)), p + "wo")
        h = R(rmsnorm(x, self.mat(p + "mlp_norm"), c.rms_eps))
        a = R(silu(self.mm(h, p + "w_gate")) * self.mm(h, p + "w_up"))
        x = x + self.mm(a, p + "w_down")
        return x, k.transpose(1, 0, 2).copy(), v.transpose(1, 0, 2).copy()

    def head(self, x: np.ndarray) -> np.ndarray:
        """Final RMSNorm + LM head: [n, d] -> [n, V]."""
        h = self.R(rmsnorm(x, self.mat("final_norm"), self.cfg.rms_eps))
        return self.mm(h, "lm_head")

    # -- one decode layer against a KV cache ---------------------------------
    def decode_layer(self, l: int, x: np.ndarray, pos: np.ndarray, K: np.ndarray,
                     V: np.ndarray):
        """x [B, d] residual in, pos [B], K/V [B, Hkv, >pos, hd] caches of layer l.

        Entries of K/V before each sequence's pos are read as given; the new
        token's k, v are computed, written at pos and returned with the
        updated residual.
        """
        c, R = self.cfg, self.R
        x = np.asarray(x).astype(self.dt, copy=False)
        B = x.shape[0]
        H, Hk, hd = c.n_heads, c.n_kv_heads, c.head_dim
        p = f"l{l}."
        h = R(rmsnorm(x, self.mat(p + "attn_norm"), c.rms_eps))
        q = self.mm(h, p + "wq").reshape(B, H, hd)
        k = self.mm(h, p + "wk").reshape(B, Hk, hd)
        v = self.mm(h, p + "wv").reshape(B, Hk, hd)
        o = np.empty((B, H, hd), self.dt)
        k_new = np.empty((B, Hk, hd), self.dt)
        v_new = np.empty((B, Hk, hd), self.dt)
        for b in range(B):
            pb = int(pos[b])
            qb = R(rope(q[b:b + 1], np.array([pb]), c.rope_theta))[0]
            kb = R(rope(k[b:b + 1], np.array([pb]), c.rope_theta))[0]
            vb = R(v[b])
            K[b, :, pb, :] = kb
            V[b, :, pb, :] = vb
            k_new[b], v_new[b] = kb, vb
            for hh in range(H):
                g = hh * Hk // H
                s = K[b, g, : pb + 1, :] @ qb[hh] / float(np.sqrt(hd))
                pr = np.exp(s - s.max())
                pr /= pr.sum()
                o[b, hh] = pr @ V[b, g, : pb + 1, :]
        x = x + self.mm(R(o.reshape(B, H * hd)), p + "wo")
        h = R(rmsnorm(x, self.mat(p + "mlp_norm"), c.rms_eps))
        a = R(silu(self.mm(h, p + "w_gate")) * self.mm(h, p + "w_up"))
        x = x + self.mm(a, p + "w_down")
        return x, k_new, v_new

    # -- a span of tokens appended to a cached sequence -----------------------
    def extend_layer(self, l: int, x: np.ndarray, pos0: int, K: np.ndarray, V: np.ndarray):
        """x [Te, d] residual of a span at positions pos0 .. pos0 + Te - 1 of one
        sequence whose K/V [Hkv, >= pos0 + Te, hd] hold positions 0 .. pos0 - 1;
        the span's k, v are written there and every row attends positions
        0 .. its own.  Returns the new residual (tool output injected into a live
        sequence, Sec. V-B)."""
        c, R = self.cfg, self.R
        x = np.asarray(x, np.float64)
        Te = x.shape[0]
        H, Hk, hd = c.n_heads, c.n_kv_heads, c.head_dim
        p = f"l{l}."
        pos = pos0 + np.arange(Te)
        h = R(rmsnorm(x, self.mat(p + "attn_norm"), c.rms_eps))
        q = R(rope(self.mm(h, p + "wq").reshape(Te, H, hd), pos, c.rope_theta))
        k = R(rope(self.mm(h, p + "wk").reshape(Te, Hk, hd), pos, c.rope_theta))
        v = R(self.mm(h, p + "wv").reshape(Te, Hk, hd))
        K[:, pos0:pos0 + Te] = k.transpose(1, 0, 2)
        V[:, pos0:pos0 + Te] = v.transpose(1, 0, 2)
        o = np.empty((Te, H, hd))
        for t in range(Te):
            n = pos0 + t + 1
            for hh in range(H):
                g = hh * Hk // H
                sc = K[g, :n] @ q[t, hh] / float(np.sqrt(hd))
                pr = np.exp(sc - sc.max())
                o[t, hh] = (pr / pr.sum()) @ V[g, :n]
        x = x + self.mm(R(o.reshape(Te, H * hd)), p + "wo")
        h = R(rmsnorm(x, self.mat(p + "mlp_norm"), c.rms_eps))
        a = R(silu(self.mm(h, p + "w_gate")) * self.mm(h, p + "w_up"))
        return x + self.mm(a, p + "w_down")

    def extend(self, tokens, pos0: int, K: np.ndarray, V: np.ndarray) -> np.ndarray:
        """Span tokens [Te] at positions pos0.. of one sequence with caches K/V
        [L, Hkv, Tmax, hd] (updated in place) -> logits of every span row [Te, V]."""
        x = self.embed(tokens)
        for l in range(self.cfg.n_layers):
            x = self.extend_layer(l, x, pos0, K[l], V[l])
        return self.head(x)

    def decode(self, tokens, pos, K: np.ndarray, V: np.ndarray, return_hidden: bool = False):
        """One decode step for B sequences; K/V [L, B, Hkv, Tmax, hd] updated in place."""
        x = self.embed(tokens)
        hidden = [x.copy()]
        for l in range(self.cfg.n_layers):
            x, _, _ = self.decode_layer(l, x, np.asarray(pos), K[l], V[l])
            hidden.append(x.copy())
        logits = self.head(x)
        return (logits, hidden) if return_hidden else logits

    # -- GRPO rollout: K samples per prompt -----------------------------------
    def rollout(self, prompts, group: int, new_tokens: int, temperature: float, top_k: int,
                seed: int, forced=None, keep_logits: bool = False, seq_ids=None):
        """Sample ``group`` completions of ``new_tokens`` tokens for every prompt.

        Sequence id of sample g of prompt p is p*group + g; the first token is
        generation step 0 (drawn from the prompt's last position), later tokens
        are steps 1..new_tokens-1 of cached decode.  ``forced`` [B, Tn] feeds the
        given tokens back instead of the oracle's own (teacher-forced replay);
        the oracle's own decision and its margin are still returned.
        """
        c = self.cfg
        prompts = np.asarray(prompts)
        P, Tp = prompts.shape
        B = P * group
        Tmax = Tp + new_tokens - 1
        L, Hk, hd = c.n_layers, c.n_kv_heads, c.head_dim
        K = np.zeros((L, B, Hk, max(Tmax, Tp), hd), self.dt)
        V = np.zeros_like(K)
        toks = np.zeros((B, new_tokens), np.int64)
        own = np.zeros((B, new_tokens), np.int64)
        logp = np.zeros((B, new_tokens))
        margin = np.zeros((B, new_tokens))
        logits_all = [] if keep_logits else None
        sid = np.arange(B) if seq_ids is None else np.asarray(seq_ids)
        first = np.zeros((B, c.vocab))
        for p in range(P):
            lg, kv = self.forward(prompts[p])
            for g in range(group):
                b = p * group + g
                for l in range(L):
                    K[l, b, :, :Tp] = kv[l][0]
                    V[l, b, :, :Tp] = kv[l][1]
                first[b] = lg[-1]
        cur = first
        for s in range(new_tokens):
            if s > 0:
                pos = np.full(B, Tp + s - 1)
                cur = self.decode(toks[:, s - 1], pos, K, V)
            if keep_logits:
                logits_all.append(cur.copy())
            for b in range(B):
                t, lp, m = sample_token(cur[b], temperature, top_k, seed, s, int(sid[b]))
                own[b, s], margin[b, s] = t, m
                toks[b, s] = t if forced is None else int(forced[b, s])
                z = cur[b] / (temperature if temperature > 0 else 1.0)
                logp[b, s] = lp if forced is None else float(log_softmax(z)[toks[b, s]])
        out = dict(tokens=toks, own_tokens=own, logp=logp, margin=margin, K=K, V=V)
        if keep_logits:
            out["logits"] = np.stack(logits_all, axis=1)
        return out

    # -- teacher-forced scoring -----------------------------------------------
    def score(self, tokens, score_from: int, temperature: float) -> np.ndarray:
        """logp[n, j - score_from] = log_softmax(l_{j-1} / T)[tok_j] for j in [score_from, T)."""
        tokens = np.asarray(tokens)
        N, T = tokens.shape
        Tt = temperature if temperature > 0 else 1.0
        out = np.zeros((N, T - score_from))
        for n in range(N):
            lg, _ = self.forward(tokens[n])
            ls = log_softmax(lg[score_from - 1:T - 1] / Tt)
            out[n] = ls[np.arange(T - score_from), tokens[n, score_from:]]
        return out
