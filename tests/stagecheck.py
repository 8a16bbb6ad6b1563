"""Rounding-point-local parity: every stage of the GPU forward, fed the GPU's
own inputs (from a grpo_trace), against the oracle's fp64 evaluation of that
stage, within the bounds of tests/bounds.py.

Stages of a layer (the precision contract's rounding points in brackets):
  h_attn = [rmsnorm(x) g]            q, k = [rope(h Wq^T, h Wk^T)], v = [h Wv^T]
  o = [softmax(q k^T / sqrt(hd)) v]  x_attn = x + o Wo^T
  h_mlp = [rmsnorm(x_attn) g]        act = [silu(h Wg^T) * (h Wu^T)]
  x' = x_attn + act Wd^T
and the head: h_final = [rmsnorm(x_L) g], logits = h_final W_head^T.
fp32 models have no rounding points: every output is an fp32 comparison.
"""
from __future__ import annotations

import numpy as np

import oracle
from bounds import (F32_GEMM, Report, attention_bound, check_bf16, check_f32, decode_gemm,
                    rmsnorm_bound, rope_bound, rows_gemm, swiglu_bound)


class StageChecker:
    def __init__(self, cfg, host, rep: Report | None = None):
        self.cfg = cfg
        self.om = oracle.OracleModel(cfg, host)
        self.rep = rep or Report()
        self.bf16 = cfg.dtype == 1

    def _round_check(self, name, gpu, y, E):
        if self.bf16:
            return check_bf16(self.rep, name, gpu, y, E)
        return check_f32(self.rep, name, gpu, y, E)

    def layer(self, l: int, tr: dict, ridx, pos, context, segments, gemms: dict):
        """Checks layer l on trace rows ridx (positions pos).

        context(i) -> (K, V) [ctx, n_kv, hd]: the GPU's cached keys and values
        that row ridx[i] attends (positions 0 .. pos[i]).
        segments(i) -> (segments, merges) of attention_bound for that row.
        gemms: Gemm structures of "qkv", "o", "gu" (gate/up) and "down"."""
        c, om = self.cfg, self.om
        ridx = np.asarray(ridx)
        pos = np.asarray(pos)
        H, Hk, hd, d = c.n_heads, c.n_kv_heads, c.head_dim, c.d_model
        qd, kvd, half = c.q_dim, c.kv_dim, c.head_dim // 2
        p = f"l{l}."
        x = tr["x"][l][ridx]
        # attention input norm
        y, E = rmsnorm_bound(x, om.mat(p + "attn_norm"), c.rms_eps)
        h = tr["h_attn"][l][ridx]
        self._round_check("h_attn", h, y, E)
        # QKV projection, RoPE on q and k
        Wqkv = np.concatenate([om.mat(p + "wq"), om.mat(p + "wk"), om.mat(p + "wv")], 0)
        yq, Eq = gemms["qkv"].bound(h, Wqkv)
        R = len(ridx)

        def rot(y_, E_, nh):
            y_ = y_.reshape(R, nh, hd)
            E_ = E_.reshape(R, nh, hd)
            lo, hi, Elo, Ehi = rope_bound(y_[..., :half], y_[..., half:], E_[..., :half],
                                          E_[..., half:], pos, c.rope_theta, hd)
            return (np.concatenate([lo, hi], -1).reshape(R, -1),
                    np.concatenate([Elo, Ehi], -1).reshape(R, -1))

        qy, qE = rot(yq[:, :qd], Eq[:, :qd], H)
        ky, kE = rot(yq[:, qd:qd + kvd], Eq[:, qd:qd + kvd], Hk)
        self._round_check("q", tr["q"][l][ridx], qy, qE)
        self._round_check("k", tr["k"][l][ridx], ky, kE)
        self._round_check("v", tr["v"][l][ridx], yq[:, qd + kvd:], Eq[:, qd + kvd:])
        # attention on the GPU's q, K, V
        qg = tr["q"][l][ridx].reshape(R, H, hd)
        oy = np.empty((R, H, hd))
        oE = np.empty((R, H, hd))
        for i in range(R):
            K, V = context(i)
            segs, merges = segments(i)
            for hh in range(H):
                g = hh * Hk // H
                oy[i, hh], oE[i, hh] = attention_bound(qg[i, hh], K[:, g], V[:, g], hd, segs,
                                                       merges)
        o = tr["o"][l][ridx]
        self._round_check("o", o, oy.reshape(R, qd), oE.reshape(R, qd))
        # O projection + residual
        y, E = gemms["o"].bound(o, om.mat(p + "wo"), resid=x)
        xa = tr["x_attn"][l][ridx]
        check_f32(self.rep, "x_attn", xa, y, E)
        # MLP input norm, SwiGLU
        y, E = rmsnorm_bound(xa, om.mat(p + "mlp_norm"), c.rms_eps)
        h2 = tr["h_mlp"][l][ridx]
        self._round_check("h_mlp", h2, y, E)
        gy, gE = gemms["gu"].bound(h2, om.mat(p + "w_gate"))
        uy, uE = gemms["gu"].bound(h2, om.mat(p + "w_up"))
        y, E = swiglu_bound(gy, uy, gE, uE)
        a = tr["act"][l][ridx]
        self._round_check("act", a, y, E)
        # down projection + residual
        y, E = gemms["down"].bound(a, om.mat(p + "w_down"), resid=xa)
        check_f32(self.rep, "x_out", tr["x"][l + 1][ridx], y, E)

    def head(self, tr: dict, hrows, xrows, gemm_head, cols=None, logit_tol=None):
        """Final norm of residual rows xrows (trace x[L]) into head rows hrows, and
        the logits (on a column subset `cols` of the vocabulary if given).
        Returns the largest |logit - oracle logit| seen."""
        c, om = self.cfg, self.om
        x = tr["x"][c.n_layers][np.asarray(xrows)]
        y, E = rmsnorm_bound(x, om.mat("final_norm"), c.rms_eps)
        h = tr["h_final"][np.asarray(hrows)]
        self._round_check("h_final", h, y, E)
        W = om.mat("lm_head")
        lg = tr["logits"][np.asarray(hrows)]
        if cols is not None:
            W, lg = W[cols], lg[:, cols]
        y, E = gemm_head.bound(h, W)
        check_f32(self.rep, "logits", lg, y, E)
        worst = float(np.abs(lg - y).max())
        if logit_tol is not None:
            self.rep.add("logits_tol", np.abs(lg - y) <= logit_tol)
        return worst


def flash_segments(ctx: int):
    """Prefill / scoring attention: one matrix-core chain over all keys."""
    return [("mfma", 0, ctx, ctx)], 0


def f32_segments(ctx: int):
    return [("f32", 0, ctx, ctx)], 0


def decode_segments(ctx: int, st: dict, base: int = 0):
    """Decode attention of a row with context ctx: prompt chunks below `base`
    (grouped steps), then the per-row spans from `base`."""
    segs = []
    if base > 0:
        segs.append(("mfma", 0, base, st["chunk"]))
    # the per-row spans from `base`: the row's positions past it cut evenly
    # into whole 128-position units, the last span running to the row's end
    n, ns = ctx - base, st["spans"]
    rspan = max(128, -(-(-(-n // ns)) // 128) * 128)
    for k in range(ns):
        a0 = base + k * rspan
        a1 = ctx if k == ns - 1 else min(a0 + rspan, ctx)
        if a0 < a1:
            segs.append(("decode", a0, a1, a1 - a0, st["waves"]))
    merges = st["waves"] + st["spans"] + (st["chunks"] + 1 if base > 0 else 0)
    return segs, merges


def gemms_decode(st: dict) -> dict:
    return dict(qkv=decode_gemm(st["splits_qkv"]), o=decode_gemm(st["splits_o"]),
                gu=decode_gemm(1), down=decode_gemm(st["splits_down"]))


def gemms_rows(cfg, M: int) -> dict:
    g = F32_GEMM if cfg.dtype == 0 else rows_gemm(M)
    return dict(qkv=g, o=g, gu=g, down=g)


def logp_bound(z, logp):
    """Bound on the GPU's fp32 log-probability z_tok - LSE(z) of a draw given its
    logits, for both ways the draw is made.  The sampler kernel: z = l / T (u |z|),
    exponent arguments z - max (u |z - m|), the exponentials (C_EXP u), a sum of V
    positive terms read by at least 256 threads (at most V / 256 per thread, then
    16 reduction levels), the log and the final subtractions (u each of |LSE| and
    |logp|).  The decode LM head's sampling epilogue: per output tile of at most
    128 ids four threads sum at most 32 terms each over 2 shuffle levels, and the
    combine rescales every tile by exp(m_s / T - M / T) (argument 2u max|z|,
    C_EXP u, one fused multiply-add) and sums V / 32 / 64 tiles per lane over 6
    levels.  The bound takes each term's larger value."""
    from bounds import C_EXP, U
    zmax = float(np.max(np.abs(z)))
    lse = float(np.max(z) + np.log(np.sum(np.exp(z - np.max(z)))))
    h_sum = max(len(z) / 256.0 + 16.0, 32.0 + 2.0 + np.ceil(len(z) / 32.0 / 64.0) + 6.0 + 1.0)
    return U * (h_sum + 8.0 + 2.0 * C_EXP + 6.0 * zmax + 3.0 * abs(lse) + abs(float(logp)))


def score_logp_bound(z, logp):
    """Bound on the scoring head's fp32 log-probability given its logits (z = l / T
    in fp64 here): the product's epilogue scales x = l * fl(log2(e) / T) (c off by
    2u, each x by u: 3u |z| in natural-log units), takes per 64-column slot the
    maximum and sum_n 2^(x_n - max) (arguments u |x - max| <= 2u max|z|, exp2 C_EXP u,
    at most 64 terms in a chain), then the combine rescales each slot by
    2^(m_s - M) (another 2u max|z| and C_EXP u, one fused multiply-add) and sums
    V / 64 / 64 slots per lane over 6 reduction levels; log2, M + log2 S, the
    product by ln 2 (u |LSE| each), z_t = l_t / T (u |z|) and the difference
    (u |logp|)."""
    from bounds import C_EXP, U
    zmax = float(np.max(np.abs(z)))
    lse = float(np.max(z) + np.log(np.sum(np.exp(z - np.max(z)))))
    h_sum = 64.0 + np.ceil(len(z) / 64.0) / 64.0 + 6.0 + 2.0
    return U * (h_sum + 2.0 * C_EXP + 4.0 + 8.0 * zmax + 3.0 * abs(lse) + abs(float(logp)))


def sampler_check(logits, toks, logps, temperature, top_k, seed, step, seq_ids,
                  band: float = 1e-5):
    """The oracle sampler on the GPU's own fp32 logits: tokens bit-exact except at a
    logged near-tie (winning margin below `band`), log-probs within logp_bound.
    Returns the number of near-ties."""
    near = 0
    T = temperature if temperature > 0 else 1.0
    for b in range(len(toks)):
        l = np.asarray(logits[b], np.float64)
        t, lp, margin = oracle.sample_token(l, temperature, top_k, seed, step, int(seq_ids[b]))
        if margin < band:
            near += 1
            continue
        assert int(toks[b]) == t, (b, int(toks[b]), t, margin)
        assert abs(float(logps[b]) - lp) <= logp_bound(l / T, lp), (b, float(logps[b]), lp)
    return near
