"""Seeded synthetic inputs for the GRPO hot path.

The paper trains on kernel-optimisation tasks whose datasets and trained
weights are not available (Sec. IV, Sec. VI-C).  These generators stand in for
them with inputs of the same structure: random-init Llama-style weights, prompts
shaped like tool-augmented kernel-optimisation rollouts (code-like token
stream, tool-call marker, arguments, result marker and a tool-output span, as in
the paper's example reasoning trace), and rewards in the paper's reward range.

This module holds none of the method's arithmetic.  It only draws random
numbers and stores them; both the HIP path and the CPU oracle consume what it
returns.  bf16 weights are produced with torch's own CPU conversion and handed
out as uint16 bit patterns.
"""
from __future__ import annotations

import concurrent.futures as cf
import os

import numpy as np
import torch

from .workloads import DTYPE_F32, ModelConfig, Workload

# Reserved token ids: BOS, the four trace markers (reasoning, tool call, tool
# result, final answer) and EOS.  EOS never stops generation: lengths are fixed.
BOS, REASONING, TOOL, RESULT, FINAL, EOS = 0, 1, 2, 3, 4, 5
FIRST_FREE_ID = 16
TOOL_ARG_LEN = 16
TOOL_OUT_LEN = 256
NUMERIC_BAND = 512

REF_MIX = 0.05       # reference weights = policy + REF_MIX * (a shifted copy of policy)
REF_SHIFT = 7919


def _children(seed: int):
    """(weights, prompts, rewards, philox, extra) seed sequences of one workload."""
    return np.random.SeedSequence(seed).spawn(5)


def tensor_names(cfg: ModelConfig) -> list[str]:
    names = ["tok_emb"]
    for i in range(cfg.n_layers):
        names += [f"l{i}.{t}" for t in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm",
                                        "w_gate", "w_up", "w_down")]
    return names + ["final_norm", "lm_head"]


def tensor_shape(cfg: ModelConfig, name: str) -> tuple[int, ...]:
    d, f, V = cfg.d_model, cfg.d_ffn, cfg.vocab
    t = name.split(".")[-1]
    return {
        "tok_emb": (V, d), "lm_head": (V, d), "final_norm": (d,),
        "attn_norm": (d,), "mlp_norm": (d,),
        "wq": (cfg.q_dim, d), "wk": (cfg.kv_dim, d), "wv": (cfg.kv_dim, d),
        "wo": (d, cfg.q_dim),
        "w_gate": (f, d), "w_up": (f, d), "w_down": (d, f),
    }[t]


def _to_bf16_bits(x32: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(x32, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _draw(cfg: ModelConfig, name: str, ss: np.random.SeedSequence, gain_noise: float,
          ref: bool, std: float) -> np.ndarray:
    shape = tensor_shape(cfg, name)
    rng = np.random.default_rng(ss)
    if name.endswith("norm"):
        x = np.ones(shape, np.float32)
        if gain_noise:
            x += np.float32(gain_noise) * rng.standard_normal(shape, dtype=np.float32)
    else:
        x = rng.standard_normal(shape, dtype=np.float32)
        x *= np.float32(std)
        if ref:
            flat = x.reshape(-1)
            x = (flat + np.float32(REF_MIX) * np.roll(flat, REF_SHIFT)).reshape(shape)
    if cfg.dtype == DTYPE_F32:
        return x
    return _to_bf16_bits(x)


def make_weights(cfg: ModelConfig, seed: int, *, ref: bool = False, gain_noise: float = 0.0,
                 std: float = 0.02, names: list[str] | None = None,
                 threads: int | None = None) -> dict[str, np.ndarray]:
    """Random-init weights, N(0, std^2) per matrix, norm gains 1 (+ optional noise).

    Every tensor has its own child seed, so any one of them can be regenerated on
    its own.  bf16 models return uint16 bit patterns (RNE of the fp32 draw), fp32
    models return float32.  ``ref=True`` gives the frozen reference copy used for
    the KL term: the policy draw plus a small shifted copy of itself.
    """
    all_names = tensor_names(cfg)
    kids = _children(seed)[0].spawn(len(all_names))
    want = all_names if names is None else names
    idx = {n: i for i, n in enumerate(all_names)}
    threads = threads or min(16, os.cpu_count() or 1)

    def one(n):
        return n, _draw(cfg, n, kids[idx[n]], gain_noise, ref, std)

    if len(want) == 1 or threads == 1:
        return dict(map(one, want))
    with cf.ThreadPoolExecutor(threads) as ex:
        return dict(ex.map(one, want))


def _code_stream(rng: np.random.Generator, n: int, V: int, perm: np.ndarray) -> np.ndarray:
    """Zipf(1.2)-ranked ids through a fixed permutation, with copied spans."""
    out = np.empty(n, np.int64)
    i = 0
    while i < n:
        if i >= 16 and rng.random() < 0.3:
            ln = int(rng.integers(4, 17))
            src = int(rng.integers(0, i - 4 + 1))
            ln = min(ln, n - i, i - src)
            out[i:i + ln] = out[src:src + ln]
            i += ln
        else:
            r = int(rng.zipf(1.2))
            out[i] = perm[(r - 1) % len(perm)]
            i += 1
    return out


def make_prompts(w: Workload) -> np.ndarray:
    """int32 [P, Tp] prompt tokens."""
    rng = np.random.default_rng(_children(w.master_seed)[1])
    V, P, Tp = w.model.vocab, w.n_prompts, w.prompt_len
    if w.prompt_kind == "uniform":
        return rng.integers(0, V, size=(P, Tp)).astype(np.int32)
    perm = rng.permutation(np.arange(FIRST_FREE_ID, V))
    band0 = int(rng.integers(FIRST_FREE_ID, V - NUMERIC_BAND))
    span = 2 + TOOL_ARG_LEN + TOOL_OUT_LEN
    out = np.empty((P, Tp), np.int64)
    for p in range(P):
        row = _code_stream(rng, Tp, V, perm)
        row[0] = BOS
        n_sp = w.tool_spans
        free = Tp - 1 - n_sp * span
        if n_sp and free > 0:
            # non-overlapping offsets: choose n_sp cut points in the free text
            cuts = np.sort(rng.choice(free + 1, size=n_sp, replace=True))
            pos = 1 + cuts + np.arange(n_sp) * span
            for s in pos:
                row[s] = TOOL
                row[s + 1:s + 1 + TOOL_ARG_LEN] = perm[rng.integers(0, 64, TOOL_ARG_LEN)]
                row[s + 1 + TOOL_ARG_LEN] = RESULT
                row[s + 2 + TOOL_ARG_LEN:s + span] = band0 + rng.integers(0, NUMERIC_BAND,
                                                                          TOOL_OUT_LEN)
        out[p] = row
    return out.astype(np.int32)


def make_rewards(w: Workload) -> np.ndarray:
    """float32 [P*G]: 0 with probability 0.3, else lognormal(0, 0.5)."""
    rng = np.random.default_rng(_children(w.master_seed)[2])
    n = w.batch
    zero = rng.random(n) < 0.3
    r = rng.lognormal(0.0, 0.5, n)
    return np.where(zero, 0.0, r).astype(np.float32)


def make_seed(w: Workload) -> int:
    """64-bit key of the counter-based sampler."""
    rng = np.random.default_rng(_children(w.master_seed)[3])
    return int(rng.integers(0, 2**63 - 1, dtype=np.int64))


def make_loss_inputs(n: int, t: int, seed: int, *, mask_p: float = 0.9,
                     drift: float = 0.05) -> dict[str, np.ndarray]:
    """Synthetic per-token log-probs and mask shaped like a rollout's."""
    rng = np.random.default_rng(seed)
    lp_old = -rng.exponential(2.0, size=(n, t))
    lp = lp_old + drift * rng.standard_normal((n, t))
    lp_ref = lp + drift * rng.standard_normal((n, t))
    mask = (rng.random((n, t)) < mask_p).astype(np.uint8)
    adv = rng.standard_normal(n)
    return {k: v.astype(np.float32) if v.dtype == np.float64 else v
            for k, v in dict(logp=lp, logp_old=lp_old, logp_ref=lp_ref, mask=mask,
                             adv=adv).items()}
