"""Shared set-up of the GPU parity tests (not collected: no test_ prefix)."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
from bounds import Report
from paper_2510_17158_amd import api, synth
from paper_2510_17158_amd.workloads import DTYPE_F32, ModelConfig
from stagecheck import (StageChecker, decode_segments, f32_segments, flash_segments,
                        gemms_decode, gemms_rows, sampler_check)
from bounds import F32_GEMM, decode_gemm, rows_gemm

LOGIT_TOL = 2e-2       # bf16 logits / log-probs (stated tolerance)
LOGIT_TOL_F32 = 1e-4   # fp32 logits / log-probs (stated tolerance)
NEAR_TIE = 1e-5        # sampler decisions closer than this are logged, not compared


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    api.lib()   # fails loudly if the HIP library is missing


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def build_model(cfg: ModelConfig, seed: int, gain_noise: float = 0.1, ref: bool = False,
                std: float = 0.02):
    host = synth.make_weights(cfg, seed, gain_noise=gain_noise, ref=ref, std=std)
    dev = api.upload_weights(cfg, host)
    return host, api.Model(cfg, dev)


def kv_view(cfg: ModelConfig, kv: torch.Tensor, n_seqs: int, max_len: int) -> np.ndarray:
    """KV buffer -> float64 array [L, 2, n_seqs, n_kv, max_len, hd]."""
    shape = (cfg.n_layers, 2, n_seqs, cfg.n_kv_heads, max_len, cfg.head_dim)
    if cfg.dtype == DTYPE_F32:
        return kv.view(torch.float32).view(shape).double().cpu().numpy()
    return kv.view(torch.bfloat16).view(shape).double().cpu().numpy()


def logit_tol(cfg) -> float:
    return LOGIT_TOL_F32 if cfg.dtype == DTYPE_F32 else LOGIT_TOL


def head_cols(V: int, logits: np.ndarray, n: int = 4096, seed: int = 0) -> np.ndarray | None:
    """Vocabulary columns on which the LM-head bound is evaluated: all of a small
    vocabulary, else n random ones plus every row's largest logits."""
    if V <= n:
        return None
    rng = np.random.default_rng(seed)
    top = np.argsort(-logits, axis=1)[:, :4].ravel()
    return np.unique(np.concatenate([rng.choice(V, n, replace=False), top]))


# ------------------------------------------------------------- decode step
def decode_traced(model: api.Model, kv, n_seqs, max_len, pos_host, tok_dev, step: int,
                  sampling, ws, group: int = 0, prefix_len: int = 0, seq_ids=None):
    """One traced decode step for the rows of pos_host (host positions, written to a
    fresh device pos array).  Returns (trace numpy dict, tokens, log-probs)."""
    cfg = model.cfg
    B = len(pos_host)
    pos = torch.from_numpy(np.asarray(pos_host, np.int32)).to("cuda")
    tr = api.Trace(cfg, B, B)
    to = torch.empty(B, 1, dtype=torch.int32, device="cuda")
    lo = torch.empty(B, 1, device="cuda")
    api.rollout_step(model, kv, n_seqs, max_len, pos, tok_dev, int(np.max(pos_host)), step, 1,
                     sampling, to, lo, seq_ids=seq_ids, trace=tr, ws=ws, group=group,
                     prefix_len=prefix_len)
    torch.cuda.synchronize()
    return tr.numpy(), to.cpu().numpy()[:, 0], lo.cpu().numpy()[:, 0]


def check_decode(cfg, host, model, tr: dict, kvnp: np.ndarray, pos, max_len: int, rows=None,
                 group: int = 0, prefix_len: int = 0, slots=None, rep: Report | None = None):
    """Rounding-point-local check of a traced decode step.  kvnp: the cache after
    the step ([L, 2, n_seqs, n_kv, max_len, hd]); pos: each row's position; slots:
    each row's cache slot (seq_ids)."""
    pos = np.asarray(pos)
    B = len(pos)
    rows = np.arange(B) if rows is None else np.asarray(rows)
    slots = np.arange(B) if slots is None else np.asarray(slots)
    chk = StageChecker(cfg, host, rep)
    if cfg.dtype == DTYPE_F32:
        gem = gemms_rows(cfg, B)
        seg = lambda i: f32_segments(int(pos[rows[i]]) + 1)   # noqa: E731
        ghead = F32_GEMM
    else:
        st = api.decode_structure(model, B, max_len, group, prefix_len)
        gem = gemms_decode(st)
        ghead = decode_gemm(st["splits_head"])
        grouped = group > 0 and prefix_len > 0

        def seg(i):
            b = rows[i]
            ctx = int(pos[b]) + 1
            base = 0
            if grouped:
                g0 = b // group * group
                base = min(prefix_len, int((pos[g0:g0 + group] + 1).min()))
            return decode_segments(ctx, st, base)
    for l in range(cfg.n_layers):
        def context(i, l=l):
            b = rows[i]
            ctx = int(pos[b]) + 1
            K = kvnp[l, 0, slots[b], :, :ctx].transpose(1, 0, 2)
            V = kvnp[l, 1, slots[b], :, :ctx].transpose(1, 0, 2)
            return K, V
        chk.layer(l, tr, rows, pos[rows], context, seg, gem)
    cols = head_cols(cfg.vocab, tr["logits"][rows])
    worst = chk.head(tr, rows, rows, ghead, cols=cols, logit_tol=logit_tol(cfg))
    return chk.rep, worst


# ------------------------------------------------------- many-row forwards
def check_rows(cfg, host, tr: dict, T: int, M_call: int, rows, rep: Report | None = None,
               head=None):
    """Rounding-point-local check of a traced prefill or scoring forward on the
    trace rows `rows` (row = seq * T + t).  M_call: rows of the call's GEMMs.
    head: None, or (head_rows, x_rows, M_head) for the LM-head check."""
    rows = np.asarray(rows)
    chk = StageChecker(cfg, host, rep)
    gem = gemms_rows(cfg, M_call)
    pos = rows % T
    for l in range(cfg.n_layers):
        seq_kv = {}

        def context(i, l=l):
            r = rows[i]
            s0 = r - r % T
            if s0 not in seq_kv:
                seq_kv.clear()
                last = int(rows[rows < s0 + T].max())      # the sequence's last checked row
                seq_kv[s0] = (tr["k"][l][s0:last + 1].reshape(-1, cfg.n_kv_heads, cfg.head_dim),
                              tr["v"][l][s0:last + 1].reshape(-1, cfg.n_kv_heads, cfg.head_dim))
            K, V = seq_kv[s0]
            return K[:r - s0 + 1], V[:r - s0 + 1]
        segf = f32_segments if cfg.dtype == DTYPE_F32 else flash_segments
        chk.layer(l, tr, rows, pos, context, lambda i: segf(int(pos[i]) + 1), gem)
    worst = None
    if head is not None:
        hrows, xrows, M_head = head
        g = F32_GEMM if cfg.dtype == DTYPE_F32 else rows_gemm(M_head)
        cols = head_cols(cfg.vocab, tr["logits"][np.asarray(hrows)])
        worst = chk.head(tr, hrows, xrows, g, cols=cols, logit_tol=logit_tol(cfg))
    return chk.rep, worst


def sample_rows(T: int, n_seqs: int, k: int, seed: int = 0, lo: int = 0, hi: int | None = None):
    """Rows to check: per sequence the first and last rows, rows around 32/64-row
    tile edges, and k random rows from [lo, hi)."""
    hi = T if hi is None else hi
    rng = np.random.default_rng(seed)
    edges = [t for e in (31, 32, 63, 64, 127, 128, 255, 256, 1023, 1024, 2047, 2048, 4095)
             for t in (e,) if lo <= t < hi]
    out = []
    for s in range(n_seqs):
        r = set([lo, hi - 1] + edges)
        r.update(rng.integers(lo, hi, k).tolist())
        out.extend(s * T + t for t in sorted(r))
    return np.array(sorted(out))


def assert_report(rep: Report, label: str):
    say(label, rep.summary())
    assert rep.ok(), rep.summary()


def check_extend(cfg, host, tr: dict, kvnp: np.ndarray, pos0, Te: int, slots,
                 rows=None, rep: Report | None = None):
    """Rounding-point-local check of a traced grpo_extend: span row r of sequence
    b = r // Te sits at position pos0[b] + r % Te of cache slot slots[b] and
    attends that slot's positions 0 .. its own (one matrix-core chain over the
    keys on bf16 models); the head on each sequence's last span row."""
    pos0 = np.asarray(pos0)
    slots = np.asarray(slots)
    B = len(pos0)
    M = B * Te
    rows = np.arange(M) if rows is None else np.asarray(rows)
    pos = pos0[rows // Te] + rows % Te
    chk = StageChecker(cfg, host, rep)
    gem = gemms_rows(cfg, M)
    segf = f32_segments if cfg.dtype == DTYPE_F32 else flash_segments
    for l in range(cfg.n_layers):
        def context(i, l=l):
            b = rows[i] // Te
            ctx = int(pos[i]) + 1
            return (kvnp[l, 0, slots[b], :, :ctx].transpose(1, 0, 2),
                    kvnp[l, 1, slots[b], :, :ctx].transpose(1, 0, 2))
        chk.layer(l, tr, rows, pos, context, lambda i: segf(int(pos[i]) + 1), gem)
    g = F32_GEMM if cfg.dtype == DTYPE_F32 else rows_gemm(B)
    hrows = np.arange(B)
    cols = head_cols(cfg.vocab, tr["logits"][hrows])
    worst = chk.head(tr, hrows, hrows * Te + Te - 1, g, cols=cols, logit_tol=logit_tol(cfg))
    return chk.rep, worst
