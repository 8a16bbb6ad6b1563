"""GPU parity of the fused scoring head (Alg. 1 scoring, log pi of each scored
token).  The LM-head product's epilogue reduces every row's logits to per-slot
log-sum-exp pieces plus the target's logit, and a combine kernel forms
log_softmax(l / T) at the target: the logits are never stored (a traced call
also writes them into its trace by a second product).  Checked per case:
the traced logits stage-locally against the oracle's fp64 head on the GPU's
own normed rows, every scored row's log-prob against log_softmax of those
logits within the bound of the fused arithmetic (stagecheck.score_logp_bound),
and the log-probs end to end against the oracle's teacher-forced scoring.
The cases cover the three product kernels (256 x 256 tiles: >= 1024 rows and a
vocabulary in multiples of 256, 32000 and 152064 ids; 128 x 128 tiles; fp32),
vocabularies that end inside a 64-column slot or leave a tile's second half
past the last column, and temperatures other than 1 (0 scores at 1)."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from bounds import F32_GEMM, Gemm
from gpu_util import assert_report, build_model, head_cols, logit_tol, require_gpu, say
from paper_2510_17158_amd import api
from paper_2510_17158_amd.workloads import DTYPE_F32, SMALL, TINY
from stagecheck import StageChecker, score_logp_bound

pytestmark = pytest.mark.gpu

S1 = dataclasses.replace(SMALL, n_layers=1)
T1 = dataclasses.replace(TINY, n_layers=1)
CASES = [
    # cfg, sequences, T, score_from, temperature; scored rows = N (T - score_from)
    (S1, 2, 1100, 500, 1.3),                                 # 1200 rows, V 32000: 256 x 256
    (dataclasses.replace(S1, vocab=152064), 2, 600, 80, 1.1),  # 1040 rows, the 32B vocabulary
    (dataclasses.replace(S1, vocab=1040), 2, 1100, 500, 0.7),  # 128 x 128, last tile half empty
    (dataclasses.replace(S1, vocab=4000), 3, 150, 20, 1.0),    # 390 rows, V % 64 = 32
    (dataclasses.replace(T1, vocab=1000), 2, 90, 30, 0.8),     # fp32, V % 64 = 40
    (T1, 2, 90, 30, 0.0),                                      # fp32, temperature 0 -> 1
]


@pytest.mark.parametrize("cfg,N,T,sf,temp", CASES)
def test_fused_scoring_head(cfg, N, T, sf, temp):
    require_gpu()
    say("fused scoring head", "fp32" if cfg.dtype == DTYPE_F32 else "bf16", cfg.vocab, N, T, sf,
        temp)
    host, model = build_model(cfg, 91, gain_noise=0.1)
    rng = np.random.default_rng(cfg.vocab + T)
    seqs = rng.integers(0, cfg.vocab, (N, T)).astype(np.int32)
    Ts, R, V = T - sf, N * (T - sf), cfg.vocab
    tok = torch.from_numpy(seqs).cuda()
    ws = api.alloc_workspace(model, api.OP_SCORE, N, T)
    tr = api.Trace(cfg, N * T, R)
    lp = torch.empty(N, Ts, device="cuda")
    api.score_sequences(model, tok, sf, temp, lp, trace=tr, ws=ws)
    torch.cuda.synchronize()
    t = tr.numpy()
    lp = lp.cpu().numpy()
    assert np.isfinite(lp).all()
    Tt = temp if temp > 0 else 1.0

    # the traced logits, stage-local on sampled rows (one product over all R rows)
    hrows = np.unique(np.concatenate([[0, Ts - 1, R - 1], rng.integers(0, R, 13)]))
    xrows = hrows // Ts * T + sf - 1 + hrows % Ts
    chk = StageChecker(cfg, host)
    # 256 x 256 tiles (32x32x16 chains) need >= 1024 rows and V in multiples of 256
    g = (F32_GEMM if cfg.dtype == DTYPE_F32
         else Gemm("mfma", 16 if R >= 1024 and V % 256 == 0 else 32))
    worst = chk.head(t, hrows, xrows, g, cols=head_cols(V, t["logits"][hrows]),
                     logit_tol=logit_tol(cfg))
    assert_report(chk.rep, f"scoring head (worst logit err {worst:.2e})")

    # every row's log-prob against log_softmax of its own logits
    tgt = seqs[:, sf:].ravel()
    flat = lp.ravel()
    worst_r = 0.0
    for r in range(R):
        z = t["logits"][r].astype(np.float64) / Tt
        ref = float(oracle.log_softmax(z)[tgt[r]])
        err = abs(float(flat[r]) - ref)
        worst_r = max(worst_r, err / score_logp_bound(z, ref))
        assert err <= score_logp_bound(z, ref), (r, float(flat[r]), ref)
    say("log-probs vs their own logits: worst error / bound", worst_r)

    # end to end against the oracle's teacher-forced scoring
    ref = oracle.OracleModel(cfg, host).score(seqs, sf, temp)
    e2e = float(np.abs(lp - ref).max())
    say("end to end vs oracle", e2e)
    assert e2e <= logit_tol(cfg)
    model.close()
