"""GPU parity on bf16 decoders: stage-local (every decode layer fed the GPU's
own residual and KV cache), the LM head + sampler on the GPU's final state, and
end to end at the small shape (12 layers, d 768, GQA 12/4) where the bf16
logit tolerance 2e-2 holds literally.

Prompt length 300 spans three 128-row GEMM tiles, five 64-row attention blocks
and two 256-position decode splits, each with a ragged tail."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2510_17158_amd import api, synth
from paper_2510_17158_amd.runner import GrpoIteration
from paper_2510_17158_amd.workloads import get, truncated

from gpu_util import bf16_ulps, build_model, kv_view, require_gpu, say

pytestmark = pytest.mark.gpu

LOGIT_TOL = 2e-2     # bf16 logits / log-probs
RESID_TOL = 2e-3     # one decode layer's residual output, fed identical inputs


def _small_workload(**kw):
    w = get("small").with_(n_prompts=2, group=4, prompt_len=300, new_tokens=6, temperature=1.0)
    return w.with_(**kw)


def _stage_local(w, host, model, it, n_steps, check_layers=True):
    """Decode n_steps one at a time; check every layer, the head and the sampler."""
    cfg = w.model
    B, L, d, V = it.B, cfg.n_layers, cfg.d_model, cfg.vocab
    om = oracle.OracleModel(cfg, host)
    it.tok.copy_(it.tok0)
    it.pos.fill_(w.prompt_len)
    worst = dict(resid=0.0, kv_flip=0.0, kv_ulps=0, logit=0.0, near=0)
    toks = []
    for s in range(n_steps):
        pos = w.prompt_len + s
        to = torch.empty(B, 1, dtype=torch.int32, device="cuda")
        lo = torch.empty(B, 1, device="cuda")
        lg = torch.empty(B, V, device="cuda")
        hid = torch.empty(L + 1, B, d, device="cuda")
        api.rollout_step(model, it.kv, B, it.max_len, it.pos, it.tok, pos, 1 + s, 1, it.sampling,
                         to, lo, logits_dbg=lg, hidden_dbg=hid, ws=it.ws_roll)
        torch.cuda.synchronize()
        hid = hid.double().cpu().numpy()
        lg = lg.cpu().numpy()
        to = to.cpu().numpy()[:, 0]
        lo = lo.cpu().numpy()[:, 0]
        toks.append(to)
        if check_layers:
            kv = kv_view(cfg, it.kv, B, it.max_len)
            posv = np.full(B, pos)
            for l in range(L):
                K = kv[l, 0].copy()
                Vv = kv[l, 1].copy()
                x1, kn, vn = om.decode_layer(l, hid[l], posv, K, Vv)
                worst["resid"] = max(worst["resid"], float(np.abs(x1 - hid[l + 1]).max()))
                u = np.concatenate([bf16_ulps(kn, kv[l, 0, :, :, pos]).ravel(),
                                    bf16_ulps(vn, kv[l, 1, :, :, pos]).ravel()])
                worst["kv_ulps"] = max(worst["kv_ulps"], int(u.max()))
                worst["kv_flip"] = max(worst["kv_flip"], float((u > 0).mean()))
        ref_logits = om.head(hid[L])
        worst["logit"] = max(worst["logit"], float(np.abs(ref_logits - lg).max()))
        for b in range(B):
            t, lp, margin = oracle.sample_token(lg[b].astype(np.float64), w.temperature, w.top_k,
                                                it.sampling.seed, 1 + s, b)
            if margin < 1e-4:
                worst["near"] += 1
                continue
            assert to[b] == t, (s, b)
            assert abs(lo[b] - lp) <= 1e-5
    say("stage-local worst:", worst)
    assert worst["resid"] <= RESID_TOL
    assert worst["kv_ulps"] <= 1
    assert worst["logit"] <= LOGIT_TOL
    return np.stack(toks, 1), worst


@pytest.fixture(scope="module")
def small():
    require_gpu()
    w = _small_workload()
    host, model = build_model(w.model, w.master_seed, gain_noise=0.1)
    return w, host, model


def test_small_end_to_end(small):
    w, host, model = small
    say("small end to end")
    prompts = synth.make_prompts(w)
    seed = synth.make_seed(w)
    it = GrpoIteration(w, model, None, prompts, synth.make_rewards(w), seed)
    lg0 = torch.empty(w.n_prompts, w.model.vocab, device="cuda")
    it.prefill(logits_dbg=lg0)
    it.decode()
    it.assemble()
    torch.cuda.synchronize()
    seqs = it.seqs.cpu().numpy()
    gpu_tokens = seqs[:, w.prompt_len:]
    om = oracle.OracleModel(w.model, host)
    ref = om.rollout(prompts, w.group, w.new_tokens, w.temperature, w.top_k, seed,
                     forced=gpu_tokens)
    # prefill: last-position logits and the layer-0 cache (exact inputs) against the oracle
    for p in range(w.n_prompts):
        lgp, kvp = om.forward(prompts[p])
        e = np.abs(lg0[p].cpu().numpy() - lgp[-1]).max()
        say("prefill logits", p, e)
        assert e <= LOGIT_TOL
        kv = kv_view(w.model, it.kv, it.B, it.max_len)
        u = bf16_ulps(kv[0, 0, p * w.group, :, : w.prompt_len], kvp[0][0])
        say("layer-0 K ulps max", int(u.max()), "flip frac", float((u > 0).mean()))
        assert u.max() <= 1
    # rollout log-probs vs the teacher-forced oracle (same token history)
    lp_gpu = it.logp_old.cpu().numpy()
    e = np.abs(lp_gpu - ref["logp"]).max()
    say("rollout logp max err", e)
    assert e <= LOGIT_TOL
    near = ref["margin"] < 2 * LOGIT_TOL / w.temperature
    mism = (gpu_tokens != ref["own_tokens"]) & ~near
    say("near ties", int(near.sum()), "mismatches", int(mism.sum()))
    assert not mism.any()
    # scoring
    ws = api.alloc_workspace(model, api.OP_SCORE, it.B, it.T)
    lp = torch.empty(it.B, w.new_tokens, device="cuda")
    api.score_sequences(model, it.seqs, w.prompt_len, w.temperature, lp, ws=ws)
    torch.cuda.synchronize()
    lp = lp.cpu().numpy()
    sc = om.score(seqs, w.prompt_len, w.temperature)
    say("score err", np.abs(lp - sc).max(), "score vs rollout", np.abs(lp - lp_gpu).max())
    assert np.abs(lp - sc).max() <= LOGIT_TOL
    assert np.abs(lp - lp_gpu).max() <= LOGIT_TOL


def test_small_stage_local(small):
    w, host, model = small
    say("small stage-local")
    it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w),
                       synth.make_seed(w))
    it.prefill()
    _stage_local(w, host, model, it, 3)


@pytest.mark.parametrize("name,layers,kw", [
    ("1b", 2, dict(n_prompts=1, group=4, prompt_len=70, new_tokens=3, temperature=0.8,
                   top_k=50)),
    ("7b", 1, dict(n_prompts=1, group=3, prompt_len=65, new_tokens=3)),
    ("32b", 1, dict(n_prompts=1, group=2, prompt_len=40, new_tokens=2)),
])
def test_full_width_stage_local(name, layers, kw):
    """Layer-truncated models at the 1B/7B/32B widths: every stage fed GPU inputs."""
    require_gpu()
    say("full width stage-local", name, layers)
    w = truncated(get(name), layers, **kw)
    host, model = build_model(w.model, w.master_seed, gain_noise=0.1)
    it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w),
                       synth.make_seed(w))
    lg0 = torch.empty(w.n_prompts, w.model.vocab, device="cuda")
    it.prefill(logits_dbg=lg0)
    torch.cuda.synchronize()
    om = oracle.OracleModel(w.model, host)
    lgp, kvp = om.forward(synth.make_prompts(w)[0])
    e = np.abs(lg0[0].cpu().numpy() - lgp[-1]).max()
    say("prefill logits err", e)
    assert e <= LOGIT_TOL
    _stage_local(w, host, model, it, w.new_tokens - 1)
    model.close()
