"""GPU parity on the 2-layer fp32 decoder (the tiny workload: 4 prompts x G=4,
64-token prompts, 64 greedy tokens): end to end against the fp64 oracle at the
fp32 tolerance 1e-4; every stage of a prefill and a decode step against the
oracle on the GPU's own inputs within the bounds of its fp32 arithmetic; the
sampler on the GPU's logits for sampled decoding."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2510_17158_amd import api, synth
from paper_2510_17158_amd.runner import GrpoIteration
from paper_2510_17158_amd.workloads import get

from gpu_util import (NEAR_TIE, assert_report, build_model, check_decode, check_rows,
                      decode_traced, kv_view, require_gpu, say)
from stagecheck import sampler_check

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _stepwise(it: GrpoIteration, n: int):
    """Decode n steps one call at a time, collecting the logits of every step."""
    B, V = it.B, it.w.model.vocab
    it.tok.copy_(it.tok0)
    it.pos.fill_(it.w.prompt_len)
    toks, lps, logits = [], [], []
    for s in range(n):
        to = torch.empty(B, 1, dtype=torch.int32, device="cuda")
        lo = torch.empty(B, 1, dtype=torch.float32, device="cuda")
        tr = api.Trace(it.w.model, B, B, fields=("logits",))
        api.rollout_step(it.policy, it.kv, it.B, it.max_len, it.pos, it.tok, it.w.prompt_len + s,
                         1 + s, 1, it.sampling, to, lo, trace=tr, ws=it.ws_roll)
        toks.append(to)
        lps.append(lo)
        logits.append(tr.t["logits"])
    torch.cuda.synchronize()
    return (torch.cat(toks, 1).cpu().numpy(), torch.cat(lps, 1).cpu().numpy(),
            torch.stack(logits, 1).cpu().numpy())


@pytest.fixture(scope="module")
def tiny():
    require_gpu()
    w = get("tiny")
    host, model = build_model(w.model, w.master_seed, gain_noise=0.1)
    return w, host, model


def test_tiny_greedy_end_to_end(tiny):
    w, host, model = tiny
    say("tiny greedy end to end")
    prompts = synth.make_prompts(w)
    it = GrpoIteration(w, model, None, prompts, synth.make_rewards(w), synth.make_seed(w))
    tr0 = api.Trace(w.model, w.n_prompts * w.prompt_len, w.n_prompts, fields=("logits",))
    it.prefill(trace=tr0)
    lg0 = tr0.t["logits"]
    n = w.new_tokens - 1
    toks, lps, logits = _stepwise(it, n)
    tok0 = it.tok0.cpu().numpy()
    gpu_tokens = np.concatenate([tok0[:, None], toks], axis=1)
    gpu_logp = np.concatenate([it.logp0.cpu().numpy()[:, None], lps], axis=1)

    om = oracle.OracleModel(w.model, host)
    ref = om.rollout(prompts, w.group, w.new_tokens, 0.0, 0, synth.make_seed(w),
                     forced=gpu_tokens, keep_logits=True)
    # logits of every step (prefill logits of each prompt appear G times)
    gpu_all = np.concatenate([np.repeat(lg0.cpu().numpy(), w.group, 0)[:, None], logits], axis=1)
    err = np.abs(gpu_all - ref["logits"]).max()
    say("max |dlogit|", err)
    assert err <= TOL
    np.testing.assert_allclose(gpu_logp, ref["logp"], rtol=0, atol=TOL)
    # greedy tokens bit-exact except at logged near-ties
    # (replay of the GPU's history: the oracle's own choice may differ only where
    # its margin is within twice the logit tolerance)
    near = ref["margin"] < 2 * TOL
    mism = (gpu_tokens != ref["own_tokens"]) & ~near
    say("near ties:", int(near.sum()), "mismatches:", int(mism.sum()))
    assert not mism.any()
    # KV cache against the oracle's (same token history)
    kv = kv_view(w.model, it.kv, it.B, it.max_len)
    L = w.model.n_layers
    ctx = w.prompt_len + w.new_tokens - 1
    for l in range(L):
        np.testing.assert_allclose(kv[l, 0, :, :, :ctx], ref["K"][l, :, :, :ctx], rtol=0,
                                   atol=TOL)
        np.testing.assert_allclose(kv[l, 1, :, :, :ctx], ref["V"][l, :, :, :ctx], rtol=0,
                                   atol=TOL)

    # the multi-step call gives the same tokens as the one-step calls
    it.prefill()
    it.decode()
    torch.cuda.synchronize()
    assert np.array_equal(it.tok_dec.cpu().numpy(), toks)
    np.testing.assert_array_equal(it.logp_dec.cpu().numpy(), lps)

    # teacher-forced scoring vs oracle, and vs the rollout's own log-probs
    it.assemble()
    ws = api.alloc_workspace(model, api.OP_SCORE, it.B, it.T)
    lp = torch.empty(it.B, w.new_tokens, device="cuda")
    api.score_sequences(model, it.seqs, w.prompt_len, 0.0, lp, ws=ws)
    torch.cuda.synchronize()
    lp = lp.cpu().numpy()
    seqs = it.seqs.cpu().numpy()
    np.testing.assert_allclose(lp, om.score(seqs, w.prompt_len, 0.0), rtol=0, atol=TOL)
    np.testing.assert_allclose(lp, gpu_logp, rtol=0, atol=TOL)


@pytest.mark.parametrize("temperature,top_k", [(1.0, 0), (0.8, 50), (1.3, 1), (0.7, 2048)])
def test_tiny_sampler_on_gpu_logits(tiny, temperature, top_k):
    w, host, model = tiny
    say("tiny sampler", temperature, top_k)
    w = w.with_(temperature=temperature, top_k=top_k, new_tokens=9)
    prompts = synth.make_prompts(w)
    seed = synth.make_seed(w) ^ 0x5DEECE66D
    it = GrpoIteration(w, model, None, prompts, synth.make_rewards(w), seed)
    it.prefill()
    toks, lps, logits = _stepwise(it, w.new_tokens - 1)
    near_total = 0
    for s in range(toks.shape[1]):
        near_total += sampler_check(logits[:, s], toks[:, s], lps[:, s], temperature, top_k, seed,
                                    1 + s, np.arange(it.B), band=NEAR_TIE)
    say("near ties", near_total)
    # tokens also agree with the oracle's own rollout when margins allow
    om = oracle.OracleModel(w.model, host)
    ref = om.rollout(prompts, w.group, w.new_tokens, temperature, top_k, seed,
                     forced=np.concatenate([it.tok0.cpu().numpy()[:, None], toks], 1))
    ok = ref["margin"][:, 1:] > 2 * TOL / temperature
    assert np.array_equal(toks[ok], ref["own_tokens"][:, 1:][ok])


@pytest.mark.parametrize("temperature,top_k", [(1.0, 0), (0.8, 50), (0.0, 0), (1.2, 1)])
def test_large_vocab_sampler_on_gpu_logits(temperature, top_k):
    """Vocabularies above 32768 ids take the sampler's streaming kernel (the row's
    logits read on every pass instead of held in registers): its tokens and
    log-probs against the oracle sampler on the GPU's own logits, at vocabulary
    40000 (one layer of the tiny widths), for a draw without a cut, a top-k cut,
    greedy and top-1."""
    require_gpu()
    w = get("tiny")
    w = w.with_(model=dataclasses.replace(w.model, vocab=40000, n_layers=1),
                temperature=temperature, top_k=top_k, new_tokens=5)
    say("large-vocabulary sampler", temperature, top_k)
    host, model = build_model(w.model, w.master_seed, gain_noise=0.1)
    seed = synth.make_seed(w) ^ 0x2545F491
    it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w), seed)
    it.prefill()
    toks, lps, logits = _stepwise(it, w.new_tokens - 1)
    assert np.all((toks >= 0) & (toks < w.model.vocab))
    near_total = 0
    for s in range(toks.shape[1]):
        near_total += sampler_check(logits[:, s], toks[:, s], lps[:, s], temperature, top_k, seed,
                                    1 + s, np.arange(it.B), band=NEAR_TIE)
    say("near ties", near_total)
    model.close()


def test_tiny_resume_and_determinism(tiny):
    w, host, model = tiny
    w = w.with_(temperature=1.0, new_tokens=11)
    it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w), 77)
    it.prefill()
    it.decode()
    torch.cuda.synchronize()
    a = it.tok_dec.cpu().numpy().copy()
    # again: bit-identical
    it.prefill()
    it.decode()
    torch.cuda.synchronize()
    assert np.array_equal(a, it.tok_dec.cpu().numpy())
    # 4 steps, then resume for 6 from the carried (tok, pos) state
    it.prefill()
    it.tok.copy_(it.tok0)
    it.pos.fill_(w.prompt_len)
    o1 = torch.empty(it.B, 4, dtype=torch.int32, device="cuda")
    o2 = torch.empty(it.B, 6, dtype=torch.int32, device="cuda")
    l1 = torch.empty(it.B, 4, device="cuda")
    l2 = torch.empty(it.B, 6, device="cuda")
    api.rollout_step(model, it.kv, it.B, it.max_len, it.pos, it.tok, w.prompt_len, 1, 4,
                     it.sampling, o1, l1, ws=it.ws_roll)
    api.rollout_step(model, it.kv, it.B, it.max_len, it.pos, it.tok, w.prompt_len + 4, 5, 6,
                     it.sampling, o2, l2, ws=it.ws_roll)
    torch.cuda.synchronize()
    assert np.array_equal(np.concatenate([o1.cpu().numpy(), o2.cpu().numpy()], 1), a)


def test_graph_replay_matches_eager(tiny, monkeypatch):
    """The captured-and-replayed decode step gives the eager step's bits."""
    w, host, model = tiny
    w = w.with_(temperature=1.0, new_tokens=7)
    it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w), 31)
    outs = []
    for flag in (None, "1", None):
        if flag:
            monkeypatch.setenv("GRPO_NO_GRAPH", flag)
        else:
            monkeypatch.delenv("GRPO_NO_GRAPH", raising=False)
        it.prefill()
        it.decode()
        torch.cuda.synchronize()
        outs.append((it.tok_dec.cpu().numpy().copy(), it.logp_dec.cpu().numpy().copy(),
                     it.pos.cpu().numpy().copy()))
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            np.testing.assert_array_equal(a, b)
    assert np.all(outs[0][2] == w.prompt_len + w.new_tokens - 1)


def test_tiny_stage_local(tiny):
    """Every stage of the prefill and of two decode steps, fed the GPU's own
    inputs, against the oracle within the bounds of fp32 arithmetic (fp32
    models have no rounding points), then the sampler (T1)."""
    w, host, model = tiny
    cfg = w.model
    say("tiny stage-local")
    it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w),
                       synth.make_seed(w))
    P, Tp = w.n_prompts, w.prompt_len
    tr = api.Trace(cfg, P * Tp, P)
    it.prefill(trace=tr)
    torch.cuda.synchronize()
    t = tr.numpy()
    rows = np.arange(P * Tp)
    hrows = np.arange(P)
    rep, worst = check_rows(cfg, host, t, Tp, P * Tp, rows,
                            head=(hrows, hrows * Tp + Tp - 1, P))
    assert_report(rep, "tiny prefill")
    it.tok.copy_(it.tok0)
    for s in range(2):
        pos = np.full(it.B, Tp + s)
        t, toks, lps = decode_traced(model, it.kv, it.B, it.max_len, pos, it.tok, 1 + s,
                                     it.sampling, it.ws_roll)
        kvnp = kv_view(cfg, it.kv, it.B, it.max_len)
        rep, worst = check_decode(cfg, host, model, t, kvnp, pos, it.max_len)
        assert_report(rep, f"tiny decode step {s}")
        sampler_check(t["logits"], toks, lps, w.temperature, w.top_k, it.sampling.seed, 1 + s,
                      np.arange(it.B), band=NEAR_TIE)
