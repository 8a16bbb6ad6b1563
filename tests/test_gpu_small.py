"""GPU parity on bf16 decoders: stage-local (every decode layer fed the GPU's
own residual and KV cache), the LM head + sampler on the GPU's final state, and
end to end at the small shape (12 layers, d 768, GQA 12/4) where the bf16
logit tolerance 2e-2 holds literally.

Prompt length 300 spans three 128-row GEMM tiles, five 64-row attention blocks
and three 128-position decode spans (8 sequences x 4 kv heads is too few pairs
for a single span), each with a ragged tail."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2510_17158_amd import api, synth
from paper_2510_17158_amd.runner import GrpoIteration
from paper_2510_17158_amd.workloads import get, truncated

from gpu_util import (FloorPool, bf16_ulps, build_model, floor_check, h_flip_allowance,
                      kv_view, require_gpu, say)

pytestmark = pytest.mark.gpu

LOGIT_TOL = 2e-2     # bf16 logits / log-probs
# Per-layer outputs (residual stream, K/V) are judged against the noise floor of
# the rounding contract: the distance between the fp32-arithmetic and the fp64
# evaluation of the same layer on the same (GPU-produced) inputs.


def _small_workload(**kw):
    w = get("small").with_(n_prompts=2, group=4, prompt_len=300, new_tokens=6, temperature=1.0)
    return w.with_(**kw)


def _stage_local(w, host, model, it, n_steps, group=0, prefix_len=0, back=None):
    """Decode n_steps one at a time; check every layer, the head and the sampler
    (group > 0: grouped steps sharing the cache below prefix_len; back: per-row
    steps back from the prompt's end, so the rows decode at ragged positions)."""
    cfg = w.model
    B, L, d, V = it.B, cfg.n_layers, cfg.d_model, cfg.vocab
    om = oracle.OracleModel(cfg, host)
    om32 = oracle.OracleModel(cfg, host, precision="fp32")
    om32s = oracle.OracleModel(cfg, host, precision="fp32-seq")
    it.tok.copy_(it.tok0)
    back = np.zeros(B, np.int64) if back is None else np.asarray(back, np.int64)
    it.pos.copy_(torch.from_numpy((w.prompt_len - back).astype(np.int32)).to("cuda"))
    pool = FloorPool()
    worst_logit, near = 0.0, 0
    toks = []
    for s in range(n_steps):
        pos = w.prompt_len + s
        posv = pos - back
        to = torch.empty(B, 1, dtype=torch.int32, device="cuda")
        lo = torch.empty(B, 1, device="cuda")
        lg = torch.empty(B, V, device="cuda")
        hid = torch.empty(L + 1, B, d, device="cuda")
        api.rollout_step(model, it.kv, B, it.max_len, it.pos, it.tok, pos, 1 + s, 1, it.sampling,
                         to, lo, logits_dbg=lg, hidden_dbg=hid, ws=it.ws_roll, group=group,
                         prefix_len=prefix_len)
        torch.cuda.synchronize()
        hid = hid.double().cpu().numpy()
        lg = lg.cpu().numpy()
        to = to.cpu().numpy()[:, 0]
        lo = lo.cpu().numpy()[:, 0]
        toks.append(to)
        kv = kv_view(cfg, it.kv, B, it.max_len)
        rows = np.arange(B)
        for l in range(L):
            x64, k64, v64 = om.decode_layer(l, hid[l], posv, kv[l, 0].copy(), kv[l, 1].copy())
            f32 = [m.decode_layer(l, hid[l], posv, kv[l, 0].astype(np.float32),
                                  kv[l, 1].astype(np.float32)) for m in (om32, om32s)]
            ak, av = h_flip_allowance(om, cfg, l, hid[l])
            pool.add("x", hid[l + 1], x64, [r[0] for r in f32])
            pool.add("k", kv[l, 0, rows, :, posv], k64, [r[1] for r in f32], bf16=True, allow=ak)
            pool.add("v", kv[l, 1, rows, :, posv], v64, [r[2] for r in f32], bf16=True, allow=av)
        worst_logit = max(worst_logit, float(np.abs(om.head(hid[L]) - lg).max()))
        for b in range(B):
            t, lp, margin = oracle.sample_token(lg[b].astype(np.float64), w.temperature, w.top_k,
                                                it.sampling.seed, 1 + s, b)
            if margin < 1e-4:
                near += 1
                continue
            assert to[b] == t, (s, b)
            assert abs(lo[b] - lp) <= 1e-5
    ok, stats = pool.check()
    say("decode stage-local:", stats, "head logit err", worst_logit, "near ties", near)
    assert ok
    assert worst_logit <= LOGIT_TOL
    return np.stack(toks, 1)


def _prefill_stage_local(w, host, model, it):
    """Prefill with every layer fed the GPU's own residual stream."""
    cfg = w.model
    L, d, P, Tp = cfg.n_layers, cfg.d_model, w.n_prompts, w.prompt_len
    lg0 = torch.empty(P, cfg.vocab, device="cuda")
    hid = torch.empty(L + 1, P * Tp, d, device="cuda")
    it.prefill(logits_dbg=lg0, hidden_dbg=hid)
    torch.cuda.synchronize()
    hid = hid.double().cpu().numpy().reshape(L + 1, P, Tp, d)
    kv = kv_view(cfg, it.kv, it.B, it.max_len)
    lg0 = lg0.cpu().numpy()
    om = oracle.OracleModel(cfg, host)
    om32 = oracle.OracleModel(cfg, host, precision="fp32")
    om32s = oracle.OracleModel(cfg, host, precision="fp32-seq")
    prompts = synth.make_prompts(w)
    pool = FloorPool()
    worst_logit, e2e = 0.0, 0.0
    for p in range(P):
        for l in range(L):
            x64, k64, v64 = om.layer(l, hid[l, p])
            f32 = [m.layer(l, hid[l, p]) for m in (om32, om32s)]
            ak, av = h_flip_allowance(om, cfg, l, hid[l, p])      # [Tp, n_kv, hd]
            pool.add("x", hid[l + 1, p], x64, [r[0] for r in f32])
            pool.add("k", kv[l, 0, p * w.group, :, :Tp], k64, [r[1] for r in f32], bf16=True,
                     allow=ak.transpose(1, 0, 2))
            pool.add("v", kv[l, 1, p * w.group, :, :Tp], v64, [r[2] for r in f32], bf16=True,
                     allow=av.transpose(1, 0, 2))
        worst_logit = max(worst_logit, float(np.abs(om.head(hid[L, p, -1:])[0] - lg0[p]).max()))
        e2e = max(e2e, float(np.abs(om.forward(prompts[p])[0][-1] - lg0[p]).max()))
    ok, stats = pool.check()
    say("prefill stage-local:", stats, "head logit err", worst_logit,
        "end-to-end logit err (reported)", e2e)
    assert ok
    assert worst_logit <= LOGIT_TOL


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
        g, r = kv[0, 0, p * w.group, :, : w.prompt_len], kvp[0][0]
        r32 = [oracle.OracleModel(w.model, host, precision=pr).forward(prompts[p])[1][0][0]
               for pr in ("fp32", "fp32-seq")]
        u = bf16_ulps(g, r)
        ok, st = floor_check(g, r, r32, bf16=True)
        say("layer-0 K ulps max", int(u.max()), "flip frac", float((u > 0).mean()), st)
        assert ok
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
    _prefill_stage_local(w, host, model, it)
    _stage_local(w, host, model, it, 3)


@pytest.mark.parametrize("name,layers,kw", [
    ("1b", 2, dict(n_prompts=2, group=4, prompt_len=70, new_tokens=4, temperature=0.8,
                   top_k=50)),
    ("7b", 1, dict(n_prompts=1, group=8, prompt_len=120, new_tokens=5)),
    ("32b", 1, dict(n_prompts=1, group=8, prompt_len=96, new_tokens=5)),
    # >= 1024 prompt rows: the 256 x 256 GEMM tiles, last row tile shifted back.
    # 8 sequences x 2 decode steps: the decode floor check pools per-row rounding
    # flip cascades, which a 4-row pool is too small to compare with the floor's
    ("small", 2, dict(n_prompts=4, group=2, prompt_len=300, new_tokens=3)),
    ("7b", 1, dict(n_prompts=2, group=4, prompt_len=520, new_tokens=3)),
])
def test_full_width_stage_local(name, layers, kw):
    """Layer-truncated models at the 1B/7B/32B widths: every stage fed GPU inputs."""
    require_gpu()
    say("full width stage-local", name, layers)
    w = truncated(get(name), layers, **kw)
    host, model = build_model(w.model, w.master_seed, gain_noise=0.1)
    it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w),
                       synth.make_seed(w))
    _prefill_stage_local(w, host, model, it)
    _stage_local(w, host, model, it, w.new_tokens - 1)
    model.close()



def test_small_graph_replay_matches_eager(small, monkeypatch):
    w, host, model = small
    it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w),
                       synth.make_seed(w))
    outs = []
    for flag in (None, "1"):
        if flag:
            monkeypatch.setenv("GRPO_NO_GRAPH", flag)
        else:
            monkeypatch.delenv("GRPO_NO_GRAPH", raising=False)
        it.prefill()
        it.decode()
        torch.cuda.synchronize()
        outs.append((it.tok_dec.cpu().numpy().copy(), it.logp_dec.cpu().numpy().copy()))
    np.testing.assert_array_equal(outs[0][0], outs[1][0])
    np.testing.assert_array_equal(outs[0][1], outs[1][1])


def test_profile_counts_launches(small):
    w, host, model = small
    it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w),
                       synth.make_seed(w))
    api.profile_begin()
    it.prefill()
    it.decode()
    torch.cuda.synchronize()
    prof = api.profile_end()
    say("profile", prof)
    L, n = w.model.n_layers, w.new_tokens - 1
    assert prof["attn_decode"][0] == L * n
    assert prof["gemm_decode_swiglu"][0] == L * n
    assert all(t >= 0 for _, t in prof.values())


def test_decode_span_count_does_not_change_results(small):
    """A KV capacity far above the context gives more decode spans, several of
    them empty; the logits agree with the tight-capacity run up to the order of
    the fp32 merge."""
    w, host, model = small
    w = w.with_(new_tokens=2)          # one decode step after the prefill draw
    cfg = w.model
    outs = []
    for cap in (None, 2000):
        it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w), 11)
        max_len = it.max_len
        if cap:
            max_len = cap
            it.kv = api.alloc_kv(cfg, it.B, cap)
            it.ws_roll = api.alloc_workspace(model, api.OP_ROLLOUT, it.B, cap)
            it.max_len = cap
        say("span check, kv capacity", max_len)
        it.prefill()
        lg = torch.empty(it.B, cfg.vocab, device="cuda")
        it.decode(logits_dbg=lg)
        torch.cuda.synchronize()
        outs.append((lg.cpu().numpy(), it.tok_dec.cpu().numpy()))
    err = np.abs(outs[0][0] - outs[1][0]).max()
    say("max |dlogit| between capacities", err)
    assert err <= 1e-3


def test_bench_launch_configuration():
    """The 7B workload's own launch configuration on a 1-layer model of the 7B
    width: 8 prompts x G 8 = 64 sequences, 2048-token prompts, 2048 sampled tokens
    (temperature 1), scoring over 4096 positions.  One grouped decode step at
    context 2049 is checked stage-locally against the oracle (the decode GEMM plans
    at batch 64, the prompt attention once per group in 8 chunks, the generated
    positions per sequence and their merge, the LM head and the sampler over 32000
    logits); then the whole rollout runs (grouped, as the workload does), and teacher-forced
    scoring of its sequences (flash attention over 4096 positions, the 256 x 256
    GEMM tiles over chunks of 16 x 4096 rows) must reproduce every rollout log-prob:
    both are log_softmax(logits / T) at the sampled token (Eq. (1)), computed by
    different kernels."""
    require_gpu()
    w = truncated(get("7b"), 1)
    assert (w.n_prompts * w.group, w.prompt_len, w.new_tokens) == (64, 2048, 2048)
    say("bench launch configuration, 1 layer of the 7B width")
    host, model = build_model(w.model, w.master_seed, gain_noise=0.1)
    it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w),
                       synth.make_seed(w))
    assert w.shared_prompt
    it.prefill()
    _stage_local(w, host, model, it, 1, group=w.group, prefix_len=w.prompt_len)
    say("full rollout and scoring")
    it.decode()
    it.assemble()
    it.score()
    torch.cuda.synchronize()
    old = it.logp_old.cpu().numpy()
    new = it.lp_pol.cpu().numpy()
    assert np.isfinite(old).all() and np.isfinite(new).all()
    err = float(np.abs(new - old).max())
    say("rollout vs scoring log-prob err", err, "mean logp", float(old.mean()))
    assert err <= LOGIT_TOL
    model.close()


@pytest.mark.parametrize("name,P,G,Tp,prefix,steps", [
    ("small", 2, 4, 300, 300, 3),      # GQ 3: two samples (6 of 8 columns) per wave
    ("small", 2, 4, 300, 100, 2),      # only part of the prompt shared
    ("small", 1, 3, 33, 33, 2),        # G not a multiple of the samples per wave
    ("7b", 2, 16, 70, 70, 2),          # GQ 4, G 16: two prefix workgroups per group
    ("7b", 4, 8, 520, 520, 2),         # several prompt chunks, ragged last tile
])
def test_grouped_decode_matches_per_row(name, P, G, Tp, prefix, steps):
    """Grouped decode (each group's prompt K/V read once) against per-row decode,
    step by step from the same state (both write the same K/V: same token, same
    projections): logits within the bf16 tolerance (the prompt part takes P as
    bf16 hi + lo on MFMA, the per-row part fp32 P on the vector units; the
    difference flips bf16 roundings of the attention output, which cascade like
    the noise floor of the stage-local checks), log-probs likewise, identical
    tokens except where the per-row winner's margin is within twice the row's
    logit change."""
    require_gpu()
    base = get(name)
    layers = 2 if name == "small" else 1
    w = truncated(base, layers, n_prompts=P, group=G, prompt_len=Tp, new_tokens=steps + 1,
                  temperature=1.0, top_k=0)
    say("grouped vs per-row decode", name, P, G, Tp, prefix)
    host, model = build_model(w.model, w.master_seed, gain_noise=0.1)
    it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w),
                       synth.make_seed(w))
    it.prefill()
    B, V = it.B, w.model.vocab
    it.tok.copy_(it.tok0)
    it.pos.fill_(Tp)
    worst, near = 0.0, 0
    for s in range(steps):
        tok_in, pos_in = it.tok.clone(), it.pos.clone()
        res = []
        for grouped in (False, True):
            it.tok.copy_(tok_in)
            it.pos.copy_(pos_in)
            to = torch.empty(B, 1, dtype=torch.int32, device="cuda")
            lo = torch.empty(B, 1, device="cuda")
            lg = torch.empty(B, V, device="cuda")
            api.rollout_step(model, it.kv, B, it.max_len, it.pos, it.tok, Tp + s, 1 + s, 1,
                             it.sampling, to, lo, logits_dbg=lg, ws=it.ws_roll,
                             group=G if grouped else 0, prefix_len=prefix if grouped else 0)
            torch.cuda.synchronize()
            res.append((to.cpu().numpy()[:, 0], lo.cpu().numpy()[:, 0], lg.cpu().numpy()))
        (t0, l0, g0), (t1, l1, g1) = res
        worst = max(worst, float(np.abs(g1 - g0).max()))
        assert np.abs(g1 - g0).max() <= LOGIT_TOL
        for b in np.flatnonzero(t0 != t1):
            # both draws use the same Gumbel noise, so the token can change only if
            # the per-row winner's margin is below twice the row's logit change / T
            _, _, margin = oracle.sample_token(g0[b].astype(np.float64), w.temperature, w.top_k,
                                               it.sampling.seed, 1 + s, b)
            delta = float(np.abs(g1[b].astype(np.float64) - g0[b]).max())
            assert margin <= 2 * delta / w.temperature + 1e-6, (s, b, margin, delta)
            near += 1
        keep = t0 == t1
        assert np.abs(l1 - l0)[keep].max() <= LOGIT_TOL
        it.tok.copy_(torch.from_numpy(t0).to("cuda"))   # both continue from the per-row token
    say("grouped vs per-row: logit err", worst, "tokens changed within the margin bound", near)
    model.close()


@pytest.mark.parametrize("name,P,G,Tp,Tn,prefix", [
    ("small", 2, 4, 300, 100, 300),    # GQ 3; own rows from position 288
    ("small", 2, 4, 300, 100, 200),    # part of the prompt shared (prefix below score_from)
    ("7b", 2, 8, 70, 60, 70),          # GQ 4; own rows from 64
    ("7b", 1, 8, 520, 40, 520),        # several 64-key tiles shared
])
def test_grouped_scoring_matches_per_row(name, P, G, Tp, Tn, prefix):
    """Teacher-forced scoring with each group's shared prompt run once against
    per-row scoring of the same sequences: under causal attention the shared
    positions' states are the same for every member, so the log-probs agree up
    to the order of additions (bf16 tolerance; bf16 roundings may flip)."""
    require_gpu()
    base = get(name)
    layers = 2 if name == "small" else 1
    w = truncated(base, layers, n_prompts=P, group=G, prompt_len=Tp, new_tokens=Tn)
    say("grouped vs per-row scoring", name, P, G, Tp, Tn, prefix)
    host, model = build_model(w.model, w.master_seed, gain_noise=0.1)
    V = w.model.vocab
    rng = np.random.default_rng(P * 1000 + Tp)
    prompts = rng.integers(0, V, (P, Tp))
    gen = rng.integers(0, V, (P * G, Tn))
    seqs = np.concatenate([np.repeat(prompts, G, 0), gen], 1).astype(np.int32)
    tok = torch.from_numpy(seqs).to("cuda")
    N, T = seqs.shape
    ws = api.alloc_workspace(model, api.OP_SCORE, N, T, "cuda")
    out = []
    for group in (0, G):
        lp = torch.empty(N, Tn, device="cuda")
        api.score_sequences(model, tok, Tp, 1.0, lp, ws=ws, group=group, prefix_len=prefix)
        torch.cuda.synchronize()
        out.append(lp.cpu().numpy())
    assert np.isfinite(out[1]).all()
    err = float(np.abs(out[1] - out[0]).max())
    say("grouped vs per-row scoring: log-prob err", err)
    assert err <= LOGIT_TOL
    model.close()


@pytest.mark.parametrize("group", [0, 4])
def test_ragged_positions_stage_local(small, group):
    """One batch whose rows decode at different positions (1 .. 9 steps back from
    the prompt's end, re-entering the prompt: each row attends its own context
    0 .. pos[b]), stage-local against the oracle; grouped with the shared length
    below every row's position."""
    require_gpu()
    w, host, model = small
    say("ragged positions stage-local, group", group)
    it = GrpoIteration(w, model, None, synth.make_prompts(w), synth.make_rewards(w),
                       synth.make_seed(w))
    it.prefill()
    back = 1 + (np.arange(it.B) * 5) % 9
    prefix = w.prompt_len - int(back.max()) if group else 0
    _stage_local(w, host, model, it, 2, group=group, prefix_len=prefix, back=back)
