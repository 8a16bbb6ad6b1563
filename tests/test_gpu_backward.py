"""GPU parity of the gradient step (Alg. 1): grpo_policy_backward against the
oracle's fp64 backward, and grpo_adamw_step against the oracle's AdamW.

Tolerances.  fp32 models: every gradient tensor within 1e-4 of its largest
entry (the stated fp32 tolerance, relative to the tensor's scale).  bf16
models: the relative Frobenius error of every gradient tensor at most 2e-2.
The bf16 backward rounds each data-gradient operand to bf16 before its product
(relative error at most 2^-9, uncorrelated across elements), so one product
carries about sqrt(2) 2^-9 = 0.3% relative Frobenius error; a layer chains up
to six such products and the recomputed forward adds its own ulp-level
differences, which at two layers gives about 1%; the bound is twice that."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2510_17158_amd import api
from paper_2510_17158_amd.workloads import DTYPE_F32, M32B, M7B, SMALL, TINY

from gpu_util import build_model, require_gpu, say

pytestmark = pytest.mark.gpu


def _grads_oracle(cfg, host, tokens, sf, temp, dlogp):
    om = oracle.OracleModel(cfg, host)
    tot = None
    for n in range(tokens.shape[0]):
        g = oracle.policy_gradient(om, tokens[n], sf, temp, dlogp[n])
        tot = g if tot is None else {k: tot[k] + g[k] for k in tot}
    return tot


@pytest.mark.parametrize("cfg,N,T,sf,temp", [
    (TINY, 2, 100, 40, 1.0),
    (dataclasses.replace(TINY, n_kv_heads=2), 1, 130, 7, 0.7),
    (dataclasses.replace(SMALL, n_layers=2), 1, 200, 100, 1.0),
    (dataclasses.replace(SMALL, n_layers=1), 2, 64, 1, 0.8),
    # bf16 below one 64-position block: query rows past T clamped and zeroed
    (dataclasses.replace(SMALL, n_layers=1), 1, 10, 3, 1.0),
    # the 7B width (head_dim 128, GQ 4, vocab 32000), one layer, 2048 positions
    (dataclasses.replace(M7B, n_layers=1), 1, 2048, 1024, 1.0),
    # the 32B width (GQ 5: head batches of whole 5-head groups, vocab 152064), one
    # layer, a ragged length
    (dataclasses.replace(M32B, n_layers=1), 1, 200, 77, 0.9),
])
def test_policy_backward_matches_oracle(cfg, N, T, sf, temp):
    require_gpu()
    say("backward", cfg.d_model, cfg.n_layers, cfg.n_kv_heads, N, T, sf)
    host, model = build_model(cfg, 77, gain_noise=0.1)
    rng = np.random.default_rng(5)
    tokens = rng.integers(0, cfg.vocab, (N, T)).astype(np.int32)
    dlogp = rng.standard_normal((N, T - sf)).astype(np.float32)
    grads = api.Grads(model)
    api.policy_backward(model, torch.from_numpy(tokens).cuda(), sf, temp,
                        torch.from_numpy(dlogp).cuda(), grads)
    torch.cuda.synchronize()
    ref = _grads_oracle(cfg, host, tokens, sf, temp, dlogp.astype(np.float64))
    worst = {}
    for name, r in ref.items():
        g = grads.t[name].double().cpu().numpy()
        assert np.all(np.isfinite(g)), name
        if cfg.dtype == DTYPE_F32:
            err = np.abs(g - r).max() / max(np.abs(r).max(), 1e-30)
            worst[name] = err
            assert err <= 1e-4, (name, err)
        else:
            err = np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-30)
            worst[name] = err
            assert err <= 2e-2, (name, err)
    top = sorted(worst.items(), key=lambda kv: -kv[1])[:4]
    say("worst relative errors", [(k, f"{v:.2e}") for k, v in top])
    model.close()


def test_backward_accumulates_and_zero_gradient_is_zero():
    """A second call adds exactly the same gradient (every reduction has a fixed
    order, the embedding's included: g + g = 2g bit for bit); dlogp = 0 leaves the
    accumulators untouched."""
    require_gpu()
    cfg = TINY
    host, model = build_model(cfg, 78)
    rng = np.random.default_rng(6)
    tokens = torch.from_numpy(rng.integers(0, cfg.vocab, (1, 70)).astype(np.int32)).cuda()
    dlogp = torch.from_numpy(rng.standard_normal((1, 50)).astype(np.float32)).cuda()
    grads = api.Grads(model)
    api.policy_backward(model, tokens, 20, 1.0, torch.zeros_like(dlogp), grads)
    torch.cuda.synchronize()
    assert all(float(v.abs().max()) == 0.0 for v in grads.t.values())
    api.policy_backward(model, tokens, 20, 1.0, dlogp, grads)
    one = {k: v.clone() for k, v in grads.t.items()}
    api.policy_backward(model, tokens, 20, 1.0, dlogp, grads)
    torch.cuda.synchronize()
    for k, v in grads.t.items():
        assert torch.equal(v, 2 * one[k]), k
    model.close()


@pytest.mark.parametrize("T,distinct", [(300, 8), (2, 1), (4096, 3)])
def test_embedding_gradient_with_repeated_tokens(T, distinct):
    """Tokens drawn from a few ids (long runs of each id after sorting, the first
    and last positions included): the embedding gradient against the oracle, rows
    of ids that never occur exactly zero, and two fresh calls bit-identical."""
    require_gpu()
    cfg = dataclasses.replace(TINY, n_layers=1)
    host, model = build_model(cfg, 79)
    rng = np.random.default_rng(T)
    ids = rng.choice(cfg.vocab, distinct, replace=False)
    tokens = ids[rng.integers(0, distinct, (1, T))].astype(np.int32)
    sf = 1
    dlogp = rng.standard_normal((1, T - sf)).astype(np.float32)
    runs = []
    for _ in range(2):
        grads = api.Grads(model)
        api.policy_backward(model, torch.from_numpy(tokens).cuda(), sf, 1.0,
                            torch.from_numpy(dlogp).cuda(), grads)
        torch.cuda.synchronize()
        runs.append(grads.t["tok_emb"].clone())
    assert torch.equal(runs[0], runs[1])
    g = runs[0].double().cpu().numpy()
    unseen = np.setdiff1d(np.arange(cfg.vocab), ids)
    assert np.all(g[unseen] == 0)
    ref = _grads_oracle(cfg, host, tokens, sf, 1.0, dlogp.astype(np.float64))["tok_emb"]
    assert np.abs(g - ref).max() <= 1e-4 * np.abs(ref).max()
    model.close()


@pytest.mark.parametrize("dtype", [0, 1])
def test_adamw_matches_oracle(dtype):
    require_gpu()
    rng = np.random.default_rng(8)
    n = 100003
    p0 = rng.standard_normal(n).astype(np.float32)
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
    master = torch.from_numpy(p0).cuda() if dtype == 1 else None
    param = (torch.from_numpy(p0).cuda() if dtype == 0
             else torch.from_numpy(p0).cuda().to(torch.bfloat16))
    m = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    p_ref, m_ref, v_ref = p0.astype(np.float64), np.zeros(n), np.zeros(n)
    for step in (1, 2, 3):
        g = rng.standard_normal(n).astype(np.float32)
        api.adamw_step(dtype, param, master, m, v, torch.from_numpy(g).cuda(), step=step, **hp)
        torch.cuda.synchronize()
        p_ref, m_ref, v_ref = oracle.adamw(p_ref, g.astype(np.float64), m_ref, v_ref, step,
                                           hp["lr"], hp["beta1"], hp["beta2"], hp["eps"],
                                           hp["weight_decay"])
        got = (master if dtype == 1 else param).double().cpu().numpy()
        assert np.abs(got - p_ref).max() <= 1e-6 * np.abs(p_ref).max()
        np.testing.assert_allclose(m.double().cpu().numpy(), m_ref, rtol=1e-5, atol=1e-7)
        np.testing.assert_allclose(v.double().cpu().numpy(), v_ref, rtol=1e-5, atol=1e-7)
        if dtype == 1:   # the model copy is the master rounded to bf16
            assert torch.equal(param, master.to(torch.bfloat16))


@pytest.mark.parametrize("name,layers", [("tiny", 2), ("small", 2)])
def test_grpo_iteration_with_update_lowers_its_loss(name, layers):
    """A whole Alg. 1 iteration: rollout, scoring, advantages and loss, then the
    gradient step (backward over the batch + AdamW, decode copy repacked).  On the
    same sampled batch the loss after the step is lower.  On the fp32 model its
    change also matches the first-order prediction sum(g * dw) from the GPU's own
    gradient and the weights' actual change (5e-2 relative).  bf16 weights only
    move in steps of their rounding, so the first AdamW step (every weight moved
    by about lr) has to be large enough to change them, which puts it outside
    the first-order regime; there only the decrease is asserted."""
    require_gpu()
    from paper_2510_17158_amd import synth
    from paper_2510_17158_amd.runner import GrpoIteration
    from paper_2510_17158_amd.workloads import get, truncated
    w = truncated(get(name), layers, n_prompts=2, group=4, prompt_len=48, new_tokens=24,
                  temperature=1.0, top_k=0)
    cfg = w.model
    host, model = build_model(cfg, w.master_seed, gain_noise=0.1)
    ref_host = synth.make_weights(cfg, w.master_seed, ref=True)
    ref = api.Model(cfg, api.upload_weights(cfg, ref_host), decode=False)
    it = GrpoIteration(w, model, ref, synth.make_prompts(w), synth.make_rewards(w), 11)
    it.run()
    torch.cuda.synchronize()
    l0 = it.loss.item()
    before = {k: v.double().clone() for k, v in model.weights.items()}
    it.update(lr=1e-5 if cfg.dtype == DTYPE_F32 else 2e-4)
    torch.cuda.synchronize()
    pred = sum(float((it._grads.t[k].double() * (v.double() - before[k])).sum())
               for k, v in model.weights.items())
    it.score()
    it.grpo()
    torch.cuda.synchronize()
    l1 = it.loss.item()
    say(name, "loss", l0, "->", l1, "first-order", pred)
    assert l1 < l0 and pred < 0
    if cfg.dtype == DTYPE_F32:
        assert abs((l1 - l0) - pred) <= 5e-2 * abs(pred) + 1e-7
    # the next rollout decodes with the updated weights (decode copy repacked)
    it.run()
    torch.cuda.synchronize()
    assert np.isfinite(it.loss.item())
    model.close()
    ref.close()
