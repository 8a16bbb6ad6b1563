"""GPU parity of tool-output injection (grpo_extend) in a rollout whose row set
changes between calls: all rows decode, half of them pause (a pending tool call)
while the others decode on through seq_ids, then every sequence receives a tool
output at its own position (rows listed in a permuted order), and all decode on
from there.  The extend is checked stage by stage against the oracle on its own
inputs, its next-token draws by the oracle sampler; paused sequences' caches
stay bit-identical; the final logits of every sequence match the oracle's full
forward over that sequence's whole token history (end to end: 1e-4 fp32,
2e-2 bf16 at widths below 2048, 0.1 at the 7B width where bf16 rounding flips
alone approach 2e-2)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2510_17158_amd import api, synth
from paper_2510_17158_amd.runner import GrpoIteration
from paper_2510_17158_amd.workloads import get, truncated

from gpu_util import (NEAR_TIE, assert_report, build_model, check_extend, decode_traced,
                      kv_view, logit_tol, require_gpu, say)
from stagecheck import sampler_check

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,layers", [("tiny", 2), ("small", 2), ("7b", 1)])
def test_tool_injection_round_trip(name, layers):
    require_gpu()
    Tp, Te = 100, 40
    w = truncated(get(name), layers, n_prompts=2, group=4, prompt_len=Tp, new_tokens=12,
                  temperature=1.0, top_k=0)
    cfg = w.model
    say("tool injection", name, layers)
    host, model = build_model(cfg, w.master_seed, gain_noise=0.1)
    prompts = synth.make_prompts(w)
    seed = 4242
    it = GrpoIteration(w, model, None, prompts, synth.make_rewards(w), seed)
    B, V = it.B, cfg.vocab
    max_len = Tp + 5 + Te + 2 + 1
    kv = api.alloc_kv(cfg, B, max_len)
    it.kv, it.max_len = kv, max_len
    it.ws_roll = api.alloc_workspace(model, api.OP_ROLLOUT, B, max_len)
    samp = it.sampling
    it.prefill()
    hist = [list(prompts[b // w.group]) for b in range(B)]   # tokens in the cache
    pending = it.tok0.cpu().numpy().astype(np.int64)          # drawn, not yet cached
    pos = np.full(B, Tp)
    step = np.ones(B, np.int64)                               # next Philox step

    def decode(ids, n):
        ids = np.asarray(ids)
        k = len(ids)
        p_dev = torch.from_numpy(pos[ids].astype(np.int32)).cuda()
        t_dev = torch.from_numpy(pending[ids].astype(np.int32)).cuda()
        to = torch.empty(k, n, dtype=torch.int32, device="cuda")
        lo = torch.empty(k, n, device="cuda")
        assert len(set(step[ids])) == 1
        api.rollout_step(model, kv, B, max_len, p_dev, t_dev, int(pos[ids].max()),
                         int(step[ids][0]), n, samp, to, lo, seq_ids=ids, ws=it.ws_roll)
        torch.cuda.synchronize()
        to = to.cpu().numpy()
        for j, b in enumerate(ids):
            hist[b].append(int(pending[b]))
            hist[b].extend(int(t) for t in to[j, :-1])
            pending[b] = to[j, -1]
            pos[b] += n
            step[b] += n

    decode(np.arange(B), 2)
    kv_before = kv_view(cfg, kv, B, max_len)
    running = np.array([0, 2, 5, 7])
    paused = np.array([1, 3, 4, 6])
    decode(running, 3)
    kv_after = kv_view(cfg, kv, B, max_len)
    np.testing.assert_array_equal(kv_after[:, :, paused], kv_before[:, :, paused])
    # every sequence gets a tool output: its pending token, then Te - 1 injected tokens
    rng = np.random.default_rng(7)
    order = rng.permutation(B)
    span = np.zeros((B, Te), np.int64)
    for j, b in enumerate(order):
        span[j, 0] = pending[b]
        span[j, 1:] = rng.integers(0, V, Te - 1)
    pos0 = pos[order].copy()
    ext_step = 20
    tr = api.Trace(cfg, B * Te, B)
    to = torch.empty(B, dtype=torch.int32, device="cuda")
    lo = torch.empty(B, device="cuda")
    ws_ext = api.alloc_workspace(model, api.OP_EXTEND, B, max_len)
    api.extend(model, kv, B, max_len, pos0, torch.from_numpy(span.astype(np.int32)).cuda(),
               ext_step, samp, to, lo, seq_ids=order, trace=tr, ws=ws_ext)
    torch.cuda.synchronize()
    t = tr.numpy()
    kvnp = kv_view(cfg, kv, B, max_len)
    rows = None
    if cfg.d_model >= 2048:      # the widest model: every sequence's span edges
        rows = np.array([j * Te + r for j in range(B) for r in (0, 1, 2, 31, 32, Te - 2, Te - 1)])
    rep, worst = check_extend(cfg, host, t, kvnp, pos0, Te, order, rows=rows)
    assert_report(rep, f"extend (worst logit err {worst:.2e})")
    to, lo = to.cpu().numpy(), lo.cpu().numpy()
    near = sampler_check(t["logits"], to, lo, w.temperature, w.top_k, seed, ext_step, order,
                         band=NEAR_TIE)
    say("extend draws: near ties", near)
    for j, b in enumerate(order):
        hist[b].extend(int(x) for x in span[j])
        pending[b] = to[j]
        pos[b] += Te
        step[b] = ext_step + 1
    # everyone decodes on from their own positions; the last step traced
    decode(np.arange(B), 1)
    tok_dev = torch.from_numpy(pending.astype(np.int32)).cuda()
    td, _, _ = decode_traced(model, kv, B, max_len, pos.copy(), tok_dev, int(step[0]), samp,
                             it.ws_roll)
    for b in range(B):
        hist[b].append(int(pending[b]))
    om = oracle.OracleModel(cfg, host)
    # End to end, two correctly rounded bf16 forwards part by one-ulp flips at
    # ambiguous rounding points; at the 7B width (logit std ~1.3) those alone
    # reach the stated 2e-2 at the worst of ~10^5 logits (plain decode: 0.019), so
    # there the stated tolerance is enforced stage by stage above and the end-to-end
    # figure checks placement only: a span or cache slot off by one sequence or
    # position moves logits by O(1).
    tol = logit_tol(cfg) if cfg.d_model < 2048 else 0.1
    worst_e2e = 0.0
    for b in range(B):
        full, _ = om.forward(np.array(hist[b]))
        assert len(hist[b]) == pos[b] + 1
        worst_e2e = max(worst_e2e, float(np.abs(full[-1] - td["logits"][b]).max()))
    say("end to end after injection: worst logit err", worst_e2e)
    assert worst_e2e <= tol
    # the extend's own next-token logits against the full forward at the span's end
    worst_ext = 0.0
    for j, b in enumerate(order):
        full, _ = om.forward(np.array(hist[b][:pos0[j] + Te]))
        worst_ext = max(worst_ext, float(np.abs(full[-1] - t["logits"][j]).max()))
    say("extend next-token logits end to end: worst err", worst_ext)
    assert worst_ext <= tol
    model.close()
