"""GPU parity of the projection GEMMs with inputs that the norm passes through
exactly: rms_eps = 0, unit gains and embedding rows of +-2^-4, so the normed
activation is exactly +-1 in bf16 and the K/V cache must equal
bf16(rope(h W^T)) of the fp64 oracle to half an ulp plus the fp32 accumulation
error.  Covers the decode GEMM (batch 5, 8, 64, 100 -> all four batch paddings)
and the prefill GEMM, at the small and 7B widths."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from oracle.numerics import rope
from paper_2510_17158_amd import api, synth
from paper_2510_17158_amd.runner import GrpoIteration
from paper_2510_17158_amd.workloads import get, truncated

from gpu_util import kv_view, require_gpu, say

pytestmark = pytest.mark.gpu


def _ulp_bf16(r):
    a = np.abs(np.asarray(r, np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return 2.0 ** (e - 7)


@pytest.mark.parametrize("name,B,Tp", [("small", 8, 130), ("small", 64, 20), ("small", 5, 33),
                                       ("small", 100, 9), ("7b", 64, 12), ("7b", 16, 70),
                                       ("7b", 16, 8), ("7b", 100, 1), ("32b", 8, 5)])
def test_kv_projection_exact_inputs(name, B, Tp):
    require_gpu()
    base = get(name)
    cfg = dataclasses.replace(base.model, n_layers=1, rms_eps=0.0)
    w = dataclasses.replace(truncated(base, 1), model=cfg, n_prompts=B, group=1, prompt_len=Tp,
                            new_tokens=2, temperature=0.0, top_k=0)
    say("exact-input KV", name, B, Tp)
    host = synth.make_weights(cfg, 99 + B)
    rng = np.random.default_rng(B * 1000 + Tp)
    signs = rng.integers(0, 2, (cfg.vocab, cfg.d_model)) * 2 - 1
    emb = (signs * 2.0 ** -4).astype(np.float32)
    host["tok_emb"] = torch.from_numpy(emb).to(torch.bfloat16).view(torch.int16).numpy().view(
        np.uint16)
    dev = api.upload_weights(cfg, host)
    model = api.Model(cfg, dev)
    prompts = rng.integers(0, cfg.vocab, (B, Tp)).astype(np.int32)
    it = GrpoIteration(w, model, None, prompts, np.zeros(B, np.float32), 5)
    it.prefill()
    it.decode()
    it.assemble()
    torch.cuda.synchronize()
    seqs = it.seqs.cpu().numpy()
    kv = kv_view(cfg, it.kv, B, it.max_len)
    Wk = oracle.bf16_bits_to_f64(host["l0.wk"])
    Wv = oracle.bf16_bits_to_f64(host["l0.wv"])
    hd, Hk = cfg.head_dim, cfg.n_kv_heads
    worst = {}
    for label, lo, hi in (("prefill", 0, Tp), ("decode", Tp, Tp + 1)):
        toks = seqs[:, lo:hi]
        h = signs[toks].astype(np.float64)                     # exactly +-1
        k = (h @ Wk.T).reshape(B, hi - lo, Hk, hd)
        v = (h @ Wv.T).reshape(B, hi - lo, Hk, hd)
        pos = np.arange(lo, hi)
        k = np.stack([rope(k[b], pos, cfg.rope_theta) for b in range(B)])
        sum_abs_k = (np.abs(h)[..., None, :] @ np.abs(Wk.T)).reshape(B, hi - lo, Hk, hd)
        gk = kv[0, 0, :, :, lo:hi].transpose(0, 2, 1, 3)
        gv = kv[0, 1, :, :, lo:hi].transpose(0, 2, 1, 3)
        for nm, g, r in (("k", gk, k), ("v", gv, v)):
            err = np.abs(g - r)
            bound = 0.5 * _ulp_bf16(r) * (1 + 2 ** -7) + 1e-6 * sum_abs_k
            frac = err / _ulp_bf16(r)
            worst[f"{label}_{nm}_max_ulp_frac"] = float(frac.max())
            nbad = int((err > bound).sum())
            worst[f"{label}_{nm}_bad"] = nbad
            if nbad:
                idx = np.argwhere(err > bound)[:3]
                say(label, nm, "bad at", idx.tolist(), "gpu", g[tuple(idx[0])], "ref",
                    r[tuple(idx[0])])
    say(worst)
    assert all(v == 0 for k_, v in worst.items() if k_.endswith("_bad"))
    model.close()


@pytest.mark.parametrize("name,B", [("7b", 100), ("7b", 300), ("small", 64)])
def test_rmsnorm_output_through_selection_projection(name, B):
    """W_k and W_v select coordinates of the normed activation h, so the K/V cache
    at position 0 (where RoPE is the identity) holds the GPU's h itself: it must be
    the bf16 rounding of the oracle's h except where the fp64 value lies within
    fp32 error of a rounding midpoint."""
    require_gpu()
    base = get(name)
    cfg = dataclasses.replace(base.model, n_layers=1)
    w = dataclasses.replace(truncated(base, 1), model=cfg, n_prompts=B, group=1, prompt_len=1,
                            new_tokens=2, temperature=0.0, top_k=0)
    say("norm through selection", name, B)
    host = synth.make_weights(cfg, 7 + B, gain_noise=0.1)
    kvd, d = cfg.kv_dim, cfg.d_model
    one = np.uint16(0x3F80)
    for t, off in (("wk", 0), ("wv", kvd)):
        m = np.zeros((kvd, d), np.uint16)
        m[np.arange(kvd), off + np.arange(kvd)] = one
        host[f"l0.{t}"] = m
    dev = api.upload_weights(cfg, host)
    model = api.Model(cfg, dev)
    prompts = np.random.default_rng(B).integers(0, cfg.vocab, (B, 1)).astype(np.int32)
    it = GrpoIteration(w, model, None, prompts, np.zeros(B, np.float32), 5)
    it.prefill()
    torch.cuda.synchronize()
    kv = kv_view(cfg, it.kv, B, it.max_len)
    got = np.concatenate([kv[0, 0, :, :, 0].reshape(B, kvd), kv[0, 1, :, :, 0].reshape(B, kvd)], 1)
    om = oracle.OracleModel(cfg, host, round_points=False)
    h64 = oracle.rmsnorm(om.embed(prompts[:, 0]), om.mat("l0.attn_norm"), cfg.rms_eps)[:, :2 * kvd]
    ref = oracle.round_bf16(h64)
    diff = got != ref
    # distance of the fp64 value from the nearest rounding midpoint, in ulps
    ulp = _ulp_bf16(ref)
    mid_dist = np.abs(np.abs(h64 - ref) - 0.5 * ulp) / ulp
    say("h flips", int(diff.sum()), "of", diff.size, "closest midpoint of a flip",
        float(mid_dist[diff].max()) if diff.any() else None)
    assert not np.any(diff & (mid_dist > 1e-3))
    model.close()
