"""Pins of the oracle decoder: brute-force attention, an independent Llama
implementation (HF transformers, fp64 on CPU), cached decode == recompute,
GQA reductions and scoring/rollout consistency."""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import OracleModel
from oracle.model import causal_attention
from paper_2510_17158_amd import synth
from paper_2510_17158_amd.workloads import DTYPE_BF16, DTYPE_F32, ModelConfig

MICRO = ModelConfig(n_layers=2, d_model=32, n_heads=4, n_kv_heads=2, head_dim=8, d_ffn=48,
                    vocab=64, dtype=DTYPE_F32)


def _brute_attention(q, k, v):
    T, H, hd = q.shape
    Hk = k.shape[1]
    o = np.zeros_like(q)
    for i in range(T):
        for h in range(H):
            g = (h * Hk) // H
            sc = [sum(q[i, h, e] * k[j, g, e] for e in range(hd)) / hd ** 0.5 for j in range(i + 1)]
            mx = max(sc)
            ex = [np.exp(s - mx) for s in sc]
            tot = sum(ex)
            for j in range(i + 1):
                for e in range(hd):
                    o[i, h, e] += ex[j] / tot * v[j, g, e]
    return o


@pytest.mark.parametrize("H,Hk", [(4, 4), (4, 2), (6, 3), (4, 1)])
def test_attention_brute_force(H, Hk):
    rng = np.random.default_rng(H * 10 + Hk)
    T, hd = 7, 8
    q, k, v = (rng.standard_normal((T, n, hd)) for n in (H, Hk, Hk))
    np.testing.assert_allclose(causal_attention(q, k, v), _brute_attention(q, k, v), rtol=1e-12,
                               atol=1e-13)


def test_attention_special_cases():
    rng = np.random.default_rng(5)
    T, H, hd = 6, 2, 8
    q = rng.standard_normal((T, H, hd))
    v = rng.standard_normal((T, H, hd))
    k = rng.standard_normal((T, H, hd))
    o = causal_attention(q, k, v)
    np.testing.assert_allclose(o[0], v[0], rtol=1e-14)               # one key: o = v
    k_eq = np.repeat(k[:1], T, axis=0)                                # all keys equal
    o2 = causal_attention(q, k_eq, v)
    for i in range(T):
        np.testing.assert_allclose(o2[i], v[: i + 1].mean(axis=0), rtol=1e-12, atol=1e-14)
    # GQA with the kv heads duplicated equals MHA
    k1, v1 = k[:, :1], v[:, :1]
    np.testing.assert_allclose(causal_attention(q, k1, v1),
                               causal_attention(q, np.repeat(k1, 2, 1), np.repeat(v1, 2, 1)),
                               rtol=1e-14)


def _hf_model(cfg: ModelConfig, w: dict, bf16: bool):
    from transformers import LlamaConfig, LlamaForCausalLM
    hc = LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.d_model, intermediate_size=cfg.d_ffn,
                     num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
                     num_key_value_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                     rms_norm_eps=cfg.rms_eps, rope_theta=cfg.rope_theta,
                     tie_word_embeddings=False, attention_bias=False, mlp_bias=False,
                     max_position_embeddings=4096)
    m = LlamaForCausalLM(hc).to(torch.float64).eval()

    def t(a):
        a = np.asarray(a)
        if bf16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).double()
        return torch.from_numpy(a).double()

    sd = {"model.embed_tokens.weight": t(w["tok_emb"]), "lm_head.weight": t(w["lm_head"]),
          "model.norm.weight": t(w["final_norm"])}
    hf = {"attn_norm": "input_layernorm", "mlp_norm": "post_attention_layernorm",
          "wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
          "wo": "self_attn.o_proj", "w_gate": "mlp.gate_proj", "w_up": "mlp.up_proj",
          "w_down": "mlp.down_proj"}
    for l in range(cfg.n_layers):
        for ours, theirs in hf.items():
            sd[f"model.layers.{l}.{theirs}.weight"] = t(w[f"l{l}.{ours}"])
    missing, unexpected = m.load_state_dict(sd, strict=False)
    assert not unexpected and all("rotary" in k for k in missing)
    return m


@pytest.mark.parametrize("cfg", [MICRO, dataclasses.replace(MICRO, n_kv_heads=4),
                                 dataclasses.replace(MICRO, dtype=DTYPE_BF16, n_kv_heads=1)])
def test_forward_matches_hf_llama(cfg):
    bf16 = cfg.dtype == DTYPE_BF16
    w = synth.make_weights(cfg, 11, gain_noise=0.2, std=0.2)
    om = OracleModel(cfg, w, round_points=False)
    tokens = np.random.default_rng(0).integers(0, cfg.vocab, 40)
    ours, _ = om.forward(tokens)
    with torch.no_grad():
        ref = _hf_model(cfg, w, bf16)(torch.from_numpy(tokens)[None]).logits[0].numpy()
    # HF evaluates the RoPE angles in fp32, hence the 1e-6 band
    np.testing.assert_allclose(ours, ref, rtol=0, atol=2e-6 * np.abs(ref).max())


def test_hf_greedy_generate_matches_oracle_rollout():
    cfg = MICRO
    w = synth.make_weights(cfg, 12, std=0.3)
    om = OracleModel(cfg, w)
    prompt = np.random.default_rng(1).integers(0, cfg.vocab, (1, 9))
    r = om.rollout(prompt, group=1, new_tokens=12, temperature=0.0, top_k=0, seed=0)
    with torch.no_grad():
        g = _hf_model(cfg, w, False).generate(torch.from_numpy(prompt), max_new_tokens=12,
                                              do_sample=False, min_new_tokens=12)
    hf_toks = g[0, 9:].numpy()
    ok = (r["margin"][0] > 1e-6)
    assert np.array_equal(r["tokens"][0][ok], hf_toks[ok])


@pytest.mark.parametrize("dtype", [DTYPE_F32, DTYPE_BF16])
def test_cached_decode_equals_recompute(dtype):
    cfg = dataclasses.replace(MICRO, dtype=dtype)
    w = synth.make_weights(cfg, 13, gain_noise=0.1, std=0.2)
    om = OracleModel(cfg, w, round_points=(dtype == DTYPE_BF16))
    prompts = np.random.default_rng(2).integers(0, cfg.vocab, (2, 5))
    r = om.rollout(prompts, group=2, new_tokens=6, temperature=1.0, top_k=0, seed=99,
                   keep_logits=True)
    for b in range(4):
        seq = np.concatenate([prompts[b // 2], r["tokens"][b]])
        full, _ = om.forward(seq)
        np.testing.assert_allclose(r["logits"][b], full[4:4 + 6], rtol=0, atol=1e-12)


def test_score_equals_rollout_logp_and_softmax_sums():
    cfg = MICRO
    w = synth.make_weights(cfg, 14, std=0.2)
    om = OracleModel(cfg, w)
    prompts = np.random.default_rng(3).integers(0, cfg.vocab, (2, 6))
    r = om.rollout(prompts, group=3, new_tokens=5, temperature=0.7, top_k=5, seed=7)
    seqs = np.concatenate([np.repeat(prompts, 3, axis=0), r["tokens"]], axis=1)
    sc = om.score(seqs, 6, 0.7)
    np.testing.assert_allclose(sc, r["logp"], rtol=0, atol=1e-12)
    assert np.all(sc <= 0)


def test_gqa_duplicated_heads_equal_mha():
    cfg = dataclasses.replace(MICRO, n_kv_heads=2)
    w = synth.make_weights(cfg, 15, std=0.2)
    mha = dataclasses.replace(cfg, n_kv_heads=4)
    w2 = dict(w)
    hd = cfg.head_dim
    for l in range(cfg.n_layers):
        for t in ("wk", "wv"):
            a = w[f"l{l}.{t}"].reshape(2, hd, cfg.d_model)
            w2[f"l{l}.{t}"] = np.repeat(a, 2, axis=0).reshape(4 * hd, cfg.d_model)
    tokens = np.arange(10) * 5 % cfg.vocab
    a, _ = OracleModel(cfg, w).forward(tokens)
    b, _ = OracleModel(mha, w2).forward(tokens)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_layer_truncation_and_hidden_states():
    cfg = MICRO
    w = synth.make_weights(cfg, 16, std=0.2)
    om = OracleModel(cfg, w)
    tokens = np.arange(8)
    logits, _, hidden = om.forward(tokens, return_hidden=True)
    assert len(hidden) == cfg.n_layers + 1
    np.testing.assert_allclose(om.head(hidden[-1]), logits, rtol=0, atol=1e-13)


@pytest.mark.parametrize("dtype", [DTYPE_F32, DTYPE_BF16])
def test_extend_then_decode_equals_full_forward(dtype):
    """A tool-output span appended to a cached sequence, then decode steps after
    it, give the logits and K/V of one full forward over the concatenated
    tokens (fp64, 1e-12): prompt prefill, 3 decode steps, a 7-token injected
    span, 2 more decode steps."""
    cfg = dataclasses.replace(MICRO, dtype=dtype)
    w = synth.make_weights(cfg, 21, gain_noise=0.1, std=0.2)
    om = OracleModel(cfg, w, round_points=(dtype == DTYPE_BF16))
    rng = np.random.default_rng(4)
    prompt = rng.integers(0, cfg.vocab, 6)
    gen1 = rng.integers(0, cfg.vocab, 3)
    span = rng.integers(0, cfg.vocab, 7)
    gen2 = rng.integers(0, cfg.vocab, 2)
    seq = np.concatenate([prompt, gen1, span, gen2])
    full, kv_full = om.forward(seq)
    L, Hk, hd = cfg.n_layers, cfg.n_kv_heads, cfg.head_dim
    Tmax = len(seq)
    K = np.zeros((L, 1, Hk, Tmax, hd))
    V = np.zeros_like(K)
    lg, kvp = om.forward(prompt)
    for l in range(L):
        K[l, 0, :, :6], V[l, 0, :, :6] = kvp[l]
    logits = [lg[-1]]
    pos = 6
    for t in gen1:
        logits.append(om.decode(np.array([t]), np.array([pos]), K, V)[0])
        pos += 1
    # the span: its own rows' logits; the last row's is the next-token logit
    ls = om.extend(span, pos, K[:, 0], V[:, 0])
    np.testing.assert_allclose(ls, full[pos:pos + len(span)], rtol=0, atol=1e-12)
    pos += len(span)
    for t in gen2:
        logits.append(om.decode(np.array([t]), np.array([pos]), K, V)[0])
        pos += 1
    want = np.concatenate([full[5:9], full[len(prompt) + 3 + len(span):]])
    np.testing.assert_allclose(np.stack(logits), want, rtol=0, atol=1e-12)
    for l in range(L):
        np.testing.assert_allclose(K[l, 0], kv_full[l][0], rtol=0, atol=1e-12)
        np.testing.assert_allclose(V[l, 0], kv_full[l][1], rtol=0, atol=1e-12)
