"""Pins of the oracle backward and optimizer: torch autograd through HF Llama in
fp64 (fp32-weight models, no rounding points), autograd through a torch forward
with straight-through bf16 rounding points, central finite differences of the
oracle's own scoring, torch.optim.AdamW, and the degenerate cases."""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import OracleModel
from oracle.backward import adamw, policy_gradient
from paper_2510_17158_amd import synth
from paper_2510_17158_amd.workloads import DTYPE_BF16, DTYPE_F32, ModelConfig

MICRO = ModelConfig(n_layers=2, d_model=32, n_heads=4, n_kv_heads=2, head_dim=8, d_ffn=48,
                    vocab=64, dtype=DTYPE_F32)
HF_NAMES = {"attn_norm": "input_layernorm", "mlp_norm": "post_attention_layernorm",
            "wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
            "wo": "self_attn.o_proj", "w_gate": "mlp.gate_proj", "w_up": "mlp.up_proj",
            "w_down": "mlp.down_proj"}


def _case(cfg, seed, T=12, score_from=5):
    w = synth.make_weights(cfg, seed, gain_noise=0.2, std=0.2)
    rng = np.random.default_rng(seed)
    tokens = rng.integers(0, cfg.vocab, T)
    dlogp = rng.standard_normal(T - score_from)
    return w, tokens, dlogp


def _hf(cfg, w):
    from transformers import LlamaConfig, LlamaForCausalLM
    hc = LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.d_model, intermediate_size=cfg.d_ffn,
                     num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
                     num_key_value_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                     rms_norm_eps=cfg.rms_eps, rope_theta=cfg.rope_theta,
                     tie_word_embeddings=False, attention_bias=False, mlp_bias=False,
                     max_position_embeddings=4096, attn_implementation="eager")
    m = LlamaForCausalLM(hc).to(torch.float64)
    sd = {"model.embed_tokens.weight": w["tok_emb"], "lm_head.weight": w["lm_head"],
          "model.norm.weight": w["final_norm"]}
    for l in range(cfg.n_layers):
        for ours, theirs in HF_NAMES.items():
            sd[f"model.layers.{l}.{theirs}.weight"] = w[f"l{l}.{ours}"]
    sd = {k: torch.from_numpy(np.asarray(v, np.float64)) for k, v in sd.items()}
    missing, unexpected = m.load_state_dict(sd, strict=False)
    assert not unexpected and all("rotary" in k for k in missing)
    return m


@pytest.mark.parametrize("cfg,temp", [(MICRO, 1.0), (dataclasses.replace(MICRO, n_kv_heads=1), 0.7),
                                      (dataclasses.replace(MICRO, n_kv_heads=4), 1.3)])
def test_gradient_matches_hf_llama_autograd(cfg, temp):
    """Every weight's gradient of sum_j g_j logp_j equals torch autograd through
    HF's Llama (fp64 on the CPU; HF takes the RoPE angles in fp32, hence 1e-6)."""
    w, tokens, dlogp = _case(cfg, 31)
    sf = 5
    ours = policy_gradient(OracleModel(cfg, w), tokens, sf, temp, dlogp)
    m = _hf(cfg, w)
    logits = m(torch.from_numpy(tokens)[None]).logits[0]
    ls = torch.log_softmax(logits[sf - 1:-1] / temp, dim=-1)
    lp = ls[torch.arange(len(tokens) - sf), torch.from_numpy(tokens[sf:])]
    (lp * torch.from_numpy(dlogp)).sum().backward()
    params = dict(m.named_parameters())
    ref = {"tok_emb": params["model.embed_tokens.weight"], "lm_head": params["lm_head.weight"],
           "final_norm": params["model.norm.weight"]}
    for l in range(cfg.n_layers):
        for o, t in HF_NAMES.items():
            ref[f"l{l}.{o}"] = params[f"model.layers.{l}.{t}.weight"]
    assert set(ref) == set(ours)
    for name, p in ref.items():
        g = p.grad.numpy()
        scale = np.abs(g).max()
        assert scale > 0, name
        np.testing.assert_allclose(ours[name], g, rtol=0, atol=1e-6 * scale, err_msg=name)


def _torch_forward_ste(cfg, w, tokens, sf, temp):
    """Independent torch forward of the bf16-rounded decoder, rounding points as
    straight-through estimators: R(x) = x + (bf16(x) - x).detach()."""
    def R(x):
        return x + (x.to(torch.bfloat16).to(torch.float64) - x).detach()

    def f64(a):
        a = np.asarray(a)
        t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16) if a.dtype == np.uint16 \
            else torch.from_numpy(a)
        return t.to(torch.float64).clone().requires_grad_(True)

    P = {k: f64(v) for k, v in w.items()}
    T = len(tokens)
    H, Hk, hd, eps = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.rms_eps
    tok = torch.from_numpy(tokens)

    def norm(x, g):
        return x * torch.rsqrt((x * x).mean(-1, keepdim=True) + eps) * g

    inv = cfg.rope_theta ** (-2.0 * torch.arange(hd // 2, dtype=torch.float64) / hd)
    ang = torch.arange(T, dtype=torch.float64)[:, None] * inv[None, :]
    cs, sn = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]

    def rot(x):
        lo, hi = x[..., : hd // 2], x[..., hd // 2:]
        return torch.cat([lo * cs - hi * sn, hi * cs + lo * sn], -1)

    x = P["tok_emb"][tok]
    mask = torch.tril(torch.ones(T, T, dtype=torch.bool))
    for l in range(cfg.n_layers):
        p = f"l{l}."
        h = R(norm(x, P[p + "attn_norm"]))
        q = R(rot((h @ P[p + "wq"].T).view(T, H, hd)))
        k = R(rot((h @ P[p + "wk"].T).view(T, Hk, hd)))
        v = R((h @ P[p + "wv"].T).view(T, Hk, hd))
        outs = []
        for hh in range(H):
            g = hh * Hk // H
            s = (q[:, hh] @ k[:, g].T) / hd ** 0.5
            outs.append(torch.softmax(s.masked_fill(~mask, float("-inf")), -1) @ v[:, g])
        o = R(torch.cat(outs, -1))
        x = x + o @ P[p + "wo"].T
        h2 = R(norm(x, P[p + "mlp_norm"]))
        gt, up = h2 @ P[p + "w_gate"].T, h2 @ P[p + "w_up"].T
        x = x + R(torch.nn.functional.silu(gt) * up) @ P[p + "w_down"].T
    logits = R(norm(x, P["final_norm"])) @ P["lm_head"].T
    ls = torch.log_softmax(logits[sf - 1:-1] / temp, -1)
    return P, ls[torch.arange(T - sf), tok[sf:]]


def test_gradient_through_bf16_rounding_points_matches_straight_through_autograd():
    cfg = dataclasses.replace(MICRO, dtype=DTYPE_BF16)
    sf, temp = 4, 0.9
    w, tokens, dlogp = _case(cfg, 32, score_from=sf)
    ours = policy_gradient(OracleModel(cfg, w), tokens, sf, temp, dlogp)
    P, lp = _torch_forward_ste(cfg, w, tokens, sf, temp)
    (lp * torch.from_numpy(dlogp)).sum().backward()
    for name, p in P.items():
        g = p.grad.numpy()
        np.testing.assert_allclose(ours[name], g, rtol=0, atol=1e-10 * np.abs(g).max(),
                                   err_msg=name)


def test_gradient_matches_finite_differences_of_the_oracle_score():
    """Central differences of sum_j g_j logp_j (OracleModel.score) for a few
    entries of several weights."""
    cfg = MICRO
    w, tokens, dlogp = _case(cfg, 33, T=10, score_from=3)
    ours = policy_gradient(OracleModel(cfg, w), tokens, 3, 1.0, dlogp)
    rng = np.random.default_rng(0)

    def objective(wd):
        return float(np.dot(OracleModel(cfg, wd).score(tokens[None], 3, 1.0)[0], dlogp))

    for name in ("tok_emb", "l0.attn_norm", "l0.wk", "l1.wv", "l0.w_up", "final_norm", "lm_head"):
        a = np.asarray(w[name], np.float64)
        idx = tuple(rng.integers(0, n) for n in a.shape)
        if name == "tok_emb":
            idx = (int(tokens[2]),) + idx[1:]
        eps = 1e-6
        wp, wm = dict(w), dict(w)
        ap, am = a.copy(), a.copy()
        ap[idx] += eps
        am[idx] -= eps
        wp[name], wm[name] = ap, am
        fd = (objective(wp) - objective(wm)) / (2 * eps)
        assert abs(fd - ours[name][idx]) <= 1e-6 * max(1.0, abs(fd)), (name, idx, fd, ours[name][idx])


def test_degenerate_cases():
    cfg = MICRO
    w, tokens, dlogp = _case(cfg, 34)
    om = OracleModel(cfg, w)
    zero = policy_gradient(om, tokens, 5, 1.0, np.zeros_like(dlogp))
    assert all(np.all(g == 0) for g in zero.values())
    # one scored token: the head gradient has rank one, rows of unseen tokens are zero
    g1 = policy_gradient(om, tokens, len(tokens) - 1, 1.0, np.array([1.0]))
    assert np.linalg.matrix_rank(g1["lm_head"]) == 1
    unseen = np.setdiff1d(np.arange(cfg.vocab), tokens)
    assert np.all(g1["tok_emb"][unseen] == 0)
    # the last token never feeds a scored log-prob: changing it changes nothing
    t2 = tokens.copy()
    t2[-1] = (t2[-1] + 1) % cfg.vocab
    g2 = policy_gradient(om, t2, 5, 1.0, np.zeros_like(dlogp))
    assert all(np.all(g == 0) for g in g2.values())


def test_adamw_matches_torch():
    rng = np.random.default_rng(5)
    p0 = rng.standard_normal(50)
    grads = [rng.standard_normal(50) for _ in range(3)]
    hp = dict(lr=1e-3, betas=(0.9, 0.95), eps=1e-8, weight_decay=0.1)
    t = torch.from_numpy(p0.copy()).requires_grad_(True)
    opt = torch.optim.AdamW([t], **hp)
    p, m, v = p0.copy(), np.zeros(50), np.zeros(50)
    for s, g in enumerate(grads, 1):
        t.grad = torch.from_numpy(g)
        opt.step()
        p, m, v = adamw(p, g, m, v, s, hp["lr"], hp["betas"][0], hp["betas"][1], hp["eps"],
                        hp["weight_decay"])
        np.testing.assert_allclose(p, t.detach().numpy(), rtol=0, atol=1e-15)
