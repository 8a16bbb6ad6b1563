"""CPU tests of the rounding-point-local checker (tests/bounds.py,
tests/stagecheck.py): an fp32 emulation that follows the arithmetic model is
accepted, and each planted mistake is rejected."""
import dataclasses

import numpy as np
import pytest

import oracle
from bounds import Gemm, Report, attention_bound, check_bf16, check_f32, rows_gemm
from emulate import emulate_layer, gemm32
from paper_2510_17158_amd import synth
from paper_2510_17158_amd.workloads import SMALL
from stagecheck import StageChecker, flash_segments

CFG = dataclasses.replace(SMALL, n_layers=1, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64,
                          d_ffn=512, vocab=512)


def _layer_case(mutate=None, B=6, seed=3):
    host = synth.make_weights(CFG, seed, gain_noise=0.1)
    om = oracle.OracleModel(CFG, host)
    rng = np.random.default_rng(seed)
    ctx_max = 80
    Kc = oracle.round_bf16(rng.standard_normal((B, CFG.n_kv_heads, ctx_max, CFG.head_dim)))
    Vc = oracle.round_bf16(rng.standard_normal((B, CFG.n_kv_heads, ctx_max, CFG.head_dim)))
    pos = rng.integers(5, ctx_max, B)
    x = rng.standard_normal((B, CFG.d_model)).astype(np.float32)
    e = emulate_layer(CFG, om, 0, x, pos, Kc, Vc, mutate)
    tr = {k: v[None] for k, v in e.items() if k != "x_out"}
    tr["x"] = np.stack([e["x"], e["x_out"]]).astype(np.float64)
    chk = StageChecker(CFG, host)
    g = Gemm("mfma", 32)
    gem = dict(qkv=g, o=g, gu=g, down=g)

    def context(i):
        return Kc[i, :, :pos[i] + 1].transpose(1, 0, 2), Vc[i, :, :pos[i] + 1].transpose(1, 0, 2)

    chk.layer(0, tr, np.arange(B), pos, context, lambda i: flash_segments(int(pos[i]) + 1), gem)
    return chk.rep


def test_emulated_layer_accepted():
    rep = _layer_case()
    print(rep.summary())
    assert rep.ok(), rep.summary()
    # the check is bit-exact on most elements: few are ambiguous (attention
    # outputs more: P enters P.V to 16 bits, hi + lo)
    for name, s in rep.summary().items():
        assert s["amb_frac"] < (0.3 if name == "o" else 0.05), (name, s)


@pytest.mark.parametrize("mutate,stage", [("drop_term", "q"), ("rope_sign", "k"),
                                          ("scale", "o"), ("reversed_v", "o"),
                                          ("no_resid", "x_attn")])
def test_planted_mistakes_rejected(mutate, stage):
    rep = _layer_case(mutate)
    s = rep.summary()
    assert not rep.ok()
    assert s[stage]["bad"] > 0, s


def test_gemm_bound_chain_models():
    """Emulated chains (exact step sums rounded once into fp32) stay inside the
    bound for 32- and 16-wide steps and for split / wave structures; a one-ulp
    bias on every step does not."""
    rng = np.random.default_rng(0)
    a = oracle.round_bf16(rng.standard_normal((16, 1024)))
    W = oracle.round_bf16(rng.standard_normal((64, 1024)) * 0.02)
    for kc in (16, 32):
        y, E = Gemm("mfma", kc).bound(a, W)
        got = gemm32(a, W, kc)
        rep = Report()
        check_f32(rep, "y", got, y, E)
        assert rep.ok()
        assert np.all(E < 1e-3 * np.abs(a) @ np.abs(W).T)
    # 4 waves x 2 splits: emulate the kernel's order exactly
    g = Gemm("mfma", 32, 2, 4)
    y, E = g.bound(a, W)
    parts = []
    for s in range(2):
        ch = []
        for w in range(4):
            acc = np.zeros((16, 64), np.float32)
            for k0 in range(s * 512 + w * 32, (s + 1) * 512, 128):
                acc = (acc.astype(np.float64) + a[:, k0:k0 + 32] @ W[:, k0:k0 + 32].T).astype(
                    np.float32)
            ch.append(acc)
        parts.append((ch[0] + ch[2]) + (ch[1] + ch[3]))
    got = parts[0] + parts[1]
    rep = Report()
    check_f32(rep, "y", got, y, E)
    assert rep.ok()
    biased = got + np.abs(got) * 2.0 ** -23 * 64
    rep = Report()
    check_f32(rep, "y", biased, y, E)
    assert not rep.ok()


def test_bf16_interval_check():
    """Exact values are unique and accepted; one ulp off is rejected unless the
    bound straddles a rounding midpoint."""
    rng = np.random.default_rng(1)
    y = rng.standard_normal(10000)
    E = np.full_like(y, 1e-7)
    g = oracle.round_bf16(y)
    rep = Report()
    check_bf16(rep, "h", g, y, E)
    s = rep.summary()["h"]
    assert s["bad"] == 0 and s["amb_frac"] < 1e-3
    ulp = 2.0 ** (np.floor(np.log2(np.abs(g))) - 7)
    rep = Report()
    ok = check_bf16(rep, "h", g + ulp, y, E)
    assert ok.mean() < 1e-3


def test_attention_bound_mfma_and_decode_chains():
    """Flash-like and decode-like fp32 evaluations of one query stay inside the
    attention bound; the bound is far below an ulp of the output."""
    rng = np.random.default_rng(2)
    hd, ctx = 128, 700
    q = oracle.round_bf16(rng.standard_normal(hd))
    K = oracle.round_bf16(rng.standard_normal((ctx, hd)))
    V = oracle.round_bf16(rng.standard_normal((ctx, hd)))
    for segs, merges in (([("mfma", 0, ctx, ctx)], 0), ([("decode", 0, ctx, 256)], 7),
                         ([("decode", 0, ctx, 256, 2)], 5),
                         ([("mfma", 0, 512, 256), ("decode", 512, ctx, 128)], 24)):
        o, E = attention_bound(q, K, V, hd, segs, merges)
        assert np.all(E < 1e-3 * np.abs(V).mean())
        from emulate import attn32
        got = attn32(q, K, V, 1.0 / np.sqrt(hd))
        rep = Report()
        check_f32(rep, "o", got, o, E)
        assert rep.ok(), rep.summary()
