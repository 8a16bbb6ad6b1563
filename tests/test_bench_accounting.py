"""The bench's algorithmic work figures (the denominators of its roofline
fractions) against hand computations from the 7B shape: 32 layers, d 4096,
32 / 8 heads of 128, ffn 14336, vocab 32000; 8 prompts x G 8, prompt 2048,
2048 sampled tokens, bf16."""
import importlib.util
import os

import pytest

from paper_2510_17158_amd.workloads import get

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


L, d, Hq, Hk, hd, f, V = 32, 4096, 32, 8, 128, 14336, 32000
P, G, Tp, Tn = 8, 8, 2048, 2048
B, T = P * G, Tp + Tn
KV_TOK = L * 2 * Hk * hd * 2                       # bytes of K and V per position, all layers
WEIGHTS = 2 * (L * (d * (Hq + 2 * Hk) * hd + Hq * hd * d + 3 * d * f + 2 * d) + d + V * d)


def test_decode_bytes_per_step():
    b = _bench()
    w = get("7b")
    n_dec = Tn - 1
    ctx = Tp + n_dec / 2
    per_row = WEIGHTS + B * d * 2 + B * ctx * KV_TOK + B * KV_TOK
    shared = WEIGHTS + B * d * 2 + (P * Tp + B * (ctx - Tp)) * KV_TOK + B * KV_TOK
    assert b.decode_bytes_per_step(w.with_(shared_prompt=False), ctx) == pytest.approx(per_row)
    assert b.decode_bytes_per_step(w, ctx) == pytest.approx(shared)
    assert per_row / 1e9 == pytest.approx(40.0, rel=2e-3)
    assert shared / 1e9 == pytest.approx(24.96, rel=2e-3)


def test_attention_bytes_per_launch():
    b = _bench()
    w = get("7b")
    n_dec = Tn - 1
    kb = b.kernel_bytes(w)
    per_layer_tok = 2 * Hk * hd * 2
    assert kb["attn_prefix"] / (n_dec * L) == pytest.approx(P * Tp * per_layer_tok)   # 67.1 MB
    own = sum(range(1, n_dec + 1)) / n_dec                                            # 1024
    assert kb["attn_decode"] / (n_dec * L) == pytest.approx(B * own * per_layer_tok)  # 268.4 MB
    kb1 = b.kernel_bytes(w.with_(shared_prompt=False))
    assert "attn_prefix" not in kb1
    assert kb1["attn_decode"] / (n_dec * L) == pytest.approx(B * (Tp + own) * per_layer_tok)


def test_score_flops():
    b = _bench()
    w = get("7b")
    proj = 2 * (d * (Hq + 2 * Hk) * hd + Hq * hd * d + 3 * d * f)       # per row and layer
    pair = 4 * L * Hq * hd                                                # per (query, key) pair
    head = 2 * V * d * (T - Tp) * B
    full = L * proj * B * T + pair * B * T * (T + 1) / 2 + head
    rows = P * Tp + B * (T - Tp)
    pairs = P * Tp * (Tp + 1) / 2 + B * (T * (T + 1) / 2 - Tp * (Tp + 1) / 2)
    shared = L * proj * rows + pair * pairs + head
    assert b.score_flops(w.with_(shared_prompt=False)) == pytest.approx(full)
    assert b.score_flops(w) == pytest.approx(shared)
    assert full / 1e15 == pytest.approx(3.975, rel=1e-3)
    assert shared / 1e15 == pytest.approx(2.3126, rel=1e-3)


def test_update_flops_per_sequence():
    """Gradient of one sequence's scored log-probs: three forwards' worth of the
    projections over all T rows, causal attention and the head on the Tn scored
    rows (186.3 TFLOP at the 7B shape)."""
    b = _bench()
    w = get("7b")
    proj = 2 * (d * (Hq + 2 * Hk) * hd + Hq * hd * d + 3 * d * f)
    fwd = L * proj * T + 4 * L * Hq * hd * T * (T + 1) / 2 + 2 * V * d * Tn
    assert b.update_flops_per_seq(w) == pytest.approx(3 * fwd)
    assert 3 * fwd / 1e12 == pytest.approx(186.33, rel=1e-3)


def test_attention_traffic_reading():
    """The counter reading at 1024 generated positions, the mean launch of the 7B
    rollout; null when the kernel source changed, at another batch or at another
    mean context."""
    b = _bench()
    t = b.ATTN_TRAFFIC
    alg = B * 1024 * 2 * Hk * hd * 2
    exp = (t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"]) * 1024
    got = b.attn_traffic(alg)
    if got is not None:
        assert got == pytest.approx(exp)
        assert 1.0 < got / alg < 1.1
    assert b.attn_traffic(alg * 1.5, 96) is None    # measured at batch 64 only
    assert b.attn_traffic(alg / 2) is None          # and at the 7B rollout's mean context
    saved = dict(t)
    try:
        t["sha256"] = "0" * 64
        assert b.attn_traffic(alg) is None
    finally:
        t.clear()
        t.update(saved)
