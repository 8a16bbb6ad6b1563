"""The C-ABI library loads without a GPU, exports what the header declares, and
rejects bad arguments before touching the device."""
import ctypes as C
import os
import re

import pytest

from paper_2510_17158_amd import api
from paper_2510_17158_amd.workloads import DTYPE_BF16, DTYPE_F32, get

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "grpo_hip.h")

pytestmark = pytest.mark.skipif(not os.path.exists(api.LIB_PATH), reason="library not built")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(grpo_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = _declared()
    assert "grpo_rollout_step" in names and "grpo_token_loss" in names
    L = api.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) >= set(api._SIGS)


def _fake_model(cfg):
    """A handle over fake (never dereferenced) device pointers."""
    L = cfg.n_layers
    fake = (C.c_void_p * L)(*[0x1000 + i for i in range(L)])
    w = api.Weights(0x1000, *[C.cast(fake, api._PP)] * 9, 0x1000, 0x1000)
    h = C.c_void_p()
    rc = api.lib().grpo_model_create(C.byref(api.config_struct(cfg)), C.byref(w), C.byref(h))
    return rc, h, fake


def test_config_validation():
    cfg = get("small").model
    rc, h, _ = _fake_model(cfg)
    assert rc == api.OK and h
    api.lib().grpo_model_destroy(h)
    for bad, code in [(dict(head_dim=96), api.UNSUPPORTED), (dict(n_kv_heads=5), api.UNSUPPORTED),
                      (dict(dtype=7), api.UNSUPPORTED), (dict(n_layers=0), api.INVALID_ARG),
                      (dict(d_model=800), api.UNSUPPORTED), (dict(n_heads=48, n_kv_heads=4),
                                                             api.UNSUPPORTED),
                      (dict(vocab=32001), api.UNSUPPORTED)]:
        import dataclasses
        rc, h, _ = _fake_model(dataclasses.replace(cfg, **bad))
        assert rc == code, (bad, rc)
        assert api.lib().grpo_last_error()


def test_sizes():
    c = get("7b").model
    assert api.kv_cache_bytes(c, 64, 4095) == 32 * 2 * 64 * 8 * 4095 * 128 * 2
    t = get("tiny").model
    assert api.kv_cache_bytes(t, 16, 127) == 2 * 2 * 16 * 4 * 127 * 64 * 4
    rc, h, keep = _fake_model(get("small").model)
    m = type("M", (), {"handle": h})()
    for op, rows, ln in [(api.OP_PREFILL, 8, 512), (api.OP_ROLLOUT, 64, 1023),
                         (api.OP_SCORE, 64, 1024)]:
        assert api.workspace_bytes(m, op, rows, ln) > 0
    assert api.workspace_bytes(None, api.OP_LOSS, 64, 2048) >= 64 * 9 * 8
    assert api.workspace_bytes(m, api.OP_ROLLOUT, 0, 10) == 0
    api.lib().grpo_model_destroy(h)


def test_decode_weights_size_and_errors():
    L = api.lib()
    c = get("small").model
    d, qd, kvd, f = c.d_model, c.q_dim, c.kv_dim, c.d_ffn
    per_layer = (qd + 2 * kvd) * d + d * qd + 2 * f * d + d * f
    want = (c.n_layers * per_layer + c.vocab * d) * 2   # every piece is a multiple of 256 bytes
    assert L.grpo_decode_weights_bytes(C.byref(api.config_struct(c))) == want
    assert L.grpo_decode_weights_bytes(C.byref(api.config_struct(get("tiny").model))) == 0
    rc, h, keep = _fake_model(c)
    p = C.c_void_p(0x1000)
    # no decode copy yet: a bf16 rollout step is refused before any device work
    s = api.Sampling(1.0, 0, 1)
    assert L.grpo_rollout_step(h, p, 64, 100, 64, p, p, 10, 1, 2, C.byref(s), p, p, None, None, p,
                               1 << 40, None) == api.INVALID_ARG
    assert b"decode weights" in L.grpo_last_error()
    assert L.grpo_model_pack_decode(h, None, 1 << 40, None) == api.INVALID_ARG
    assert L.grpo_model_pack_decode(h, C.c_void_p(0x100000), want - 1, None) == api.INVALID_ARG
    assert L.grpo_model_pack_decode(h, C.c_void_p(0x100010), want, None) == api.INVALID_ARG
    assert L.grpo_model_pack_decode(None, p, want, None) == api.INVALID_ARG
    L.grpo_model_destroy(h)
    rc, h, keep = _fake_model(get("tiny").model)   # fp32: nothing to pack
    assert L.grpo_model_pack_decode(h, None, 0, None) == api.OK
    L.grpo_model_destroy(h)


def test_argument_errors_before_device_work():
    L = api.lib()
    rc, h, keep = _fake_model(get("small").model)
    s = api.Sampling(1.0, 0, 1)
    p = C.c_void_p(0x1000)
    # KV capacity: max_pos + n_steps > max_len
    r = L.grpo_rollout_step(h, p, 64, 100, 64, p, p, 99, 1, 2, C.byref(s), p, p, None, None, p,
                            1 << 40, None)
    assert r == api.KV_CAPACITY
    # workspace too small
    r = L.grpo_rollout_step(h, p, 64, 100, 64, p, p, 10, 1, 2, C.byref(s), p, p, None, None, p, 16,
                            None)
    assert r == api.WORKSPACE_TOO_SMALL
    # grouped steps: G must divide B, 0 <= prefix_len <= max_len; the per-row
    # checks still apply
    def grouped(G, prefix, max_pos=10):
        return L.grpo_rollout_step_grouped(h, p, 64, 100, 64, G, prefix, p, p, max_pos, 1, 2,
                                           C.byref(s), p, p, None, None, p, 1 << 40, None)
    assert grouped(0, 50) == api.INVALID_ARG
    assert grouped(3, 50) == api.INVALID_ARG
    assert grouped(8, 101) == api.INVALID_ARG
    assert grouped(8, -1) == api.INVALID_ARG
    assert grouped(8, 50, max_pos=99) == api.KV_CAPACITY
    # B above n_seqs, bad temperature, bad top_k
    assert L.grpo_rollout_step(h, p, 8, 100, 64, p, p, 10, 1, 2, C.byref(s), p, p, None, None, p,
                               1 << 40, None) == api.INVALID_ARG
    bad = api.Sampling(-1.0, 0, 1)
    assert L.grpo_rollout_step(h, p, 64, 100, 64, p, p, 10, 1, 2, C.byref(bad), p, p, None, None,
                               p, 1 << 40, None) == api.INVALID_ARG
    bad = api.Sampling(1.0, 40000, 1)
    assert L.grpo_prefill(h, p, 64, 100, p, 8, 10, 8, C.byref(bad), p, p, None, None, p, 1 << 40,
                          None) == api.INVALID_ARG
    # prefill: P*G > n_seqs, prompt longer than the cache
    assert L.grpo_prefill(h, p, 8, 100, p, 8, 10, 8, C.byref(s), p, p, None, None, p, 1 << 40,
                          None) == api.INVALID_ARG
    assert L.grpo_prefill(h, p, 64, 100, p, 8, 200, 8, C.byref(s), p, p, None, None, p, 1 << 40,
                          None) == api.KV_CAPACITY
    # grouped scoring: G must divide N, 0 <= prefix_len <= score_from
    assert L.grpo_score_sequences_grouped(h, p, 8, 100, 50, 1.0, 3, 50, p, p, 1 << 40,
                                          None) == api.INVALID_ARG
    assert L.grpo_score_sequences_grouped(h, p, 8, 100, 50, 1.0, 4, 51, p, p, 1 << 40,
                                          None) == api.INVALID_ARG
    assert L.grpo_score_sequences_grouped(h, p, 8, 100, 50, 1.0, 0, 50, p, p, 1 << 40,
                                          None) == api.INVALID_ARG
    # scoring range
    assert L.grpo_score_sequences(h, p, 4, 10, 0, 1.0, p, p, 1 << 40, None) == api.INVALID_ARG
    assert L.grpo_score_sequences(h, p, 4, 10, 10, 1.0, p, p, 1 << 40, None) == api.INVALID_ARG
    # advantages and loss
    assert L.grpo_advantages(p, 4, 1, 1e-6, p, None) == api.INVALID_ARG
    assert L.grpo_advantages(None, 4, 2, 1e-6, p, None) == api.INVALID_ARG
    assert L.grpo_token_loss(p, p, p, p, p, 4, 8, 0.2, 0.04, 2, p, None, None, None, p, 1 << 20,
                             None) == api.INVALID_ARG
    assert L.grpo_token_loss(p, p, p, p, p, 4, 8, 1.5, 0.04, 0, p, None, None, None, p, 1 << 20,
                             None) == api.INVALID_ARG
    assert L.grpo_token_loss(p, p, p, p, p, 4, 8, 0.2, 0.04, 0, p, None, None, None, p, 8,
                             None) == api.WORKSPACE_TOO_SMALL
    assert b"workspace" in L.grpo_last_error()
    L.grpo_model_destroy(h)


def test_product_path_has_no_cpu_fallback():
    import paper_2510_17158_amd.api as a
    import paper_2510_17158_amd.runner as r
    for mod in (a, r):
        src = open(mod.__file__).read()
        assert "import oracle" not in src and "from oracle" not in src
