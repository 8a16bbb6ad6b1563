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
    assert L.grpo_rollout_step(h, p, 64, 100, 64, None, p, p, 10, 1, 2, C.byref(s), p, p, None, p,
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
    BIG = 1 << 40

    def roll(n_seqs=64, B=64, max_pos=10, ids=None, ws_bytes=BIG, samp=s):
        return L.grpo_rollout_step(h, p, n_seqs, 100, B, ids, p, p, max_pos, 1, 2, C.byref(samp),
                                   p, p, None, p, ws_bytes, None)
    # KV capacity: max_pos + n_steps > max_len
    assert roll(max_pos=99) == api.KV_CAPACITY
    # workspace too small
    assert roll(ws_bytes=16) == api.WORKSPACE_TOO_SMALL
    # grouped steps: G must divide B, 0 <= prefix_len <= max_len; the per-row
    # checks still apply
    def grouped(G, prefix, max_pos=10, ids=None):
        return L.grpo_rollout_step_grouped(h, p, 64, 100, 64, G, prefix, ids, p, p, max_pos, 1, 2,
                                           C.byref(s), p, p, None, p, BIG, None)
    assert grouped(0, 50) == api.INVALID_ARG
    assert grouped(3, 50) == api.INVALID_ARG
    assert grouped(8, 101) == api.INVALID_ARG
    assert grouped(8, -1) == api.INVALID_ARG
    assert grouped(8, 50, max_pos=99) == api.KV_CAPACITY
    # B above n_seqs or above 128 for a bf16 model, bad temperature, bad top_k
    assert roll(n_seqs=8) == api.INVALID_ARG
    assert roll(n_seqs=200, B=130) == api.UNSUPPORTED
    assert roll(samp=api.Sampling(-1.0, 0, 1)) == api.INVALID_ARG
    # seq_ids: each in [0, n_seqs), no repeats (host array, checked before any work)
    ids = lambda v: (C.c_int32 * len(v))(*v)  # noqa: E731
    good = list(range(63, -1, -1))
    assert roll(ids=ids(good), ws_bytes=16) == api.WORKSPACE_TOO_SMALL   # ids accepted
    assert roll(ids=ids(good[:-1] + [64])) == api.INVALID_ARG
    assert b"seq_ids" in L.grpo_last_error()
    assert roll(ids=ids(good[:-1] + [-1])) == api.INVALID_ARG
    assert roll(ids=ids(good[:-1] + [5])) == api.INVALID_ARG
    assert b"repeats" in L.grpo_last_error()
    assert roll(n_seqs=100, B=4, ids=ids([99, 0, 50, 7]), ws_bytes=16) == api.WORKSPACE_TOO_SMALL
    assert grouped(8, 50, ids=ids(good[:-1] + [70])) == api.INVALID_ARG
    bad = api.Sampling(1.0, 40000, 1)
    assert L.grpo_prefill(h, p, 64, 100, p, 8, 10, 8, C.byref(bad), p, p, None, p, BIG,
                          None) == api.INVALID_ARG
    # prefill: P*G > n_seqs, prompt longer than the cache
    assert L.grpo_prefill(h, p, 8, 100, p, 8, 10, 8, C.byref(s), p, p, None, p, BIG,
                          None) == api.INVALID_ARG
    assert L.grpo_prefill(h, p, 64, 100, p, 8, 200, 8, C.byref(s), p, p, None, p, BIG,
                          None) == api.KV_CAPACITY
    # grouped scoring: G must divide N, 0 <= prefix_len <= score_from
    assert L.grpo_score_sequences_grouped(h, p, 8, 100, 50, 1.0, 3, 50, p, None, p, BIG,
                                          None) == api.INVALID_ARG
    assert L.grpo_score_sequences_grouped(h, p, 8, 100, 50, 1.0, 4, 51, p, None, p, BIG,
                                          None) == api.INVALID_ARG
    assert L.grpo_score_sequences_grouped(h, p, 8, 100, 50, 1.0, 0, 50, p, None, p, BIG,
                                          None) == api.INVALID_ARG
    # scoring range
    assert L.grpo_score_sequences(h, p, 4, 10, 0, 1.0, p, None, p, BIG, None) == api.INVALID_ARG
    assert L.grpo_score_sequences(h, p, 4, 10, 10, 1.0, p, None, p, BIG, None) == api.INVALID_ARG
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


def test_extend_argument_errors_before_device_work():
    """grpo_extend checks its host arrays (positions, sequence ids) and the span
    length before any device work."""
    L = api.lib()
    rc, h, keep = _fake_model(get("small").model)
    s = api.Sampling(1.0, 0, 1)
    p = C.c_void_p(0x1000)
    BIG = 1 << 40
    arr = lambda v: (C.c_int32 * len(v))(*v)  # noqa: E731

    def ext(pos0, ids=None, n_seqs=8, B=4, Te=16, ws_bytes=16, max_len=100):
        return L.grpo_extend(h, p, n_seqs, max_len, B, ids, arr(pos0), p, Te, 3, C.byref(s), p, p,
                             None, p, ws_bytes, None)
    ok = [10, 84, 0, 50]
    assert ext(ok) == api.WORKSPACE_TOO_SMALL                 # arguments accepted
    assert ext([10, 85, 0, 50]) == api.KV_CAPACITY             # 85 + 16 > 100
    assert ext([10, -1, 0, 50]) == api.INVALID_ARG
    assert b"negative" in L.grpo_last_error()
    assert ext(ok, Te=0) == api.INVALID_ARG
    assert ext(ok, Te=api.EXTEND_CHUNK + 1, max_len=2000) == api.INVALID_ARG
    assert ext(ok, n_seqs=3) == api.INVALID_ARG                # B > n_seqs without ids
    assert ext(ok, ids=arr([7, 0, 3, 5])) == api.WORKSPACE_TOO_SMALL
    assert ext(ok, ids=arr([7, 0, 3, 7])) == api.INVALID_ARG
    assert b"repeats" in L.grpo_last_error()
    assert ext(ok, ids=arr([7, 0, 3, 8])) == api.INVALID_ARG
    assert L.grpo_extend(h, p, 8, 100, 4, None, None, p, 16, 3, C.byref(s), p, p, None, p, BIG,
                         None) == api.INVALID_ARG
    need = L.grpo_workspace_bytes(h, api.OP_EXTEND, 4, 100)
    assert need > 0 and ext(ok, ws_bytes=need - 1) == api.WORKSPACE_TOO_SMALL
    L.grpo_model_destroy(h)


def test_backward_and_adamw_argument_errors():
    """grpo_policy_backward and grpo_adamw_step reject bad arguments before any
    device work."""
    L = api.lib()
    cfg = get("small").model
    rc, h, keep = _fake_model(cfg)
    p = C.c_void_p(0x1000)
    BIG = 1 << 44
    Lc = cfg.n_layers
    arrs = [(C.c_void_p * Lc)(*([0x2000] * Lc)) for _ in range(9)]
    g = api.GradsStruct(p, *[C.cast(a, api._PP) for a in arrs], p, p)

    def bwd(N=2, T=100, sf=10, temp=1.0, grads=g, ws_bytes=BIG):
        return L.grpo_policy_backward(h, p, N, T, sf, temp, p, C.byref(grads) if grads else None,
                                      p, ws_bytes, None)
    assert bwd(ws_bytes=16) == api.WORKSPACE_TOO_SMALL          # arguments accepted
    assert bwd(sf=0) == api.INVALID_ARG
    assert bwd(sf=100) == api.INVALID_ARG
    assert bwd(T=1, sf=1) == api.INVALID_ARG
    assert bwd(temp=-1.0) == api.INVALID_ARG
    assert bwd(T=20000) == api.UNSUPPORTED
    assert bwd(grads=None) == api.INVALID_ARG
    holes = (C.c_void_p * Lc)(*([0x2000] * (Lc - 1) + [0]))
    g2 = api.GradsStruct(p, *[C.cast(a, api._PP) for a in arrs[:4]], C.cast(holes, api._PP),
                         *[C.cast(a, api._PP) for a in arrs[5:]], p, p)
    assert bwd(grads=g2) == api.INVALID_ARG
    assert b"layer" in L.grpo_last_error()
    need = L.grpo_workspace_bytes(h, api.OP_BACKWARD, 2, 100)
    assert need > 0 and bwd(ws_bytes=need - 1) == api.WORKSPACE_TOO_SMALL
    assert L.grpo_workspace_bytes(h, api.OP_BACKWARD, 2, 20000) == 0
    hp = api.AdamW(1e-3, 0.9, 0.95, 1e-8, 0.1)
    assert L.grpo_adamw_step(1, p, None, p, p, p, 10, C.byref(hp), 1, None) == api.INVALID_ARG
    assert L.grpo_adamw_step(0, p, None, p, p, p, 10, C.byref(hp), 0, None) == api.INVALID_ARG
    assert L.grpo_adamw_step(2, p, p, p, p, p, 10, C.byref(hp), 1, None) == api.INVALID_ARG
    bad = api.AdamW(1e-3, 1.0, 0.95, 1e-8, 0.1)
    assert L.grpo_adamw_step(0, p, None, p, p, p, 10, C.byref(bad), 1, None) == api.INVALID_ARG
    L.grpo_model_destroy(h)


def test_decode_structure_query():
    """The reduction structure the tests' error bounds use comes from the library's
    own planner; its arguments are checked."""
    L = api.lib()
    rc, h, keep = _fake_model(get("7b").model)
    out = (C.c_int32 * 9)()
    assert L.grpo_decode_structure(h, 64, 4095, 8, 2048, out) == api.OK
    v = list(out)
    assert all(x >= 1 for x in v[:6]) and v[3] == 1       # the LM head is never split
    assert v[6] > 0 and v[7] >= 1 and v[6] * v[7] >= 2048
    assert v[8] == 4                       # 512 per-row workgroups fit on the chip at once
    assert L.grpo_decode_structure(h, 96, 4095, 12, 2048, out) == api.OK and out[8] == 4
    assert L.grpo_decode_structure(h, 128, 4095, 8, 2048, out) == api.OK and out[8] == 2
    assert L.grpo_decode_structure(h, 64, 4095, 0, 0, out) == api.OK and list(out)[6:8] == [0, 0]
    assert L.grpo_decode_structure(h, 129, 4095, 0, 0, out) == api.INVALID_ARG
    assert L.grpo_decode_structure(h, 64, 4095, 3, 100, out) == api.INVALID_ARG
    assert L.grpo_decode_structure(None, 64, 4095, 0, 0, out) == api.INVALID_ARG
    L.grpo_model_destroy(h)


def test_product_path_has_no_cpu_fallback():
    import paper_2510_17158_amd.api as a
    import paper_2510_17158_amd.runner as r
    for mod in (a, r):
        src = open(mod.__file__).read()
        assert "import oracle" not in src and "from oracle" not in src


def test_reward_host_call_matches_the_oracle_and_checks_arguments():
    """grpo_reward computes on the host (no GPU): every branch of Eq. 2-4 against
    the oracle, and bad times / tool counts rejected before any output."""
    import numpy as np
    import oracle
    rng = np.random.default_rng(3)
    n = 2000
    c = rng.random(n) < 0.7
    tb = rng.lognormal(0, 1, n)
    t = tb * rng.lognormal(0, 1.2, n)
    t[:5] = tb[:5]                          # exactly as fast: r_perf 0
    avail = rng.integers(4, 7, n)
    used = (rng.random(n) * (avail + 1)).astype(np.int32)
    got = api.reward(c, tb, t, used, avail)
    want = oracle.reward(c, tb, t, used, avail)
    # fp32 output of an fp64 evaluation
    np.testing.assert_allclose(got, want, rtol=2.0 ** -24, atol=0)
    assert got.min() >= -2.0 and got.max() <= 10.5
    for bad in (dict(t=-1.0), dict(t_base=0.0), dict(used=5, avail=4), dict(avail=0)):
        args = dict(c=1, t_base=1.0, t=0.5, used=1, avail=4)
        args.update(bad)
        with pytest.raises(api.GrpoError) as e:
            api.reward([args["c"]], [args["t_base"]], [args["t"]], [args["used"]],
                       [args["avail"]])
        assert e.value.code == api.INVALID_ARG
