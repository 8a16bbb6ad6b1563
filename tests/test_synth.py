"""The seeded input generators are deterministic and per-tensor reproducible."""
import numpy as np

from paper_2510_17158_amd import synth, workloads


def test_weights_deterministic_and_per_tensor():
    cfg = workloads.truncated(workloads.get("small"), 1).model
    a = synth.make_weights(cfg, 5)
    b = synth.make_weights(cfg, 5, names=["l0.wk"])
    assert np.array_equal(a["l0.wk"], b["l0.wk"])
    assert a["l0.wq"].dtype == np.uint16 and a["l0.wq"].shape == (cfg.q_dim, cfg.d_model)
    r = synth.make_weights(cfg, 5, ref=True, names=["l0.wq"])["l0.wq"]
    assert not np.array_equal(r, a["l0.wq"])
    assert np.all(a["l0.attn_norm"] == 0x3F80)        # gains 1.0 in bf16


def test_prompts_structure_and_rewards():
    w = workloads.get("7b").with_(n_prompts=2)
    p = synth.make_prompts(w)
    assert p.shape == (2, 2048) and p.dtype == np.int32
    assert np.all(p[:, 0] == synth.BOS)
    assert np.all((p >= 0) & (p < w.model.vocab))
    assert np.all((p == synth.TOOL).sum(axis=1) >= w.tool_spans)
    r = synth.make_rewards(workloads.get("small"))
    assert r.shape == (64,) and np.all(r >= 0)
    assert np.array_equal(r, synth.make_rewards(workloads.get("small")))
    assert 0 < synth.make_seed(w) < 2**63
