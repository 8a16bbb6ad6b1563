"""Pins of the oracle's elementwise pieces against library routines and closed forms."""
import numpy as np
import pytest
import torch
from scipy.special import expit

from oracle import bf16_bits_to_f64, rmsnorm, rope, round_bf16, silu


def _torch_bf16(x32: np.ndarray) -> np.ndarray:
    return torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()


def test_round_bf16_matches_torch_rne():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(1_000_000) * np.exp(rng.uniform(-30, 30, 1_000_000))).astype(np.float32)
    # exact ties: bf16 value + half an ulp, both even and odd mantissas
    base = rng.standard_normal(20000).astype(np.float32)
    bits = base.view(np.uint32) & np.uint32(0xFFFF0000)
    ties = (bits | np.uint32(0x8000)).view(np.float32)
    sub = (rng.integers(1, 2**23, 20000).astype(np.uint32)).view(np.float32)  # subnormals
    special = np.array([0.0, -0.0, np.inf, -np.inf, 3.3895314e38, -3.3895314e38,
                        1.1754944e-38], np.float32)
    allx = np.concatenate([x, ties, sub, -sub, special])
    ours = round_bf16(allx)
    ref = _torch_bf16(allx)
    assert np.array_equal(ours.view(np.uint64), ref.view(np.uint64))
    assert np.isnan(round_bf16(np.array([np.nan]))[0])


def test_round_bf16_rounds_via_fp32():
    # a float64 value just above a bf16 tie that becomes an exact tie in fp32
    tie32 = np.float32(np.uint32(0x3F808000).view(np.float32))  # 1.00390625: halfway
    x = np.float64(tie32) + 1e-12
    assert round_bf16(np.array([x]))[0] == 1.0  # tie to even after fp32 rounding


def test_bf16_bits_roundtrip():
    bits = np.arange(0, 65536, dtype=np.uint32).astype(np.uint16)
    f = bf16_bits_to_f64(bits)
    ok = ~np.isnan(f)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(f[ok], ref[ok])
    assert np.array_equal(round_bf16(f[ok]), f[ok])


def test_rmsnorm_unit_rms_and_gain():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 96)) * 3.0
    eps = 1e-6
    y = rmsnorm(x, np.ones(96), eps)
    ms = np.mean(x * x, axis=-1)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), np.sqrt(ms / (ms + eps)), rtol=1e-14)
    g = rng.standard_normal(96)
    np.testing.assert_allclose(rmsnorm(x, g, eps), y * g, rtol=1e-14)
    # scale invariance up to eps: rmsnorm(c x) -> rmsnorm(x)
    np.testing.assert_allclose(rmsnorm(1e3 * x, g, 0.0), rmsnorm(x, g, 0.0), rtol=1e-13)


def test_silu_matches_logistic():
    z = np.linspace(-40, 40, 10001)
    np.testing.assert_allclose(silu(z), z * expit(z), rtol=1e-13, atol=1e-300)
    assert silu(np.array([0.0]))[0] == 0.0


def _rope_complex(v, pos, theta):
    """Independent form: pair (i, i+hd/2) as the complex number a + ib times e^{i pos w_i}."""
    hd = v.shape[-1]
    w = np.array([theta ** (-2.0 * i / hd) for i in range(hd // 2)])
    zc = v[..., : hd // 2] + 1j * v[..., hd // 2:]
    r = zc * np.exp(1j * np.asarray(pos)[:, None, None] * w[None, None, :])
    return np.concatenate([r.real, r.imag], axis=-1)


def test_rope_complex_form_norm_and_identity():
    rng = np.random.default_rng(2)
    v = rng.standard_normal((5, 3, 16))
    pos = np.array([0, 1, 7, 1000, 12287])
    out = rope(v, pos, 10000.0)
    np.testing.assert_allclose(out, _rope_complex(v, pos, 10000.0), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(np.linalg.norm(out, axis=-1), np.linalg.norm(v, axis=-1), rtol=1e-13)
    np.testing.assert_array_equal(rope(v[:1], np.array([0]), 10000.0), v[:1])


def test_rope_relative_position():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 1, 64))
    k = rng.standard_normal((1, 1, 64))
    for m, n, s in [(5, 2, 100), (0, 0, 4000), (17, 30, 9)]:
        a = (rope(q, np.array([m]), 1e4) * rope(k, np.array([n]), 1e4)).sum()
        b = (rope(q, np.array([m + s]), 1e4) * rope(k, np.array([n + s]), 1e4)).sum()
        assert abs(a - b) < 1e-11


@pytest.mark.parametrize("hd", [64, 128])
def test_rope_matches_rotate_half_reference(hd):
    # Llama's published rotate_half formulation, evaluated through torch in fp64
    rng = np.random.default_rng(4)
    v = rng.standard_normal((6, 2, hd))
    pos = np.arange(6) * 13
    inv = 1.0 / (10000.0 ** (torch.arange(0, hd, 2, dtype=torch.float64) / hd))
    ang = torch.outer(torch.from_numpy(pos).double(), inv)
    emb = torch.cat([ang, ang], dim=-1)[:, None, :]
    t = torch.from_numpy(v)
    rot = torch.cat([-t[..., hd // 2:], t[..., : hd // 2]], dim=-1)
    ref = (t * emb.cos() + rot * emb.sin()).numpy()
    np.testing.assert_allclose(rope(v, pos, 10000.0), ref, rtol=1e-12, atol=1e-12)
