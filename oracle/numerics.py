"""Elementwise building blocks of the decoder, in fp64.

The paper's policy is a Llama3 decoder (Sec. VI-C); these are that family's
published definitions: RMSNorm, the SiLU-gated MLP and rotary position
embeddings with the half-split pairing (i, i + hd/2).

bf16 rounding: the bf16 models keep weights in bf16 and round a few
activations to bf16 before they enter a matrix product (the precision
contract).  ``round_bf16`` is round-to-nearest-even of the value's fp32
rounding, written out on the bit pattern.
"""
from __future__ import annotations

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns -> float64 (exact)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):
        return u.view(np.float32).astype(np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bf16 value (ties to even), via fp32; returns float64."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    b = f.view(np.uint32).astype(np.uint64)
    lsb = (b >> np.uint64(16)) & np.uint64(1)
    r = (b + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    nan = np.isnan(f)
    r = np.where(nan, (b >> np.uint64(16)) | np.uint64(0x40), r)
    return bf16_bits_to_f64((r & np.uint64(0xFFFF)).astype(np.uint16))


def _float(x) -> np.ndarray:
    return np.asarray(x, np.float64)


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = _float(x)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + float(eps)) * np.asarray(g, x.dtype)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def rope_angles(pos: np.ndarray, head_dim: int, theta: float) -> np.ndarray:
    """[len(pos), hd/2] rotation angles pos * theta^(-2i/hd)."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv = theta ** (-2.0 * i / head_dim)
    return np.asarray(pos, np.float64)[:, None] * inv[None, :]


def rope(v: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate [T, n_heads, hd] vectors at positions pos[T], half-split pairing.

    Angles, cos, sin and the rotation are fp64."""
    v = _float(v)
    hd = v.shape[-1]
    a = rope_angles(pos, hd, theta)[:, None, :]
    c, s = np.cos(a).astype(v.dtype), np.sin(a).astype(v.dtype)
    lo, hi = v[..., : hd // 2], v[..., hd // 2:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)
