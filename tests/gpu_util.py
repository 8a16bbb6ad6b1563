"""Shared set-up of the GPU parity tests (not collected: no test_ prefix)."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

from paper_2510_17158_amd import api, synth
from paper_2510_17158_amd.workloads import DTYPE_F32, ModelConfig


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    api.lib()   # fails loudly if the HIP library is missing


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def build_model(cfg: ModelConfig, seed: int, gain_noise: float = 0.1, ref: bool = False,
                std: float = 0.02):
    host = synth.make_weights(cfg, seed, gain_noise=gain_noise, ref=ref, std=std)
    dev = api.upload_weights(cfg, host)
    return host, api.Model(cfg, dev)


def kv_view(cfg: ModelConfig, kv: torch.Tensor, n_seqs: int, max_len: int) -> np.ndarray:
    """KV buffer -> float64 array [L, 2, n_seqs, n_kv, max_len, hd]."""
    shape = (cfg.n_layers, 2, n_seqs, cfg.n_kv_heads, max_len, cfg.head_dim)
    if cfg.dtype == DTYPE_F32:
        return kv.view(torch.float32).view(shape).double().cpu().numpy()
    return kv.view(torch.bfloat16).view(shape).double().cpu().numpy()


def bf16_ulps(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Distance in bf16 units in the last place between bf16-representable values."""
    def key(x):
        u = (np.asarray(x, np.float32).view(np.uint32) >> 16).astype(np.int64)
        return np.where(u & 0x8000, -(u & 0x7FFF), u)
    return np.abs(key(a) - key(b))
