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


BF16_ABS = 1e-5


def bf16_bad(gpu: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Elements of a bf16-stored GPU output outside the contract: more than one
    bf16 ulp from the oracle's bf16 value AND more than BF16_ABS away (near zero
    the fp32 accumulation error alone exceeds an ulp)."""
    return (bf16_ulps(gpu, ref) > 1) & (np.abs(np.asarray(gpu) - np.asarray(ref)) > BF16_ABS)


def ulp_bf16(r):
    a = np.abs(np.asarray(r, np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return 2.0 ** (e - 7)


def floor_check(gpu, ref64, ref32, bf16: bool = False, kmax: float = 2.0, kmean: float = 1.5):
    """GPU vs the fp64 oracle, judged against the noise floor |oracle_fp32 - oracle_fp64|
    of the same rounding contract.  bf16-stored outputs may also differ by one ulp."""
    gpu, ref64, ref32 = (np.asarray(a, np.float64) for a in (gpu, ref64, ref32))
    e = np.abs(gpu - ref64)
    f = np.abs(ref32 - ref64)
    slack = ulp_bf16(ref64) if bf16 else 1e-6 * float(np.abs(ref64).max())
    ok_max = bool(np.all(e <= kmax * f.max() + slack))
    ok_mean = bool(e.mean() <= kmean * f.mean() + (np.mean(slack) * 0.05 if bf16 else 1e-7))
    return ok_max and ok_mean, dict(err_max=float(e.max()), floor_max=float(f.max()),
                                    err_mean=float(e.mean()), floor_mean=float(f.mean()))


class FloorPool:
    """Pools GPU and noise-floor errors of one output kind over layers, steps and
    sequences, then applies the floor criterion once: a single rounding flip more
    or less in one small instance is chance, a systematic excess is not."""

    def __init__(self):
        self.g, self.r64, self.r32, self.bf = {}, {}, {}, {}

    def add(self, name, gpu, ref64, ref32, bf16=False):
        for d, a in ((self.g, gpu), (self.r64, ref64), (self.r32, ref32)):
            d.setdefault(name, []).append(np.asarray(a, np.float64).ravel())
        self.bf[name] = bf16

    def check(self):
        out, ok = {}, True
        for n in self.g:
            o, st = floor_check(np.concatenate(self.g[n]), np.concatenate(self.r64[n]),
                                np.concatenate(self.r32[n]), bf16=self.bf[n])
            out[n] = st
            ok &= o
        return ok, out
