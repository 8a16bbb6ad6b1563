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


def floor_check(gpu, ref64, refs32, bf16: bool = False, kmax: float = 3.0, kmean: float = 2.5,
                allow=None):
    """GPU vs the fp64 oracle, judged against the noise floor of the same rounding
    contract: the larger elementwise distance from fp64 of the fp32 evaluations
    in `refs32` (BLAS order and matrix-core order).  fp32 outputs: max and mean
    within kmax / kmean of the floor.  bf16-stored outputs: every element within
    kmax floor maxima plus one ulp, and no more than kmax times the floor's
    fraction of differing elements (at least 2e-3).  `allow` (bf16 outputs) adds a
    per-element allowance, e.g. the reach of rounding flips of an input that the
    rounding contract leaves open (see h_flip_allowance)."""
    gpu, ref64 = (np.asarray(a, np.float64) for a in (gpu, ref64))
    if not isinstance(refs32, (list, tuple)):
        refs32 = [refs32]
    e = np.abs(gpu - ref64)
    f = np.max([np.abs(np.asarray(r, np.float64) - ref64) for r in refs32], axis=0)
    st = dict(err_max=float(e.max()), floor_max=float(f.max()), err_mean=float(e.mean()),
              floor_mean=float(f.mean()))
    if bf16:
        ulp = ulp_bf16(ref64)
        extra = 0.0 if allow is None else np.asarray(allow, np.float64)
        bad = e > kmax * f.max() + ulp + extra
        ok = not bool(bad.any())
        frac, ffrac = float((e > 0).mean()), float((f > 0).mean())
        st.update(flip_frac=frac, floor_flip_frac=ffrac)
        if not ok:
            idx = np.argsort(-(e - ulp))[:4]
            st["worst"] = [dict(i=int(i), gpu=float(gpu[i]), ref=float(ref64[i]), err=float(e[i]),
                                ulp=float(ulp[i]), floor=float(f[i])) for i in idx]
        return ok and frac <= max(kmax * ffrac, 2e-3), st
    slack = 1e-6 * float(np.abs(ref64).max())
    ok = bool(e.max() <= kmax * f.max() + slack) and bool(e.mean() <= kmean * f.mean() + 1e-7)
    return ok, st


class FloorPool:
    """Pools GPU and noise-floor errors of one output kind over layers, steps and
    sequences, then applies the floor criterion once: a single rounding flip more
    or less in one small instance is chance, a systematic excess is not."""

    def __init__(self):
        self.g, self.r64, self.r32, self.bf, self.al = {}, {}, {}, {}, {}

    def add(self, name, gpu, ref64, refs32, bf16=False, allow=None):
        if not isinstance(refs32, (list, tuple)):
            refs32 = [refs32]
        a = np.zeros(np.size(gpu)) if allow is None else np.asarray(allow, np.float64).ravel()
        self.al.setdefault(name, []).append(a)
        self.g.setdefault(name, []).append(np.asarray(gpu, np.float64).ravel())
        self.r64.setdefault(name, []).append(np.asarray(ref64, np.float64).ravel())
        self.r32.setdefault(name, []).append([np.asarray(r, np.float64).ravel() for r in refs32])
        self.bf[name] = bf16

    def check(self):
        out, ok = {}, True
        for n in self.g:
            refs = [np.concatenate([r[i] for r in self.r32[n]]) for i in range(len(self.r32[n][0]))]
            o, st = floor_check(np.concatenate(self.g[n]), np.concatenate(self.r64[n]), refs,
                                bf16=self.bf[n], allow=np.concatenate(self.al[n]))
            out[n] = st
            ok &= o
        return ok, out


def h_flip_allowance(om, cfg, l, x, rel=4e-6):
    """Per-element reach of rounding flips of the normed attention input of layer l
    on its K and V outputs.  h = R1(rms(x) g) is rounded to bf16; where the fp64
    value of an element lies within `rel` (relative) of a rounding midpoint, an
    fp32 evaluation of the norm (relative error below 1e-6 at these widths) may
    round it either way, moving every K/V output j by up to sum_i |W[j, i]| ulp(h_i)
    over those elements (K: also its RoPE partner dimension).
    x: [..., d] residual fed to the layer; returns (allow_k, allow_v) [..., n_kv, hd]."""
    import oracle
    x = np.asarray(x, np.float64)
    h = oracle.rmsnorm(x, om.mat(f"l{l}.attn_norm"), cfg.rms_eps)
    r = oracle.round_bf16(h)
    a, ar = np.abs(h), np.abs(r)
    u = ulp_bf16(r)
    pow2 = ar == 2.0 ** np.floor(np.log2(np.maximum(ar, 2.0 ** -126)))
    half = np.where(a >= ar, u / 2, np.where(pow2, u / 4, u / 2))   # to the midpoint beyond h
    near = (half - np.abs(a - ar)) <= rel * a
    dh = np.where(near, u, 0.0)
    hd, hk = cfg.head_dim, cfg.n_kv_heads
    lead = x.shape[:-1]
    ak = (dh @ np.abs(om.mat(f"l{l}.wk")).T).reshape(*lead, hk, hd)
    ak = ak + np.roll(ak, hd // 2, axis=-1)
    av = (dh @ np.abs(om.mat(f"l{l}.wv")).T).reshape(*lead, hk, hd)
    return ak, av
