"""ctypes binding of libgrpo_hip.so (declared in include/grpo_hip.h).

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels.  torch supplies device memory (tensors on ``cuda``) and the
stream; nothing here computes.  The functions keep the C names without the
``grpo_`` prefix and raise ``GrpoError`` on a negative status.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
import torch

from .workloads import DTYPE_F32, ModelConfig

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgrpo_hip.so")

OK, INVALID_ARG, UNSUPPORTED, WORKSPACE_TOO_SMALL, HIP_ERROR, KV_CAPACITY = 0, -1, -2, -3, -4, -5
OP_PREFILL, OP_ROLLOUT, OP_SCORE, OP_LOSS, OP_EXTEND, OP_BACKWARD = 0, 1, 2, 3, 4, 5
EXTEND_CHUNK = 512


class GrpoError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"grpo status {code}: {msg}")
        self.code = code


class Config(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("d_ffn", C.c_int32),
                ("vocab", C.c_int32), ("rms_eps", C.c_float), ("rope_theta", C.c_float),
                ("dtype", C.c_int32)]


_PP = C.POINTER(C.c_void_p)


class Weights(C.Structure):
    _fields_ = [("tok_emb", C.c_void_p), ("attn_norm", _PP), ("wq", _PP), ("wk", _PP),
                ("wv", _PP), ("wo", _PP), ("mlp_norm", _PP), ("w_gate", _PP), ("w_up", _PP),
                ("w_down", _PP), ("final_norm", C.c_void_p), ("lm_head", C.c_void_p)]


class GradsStruct(C.Structure):
    _fields_ = Weights._fields_


class AdamW(C.Structure):
    _fields_ = [("lr", C.c_float), ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float),
                ("weight_decay", C.c_float)]


class Sampling(C.Structure):
    _fields_ = [("temperature", C.c_float), ("top_k", C.c_int32), ("seed", C.c_uint64)]


TRACE_FIELDS = ("x", "x_attn", "h_attn", "q", "k", "v", "o", "h_mlp", "act", "h_final", "logits")


class TraceStruct(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in TRACE_FIELDS]


class Trace:
    """Device buffers of a grpo_trace for a call with `rows` forward rows and
    `head_rows` LM-head rows (see include/grpo_hip.h), filled with NaN so that
    rows a call leaves unwritten stay recognisable."""

    def __init__(self, cfg: ModelConfig, rows: int, head_rows: int, fields=TRACE_FIELDS,
                 device="cuda"):
        L, d, f = cfg.n_layers, cfg.d_model, cfg.d_ffn
        shapes = dict(x=(L + 1, rows, d), x_attn=(L, rows, d), h_attn=(L, rows, d),
                      q=(L, rows, cfg.q_dim), k=(L, rows, cfg.kv_dim), v=(L, rows, cfg.kv_dim),
                      o=(L, rows, cfg.q_dim), h_mlp=(L, rows, d), act=(L, rows, f),
                      h_final=(head_rows, d), logits=(head_rows, cfg.vocab))
        self.t = {n: torch.full(shapes[n], float("nan"), dtype=torch.float32, device=device)
                  for n in fields}
        self._s = TraceStruct(*[_ptr(self.t.get(n)) for n in TRACE_FIELDS])

    def struct(self):
        return C.byref(self._s)

    def numpy(self) -> dict:
        return {n: t.cpu().numpy().astype(np.float64) for n, t in self.t.items()}

    def lazy(self) -> dict:
        """Members that copy only the rows they are indexed with to the host:
        lazy()["x"][layer][rows] -> float64 array."""
        return {n: _LazyMember(t) for n, t in self.t.items()}


class _LazyMember:
    def __init__(self, t):
        self.t = t

    def __getitem__(self, i):
        if self.t.dim() == 3 and isinstance(i, (int, np.integer)):
            return _LazyMember(self.t[int(i)])
        if isinstance(i, slice):
            return self.t[i].cpu().numpy().astype(np.float64)
        idx = torch.as_tensor(np.asarray(i), device=self.t.device, dtype=torch.long)
        return self.t[idx].cpu().numpy().astype(np.float64)


def _trace(tr):
    return tr.struct() if tr is not None else None


def _ids(seq_ids, B):
    if seq_ids is None:
        return None
    a = np.ascontiguousarray(np.asarray(seq_ids, np.int32).ravel())
    if a.size != B:
        raise ValueError(f"seq_ids has {a.size} entries, the batch {B}")
    return (C.c_int32 * B)(*a.tolist())


_lib = None

_VP, _I32, _F32, _SZ = C.c_void_p, C.c_int32, C.c_float, C.c_size_t
_IP = C.POINTER(C.c_int32)
_TP = C.POINTER(TraceStruct)
_SIGS = {
    "grpo_model_create": (_I32, [C.POINTER(Config), C.POINTER(Weights), C.POINTER(_VP)]),
    "grpo_model_destroy": (_I32, [_VP]),
    "grpo_decode_weights_bytes": (_SZ, [C.POINTER(Config)]),
    "grpo_model_pack_decode": (_I32, [_VP, _VP, _SZ, _VP]),
    "grpo_kv_cache_bytes": (_SZ, [C.POINTER(Config), _I32, _I32]),
    "grpo_workspace_bytes": (_SZ, [_VP, _I32, _I32, _I32]),
    "grpo_last_error": (C.c_char_p, []),
    "grpo_prefill": (_I32, [_VP, _VP, _I32, _I32, _VP, _I32, _I32, _I32, C.POINTER(Sampling),
                            _VP, _VP, _TP, _VP, _SZ, _VP]),
    "grpo_rollout_step": (_I32, [_VP, _VP, _I32, _I32, _I32, _IP, _VP, _VP, _I32, _I32, _I32,
                                 C.POINTER(Sampling), _VP, _VP, _TP, _VP, _SZ, _VP]),
    "grpo_rollout_step_grouped": (_I32, [_VP, _VP, _I32, _I32, _I32, _I32, _I32, _IP, _VP, _VP,
                                         _I32, _I32, _I32, C.POINTER(Sampling), _VP, _VP, _TP,
                                         _VP, _SZ, _VP]),
    "grpo_extend": (_I32, [_VP, _VP, _I32, _I32, _I32, _IP, _IP, _VP, _I32, _I32,
                           C.POINTER(Sampling), _VP, _VP, _TP, _VP, _SZ, _VP]),
    "grpo_score_sequences": (_I32, [_VP, _VP, _I32, _I32, _I32, _F32, _VP, _TP, _VP, _SZ, _VP]),
    "grpo_score_sequences_grouped": (_I32, [_VP, _VP, _I32, _I32, _I32, _F32, _I32, _I32, _VP,
                                            _TP, _VP, _SZ, _VP]),
    "grpo_advantages": (_I32, [_VP, _I32, _I32, _F32, _VP, _VP]),
    "grpo_token_loss": (_I32, [_VP, _VP, _VP, _VP, _VP, _I32, _I32, _F32, _F32, _I32, _VP, _VP,
                               _VP, _VP, _VP, _SZ, _VP]),
    "grpo_decode_structure": (_I32, [_VP, _I32, _I32, _I32, _I32, _IP]),
    "grpo_token_loss_noalloc": (_I32, [_VP, _VP, _VP, _VP, _VP, _I32, _I32, _F32, _F32, _I32, _VP,
                                       _VP, _VP, _VP, _VP]),
    "grpo_reward": (_I32, [_VP, _VP, _VP, _VP, _VP, _I32, _VP]),
    "grpo_sft_loss": (_I32, [_VP, _VP, _I32, _I32, _I32, _VP, _VP, _VP, _SZ, _VP]),
    "grpo_exact_kl": (_I32, [_VP, _VP, _I32, _I32, _I32, _F32, _VP, _VP]),
    "grpo_policy_backward": (_I32, [_VP, _VP, _I32, _I32, _I32, _F32, _VP, C.POINTER(GradsStruct),
                                     _VP, _SZ, _VP]),
    "grpo_adamw_step": (_I32, [_I32, _VP, _VP, _VP, _VP, _VP, _SZ, C.POINTER(AdamW), _I32, _VP]),
    "grpo_profile_begin": (_I32, []),
    "grpo_profile_end": (_I32, [C.c_char_p, _SZ]),
}


def lib() -> C.CDLL:
    """The in-tree HIP library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} missing: run __graft_entry__.build() first")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _lib = L
    return _lib


def _check(rc: int):
    if rc != OK:
        raise GrpoError(rc, lib().grpo_last_error().decode())


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, torch.Tensor):
        if t.device.type != "cuda":
            raise ValueError("device tensors only")
        if not t.is_contiguous():
            raise ValueError("contiguous tensors only")
        return t.data_ptr()
    return int(t)


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return int(getattr(stream, "cuda_stream", stream))


def config_struct(cfg: ModelConfig) -> Config:
    return Config(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ffn,
                  cfg.vocab, cfg.rms_eps, cfg.rope_theta, cfg.dtype)


def upload_weights(cfg: ModelConfig, host: dict, device="cuda") -> dict:
    """Host weights (uint16 bf16 bits or float32) -> device tensors of the model dtype."""
    out = {}
    for k, a in host.items():
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
        else:
            t = torch.from_numpy(a.astype(np.float32, copy=False))
        out[k] = t.to(device, non_blocking=False)
    return out


class Model:
    """A model handle over device weight tensors (which it keeps alive).

    ``decode=True`` (bf16 models) also allocates the decode copy of the
    projections and has the library pack it (``grpo_model_pack_decode``), which
    ``rollout_step`` needs; a model that is only scored can skip it.  Call
    ``pack_decode()`` again after changing the weights in place.
    """

    def __init__(self, cfg: ModelConfig, weights: dict, decode: bool = True):
        self.cfg = cfg
        self.weights = weights
        L = cfg.n_layers

        def arr(t):
            a = (C.c_void_p * L)(*[_ptr(weights[f"l{i}.{t}"]) for i in range(L)])
            return a

        self._arrays = {t: arr(t) for t in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm",
                                            "w_gate", "w_up", "w_down")}
        cast = lambda a: C.cast(a, _PP)  # noqa: E731
        w = Weights(_ptr(weights["tok_emb"]), *[cast(self._arrays[t]) for t in (
            "attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")],
            _ptr(weights["final_norm"]), _ptr(weights["lm_head"]))
        self._cfg_s = config_struct(cfg)
        h = C.c_void_p()
        _check(lib().grpo_model_create(C.byref(self._cfg_s), C.byref(w), C.byref(h)))
        self.handle = h
        self.decode_weights = None
        if decode:
            n = lib().grpo_decode_weights_bytes(C.byref(self._cfg_s))
            if n:
                self.decode_weights = torch.empty(n, dtype=torch.uint8, device="cuda")
                self.pack_decode()

    def pack_decode(self, stream=None):
        t = self.decode_weights
        if t is not None:
            _check(lib().grpo_model_pack_decode(self.handle, _ptr(t), t.numel(), _stream(stream)))

    def close(self):
        if getattr(self, "handle", None):
            lib().grpo_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def act_dtype(self):
        return torch.float32 if self.cfg.dtype == DTYPE_F32 else torch.bfloat16


def kv_cache_bytes(cfg: ModelConfig, n_seqs: int, max_len: int) -> int:
    return lib().grpo_kv_cache_bytes(C.byref(config_struct(cfg)), n_seqs, max_len)


def workspace_bytes(model: Model | None, op: int, n_rows: int, seq_len: int) -> int:
    return lib().grpo_workspace_bytes(model.handle if model else None, op, n_rows, seq_len)


def alloc_workspace(model: Model | None, op: int, n_rows: int, seq_len: int, device="cuda"):
    n = workspace_bytes(model, op, n_rows, seq_len)
    if n == 0:
        raise GrpoError(INVALID_ARG, "workspace size query failed")
    return torch.empty(n, dtype=torch.uint8, device=device)


def alloc_kv(cfg: ModelConfig, n_seqs: int, max_len: int, device="cuda"):
    n = kv_cache_bytes(cfg, n_seqs, max_len)
    if n == 0:
        raise GrpoError(INVALID_ARG, "kv size query failed")
    return torch.empty(n, dtype=torch.uint8, device=device)


def prefill(model: Model, kv, n_seqs: int, max_len: int, prompts, G: int, sampling: Sampling,
            tok_out, logp_out, trace: Trace | None = None, ws=None, stream=None):
    P, Tp = prompts.shape
    _check(lib().grpo_prefill(model.handle, _ptr(kv), n_seqs, max_len, _ptr(prompts), P, Tp, G,
                              C.byref(sampling), _ptr(tok_out), _ptr(logp_out), _trace(trace),
                              _ptr(ws), ws.numel() if ws is not None else 0, _stream(stream)))


def rollout_step(model: Model, kv, n_seqs: int, max_len: int, pos, tok, max_pos: int, step0: int,
                 n_steps: int, sampling: Sampling, tok_out, logp_out, seq_ids=None,
                 trace: Trace | None = None, ws=None, stream=None, group: int = 0,
                 prefix_len: int = 0):
    """grpo_rollout_step, or grpo_rollout_step_grouped when group > 0 (rows in
    groups of `group` sharing cache positions below prefix_len).  seq_ids: host
    sequence of B ints (cache slot and Philox sequence id of each row) or None."""
    B = pos.numel()
    nws = ws.numel() if ws is not None else 0
    ids = _ids(seq_ids, B)
    if group > 0:
        _check(lib().grpo_rollout_step_grouped(
            model.handle, _ptr(kv), n_seqs, max_len, B, group, prefix_len, ids, _ptr(pos),
            _ptr(tok), max_pos, step0, n_steps, C.byref(sampling), _ptr(tok_out), _ptr(logp_out),
            _trace(trace), _ptr(ws), nws, _stream(stream)))
        return
    _check(lib().grpo_rollout_step(model.handle, _ptr(kv), n_seqs, max_len, B, ids, _ptr(pos),
                                   _ptr(tok), max_pos, step0, n_steps, C.byref(sampling),
                                   _ptr(tok_out), _ptr(logp_out), _trace(trace), _ptr(ws), nws,
                                   _stream(stream)))


def extend(model: Model, kv, n_seqs: int, max_len: int, pos0, tokens, step: int,
           sampling: Sampling, tok_out, logp_out, seq_ids=None, trace: Trace | None = None,
           ws=None, stream=None):
    """grpo_extend: tokens [B, Te] (device) injected at host positions pos0[b] of
    sequences seq_ids[b] (host, None: b); the next token of each row drawn at `step`."""
    B, Te = tokens.shape
    _check(lib().grpo_extend(model.handle, _ptr(kv), n_seqs, max_len, B, _ids(seq_ids, B),
                             _ids(pos0, B), _ptr(tokens), Te, step, C.byref(sampling),
                             _ptr(tok_out), _ptr(logp_out), _trace(trace), _ptr(ws),
                             ws.numel() if ws is not None else 0, _stream(stream)))


def score_sequences(model: Model, tokens, score_from: int, temperature: float, logp_out,
                    trace: Trace | None = None, ws=None, stream=None, group: int = 0,
                    prefix_len: int = 0):
    """grpo_score_sequences, or grpo_score_sequences_grouped when group > 0 (rows in
    groups of `group` sharing their first prefix_len tokens)."""
    N, T = tokens.shape
    nws = ws.numel() if ws is not None else 0
    if group > 0:
        _check(lib().grpo_score_sequences_grouped(model.handle, _ptr(tokens), N, T, score_from,
                                                  temperature, group, prefix_len, _ptr(logp_out),
                                                  _trace(trace), _ptr(ws), nws, _stream(stream)))
        return
    _check(lib().grpo_score_sequences(model.handle, _ptr(tokens), N, T, score_from, temperature,
                                      _ptr(logp_out), _trace(trace), _ptr(ws), nws,
                                      _stream(stream)))


def advantages(rewards, P: int, G: int, eps: float, adv_out, stream=None):
    _check(lib().grpo_advantages(_ptr(rewards), P, G, eps, _ptr(adv_out), _stream(stream)))


def token_loss(logp, logp_old, logp_ref, mask, adv, clip_eps: float, beta: float, agg: int,
               loss_out, tok_loss=None, dloss_dlogp=None, stats=None, ws=None, stream=None):
    N, Tr = logp.shape
    _check(lib().grpo_token_loss(_ptr(logp), _ptr(logp_old), _ptr(logp_ref), _ptr(mask), _ptr(adv),
                                 N, Tr, clip_eps, beta, agg, _ptr(loss_out), _ptr(tok_loss),
                                 _ptr(dloss_dlogp), _ptr(stats), _ptr(ws),
                                 ws.numel() if ws is not None else 0, _stream(stream)))


def decode_structure(model: Model, B: int, max_len: int, G: int = 0, prefix_len: int = 0) -> dict:
    """grpo_decode_structure as a dict."""
    out = (C.c_int32 * 9)()
    _check(lib().grpo_decode_structure(model.handle, B, max_len, G, prefix_len, out))
    v = list(out)
    return dict(splits_qkv=v[0], splits_o=v[1], splits_down=v[2], splits_head=v[3], span=v[4],
                spans=v[5], chunk=v[6], chunks=v[7], waves=v[8])


def token_loss_noalloc(logp, logp_old, logp_ref, mask, adv, clip_eps: float, beta: float,
                       agg: int, loss_out, tok_loss=None, dloss_dlogp=None, stats=None,
                       stream=None):
    """grpo_token_loss_noalloc: grpo_token_loss with the library's static scratch."""
    N, Tr = logp.shape
    _check(lib().grpo_token_loss_noalloc(_ptr(logp), _ptr(logp_old), _ptr(logp_ref), _ptr(mask),
                                         _ptr(adv), N, Tr, clip_eps, beta, agg, _ptr(loss_out),
                                         _ptr(tok_loss), _ptr(dloss_dlogp), _ptr(stats),
                                         _stream(stream)))


def reward(correct, t_base, t, tools_used, tools_avail) -> np.ndarray:
    """grpo_reward on host arrays; returns fp32 rewards."""
    c = np.ascontiguousarray(np.asarray(correct, np.uint8))
    tb = np.ascontiguousarray(np.asarray(t_base, np.float64))
    tt = np.ascontiguousarray(np.asarray(t, np.float64))
    u = np.ascontiguousarray(np.asarray(tools_used, np.int32))
    a = np.ascontiguousarray(np.asarray(tools_avail, np.int32))
    out = np.empty(c.size, np.float32)
    _check(lib().grpo_reward(c.ctypes.data, tb.ctypes.data, tt.ctypes.data, u.ctypes.data,
                             a.ctypes.data, c.size, out.ctypes.data))
    return out


def sft_loss(logp, mask, agg: int, loss_out, dloss_dlogp=None, ws=None, stream=None):
    N, Tr = logp.shape
    _check(lib().grpo_sft_loss(_ptr(logp), _ptr(mask), N, Tr, agg, _ptr(loss_out),
                               _ptr(dloss_dlogp), _ptr(ws), ws.numel() if ws is not None else 0,
                               _stream(stream)))


def exact_kl(logits, logits_ref, temperature: float, kl_out, stream=None):
    R, V = logits.shape
    _check(lib().grpo_exact_kl(_ptr(logits), _ptr(logits_ref), R, V, V, temperature,
                               _ptr(kl_out), _stream(stream)))


def profile_begin():
    _check(lib().grpo_profile_begin())


def profile_end() -> dict:
    """Per-kernel {name: (launches, total_ms)} since profile_begin()."""
    import json
    buf = C.create_string_buffer(1 << 16)
    _check(lib().grpo_profile_end(buf, len(buf)))
    return {k: tuple(v) for k, v in json.loads(buf.value.decode()).items()}


# ---- gradient step ------------------------------------------------------------------
WEIGHT_NAMES_LAYER = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")


class Grads:
    """fp32 gradient accumulators shaped like a model's weights (zeroed).  Each
    layer's q, k and v gradients are views of one buffer in that order, and so
    are its gate and up gradients: the backward then forms each group's weight
    gradient in a single product."""

    GROUPS = (("wq", "wk", "wv"), ("w_gate", "w_up"))

    def __init__(self, model: "Model"):
        L = model.cfg.n_layers
        self.t = {}
        for i in range(L):
            for grp in self.GROUPS:
                names = [f"l{i}.{n}" for n in grp]
                ws = [model.weights[n] for n in names]
                flat = torch.zeros(sum(w.numel() for w in ws), dtype=torch.float32,
                                   device=ws[0].device)
                off = 0
                for n, w in zip(names, ws):
                    self.t[n] = flat[off:off + w.numel()].view(w.shape)
                    off += w.numel()
        for k, v in model.weights.items():
            if k not in self.t:
                self.t[k] = torch.zeros(v.shape, dtype=torch.float32, device=v.device)
        self._arrays = {n: (C.c_void_p * L)(*[_ptr(self.t[f"l{i}.{n}"]) for i in range(L)])
                        for n in WEIGHT_NAMES_LAYER}
        self.struct = GradsStruct(_ptr(self.t["tok_emb"]),
                                  *[C.cast(self._arrays[n], _PP) for n in WEIGHT_NAMES_LAYER],
                                  _ptr(self.t["final_norm"]), _ptr(self.t["lm_head"]))

    def zero_(self):
        for v in self.t.values():
            v.zero_()


def policy_backward(model: "Model", tokens, score_from: int, temperature: float, dlogp,
                    grads: Grads, ws=None, stream=None):
    """grpo_policy_backward: tokens int32 [N, T], dlogp fp32 [N, T - score_from] (device)."""
    N, T = tokens.shape
    if ws is None:
        ws = alloc_workspace(model, OP_BACKWARD, N, T)
    _check(lib().grpo_policy_backward(model.handle, _ptr(tokens), N, T, score_from, temperature,
                                      _ptr(dlogp), C.byref(grads.struct), _ptr(ws), ws.numel(),
                                      _stream(stream)))


def adamw_step(dtype: int, param, master, m, v, grad, lr: float, beta1: float, beta2: float,
               eps: float, weight_decay: float, step: int, stream=None):
    """grpo_adamw_step over one tensor (master None for fp32 parameters)."""
    hp = AdamW(lr, beta1, beta2, eps, weight_decay)
    _check(lib().grpo_adamw_step(dtype, _ptr(param), _ptr(master) if master is not None else None,
                                 _ptr(m), _ptr(v), _ptr(grad), grad.numel(), C.byref(hp), step,
                                 _stream(stream)))
