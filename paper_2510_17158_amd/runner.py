"""One GRPO iteration's hot path through the C-ABI (Alg. 1 minus the update).

  prefill          prompt forward once per prompt, first token of each of the
                   G group members (generation step 0)
  rollout_step     the remaining new_tokens - 1 batched decode steps
  score_sequences  teacher-forced log-probs of the sampled completions under
                   the policy and under the frozen reference
  advantages       group-normalised rewards
  token_loss       clipped-ratio + KL loss and its gradient w.r.t. logp

torch only allocates buffers and moves tokens between them; every arithmetic
step is a library kernel.
"""
from __future__ import annotations

import numpy as np
import torch

from . import api
from .workloads import Workload


class GrpoIteration:
    def __init__(self, w: Workload, policy: api.Model, ref: api.Model | None, prompts: np.ndarray,
                 rewards: np.ndarray, seed: int, device="cuda", mask: np.ndarray | None = None):
        self.w = w
        self.policy, self.ref = policy, ref
        cfg = w.model
        P, G, Tp, Tn = w.n_prompts, w.group, w.prompt_len, w.new_tokens
        B = P * G
        self.B, self.T = B, Tp + Tn
        self.max_len = max(w.max_len, Tp)
        dev = device
        i32 = dict(dtype=torch.int32, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        self.sampling = api.Sampling(w.temperature, w.top_k, seed)
        self.prompts = torch.from_numpy(np.ascontiguousarray(prompts, np.int32)).to(dev)
        self.kv = api.alloc_kv(cfg, B, self.max_len, dev)
        self.ws_prefill = api.alloc_workspace(policy, api.OP_PREFILL, P, Tp, dev)
        self.ws_roll = api.alloc_workspace(policy, api.OP_ROLLOUT, B, self.max_len, dev)
        self.ws_score = (api.alloc_workspace(policy, api.OP_SCORE, B, self.T, dev)
                         if w.score else None)
        self.ws_loss = api.alloc_workspace(None, api.OP_LOSS, B, Tn, dev)
        self.tok0 = torch.empty(B, **i32)
        self.logp0 = torch.empty(B, **f32)
        self.tok = torch.empty(B, **i32)
        self.pos = torch.empty(B, **i32)
        n_dec = max(Tn - 1, 1)
        self.tok_dec = torch.empty(B, n_dec, **i32)
        self.logp_dec = torch.empty(B, n_dec, **f32)
        self.seqs = torch.empty(B, self.T, **i32)
        self.logp_old = torch.empty(B, Tn, **f32)
        self.lp_pol = torch.empty(B, Tn, **f32)
        self.lp_ref = torch.empty(B, Tn, **f32)
        self.rewards = torch.from_numpy(np.ascontiguousarray(rewards, np.float32)).to(dev)
        self.adv = torch.empty(B, **f32)
        m = np.ones((B, Tn), np.uint8) if mask is None else mask
        self.mask = torch.from_numpy(np.ascontiguousarray(m, np.uint8)).to(dev)
        self.loss = torch.empty(1, **f32)
        self.tok_loss = torch.empty(B, Tn, **f32)
        self.dloss = torch.empty(B, Tn, **f32)
        self.stats = torch.empty(4, **f32)

    # --- phases -----------------------------------------------------------------------
    def prefill(self, trace=None):
        w = self.w
        api.prefill(self.policy, self.kv, self.B, self.max_len, self.prompts, w.group,
                    self.sampling, self.tok0, self.logp0, trace=trace, ws=self.ws_prefill)

    def decode(self, trace=None):
        """Generation steps 1 .. new_tokens-1 for the whole batch."""
        w = self.w
        n = w.new_tokens - 1
        if n <= 0:
            return
        self.tok.copy_(self.tok0)
        self.pos.fill_(w.prompt_len)
        api.rollout_step(self.policy, self.kv, self.B, self.max_len, self.pos, self.tok,
                         w.prompt_len, 1, n, self.sampling, self.tok_dec, self.logp_dec,
                         trace=trace, ws=self.ws_roll,
                         group=w.group if w.shared_prompt else 0,
                         prefix_len=w.prompt_len if w.shared_prompt else 0)

    def assemble(self):
        """Sequences [B, Tp + Tn] and rollout log-probs [B, Tn] from the phase outputs."""
        w = self.w
        G, Tp, Tn = w.group, w.prompt_len, w.new_tokens
        self.seqs[:, :Tp] = self.prompts.repeat_interleave(G, dim=0)
        self.seqs[:, Tp] = self.tok0
        self.logp_old[:, 0] = self.logp0
        if Tn > 1:
            self.seqs[:, Tp + 1:] = self.tok_dec
            self.logp_old[:, 1:] = self.logp_dec

    def score(self):
        w = self.w
        grp = dict(group=w.group, prefix_len=w.prompt_len) if w.shared_prompt else {}
        api.score_sequences(self.policy, self.seqs, w.prompt_len, w.temperature, self.lp_pol,
                            ws=self.ws_score, **grp)
        if self.ref is not None:
            api.score_sequences(self.ref, self.seqs, w.prompt_len, w.temperature, self.lp_ref,
                                ws=self.ws_score, **grp)

    def grpo(self):
        w = self.w
        api.advantages(self.rewards, w.n_prompts, w.group, w.adv_eps, self.adv)
        lp_ref = self.lp_ref if self.ref is not None else self.lp_pol
        api.token_loss(self.lp_pol, self.logp_old, lp_ref, self.mask, self.adv, w.clip_eps,
                       w.beta, 0, self.loss, self.tok_loss, self.dloss, self.stats,
                       ws=self.ws_loss)

    def update(self, lr: float = 1e-5, beta1: float = 0.9, beta2: float = 0.95,
               eps: float = 1e-8, weight_decay: float = 0.0, micro_batch: int = 1):
        """The gradient step that closes the iteration (Alg. 1): the policy's
        weight gradient of the token loss (grpo_policy_backward over the batch,
        micro_batch sequences per call, dL/dlogp from grpo()), then AdamW on fp32
        master weights (created on the first call) and a repack of the decode
        copy.  Returns the step number."""
        w, pol = self.w, self.policy
        if not hasattr(self, "_opt"):
            self._opt = {k: (v.float() if w.model.dtype == 1 else None,
                             torch.zeros(v.shape, dtype=torch.float32, device=v.device),
                             torch.zeros(v.shape, dtype=torch.float32, device=v.device))
                         for k, v in pol.weights.items()}
            self._grads = api.Grads(pol)
            self._ws_bwd = api.alloc_workspace(pol, api.OP_BACKWARD, micro_batch, self.T)
            self._step = 0
        self._grads.zero_()
        for n0 in range(0, self.B, micro_batch):
            n1 = min(self.B, n0 + micro_batch)
            api.policy_backward(pol, self.seqs[n0:n1], w.prompt_len, w.temperature,
                                self.dloss[n0:n1], self._grads, ws=self._ws_bwd)
        self._step += 1
        for k, v in pol.weights.items():
            mst, m1, m2 = self._opt[k]
            api.adamw_step(w.model.dtype, v, mst, m1, m2, self._grads.t[k], lr=lr, beta1=beta1,
                           beta2=beta2, eps=eps, weight_decay=weight_decay, step=self._step)
        pol.pack_decode()
        return self._step

    def run(self):
        """One full pass of the hot path."""
        self.prefill()
        self.decode()
        self.assemble()
        if self.w.score:
            self.score()
        else:
            self.lp_pol.copy_(self.logp_old)
        self.grpo()
