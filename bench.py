#!/usr/bin/env python3
"""GRPO hot-path benchmark on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
prompt prefill + G-sample decode (the rollout), teacher-forced scoring of the
completions under the policy and the frozen reference, group advantages and the
clipped-ratio + KL token loss.  Prints ONE JSON line.

  value      sampled (rollout) tokens per second of whole steps
  roofline   the dominant kernel's algorithmic bytes / its measured duration
  cpu_baseline  the CPU oracle on a bounded sample of the same workload
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0

# HBM bytes of the per-row decode attention kernel of a grouped step (the generated
# positions of every sequence, the prompt chunks' partials merged in) from rocprofv3
# FETCH_SIZE / WRITE_SIZE runs at the 7B shape (64 sequences, 2048-token prompt shared
# per group of 8, 1 .. 48 generated positions; 32 launches per position count), each
# counter scaled by what it reads for a 1 GiB device copy.  The fetch per launch fits
# fixed + per_position x (generated positions): the fixed part is mostly the prompt
# chunks' partial rows.  Valid only for the kernel source it was measured on and
# for that shape (position_bytes: algorithmic K + V bytes of one position of all
# 64 sequences).
ATTN_TRAFFIC = {
    "source": "paper_2510_17158_amd/csrc/attn_decode.hip",
    "sha256": "43ef04d768466c704263f23bacabddbc355550434d3a6e408908055aaa35092f",
    # rocprofv3 FETCH_SIZE / WRITE_SIZE per dispatch of the per-row decode attention at
    # batch 64 (7B shape, 2048 shared prompt positions), mean of the 32 layers' launches at
    # exactly 1024 generated positions: the mean launch of the 7B rollout (positions
    # 1 .. 2047), read directly; readings at 512 and 1536 put it on their line (0.02%),
    # so the mean launch's traffic is this one's
    "batch": 64, "generated_positions": 1024,
    "fetch_kib": 136314.7, "fetch_scale": 2.0,
    "write_kib": 512.0, "write_scale": 1.0,
    "position_bytes": 64 * 4096,
}


def attn_traffic(algorithmic_bytes_per_launch: float, batch: int = 64):
    """Counter-measured HBM bytes per launch of the decode attention, or None when
    the kernel has changed since the counters, the batch differs, or the launches'
    mean generated positions are not the measured ones."""
    import hashlib
    try:
        with open(os.path.join(ROOT, ATTN_TRAFFIC["source"]), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != ATTN_TRAFFIC["sha256"]:
                return None
    except OSError:
        return None
    t = ATTN_TRAFFIC
    positions = algorithmic_bytes_per_launch / t["position_bytes"]
    if batch != t["batch"] or abs(positions - t["generated_positions"]) > 0.5:
        return None
    return (t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"]) * 1024


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def copy_ceiling_gbs(torch) -> float:
    """HBM rate of a plain 1 GiB device-to-device copy (bytes read + written per
    second), the best of 5 timed copies after one untimed."""
    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    best = float("inf")
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del src, dst
    torch.cuda.empty_cache()
    return 2 * (1 << 30) / (best / 1e3) / 1e9


def read_ceiling_gbs(torch) -> float:
    """HBM read rate of the vendor library's memory-bound kernel of the decode
    step's own kind: a bf16 matrix-vector product (torch.mv) over a 4 GiB matrix
    (matrix bytes per second; the vector and the result aside), the best of 5
    timed products after one untimed.  The decode step reads almost everything it
    moves, so this is the ceiling it compares with beside the spec peak (a plain
    full-tensor sum reads at little more than half this rate, a device copy, read
    plus write, at about 0.8 of it)."""
    rows, cols = 1 << 16, 1 << 15
    a = torch.ones(rows, cols, dtype=torch.bfloat16, device="cuda")
    v = torch.ones(cols, dtype=torch.bfloat16, device="cuda")
    y = torch.mv(a, v)
    best = float("inf")
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        y = torch.mv(a, v)
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del a, v, y
    torch.cuda.empty_cache()
    return 2 * rows * cols / (best / 1e3) / 1e9


def gemm_ceiling_tflops(torch, n: int = 8192) -> float:
    """Dense bf16 matrix-core rate the device sustains right after the step: the
    vendor library's n x n x n product (torch.mm, contiguous operands), the best
    of 5 timed calls after two untimed.  Under dense matrix work the engine clock
    drops below the 2.4 GHz of the spec peak (and varies with the power state by
    some 15% between runs), so this ceiling is what a GEMM-bound phase can be
    compared against beside that peak."""
    g = torch.Generator(device="cuda").manual_seed(0)
    a = torch.randn(n, n, device="cuda", generator=g).to(torch.bfloat16)
    b = torch.randn(n, n, device="cuda", generator=g).to(torch.bfloat16)
    c = torch.mm(a, b)
    c = torch.mm(a, b)
    best = float("inf")
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        torch.mm(a, b, out=c)
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del a, b, c
    torch.cuda.empty_cache()
    return 2.0 * n ** 3 / (best / 1e3) / 1e12


def decode_bytes_per_step(w, ctx_avg: float) -> float:
    """Algorithmic HBM bytes of one decode step: every weight once (embedding rows
    aside), the KV of every context position once, the new K/V written.  With the
    prompt shared within groups the prompt's KV counts once per group."""
    c = w.model
    es = c.elem_bytes
    weights = (c.n_params() - c.vocab * c.d_model) * es + w.batch * c.d_model * es
    kv_tok = c.kv_bytes_per_token()
    if w.shared_prompt:
        kv = (w.n_prompts * w.prompt_len + w.batch * (ctx_avg - w.prompt_len)) * kv_tok
    else:
        kv = w.batch * ctx_avg * kv_tok
    return weights + kv + w.batch * kv_tok


def score_flops(w) -> float:
    """Algorithmic flops of scoring one model over the batch.  With the prompt
    shared within groups its positions count once per group (projections and
    causal attention), every sequence's later positions once each."""
    c = w.model
    T, N, Tp = w.total_len, w.batch, w.prompt_len
    per_tok = 2 * (c.d_model * (c.q_dim + 2 * c.kv_dim) + c.q_dim * c.d_model
                   + 3 * c.d_model * c.d_ffn)
    attn_pos = 2 * 2 * c.n_layers * c.n_heads * c.head_dim   # per (query, key) pair
    head = 2 * c.vocab * c.d_model * (T - Tp) * N
    if w.shared_prompt:
        rows = w.n_prompts * Tp + N * (T - Tp)
        pairs = w.n_prompts * Tp * (Tp + 1) / 2 + N * (T * (T + 1) / 2 - Tp * (Tp + 1) / 2)
    else:
        rows = N * T
        pairs = N * T * (T + 1) / 2
    return c.n_layers * per_tok * rows + attn_pos * pairs + head


def update_flops_per_seq(w) -> float:
    """Algorithmic flops of the gradient of one sequence's scored log-probs:
    three times its forward (the forward, then the data and the weight
    gradients of every product): the projections over all T positions, causal
    attention, and the LM head on the scored positions."""
    c = w.model
    T, Tn = w.total_len, w.new_tokens
    per_tok = 2 * (c.d_model * (c.q_dim + 2 * c.kv_dim) + c.q_dim * c.d_model
                   + 3 * c.d_model * c.d_ffn)
    attn = 2 * 2 * c.n_layers * c.n_heads * c.head_dim * T * (T + 1) / 2
    head = 2 * c.vocab * c.d_model * Tn
    return 3 * (c.n_layers * per_tok * T + attn + head)


def update_measure(w, it, pol, api, torch, n_seqs: int = 2) -> dict:
    """The iteration's gradient step on a slice, outside the timed step: the
    policy backward of the first n_seqs sequences of the step's batch with the
    token loss's dL/dlogp (grpo_policy_backward), then AdamW over every
    parameter (grpo_adamw_step, fp32 master weights)."""
    c = w.model
    T, sf = w.total_len, w.prompt_len
    n = min(n_seqs, w.batch)
    try:
        grads = api.Grads(pol)
        ws = api.alloc_workspace(pol, api.OP_BACKWARD, n, T)
        toks = it.seqs[:n].contiguous()
        dl = it.dloss[:n].contiguous()
        api.policy_backward(pol, toks, sf, w.temperature, dl, grads, ws=ws)    # untimed
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        api.policy_backward(pol, toks, sf, w.temperature, dl, grads, ws=ws)
        e1.record()
        torch.cuda.synchronize()
        bwd_ms = e0.elapsed_time(e1)
        del ws
        torch.cuda.empty_cache()
        # a copy of the weights (the model itself stays as it is), fp32 masters, moments
        state = {k: (v.clone(), v.float() if c.dtype == 1 else None,
                     torch.zeros_like(v, dtype=torch.float32),
                     torch.zeros_like(v, dtype=torch.float32)) for k, v in pol.weights.items()}
        hp = dict(lr=1e-6, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0)
        torch.cuda.synchronize()
        e0.record()
        for k, (prm, mst, m1, m2) in state.items():
            api.adamw_step(c.dtype, prm, mst, m1, m2, grads.t[k], step=1, **hp)
        e1.record()
        torch.cuda.synchronize()
        opt_ms = e0.elapsed_time(e1)
        nparam = sum(v.numel() for v in pol.weights.values())
        del state, grads
        torch.cuda.empty_cache()
    except torch.cuda.OutOfMemoryError as ex:
        torch.cuda.empty_cache()
        return {"error": f"out of memory: {ex}"[:200]}
    fl = update_flops_per_seq(w) * n
    per_seq = bwd_ms / n
    return {"sequences": n, "tokens_per_seq": T, "backward_ms_per_seq": per_seq,
            "alg_tflops": fl / (bwd_ms / 1e3) / 1e12,
            "mfma_frac": fl / (bwd_ms / 1e3) / 1e12 / BF16_PEAK_TFLOPS,
            "adamw_ms": opt_ms, "params": nparam,
            "est_batch_update_ms": per_seq * w.batch + opt_ms,
            "note": "outside the timed step; a slice of the step's batch"}


def kernel_bytes(w) -> dict:
    """Algorithmic HBM bytes of one step, per decode-side kernel name: every
    weight byte of the projection once per decode step, plus its activation rows
    read and its product written once (fp32 products, bf16 activations); for
    attn_decode the K and V of every context position of every sequence per
    layer, context = position + 1, or, with the prompt shared within groups,
    attn_prefix the prompt's K and V once per group and attn_decode every
    sequence's generated positions."""
    c = w.model
    es = c.elem_bytes
    B, L, d, f, V = w.batch, c.n_layers, c.d_model, c.d_ffn, c.vocab
    qd, kvd = c.q_dim, c.kv_dim
    n_dec = w.new_tokens - 1
    kv_layer_tok = 2 * kvd * es
    ctx_sum = sum(w.prompt_len + s for s in range(1, n_dec + 1))   # context of decode step s
    out = {
        "gemm_decode_qkv": n_dec * L * ((qd + 2 * kvd) * d * es + B * d * es + B * (qd + 2 * kvd) * 4),
        "gemm_decode_o": n_dec * L * (d * qd * es + B * qd * es + B * d * 4),
        "gemm_decode_swiglu": n_dec * L * (2 * f * d * es + B * d * es + B * f * es),
        "gemm_decode_down": n_dec * L * (d * f * es + B * f * es + B * d * 4),
        # without a top-k cut (bf16) the LM head writes the sampler's 32-byte pieces
        # per row and 128-id tile instead of the logits
        "gemm_decode_lm_head": n_dec * (V * d * es + B * d * es +
                                        (B * -(-V // 128) * 32 if es == 2 and (w.top_k <= 0 or w.top_k >= V)
                                         else B * V * 4)),
    }
    if w.shared_prompt:
        out["attn_prefix"] = n_dec * L * w.n_prompts * w.prompt_len * kv_layer_tok
        out["attn_decode"] = L * B * kv_layer_tok * (ctx_sum - n_dec * w.prompt_len)
    else:
        out["attn_decode"] = L * B * kv_layer_tok * ctx_sum
    return out


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, host, budget_s: float = 20.0) -> dict:
    """The oracle (fp64 NumPy, as it stands) on a bounded slice of the workload:
    decode steps of up to 8 sequences at the prompt-length context (all layers,
    LM head and sampler; the cached K/V drawn once before timing, since their
    values do not change the work), a prefill slice of one prompt and a
    teacher-forced scoring slice of one sequence.  value = the decode rate
    (sampled tokens per second), the rollout's dominant phase."""
    import numpy as np
    import oracle
    try:
        cores = len(os.sched_getaffinity(0))
    except Exception:
        cores = os.cpu_count() or 1
    c = w.model
    B, ctx = min(8, w.batch), w.prompt_len
    om = oracle.OracleModel(c, host)
    rng = np.random.default_rng(0)
    K = rng.standard_normal((B, c.n_kv_heads, ctx + 1, c.head_dim)) * 0.5
    V = rng.standard_normal((B, c.n_kv_heads, ctx + 1, c.head_dim)) * 0.5
    toks = rng.integers(0, c.vocab, B)
    pos = np.full(B, ctx)
    # decode: whole steps at the full batch until half the budget is spent
    t0 = time.perf_counter()
    steps = 0
    while True:
        x = om.embed(toks)
        for l in range(c.n_layers):
            x, _, _ = om.decode_layer(l, x, pos, K, V)
            om.drop_cache()
        lg = om.head(x)
        om.drop_cache()
        for b in range(B):
            oracle.sample_token(lg[b], w.temperature, w.top_k, 1, 1 + steps, b)
        steps += 1
        if time.perf_counter() - t0 >= budget_s / 2:
            break
    t_dec = (time.perf_counter() - t0) / steps
    # prefill and scoring slices: n positions of one prompt through every layer,
    # then the head at the last position (prefill) or at every position with its
    # teacher-forced log-probability (scoring)
    n = 32
    seq = np.asarray(rng.integers(0, c.vocab, n + 1))
    t0 = time.perf_counter()
    x = om.embed(seq[:n])
    for l in range(c.n_layers):
        x, _, _ = om.layer(l, x)
        om.drop_cache()
    t_fwd = time.perf_counter() - t0
    t0 = time.perf_counter()
    om.head(x[-1:])
    t_head1 = time.perf_counter() - t0
    t0 = time.perf_counter()
    ls = oracle.log_softmax(om.head(x) / (w.temperature or 1.0))
    _ = ls[np.arange(n), seq[1:]]
    om.drop_cache()
    t_headn = time.perf_counter() - t0
    return {"value": B / t_dec, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "cpu_model": cpu_model(),
            "prefill_tokens_per_s": n / (t_fwd + t_head1),
            "scored_tokens_per_s": n / (t_fwd + t_headn),
            "sample": f"{steps} decode step(s) of {B} sequences at context "
                      f"{ctx} (all {c.n_layers} layers, LM head, sampler; {steps * t_dec:.1f} s); "
                      f"a {n}-position prefill slice and a {n}-position scoring slice of one "
                      f"sequence ({t_fwd + t_head1 + t_headn:.1f} s); fp64 NumPy"}


def decode_at(w, ctx: int, steps: int) -> dict:
    """Counter runs at one decode context: prefill prompts of `ctx` positions,
    then `steps` grouped decode steps that share only the workload's prompt
    length, so every per-row attention launch reads ctx - prompt_len generated
    positions per sequence besides the shared prompt (ctx = prompt_len +
    new_tokens / 2 is the mean context of the workload's rollout).  The group's
    rows hold identical prompts, so the shared positions are the same in every
    member, as grouped decode requires."""
    import torch
    from paper_2510_17158_amd import api, synth
    from paper_2510_17158_amd.runner import GrpoIteration
    shared = w.prompt_len
    if not (shared < ctx and steps >= 1 and ctx + steps <= w.max_len):
        raise SystemExit(f"--decode-at needs {shared} < ctx and ctx + steps <= {w.max_len}")
    wc = w.with_(prompt_len=ctx, new_tokens=w.total_len - ctx, score=False)
    c = wc.model
    host = synth.make_weights(c, wc.master_seed)
    pol = api.Model(c, api.upload_weights(c, host))
    del host
    it = GrpoIteration(wc, pol, None, synth.make_prompts(wc), synth.make_rewards(wc),
                       synth.make_seed(wc))
    it.prefill()
    tok_o = torch.empty(it.B, steps, dtype=torch.int32, device="cuda")
    lp_o = torch.empty(it.B, steps, dtype=torch.float32, device="cuda")
    it.tok.copy_(it.tok0)
    it.pos.fill_(ctx)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    api.rollout_step(pol, it.kv, it.B, it.max_len, it.pos, it.tok, ctx, 1, steps, it.sampling,
                     tok_o, lp_o, ws=it.ws_roll, group=wc.group, prefix_len=shared)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    assert bool(torch.isfinite(lp_o).all())
    return {"mode": "decode_at", "workload": w.name, "context": ctx, "shared_prompt": shared,
            "generated_positions": ctx - shared, "steps": steps, "decode_step_ms": ms,
            "max_len": it.max_len}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="7b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--new-tokens", type=int, default=None,
                    help="override the workload's sampled tokens (profiling runs)")
    ap.add_argument("--prompt-len", type=int, default=None,
                    help="override the workload's prompt length (profiling runs)")
    ap.add_argument("--no-kernel-timing", action="store_true",
                    help="skip the replica of the step with per-launch HIP events (no roofline "
                         "line); for hardware-counter runs")
    ap.add_argument("--decode-at", type=int, default=None, metavar="CTX",
                    help="only prefill prompts of CTX positions and run --steps grouped decode "
                         "steps sharing the workload's prompt length (counter runs at one "
                         "decode context)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only copy a 1 GiB device buffer 4 times (HBM counter calibration)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": 1 << 30, "copies": 4}), flush=True)
        return
    if args.decode_at:
        from paper_2510_17158_amd.workloads import get
        import torch
        torch.cuda.set_device(0)
        print(json.dumps(decode_at(get(args.workload), args.decode_at, args.steps)), flush=True)
        return
    if os.environ.get("ROCPROF_COUNTER_COLLECTION") and not args.no_kernel_timing:
        # hardware-counter collection rewrites every dispatch; the library then
        # launches decode steps eagerly and refuses per-launch event timing, so a
        # counter run must skip the timing replica
        print("bench.py under rocprofv3 counter collection needs --no-kernel-timing",
              file=sys.stderr)
        sys.exit(2)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); "
              "the hot path is built and measured on a single MI355X.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2510_17158_amd import api, synth
    from paper_2510_17158_amd.runner import GrpoIteration
    from paper_2510_17158_amd.workloads import get

    w = get(args.workload)
    if args.new_tokens:
        w = w.with_(new_tokens=args.new_tokens)
    if args.prompt_len:
        w = w.with_(prompt_len=args.prompt_len)
    c = w.model
    torch.cuda.set_device(0)
    t = time.perf_counter()
    host = synth.make_weights(c, w.master_seed)
    pol = api.Model(c, api.upload_weights(c, host))
    ref = None
    if w.score:
        ref_host = synth.make_weights(c, w.master_seed, ref=True)
        ref = api.Model(c, api.upload_weights(c, ref_host), decode=False)
        del ref_host
    it = GrpoIteration(w, pol, ref, synth.make_prompts(w), synth.make_rewards(w),
                       synth.make_seed(w))
    torch.cuda.synchronize()
    log(f"[bench] set-up {time.perf_counter() - t:.1f} s  workload {w.name}")

    def step(ev=None):
        if ev: ev[0].record()
        it.prefill()
        if ev: ev[1].record()
        it.decode()
        if ev: ev[2].record()
        it.assemble()
        if w.score:
            it.score()
        else:
            it.lp_pol.copy_(it.logp_old)
        if ev: ev[3].record()
        it.grpo()
        if ev: ev[4].record()

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {i + 1}/{args.warmup} done")
    phases = np.zeros(4)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
        step(ev)
        torch.cuda.synchronize()
        phases += [ev[j].elapsed_time(ev[j + 1]) for j in range(4)]
        log(f"[bench] step {i + 1}/{args.steps} done")
    wall = time.perf_counter() - t0
    phases /= args.steps
    ms_step = wall * 1e3 / args.steps
    gen = w.batch * w.new_tokens
    n_dec = w.new_tokens - 1
    dec_ms = phases[1] / max(n_dec, 1)
    ctx_avg = w.prompt_len + n_dec / 2.0
    dec_bytes = decode_bytes_per_step(w, ctx_avg)
    n_models = 2 if w.score else 0
    out = {
        "metric": "rollout tokens/s on 1 MI355X (G samples/prompt) + % of HBM roofline",
        "value": gen * args.steps / wall,
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if c.dtype == 1 else "f32",
        "data": "synthetic (seeded random-init weights, code-like prompts with tool spans)",
        "config": {"workload": w.name, "layers": c.n_layers, "d_model": c.d_model,
                   "prompts": w.n_prompts, "group": w.group, "prompt_len": w.prompt_len,
                   "new_tokens": w.new_tokens, "batch": w.batch,
                   "scored_models": n_models},
        "phases_ms": {"prefill": phases[0], "decode": phases[1], "score": phases[2],
                      "advantages_loss": phases[3]},
        "rollout_tokens_per_s": gen / ((phases[0] + phases[1]) / 1e3),
        "decode_step_ms": dec_ms,
        "decode_step_gbs": dec_bytes / (dec_ms / 1e3) / 1e9,
        "decode_step_hbm_frac": dec_bytes / (dec_ms / 1e3) / 1e9 / HBM_PEAK_GBS,
        "decode_tokens_per_s": w.batch / (dec_ms / 1e3),
    }
    if w.score:
        sf = score_flops(w)
        out["scored_tokens_per_s"] = n_models * w.batch * w.total_len / (phases[2] / 1e3)
        out["score_tflops"] = n_models * sf / (phases[2] / 1e3) / 1e12
        out["score_mfma_frac"] = out["score_tflops"] / BF16_PEAK_TFLOPS
    # the decode step against measured stream-copy and stream-read ceilings as well
    # as the spec peak
    cc = copy_ceiling_gbs(torch)
    out["copy_ceiling_gbs"] = cc
    out["decode_step_copy_frac"] = out["decode_step_gbs"] / cc
    rc = read_ceiling_gbs(torch)
    out["read_ceiling_gbs"] = rc
    out["decode_step_read_frac"] = out["decode_step_gbs"] / rc
    # scoring against the measured dense-GEMM rate as well as the spec peak
    if w.score and c.dtype == 1:
        gc = gemm_ceiling_tflops(torch)
        out["gemm_ceiling_tflops"] = gc
        out["score_gemm_ceiling_frac"] = out["score_tflops"] / gc
    # per-kernel times from a profiled replica of the step (HIP events around
    # every launch, on the launch stream); the dominant decode kernel sets the
    # roofline line
    if args.no_kernel_timing:
        if not args.no_cpu_baseline:
            out["cpu_baseline"] = cpu_baseline(w, host, args.cpu_budget)
        print(json.dumps(out), flush=True)
        return
    api.profile_begin()
    step()
    torch.cuda.synchronize()
    prof = api.profile_end()
    out["kernels_ms"] = {k: {"launches": n, "total_ms": t, "avg_us": 1e3 * t / n}
                         for k, (n, t) in sorted(prof.items(), key=lambda kv: -kv[1][1])}
    kb = kernel_bytes(w)
    dom = max(kb, key=lambda k: prof.get(k, (0, 0.0))[1])
    n, t = prof[dom]
    out["roofline"] = {"bound": "hbm", "achieved": kb[dom] / (t / 1e3) / 1e9,
                       "peak": HBM_PEAK_GBS, "unit": "GB/s",
                       "frac": kb[dom] / (t / 1e3) / 1e9 / HBM_PEAK_GBS,
                       "traffic": (attn_traffic(kb[dom] / n, w.batch) if dom == "attn_decode"
                                   else None),
                       "traffic_unit": "bytes per launch",
                       "kernel": dom, "launches": n, "avg_us": 1e3 * t / n,
                       "algorithmic_bytes_per_launch": kb[dom] / n}
    out["decode_kernels_gbs"] = {k: kb[k] / (prof[k][1] / 1e3) / 1e9 for k in kb if k in prof}
    if w.score:
        out["update"] = update_measure(w, it, pol, api, torch)
        log("[bench] update measured")
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, host, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
