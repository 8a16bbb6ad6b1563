"""Error bounds of the GPU arithmetic, for rounding-point-local parity.

Each stage of the forward is checked on the GPU's own inputs (read from a
grpo_trace): the oracle evaluates the stage's plain definition in fp64 on
exactly those inputs, and the GPU's output must lie within a bound derived
from the arithmetic the kernel performs.  No constant here is fitted to the
GPU's results; each follows from a stated model of the hardware arithmetic:

* u = 2^-24.  Every fp32 add, multiply, fused multiply-add, divide and square
  root on the vector units is correctly rounded (round to nearest even): its
  error is at most u * |exact result of that operation|.  (HIP's default
  compilation keeps division and sqrtf correctly rounded.)
* Products of two bf16 values are exact in fp32 (8 + 8 significand bits).
* One bf16 matrix-core instruction (v_mfma_f32_16x16x32_bf16 adds 32 products
  per output, v_mfma_f32_32x32x16_bf16 adds 16) returns acc + sum(products)
  with an error of at most C_MFMA * u * (|acc| + sum |products|).  The
  instruction adds its products in one pass and truncates rather than
  rounding to nearest; a probe of 2 x 10^6 instruction outputs on gfx950
  (normal and exponent-spread data) measured at most 5.9 u * (|acc| +
  sum|products|), so C_MFMA = 12 is twice the worst case observed.
* The hardware exp2 and the exponentials built on it are within 2 ulp
  (relative 4u) of the exact value of their (rounded) argument.

A bound is first order in u (second-order terms are below 10^-9 of it at
these sizes); a 1% margin covers them.

bf16 outputs: the GPU rounds its fp32 value z to bf16 (nearest even).  With
|z - y| <= E for the exact value y, the GPU's bf16 value must lie in
[RNE(y - E), RNE(y + E)] (rounding is monotone).  Where both ends agree the
result is unique and the check is bit-exact; elsewhere both neighbours are
valid results of the arithmetic.  The fraction of such elements is reported.
"""
from __future__ import annotations

import numpy as np

import oracle

U = 2.0 ** -24
C_MFMA = 12.0
C_EXP = 4.0          # relative error of a hardware exponential, in u
MARGIN = 1.01        # second-order terms


# ----------------------------------------------------------------- checks
class Report:
    """Collects per-stage results: violations, element counts, ambiguous counts."""

    def __init__(self):
        self.st = {}

    def add(self, name, ok, amb=None, err=None):
        ok = np.asarray(ok, bool)
        s = self.st.setdefault(name, dict(n=0, bad=0, amb=0, worst=[]))
        s["n"] += ok.size
        s["bad"] += int((~ok).sum())
        if amb is not None:
            s["amb"] += int(np.asarray(amb, bool).sum())
        if err is not None and (~ok).any():
            s["worst"].extend(err[:3])

    def ok(self):
        return all(s["bad"] == 0 for s in self.st.values())

    def summary(self):
        return {k: dict(n=v["n"], bad=v["bad"], amb_frac=round(v["amb"] / max(v["n"], 1), 5),
                        **({"worst": v["worst"][:3]} if v["bad"] else {}))
                for k, v in self.st.items()}


def check_bf16(rep: Report, name: str, gpu, y, E):
    """gpu: bf16 values (exact, as float); y: exact value; E: bound on |z - y|."""
    gpu, y, E = (np.asarray(a, np.float64) for a in (gpu, y, E))
    E = np.broadcast_to(E * MARGIN, y.shape)
    lo, hi = oracle.round_bf16(y - E), oracle.round_bf16(y + E)
    ok = (gpu >= lo) & (gpu <= hi)
    err = None
    if not ok.all():
        idx = np.flatnonzero(~ok.ravel())[:3]
        err = [dict(i=int(i), gpu=float(gpu.ravel()[i]), y=float(y.ravel()[i]),
                    E=float(E.ravel()[i])) for i in idx]
    rep.add(name, ok, lo != hi, err)
    return ok


def check_f32(rep: Report, name: str, gpu, y, E):
    gpu, y, E = (np.asarray(a, np.float64) for a in (gpu, y, E))
    ok = np.abs(gpu - y) <= E * MARGIN + 1e-300
    err = None
    if not ok.all():
        idx = np.flatnonzero(~ok.ravel())[:3]
        err = [dict(i=int(i), gpu=float(gpu.ravel()[i]), y=float(y.ravel()[i]),
                    E=float(np.broadcast_to(E, y.shape).ravel()[i])) for i in idx]
    rep.add(name, ok, None, err)
    return ok


# ------------------------------------------------------------- GEMM bounds
class Gemm:
    """Accumulation structure of one GEMM kernel.

    kind "mfma": chains of matrix-core instructions of `kc` products each;
    kind "fma": chains of scalar fused multiply-adds (kc = 1).  K is cut into
    `splits` contiguous ranges; inside a range the kc-wide steps are dealt
    round-robin to `waves` chains.  The chains of a range are added as
    ((c0 + c2) + (c1 + c3)) for four waves (in order otherwise), then the
    ranges one after another (after the residual, when there is one)."""

    def __init__(self, kind: str, kc: int, splits: int = 1, waves: int = 1):
        self.kind, self.kc, self.splits, self.waves = kind, kc, splits, waves

    def bound(self, a, W, resid=None, block_cols: int = 8192):
        """a [R, K], W [N, K] exact fp64 values -> (exact y [R, N], bound E [R, N]).
        resid [R, N] (optional): y = resid + a W^T, the residual added first."""
        a = np.asarray(a, np.float64)
        W = np.asarray(W, np.float64)
        R, K = a.shape
        N = W.shape[0]
        y = np.empty((R, N))
        E = np.empty((R, N))
        for n0 in range(0, N, block_cols):
            sl = slice(n0, min(N, n0 + block_cols))
            r = None if resid is None else np.asarray(resid, np.float64)[:, sl]
            y[:, sl], E[:, sl] = self._bound(a, W[sl], r)
        return y, E

    def _bound(self, a, W, resid):
        R, K = a.shape
        N = W.shape[0]
        kc = self.kc
        kper = K // self.splits
        assert kper * self.splits == K and kper % (kc * self.waves) == 0, (K, self.splits)
        aa, Wa = np.abs(a), np.abs(W)
        E = np.zeros((R, N))
        split_vals = []
        for s in range(self.splits):
            chains = []
            for w in range(self.waves):
                A = np.zeros((R, N))
                steps = range(s * kper + w * kc, (s + 1) * kper, kc * self.waves)
                for k0 in steps:
                    ks = slice(k0, k0 + kc)
                    P = a[:, ks] @ W[:, ks].T
                    if self.kind == "mfma":
                        E += C_MFMA * U * (np.abs(A) + aa[:, ks] @ Wa[:, ks].T)
                        A = A + P
                    else:
                        # one fma per product, each rounded: u * |partial sum|
                        for k in range(k0, k0 + kc):
                            A = A + np.outer(a[:, k], W[:, k])
                            E += U * np.abs(A)
                chains.append(A)
            if self.waves == 4:
                c02, c13 = chains[0] + chains[2], chains[1] + chains[3]
                tot = c02 + c13
                E += U * (np.abs(c02) + np.abs(c13) + np.abs(tot))
            else:
                tot = chains[0]
                for c in chains[1:]:
                    tot = tot + c
                    E += U * np.abs(tot)
            split_vals.append(tot)
        y = np.zeros((R, N)) if resid is None else resid.copy()
        first = resid is None
        for v in split_vals:
            if first:
                y = v.copy()
                first = False
            else:
                y = y + v
                E += U * np.abs(y)
        return y, E


def decode_gemm(splits: int) -> Gemm:
    """The decode GEMM: 32-wide steps dealt to 4 waves, `splits` K ranges."""
    return Gemm("mfma", 32, splits, 4)


def rows_gemm(M: int) -> Gemm:
    """Prefill / scoring GEMM over M rows: 256 x 256 tiles on 32x32x16 from 1024
    rows on (one chain of 16-wide steps), 128 x 128 tiles on 16x16x32 below."""
    return Gemm("mfma", 16) if M >= 1024 else Gemm("mfma", 32)


F32_GEMM = Gemm("fma", 1)


def gemm_for(cfg, rows: int, decode_splits: int | None = None) -> Gemm:
    if cfg.dtype == 0:
        return F32_GEMM
    if decode_splits is not None:
        return decode_gemm(decode_splits)
    return rows_gemm(rows)


# ---------------------------------------------------------- elementwise
def rmsnorm_bound(x, g, eps):
    """h = x / sqrt(mean(x^2) + eps) * g, evaluated in fp32: the sum of squares
    (all terms positive) passes through at most 30 roundings (16 per thread,
    6 wave levels, 8 wave partials), then /d, +eps, sqrt, 1/x, *r, *g: relative
    error <= (30u + 2u) / 2 + 4u... <= 20u of |h|."""
    h = oracle.rmsnorm(np.asarray(x, np.float64), np.asarray(g, np.float64), eps)
    return h, 20.0 * U * np.abs(h)


def rope_bound(lo, hi, Elo, Ehi, pos, theta, hd):
    """Rotation of the pre-rotation (lo, hi) halves [..., hd/2] at positions pos
    (broadcast over the leading axes): cos/sin rounded to fp32 (u each), two
    products and a sum, plus the inputs' own bounds."""
    ang = oracle.numerics.rope_angles(np.atleast_1d(pos), hd, theta)
    c, s = np.cos(ang), np.sin(ang)
    while c.ndim < lo.ndim:
        c, s = c[:, None, :], s[:, None, :]
    ylo = lo * c - hi * s
    yhi = hi * c + lo * s
    base = 3.0 * U * (np.abs(lo * c) + np.abs(hi * s))
    Ec = np.abs(c) * Elo + np.abs(s) * Ehi + base
    Es = np.abs(c) * Ehi + np.abs(s) * Elo + 3.0 * U * (np.abs(hi * c) + np.abs(lo * s))
    return ylo, yhi, Ec, Es


def swiglu_bound(g, up, Eg, Eu):
    """a = silu(g) * up in fp32 with a hardware exponential: the inputs' bounds
    through the derivatives, plus the evaluation (exp argument u|g|, exp C_EXP u,
    then 4u for the rest: 1 + e (u/2), the hardware reciprocal (within 1 ulp,
    u) or an IEEE division (u/2), and the products by g and up (u/2 each))."""
    sg = 1.0 / (1.0 + np.exp(-g))
    silu = g * sg
    y = silu * up
    dsilu = sg * (1.0 + g * (1.0 - sg))
    E = np.abs(dsilu * up) * Eg + np.abs(silu) * Eu + np.abs(y) * U * (np.abs(g) + C_EXP + 4.0)
    return y, E


# ------------------------------------------------------------ attention
def attention_bound(q, Kc, Vc, hd, segments, merges=0):
    """One query row and head against its context (positions 0..ctx-1 in order).

    q [hd], Kc/Vc [ctx, hd] exact fp64 (the GPU's bf16 or fp32 values).  Returns
    (o, E) with E bounding |o_gpu (fp32, before any bf16 rounding) - o|.

    segments: how the kernels sum P.V over the context, a list of
    (kind, start, end, chunk):
      "mfma":   P.V on matrix cores, P as bf16 hi + lo, chains of `chunk`
                positions from `start` (flash attention: one chain over all
                keys; the grouped step's prompt chunks), 32-key steps of two
                instructions each, at most one rescale per step;
      "decode": the per-row decode kernel: spans of `chunk` positions from
                `start`, each cut into 32-position tiles dealt to the
                workgroup's waves (a fifth tuple element, 4 when absent); a
                lane fuses P.V of positions iv * PPW + ts of its tiles in one
                fma chain (a rescale per tile), lanes then meet in a butterfly;
      "f32":    one fma chain over the positions (fp32 models).
    merges: weighted additions of partial results any term passes through
    (waves, spans, prompt chunks).

    First-order structure (p_j = exp(s_j - max s), L = sum p):
      o_gpu - o = sum_j p_j rho_j (v_j - o) / L        (weight errors)
                + (P.V summation errors + hi/lo split) / L
                + |o| (denominator summation + final division)
    rho_j: the score's dot product over hd (hd/32 matrix-core steps, or hd
    fmas), the scale's rounding, the exponent argument's rounding and the
    exponential's own error."""
    q = np.asarray(q, np.float64)
    Kc = np.asarray(Kc, np.float64)
    Vc = np.asarray(Vc, np.float64)
    ctx = Kc.shape[0]
    scale = 1.0 / np.sqrt(hd)
    s = (Kc @ q) * scale
    p = np.exp(s - s.max())
    L = p.sum()
    o = (p @ Vc) / L
    prods = Kc * q[None, :]
    if any(k == "f32" for k, *_ in segments):
        Es = U * np.abs(np.cumsum(prods, axis=1)).sum(axis=1) * scale
    else:
        steps = prods.reshape(ctx, hd // 32, 32)
        sums = steps.sum(-1)
        prev = np.concatenate([np.zeros((ctx, 1)), np.cumsum(sums, axis=1)[:, :-1]], axis=1)
        Es = C_MFMA * U * (np.abs(prev) + np.abs(steps).sum(-1)).sum(axis=1) * scale
    smax = np.abs(s).max()
    rho = Es + 4.0 * U * np.abs(s) + 3.0 * U * (np.abs(s) + smax + 8.0) + C_EXP * U
    E = (p * rho) @ np.abs(Vc - o[None, :]) / L
    pv = p[:, None] * Vc
    apv = np.abs(pv)
    for kind, a0, a1, chunk, *rest in segments:
        if a1 <= a0:
            continue
        if kind == "mfma":
            E += 2.0 ** -16 * apv[a0:a1].sum(0) / L        # |p - (hi + lo)| <= 2^-16 p
            for c0 in range(a0, a1, chunk):
                cp, ca = pv[c0:min(a1, c0 + chunk)], apv[c0:min(a1, c0 + chunk)]
                nst = (cp.shape[0] + 31) // 32
                pad = ((0, nst * 32 - cp.shape[0]), (0, 0))
                cps = np.pad(cp, pad).reshape(nst, 32, hd).sum(1)
                cas = np.pad(ca, pad).reshape(nst, 32, hd).sum(1)
                cum = np.cumsum(cps, 0)
                prev = np.concatenate([np.zeros((1, hd)), cum[:-1]], 0)
                E += 2.0 * C_MFMA * U * (np.abs(prev) + cas).sum(0) * (1 + 2.0 ** -7) / L
                E += U * np.abs(cum).sum(0) / L             # rescales
        elif kind == "decode":
            PPW = 64 // (hd // 8)
            nvt = 32 // PPW
            for t0 in range(a0, a1, chunk):
                seg = pv[t0:min(a1, t0 + chunk)]
                tiles = (seg.shape[0] + 31) // 32
                pp = np.pad(seg, ((0, tiles * 32 - seg.shape[0]), (0, 0)))
                pp = pp.reshape(tiles, nvt, PPW, hd)
                waves = rest[0] if rest else 4
                for w in range(waves):
                    t = pp[w::waves]
                    if t.shape[0] == 0:
                        continue
                    chain = t.transpose(2, 0, 1, 3).reshape(PPW, -1, hd)
                    E += 2.0 * U * np.abs(np.cumsum(chain, axis=1)).sum(axis=(0, 1)) / L
                    E += U * np.log2(PPW) * np.abs(chain).sum(axis=(0, 1)) / L
        elif kind == "f32":
            E += U * np.abs(np.cumsum(pv[a0:a1], 0)).sum(0) / L
        else:
            raise ValueError(kind)
    E += U * merges * apv.sum(0) / L
    # denominator: positive terms through at most ctx/16 + 64 + merges roundings;
    # then the reciprocal / division and the product
    E += np.abs(o) * U * (ctx / 16.0 + 64 + merges + 3.0)
    return o, E
