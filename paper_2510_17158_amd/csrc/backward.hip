// Backward pass of the teacher-forced policy log-probs and the AdamW step.
//
// The weight gradient of sum_t g_t logp_t (g = dL/dlogp from the GRPO token
// loss) runs as matrix products on the tiled MFMA GEMMs plus the element-wise
// and row-wise kernels here.  Every product is cast as Y[M, N] = X[M, K] W[N, K]^T
// with both operands K-contiguous (the layout the matrix cores read); the
// operands that are not stored that way are transposed first (k_transpose):
//   data gradient   dX = dY W      -> X operand dY, W operand W^T
//   weight gradient dW += dY^T X   -> X operand dY^T, W operand X^T (K = tokens)
// Attention's backward materialises, per head, the T x T scores S = q k^T and
// dP = do v^T (fp32), turns them into P and dS' = P (dP - rowsum(P dP)) / sqrt(hd)
// (row statistics, then 64 x 64 tiles that also write P^T and dS'^T), and finishes with three products per head, batched over
// a block of heads: dq_h = dS'_h k, dk_h = dS'_h^T q_h, dv_h = P_h^T do_h, the
// last two summed over each kv group's heads in a fixed order (k_sum_heads).
// The causal upper triangle is computed and zeroed.
//
// Gradients accumulate in fp32; GEMM operands are the model's dtype (bf16
// products on MFMA, fp32 on the vector units for fp32 models).  Every reduction
// runs in a fixed order, the embedding gradient's scatter-add included (its
// positions are sorted by token first): the result is bit-deterministic.
#include "common.h"
#include "kernels.h"

namespace grpo {

namespace {

constexpr int BT = 64;    // transpose tile

// two finite fp32 values rounded to bf16 (round to nearest even, the hardware
// conversion: the same bits as f2bf for finite inputs), a in the low half
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// out[c][r] = in[r][c] (r < R, c < C); out columns R .. Rpad-1 are zero.
// Batch element b: in + b * in_bs, out + (b / div) * s1 + (b % div) * s2.
// vec (16-byte aligned rows and batch offsets on both sides): a tile inside
// [0, R) x [0, C) is read and written in 16-byte pieces (all loads in flight
// together, a 64-element output row by 8 or 16 lanes); edge tiles element-wise.
template <typename TI, typename TO>
__global__ __launch_bounds__(256) void k_transpose(const TI* __restrict__ in, int ldi, size_t in_bs,
                                                   int R, int C, TO* __restrict__ out, int ldo,
                                                   size_t s1, size_t s2, int div, int Rpad,
                                                   int vec) {
  __shared__ float tile[BT][BT + 1];
  const int b = blockIdx.z, r0 = blockIdx.x * BT, c0 = blockIdx.y * BT;
  in += (size_t)b * in_bs;
  out += (size_t)(b / div) * s1 + (size_t)(b % div) * s2;
  if (vec && r0 + BT <= R && c0 + BT <= C) {
    constexpr int VI = 16 / sizeof(TI), TPI = BT / VI, RPI = 256 / TPI;
    u32x4_t v[BT / RPI];
#pragma unroll
    for (int p = 0; p < BT / RPI; ++p) {
      const int r = p * RPI + threadIdx.x / TPI, c = (threadIdx.x % TPI) * VI;
      v[p] = *(const u32x4_t*)(in + (size_t)(r0 + r) * ldi + c0 + c);
    }
#pragma unroll
    for (int p = 0; p < BT / RPI; ++p) {
      const int r = p * RPI + threadIdx.x / TPI, c = (threadIdx.x % TPI) * VI;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if constexpr (sizeof(TI) == 4) {
          tile[r][c + k] = __uint_as_float(v[p][k]);
        } else {
          tile[r][c + 2 * k] = __uint_as_float(v[p][k] << 16);
          tile[r][c + 2 * k + 1] = __uint_as_float(v[p][k] & 0xffff0000u);
        }
      }
    }
    __syncthreads();
    constexpr int VO = 16 / sizeof(TO), TPO = BT / VO, RPO = 256 / TPO;
#pragma unroll
    for (int p = 0; p < BT / RPO; ++p) {
      const int c = p * RPO + threadIdx.x / TPO, r = (threadIdx.x % TPO) * VO;
      u32x4_t w;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if constexpr (sizeof(TO) == 4)
          w[k] = __float_as_uint(tile[r + k][c]);
        else
          w[k] = pack_bf16x2(tile[r + 2 * k][c], tile[r + 2 * k + 1][c]);
      }
      *(u32x4_t*)(out + (size_t)(c0 + c) * ldo + r0 + r) = w;
    }
    return;
  }
  for (int i = threadIdx.x; i < BT * BT; i += 256) {
    const int r = i / BT, c = i % BT;
    tile[r][c] = (r0 + r < R && c0 + c < C) ? ldf(in, (size_t)(r0 + r) * ldi + c0 + c) : 0.f;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < BT * BT; i += 256) {
    const int c = i / BT, r = i % BT;
    if (c0 + c < C && r0 + r < Rpad) stf(out, (size_t)(c0 + c) * ldo + r0 + r, tile[r][c]);
  }
}

// dz[r, v] = g_r / T (onehot(tgt_r) - softmax(z_r / T)); one workgroup per row.
template <typename TO>
__global__ __launch_bounds__(256) void k_dlogits(const float* __restrict__ z, int V, int ldz,
                                                 const int32_t* __restrict__ tgt, int tstride,
                                                 const float* __restrict__ g, float inv_t,
                                                 TO* __restrict__ dz, int ldo) {
  __shared__ float sh[4];
  const int r = blockIdx.x;
  const float* zr = z + (size_t)r * ldz;
  float m = -INFINITY;
  for (int v = threadIdx.x; v < V; v += 256) m = fmaxf(m, zr[v] * inv_t);
  m = block_max<256>(m, sh);
  float s = 0.f;
  for (int v = threadIdx.x; v < V; v += 256) s += __expf(zr[v] * inv_t - m);
  s = block_sum<256>(s, sh);
  const float c = g[r] * inv_t, rs = 1.f / s;
  const int t = tgt[(size_t)r * tstride];
  TO* o = dz + (size_t)r * ldo;
  for (int v = threadIdx.x; v < V; v += 256) {
    const float p = __expf(zr[v] * inv_t - m) * rs;
    stf(o, v, c * ((v == t ? 1.f : 0.f) - p));
  }
}

// RMSNorm backward of one row: y = x r g, r = (mean x^2 + eps)^-1/2.
// dres[t] += r (g dy) - x r^3 sum(g dy x) / d; dres_e = dres in the GEMM dtype
// (optional); rr[t] = r for the gain gradient.
template <typename TG>
__global__ __launch_bounds__(256) void k_rmsnorm_bwd(const float* __restrict__ x, int ldx,
                                                     const TG* __restrict__ g,
                                                     const float* __restrict__ dy, int ldy, int d,
                                                     float eps, float* __restrict__ dres,
                                                     TG* __restrict__ dres_e, float* __restrict__ rr) {
  __shared__ float sh[4];
  const int t = blockIdx.x;
  const float* xr = x + (size_t)t * ldx;
  const float* dr = dy + (size_t)t * ldy;
  float ss = 0.f, sd = 0.f;
  for (int k = threadIdx.x; k < d; k += 256) {
    const float xv = xr[k];
    ss = fmaf(xv, xv, ss);
    sd = fmaf(ldf(g, k) * dr[k], xv, sd);
  }
  ss = block_sum<256>(ss, sh);
  sd = block_sum<256>(sd, sh);
  const float r = 1.f / sqrtf(ss / (float)d + eps);
  const float c = r * r * r * sd / (float)d;
  float* o = dres + (size_t)t * d;
  for (int k = threadIdx.x; k < d; k += 256) {
    const float v = o[k] + r * ldf(g, k) * dr[k] - xr[k] * c;
    o[k] = v;
    if (dres_e) stf(dres_e, (size_t)t * d + k, v);
  }
  if (threadIdx.x == 0) rr[t] = r;
}

// Gain gradient partials: part[chunk][k] = sum over the chunk's 64 rows of
// dy[t, k] x[t, k] rr[t]; then dg[k] += sum over chunks in order.
__global__ __launch_bounds__(256) void k_norm_dg_part(const float* __restrict__ x, int ldx,
                                                      const float* __restrict__ dy, int ldy,
                                                      const float* __restrict__ rr, int T, int d,
                                                      float* __restrict__ part) {
  const int k = blockIdx.x * 256 + threadIdx.x, c = blockIdx.y;
  if (k >= d) return;
  float s = 0.f;
  const int t1 = min(T, (c + 1) * 64);
  for (int t = c * 64; t < t1; ++t) s = fmaf(dy[(size_t)t * ldy + k] * x[(size_t)t * ldx + k], rr[t], s);
  part[(size_t)c * d + k] = s;
}
__global__ __launch_bounds__(256) void k_norm_dg_sum(const float* __restrict__ part, int chunks,
                                                     int d, float* __restrict__ dg) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k >= d) return;
  float s = 0.f;
  for (int c = 0; c < chunks; ++c) s += part[(size_t)c * d + k];
  dg[k] += s;
}

// SwiGLU: gu = [gate | up] fp32 [T, 2F].  Forward a = silu(gate) up (activation
// dtype); backward dgate = da up silu'(gate), dup = da silu(gate) into dgu [T, 2F].
template <typename TO>
__global__ __launch_bounds__(256) void k_swiglu_fwd(const float* __restrict__ gu, int T, int F,
                                                    TO* __restrict__ a) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)T * F) return;
  const size_t t = i / F, n = i % F;
  const float gt = gu[t * 2 * F + n], up = gu[t * 2 * F + F + n];
  stf(a, i, silu_mul(gt, up));
}
template <typename TO>
__global__ __launch_bounds__(256) void k_swiglu_bwd(const float* __restrict__ gu,
                                                    const float* __restrict__ da, int T, int F,
                                                    TO* __restrict__ dgu) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)T * F) return;
  const size_t t = i / F, n = i % F;
  const float gt = gu[t * 2 * F + n], up = gu[t * 2 * F + F + n], d = da[i];
  const float sg = 1.f / (1.f + __expf(-gt));
  stf(dgu, t * 2 * F + n, d * up * sg * (1.f + gt * (1.f - sg)));
  stf(dgu, t * 2 * F + F + n, d * gt * sg);
}

// The same, four consecutive outputs per thread (F a multiple of 4, 16-byte
// aligned rows): 16-byte loads, 32-bit index arithmetic, the same expressions.
template <typename TO>
__device__ __forceinline__ void st4(TO* p, size_t i, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void st4<float>(float* p, size_t i, float a, float b, float c, float d) {
  *(f32x4_t*)(p + i) = (f32x4_t){a, b, c, d};
}
template <>
__device__ __forceinline__ void st4<bf16_t>(bf16_t* p, size_t i, float a, float b, float c, float d) {
  *(uint2*)(p + i) = make_uint2(pack_bf16x2(a, b), pack_bf16x2(c, d));
}
template <typename TO>
__global__ __launch_bounds__(256) void k_swiglu_fwd4(const float* __restrict__ gu, int T, int F,
                                                     TO* __restrict__ a) {
  const uint32_t F4 = (uint32_t)F / 4, idx = blockIdx.x * 256u + threadIdx.x;
  if (idx >= (uint32_t)T * F4) return;
  const uint32_t t = idx / F4, n = 4 * (idx - t * F4);
  const f32x4_t g = *(const f32x4_t*)(gu + (size_t)t * 2 * F + n);
  const f32x4_t u = *(const f32x4_t*)(gu + (size_t)t * 2 * F + F + n);
  st4(a, (size_t)t * F + n, silu_mul(g[0], u[0]), silu_mul(g[1], u[1]), silu_mul(g[2], u[2]),
      silu_mul(g[3], u[3]));
}
template <typename TO>
__global__ __launch_bounds__(256) void k_swiglu_bwd4(const float* __restrict__ gu,
                                                     const float* __restrict__ da, int T, int F,
                                                     TO* __restrict__ dgu) {
  const uint32_t F4 = (uint32_t)F / 4, idx = blockIdx.x * 256u + threadIdx.x;
  if (idx >= (uint32_t)T * F4) return;
  const uint32_t t = idx / F4, n = 4 * (idx - t * F4);
  const f32x4_t g = *(const f32x4_t*)(gu + (size_t)t * 2 * F + n);
  const f32x4_t u = *(const f32x4_t*)(gu + (size_t)t * 2 * F + F + n);
  const f32x4_t d = *(const f32x4_t*)(da + (size_t)t * F + n);
  float dg[4], du[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float sg = 1.f / (1.f + __expf(-g[e]));
    dg[e] = d[e] * u[e] * sg * (1.f + g[e] * (1.f - sg));
    du[e] = d[e] * g[e] * sg;
  }
  st4(dgu, (size_t)t * 2 * F + n, dg[0], dg[1], dg[2], dg[3]);
  st4(dgu, (size_t)t * 2 * F + F + n, du[0], du[1], du[2], du[3]);
}

// RoPE adjoint on the q and k heads of dqkv [T, (H + 2 Hkv) hd] (fp32, in place:
// lo' = lo c + hi s, hi' = hi c - lo s), and the whole row in the GEMM dtype.
template <typename TO>
__global__ __launch_bounds__(256) void k_rope_bwd(float* __restrict__ dqkv, int T, int heads,
                                                  int n_rot, int hd, const float2* __restrict__ cs,
                                                  TO* __restrict__ out) {
  const int half = hd / 2;
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)T * heads * half) return;
  const int e = (int)(i % half);
  const int h = (int)((i / half) % heads);
  const size_t t = i / ((size_t)half * heads);
  float* p = dqkv + (t * heads + h) * hd;
  float lo = p[e], hi = p[e + half];
  if (h < n_rot) {
    const float2 c = cs[t * half + e];
    const float l2 = lo * c.x + hi * c.y, h2 = hi * c.x - lo * c.y;
    lo = l2; hi = h2;
    p[e] = lo; p[e + half] = hi;
  }
  stf(out, (t * heads + h) * hd + e, lo);
  stf(out, (t * heads + h) * hd + e + half, hi);
}

// Attention softmax backward, pass 1: per query row i of head-batch element b,
// from the raw scores S [T, ldS = Tp] (q.k, fp32) and dP = do.v: the row maximum
// m of S s over j <= i, l = sum_j e^(S s - m) and D = sum_j P dP (P = e^(..) / l).
__global__ __launch_bounds__(256) void k_attn_row_stats(const float* __restrict__ S,
                                                        const float* __restrict__ dP, int T, int Tp,
                                                        float s, float* __restrict__ stats) {
  __shared__ float sh[4];
  const int i = blockIdx.x, b = blockIdx.y;
  const size_t row = ((size_t)b * T + i) * Tp;
  const float* sr = S + row;
  const float* dr = dP + row;
  // one pass: each thread reads 4 consecutive columns per step (16-byte loads;
  // columns past i, still inside the row's Tp, are masked) and keeps its own
  // running maximum, with its sums rescaled when that moves; the threads' sums
  // are then brought to the row maximum and added in a fixed order
  float m = -INFINITY, l = 0.f, dd = 0.f;
  for (int j4 = 4 * threadIdx.x; j4 <= i; j4 += 1024) {
    const f32x4_t sv = *(const f32x4_t*)(sr + j4), dv = *(const f32x4_t*)(dr + j4);
    float x[4], mx = m;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x[k] = j4 + k <= i ? sv[k] * s : -INFINITY;
      mx = fmaxf(mx, x[k]);
    }
    const float c = __expf(m - mx);   // 0 while m is -inf
    l *= c;
    dd *= c;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float e = __expf(x[k] - mx);   // 0 for masked columns
      l += e;
      dd = fmaf(e, j4 + k <= i ? dv[k] : 0.f, dd);
    }
    m = mx;
  }
  const float M = block_max<256>(m, sh);
  const float w = m == -INFINITY ? 0.f : __expf(m - M);
  const float L = block_sum<256>(l * w, sh);
  const float DD = block_sum<256>(dd * w, sh);
  if (threadIdx.x == 0) {
    float* o = stats + ((size_t)b * T + i) * 3;
    o[0] = M; o[1] = 1.f / L; o[2] = DD / L;
  }
}

// Pass 2, one 64 x 64 tile (query rows i0.., key columns j0..) per workgroup:
// P = e^(S s - m) / l and dS' = P (dP - D) s on j <= i < T (zero elsewhere),
// written as dS' [T][Tp] (rows i) and, through LDS, as P^T and dS'^T [Tp][Tp]
// (rows j, columns i; zero for i >= T).  fp32 models only: their products read
// every tile, so every tile is written, the zeros above the diagonal included.
__global__ __launch_bounds__(256) void k_attn_tiles(const float* __restrict__ S,
                                                    const float* __restrict__ dP,
                                                    const float* __restrict__ stats, int T, int Tp,
                                                    float s, float* __restrict__ dS,
                                                    float* __restrict__ dST,
                                                    float* __restrict__ PT) {
  __shared__ float tp[BT][BT + 1], td[BT][BT + 1];
  const int j0 = blockIdx.x * BT, i0 = blockIdx.y * BT, b = blockIdx.z;
  const size_t base = (size_t)b * T * Tp;
  const bool live = j0 <= i0 + BT - 1 && i0 < T;     // some (i, j) with j <= i < T
  for (int e = threadIdx.x; e < BT * BT; e += 256) {
    const int r = e / BT, c = e % BT, i = i0 + r, j = j0 + c;
    float p = 0.f, ds = 0.f;
    if (live && i < T && j <= i) {
      const float* st = stats + ((size_t)b * T + i) * 3;
      const size_t o = base + (size_t)i * Tp + j;
      p = __expf(S[o] * s - st[0]) * st[1];
      ds = p * (dP[o] - st[2]) * s;
    }
    if (i < T) dS[base + (size_t)i * Tp + j] = ds;
    tp[r][c] = p;
    td[r][c] = ds;
  }
  __syncthreads();
  const size_t tb = (size_t)b * Tp * Tp;
  for (int e = threadIdx.x; e < BT * BT; e += 256) {
    const int c = e / BT, r = e % BT;
    const size_t o = tb + (size_t)(j0 + c) * Tp + i0 + r;
    PT[o] = tp[r][c];
    dST[o] = td[r][c];
  }
}

// Pass 1 and 2 of the attention backward for bf16 models with the scores never
// stored.  One workgroup per (64-query block, head of the batch), wave w the
// queries 16 w .. 16 w + 15 of the block.  For every key block at or below the
// diagonal, S = q k^T and dP = do v^T come from the matrix cores (16x16x32 bf16
// products, fp32 sums over the head dimension in k-step order; the block's K and
// V rows staged in LDS, the next block's rows loaded into registers meanwhile).
// The first pass keeps each lane's running maximum of S s and its rescaled sums
// of e^(S s - max) and e^(S s - max) dP over its own columns; the 16 lanes of a
// row then combine theirs in a fixed butterfly, so every lane holds the row's
// max m, 1/l and D = sum P dP.  The second pass forms P = e^(S s - m) / l and
// dS' = P (dP - D) s (the tile kernel's expressions) and writes them as that
// kernel does: dS' by rows, P^T and dS'^T through LDS, in 16-byte pieces.  Above
// the diagonal only the band tile the causal products read (row tiles of
// kTiledRows) is written, as zeros.  Rows at or past T are zeros (their query
// loads re-read row T - 1); key rows past T are read from the padded K and V
// (within Tp) and masked.
template <int HD>
__global__ __launch_bounds__(256) void k_attn_bwd_scores(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ dO, int ldq,
    const bf16_t* __restrict__ kb, const bf16_t* __restrict__ vb, int gq, int T, int Tp, float s,
    bf16_t* __restrict__ dS, bf16_t* __restrict__ dST, bf16_t* __restrict__ PT) {
  constexpr int QS = HD / 32;            // MFMA k-steps over the head dimension
  constexpr int KROW = HD + 8;           // LDS row of a K or V tile (16-byte pad)
  constexpr int PR = HD / 8;             // 16-byte pieces per row
  constexpr int PPT = 64 * PR / 256;     // pieces per thread and tile
  static_assert(kTiledRows == 128, "band of two 64-row blocks");
  __shared__ __attribute__((aligned(16))) bf16_t ks[64 * KROW];
  __shared__ __attribute__((aligned(16))) bf16_t vs[64 * KROW];
  __shared__ float tp[64][65], td[64][65];

  const int nqb = Tp / 64;
  const int qb = nqb - 1 - (int)blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
  const int j = lane & 15, lg = lane >> 4;
  const int i0 = qb * 64;
  const bf16_t* kg = kb + (size_t)(b / gq) * Tp * HD;
  const bf16_t* vg = vb + (size_t)(b / gq) * Tp * HD;
  bf16_t* dSb = dS + (size_t)b * T * Tp;
  const size_t tb = (size_t)b * Tp * Tp;
  const u32x4_t zero = {0u, 0u, 0u, 0u};

  // the band tile above the diagonal (read by the causal products): zeros
  if (qb % 2 == 0 && qb + 1 < nqb) {
    const int j0 = i0 + 64;
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      const int r = pass * 32 + tid / 8, u = tid % 8;
      if (i0 + r < T) *(u32x4_t*)(dSb + (size_t)(i0 + r) * Tp + j0 + 8 * u) = zero;
      *(u32x4_t*)(PT + tb + (size_t)(j0 + r) * Tp + i0 + 8 * u) = zero;
      *(u32x4_t*)(dST + tb + (size_t)(j0 + r) * Tp + i0 + 8 * u) = zero;
    }
  }

  // A operands: this lane's query row (clamped below T), k-step st taking the
  // head-dimension elements 32 st + 8 lg .. 32 st + 8 lg + 7
  const int qrow = min(i0 + 16 * wave + j, T - 1);
  bf16x8_t qa[QS], da[QS];
#pragma unroll
  for (int st = 0; st < QS; ++st) {
    qa[st] = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(q + (size_t)qrow * ldq + b * HD + 32 * st + 8 * lg));
    da[st] = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(dO + (size_t)qrow * ldq + b * HD + 32 * st + 8 * lg));
  }

  // key block jb: piece p of a tile is row p / PR, elements (p % PR) 8 ..
  u32x4_t pk[PPT], pv[PPT];
  auto fetch = [&](int jb) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < PPT; ++u) {
      const int p = tid + 256 * u, row = p / PR, col = (p % PR) * 8;
      pk[u] = *(const u32x4_t*)(kg + (size_t)(jb * 64 + row) * HD + col);
      pv[u] = *(const u32x4_t*)(vg + (size_t)(jb * 64 + row) * HD + col);
    }
  };
  auto stash = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < PPT; ++u) {
      const int p = tid + 256 * u, row = p / PR, col = (p % PR) * 8;
      *(u32x4_t*)(ks + row * KROW + col) = pk[u];
      *(u32x4_t*)(vs + row * KROW + col) = pv[u];
    }
  };
  // S and dP of the staged block: column block c holds keys 16 c .. 16 c + 15;
  // lane (j, lg) gets rows 4 lg .. 4 lg + 3 of its wave's queries, column j
  f32x4_t as[4], ap[4];
  auto products = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      f32x4_t x = {0.f, 0.f, 0.f, 0.f}, y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < QS; ++st) {
        const bf16x8_t kf = *(const bf16x8_t*)(ks + (16 * c + j) * KROW + 32 * st + 8 * lg);
        const bf16x8_t vf = *(const bf16x8_t*)(vs + (16 * c + j) * KROW + 32 * st + 8 * lg);
        x = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[st], kf, x, 0, 0, 0);
        y = __builtin_amdgcn_mfma_f32_16x16x32_bf16(da[st], vf, y, 0, 0, 0);
      }
      as[c] = x;
      ap[c] = y;
    }
  };

  // pass 1: row statistics
  float m[4], l[4], dd[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) { m[v] = -INFINITY; l[v] = 0.f; dd[v] = 0.f; }
  fetch(0);
  for (int jb = 0; jb <= qb; ++jb) {
    __syncthreads();
    stash();
    __syncthreads();
    if (jb < qb) fetch(jb + 1);
    products();
    const bool diag = jb == qb;   // below it every key precedes every query
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int i = i0 + 16 * wave + 4 * lg + v;
      float x[4], mx = m[v];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        x[c] = !diag || jb * 64 + 16 * c + j <= i ? as[c][v] * s : -INFINITY;
        mx = fmaxf(mx, x[c]);
      }
      if (mx != -INFINITY) {
        const float cf = __expf(m[v] - mx);   // 0 while m is -inf
        l[v] *= cf;
        dd[v] *= cf;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const float e = __expf(x[c] - mx);   // 0 for masked keys
          l[v] += e;
          dd[v] = fmaf(e, x[c] != -INFINITY ? ap[c][v] : 0.f, dd[v]);
        }
        m[v] = mx;
      }
    }
  }
  float il[4], D[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      const float m2 = __shfl_xor(m[v], off, 64), l2 = __shfl_xor(l[v], off, 64),
                  d2 = __shfl_xor(dd[v], off, 64);
      const float M = fmaxf(m[v], m2);
      const float a = m[v] == -INFINITY ? 0.f : __expf(m[v] - M);
      const float c2 = m2 == -INFINITY ? 0.f : __expf(m2 - M);
      l[v] = l[v] * a + l2 * c2;
      dd[v] = dd[v] * a + d2 * c2;
      m[v] = M;
    }
    il[v] = 1.f / l[v];
    D[v] = dd[v] / l[v];
  }

  // pass 2: P and dS' of every block, written as the tile kernel writes them
  fetch(0);
  for (int jb = 0; jb <= qb; ++jb) {
    __syncthreads();
    stash();
    __syncthreads();
    if (jb < qb) fetch(jb + 1);
    products();
    const bool diag = jb == qb;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = 16 * wave + 4 * lg + v, i = i0 + r;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const bool ok = (!diag || jb * 64 + 16 * c + j <= i) && i < T;
        const float pv_ = __expf(as[c][v] * s - m[v]) * il[v];
        const float dsv = pv_ * (ap[c][v] - D[v]) * s;
        tp[r][16 * c + j] = ok ? pv_ : 0.f;
        td[r][16 * c + j] = ok ? dsv : 0.f;
      }
    }
    __syncthreads();
    const int j0 = jb * 64;
    {
      const int r = tid / 4, qq = tid % 4, i = i0 + r;
      if (i < T) {
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          u32x4_t w;
#pragma unroll
          for (int k = 0; k < 4; ++k)
            w[k] = pack_bf16x2(td[r][32 * g + 8 * qq + 2 * k], td[r][32 * g + 8 * qq + 2 * k + 1]);
          *(u32x4_t*)(dSb + (size_t)i * Tp + j0 + 32 * g + 8 * qq) = w;
        }
      }
    }
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      const int c = pass * 32 + tid / 8, u = tid % 8;
      u32x4_t wp, wd;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        wp[k] = pack_bf16x2(tp[8 * u + 2 * k][c], tp[8 * u + 2 * k + 1][c]);
        wd[k] = pack_bf16x2(td[8 * u + 2 * k][c], td[8 * u + 2 * k + 1][c]);
      }
      const size_t o = tb + (size_t)(j0 + c) * Tp + i0 + 8 * u;
      *(u32x4_t*)(PT + o) = wp;
      *(u32x4_t*)(dST + o) = wd;
    }
  }
}

// Sum over each kv group's heads: out[t][g hd + e] = sum_j tmp[g gq + j][t][e].
__global__ __launch_bounds__(256) void k_sum_heads(const float* __restrict__ tmp, int T, int hd,
                                                   int gq, int groups, float* __restrict__ out,
                                                   int ldo) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)groups * T * hd) return;
  const int e = (int)(i % hd);
  const size_t t = (i / hd) % T;
  const int g = (int)(i / ((size_t)hd * T));
  float s = 0.f;
  for (int j = 0; j < gq; ++j) s += tmp[(((size_t)g * gq + j) * T + t) * hd + e];
  out[t * ldo + (size_t)g * hd + e] = s;
}

// Embedding gradient demb[tok[t]] += dx[t] without atomics, in a fixed order:
// the keys (tok[t] << 14) | t are sorted (one workgroup, bitonic in LDS), then
// every run of equal tokens is summed in increasing t by the workgroup at its
// first sorted index, which alone owns that embedding row in this call.
constexpr int kEmbedKeyBits = 14;                    // t < 16384
constexpr int kEmbedSortMax = 1 << kEmbedKeyBits;    // keys sorted in LDS

__global__ __launch_bounds__(1024) void k_embed_sort(const int32_t* __restrict__ tok, int T, int V,
                                                     uint32_t* __restrict__ keys) {
  __shared__ uint32_t k[kEmbedSortMax];
  int n = 1;
  while (n < T) n <<= 1;
  for (int i = threadIdx.x; i < n; i += 1024)
    k[i] = i < T ? ((uint32_t)clampi(tok[i], 0, V - 1) << kEmbedKeyBits) | (uint32_t)i
                 : 0xffffffffu;
  __syncthreads();
  for (int w = 2; w <= n; w <<= 1)
    for (int j = w >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < n; i += 1024) {
        const int l = i ^ j;
        if (l > i) {
          const uint32_t a = k[i], b = k[l];
          if ((a > b) == ((i & w) == 0)) { k[i] = b; k[l] = a; }
        }
      }
      __syncthreads();
    }
  for (int i = threadIdx.x; i < T; i += 1024) keys[i] = k[i];
}

__global__ __launch_bounds__(256) void k_embed_bwd(const uint32_t* __restrict__ keys, int T,
                                                   const float* __restrict__ dx, int d,
                                                   float* __restrict__ demb) {
  const int i = blockIdx.x;
  const uint32_t v = keys[i] >> kEmbedKeyBits;
  if (i > 0 && (keys[i - 1] >> kEmbedKeyBits) == v) return;   // not the run's first
  float* row = demb + (size_t)v * d;
  for (int c = threadIdx.x; c < d; c += 256) {
    float acc = 0.f;
    for (int j = i; j < T && (keys[j] >> kEmbedKeyBits) == v; ++j)
      acc += dx[(size_t)(keys[j] & (kEmbedSortMax - 1)) * d + c];
    row[c] += acc;
  }
}

__global__ __launch_bounds__(256) void k_fill_f32(float* p, size_t n, float v) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

template <typename TI, typename TO>
__global__ __launch_bounds__(256) void k_cast(const TI* __restrict__ in, size_t n, TO* __restrict__ out) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) stf(out, i, ldf(in, i));
}

// AdamW: m = b1 m + (1 - b1) g, v = b2 v + (1 - b2) g^2, p -= lr wd p + lr mhat /
// (sqrt(vhat) + eps) on the fp32 master; the model copy gets the rounded value.
template <typename TP>
__global__ __launch_bounds__(256) void k_adamw(TP* __restrict__ param, float* __restrict__ master,
                                               float* __restrict__ m, float* __restrict__ v,
                                               const float* __restrict__ grad, size_t n, float lr,
                                               float b1, float b2, float eps, float wd, float bc1,
                                               float bc2) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const float g = grad[i];
  const float mi = b1 * m[i] + (1.f - b1) * g;
  const float vi = b2 * v[i] + (1.f - b2) * g * g;
  m[i] = mi;
  v[i] = vi;
  float p = master ? master[i] : ldf(param, i);
  p = p - lr * wd * p - lr * (mi / bc1) / (sqrtf(vi / bc2) + eps);
  if (master) master[i] = p;
  stf(param, i, p);
}

inline unsigned blocks(size_t n) { return (unsigned)((n + 255) / 256); }

}  // namespace

hipError_t transpose(int tin, int tout, const void* in, int ldi, size_t in_bs, int R, int C,
                     void* out, int ldo, size_t s1, size_t s2, int div, int Rpad, int batch,
                     hipStream_t st) {
  if (R <= 0 || C <= 0 || batch <= 0) return hipSuccess;
  if (Rpad < R || div < 1) return hipErrorInvalidValue;
  dim3 grid((Rpad + BT - 1) / BT, (C + BT - 1) / BT, batch);
  Prof pf("transpose", st);
  const size_t ei = tin == 0 ? 4 : 2, eo = tout == 0 ? 4 : 2;
  const int vec = (uintptr_t)in % 16 == 0 && (uintptr_t)out % 16 == 0 && ldi * ei % 16 == 0 &&
                  in_bs * ei % 16 == 0 && ldo * eo % 16 == 0 && s1 * eo % 16 == 0 &&
                  s2 * eo % 16 == 0;
  if (tin == 0 && tout == 0)
    k_transpose<float, float><<<grid, 256, 0, st>>>((const float*)in, ldi, in_bs, R, C, (float*)out,
                                                    ldo, s1, s2, div, Rpad, vec);
  else if (tin == 0)
    k_transpose<float, bf16_t><<<grid, 256, 0, st>>>((const float*)in, ldi, in_bs, R, C,
                                                     (bf16_t*)out, ldo, s1, s2, div, Rpad, vec);
  else if (tout == 1)
    k_transpose<bf16_t, bf16_t><<<grid, 256, 0, st>>>((const bf16_t*)in, ldi, in_bs, R, C,
                                                      (bf16_t*)out, ldo, s1, s2, div, Rpad, vec);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t dlogits(int dtype, const float* z, int R, int V, int ldz, const int32_t* tgt,
                   int tstride, const float* g, float temperature, void* dz, int ldo,
                   hipStream_t st) {
  if (R <= 0) return hipSuccess;
  const float inv_t = 1.f / (temperature > 0.f ? temperature : 1.f);
  Prof pf("dlogits", st);
  if (dtype == 0) k_dlogits<float><<<R, 256, 0, st>>>(z, V, ldz, tgt, tstride, g, inv_t, (float*)dz, ldo);
  else k_dlogits<bf16_t><<<R, 256, 0, st>>>(z, V, ldz, tgt, tstride, g, inv_t, (bf16_t*)dz, ldo);
  return hipGetLastError();
}

hipError_t rmsnorm_bwd(int dtype, const float* x, int ldx, const void* g, const float* dy, int ldy,
                       int T, int d, float eps, float* dres, void* dres_e, float* rr, float* part,
                       float* dg, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  Prof pf("rmsnorm_bwd", st);
  if (dtype == 0)
    k_rmsnorm_bwd<float><<<T, 256, 0, st>>>(x, ldx, (const float*)g, dy, ldy, d, eps, dres,
                                            (float*)dres_e, rr);
  else
    k_rmsnorm_bwd<bf16_t><<<T, 256, 0, st>>>(x, ldx, (const bf16_t*)g, dy, ldy, d, eps, dres,
                                             (bf16_t*)dres_e, rr);
  const int chunks = (T + 63) / 64;
  k_norm_dg_part<<<dim3((d + 255) / 256, chunks), 256, 0, st>>>(x, ldx, dy, ldy, rr, T, d, part);
  k_norm_dg_sum<<<(d + 255) / 256, 256, 0, st>>>(part, chunks, d, dg);
  return hipGetLastError();
}

hipError_t swiglu_fwd(int dtype, const float* gu, int T, int F, void* a, hipStream_t st) {
  const size_t n = (size_t)T * F;
  if (n == 0) return hipSuccess;
  Prof pf("swiglu_fwd", st);
  if (F % 4 == 0 && n / 4 < (1u << 31) && (uintptr_t)gu % 16 == 0 && (uintptr_t)a % 16 == 0) {
    if (dtype == 0) k_swiglu_fwd4<float><<<blocks(n / 4), 256, 0, st>>>(gu, T, F, (float*)a);
    else k_swiglu_fwd4<bf16_t><<<blocks(n / 4), 256, 0, st>>>(gu, T, F, (bf16_t*)a);
  } else if (dtype == 0) {
    k_swiglu_fwd<float><<<blocks(n), 256, 0, st>>>(gu, T, F, (float*)a);
  } else {
    k_swiglu_fwd<bf16_t><<<blocks(n), 256, 0, st>>>(gu, T, F, (bf16_t*)a);
  }
  return hipGetLastError();
}

hipError_t swiglu_bwd(int dtype, const float* gu, const float* da, int T, int F, void* dgu,
                      hipStream_t st) {
  const size_t n = (size_t)T * F;
  if (n == 0) return hipSuccess;
  Prof pf("swiglu_bwd", st);
  if (F % 4 == 0 && n / 4 < (1u << 31) && (uintptr_t)gu % 16 == 0 && (uintptr_t)da % 16 == 0 &&
      (uintptr_t)dgu % 16 == 0) {
    if (dtype == 0) k_swiglu_bwd4<float><<<blocks(n / 4), 256, 0, st>>>(gu, da, T, F, (float*)dgu);
    else k_swiglu_bwd4<bf16_t><<<blocks(n / 4), 256, 0, st>>>(gu, da, T, F, (bf16_t*)dgu);
  } else if (dtype == 0) {
    k_swiglu_bwd<float><<<blocks(n), 256, 0, st>>>(gu, da, T, F, (float*)dgu);
  } else {
    k_swiglu_bwd<bf16_t><<<blocks(n), 256, 0, st>>>(gu, da, T, F, (bf16_t*)dgu);
  }
  return hipGetLastError();
}

hipError_t rope_bwd(int dtype, float* dqkv, int T, int heads, int n_rot, int hd, const float2* cs,
                    void* out, hipStream_t st) {
  const size_t n = (size_t)T * heads * (hd / 2);
  if (n == 0) return hipSuccess;
  Prof pf("rope_bwd", st);
  if (dtype == 0) k_rope_bwd<float><<<blocks(n), 256, 0, st>>>(dqkv, T, heads, n_rot, hd, cs, (float*)out);
  else k_rope_bwd<bf16_t><<<blocks(n), 256, 0, st>>>(dqkv, T, heads, n_rot, hd, cs, (bf16_t*)out);
  return hipGetLastError();
}

hipError_t attn_softmax_bwd(int dtype, const float* S, const float* dP, int T, int Tp, int batch,
                            float scale, float* stats, void* dS, void* dST, void* PT,
                            hipStream_t st) {
  if (T <= 0 || batch <= 0) return hipSuccess;
  // fp32 models only: bf16 models form the scores inside attn_scores_bwd
  if (dtype != 0 || Tp % BT || Tp < T) return hipErrorInvalidValue;
  Prof pf("attn_softmax_bwd", st);
  k_attn_row_stats<<<dim3(T, batch), 256, 0, st>>>(S, dP, T, Tp, scale, stats);
  const dim3 grid(Tp / BT, Tp / BT, batch);
  k_attn_tiles<<<grid, 256, 0, st>>>(S, dP, stats, T, Tp, scale, (float*)dS, (float*)dST,
                                     (float*)PT);
  return hipGetLastError();
}

hipError_t attn_scores_bwd(const void* q, const void* dO, int ldq, const void* kb, const void* vb,
                          int gq, int T, int Tp, int batch, int hd, float scale, void* dS,
                          void* dST, void* PT, hipStream_t st) {
  if (T <= 0 || batch <= 0) return hipSuccess;
  auto a16 = [](const void* p) { return (uintptr_t)p % 16 == 0; };
  if (Tp % 64 || Tp < T || (hd != 64 && hd != 128) || gq < 1 || batch % gq || ldq % 8 ||
      !a16(q) || !a16(dO) || !a16(kb) || !a16(vb) || !a16(dS) || !a16(dST) || !a16(PT))
    return hipErrorInvalidValue;
  Prof pf("attn_scores_bwd", st);
  const dim3 grid(Tp / 64, batch);
  if (hd == 128)
    k_attn_bwd_scores<128><<<grid, 256, 0, st>>>((const bf16_t*)q, (const bf16_t*)dO, ldq,
                                                 (const bf16_t*)kb, (const bf16_t*)vb, gq, T, Tp,
                                                 scale, (bf16_t*)dS, (bf16_t*)dST, (bf16_t*)PT);
  else
    k_attn_bwd_scores<64><<<grid, 256, 0, st>>>((const bf16_t*)q, (const bf16_t*)dO, ldq,
                                                (const bf16_t*)kb, (const bf16_t*)vb, gq, T, Tp,
                                                scale, (bf16_t*)dS, (bf16_t*)dST, (bf16_t*)PT);
  return hipGetLastError();
}

hipError_t sum_heads(const float* tmp, int T, int hd, int gq, int groups, float* out, int ldo,
                     hipStream_t st) {
  const size_t n = (size_t)groups * T * hd;
  if (n == 0) return hipSuccess;
  Prof pf("sum_heads", st);
  k_sum_heads<<<blocks(n), 256, 0, st>>>(tmp, T, hd, gq, groups, out, ldo);
  return hipGetLastError();
}

hipError_t embed_bwd(const int32_t* tok, const float* dx, int T, int d, int V, uint32_t* keys,
                     float* demb, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  if (T > kEmbedSortMax || V < 1 || V > (1 << (32 - kEmbedKeyBits))) return hipErrorInvalidValue;
  Prof pf("embed_bwd", st);
  k_embed_sort<<<1, 1024, 0, st>>>(tok, T, V, keys);
  k_embed_bwd<<<T, 256, 0, st>>>(keys, T, dx, d, demb);
  return hipGetLastError();
}

hipError_t fill_f32(float* p, size_t n, float v, hipStream_t st) {
  if (n == 0) return hipSuccess;
  k_fill_f32<<<blocks(n), 256, 0, st>>>(p, n, v);
  return hipGetLastError();
}

hipError_t cast_f32(const float* in, size_t n, int dtype, void* out, hipStream_t st) {
  if (n == 0) return hipSuccess;
  if (dtype == 0) k_cast<float, float><<<blocks(n), 256, 0, st>>>(in, n, (float*)out);
  else k_cast<float, bf16_t><<<blocks(n), 256, 0, st>>>(in, n, (bf16_t*)out);
  return hipGetLastError();
}

hipError_t adamw(int dtype, void* param, float* master, float* m, float* v, const float* grad,
                 size_t n, float lr, float b1, float b2, float eps, float wd, int step,
                 hipStream_t st) {
  if (n == 0) return hipSuccess;
  const float bc1 = (float)(1.0 - pow((double)b1, (double)step));
  const float bc2 = (float)(1.0 - pow((double)b2, (double)step));
  Prof pf("adamw", st);
  if (dtype == 0)
    k_adamw<float><<<blocks(n), 256, 0, st>>>((float*)param, master, m, v, grad, n, lr, b1, b2, eps,
                                              wd, bc1, bc2);
  else
    k_adamw<bf16_t><<<blocks(n), 256, 0, st>>>((bf16_t*)param, master, m, v, grad, n, lr, b1, b2,
                                               eps, wd, bc1, bc2);
  return hipGetLastError();
}

}  // namespace grpo
