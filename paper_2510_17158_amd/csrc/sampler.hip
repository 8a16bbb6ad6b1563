// Next-token sampling over the LM-head logits and its log-probability.
//
// One workgroup per (row, draw).  Vocabularies up to 32768 ids are read once into
// registers (1024 threads x 32 logits); larger ones are read from L2 per pass:
//   1. max and arg-max of z = l / T (lowest id among equal maxima),
//   2. sum of exp(z - max) -> log-sum-exp (full vocabulary),
//   3. with top_k > 0: radix select (four 8-bit passes, LDS histograms with
//      integer atomics) of the k-th largest logit, ties at the cut ordered by id,
//   4. Gumbel-max over the allowed ids with Philox4x32-10 draws: one Philox
//      block per 4 consecutive ids, u = (2*(w >> 9) + 1) * 2^-24,
//      key = z - ln(-ln u); the largest key wins, the lowest id among equals.
// Every reduction is in a fixed order, so draws are bit-deterministic.
#include "common.h"
#include "kernels.h"

namespace grpo {

namespace {

constexpr int NT = 256;

__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

template <int NTH = NT>
__device__ __forceinline__ void block_argmax(float& bv, int& bi, float* shv, int* shi) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o, 64);
    const int oi = __shfl_xor(bi, o, 64);
    better(bv, bi, ov, oi);
  }
  const int w = threadIdx.x / 64;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) { shv[w] = bv; shi[w] = bi; }
  __syncthreads();
  bv = shv[0]; bi = shi[0];
  for (int i = 1; i < NTH / 64; ++i) better(bv, bi, shv[i], shi[i]);
}

__global__ __launch_bounds__(NT) void k_sample(const float* __restrict__ logits, int V, int ld,
                                               SampleArgs a) {
  __shared__ float sh[4];
  __shared__ float shv[4];
  __shared__ int shi[4];
  __shared__ int hist[256];
  __shared__ uint32_t s_prefix;
  __shared__ int s_krem, s_eq, s_cut;
  const int r = blockIdx.x, gdraw = blockIdx.y;
  const int seq = r * a.G + gdraw;
  const int pid = a.seq_ids ? a.seq_ids[seq] : seq;   // Philox sequence id
  const int col = a.step_ctr ? *a.step_ctr : 0;
  const int step = a.step + col;
  const float* l = logits + (size_t)r * ld;
  const int tid = threadIdx.x;
  const bool greedy = !(a.temperature > 0.f);
  const float T = greedy ? 1.f : a.temperature;

  // 1-2: max / arg-max and log-sum-exp of z
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int i = tid; i < V; i += NT) better(bv, bi, l[i], i);
  block_argmax(bv, bi, shv, shi);
  const float zmax = bv / T;
  float s = 0.f;
  for (int i = tid; i < V; i += NT) s += __expf(l[i] / T - zmax);
  s = block_sum<NT>(s, sh);
  const float lse = zmax + logf(s);

  int tok = bi;
  if (!greedy) {
    // 3: top-k cut
    uint32_t thr = 0;
    int cut = 0x7fffffff;
    const bool use_k = a.top_k > 0 && a.top_k < V;
    if (use_k) {
      uint32_t prefix = 0, pmask = 0;
      int krem = a.top_k;
      for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += NT) hist[i] = 0;
        __syncthreads();
        for (int i = tid; i < V; i += NT) {
          const uint32_t u = order_key(l[i]);
          if ((u & pmask) == prefix) atomicAdd(&hist[(u >> shift) & 255], 1);
        }
        __syncthreads();
        if (tid == 0) {
          int cum = 0, sel = 0;
          for (int bin = 255; bin >= 0; --bin) {
            if (cum + hist[bin] >= krem) { sel = bin; break; }
            cum += hist[bin];
          }
          s_krem = krem - cum;
          s_eq = hist[sel];
          s_prefix = prefix | ((uint32_t)sel << shift);
        }
        __syncthreads();
        krem = s_krem;
        prefix = s_prefix;
        pmask |= 255u << shift;
        __syncthreads();
      }
      thr = prefix;
      // ids equal to the cut value: keep the lowest krem of them
      if (tid == 0) {
        int c = 0x7fffffff;
        if (s_eq > krem) {
          int seen = 0;
          for (int i = 0; i < V; ++i)
            if (order_key(l[i]) == thr && ++seen == krem) { c = i; break; }
        }
        s_cut = c;
      }
      __syncthreads();
      cut = s_cut;
    }
    // 4: Gumbel-max over the allowed ids
    const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
    float gv = -INFINITY;
    int gi = 0x7fffffff;
    const int nblk = (V + 3) / 4;
    for (int c = tid; c < nblk; c += NT) {
      const uint4 w = philox4x32_10(make_uint4((uint32_t)c, (uint32_t)step, (uint32_t)pid, 0u),
                                    k0, k1);
      const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = 4 * c + j;
        if (i >= V) break;
        const float li = l[i];
        if (use_k) {
          const uint32_t u = order_key(li);
          if (!(u > thr || (u == thr && i <= cut))) continue;
        }
        better(gv, gi, gumbel_key(li, T, ws[j]), i);
      }
    }
    block_argmax(gv, gi, shv, shi);
    tok = gi;
  }
  if (tid == 0) {
    tok = clampi(tok, 0, V - 1);
    a.tok_out[(size_t)seq * a.out_stride + col] = tok;
    a.logp_out[(size_t)seq * a.out_stride + col] = l[tok] / T - lse;
    if (a.tok_state) a.tok_state[seq] = tok;
    if (a.pos_state) a.pos_state[seq] += 1;
  }
}

// The same for a vocabulary of at most NTR * 4 * R4 ids, read from memory once:
// NTR threads each hold R4 groups of 4 consecutive logits (group c = thread + NTR j,
// which is also its Philox block) in registers for every pass.
constexpr int NTR = 1024, R4 = 8;

__global__ __launch_bounds__(NTR) void k_sample_reg(const float* __restrict__ logits, int V,
                                                    int ld, SampleArgs a) {
  __shared__ float sh[NTR / 64];
  __shared__ float shv[NTR / 64];
  __shared__ int shi[NTR / 64];
  __shared__ int hist[NTR / 64][256];   // one histogram per wave
  __shared__ int hsum[256];
  __shared__ uint32_t s_prefix;
  __shared__ int s_krem, s_eq, s_cut;
  const int r = blockIdx.x, gdraw = blockIdx.y;
  const int seq = r * a.G + gdraw;
  const int pid = a.seq_ids ? a.seq_ids[seq] : seq;   // Philox sequence id
  const int col = a.step_ctr ? *a.step_ctr : 0;
  const int step = a.step + col;
  const float* l = logits + (size_t)r * ld;
  const int tid = threadIdx.x;
  const bool greedy = !(a.temperature > 0.f);
  const float T = greedy ? 1.f : a.temperature;

  // ids past V hold -inf (never the maximum, exp gives 0, excluded below)
  float x[R4][4];
#pragma unroll
  for (int j = 0; j < R4; ++j) {
    const int i0 = 4 * (tid + NTR * j);
    if (i0 + 3 < V && (ld & 3) == 0) {
      const float4 v = *(const float4*)(l + i0);
      x[j][0] = v.x; x[j][1] = v.y; x[j][2] = v.z; x[j][3] = v.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) x[j][e] = i0 + e < V ? l[i0 + e] : -INFINITY;
    }
  }

  // 1-2: max / arg-max and log-sum-exp of z
  float bv = -INFINITY;
  int bi = 0x7fffffff;
#pragma unroll
  for (int j = 0; j < R4; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) better(bv, bi, x[j][e], 4 * (tid + NTR * j) + e);
  block_argmax<NTR>(bv, bi, shv, shi);
  const float zmax = bv / T;
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < R4; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) s += __expf(x[j][e] / T - zmax);
  s = block_sum<NTR>(s, sh);
  const float lse = zmax + logf(s);

  int tok = bi;
  if (!greedy) {
    // 3: top-k cut
    uint32_t thr = 0;
    int cut = 0x7fffffff;
    const bool use_k = a.top_k > 0 && a.top_k < V;
    if (use_k) {
      uint32_t prefix = 0, pmask = 0;
      int krem = a.top_k;
      const int wave = tid / 64, lane = tid % 64;
      for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = tid; i < (NTR / 64) * 256; i += NTR) (&hist[0][0])[i] = 0;
        __syncthreads();
#pragma unroll
        for (int j = 0; j < R4; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t u = order_key(x[j][e]);
            if (4 * (tid + NTR * j) + e < V && (u & pmask) == prefix)
              atomicAdd(&hist[wave][(u >> shift) & 255], 1);
          }
        __syncthreads();
        for (int b = tid; b < 256; b += NTR) {
          int t = 0;
#pragma unroll
          for (int w = 0; w < NTR / 64; ++w) t += hist[w][b];
          hsum[b] = t;
        }
        __syncthreads();
        // the highest bin whose count, added to those of all higher bins, reaches
        // krem: lane l holds bins 255 - 4 l .. 252 - 4 l, the counts above its
        // first bin come from a scan over the lanes
        if (wave == 0) {
          const int* hb = hsum + 252 - 4 * lane;   // this lane's bins, hb[3] the highest
          const int own = hb[0] + hb[1] + hb[2] + hb[3];
          int above = own;   // inclusive scan over lanes 0 .. lane
#pragma unroll
          for (int off = 1; off < 64; off <<= 1) {
            const int v = __shfl_up(above, off, 64);
            if (lane >= off) above += v;
          }
          int cum = above - own, sel = -1, before = 0;
#pragma unroll
          for (int q = 3; q >= 0; --q) {
            const int cq = hb[q];
            if (sel < 0 && cum + cq >= krem) { sel = 252 - 4 * lane + q; before = cum; }
            cum += cq;
          }
          const unsigned long long found = __ballot(sel >= 0);
          if (found) {
            const int first = __ffsll((long long)found) - 1;
            sel = __shfl(sel, first, 64);
            before = __shfl(before, first, 64);
          } else {   // not reached: every count summed, the lowest bin
            sel = 0;
            before = __shfl(above, 63, 64);
          }
          if (lane == 0) {
            s_krem = krem - before;
            s_eq = hsum[sel];
            s_prefix = prefix | ((uint32_t)sel << shift);
          }
        }
        __syncthreads();
        krem = s_krem;
        prefix = s_prefix;
        pmask |= 255u << shift;
        __syncthreads();
      }
      thr = prefix;
      // ids equal to the cut value: keep the lowest krem of them
      if (tid == 0) {
        int c = 0x7fffffff;
        if (s_eq > krem) {
          int seen = 0;
          for (int i = 0; i < V; ++i)
            if (order_key(l[i]) == thr && ++seen == krem) { c = i; break; }
        }
        s_cut = c;
      }
      __syncthreads();
      cut = s_cut;
    }
    // 4: Gumbel-max over the allowed ids
    const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
    float gv = -INFINITY;
    int gi = 0x7fffffff;
#pragma unroll
    for (int j = 0; j < R4; ++j) {
      const int c = tid + NTR * j;
      if (4 * c < V) {
        const uint4 w = philox4x32_10(make_uint4((uint32_t)c, (uint32_t)step, (uint32_t)pid, 0u),
                                      k0, k1);
        const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = 4 * c + e;
          const float li = x[j][e];
          bool ok = i < V;
          if (use_k) {
            const uint32_t u = order_key(li);
            ok = ok && (u > thr || (u == thr && i <= cut));
          }
          if (ok) better(gv, gi, gumbel_key(li, T, ws[e]), i);
        }
      }
    }
    block_argmax<NTR>(gv, gi, shv, shi);
    tok = gi;
  }
  if (tid == 0) {
    tok = clampi(tok, 0, V - 1);
    a.tok_out[(size_t)seq * a.out_stride + col] = tok;
    a.logp_out[(size_t)seq * a.out_stride + col] = l[tok] / T - lse;
    if (a.tok_state) a.tok_state[seq] = tok;
    if (a.pos_state) a.pos_state[seq] += 1;
  }
}

// One wave per row over the decode LM head's per-tile pieces (tiles read
// lane-strided, merged in a fixed order): the arg-max, the log-sum-exp and the
// Gumbel-max of the whole vocabulary, then the sampler's outputs.
__global__ __launch_bounds__(256) void k_sample_combine(const float* __restrict__ part, int tiles,
                                                        int R, int V, SampleArgs a) {
  const int r = blockIdx.x * 4 + threadIdx.x / 64, lane = threadIdx.x % 64;
  if (r >= R) return;                      // whole waves
  const bool greedy = !(a.temperature > 0.f);
  const float T = greedy ? 1.f : a.temperature;
  const float* p = part + (size_t)r * tiles * 8;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int t = lane; t < tiles; t += 64) better(bv, bi, p[t * 8], __float_as_int(p[t * 8 + 2]));
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o, 64);
    const int oi = __shfl_xor(bi, o, 64);
    better(bv, bi, ov, oi);
  }
  const float zmax = bv / T;
  float s = 0.f;
  for (int t = lane; t < tiles; t += 64) s = fmaf(p[t * 8 + 1], __expf(p[t * 8] / T - zmax), s);
  s = wave_sum(s);
  int tok = bi;
  float xt = bv;
  if (!greedy) {
    float gk = -INFINITY, gz = 0.f;
    int gi = 0x7fffffff;
    for (int t = lane; t < tiles; t += 64) {
      const float k = p[t * 8 + 3];
      const int i = __float_as_int(p[t * 8 + 4]);
      if (k > gk || (k == gk && i < gi)) { gk = k; gi = i; gz = p[t * 8 + 5]; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ok = __shfl_xor(gk, o, 64), oz = __shfl_xor(gz, o, 64);
      const int oi = __shfl_xor(gi, o, 64);
      if (ok > gk || (ok == gk && oi < gi)) { gk = ok; gi = oi; gz = oz; }
    }
    tok = gi;
    xt = gz;
  }
  if (lane == 0) {
    const int col = a.step_ctr ? *a.step_ctr : 0;
    tok = clampi(tok, 0, V - 1);
    a.tok_out[(size_t)r * a.out_stride + col] = tok;
    a.logp_out[(size_t)r * a.out_stride + col] = xt / T - (zmax + logf(s));
    if (a.tok_state) a.tok_state[r] = tok;
    if (a.pos_state) a.pos_state[r] += 1;
  }
}

}  // namespace

hipError_t sample_combine(const float* part, int tiles, int R, int V, const SampleArgs& a,
                          hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (tiles < 1 || a.G != 1 || (a.top_k > 0 && a.top_k < V)) return hipErrorInvalidValue;
  Prof pf("sample", st);
  k_sample_combine<<<(R + 3) / 4, 256, 0, st>>>(part, tiles, R, V, a);
  return hipGetLastError();
}

hipError_t sample(const float* logits, int R, int V, int ld, const SampleArgs& a, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  dim3 grid(R, a.G);
  Prof pf("sample", st);
  if (V <= NTR * 4 * R4)
    k_sample_reg<<<grid, NTR, 0, st>>>(logits, V, ld, a);
  else
    k_sample<<<grid, NT, 0, st>>>(logits, V, ld, a);
  return hipGetLastError();
}

}  // namespace grpo
