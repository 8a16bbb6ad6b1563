// Embedding gather, RMSNorm, rotary embedding + KV-cache write, and the
// teacher-forced token log-probability.  All are bandwidth-trivial next to the
// weight and KV streams; they exist as separate kernels so that every rounding
// point of the precision contract sits in one obvious place.
#include "common.h"
#include "kernels.h"

namespace grpo {

namespace {

template <typename T>
__global__ void k_embed(const T* emb, const int32_t* tok, int d, int vocab, float* x,
                        int32_t* ctr) {
  const int m = blockIdx.x;
  if (ctr && m == 0 && threadIdx.x == 0) *ctr += 1;
  const int t = clampi(tok[m], 0, vocab - 1);
  const T* e = emb + (size_t)t * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) x[(size_t)m * d + i] = ldf(e, i);
}

// x += pending split-K partials (split order), then
// h = round(x * (1 / sqrt(mean(x^2) + eps)) * g); one workgroup per row.
// Rows are read as float4 with every load of a thread issued before any use
// (the row and its partials are a few hundred KB in L2: latency, not bandwidth,
// bounds this kernel).  d must be a multiple of 4 and at most 4 * NT * VPT.
constexpr int NORM_NT = 512, NORM_VPT = 4;

template <typename T>
__device__ __forceinline__ void store4(T* out, size_t i, float4 v);
template <>
__device__ __forceinline__ void store4<float>(float* out, size_t i, float4 v) {
  *(float4*)(out + i) = v;
}
template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t* out, size_t i, float4 v) {
  const uint32_t lo = (uint32_t)f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16);
  const uint32_t hi = (uint32_t)f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16);
  *(uint2*)(out + i) = make_uint2(lo, hi);
}
template <typename T>
__device__ __forceinline__ float4 load4(const T* g, size_t i);
template <>
__device__ __forceinline__ float4 load4<float>(const float* g, size_t i) {
  return *(const float4*)(g + i);
}
template <>
__device__ __forceinline__ float4 load4<bf16_t>(const bf16_t* g, size_t i) {
  const uint2 u = *(const uint2*)(g + i);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
}

template <typename T>
__global__ __launch_bounds__(NORM_NT) void k_rmsnorm(float* x, int ldx, RowMap rm, Partials pp,
                                                     const T* g, int d, float eps, T* out,
                                                     int ldo, int pack_nb) {
  __shared__ float sh[NORM_NT / 64];
  const int m = blockIdx.x;
  const int gi = rm.i0 + m;
  const size_t src = (size_t)(gi / rm.per) * rm.stride + rm.off + gi % rm.per;
  float* xr = x + src * ldx;
  const int n4 = d / 4;
  float4 v[NORM_VPT], gv[NORM_VPT];
#pragma unroll
  for (int k = 0; k < NORM_VPT; ++k) {
    const int i4 = threadIdx.x + k * NORM_NT;
    v[k] = i4 < n4 ? *(const float4*)(xr + 4 * i4) : make_float4(0.f, 0.f, 0.f, 0.f);
    // the gain is loaded up front with the row (no second memory round trip)
    gv[k] = g && i4 < n4 ? load4(g, 4 * (size_t)i4) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  if (pp.splits > 0) {
    // four splits' loads in flight at a time (a split past the last re-reads the
    // last one and is not added), then added in split order
    const float* pr = pp.part + src * pp.ld;
    for (int sp0 = 0; sp0 < pp.splits; sp0 += 4) {
      float4 t[4][NORM_VPT];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const size_t so = (size_t)min(sp0 + u, pp.splits - 1) * pp.split_stride;
#pragma unroll
        for (int k = 0; k < NORM_VPT; ++k) {
          const int i4 = threadIdx.x + k * NORM_NT;
          t[u][k] = i4 < n4 ? *(const float4*)(pr + so + 4 * i4) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (sp0 + u < pp.splits) {
#pragma unroll
          for (int k = 0; k < NORM_VPT; ++k) {
            v[k].x += t[u][k].x; v[k].y += t[u][k].y; v[k].z += t[u][k].z; v[k].w += t[u][k].w;
          }
        }
      }
    }
#pragma unroll
    for (int k = 0; k < NORM_VPT; ++k) {
      const int i4 = threadIdx.x + k * NORM_NT;
      if (i4 < n4) *(float4*)(xr + 4 * i4) = v[k];
    }
  }
  if (!g) return;
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < NORM_VPT; ++k) {
    ss = fmaf(v[k].x, v[k].x, ss);
    ss = fmaf(v[k].y, v[k].y, ss);
    ss = fmaf(v[k].z, v[k].z, ss);
    ss = fmaf(v[k].w, v[k].w, ss);
  }
  ss = block_sum<NORM_NT>(ss, sh);
  const float r = 1.f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int k = 0; k < NORM_VPT; ++k) {
    const int i4 = threadIdx.x + k * NORM_NT;
    if (i4 < n4)
      store4(out, pack_nb ? act_frag_index(m, 4 * i4, pack_nb) : (size_t)m * ldo + 4 * i4,
             make_float4(v[k].x * r * gv[k].x, v[k].y * r * gv[k].y, v[k].z * r * gv[k].z,
                         v[k].w * r * gv[k].w));
  }
}

// one thread per (row, head, rotation pair); q heads first, then k heads, then v
template <typename T>
__global__ void k_rope_kv(const float* qkv, int M, T* q_out, RopeArgs a) {
  const int half = a.hd / 2;
  const int heads = a.n_heads + 2 * a.n_kv;
  const size_t total = (size_t)M * heads * half;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int i = (int)(idx % half);
  const int h = (int)((idx / half) % heads);
  const int m = (int)(idx / ((size_t)half * heads));
  int seq, pos;
  if (a.mode == 0) { seq = m; pos = a.pos_arr[m]; }
  else { seq = m / a.T; pos = (a.pos_arr ? a.pos_arr[seq] : a.pos0) + m % a.T; }
  const int ldq = heads * a.hd;
  const float* src = qkv + (size_t)m * ldq + h * a.hd;
  const bool rotate = h < a.n_heads + a.n_kv;
  // the cos/sin pair and up to four splits' values are loaded together, then the
  // splits are added in split order
  const float2 cs = rotate ? a.cs[(size_t)(a.mode == 0 ? m : pos) * half + i] : make_float2(1.f, 0.f);
  float lo = src[i], hi = src[i + half];
  for (int sp0 = 1; sp0 < a.splits; sp0 += 4) {
    float tl[4], th[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const size_t so = (size_t)min(sp0 + u, a.splits - 1) * a.split_stride;
      tl[u] = src[so + i];
      th[u] = src[so + i + half];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (sp0 + u < a.splits) { lo += tl[u]; hi += th[u]; }
  }
  if (rotate) {
    const float c = cs.x, s = cs.y;
    const float l2 = lo * c - hi * s;
    const float h2 = hi * c + lo * s;
    lo = l2; hi = h2;
  }
  if (a.tq || a.tk || a.tv) {
    // trace: the values as stored, fp32 rows at tmap(m) (and its copies)
    const bool is_q = h < a.n_heads, is_k = !is_q && h < a.n_heads + a.n_kv;
    float* tb = is_q ? a.tq : (is_k ? a.tk : a.tv);
    const int width = (is_q ? a.n_heads : a.n_kv) * a.hd;
    const int col = (is_q ? h : (is_k ? h - a.n_heads : h - a.n_heads - a.n_kv)) * a.hd;
    if (tb) {
      const TraceMap& tm = a.tmap;
      const size_t r0 = (size_t)(m / tm.per) * tm.stride + tm.off + m % tm.per;
      for (int r = 0; r < tm.dup; ++r) {
        float* d = tb + (r0 + (size_t)r * tm.dup_stride) * width + col;
        d[i] = rnd<T>(lo);
        d[i + half] = rnd<T>(hi);
      }
    }
  }
  if (h < a.n_heads) {
    T* qo = q_out + (size_t)m * a.n_heads * a.hd + h * a.hd;
    stf(qo, i, lo);
    stf(qo, i + half, hi);
    return;
  }
  if (pos < 0 || pos >= a.max_len) return;
  const bool is_v = h >= a.n_heads + a.n_kv;
  const int g = is_v ? h - a.n_heads - a.n_kv : h - a.n_heads;
  T* base = (T*)(is_v ? a.vcache : a.kcache);
  // with a slot map: the sequence's own cache slot; else slots seq*G .. seq*G+G-1
  const int slot0 = a.slots ? a.slots[seq] : seq * a.G;
  for (int r = 0; base && r < a.G; ++r) {
    const int slot = slot0 + r;
    if (slot < 0 || slot >= a.n_seqs) break;
    T* dst = base + (((size_t)slot * a.n_kv + g) * a.max_len + pos) * a.hd;
    stf(dst, i, lo);
    stf(dst, i + half, hi);
  }
}

// cos / sin of the rotary angles: row r of the table is position pos_arr[r]
// (pos_arr != NULL) or position r.  Angle pos * theta^(-2i/hd) in fp64, reduced
// to [-pi, pi] in fp64 (keeps sincos on its short path), cos/sin rounded to fp32.
__global__ void k_rope_table(const int32_t* pos_arr, int rows, int half, float theta,
                             float2* cs) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * half) return;
  const int r = idx / half, i = idx % half;
  const int pos = pos_arr ? pos_arr[r] : r;
  const double inv = pow((double)theta, -2.0 * (double)i / (double)(2 * half));
  const double two_pi = 6.283185307179586476925286766559;
  double ang = (double)pos * inv;
  ang -= rint(ang / two_pi) * two_pi;
  double sd, cd;
  sincos(ang, &sd, &cd);
  cs[idx] = make_float2((float)cd, (float)sd);
}

// V^T for the prefill/scoring attention: vt[slot][g][d][pos0 + p] = bf16 of the V
// part of qkv (sum of its splits) for row seq * T + p, for slots seq * vt_G ..
// seq * vt_G + vt_G - 1 (one when vt_G <= 1).  A workgroup moves a 64-position x hd
// tile through LDS, reading rows along d and writing along positions.
__global__ __launch_bounds__(256) void k_v_transpose(const float* qkv, int T, RopeArgs a,
                                                     bf16_t* vt) {
  __shared__ float tile[64][129];
  const int p0 = blockIdx.x * 64, g = blockIdx.y, seq = blockIdx.z;
  const int hd = a.hd;
  const int ldq = (a.n_heads + 2 * a.n_kv) * hd;
  const float* src = qkv + (size_t)seq * T * ldq + (size_t)(a.n_heads + a.n_kv + g) * hd;
  for (int e = threadIdx.x; e < 64 * hd; e += 256) {
    const int p = e / hd, d = e % hd;
    float v = 0.f;
    if (p0 + p < T) {
      const float* r = src + (size_t)(p0 + p) * ldq + d;
      v = r[0];
      for (int sp = 1; sp < a.splits; ++sp) v += r[sp * a.split_stride];
    }
    tile[p][d] = v;
  }
  __syncthreads();
  const int vg = max(a.vt_G, 1);
  for (int r = 0; r < vg; ++r) {
    bf16_t* dst = vt + (((size_t)seq * vg + r) * a.n_kv + g) * hd * a.vt_len;
    for (int e = threadIdx.x; e < 64 * hd; e += 256) {
      const int d = e / 64, p = e % 64, t = a.pos0 + p0 + p;
      if (t < a.vt_len) dst[(size_t)d * a.vt_len + t] = p0 + p < T ? f2bf(tile[p][d]) : 0;
    }
  }
}

// Trace copy (debug path): element (m, i) of a source laid out as `layout`
// into fp32 row map(m) of dst; one thread per element.
__global__ void k_trace_rows(const void* src, int layout, int ld, int M, int width, TraceMap tm,
                             float* dst) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)M * width) return;
  const int m = (int)(idx / width), i = (int)(idx % width);
  float v;
  if (layout == TR_F32) v = ((const float*)src)[(size_t)m * ld + i];
  else if (layout == TR_BF16) v = bf2f(((const bf16_t*)src)[(size_t)m * ld + i]);
  else v = bf2f(((const bf16_t*)src)[act_frag_index(m, i, ld)]);
  const size_t r0 = (size_t)(m / tm.per) * tm.stride + tm.off + m % tm.per;
  for (int r = 0; r < tm.dup; ++r) dst[(r0 + (size_t)r * tm.dup_stride) * width + i] = v;
}

struct I32Block {
  int32_t v[128];
};
__global__ void k_set_i32(int32_t* dst, I32Block b, int n) {
  if ((int)threadIdx.x < n) dst[threadIdx.x] = b.v[threadIdx.x];
}

// V^T of cached sequences for the prefill/scoring attention: vt[b][g][d][t] =
// V[slots[b]][g][t][d] for t < pos0[b] + T, 0 up to vt_len.  A workgroup moves a
// 64-position x hd tile through LDS.
__global__ __launch_bounds__(256) void k_cache_vt(const bf16_t* vc, const int32_t* slots,
                                                  const int32_t* pos0, int T, int n_kv,
                                                  int max_len, int hd, int vt_len, bf16_t* vt) {
  __shared__ bf16_t tile[64][130];
  const int p0 = blockIdx.x * 64, g = blockIdx.y, b = blockIdx.z;
  const int len = pos0[b] + T;
  const bf16_t* src = vc + ((size_t)slots[b] * n_kv + g) * max_len * hd;
  for (int e = threadIdx.x; e < 64 * hd; e += 256) {
    const int p = e / hd, d = e % hd;
    tile[p][d] = p0 + p < len ? src[(size_t)(p0 + p) * hd + d] : (bf16_t)0;
  }
  __syncthreads();
  bf16_t* dst = vt + ((size_t)b * n_kv + g) * hd * vt_len;
  for (int e = threadIdx.x; e < 64 * hd; e += 256) {
    const int d = e / 64, p = e % 64;
    if (p0 + p < vt_len) dst[(size_t)d * vt_len + p0 + p] = tile[p][d];
  }
}

// per-row position and cache slot of B sequences x T rows: row m of sequence b
// is position pos0[b] + m % T of slot slots[b]
__global__ void k_row_positions(const int32_t* pos0, const int32_t* slots, int B, int T,
                                int32_t* row_pos, int32_t* row_slot) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= B * T) return;
  row_pos[m] = pos0[m / T] + m % T;
  row_slot[m] = slots[m / T];
}

__global__ void k_fill_i32(int32_t* p, size_t n, int32_t v) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// logp[r] from the LM head's log-sum-exp pieces: one wave per row, slots read
// lane-strided (fixed order), then the wave's max and sum.
__global__ __launch_bounds__(256) void k_lse_combine(const float2* __restrict__ part, int slots,
                                                     const float* __restrict__ tgt_z, int R,
                                                     float temp, float* __restrict__ logp) {
  const int r = blockIdx.x * 4 + threadIdx.x / 64, lane = threadIdx.x % 64;
  if (r >= R) return;                       // whole waves
  const float2* p = part + (size_t)r * slots;
  float mx = -INFINITY;
  for (int s = lane; s < slots; s += 64) mx = fmaxf(mx, p[s].x);
  mx = wave_max(mx);
  float sum = 0.f;
  for (int s = lane; s < slots; s += 64) {
    const float2 v = p[s];
    sum = fmaf(v.y, __builtin_amdgcn_exp2f(v.x - mx), sum);
  }
  sum = wave_sum(sum);
  if (lane == 0) logp[r] = tgt_z[r] / temp - 0.693147180559945309f * (mx + __log2f(sum));
}

}  // namespace

hipError_t embed(int dtype, const void* emb, const int32_t* tok, int M, int d, int vocab, float* x,
                 hipStream_t st, int32_t* ctr) {
  if (M <= 0) return hipSuccess;
  Prof pf("embed", st);
  if (dtype == 0) k_embed<float><<<M, 256, 0, st>>>((const float*)emb, tok, d, vocab, x, ctr);
  else k_embed<bf16_t><<<M, 256, 0, st>>>((const bf16_t*)emb, tok, d, vocab, x, ctr);
  return hipGetLastError();
}

hipError_t rmsnorm(int dtype, float* x, int ldx, RowMap rows, Partials p, const void* g, int M,
                   int d, float eps, void* out, int ldo, hipStream_t st, int pack_nb) {
  if (M <= 0) return hipSuccess;
  if (pack_nb && (dtype == 0 || M > pack_nb || pack_nb % 16 || d % 32)) return hipErrorInvalidValue;
  Prof pf(M <= 128 ? "rmsnorm" : "rmsnorm_rows", st);
  if (d % 4 || d > 4 * NORM_NT * NORM_VPT) return hipErrorInvalidValue;
  if (dtype == 0)
    k_rmsnorm<float><<<M, NORM_NT, 0, st>>>(x, ldx, rows, p, (const float*)g, d, eps,
                                            (float*)out, ldo, 0);
  else
    k_rmsnorm<bf16_t><<<M, NORM_NT, 0, st>>>(x, ldx, rows, p, (const bf16_t*)g, d, eps,
                                             (bf16_t*)out, ldo, pack_nb);
  return hipGetLastError();
}

hipError_t fill_i32(int32_t* p, size_t n, int32_t v, hipStream_t st) {
  if (n == 0) return hipSuccess;
  Prof pf("fill", st);
  k_fill_i32<<<(int)((n + 255) / 256), 256, 0, st>>>(p, n, v);
  return hipGetLastError();
}

hipError_t set_i32(int32_t* dst, const int32_t* host_vals, int n, hipStream_t st) {
  for (int i0 = 0; i0 < n; i0 += 128) {
    const int k = n - i0 < 128 ? n - i0 : 128;
    I32Block b{};
    for (int i = 0; i < k; ++i) b.v[i] = host_vals[i0 + i];
    Prof pf("set", st);
    k_set_i32<<<1, 128, 0, st>>>(dst + i0, b, k);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t trace_rows(const void* src, int layout, int ld, int M, int width, TraceMap map,
                      float* dst, hipStream_t st) {
  const size_t n = (size_t)M * width;
  if (n == 0 || !dst) return hipSuccess;
  if (map.per <= 0 || map.dup < 1 || (layout == TR_FRAG && (ld % 16 || width % 32 || M > ld)))
    return hipErrorInvalidValue;
  Prof pf("trace", st);
  k_trace_rows<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(src, layout, ld, M, width, map, dst);
  return hipGetLastError();
}

hipError_t cache_vt(const void* vc, const int32_t* slots, const int32_t* pos0, int B, int T,
                    int n_kv, int max_len, int hd, int vt_len, uint16_t* vt, hipStream_t st) {
  if (B <= 0) return hipSuccess;
  Prof pf("cache_vt", st);
  k_cache_vt<<<dim3((vt_len + 63) / 64, n_kv, B), 256, 0, st>>>(
      (const bf16_t*)vc, slots, pos0, T, n_kv, max_len, hd, vt_len, (bf16_t*)vt);
  return hipGetLastError();
}

hipError_t row_positions(const int32_t* pos0, const int32_t* slots, int B, int T,
                         int32_t* row_pos, int32_t* row_slot, hipStream_t st) {
  const int n = B * T;
  if (n <= 0) return hipSuccess;
  Prof pf("row_positions", st);
  k_row_positions<<<(n + 255) / 256, 256, 0, st>>>(pos0, slots, B, T, row_pos, row_slot);
  return hipGetLastError();
}

hipError_t rope_table(const int32_t* pos_arr, int rows, int hd, float theta, float2* cs,
                      hipStream_t st) {
  const int n = rows * (hd / 2);
  if (n <= 0) return hipSuccess;
  Prof pf("rope_table", st);
  k_rope_table<<<(n + 255) / 256, 256, 0, st>>>(pos_arr, rows, hd / 2, theta, cs);
  return hipGetLastError();
}

hipError_t rope_kv(int dtype, const float* qkv, int M, void* q_out, const RopeArgs& a,
                   hipStream_t st) {
  const size_t total = (size_t)M * (a.n_heads + 2 * a.n_kv) * (a.hd / 2);
  if (total == 0) return hipSuccess;
  if (!a.cs || a.hd > 128) return hipErrorInvalidValue;
  const int grid = (int)((total + 255) / 256);
  {
    Prof pf(a.mode == 0 ? "rope_kv" : "rope_kv_rows", st);
    if (dtype == 0) k_rope_kv<float><<<grid, 256, 0, st>>>(qkv, M, (float*)q_out, a);
    else k_rope_kv<bf16_t><<<grid, 256, 0, st>>>(qkv, M, (bf16_t*)q_out, a);
  }
  if (a.vt && a.mode == 1 && a.T > 0) {
    Prof pf("v_transpose", st);
    dim3 grid_t((a.T + 63) / 64, a.n_kv, M / a.T);
    k_v_transpose<<<grid_t, 256, 0, st>>>(qkv, a.T, a, a.vt);
  }
  return hipGetLastError();
}

hipError_t lse_combine(const float* part, int slots, const float* tgt_z, int R,
                       float temperature, float* logp, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (slots < 1) return hipErrorInvalidValue;
  const float t = temperature > 0.f ? temperature : 1.f;
  Prof pf("lse_combine", st);
  k_lse_combine<<<(R + 3) / 4, 256, 0, st>>>((const float2*)part, slots, tgt_z, R, t, logp);
  return hipGetLastError();
}

}  // namespace grpo
