// Shared device helpers of the HIP path (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define GRPO_WAVE 64

typedef uint16_t bf16_t;  // bf16 stored as its bit pattern

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// ---- bf16 <-> fp32 ---------------------------------------------------------
__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// round-to-nearest-even fp32 -> bf16 (NaN stays a quiet NaN)
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// storage-type generic loads/stores: T is float (fp32 models) or bf16_t
template <typename T> __device__ __forceinline__ float ldf(const T* p, size_t i);
template <> __device__ __forceinline__ float ldf<float>(const float* p, size_t i) { return p[i]; }
template <> __device__ __forceinline__ float ldf<bf16_t>(const bf16_t* p, size_t i) {
  return bf2f(p[i]);
}
template <typename T> __device__ __forceinline__ void stf(T* p, size_t i, float v);
template <> __device__ __forceinline__ void stf<float>(float* p, size_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void stf<bf16_t>(bf16_t* p, size_t i, float v) {
  p[i] = f2bf(v);
}
// value as it is stored: identity for fp32, bf16 rounding for bf16
template <typename T> __device__ __forceinline__ float rnd(float v);
template <> __device__ __forceinline__ float rnd<float>(float v) { return v; }
template <> __device__ __forceinline__ float rnd<bf16_t>(float v) { return bf2f(f2bf(v)); }

// ---- wavefront reductions (DPP/shuffle via __shfl_xor) ----------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, GRPO_WAVE);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, GRPO_WAVE));
  return v;
}
__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, GRPO_WAVE);
  return v;
}

// block-wide sum in a fixed order (wave partials summed by wave index)
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x / GRPO_WAVE, l = threadIdx.x % GRPO_WAVE;
  __syncthreads();
  if (l == 0) sh[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < NT / GRPO_WAVE; ++i) t += sh[i];
  return t;
}
template <int NT>
__device__ __forceinline__ float block_max(float v, float* sh) {
  v = wave_max(v);
  const int w = threadIdx.x / GRPO_WAVE, l = threadIdx.x % GRPO_WAVE;
  __syncthreads();
  if (l == 0) sh[w] = v;
  __syncthreads();
  float t = -INFINITY;
#pragma unroll
  for (int i = 0; i < NT / GRPO_WAVE; ++i) t = fmaxf(t, sh[i]);
  return t;
}

__device__ __forceinline__ int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// SwiGLU's silu(g) * u in fp32: g / (1 + e^-g) with the hardware exponential and
// reciprocal (each within about 1 ulp), then the product by u.
__device__ __forceinline__ float silu_mul(float g, float u) {
  return g * __builtin_amdgcn_rcpf(1.f + __expf(-g)) * u;
}

// ---- fragment order of the decode GEMM's activations ---------------------------
// Element (b, k) of an activation [nb][K] (nb: the padded batch, a multiple of 16)
// stored as MFMA B-operand fragments: fragment (k / 32, b / 16) is 1 KB, lane
// (b % 16) + 16 ((k / 8) % 4) holding elements k % 8 = 0..7; fragments ordered by
// k step, then batch block.
__device__ __forceinline__ size_t act_frag_index(int b, int k, int nb) {
  return ((size_t)(k >> 5) * (nb >> 4) + (b >> 4)) * 512 + ((b & 15) + 16 * ((k >> 3) & 3)) * 8 +
         (k & 7);
}

// ---- direct-to-LDS copies ---------------------------------------------------------
// One copy of 16 bytes per lane (global_load_lds_dwordx4): the 64 lanes of the wave
// fill the 1 KB at LDS byte address `lds` (wave-uniform) in lane order, each lane
// naming its own source.  Issued as one asm statement that also sets M0, so the
// compiler does not serialise consecutive copies (it cannot prove they write
// disjoint LDS); the kernel waits for them itself (s_waitcnt vmcnt) before the
// barrier that publishes the data.
__device__ __forceinline__ void dma16(const bf16_t* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(g) : "memory");
}
// The same with a wave-uniform base address and a 32-bit byte offset per lane.
__device__ __forceinline__ void dma16s(const bf16_t* base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"(off), "s"(base)
               : "memory");
}
__device__ __forceinline__ void dma_wait() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
__device__ __forceinline__ uint32_t lds_addr(const bf16_t* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// ---- sampling draws (the sampler and the decode LM head's sampling epilogue) ------
// Philox4x32-10 (Salmon et al., SC'11): counter c, key (k0, k1), ten rounds.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
  }
  return c;
}
// Gumbel-max key of logit x at temperature T from one Philox word w:
// u = (2 (w >> 9) + 1) 2^-24 in (0, 1), key = x / T - ln(-ln u).
__device__ __forceinline__ float gumbel_key(float x, float T, uint32_t w) {
  const float u = (float)(2u * (w >> 9) + 1u) * 5.9604644775390625e-8f;   // 2^-24
  return x / T - logf(-logf(u));
}
// (value desc, id asc) arg-max merge
__device__ __forceinline__ void better(float& bv, int& bi, float v, int i) {
  if (v > bv || (v == bv && i < bi)) { bv = v; bi = i; }
}

