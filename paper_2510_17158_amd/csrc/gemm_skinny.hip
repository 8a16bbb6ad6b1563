// Decode GEMM: Y[B, N] = X[B, K] . W[N, K]^T with few rows (B <= 128).
//
// Decode is bound by streaming the weights from HBM once per step; each weight
// element is used B times, which at B = 64 is 64 flop per 2 bytes: more than the
// fp32 vector units deliver at full HBM rate, so the products run on MFMA
// (v_mfma_f32_16x16x32_bf16) with the weights as the A operand (16 output rows
// per wave) and the activations as the B operand (16 batch columns per MFMA).
//
// Work split: a workgroup of 4 waves owns 64 weight rows (a 32-row output tile of
// (gate, up) pairs for SwiGLU) and one K range.  The activation chunk X[:, k..k+KC)
// is staged once in LDS and shared by the 4 waves; each lane streams 2*KC/4 bytes
// of one weight row per chunk with 16-byte loads, up to three chunks ahead of the
// MFMAs.
// The contraction order inside a chunk is permuted (MFMA step s of lane group g
// covers the 8 elements at 32 s + 8 g, so a load instruction reads 64 contiguous
// bytes of a weight row); X is read with the same permutation, so the sum is
// unchanged.  Split-K workgroups write fp32 partial products [split][B][N]; the
// kernel that consumes the product (RMSNorm with the residual add, or RoPE)
// adds the splits in split order.  No cross-workgroup synchronisation, no
// atomics, and the result is deterministic.
#include "common.h"
#include "kernels.h"

namespace grpo {

namespace {

constexpr int NT = 256;

struct SkArgs {
  const bf16_t* X; int ldx; int B;
  const bf16_t* w0; const bf16_t* w1; const bf16_t* w2; int n1, n2;
  int N, K, kper, tiles, splits;
  float* out_f32; bf16_t* out_act; int ld_out;
  const char* name;
};

__device__ __forceinline__ const bf16_t* wrow(const SkArgs& a, int r) {
  if (r < a.n1) return a.w0 + (size_t)r * a.K;
  if (r < a.n2) return a.w1 + (size_t)(r - a.n1) * a.K;
  return a.w2 + (size_t)(r - a.n2) * a.K;
}

template <int NB, int KC, int EPI>
__global__ __launch_bounds__(NT) void k_gemm_skinny(SkArgs a) {
  constexpr int NJ = NB / 16;            // MFMA batch blocks
  constexpr int LPR = KC / 4;            // elements per lane per chunk (one weight row)
  constexpr int NLD = LPR / 8;           // 16-byte loads per lane per chunk
  constexpr int XROW = KC + 8;           // padded LDS row (elements)
  constexpr int XV = NB * KC / 8 / NT;   // 16-byte X loads per thread per chunk
  constexpr int WSTAGES = NB >= 128 ? 3 : 4;
  static_assert(NLD >= 1 && XV >= 1, "chunk too small");
  __shared__ __attribute__((aligned(16))) bf16_t xs[2][NB * XROW];

  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
  const int tile = blockIdx.x % a.tiles;
  const int ks = blockIdx.x / a.tiles;
  const int k0 = ks * a.kper;
  const int nchunk = a.kper / KC;

  // weight row of this lane
  int row;
  if (EPI == EPI_SWIGLU) {
    const int n = tile * 32 + (wave & 1) * 16 + (lane & 15);
    row = (wave < 2 ? 0 : a.n1) + min(n, a.n1 - 1);
  } else {
    row = min(tile * 64 + wave * 16 + (lane & 15), a.N - 1);
  }
  const bf16_t* wp = wrow(a, row) + k0 + (lane >> 4) * 8;

  // X staging: thread -> (batch row, 8-element column group)
  auto load_x = [&](int c, u32x4_t* xr) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int e = (tid + i * NT) * 8;      // element index in [NB, KC]
      const int b = e / KC, col = e % KC;
      if (b < a.B)
        xr[i] = *(const u32x4_t*)(a.X + (size_t)b * a.ldx + k0 + c * KC + col);
      else
        xr[i] = (u32x4_t){0u, 0u, 0u, 0u};
    }
  };
  auto store_x = [&](int buf, const u32x4_t* xr) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int e = (tid + i * NT) * 8;
      const int b = e / KC, col = e % KC;
      *(u32x4_t*)(&xs[buf][b * XROW + col]) = xr[i];
    }
  };

  f32x4_t acc[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) acc[j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

  // WSTAGES weight stages in registers: chunk c is multiplied while chunks
  // c+1 .. c+WSTAGES-1 are in flight.  X chunk c+1 is requested before the
  // youngest weight chunk so that waiting for X (needed at the end of the
  // iteration) does not wait for the younger weight loads.
  u32x4_t wst[WSTAGES][NLD], xr[XV];
#pragma unroll
  for (int p = 0; p < WSTAGES - 1; ++p) {
    if (p < nchunk) {
#pragma unroll
      for (int i = 0; i < NLD; ++i) wst[p][i] = *(const u32x4_t*)(wp + p * KC + i * 32);
    }
    if (p == 0) load_x(0, xr);
  }
  store_x(0, xr);
  __syncthreads();

  for (int c = 0; c < nchunk; ++c) {
    const int buf = c & 1;
    if (c + 1 < nchunk) load_x(c + 1, xr);
    if (c + WSTAGES - 1 < nchunk) {
#pragma unroll
      for (int i = 0; i < NLD; ++i)
        wst[WSTAGES - 1][i] = *(const u32x4_t*)(wp + (c + WSTAGES - 1) * KC + i * 32);
    }
    const bf16_t* xb = &xs[buf][0];
#pragma unroll
    for (int s = 0; s < NLD; ++s) {
      const bf16x8_t av = __builtin_bit_cast(bf16x8_t, wst[0][s]);
      const int col = s * 32 + (lane >> 4) * 8;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int b = (lane & 15) + 16 * j;
        const bf16x8_t bv = *(const bf16x8_t*)(xb + b * XROW + col);
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc[j], 0, 0, 0);
      }
    }
    if (c + 1 < nchunk) store_x(buf ^ 1, xr);
#pragma unroll
    for (int p = 0; p < WSTAGES - 1; ++p)
#pragma unroll
      for (int i = 0; i < NLD; ++i) wst[p][i] = wst[p + 1][i];
    __syncthreads();
  }

  // ---- tile result -> LDS ct[64][NB] fp32 (reuses the X buffers) ----
  float* ct = (float*)&xs[0][0];
  static_assert(64 * NB * 4 <= 2 * NB * XROW * 2, "epilogue tile does not fit");
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = wave * 16 + (lane >> 4) * 4 + v;
      const int b = (lane & 15) + 16 * j;
      ct[r * NB + b] = acc[j][v];
    }
  __syncthreads();

  // ---- epilogue: consecutive threads take consecutive output columns ----
  if (EPI == EPI_SWIGLU) {
    for (int i = tid; i < 32 * NB; i += NT) {
      const int r = i % 32, b = i / 32;
      const int n = tile * 32 + r;
      if (b < a.B && n < a.n1) {
        const float g = ct[r * NB + b], u = ct[(r + 32) * NB + b];
        const float sg = g / (1.f + __expf(-g));
        a.out_act[(size_t)b * a.ld_out + n] = f2bf(sg * u);
      }
    }
  } else {
    // this split's partial product: out[ks][b][n]
    float* out = a.out_f32 + (size_t)ks * a.B * a.ld_out;
    for (int i = tid; i < 64 * NB; i += NT) {
      const int r = i % 64, b = i / 64;
      const int n = tile * 64 + r;
      if (b < a.B && n < a.N) out[(size_t)b * a.ld_out + n] = ct[r * NB + b];
    }
  }
}

template <int NB, int KC>
hipError_t launch_nb(const SkArgs& a, int epi, int grid, hipStream_t st) {
  if (epi == EPI_SWIGLU) {
    Prof pf(a.name ? a.name : "gemm_decode_swiglu", st);
    k_gemm_skinny<NB, KC, EPI_SWIGLU><<<grid, NT, 0, st>>>(a);
  } else {
    Prof pf(a.name ? a.name : "gemm_decode", st);
    k_gemm_skinny<NB, KC, EPI_PARTIAL><<<grid, NT, 0, st>>>(a);
  }
  return hipGetLastError();
}

}  // namespace

SkinnyPlan skinny_plan(int B, int N, int K, int epi, int target_wgs, int max_splits) {
  SkinnyPlan p{};
  p.nb = B <= 16 ? 16 : B <= 32 ? 32 : B <= 64 ? 64 : 128;
  p.kc = 128;
  p.tiles = epi == EPI_SWIGLU ? (N + 31) / 32 : (N + 63) / 64;
  const int nchunk = K / p.kc;
  p.splits = 1;
  if (target_wgs <= 0) target_wgs = 512;
  // SwiGLU needs complete gate and up sums in one workgroup: never split
  for (int d = 1; epi != EPI_SWIGLU && d <= nchunk && d <= max_splits; ++d) {
    if (nchunk % d) continue;
    p.splits = d;
    if ((long)p.tiles * d >= target_wgs) break;
  }
  return p;
}

hipError_t gemm_skinny_bf16(const uint16_t* X, int ldx, int B, WStack W, int N, int K, int epi,
                            EpiArgs ep, const SkinnyPlan& p, hipStream_t st) {
  SkArgs a;
  a.X = X; a.ldx = ldx; a.B = B;
  a.w0 = (const bf16_t*)W.w[0]; a.w1 = (const bf16_t*)W.w[1]; a.w2 = (const bf16_t*)W.w[2];
  a.n1 = W.n1; a.n2 = W.n2;
  a.N = N; a.K = K; a.kper = K / p.splits; a.tiles = p.tiles; a.splits = p.splits;
  a.out_f32 = ep.out_f32; a.out_act = (bf16_t*)ep.out_act; a.ld_out = ep.ld_out;
  a.name = ep.name;
  const int grid = p.tiles * p.splits;
  if (p.kc == 128) {
    switch (p.nb) {
      case 16: return launch_nb<16, 128>(a, epi, grid, st);
      case 32: return launch_nb<32, 128>(a, epi, grid, st);
      case 64: return launch_nb<64, 128>(a, epi, grid, st);
      case 128: return launch_nb<128, 128>(a, epi, grid, st);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace grpo
