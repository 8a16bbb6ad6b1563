// Decode GEMM: Y[B, N] = X[B, K] . W[N, K]^T with few rows (B <= 128), on
// operands stored in MFMA fragment order.
//
// Decode is bound by streaming the weights from HBM once per step; each weight
// element is used B times, which at B = 64 is 64 flop per 2 bytes: more than the
// fp32 vector units deliver at full HBM rate, so the products run on MFMA
// (v_mfma_f32_16x16x32_bf16) with the weights as the A operand (16 output rows
// per MFMA) and the activations as the B operand (16 batch columns per MFMA).
//
// Fragment order.  The A operand of one MFMA is 16 rows x 32 k, lane l holding
// row l & 15, elements 8 (l >> 4) .. 8 (l >> 4) + 7: 64 lanes x 16 bytes.  The
// decode copy of a weight matrix stores each such fragment as 1 KB in lane order,
// k-major: the fragments of all 16-row blocks at one 32-wide k step are
// consecutive ([K/32][N/16][64][8]).  Every weight load instruction of a wave
// reads 1 KB of contiguous memory (a row-major matrix gives 64-byte pieces of 16
// rows per instruction, measurably slower to stream), and the workgroups, which
// advance along k at about the same pace, read neighbouring memory at any moment
// (measured 4-13% faster streaming than row-block-major fragments).  The activations entering a decode GEMM are written by their producer
// (RMSNorm, attention, the SwiGLU epilogue below) in the same order with the
// batch as the row ([K/32][nb/16][64][8], nb = padded batch), so they too arrive
// in 1 KB contiguous loads.
//
// Work split: a workgroup of 4 waves owns RB fragment rows (16 RB weight rows;
// for SwiGLU each 16-row block holds 8 gate rows and the up rows of the same
// outputs; RB per projection shape evens out the grid over the compute units)
// and one K range cut into 32-wide steps dealt round-robin to the waves.  Each
// wave keeps D steps of weight and activation fragments in a register ring that
// is unrolled at compile time, so loads run D - 1 steps ahead of the MFMAs and no
// in-flight register is ever copied (a copy would make the wave wait for the
// load).  Weight loads are non-temporal: each weight byte is used once per step,
// and keeping it out of the way of the activations (read by every workgroup)
// measured faster.  At the end the four waves' accumulators go to LDS (one
// barrier) and are added in a fixed order ((w0 + w2) + (w1 + w3)) as they are
// written out: split-K partial products [split][B][N] in fp32 for the
// consuming kernel (RMSNorm with the residual add, or RoPE) to add in split
// order, or silu(gate) * up rounded to bf16 in fragment order for the down
// projection.  No atomics; the result does not depend on timing.
#include "common.h"
#include "kernels.h"

namespace grpo {

namespace {

constexpr int NT = 256;
constexpr int FRAG = 512;              // elements of one fragment (1 KB)
constexpr int KGRAN = 128;             // k granularity of a split (4 waves x 32)

struct DArgs {
  const bf16_t* X;    // fragment order [K/32][NB/16]
  const bf16_t* W;    // fragment order [K/32][N/16]
  int B, N, K, kper, tiles;
  float* out_f32; bf16_t* out_act; int ld_out;
  DecSample smp;      // EPI_SAMPLE
};

// Gumbel-max merge carrying the winner's logit: (key desc, id asc)
__device__ __forceinline__ void better_g(float& gk, int& gi, float& gz, float k, int i, float z) {
  if (k > gk || (k == gk && i < gi)) { gk = k; gi = i; gz = z; }
}

// ring slot S <- step i (clamped to the last step: the repeat is never used)
#define DG_LOAD(S, i)                                                           \
  do {                                                                          \
    const int i_ = min((i), nst - 1);                                           \
    _Pragma("unroll") for (int rb = 0; rb < RB; ++rb)                           \
        wr[S][rb] = __builtin_nontemporal_load(                                 \
            (const u32x4_t*)(wp[rb] + (size_t)i_ * wstep));                     \
    _Pragma("unroll") for (int j = 0; j < NJ; ++j)                              \
        xr[S][j] = *(const u32x4_t*)(xp + (size_t)i_ * (4 * NJ * FRAG) + j * FRAG); \
  } while (0)

#define DG_MMA(S)                                                               \
  do {                                                                          \
    _Pragma("unroll") for (int rb = 0; rb < RB; ++rb)                           \
    _Pragma("unroll") for (int j = 0; j < NJ; ++j)                              \
        acc[rb][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(                   \
            __builtin_bit_cast(bf16x8_t, wr[S][rb]),                            \
            __builtin_bit_cast(bf16x8_t, xr[S][j]), acc[rb][j], 0, 0, 0);       \
  } while (0)

template <int NB, int RB, int D, int EPI>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(RB > 4 ? 1 : 2)))
void k_gemm_decode(DArgs a) {
  constexpr int NJ = NB / 16;            // MFMA batch blocks
  constexpr int ROWS = 16 * RB;          // weight rows of the tile
  constexpr int CT = ROWS + 4;           // padded row of the [batch][row] LDS tile
  __shared__ __attribute__((aligned(16))) float red[4 * NB * CT];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int tile = blockIdx.x % a.tiles, ks = blockIdx.x / a.tiles;
  const int NR = a.N / 16;                             // 16-row blocks
  const int kt0 = ks * (a.kper / 32) + wave;           // this wave's first k step
  const size_t wstep = (size_t)4 * NR * FRAG;          // a wave's next k step (4 later)
  const int nst = a.kper / KGRAN;                      // steps per wave

  // fragment rows past the end repeat the last one (their outputs are never written)
  const bf16_t* wp[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
    wp[rb] = a.W + ((size_t)kt0 * NR + min(tile * RB + rb, NR - 1)) * FRAG + lane * 8;
  // batch rows past B hold whatever the producer left there: MFMA columns are
  // independent and those columns are never written
  const bf16_t* xp = a.X + (size_t)kt0 * NJ * FRAG + lane * 8;

  f32x4_t acc[RB][NJ];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[rb][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

  u32x4_t wr[D][RB], xr[D][NJ];
#pragma unroll
  for (int p = 0; p < D - 1; ++p) DG_LOAD(p, p);
  // whole ring turns without a branch, then the remaining nst % D steps
  int i0 = 0;
  for (; i0 + D <= nst; i0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      // fences keep the scheduler from sinking the loads below the MFMAs
      DG_LOAD((u + D - 1) % D, i0 + u + D - 1);
      __builtin_amdgcn_sched_barrier(0);
      DG_MMA(u);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  const int rem = nst - i0;
#pragma unroll
  for (int u = 0; u < D - 1; ++u)
    if (u < rem) DG_MMA(u);

  // ---- the four waves' products in LDS [wave][batch][row], one barrier; the
  // epilogue adds them in a fixed order ((w0 + w2) + (w1 + w3)) ----
  // C layout of the 16x16 MFMA: row 4 g + v, column r16.
  {
    float* dst = red + wave * NB * CT;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        *(f32x4_t*)(dst + (16 * j + r16) * CT + rb * 16 + 4 * g) = acc[rb][j];
  }
  __syncthreads();
  // four consecutive rows r .. r + 3 of batch row b (r a multiple of 4)
  auto val4 = [&](int b, int r) {
    const int o = b * CT + r;
    const f32x4_t p0 = *(const f32x4_t*)(red + o), p1 = *(const f32x4_t*)(red + NB * CT + o);
    const f32x4_t p2 = *(const f32x4_t*)(red + 2 * NB * CT + o);
    const f32x4_t p3 = *(const f32x4_t*)(red + 3 * NB * CT + o);
    return (p0 + p2) + (p1 + p3);
  };

  // ---- epilogue: 16-byte stores, consecutive threads on consecutive columns ----
  if (EPI == EPI_SWIGLU) {
    // 16-row block o_b of the tile: gate rows of outputs 8 o_b .. 8 o_b + 7, then
    // their up rows; a thread makes those 8 consecutive outputs (one 16-byte
    // piece of a fragment row)
    constexpr int HO = ROWS / 2;
    for (int i = tid; i < HO / 8 * NB; i += NT) {
      const int o = i % (HO / 8) * 8, b = i / (HO / 8);
      const int n = tile * HO + o;
      if (b < a.B && n < a.ld_out) {
        const int rg = (o >> 3) * 16;
        float y[8];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const f32x4_t gt = val4(b, rg + 4 * h), up = val4(b, rg + 8 + 4 * h);
#pragma unroll
          for (int e = 0; e < 4; ++e) y[4 * h + e] = silu_mul(gt[e], up[e]);
        }
        u32x4_t w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = (uint32_t)f2bf(y[2 * e]) | ((uint32_t)f2bf(y[2 * e + 1]) << 16);
        *(u32x4_t*)(a.out_act + act_frag_index(b, n, NB)) = w;
      }
    }
  } else if (EPI == EPI_SAMPLE) {
    // the tile's pieces of the sampler (DecSample): four threads per batch row,
    // thread t taking rows (vocabulary ids) 4 RB t .. 4 RB t + 4 RB - 1 in groups
    // of four (one Philox block each); the four merged by shuffles in a fixed order
    const bool greedy = !(a.smp.temperature > 0.f);
    const float T = greedy ? 1.f : a.smp.temperature;
    const int step = a.smp.step + (a.smp.step_ctr ? *a.smp.step_ctr : 0);
    const uint32_t k0 = (uint32_t)a.smp.seed, k1 = (uint32_t)(a.smp.seed >> 32);
    for (int i = tid; i < 4 * NB; i += NT) {       // whole waves (NB >= 16)
      const int b = i >> 2, t4 = i & 3;
      const bool live = b < a.B;
      float x[RB][4];
      float m = -INFINITY;
      int mi = 0x7fffffff;
#pragma unroll
      for (int q = 0; q < RB; ++q) {
        const int r = (t4 * RB + q) * 4, n0 = tile * ROWS + r;
        const f32x4_t v = val4(b, r);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[q][e] = n0 + e < a.N ? v[e] : -INFINITY;
          better(m, mi, x[q][e], n0 + e);
        }
        if (a.out_f32 && live && n0 < a.N)
          *(f32x4_t*)(a.out_f32 + (size_t)b * a.ld_out + n0) = v;
      }
#pragma unroll
      for (int o = 1; o < 4; o <<= 1) {
        const float om = __shfl_xor(m, o, 64);
        const int oi = __shfl_xor(mi, o, 64);
        better(m, mi, om, oi);
      }
      const float zm = m / T;
      float sum = 0.f;
#pragma unroll
      for (int q = 0; q < RB; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) sum += __expf(x[q][e] / T - zm);
      sum += __shfl_xor(sum, 1, 64);
      sum += __shfl_xor(sum, 2, 64);
      float gk = -INFINITY, gz = 0.f;
      int gi = 0x7fffffff;
      if (!greedy) {
        const int pid = live ? (a.smp.seq_ids ? a.smp.seq_ids[b] : b) : 0;
#pragma unroll
        for (int q = 0; q < RB; ++q) {
          const int n0 = tile * ROWS + (t4 * RB + q) * 4;
          const uint4 w = philox4x32_10(
              make_uint4((uint32_t)(n0 >> 2), (uint32_t)step, (uint32_t)pid, 0u), k0, k1);
          const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (n0 + e < a.N) better_g(gk, gi, gz, gumbel_key(x[q][e], T, ws[e]), n0 + e, x[q][e]);
        }
#pragma unroll
        for (int o = 1; o < 4; o <<= 1) {
          const float ok = __shfl_xor(gk, o, 64), oz = __shfl_xor(gz, o, 64);
          const int oi = __shfl_xor(gi, o, 64);
          better_g(gk, gi, gz, ok, oi, oz);
        }
      }
      if (live && t4 == 0) {
        float* o = a.smp.part + ((size_t)b * a.tiles + tile) * 8;
        *(f32x4_t*)o = (f32x4_t){m, sum, __int_as_float(mi), gk};
        *(f32x4_t*)(o + 4) = (f32x4_t){__int_as_float(gi), gz, 0.f, 0.f};
      }
    }
  } else {
    float* out = a.out_f32 + (size_t)ks * a.B * a.ld_out;
    for (int i = tid; i < ROWS / 4 * NB; i += NT) {
      const int r = i % (ROWS / 4) * 4, b = i / (ROWS / 4);
      const int n = tile * ROWS + r;
      if (b < a.B && n < a.N) *(f32x4_t*)(out + (size_t)b * a.ld_out + n) = val4(b, r);
    }
  }
}

#undef DG_LOAD
#undef DG_MMA

template <int NB, int RB>
hipError_t launch_rb(const DArgs& a, int epi, int grid, const char* name, hipStream_t st) {
  constexpr int D = 3;
  if (epi == EPI_SWIGLU) {
    Prof pf(name ? name : "gemm_decode_swiglu", st);
    k_gemm_decode<NB, RB, D, EPI_SWIGLU><<<grid, NT, 0, st>>>(a);
  } else if (epi == EPI_SAMPLE) {
    Prof pf(name ? name : "gemm_decode_sample", st);
    k_gemm_decode<NB, RB, D, EPI_SAMPLE><<<grid, NT, 0, st>>>(a);
  } else {
    Prof pf(name ? name : "gemm_decode", st);
    k_gemm_decode<NB, RB, D, EPI_PARTIAL><<<grid, NT, 0, st>>>(a);
  }
  return hipGetLastError();
}

template <int NB>
hipError_t launch_nb(const DArgs& a, int epi, int grid, int rb, const char* name, hipStream_t st) {
  if constexpr (NB >= 128) {
    return rb == 2   ? launch_rb<NB, 2>(a, epi, grid, name, st)
           : rb == 4 ? launch_rb<NB, 4>(a, epi, grid, name, st)
                     : hipErrorInvalidValue;
  } else {
    switch (rb) {
      case 4: return launch_rb<NB, 4>(a, epi, grid, name, st);
      case 6: return launch_rb<NB, 6>(a, epi, grid, name, st);
      case 7: return launch_rb<NB, 7>(a, epi, grid, name, st);
      case 8: return launch_rb<NB, 8>(a, epi, grid, name, st);
    }
    return hipErrorInvalidValue;
  }
}

// One thread per 16-byte piece of the fragment-order copy: piece u is lane
// u % 64 of fragment (kt, R) = (u / 64 / NR, u / 64 % NR).
__global__ __launch_bounds__(256) void k_pack_frag(PackSrc s, int N, int K, bf16_t* __restrict__ dst) {
  const size_t u = (size_t)blockIdx.x * 256 + threadIdx.x;
  const int NR = N / 16;
  const size_t total = (size_t)NR * (K / 32) * 64;
  if (u >= total) return;
  const int l = (int)(u % 64);
  const size_t f = u / 64;
  const int R = (int)(f % NR), kt = (int)(f / NR);
  const int k = kt * 32 + 8 * (l >> 4);
  const bf16_t* row;
  if (s.interleave) {
    // fragment row R: rows 8 R .. 8 R + 7 of s.w[0], then the same rows of s.w[1]
    const int n = R * 8 + (l & 7);
    row = (const bf16_t*)s.w[(l & 15) >> 3] + (size_t)n * K;
  } else {
    const int n = R * 16 + (l & 15);
    if (n < s.n1) row = (const bf16_t*)s.w[0] + (size_t)n * K;
    else if (n < s.n2) row = (const bf16_t*)s.w[1] + (size_t)(n - s.n1) * K;
    else row = (const bf16_t*)s.w[2] + (size_t)(n - s.n2) * K;
  }
  *(u32x4_t*)(dst + u * 8) = *(const u32x4_t*)(row + k);
}

}  // namespace

int decode_nb(int B) { return B <= 16 ? 16 : B <= 32 ? 32 : B <= 64 ? 64 : 128; }

// Split-K factor of a plan: the first divisor of K / KGRAN reaching the target
// grid (SwiGLU needs complete gate and up sums in one workgroup: never split).
static int decode_splits(int tiles, int K, int epi, int target_wgs, int max_splits) {
  // the most splits (dividing the K chunks) that keep the grid within the target
  // (one workgroup per compute unit): a grid past it leaves some units with two
  // workgroups and others with one (1B QKV: 4 splits, 384 workgroups, 12.9 us;
  // 2 splits, 192 workgroups, 10.8 us)
  const int nchunk = K / KGRAN;
  int splits = 1;
  for (int d = 2; epi != EPI_SWIGLU && d <= nchunk && d <= max_splits; ++d)
    if (nchunk % d == 0 && (long)tiles * d <= target_wgs) splits = d;
  return splits;
}

// Tile height: of 4, 6, 7 and 8 blocks of 16 rows, the one whose grid fills
// the compute units most evenly (workgroups over the next multiple of 256); on
// ties fewer splits (less partial traffic), then the taller tile (fewer
// activation reloads).  At the 7B shape: QKV 6 (64 tiles x 4 splits), SwiGLU 7
// (256 tiles), O and down 4 (64 x 4), LM head 8.  At nb = 128 the accumulators
// of a taller tile leave room for one wave per SIMD only: 4 blocks for weight
// matrices of 32 MiB or more (a long stream, where four times the activation
// reuse pays; 1B shape: SwiGLU, down and the LM head 15-20% faster), else 2
// (QKV and O of the 1B shape were 10-25% slower at 4).
DecodePlan decode_plan(int B, int N, int K, int epi, int target_wgs, int max_splits) {
  DecodePlan p{};
  p.nb = decode_nb(B);
  if (target_wgs <= 0) target_wgs = 512;
  const int blocks = N / 16;
  const int cands[4] = {4, 6, 7, 8};
  const int rb128 = (size_t)N * K * 2 >= ((size_t)32 << 20) ? 4 : 2;
  double best = -1.0;
  for (int c = 0; c < (p.nb >= 128 ? 1 : 4); ++c) {
    const int rb = p.nb >= 128 ? rb128 : cands[c];
    const int tiles = (blocks + rb - 1) / rb;
    const int splits = decode_splits(tiles, K, epi, target_wgs, max_splits);
    const long wgs = (long)tiles * splits;
    const double fill = (double)wgs / (double)(((wgs + 255) / 256) * 256);
    const bool tie = fill > best - 1e-9 && fill < best + 1e-9;
    if (fill > best + 1e-9 || (tie && (splits < p.splits || (splits == p.splits && rb > p.rb)))) {
      best = fill;
      p.rb = rb; p.tiles = tiles; p.splits = splits;
    }
  }
  return p;
}

hipError_t gemm_decode_bf16(const uint16_t* Xf, int B, const uint16_t* Wf, int N, int K, int epi,
                            EpiArgs ep, const DecodePlan& p, hipStream_t st) {
  if (B < 1 || B > p.nb || p.nb != decode_nb(B) || N % 16 || K % KGRAN || p.splits < 1 ||
      p.tiles * 16 * p.rb < N ||
      K % p.splits || (K / p.splits) % KGRAN || (epi == EPI_SWIGLU && (N % 32 || ep.ld_out != N / 2)) ||
      (epi == EPI_SAMPLE && (p.splits != 1 || !ep.smp.part || (ep.out_f32 && ep.ld_out < N))))
    return hipErrorInvalidValue;
  DArgs a;
  a.smp = ep.smp;
  a.X = (const bf16_t*)Xf; a.W = (const bf16_t*)Wf;
  a.B = B; a.N = N; a.K = K; a.kper = K / p.splits; a.tiles = p.tiles;
  a.out_f32 = ep.out_f32; a.out_act = (bf16_t*)ep.out_act; a.ld_out = ep.ld_out;
  const int grid = p.tiles * p.splits;
  switch (p.nb) {
    case 16: return launch_nb<16>(a, epi, grid, p.rb, ep.name, st);
    case 32: return launch_nb<32>(a, epi, grid, p.rb, ep.name, st);
    case 64: return launch_nb<64>(a, epi, grid, p.rb, ep.name, st);
    case 128: return launch_nb<128>(a, epi, grid, p.rb, ep.name, st);
  }
  return hipErrorInvalidValue;
}

hipError_t pack_frag(const PackSrc& s, int N, int K, uint16_t* dst, hipStream_t st) {
  if (N % 16 || K % 32 || N <= 0 || K <= 0) return hipErrorInvalidValue;
  const size_t total = (size_t)N / 16 * (K / 32) * 64;
  Prof pf("pack_frag", st);
  k_pack_frag<<<(unsigned)((total + 255) / 256), 256, 0, st>>>(s, N, K, (bf16_t*)dst);
  return hipGetLastError();
}

}  // namespace grpo
