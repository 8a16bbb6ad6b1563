// Tiled GEMM for many rows (prompt prefill and teacher-forced scoring):
// C[M, N] = X[M, K] . W[N, K]^T, bf16 in, fp32 accumulate, on MFMA.
//
// Both operands are K-contiguous, which is the layout the bf16 MFMA wants for
// both A and B.  A workgroup of 4 waves computes a 128x128 tile (2x2 waves of
// 64x64, each 4x4 v_mfma_f32_16x16x32_bf16 blocks) over K in steps of 64; the
// X and W tiles are staged through LDS (rows padded by 16 bytes against bank
// conflicts), double-buffered, the next tile's global loads in flight while the
// current one is multiplied.  Output tiles are walked in groups of 8 row-tiles
// so that neighbouring workgroups share weight tiles in L2.
//
// SwiGLU epilogue: each wave's 64 columns are 32 gate rows and the 32 up rows of
// the same outputs, so silu(gate) * up is formed in registers.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace grpo {

namespace {

constexpr int NT = 256, BM = 128, BN = 128, BK = 64, LROW = BK + 8;
static_assert(BM == kTiledRows && BM % BK == 0, "the causal hints' band");
constexpr int kBigTileRows = 1024;   // rows from which the 256 x 256 tiles are used

struct TArgs {
  const bf16_t* X; int ldx; int M;
  const bf16_t* w0; const bf16_t* w1; const bf16_t* w2; int n1, n2;
  int N, K, tiles_m, tiles_n;
  float* out_f32; bf16_t* out_act; int ld_out;
  GemmBatch bt;     // product b of a batch: blockIdx.y of the tiled kernel
  LseArgs lse;      // EPI_LSE
};

// EPI_LSE: the target column of product row m (clamped to the columns)
__device__ __forceinline__ int lse_target(const LseArgs& l, int m, int N) {
  const int g = l.i0 + m;
  const int t = l.tokens[(size_t)(g / l.Ts) * l.T + l.score_from + g % l.Ts];
  return min(max(t, 0), N - 1);
}

// operands and output of batch product b
__device__ __forceinline__ void batch_offset(TArgs& a, int b) {
  const size_t wo = (size_t)(b / a.bt.wdiv) * a.bt.sw;
  a.X += (size_t)b * a.bt.sx;
  a.w0 += wo; a.w1 += wo; a.w2 += wo;
  a.out_f32 += (size_t)b * a.bt.so;
}

template <int EPI>
__device__ __forceinline__ const bf16_t* tile_wrow(const TArgs& a, int tn, int r) {
  if (EPI == EPI_SWIGLU) {
    // B-tile row r: wave half wn = r / 64, within it 32 gate rows then 32 up rows
    const int wn = r >> 6, q = r & 63;
    const int n = min(tn * 64 + wn * 32 + (q & 31), a.n1 - 1);
    return (q < 32 ? a.w0 + (size_t)n * a.K : a.w1 + (size_t)n * a.K);
  }
  const int n = min(tn * BN + r, a.N - 1);
  if (n < a.n1) return a.w0 + (size_t)n * a.K;
  if (n < a.n2) return a.w1 + (size_t)(n - a.n1) * a.K;
  return a.w2 + (size_t)(n - a.n2) * a.K;
}

template <int EPI>
__global__ __launch_bounds__(NT) void k_gemm_tiled(TArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * LROW];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN * LROW];
  if (gridDim.y > 1) batch_offset(a, blockIdx.y);
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
  const int wm = wave >> 1, wn = wave & 1;

  // grouped tile order: 8 row-tiles share each column-tile sweep
  const int bid = blockIdx.x;
  const int group = 8;
  const int per_group = group * a.tiles_n;
  const int g = bid / per_group;
  const int first_m = g * group;
  const int gsize = min(a.tiles_m - first_m, group);
  const int tm = first_m + (bid % per_group) % gsize;
  const int tn = (bid % per_group) / gsize;
  // causal products (GemmBatch::tri): tiles above the diagonal, and the k range
  // where X is zero, are skipped (the skipped products are exact zeros)
  if (a.bt.tri == 1 && tn * BN > tm * BM + BM - 1) return;
  int kt0 = 0, nk = a.K / BK;
  if (a.bt.tri == 2) nk = min(nk, (tm * BM + BM + BK - 1) / BK);
  if (a.bt.tri == 3) kt0 = min(tm * BM / BK, nk);

  // loader mapping: 4 x 16-byte loads per operand per thread (128 rows x 64 cols)
  const bf16_t* ap[4];
  const bf16_t* bp[4];
  int lr[4], lc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int e = (tid + i * NT) * 8;
    lr[i] = e / BK;
    lc[i] = e % BK;
    const int m = min(tm * BM + lr[i], a.M - 1);
    ap[i] = a.X + (size_t)m * a.ldx + lc[i];
    bp[i] = tile_wrow<EPI>(a, tn, lr[i]) + lc[i];
  }
  u32x4_t ra[4], rb[4];

  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

  if (kt0 < nk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = *(const u32x4_t*)(ap[i] + kt0 * BK);
      rb[i] = *(const u32x4_t*)(bp[i] + kt0 * BK);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *(u32x4_t*)(&As[0][lr[i] * LROW + lc[i]]) = ra[i];
      *(u32x4_t*)(&Bs[0][lr[i] * LROW + lc[i]]) = rb[i];
    }
  }
  __syncthreads();
  for (int kt = kt0; kt < nk; ++kt) {
    const int buf = (kt - kt0) & 1;
    if (kt + 1 < nk) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ra[i] = *(const u32x4_t*)(ap[i] + (kt + 1) * BK);
        rb[i] = *(const u32x4_t*)(bp[i] + (kt + 1) * BK);
      }
    }
#pragma unroll
    for (int s = 0; s < BK / 32; ++s) {
      bf16x8_t af[4], bfr[4];
      const int col = s * 32 + (lane >> 4) * 8;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *(const bf16x8_t*)(&As[buf][(wm * 64 + i * 16 + (lane & 15)) * LROW + col]);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bfr[j] = *(const bf16x8_t*)(&Bs[buf][(wn * 64 + j * 16 + (lane & 15)) * LROW + col]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *(u32x4_t*)(&As[buf ^ 1][lr[i] * LROW + lc[i]]) = ra[i];
      *(u32x4_t*)(&Bs[buf ^ 1][lr[i] * LROW + lc[i]]) = rb[i];
    }
    }
    __syncthreads();
  }

  // ---- epilogue ----
  // the residual's values are all loaded before any is written back (one memory
  // round trip; the compiler cannot tell the addresses apart)
  float old[4][4][4];
  if (EPI == EPI_RESID) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = tm * BM + wm * 64 + i * 16 + (lane >> 4) * 4 + v;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = tn * BN + wn * 64 + j * 16 + (lane & 15);
          old[i][v][j] = (m < a.M && n < a.N) ? a.out_f32[(size_t)m * a.ld_out + n] : 0.f;
        }
      }
  }
  if (EPI == EPI_LSE) {
    // slot tn * 2 + wn = the wave's 64 columns; a row's 64 values sit in the 16
    // lanes of its lane group (4 columns each): in-lane, then across the group
    const int slot = tn * 2 + wn;
    if (slot >= a.ld_out) return;            // (tile half past the last column)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = tm * BM + wm * 64 + i * 16 + (lane >> 4) * 4 + v;
        float x[4], mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = tn * BN + wn * 64 + j * 16 + (lane & 15);
          x[j] = n < a.N ? acc[i][j][v] * a.lse.c : -INFINITY;
          mx = fmaxf(mx, x[j]);
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) s += __builtin_amdgcn_exp2f(x[j] - mx);
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) s += __shfl_xor(s, o, 64);
        if (m < a.M) {
          if ((lane & 15) == 0)
            *(float2*)(a.out_f32 + ((size_t)m * a.ld_out + slot) * 2) = make_float2(mx, s);
          const int t = lse_target(a.lse, m, a.N);
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (tn * BN + wn * 64 + j * 16 + (lane & 15) == t) a.lse.tgt_z[m] = acc[i][j][v];
        }
      }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int m = tm * BM + wm * 64 + i * 16 + (lane >> 4) * 4 + v;
      if (m >= a.M) continue;
      if (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int n = tn * 64 + wn * 32 + j * 16 + (lane & 15);
          if (n < a.n1) {
            const float gt = acc[i][j][v], up = acc[i][j + 2][v];
            a.out_act[(size_t)m * a.ld_out + n] = f2bf(silu_mul(gt, up));
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = tn * BN + wn * 64 + j * 16 + (lane & 15);
          if (n < a.N) {
            float* o = a.out_f32 + (size_t)m * a.ld_out + n;
            if (EPI == EPI_RESID) *o = old[i][v][j] + acc[i][j][v];
            else *o = acc[i][j][v];
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Large tiles for large M (scoring, long prefill): a workgroup of 4 waves (one per
// SIMD) owns a 256 x 256 output tile, each wave a 128 x 128 quarter as 4 x 4
// blocks of v_mfma_f32_32x32x16_bf16, so every 1 KB fragment read from LDS feeds
// four MFMAs (the LDS bytes per MFMA cycle are what bounds these kernels: a wave
// reads LDS at a limited rate, and a 128 x 64 quarter per wave needs half again
// as many bytes per MFMA).  Operand k-tiles of 32 (256 rows x 64 B each for X
// and W) sit in a 4-stage LDS ring (32 KB per stage) filled by direct-to-LDS
// copies (global_load_lds_dwordx4: each lane names its own source, the 64 lanes
// fill 1 KB in lane order) three k-tiles ahead.  Per k-tile each wave issues
// its 32 MFMAs as two phases of 16 with one instruction between consecutive
// MFMAs: in phase 1 (step 0 of the tile) the fragment reads of step 1 and half
// of its copies, in phase 2 (step 1) the reads of the next tile's step 0 and
// the other half; scheduling fences keep that order, so the LDS reads and the
// copies run in the shadow of the matrix core.  Between the phases each wave
// waits for its copies of the next tile and a barrier publishes that tile.
// A stage is refilled (tile t + 3 during tile t) only after every wave passed
// the barrier of tile t - 1, which follows the last read of its old contents.
// Rows of a stage are 64 bytes, their four 16-byte pieces XOR-swizzled by
// (row >> 2) & 3 (conflict-free fragment reads).  XCD-aware tile order:
// super-tiles of 4 x 8 tiles per XCD.  Measured on the scoring shapes (65536
// rows, K = 4096): 1010-1160 TFLOP/s, against 890-990 for an 8-wave ping-pong
// design (two waves per SIMD alternating MFMA and LDS phases, 128 x 64 per
// wave) whose LDS phases outlasted its MFMA phases.
constexpr int GB = 256, PBK = 32, PST = 4;

__device__ __forceinline__ int pswz(int r) { return (r >> 2) & 3; }

// W row of B-tile row r.  SwiGLU: the B-tile rows form two halves (one per wave
// column wn), each 64 gate rows then the 64 up rows of the same outputs.
// Otherwise rows of the (q, k, v) stack in order (the host guarantees that a
// tile lies inside one matrix of the stack).
template <int EPI>
__device__ __forceinline__ const bf16_t* big_wrow(const TArgs& a, int tn, int r) {
  if (EPI == EPI_SWIGLU) {
    const int wn = r >> 7, q = r & 127;
    const int n = min(tn * 128 + wn * 64 + (q & 63), a.n1 - 1);
    return (q < 64 ? a.w0 + (size_t)n * a.K : a.w1 + (size_t)n * a.K);
  }
  const int n = min(tn * GB + r, a.N - 1);
  if (n < a.n1) return a.w0 + (size_t)n * a.K;
  if (n < a.n2) return a.w1 + (size_t)(n - a.n1) * a.K;
  return a.w2 + (size_t)(n - a.n2) * a.K;
}

template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_big(TArgs a) {
  __shared__ __attribute__((aligned(1024))) bf16_t lds[PST][2][GB * PBK];
  const int tid = threadIdx.x, lane = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
  const int wm = wave >> 1, wn = wave & 1;
  const int xcd = blockIdx.x % 8, within = blockIdx.x / 8;
  const int st = (within / 32) * 8 + xcd, loc = within % 32;
  const int st_n = (a.tiles_n + 7) / 8;
  const int tm = (st / st_n) * 4 + loc / 8;
  const int tn = (st % st_n) * 8 + loc % 8;
  if (tm >= a.tiles_m || tn >= a.tiles_n) return;

  // copy instruction j (0..7): j < 4 -> X rows 64 wave + 16 j .., else W rows
  // 64 wave + 16 (j - 4) ..; lane -> row + lane / 4, piece (lane % 4) ^ pswz(row)
  const int m0 = min(tm * GB, a.M - GB);
  const int r0 = wave * 64 + lane / 4;
  const int pbase = ((lane % 4) ^ pswz(r0)) * 8;
  const bf16_t* ab = a.X + (size_t)(m0 + r0) * a.ldx + pbase;
  const size_t astep = (size_t)16 * a.ldx;
  const bf16_t* bsrc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) bsrc[j] = big_wrow<EPI>(a, tn, r0 + 16 * j) + pbase;
  auto dma = [&](int j, int kt) {
    const int buf = kt % PST;
    if (j < 4)
      dma16(ab + j * astep + kt * PBK, lds_addr(&lds[buf][0][(wave * 4 + j) * 16 * PBK]));
    else
      dma16(bsrc[j - 4] + kt * PBK, lds_addr(&lds[buf][1][(wave * 4 + j - 4) * 16 * PBK]));
  };

  const int sw = pswz(lane & 31);
  const int g2 = lane >> 5;
  int aoff[2], boff[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int pc = ((s * 2 + g2) ^ sw) * 8;
    aoff[s] = (wm * 128 + (lane & 31)) * PBK + pc;
    boff[s] = (wn * 128 + (lane & 31)) * PBK + pc;
  }
  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  bf16x8_t F[2][8];   // [step parity][A0..A3, B0..B3]
  auto rd = [&](int set, int f, int kt, int s) {
    const bf16_t* base = &lds[kt % PST][f < 4 ? 0 : 1][0];
    const int off = (f < 4 ? aoff[s] : boff[s]) + (f & 3) * 32 * PBK;
    F[set][f] = *(const bf16x8_t*)(base + off);
  };
  auto mf = [&](int set, int q) {
    const int i = q >> 2, j = q & 3;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(F[set][i], F[set][4 + j], acc[i][j], 0, 0, 0);
  };

  const int nk = a.K / PBK;
#pragma unroll
  for (int p = 0; p < 3; ++p)
    if (p < nk)
#pragma unroll
      for (int j = 0; j < 8; ++j) dma(j, p);
  if (nk > 2) asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
  else if (nk > 1) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
#pragma unroll
  for (int f = 0; f < 8; ++f) rd(0, f, 0, 0);

  auto tile = [&](int t, auto cp_c, auto nx_c) __attribute__((always_inline)) {
    constexpr bool CP = decltype(cp_c)::value, NX = decltype(nx_c)::value;
    // phase 1: MFMAs of step 0 (set 0), reads of step 1 (set 1), first half of copies
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      mf(0, q);
      __builtin_amdgcn_sched_barrier(0);
      if ((q & 1) == 0) rd(1, q >> 1, t, 1);
      else if (CP && (q >> 1) < 4) dma(q >> 1, t + 3);
      __builtin_amdgcn_sched_barrier(0);
    }
    // tile t + 1 landed (newer copies may remain), then publish it
    if (CP) asm volatile("s_waitcnt vmcnt(12)" ::: "memory");
    else if (t + 2 < nk) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    // phase 2: MFMAs of step 1 (set 1), reads of the next tile's step 0 (set 0),
    // second half of copies
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      mf(1, q);
      __builtin_amdgcn_sched_barrier(0);
      if ((q & 1) == 0) { if (NX) rd(0, q >> 1, t + 1, 0); }
      else if (CP && (q >> 1) < 4) dma(4 + (q >> 1), t + 3);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  int t = 0;
  for (; t + 3 < nk; ++t) tile(t, std::true_type{}, std::true_type{});
  for (; t + 1 < nk; ++t) tile(t, std::false_type{}, std::true_type{});
  tile(t, std::false_type{}, std::false_type{});

  // ---- epilogue through LDS (the ring is free once every wave passed this
  // barrier): 32 rows of the wave's quarter at a time are staged row-major
  // (rows padded: conflict-free stores), then moved out in 16-byte pieces, whole
  // 512-byte (fp32) or 128-byte (bf16) row segments per 32 or 8 lanes.
  // acc[i][j][r] is row 32 i + 8 (r / 4) + 4 (lane / 32) + r % 4, column
  // 32 j + (lane & 31) of the wave's 128 x 128 quarter.
  __syncthreads();
  if (EPI == EPI_LSE) {
    // 32 rows of the wave's quarter staged as for the store; lane (row, half)
    // then reduces that row's 64 columns of slot half (its 16-byte pieces read
    // back in order) and, when the row's target lies there, passes its logit on
    constexpr int SR = 132;
    float* stg = reinterpret_cast<float*>(&lds[0][0][0]) + wave * 32 * SR;
    const int row = lane & 31, half = lane >> 5;
    const int c0 = tn * GB + wn * 128 + half * 64;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          stg[((r / 4) * 8 + (lane >> 5) * 4 + (r % 4)) * SR + j * 32 + (lane & 31)] = acc[i][j][r];
      float x[64], mx = -INFINITY;
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const float4 v = *(const float4*)(stg + row * SR + half * 64 + 4 * k);
        x[4 * k] = v.x * a.lse.c; x[4 * k + 1] = v.y * a.lse.c;
        x[4 * k + 2] = v.z * a.lse.c; x[4 * k + 3] = v.w * a.lse.c;
#pragma unroll
        for (int e = 0; e < 4; ++e) mx = fmaxf(mx, x[4 * k + e]);
      }
      float s = 0.f;
#pragma unroll
      for (int k = 0; k < 64; ++k) s += __builtin_amdgcn_exp2f(x[k] - mx);
      const int m = m0 + wm * 128 + i * 32 + row;
      if (m >= tm * GB) {
        *(float2*)(a.out_f32 + ((size_t)m * a.ld_out + c0 / 64) * 2) = make_float2(mx, s);
        const int t = lse_target(a.lse, m, a.N);
        if (t >= c0 && t < c0 + 64) a.lse.tgt_z[m] = stg[row * SR + half * 64 + (t - c0)];
      }
    }
  } else if (EPI == EPI_SWIGLU) {
    constexpr int SR = 72;   // staged row: 64 outputs + 8 pad (bf16)
    bf16_t* stg = &lds[0][0][0] + wave * 32 * SR;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        // the two outputs of the lane's column pair, rounded together (hardware RNE)
        const uint32_t y = __builtin_bit_cast(
            uint32_t, __builtin_convertvector((f32x2_t){silu_mul(acc[i][0][r], acc[i][2][r]),
                                                        silu_mul(acc[i][1][r], acc[i][3][r])},
                                              bf16x2_t));
        bf16_t* row = stg + ((r / 4) * 8 + (lane >> 5) * 4 + (r % 4)) * SR + (lane & 31);
        row[0] = (bf16_t)(y & 0xffffu);
        row[32] = (bf16_t)(y >> 16);
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int idx = lane + 64 * k, row = idx >> 3, c8 = (idx & 7) * 8;
        const int m = m0 + wm * 128 + i * 32 + row;
        const int n = tn * 128 + wn * 64 + c8;
        const u32x4_t v = *(const u32x4_t*)(stg + row * SR + c8);
        if (m >= tm * GB && n < a.n1) *(u32x4_t*)(a.out_act + (size_t)m * a.ld_out + n) = v;
      }
    }
  } else {
    constexpr int SR = 132;  // staged row: 128 columns + 4 pad (fp32)
    float* stg = reinterpret_cast<float*>(&lds[0][0][0]) + wave * 32 * SR;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // the residual's 16 pieces of these 32 rows are all loaded before any is
      // written back (one memory round trip instead of one per piece: the
      // compiler cannot tell the pieces' addresses apart)
      float4 w[16];
      if (EPI == EPI_RESID) {
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const int idx = lane + 64 * k, row = idx >> 5, c4 = (idx & 31) * 4;
          const int m = m0 + wm * 128 + i * 32 + row;
          const int n = tn * GB + wn * 128 + c4;
          w[k] = (m >= tm * GB && n < a.N)
                     ? *(const float4*)(a.out_f32 + (size_t)m * a.ld_out + n)
                     : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          stg[((r / 4) * 8 + (lane >> 5) * 4 + (r % 4)) * SR + j * 32 + (lane & 31)] = acc[i][j][r];
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int idx = lane + 64 * k, row = idx >> 5, c4 = (idx & 31) * 4;
        const int m = m0 + wm * 128 + i * 32 + row;
        const int n = tn * GB + wn * 128 + c4;
        const float4 v = *(const float4*)(stg + row * SR + c4);
        if (m >= tm * GB && n < a.N) {
          float4* o = (float4*)(a.out_f32 + (size_t)m * a.ld_out + n);
          if (EPI == EPI_RESID)
            *o = make_float4(w[k].x + v.x, w[k].y + v.y, w[k].z + v.z, w[k].w + v.w);
          else
            *o = v;
        }
      }
    }
  }
}
// ---------------------------------------------------------------------------
// fp32 GEMM for fp32 models (VALU, 64x64 tiles, 4x4 outputs per thread).
struct FArgs {
  const float* X; int ldx; int M;
  const float* w0; const float* w1; const float* w2; int n1, n2;
  int N, K, epi;
  float* out_f32; float* out_act; int ld_out;
  GemmBatch bt;     // product b of a batch: blockIdx.z
  LseArgs lse;      // EPI_LSE
};

__device__ __forceinline__ const float* frow(const FArgs& a, int n) {
  if (n < a.n1) return a.w0 + (size_t)n * a.K;
  if (n < a.n2) return a.w1 + (size_t)(n - a.n1) * a.K;
  return a.w2 + (size_t)(n - a.n2) * a.K;
}

__global__ __launch_bounds__(256) void k_gemm_f32(FArgs a) {
  __shared__ float xs[16][65];
  __shared__ float ws[16][65];
  if (gridDim.z > 1) {
    const int b = blockIdx.z;
    const size_t wo = (size_t)(b / a.bt.wdiv) * a.bt.sw;
    a.X += (size_t)b * a.bt.sx;
    a.w0 += wo; a.w1 += wo; a.w2 += wo;
    a.out_f32 += (size_t)b * a.bt.so;
  }
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  const bool swiglu = a.epi == EPI_SWIGLU;
  float acc[4][4] = {};
  float acc2[4][4] = {};
  for (int k0 = 0; k0 < a.K; k0 += 16) {
    for (int pass = 0; pass < (swiglu ? 2 : 1); ++pass) {
      for (int i = tid; i < 64 * 16; i += 256) {
        const int r = i / 16, c = i % 16;
        const int m = min(m0 + r, a.M - 1);
        xs[c][r] = a.X[(size_t)m * a.ldx + k0 + c];
        const int n = n0 + r;
        float wv = 0.f;
        if (swiglu) {
          if (n < a.n1) wv = (pass == 0 ? a.w0 : a.w1)[(size_t)n * a.K + k0 + c];
        } else if (n < a.N) {
          wv = frow(a, n)[k0 + c];
        }
        ws[c][r] = wv;
      }
      __syncthreads();
      float (*ac)[4] = pass == 0 ? acc : acc2;
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        float xv[4], wv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) xv[i] = xs[k][ty * 4 + i];
#pragma unroll
        for (int j = 0; j < 4; ++j) wv[j] = ws[k][tx * 4 + j];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) ac[i][j] = fmaf(xv[i], wv[j], ac[i][j]);
      }
      __syncthreads();
    }
  }
  if (a.epi == EPI_LSE) {
    // slot blockIdx.x = the tile's 64 columns; a row's values sit in the 16
    // lanes tx of its lane group (4 columns each)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + ty * 4 + i;
      float x[4], mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[j] = n0 + tx * 4 + j < a.N ? acc[i][j] * a.lse.c : -INFINITY;
        mx = fmaxf(mx, x[j]);
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) s += __builtin_amdgcn_exp2f(x[j] - mx);
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) s += __shfl_xor(s, o, 64);
      if (m < a.M) {
        if (tx == 0)
          *(float2*)(a.out_f32 + ((size_t)m * a.ld_out + blockIdx.x) * 2) = make_float2(mx, s);
        const int t = lse_target(a.lse, m, a.N);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (n0 + tx * 4 + j == t) a.lse.tgt_z[m] = acc[i][j];
      }
    }
    return;
  }
  // the residual's values are all loaded before any is written back
  float old[4][4];
  if (a.epi == EPI_RESID) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
        old[i][j] = (m < a.M && n < a.N) ? a.out_f32[(size_t)m * a.ld_out + n] : 0.f;
      }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= a.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (swiglu) {
        if (n < a.n1) {
          const float gt = acc[i][j];
          a.out_act[(size_t)m * a.ld_out + n] = silu_mul(gt, acc2[i][j]);
        }
      } else if (n < a.N) {
        float* o = a.out_f32 + (size_t)m * a.ld_out + n;
        if (a.epi == EPI_RESID) *o = old[i][j] + acc[i][j];
        else *o = acc[i][j];
      }
    }
  }
}


}  // namespace

hipError_t gemm_tiled_bf16(const uint16_t* X, int ldx, int M, WStack W, int N, int K, int epi,
                           EpiArgs ep, hipStream_t st, GemmBatch bt) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (K % BK || bt.count < 1 || bt.wdiv < 1 ||
      (bt.count > 1 && (epi == EPI_SWIGLU || epi == EPI_LSE)) ||
      (epi == EPI_LSE && (ep.ld_out != lse_slots(N) || !ep.lse.tokens || !ep.lse.tgt_z ||
                          ep.lse.Ts < 1)))
    return hipErrorInvalidValue;
  TArgs a;
  a.bt = bt;
  a.lse = ep.lse;
  a.X = X; a.ldx = ldx; a.M = M;
  a.w0 = (const bf16_t*)W.w[0]; a.w1 = (const bf16_t*)W.w[1]; a.w2 = (const bf16_t*)W.w[2];
  a.n1 = W.n1; a.n2 = W.n2; a.N = N; a.K = K;
  a.out_f32 = ep.out_f32; a.out_act = (bf16_t*)ep.out_act; a.ld_out = ep.ld_out;
  Prof pf(epi == EPI_SWIGLU ? "gemm_tiled_swiglu" : epi == EPI_LSE ? "gemm_tiled_lse" : "gemm_tiled",
          st);
  // the big tiles store 16-byte pieces of output rows (LSE: 8-byte pairs)
  const bool out16 = epi == EPI_SWIGLU ? ep.ld_out % 8 == 0 && (uintptr_t)ep.out_act % 16 == 0
                     : epi == EPI_LSE  ? (uintptr_t)ep.out_f32 % 8 == 0
                                       : ep.ld_out % 4 == 0 && (uintptr_t)ep.out_f32 % 16 == 0;
  const bool aligned = out16 && (epi == EPI_SWIGLU
                           ? W.n1 % 128 == 0
                           : N % GB == 0 && (W.n1 >= N || W.n1 % GB == 0) && (W.n2 >= N || W.n2 % GB == 0));
  if (M >= kBigTileRows && aligned && bt.count == 1 && bt.tri == 0) {
    a.tiles_m = (M + GB - 1) / GB;
    a.tiles_n = epi == EPI_SWIGLU ? (N + 127) / 128 : (N + GB - 1) / GB;
    // super-tiles of 4 x 8 tiles, a whole number of rounds of 8 (one per XCD)
    const int n_st = ((a.tiles_m + 3) / 4) * ((a.tiles_n + 7) / 8);
    const int grid = (n_st + 7) / 8 * 8 * 32;
    switch (epi) {
      case EPI_STORE: k_gemm_big<EPI_STORE><<<grid, 256, 0, st>>>(a); break;
      case EPI_RESID: k_gemm_big<EPI_RESID><<<grid, 256, 0, st>>>(a); break;
      case EPI_LSE: k_gemm_big<EPI_LSE><<<grid, 256, 0, st>>>(a); break;
      default: k_gemm_big<EPI_SWIGLU><<<grid, 256, 0, st>>>(a); break;
    }
    return hipGetLastError();
  }
  a.tiles_m = (M + BM - 1) / BM;
  a.tiles_n = epi == EPI_SWIGLU ? (N + 63) / 64 : (N + BN - 1) / BN;
  const dim3 grid(a.tiles_m * a.tiles_n, bt.count);
  switch (epi) {
    case EPI_STORE: k_gemm_tiled<EPI_STORE><<<grid, NT, 0, st>>>(a); break;
    case EPI_RESID: k_gemm_tiled<EPI_RESID><<<grid, NT, 0, st>>>(a); break;
    case EPI_LSE: k_gemm_tiled<EPI_LSE><<<grid, NT, 0, st>>>(a); break;
    default: k_gemm_tiled<EPI_SWIGLU><<<grid, NT, 0, st>>>(a); break;
  }
  return hipGetLastError();
}

hipError_t gemm_f32(const float* X, int ldx, int M, WStack W, int N, int K, int epi, EpiArgs ep,
                    hipStream_t st, GemmBatch bt) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (K % 16 || bt.count < 1 || bt.wdiv < 1 ||
      (epi == EPI_LSE && (bt.count > 1 || ep.ld_out != lse_slots(N) || !ep.lse.tokens ||
                          !ep.lse.tgt_z || ep.lse.Ts < 1)))
    return hipErrorInvalidValue;
  FArgs a;
  a.bt = bt;
  a.lse = ep.lse;
  a.X = X; a.ldx = ldx; a.M = M;
  a.w0 = (const float*)W.w[0]; a.w1 = (const float*)W.w[1]; a.w2 = (const float*)W.w[2];
  a.n1 = W.n1; a.n2 = W.n2; a.N = N; a.K = K; a.epi = epi;
  a.out_f32 = ep.out_f32; a.out_act = (float*)ep.out_act; a.ld_out = ep.ld_out;
  dim3 grid((N + 63) / 64, (M + 63) / 64, bt.count);
  Prof pf("gemm_f32", st);
  k_gemm_f32<<<grid, 256, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace grpo
