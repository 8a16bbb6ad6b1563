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
#include "common.h"
#include "kernels.h"

namespace grpo {

namespace {

constexpr int NT = 256, BM = 128, BN = 128, BK = 64, LROW = BK + 8;
constexpr int kBigTileRows = 1024;   // rows from which the 256 x 256 tiles are used

struct TArgs {
  const bf16_t* X; int ldx; int M;
  const bf16_t* w0; const bf16_t* w1; const bf16_t* w2; int n1, n2;
  int N, K, tiles_m, tiles_n;
  float* out_f32; bf16_t* out_act; int ld_out;
};

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

  const int nk = a.K / BK;
  {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = *(const u32x4_t*)(ap[i] + 0);
      rb[i] = *(const u32x4_t*)(bp[i] + 0);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *(u32x4_t*)(&As[0][lr[i] * LROW + lc[i]]) = ra[i];
      *(u32x4_t*)(&Bs[0][lr[i] * LROW + lc[i]]) = rb[i];
    }
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
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
            a.out_act[(size_t)m * a.ld_out + n] = f2bf(gt / (1.f + __expf(-gt)) * up);
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = tn * BN + wn * 64 + j * 16 + (lane & 15);
          if (n < a.N) {
            float* o = a.out_f32 + (size_t)m * a.ld_out + n;
            if (EPI == EPI_RESID) *o += acc[i][j][v];
            else *o = acc[i][j][v];
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Large tiles for large M (scoring, long prefill): a workgroup owns a 256 x 256
// output tile on v_mfma_f32_32x32x16_bf16, with 8 waves, two per SIMD: waves w
// and w + 4 share a SIMD (the hardware places a workgroup's waves on SIMDs with
// period 4) and its 128 x 128 quarter of the tile, 64 columns each (4 x 2 blocks
// of 32 x 32, 128 accumulators).  The two waves of a SIMD take turns: while one
// runs the 16 MFMAs of a 32-wide k-tile on fragments already in registers, the
// other reads its fragments of the next k-tile from LDS and issues its half of
// the direct-to-LDS copies (global_load_lds_dwordx4: each lane names its own
// source, the 64 lanes fill 1 KB of LDS in lane order) three k-tiles ahead; a
// barrier swaps the roles, so the wave feeding the matrix core never stops for a
// memory instruction.  Four LDS stages (k-tile t in stage t % 4, 32 KB each).
// Schedule (slot = the time between two barriers; A = waves 0-3, B = 4-7):
//   slot 2t:   A copies its half of tile t + 3 into stage (t + 3) % 4 and reads
//              tile t; B multiplies tile t - 1
//   slot 2t+1: A multiplies tile t, then waits until its copies of tile t + 1
//              have landed; B copies its half of tile t + 3, reads tile t and
//              waits for its copies of tile t + 1
// A stage is refilled (slots 2t, 2t + 1) only after both groups read its previous
// tile (slots 2t - 2, 2t - 1), and a copied tile is published by the barrier after
// both groups' waits, before its first read (slot 2t + 2).
// Rows of a stage are 64 bytes, their four 16-byte pieces XOR-swizzled by
// (row >> 2) & 3 (conflict-free fragment reads).
// Measured on the scoring shapes, the operand copies alone (no MFMA) take about
// 70% of this kernel's time and the MFMAs with their LDS reads alone about 63%
// of it: the two overlap only partly, which is what holds the kernel near 40%
// of the bf16 peak.
constexpr int GB = 256, PBK = 32, PST = 4;

__device__ __forceinline__ int pswz(int r) { return (r >> 2) & 3; }

// W row of B-tile row r.  SwiGLU: the B-tile rows form 4 slices of 64 (one per
// wave column range), each 32 gate rows then the 32 up rows of the same outputs.
// Otherwise rows of the (q, k, v) stack in order (the host guarantees that a
// tile lies inside one matrix of the stack).
template <int EPI>
__device__ __forceinline__ const bf16_t* pp_wrow(const TArgs& a, int tn, int r) {
  if (EPI == EPI_SWIGLU) {
    const int slice = r >> 6, q = r & 63;
    const int n = min(tn * 128 + slice * 32 + (q & 31), a.n1 - 1);
    return (q < 32 ? a.w0 + (size_t)n * a.K : a.w1 + (size_t)n * a.K);
  }
  const int n = min(tn * GB + r, a.N - 1);
  if (n < a.n1) return a.w0 + (size_t)n * a.K;
  if (n < a.n2) return a.w1 + (size_t)(n - a.n1) * a.K;
  return a.w2 + (size_t)(n - a.n2) * a.K;
}

#define PP_BARRIER()                          \
  do {                                        \
    __builtin_amdgcn_sched_barrier(0);        \
    asm volatile("s_barrier" ::: "memory");   \
    __builtin_amdgcn_sched_barrier(0);        \
  } while (0)

template <int EPI>
__global__ __launch_bounds__(512) void k_gemm_pp(TArgs a) {
  // [stage][X tile, W tile]
  __shared__ __attribute__((aligned(1024))) bf16_t lds[PST][2][GB * PBK];
  const int tid = threadIdx.x, lane = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
  const int sq = wave & 3, grp = wave >> 2;
  const int wm = sq >> 1, wn = sq & 1;

  // XCD-aware tile order: workgroups are dealt to the 8 XCDs round-robin
  // (blockIdx % 8), each XCD with its own L2.  The tiles form super-tiles of
  // 4 row tiles x 8 column tiles; the 32 workgroups an XCD runs at a time (one
  // per compute unit) take one super-tile, so each X and W k-slice is fetched
  // into that XCD's L2 once for 8 (X) or 4 (W) users.
  const int xcd = blockIdx.x % 8, within = blockIdx.x / 8;
  const int st = (within / 32) * 8 + xcd, loc = within % 32;
  const int st_n = (a.tiles_n + 7) / 8;
  const int tm = (st / st_n) * 4 + loc / 8;
  const int tn = (st % st_n) * 8 + loc % 8;
  if (tm >= a.tiles_m || tn >= a.tiles_n) return;

  // Copies: instruction j (0..3) of wave sq fills tile rows 64 sq + 16 j .. + 16
  // of both operands, group A issuing j = 0, 1 and group B j = 2, 3 (lane -> row
  // + lane / 4, piece lane % 4 holding source piece (lane % 4) ^ pswz(row), the
  // same for every j); SwiGLU W rows switch from gate to up at j = 2.
  const int m0 = min(tm * GB, a.M - GB);
  const int r0 = sq * 64 + lane / 4;
  const int pbase = ((lane % 4) ^ pswz(r0)) * 8;
  const bf16_t* ab = a.X + (size_t)m0 * a.ldx + (size_t)r0 * a.ldx + pbase;
  const bf16_t* bb0 = pp_wrow<EPI>(a, tn, r0) + pbase;
  const bf16_t* bb1 = pp_wrow<EPI>(a, tn, r0 + 32) + pbase;
  const size_t astep = (size_t)16 * a.ldx, bstep = (size_t)16 * a.K;
  auto copy = [&](int buf, int kt) {
#pragma unroll
    for (int j = 2 * grp; j < 2 * grp + 2; ++j) {
      const int off = (sq * 4 + j) * 16 * PBK;
      dma16(ab + j * astep + kt * PBK, lds_addr(&lds[buf][0][off]));
      const bf16_t* bsrc = (EPI == EPI_SWIGLU && j >= 2) ? bb1 + (j - 2) * bstep : bb0 + j * bstep;
      dma16(bsrc + kt * PBK, lds_addr(&lds[buf][1][off]));
    }
  };

  // fragments: X rows wm * 128 + 32 i + (lane & 31); W rows (tile columns)
  // wn * 128 + grp * 64 + 32 j + (lane & 31); k-step s takes piece 2 s + (lane >> 5)
  const int sw = pswz(lane & 31);
  const int g2 = lane >> 5;
  int aoff[PBK / 16], boff[PBK / 16];
#pragma unroll
  for (int s = 0; s < PBK / 16; ++s) {
    const int pc = ((s * 2 + g2) ^ sw) * 8;
    aoff[s] = (wm * 128 + (lane & 31)) * PBK + pc;
    boff[s] = (wn * 128 + grp * 64 + (lane & 31)) * PBK + pc;
  }
  f32x16_t acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  bf16x8_t fa[PBK / 16][4], fb[PBK / 16][2];
  auto frags = [&](int buf) {
#pragma unroll
    for (int s = 0; s < PBK / 16; ++s) {
#pragma unroll
      for (int i = 0; i < 4; ++i) fa[s][i] = *(const bf16x8_t*)(&lds[buf][0][aoff[s] + i * 32 * PBK]);
#pragma unroll
      for (int j = 0; j < 2; ++j) fb[s][j] = *(const bf16x8_t*)(&lds[buf][1][boff[s] + j * 32 * PBK]);
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  };
  auto mma = [&]() {
#pragma unroll
    for (int s = 0; s < PBK / 16; ++s)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s][i], fb[s][j], acc[i][j], 0, 0, 0);
  };

  const int nk = a.K / PBK;    // >= 4 (K is a multiple of 128)
  copy(0, 0);
  copy(1, 1);
  copy(2, 2);
  asm volatile("s_waitcnt vmcnt(8)" ::: "memory");   // tile 0 (4 copies per wave per tile)
  PP_BARRIER();
  auto wait_next = [&](int t) {
    // tile t + 1 landed: only the copies of tiles t + 2 and t + 3 may remain
    if (t + 3 < nk) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
    else if (t + 2 < nk) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  };
  if (grp == 0) {
    for (int t = 0; t < nk; ++t) {
      if (t + 3 < nk) copy((t + 3) % PST, t + 3);
      frags(t % PST);
      PP_BARRIER();
      mma();
      wait_next(t);
      PP_BARRIER();
    }
    PP_BARRIER();
  } else {
    PP_BARRIER();
    for (int t = 0; t < nk; ++t) {
      if (t + 3 < nk) copy((t + 3) % PST, t + 3);
      frags(t % PST);
      wait_next(t);
      PP_BARRIER();
      mma();
      PP_BARRIER();
    }
  }

  // ---- epilogue: acc[i][j][r] is row 32 i + 8 (r / 4) + 4 (lane / 32) + r % 4 of
  // the SIMD's 128 rows, column 32 j + (lane & 31) of the wave's 64 columns ----
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm * 128 + i * 32 + (r / 4) * 8 + (lane >> 5) * 4 + (r % 4);
      if (m < tm * GB) continue;
      if (EPI == EPI_SWIGLU) {
        const int n = tn * 128 + (wn * 2 + grp) * 32 + (lane & 31);
        if (n < a.n1) {
          const float gt = acc[i][0][r], up = acc[i][1][r];
          a.out_act[(size_t)m * a.ld_out + n] = f2bf(gt / (1.f + __expf(-gt)) * up);
        }
      } else {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int n = tn * GB + wn * 128 + grp * 64 + j * 32 + (lane & 31);
          if (n < a.N) {
            float* o = a.out_f32 + (size_t)m * a.ld_out + n;
            if (EPI == EPI_RESID) *o += acc[i][j][r];
            else *o = acc[i][j][r];
          }
        }
      }
    }
  }
}
#undef PP_BARRIER

// ---------------------------------------------------------------------------
// fp32 GEMM for fp32 models (VALU, 64x64 tiles, 4x4 outputs per thread).
struct FArgs {
  const float* X; int ldx; int M;
  const float* w0; const float* w1; const float* w2; int n1, n2;
  int N, K, epi;
  float* out_f32; float* out_act; int ld_out;
};

__device__ __forceinline__ const float* frow(const FArgs& a, int n) {
  if (n < a.n1) return a.w0 + (size_t)n * a.K;
  if (n < a.n2) return a.w1 + (size_t)(n - a.n1) * a.K;
  return a.w2 + (size_t)(n - a.n2) * a.K;
}

__global__ __launch_bounds__(256) void k_gemm_f32(FArgs a) {
  __shared__ float xs[16][65];
  __shared__ float ws[16][65];
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
          a.out_act[(size_t)m * a.ld_out + n] = gt / (1.f + __expf(-gt)) * acc2[i][j];
        }
      } else if (n < a.N) {
        float* o = a.out_f32 + (size_t)m * a.ld_out + n;
        if (a.epi == EPI_RESID) *o += acc[i][j];
        else *o = acc[i][j];
      }
    }
  }
}

}  // namespace

hipError_t gemm_tiled_bf16(const uint16_t* X, int ldx, int M, WStack W, int N, int K, int epi,
                           EpiArgs ep, hipStream_t st) {
  TArgs a;
  a.X = X; a.ldx = ldx; a.M = M;
  a.w0 = (const bf16_t*)W.w[0]; a.w1 = (const bf16_t*)W.w[1]; a.w2 = (const bf16_t*)W.w[2];
  a.n1 = W.n1; a.n2 = W.n2; a.N = N; a.K = K;
  a.out_f32 = ep.out_f32; a.out_act = (bf16_t*)ep.out_act; a.ld_out = ep.ld_out;
  Prof pf(epi == EPI_SWIGLU ? "gemm_tiled_swiglu" : "gemm_tiled", st);
  const bool aligned = epi == EPI_SWIGLU
                           ? W.n1 % 128 == 0
                           : N % GB == 0 && (W.n1 >= N || W.n1 % GB == 0) && (W.n2 >= N || W.n2 % GB == 0);
  if (M >= kBigTileRows && aligned) {
    a.tiles_m = (M + GB - 1) / GB;
    a.tiles_n = epi == EPI_SWIGLU ? (N + 127) / 128 : (N + GB - 1) / GB;
    // super-tiles of 4 x 8 tiles, a whole number of rounds of 8 (one per XCD)
    const int n_st = ((a.tiles_m + 3) / 4) * ((a.tiles_n + 7) / 8);
    const int grid = (n_st + 7) / 8 * 8 * 32;
    switch (epi) {
      case EPI_STORE: k_gemm_pp<EPI_STORE><<<grid, 512, 0, st>>>(a); break;
      case EPI_RESID: k_gemm_pp<EPI_RESID><<<grid, 512, 0, st>>>(a); break;
      default: k_gemm_pp<EPI_SWIGLU><<<grid, 512, 0, st>>>(a); break;
    }
    return hipGetLastError();
  }
  a.tiles_m = (M + BM - 1) / BM;
  a.tiles_n = epi == EPI_SWIGLU ? (N + 63) / 64 : (N + BN - 1) / BN;
  const int grid = a.tiles_m * a.tiles_n;
  switch (epi) {
    case EPI_STORE: k_gemm_tiled<EPI_STORE><<<grid, NT, 0, st>>>(a); break;
    case EPI_RESID: k_gemm_tiled<EPI_RESID><<<grid, NT, 0, st>>>(a); break;
    default: k_gemm_tiled<EPI_SWIGLU><<<grid, NT, 0, st>>>(a); break;
  }
  return hipGetLastError();
}

hipError_t gemm_f32(const float* X, int ldx, int M, WStack W, int N, int K, int epi, EpiArgs ep,
                    hipStream_t st) {
  FArgs a;
  a.X = X; a.ldx = ldx; a.M = M;
  a.w0 = (const float*)W.w[0]; a.w1 = (const float*)W.w[1]; a.w2 = (const float*)W.w[2];
  a.n1 = W.n1; a.n2 = W.n2; a.N = N; a.K = K; a.epi = epi;
  a.out_f32 = ep.out_f32; a.out_act = (float*)ep.out_act; a.ld_out = ep.ld_out;
  dim3 grid((N + 63) / 64, (M + 63) / 64);
  Prof pf("gemm_f32", st);
  k_gemm_f32<<<grid, 256, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace grpo
