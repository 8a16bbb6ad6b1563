// Causal attention of the decoder for prompt prefill and teacher-forced scoring.
//
// bf16: flash attention, one workgroup per (32 queries, kv head, sequence) with
// one wave per query head of the group sharing the K and V^T tiles (V^T is
// written transposed by the rotary kernel); details at the kernel.
//
// fp32 models use a plain vector kernel (one workgroup per query row and head),
// also for decode.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace grpo {

namespace {

// ----------------------------------------------------------- flash attention, bf16
// One workgroup per (32 query rows, kv head, sequence) with one wave per query
// head of the group: every K / V^T tile is staged in LDS once for all of them.
// Each wave computes S^T = K Q^T (keys as MFMA rows, its 32 queries as two
// 16-column blocks), so a query's scores sit in the lanes of one column and the
// online-softmax statistics are per lane.  Inside each 32-key step the key order
// of the two 16-row MFMA blocks is permuted (block b, row i -> key
// 8 (i >> 2) + 4 b + (i & 3)) so that a lane's eight scores of a column are keys
// 8 g .. 8 g + 7: exactly the B operand of O^T += V^T P^T, which therefore never
// leaves registers.  P enters that product as two bf16 terms (hi + lo), so no
// rounding point is added.  K and V^T tiles of 64 keys are double-buffered in
// LDS and filled by direct-to-LDS copies one tile ahead (no staging registers);
// one barrier per tile.  The latest query blocks (the most key tiles under the
// causal mask) start first.
// Tile rows in LDS are unpadded, their 16-byte pieces XOR-swizzled.  K: the 16
// key rows one fragment read touches (8 (i >> 2) + (i & 3) plus a multiple of 4)
// fall in 16 distinct bank groups (HD 128: 256-byte rows, the swizzle takes row
// bits 0-1 and 3-4; HD 64: 128-byte rows, bits 1 and 3-4).
template <int HD>
__device__ __forceinline__ int kswz(int r) {
  return HD == 128 ? ((r & 3) | (((r >> 3) & 3) << 2)) : (((r >> 1) & 1) | (((r >> 3) & 3) << 1));
}
// V^T tile rows (one head dimension, 64 keys = 128 bytes): the 16 consecutive rows
// one fragment read touches, all at the same piece, fall in 16 distinct bank groups
// (row bit 0 selects the half of the 256-byte bank line, bits 1-3 the piece).
__device__ __forceinline__ int vswz(int r) { return (r >> 1) & 7; }

template <int HD, int GQ>
__global__ __launch_bounds__(64 * GQ) __attribute__((amdgpu_waves_per_eu(2))) void k_flash_bf16(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ vt,
    int T, int H, int n_kv, int k_len, int k_seq_stride, int vt_len, float scale,
    bf16_t* __restrict__ out, int q_pos0, int vt_seq_stride, const int32_t* __restrict__ qpos,
    const int32_t* __restrict__ kslots) {
  constexpr int QSTEPS = HD / 32, HB = HD / 16;
  constexpr int NCP = HD / 8;   // 1 KB copies per K tile (and per V^T tile)
  __shared__ __attribute__((aligned(1024))) bf16_t ks[2][64 * HD];
  __shared__ __attribute__((aligned(1024))) bf16_t vs[2][HD * 64];

  const int qblk = gridDim.x - 1 - blockIdx.x;
  const int g = blockIdx.y, n = blockIdx.z;
  const int tid = threadIdx.x, lane = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
  const int h = g * GQ + wave;
  const int ldq = H * HD;
  const int q0 = qblk * 32;
  const int lq = lane & 15, lg = lane >> 4;

  // Q as the B operand: column lq of block qb = query q0 + 16 qb + lq; MFMA step st
  // takes the 8-element piece (4 st + lg) of the head dimension
  bf16x8_t qf[2][QSTEPS];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int r = min(q0 + qb * 16 + lq, T - 1);
    const bf16_t* qp = q + ((size_t)n * T + r) * ldq + h * HD + lg * 8;
#pragma unroll
    for (int st = 0; st < QSTEPS; ++st) qf[qb][st] = *(const bf16x8_t*)(qp + st * 32);
  }
  // sequence n's first query position (per sequence when qpos is given) and
  // its K slot (kslots, else n * k_seq_stride)
  const int qp0 = qpos ? qpos[n] : q_pos0;
  const size_t kslot = kslots ? (size_t)kslots[n] : (size_t)n * k_seq_stride;
  const bf16_t* kbase = k + (kslot * n_kv + g) * (size_t)k_len * HD;
  const bf16_t* vbase = vt + ((size_t)n * vt_seq_stride * n_kv + g) * (size_t)HD * vt_len;
  // query rows are positions qp0 + row; keys run to position Tk - 1
  const int Tk = qp0 + T;

  // Tile t of 64 keys into stage buf by direct-to-LDS copies, NCP of K and NCP of
  // V^T dealt round-robin to the waves.  Copy i, lane l fills the 16-byte LDS
  // piece o = 64 i + l: for K, row o / (HD / 8) (a key), piece o % (HD / 8) holding
  // source piece (o % (HD / 8)) ^ kswz(row); for V^T, row o / 8 (a head dimension),
  // piece o % 8 holding keys 8 ((o % 8) ^ vswz(row)) .. + 8.  A tile inside the
  // sequence is addressed as a wave-uniform base plus a 32-bit lane offset; in the
  // last tile of a sequence whose length is not a multiple of 64, keys past T - 1
  // read clamped positions: their scores are masked (P = 0) and the V^T values
  // they read are finite.
  constexpr int KRPC = 512 / HD;   // K rows per copy
  auto copy_tile = [&](int t, int buf) __attribute__((always_inline)) {
    if ((t + 1) * 64 <= Tk) {
#pragma unroll
      for (int i0 = 0; i0 < NCP; i0 += GQ) {
        const int i = i0 + wave;
        if (NCP % GQ != 0 && i >= NCP) break;
        const int o = i * 64 + lane;
        const int kr_ = o / (HD / 8), kp = (o % (HD / 8)) ^ kswz<HD>(kr_);
        const int vr_ = o / 8, vp = (o % 8) ^ vswz(vr_);
        dma16s(kbase + (size_t)(t * 64 + i * KRPC) * HD, ((kr_ - i * KRPC) * HD + kp * 8) * 2,
               lds_addr(&ks[buf][i * 512]));
        dma16s(vbase + (size_t)(i * 8) * vt_len + t * 64, ((vr_ - i * 8) * vt_len + vp * 8) * 2,
               lds_addr(&vs[buf][i * 512]));
      }
    } else {
#pragma unroll
      for (int i0 = 0; i0 < NCP; i0 += GQ) {
        const int i = i0 + wave;
        if (NCP % GQ != 0 && i >= NCP) break;
        const int o = i * 64 + lane;
        const int kr_ = o / (HD / 8), kp = (o % (HD / 8)) ^ kswz<HD>(kr_);
        const int vr_ = o / 8, vp = (o % 8) ^ vswz(vr_);
        const int key = min(t * 64 + kr_, Tk - 1);
        dma16(kbase + (size_t)key * HD + kp * 8, lds_addr(&ks[buf][i * 512]));
        const int key0 = min(t * 64 + vp * 8, vt_len - 8);
        dma16(vbase + (size_t)vr_ * vt_len + key0, lds_addr(&vs[buf][i * 512]));
      }
    }
  };

  f32x4_t oacc[HB][2];
#pragma unroll
  for (int hb = 0; hb < HB; ++hb)
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) oacc[hb][qb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
  float mq[2] = {-1e30f, -1e30f}, lq_sum[2] = {0.f, 0.f};

  const float scale2 = scale * 1.4426950408889634f;   // log2(e)
  const int qlast = qp0 + min(q0 + 31, T - 1);
  const int n_tiles = qlast / 64 + 1;
  copy_tile(0, 0);
  dma_wait();
  __syncthreads();

  // One key tile: scores, online softmax and P.V.  Only the last tile holds
  // masked keys (the causal diagonal and keys past T - 1): every key of an
  // earlier tile is below q0, so MASK is set for the last tile only.
  auto tile_step = [&](int t, auto mask_c) __attribute__((always_inline)) {
    constexpr bool MASK = decltype(mask_c)::value;
    // copy tile t + 1 into the other stage (last read in iteration t - 1, which
    // every wave has left); it lands while tile t is used
    if (t + 1 < n_tiles) copy_tile(t + 1, (t + 1) & 1);
    const bf16_t* ksb = &ks[t & 1][0];
    const bf16_t* vsb = &vs[t & 1][0];
    const int k0 = t * 64;
    // S^T for the two 32-key steps: sacc[s2][b][qb], lane rows 4 lg + v -> key
    // k0 + 32 s2 + 8 lg + 4 b + v, column lq -> query q0 + 16 qb + lq
    f32x4_t sacc[2][2][2];
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int kr_ = 32 * s2 + 8 * (lq >> 2) + 4 * b + (lq & 3);   // this lane's A row
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) sacc[s2][b][qb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < QSTEPS; ++st) {
          const bf16x8_t kf = *(const bf16x8_t*)(ksb + kr_ * HD + ((st * 4 + lg) ^ kswz<HD>(kr_)) * 8);
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
            sacc[s2][b][qb] =
                __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[qb][st], sacc[s2][b][qb], 0, 0, 0);
        }
      }
    // online softmax per query column in base 2 (P = 2^(s scale log2 e - m) for a
    // reference maximum m of the column, the scaling folded into one fused
    // multiply-add; the tile maximum is taken over the raw scores, which commutes
    // with the positive scaling): tile maximum and rescale first, then per 32-key step the P^T operands (hi, lo: hardware
    // round-to-nearest-even conversions) and their products with V^T.  A masked
    // score is -inf and gives P = 0; the running maximum starts finite, so the
    // exponent is never inf - inf.
    float mnew[2], psum[2] = {0.f, 0.f};
    bool moved = false;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      // (last tile) key k0 + 32 s2 + 8 lg + 4 b + v is visible iff 32 s2 + 4 b + v <= lim
      const int lim = qp0 + min(q0 + qb * 16 + lq, T - 1) - k0 - 8 * lg;
      float mx = -INFINITY;
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            if (MASK && 32 * s2 + 4 * b + v > lim) sacc[s2][b][qb][v] = -INFINITY;
            mx = fmaxf(mx, sacc[s2][b][qb][v]);
          }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      // the reference maximum moves only when the column maximum exceeds it by
      // more than 8 (so P <= 2^8; the hi + lo terms keep their relative precision
      // and the fp32 sums their range), which makes the rescale rare
      mnew[qb] = mx * scale2 > mq[qb] + 8.f ? mx * scale2 : mq[qb];
      moved |= mnew[qb] != mq[qb];
    }
    // rescale only when some column's reference maximum moved (a factor of exactly
    // 1 otherwise)
    if (__builtin_amdgcn_ballot_w64(moved)) {
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        const float alpha = __builtin_amdgcn_exp2f(mq[qb] - mnew[qb]);
        lq_sum[qb] *= alpha;
#pragma unroll
        for (int hb = 0; hb < HB; ++hb)
#pragma unroll
          for (int v = 0; v < 4; ++v) oacc[hb][qb][v] *= alpha;
      }
    }
    mq[0] = mnew[0];
    mq[1] = mnew[1];
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      bf16x8_t ph[2], pl[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int v = 0; v < 4; v += 2) {
            const float p0 =
                __builtin_amdgcn_exp2f(fmaf(sacc[s2][b][qb][v], scale2, -mnew[qb]));
            const float p1 =
                __builtin_amdgcn_exp2f(fmaf(sacc[s2][b][qb][v + 1], scale2, -mnew[qb]));
            psum[qb] += p0;
            psum[qb] += p1;
            const bf16x2_t hi = __builtin_convertvector((f32x2_t){p0, p1}, bf16x2_t);
            const bf16x2_t lo = __builtin_convertvector(
                (f32x2_t){p0 - (float)hi[0], p1 - (float)hi[1]}, bf16x2_t);
            ph[qb][4 * b + v] = hi[0];
            ph[qb][4 * b + v + 1] = hi[1];
            pl[qb][4 * b + v] = lo[0];
            pl[qb][4 * b + v + 1] = lo[1];
          }
      }
      // O^T += V^T P^T: A = V^T rows (dims 16 hb + lq), keys 32 s2 + 8 lg .. + 8
#pragma unroll
      for (int hb = 0; hb < HB; ++hb) {
        const int vr_ = hb * 16 + lq;
        const bf16x8_t vf = *(const bf16x8_t*)(vsb + vr_ * 64 + ((4 * s2 + lg) ^ vswz(vr_)) * 8);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          oacc[hb][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, ph[qb], oacc[hb][qb], 0, 0, 0);
          oacc[hb][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pl[qb], oacc[hb][qb], 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      float sum = psum[qb];
      sum += __shfl_xor(sum, 16, 64);
      sum += __shfl_xor(sum, 32, 64);
      lq_sum[qb] += sum;
    }
    dma_wait();
    __syncthreads();
  };
  // key tiles from the one holding the block's first query position on hold
  // keys past some query of the block (only the last one when qp0 is a
  // multiple of 32)
  const int tm = min((qp0 + q0) / 64, n_tiles - 1);
  for (int t = 0; t < tm; ++t) tile_step(t, std::false_type{});
  for (int t = tm; t < n_tiles; ++t) tile_step(t, std::true_type{});

  // O^T: lane holds dims 16 hb + 4 lg + v of query column lq
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int row = q0 + qb * 16 + lq;
    if (row >= T) continue;
    const float inv = 1.f / lq_sum[qb];
    bf16_t* op = out + ((size_t)n * T + row) * ldq + h * HD + 4 * lg;
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) {
      const uint32_t w0 = (uint32_t)f2bf(oacc[hb][qb][0] * inv) |
                          ((uint32_t)f2bf(oacc[hb][qb][1] * inv) << 16);
      const uint32_t w1 = (uint32_t)f2bf(oacc[hb][qb][2] * inv) |
                          ((uint32_t)f2bf(oacc[hb][qb][3] * inv) << 16);
      *(uint2*)(op + hb * 16) = make_uint2(w0, w1);
    }
  }
}

template <int HD>
hipError_t launch_flash(int gq, dim3 grid, hipStream_t st, const bf16_t* q, const bf16_t* k,
                        const bf16_t* vt, int T, int H, int n_kv, int k_len, int k_seq_stride,
                        int vt_len, float scale, bf16_t* out, int q_pos0, int vt_seq_stride,
                        const int32_t* qpos, const int32_t* kslots) {
#define GRPO_FLASH(G)                                                                        \
  case G:                                                                                   \
    k_flash_bf16<HD, G><<<grid, 64 * G, 0, st>>>(q, k, vt, T, H, n_kv, k_len, k_seq_stride, \
                                                 vt_len, scale, out, q_pos0, vt_seq_stride, \
                                                 qpos, kslots);                             \
    break;
  switch (gq) {
    GRPO_FLASH(1) GRPO_FLASH(2) GRPO_FLASH(3) GRPO_FLASH(4)
    GRPO_FLASH(5) GRPO_FLASH(6) GRPO_FLASH(7) GRPO_FLASH(8)
    default: return hipErrorInvalidValue;
  }
#undef GRPO_FLASH
  return hipGetLastError();
}

// ------------------------------------------------------------------- fp32 path
// One workgroup per (query row, head).  Decode rows: seq = m, pos = pos_arr[m];
// sequence rows: seq = m / T, pos = m % T (K/V of sequence seq at cache slot
// seq * slot_mul).  Scores live in dynamic LDS (ctx floats).
__global__ __launch_bounds__(256) void k_attn_rows_f32(const float* __restrict__ q, int ldq,
                                                       const float* __restrict__ kc,
                                                       const float* __restrict__ vc,
                                                       const int32_t* pos_arr,
                                                       const int32_t* slots, int T, int slot_mul,
                                                       int H, int n_kv, int hd, int k_len,
                                                       float scale, float* __restrict__ out) {
  extern __shared__ float sc[];
  __shared__ float sh[4];
  const int m = blockIdx.x, h = blockIdx.y;
  int seq, p;
  if (pos_arr) { seq = slots ? slots[m] : m; p = pos_arr[m]; }
  else { seq = m / T; p = m % T; }
  p = min(p, k_len - 1);
  const int ctx = p + 1;
  const int g = h * n_kv / H;
  const float* qp = q + (size_t)m * ldq + h * hd;
  const size_t base = (((size_t)seq * slot_mul) * n_kv + g) * (size_t)k_len * hd;
  float mx = -INFINITY;
  for (int t = threadIdx.x; t < ctx; t += 256) {
    const float* kp = kc + base + (size_t)t * hd;
    float s = 0.f;
    for (int e = 0; e < hd; ++e) s = fmaf(qp[e], kp[e], s);
    s *= scale;
    sc[t] = s;
    mx = fmaxf(mx, s);
  }
  mx = block_max<256>(mx, sh);
  float sum = 0.f;
  for (int t = threadIdx.x; t < ctx; t += 256) {
    const float e = __expf(sc[t] - mx);
    sc[t] = e;
    sum += e;
  }
  sum = block_sum<256>(sum, sh);
  __syncthreads();
  for (int e = threadIdx.x; e < hd; e += 256) {
    float acc = 0.f;
    for (int t = 0; t < ctx; ++t) acc = fmaf(sc[t], vc[base + (size_t)t * hd + e], acc);
    out[(size_t)m * H * hd + h * hd + e] = acc / sum;
  }
}

}  // namespace

hipError_t attn_rows_f32(const float* q, const float* kc, const float* vc, const int32_t* pos,
                         const int32_t* slots, int rows, int T, int slot_mul, int H, int n_kv, int hd, int k_len,
                         float* out, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const float scale = 1.f / sqrtf((float)hd);
  dim3 grid(rows, H);
  Prof pf("attn_f32", st);
  k_attn_rows_f32<<<grid, 256, k_len * sizeof(float), st>>>(q, H * hd, kc, vc, pos, slots, T, slot_mul,
                                                            H, n_kv, hd, k_len, scale, out);
  return hipGetLastError();
}

hipError_t attn_prefill(int dtype, const void* q, const void* k, const void* v_or_vt, int N,
                        int T, int H, int n_kv, int hd, int k_len, int k_seq_stride, void* out,
                        hipStream_t st, int q_pos0, int vt_seq_stride, int vt_len_in,
                        const int32_t* qpos, const int32_t* kslots) {
  if (N <= 0 || T <= 0) return hipSuccess;
  const float scale = 1.f / sqrtf((float)hd);
  // (per-sequence offsets qpos: the caller guarantees qpos[n] + T <= k_len and
  // <= vt_len)
  if (q_pos0 < 0 || q_pos0 + T > k_len || vt_seq_stride < 1 ||
      (dtype == 0 && (q_pos0 || vt_seq_stride != 1 || qpos || kslots)))
    return hipErrorInvalidValue;
  if (dtype == 0) {
    dim3 grid(N * T, H);
    Prof pf("attn_f32", st);
    k_attn_rows_f32<<<grid, 256, T * sizeof(float), st>>>(
        (const float*)q, H * hd, (const float*)k, (const float*)v_or_vt, nullptr, nullptr, T,
        k_seq_stride,
        H, n_kv, hd, k_len, scale, (float*)out);
    return hipGetLastError();
  }
  const int vt_len = vt_len_in > 0 ? vt_len_in : (q_pos0 + T + 7) / 8 * 8;
  if (vt_len < q_pos0 + T) return hipErrorInvalidValue;
  dim3 grid((T + 31) / 32, n_kv, N);
  Prof pf("flash_attn", st);
  const int gq = H / n_kv;
  if (hd == 128)
    return launch_flash<128>(gq, grid, st, (const bf16_t*)q, (const bf16_t*)k,
                             (const bf16_t*)v_or_vt, T, H, n_kv, k_len, k_seq_stride, vt_len,
                             scale, (bf16_t*)out, q_pos0, vt_seq_stride, qpos, kslots);
  return launch_flash<64>(gq, grid, st, (const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v_or_vt,
                          T, H, n_kv, k_len, k_seq_stride, vt_len, scale, (bf16_t*)out, q_pos0,
                          vt_seq_stride, qpos, kslots);
}

}  // namespace grpo
