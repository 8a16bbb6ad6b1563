// Attention of the decoder: decode against the per-sequence KV cache
// (split-K over the context) and causal attention for prompt prefill and
// teacher-forced scoring.
//
// Decode (bf16): one workgroup per (context split of 256 positions, kv head,
// sequence).  The K tile is streamed straight into MFMA operands (16 positions x
// head_dim per MFMA, the group's query heads as the 16 B-columns), scores go to
// LDS, softmax statistics are block reductions, and P.V runs on the vector
// units with 16-byte coalesced V loads (each lane owns 8 head-dim elements of
// one position).  Each split writes (max, sum, unnormalised o); a second kernel
// merges the splits in split order.
//
// Prefill / scoring (bf16): flash attention.  One workgroup per (64 queries,
// head, sequence), 16 query rows per wave; K tiles and transposed V tiles
// (written transposed by the rotary kernel) staged in LDS; S = Q K^T and
// O += P V on v_mfma_f32_16x16x32_bf16 with an fp32 online softmax; P enters
// the second product as a sum of two bf16 terms, so no extra rounding point is
// introduced.  Key tiles above the diagonal are skipped.
//
// fp32 models use a plain vector kernel (one workgroup per query row and head).
#include "common.h"
#include "kernels.h"

namespace grpo {

namespace {

constexpr int TC = 256;  // decode positions per split

// ---------------------------------------------------------------- decode, bf16
// All K and V loads of the split are issued before any arithmetic (K straight
// into MFMA operand registers, V into the registers P.V consumes), so the
// workgroup keeps its whole 2 x 64 KB tile in flight.
template <int HD>
__global__ __launch_bounds__(256) void k_attn_decode_bf16(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    const int32_t* __restrict__ pos, int H, int n_kv, int max_len, int S, float scale,
    float* __restrict__ part_o, float* __restrict__ part_ml) {
  constexpr int QSTEPS = HD / 32;     // MFMA k-steps over the head dim
  constexpr int LPT = HD / 8;         // lanes per position in P.V
  constexpr int PPW = 64 / LPT;       // positions per wave per P.V step
  constexpr int NV = TC / (4 * PPW);  // V loads per lane
  constexpr int MAXG = 8;
  __shared__ __attribute__((aligned(16))) float pt[TC][MAXG];
  __shared__ float red[4][MAXG * HD];
  __shared__ float wm[4][MAXG], wl[4][MAXG];

  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int GQ = H / n_kv;
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
  const int ctx = min(pos[b], max_len - 1) + 1;
  const int t0 = split * TC;
  if (t0 >= ctx) return;
  const size_t head_base = ((size_t)b * n_kv + g) * max_len;
  const bf16_t* kb = kc + head_base * HD;
  const bf16_t* vb = vc + head_base * HD;
  const int lg = lane >> 4;           // lane group: owns dims [lg*HD/4, (lg+1)*HD/4)
  const int j = lane & 15;            // query head of this lane's MFMA column
  const int ts = lane / LPT, hg = lane % LPT;

  // ---- issue every load of the split ----
  u32x4_t kreg[4][QSTEPS];
#pragma unroll
  for (int grp = 0; grp < 4; ++grp) {
    const int t = min(t0 + wave * 64 + grp * 16 + j, ctx - 1);
    const bf16_t* kp = kb + (size_t)t * HD + lg * (HD / 4);
#pragma unroll
    for (int st = 0; st < QSTEPS; ++st) kreg[grp][st] = *(const u32x4_t*)(kp + st * 8);
  }
  u32x4_t vreg[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int t = min(t0 + k * 4 * PPW + wave * PPW + ts, ctx - 1);
    vreg[k] = *(const u32x4_t*)(vb + (size_t)t * HD + hg * 8);
  }
  bf16x8_t qf[QSTEPS];
  {
    const bf16_t* qp = q + ((size_t)b * H + g * GQ + min(j, GQ - 1)) * HD + lg * (HD / 4);
#pragma unroll
    for (int st = 0; st < QSTEPS; ++st) {
      u32x4_t v = *(const u32x4_t*)(qp + st * 8);
      if (j >= GQ) v = (u32x4_t){0u, 0u, 0u, 0u};
      qf[st] = __builtin_bit_cast(bf16x8_t, v);
    }
  }

  // ---- S = K Q^T on MFMA: lane holds positions grp*16 + 4*lg + v of head j ----
  float sv[4][4];
  float mx = -INFINITY;
#pragma unroll
  for (int grp = 0; grp < 4; ++grp) {
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < QSTEPS; ++st)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kreg[grp][st]),
                                                    qf[st], acc, 0, 0, 0);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int tt = wave * 64 + grp * 16 + lg * 4 + v;
      const float sc = (t0 + tt < ctx) ? acc[v] * scale : -INFINITY;
      sv[grp][v] = sc;
      mx = fmaxf(mx, sc);
    }
  }
  // per-head max: over this lane's 16 values, then the 4 lane groups, then the waves
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  if (lg == 0 && j < MAXG) wm[wave][j] = mx;
  __syncthreads();
  const float m = (j < GQ) ? fmaxf(fmaxf(wm[0][j], wm[1][j]), fmaxf(wm[2][j], wm[3][j])) : 0.f;
  float sum = 0.f;
#pragma unroll
  for (int grp = 0; grp < 4; ++grp)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float p = (sv[grp][v] == -INFINITY) ? 0.f : __expf(sv[grp][v] - m);
      sum += p;
      if (j < GQ) pt[wave * 64 + grp * 16 + lg * 4 + v][j] = p;
    }
  sum += __shfl_xor(sum, 16, 64);
  sum += __shfl_xor(sum, 32, 64);
  if (lg == 0 && j < MAXG) wl[wave][j] = sum;
  __syncthreads();

  // ---- o = P V on the vector units, V already in registers ----
  float o[MAXG][8];
#pragma unroll
  for (int jj = 0; jj < MAXG; ++jj)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[jj][e] = 0.f;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int tt = k * 4 * PPW + wave * PPW + ts;
    const u32x4_t raw = vreg[k];
    float v[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[2 * e] = __uint_as_float(raw[e] << 16);
      v[2 * e + 1] = __uint_as_float(raw[e] & 0xffff0000u);
    }
#pragma unroll
    for (int jj = 0; jj < MAXG; ++jj) {
      if (jj < GQ) {
        const float p = pt[tt][jj];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[jj][e] = fmaf(p, v[e], o[jj][e]);
      }
    }
  }
  // reduce the positions of a wave (lanes with equal hg), then the 4 waves
#pragma unroll
  for (int jj = 0; jj < MAXG; ++jj) {
    if (jj < GQ) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float x = o[jj][e];
#pragma unroll
        for (int off = LPT; off < 64; off <<= 1) x += __shfl_xor(x, off, 64);
        o[jj][e] = x;
      }
    }
  }
  if (ts == 0) {
#pragma unroll
    for (int jj = 0; jj < MAXG; ++jj)
      if (jj < GQ) {
#pragma unroll
        for (int e = 0; e < 8; ++e) red[wave][jj * HD + hg * 8 + e] = o[jj][e];
      }
  }
  __syncthreads();
  for (int i = tid; i < GQ * HD; i += 256) {
    const int jj = i / HD, e = i % HD;
    const float x = red[0][i] + red[1][i] + red[2][i] + red[3][i];
    const size_t row = ((size_t)b * H + g * GQ + jj) * S + split;
    part_o[row * HD + e] = x;
    if (e == 0) {
      part_ml[row * 2] = fmaxf(fmaxf(wm[0][jj], wm[1][jj]), fmaxf(wm[2][jj], wm[3][jj]));
      part_ml[row * 2 + 1] = (wl[0][jj] + wl[1][jj]) + (wl[2][jj] + wl[3][jj]);
    }
  }
}

template <int HD>
__global__ __launch_bounds__(HD) void k_attn_combine(const float* __restrict__ part_o,
                                                     const float* __restrict__ part_ml,
                                                     const int32_t* __restrict__ pos, int H,
                                                     int max_len, int S, bf16_t* __restrict__ out) {
  const int h = blockIdx.x, b = blockIdx.y, e = threadIdx.x;
  const int ctx = min(pos[b], max_len - 1) + 1;
  const int ns = min(S, (ctx + TC - 1) / TC);
  const size_t row0 = ((size_t)b * H + h) * S;
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, part_ml[(row0 + s) * 2]);
  float L = 0.f, acc = 0.f;
  for (int s = 0; s < ns; ++s) {
    const float w = __expf(part_ml[(row0 + s) * 2] - M);
    L = fmaf(part_ml[(row0 + s) * 2 + 1], w, L);
    acc = fmaf(part_o[(row0 + s) * HD + e], w, acc);
  }
  out[((size_t)b * H + h) * HD + e] = f2bf(acc / L);
}

// ----------------------------------------------------------- flash attention, bf16
template <int HD>
__global__ __launch_bounds__(256) void k_flash_bf16(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ vt,
    int T, int H, int n_kv, int k_len, int k_seq_stride, int vt_len, float scale,
    bf16_t* __restrict__ out) {
  constexpr int KROW = HD + 8, VROW = 64 + 8, PROW = 64 + 8;
  constexpr int QSTEPS = HD / 32, HB = HD / 16;
  __shared__ __attribute__((aligned(16))) bf16_t ks[64 * KROW];
  __shared__ __attribute__((aligned(16))) bf16_t vs[HD * VROW];
  __shared__ __attribute__((aligned(16))) bf16_t ps[2][4][16 * PROW];   // P = hi + lo

  const int qb = blockIdx.x, h = blockIdx.y, n = blockIdx.z;
  const int g = h * n_kv / H;
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
  const int ldq = H * HD;
  const int r0 = qb * 64 + wave * 16;

  bf16x8_t qf[QSTEPS];
  {
    const int r = min(r0 + (lane & 15), T - 1);
    const bf16_t* qp = q + ((size_t)n * T + r) * ldq + h * HD + (lane >> 4) * 8;
#pragma unroll
    for (int st = 0; st < QSTEPS; ++st) qf[st] = *(const bf16x8_t*)(qp + st * 32);
  }
  const bf16_t* kbase = k + ((size_t)n * k_seq_stride * n_kv + g) * (size_t)k_len * HD;
  const bf16_t* vbase = vt + ((size_t)n * n_kv + g) * (size_t)HD * vt_len;

  f32x4_t oacc[HB];
#pragma unroll
  for (int i = 0; i < HB; ++i) oacc[i] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
  float mrow[4], lrow[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) { mrow[v] = -1e30f; lrow[v] = 0.f; }

  const int last_kb = min(qb, (T - 1) / 64);
  for (int kb = 0; kb <= last_kb; ++kb) {
    // stage K [64 keys][HD] and Vt [HD][64 keys]
    for (int i = tid; i < 64 * HD / 8; i += 256) {
      const int r = i / (HD / 8), c = (i % (HD / 8)) * 8;
      const int key = min(kb * 64 + r, T - 1);
      *(u32x4_t*)(&ks[r * KROW + c]) = *(const u32x4_t*)(kbase + (size_t)key * HD + c);
    }
    for (int i = tid; i < HD * 8; i += 256) {
      const int r = i / 8, c = (i % 8) * 8;
      const int key0 = kb * 64 + c;
      u32x4_t v = (u32x4_t){0u, 0u, 0u, 0u};
      if (key0 < T) {
        v = *(const u32x4_t*)(vbase + (size_t)r * vt_len + key0);
        const int nv = T - key0;   // keys past T are zeroed
        if (nv < 8) {
          uint32_t w[4] = {v[0], v[1], v[2], v[3]};
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (e >= nv) w[e / 2] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
          v = (u32x4_t){w[0], w[1], w[2], w[3]};
        }
      }
      *(u32x4_t*)(&vs[r * VROW + c]) = v;
    }
    __syncthreads();

    // S = Q K^T: 16 rows x 64 keys per wave
    f32x4_t sacc[4];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      sacc[cb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < QSTEPS; ++st) {
        const bf16x8_t kf =
            *(const bf16x8_t*)(&ks[(cb * 16 + (lane & 15)) * KROW + st * 32 + (lane >> 4) * 8]);
        sacc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[st], kf, sacc[cb], 0, 0, 0);
      }
    }
    // online softmax; lane holds rows 4*(lane>>4)+v, keys cb*16 + (lane&15)
    float mnew[4], alpha[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = r0 + (lane >> 4) * 4 + v;
      float mx = -1e30f;
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        const int key = kb * 64 + cb * 16 + (lane & 15);
        float s = sacc[cb][v] * scale;
        s = (key <= row && key < T) ? s : -INFINITY;
        sacc[cb][v] = s;
        mx = fmaxf(mx, s);
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
      mnew[v] = fmaxf(mrow[v], mx);
      alpha[v] = __expf(mrow[v] - mnew[v]);
      float sum = 0.f;
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        const float p = (sacc[cb][v] == -INFINITY) ? 0.f : __expf(sacc[cb][v] - mnew[v]);
        const bf16_t ph = f2bf(p);
        const bf16_t pl = f2bf(p - bf2f(ph));
        sum += p;
        const int at = ((lane >> 4) * 4 + v) * PROW + cb * 16 + (lane & 15);
        ps[0][wave][at] = ph;
        ps[1][wave][at] = pl;
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) sum += __shfl_xor(sum, off, 64);
      lrow[v] = lrow[v] * alpha[v] + sum;
      mrow[v] = mnew[v];
    }
#pragma unroll
    for (int hb = 0; hb < HB; ++hb)
#pragma unroll
      for (int v = 0; v < 4; ++v) oacc[hb][v] *= alpha[v];
    __syncthreads();   // ps visible within the wave (and vs/ks reads ordered)

    // O += P V: A = P (16 rows x 32 keys), B = V (32 keys x 16 dims).  P enters
    // as two bf16 terms (hi + lo), so P V is accurate to fp32 level.
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int at = (lane & 15) * PROW + kk * 32 + (lane >> 4) * 8;
      const bf16x8_t ph = *(const bf16x8_t*)(&ps[0][wave][at]);
      const bf16x8_t pl = *(const bf16x8_t*)(&ps[1][wave][at]);
#pragma unroll
      for (int hb = 0; hb < HB; ++hb) {
        const bf16x8_t vf =
            *(const bf16x8_t*)(&vs[(hb * 16 + (lane & 15)) * VROW + kk * 32 + (lane >> 4) * 8]);
        oacc[hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph, vf, oacc[hb], 0, 0, 0);
        oacc[hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl, vf, oacc[hb], 0, 0, 0);
      }
    }
    __syncthreads();
  }

#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int row = r0 + (lane >> 4) * 4 + v;
    if (row >= T) continue;
    const float inv = 1.f / lrow[v];
    bf16_t* op = out + ((size_t)n * T + row) * ldq + h * HD;
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) op[hb * 16 + (lane & 15)] = f2bf(oacc[hb][v] * inv);
  }
}

// ------------------------------------------------------------------- fp32 path
// One workgroup per (query row, head).  Decode rows: seq = m, pos = pos_arr[m];
// sequence rows: seq = m / T, pos = m % T (K/V of sequence seq at cache slot
// seq * slot_mul).  Scores live in dynamic LDS (ctx floats).
__global__ __launch_bounds__(256) void k_attn_rows_f32(const float* __restrict__ q, int ldq,
                                                       const float* __restrict__ kc,
                                                       const float* __restrict__ vc,
                                                       const int32_t* pos_arr, int T, int slot_mul,
                                                       int H, int n_kv, int hd, int k_len,
                                                       float scale, float* __restrict__ out) {
  extern __shared__ float sc[];
  __shared__ float sh[4];
  const int m = blockIdx.x, h = blockIdx.y;
  int seq, p;
  if (pos_arr) { seq = m; p = pos_arr[m]; }
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

DecodeAttnPlan decode_attn_plan(int B, int H, int hd, int max_len) {
  DecodeAttnPlan p;
  p.tc = TC;
  p.splits = (max_len + TC - 1) / TC;
  p.part_floats = (size_t)B * H * p.splits * (hd + 2);
  return p;
}

hipError_t attn_decode(int dtype, const void* q, const void* kc, const void* vc,
                       const int32_t* pos, int B, int H, int n_kv, int hd, int n_seqs, int max_len,
                       const DecodeAttnPlan& p, float* part, void* out, hipStream_t st) {
  (void)n_seqs;
  if (B <= 0) return hipSuccess;
  const float scale = 1.f / sqrtf((float)hd);
  if (dtype == 0) {
    dim3 grid(B, H);
    Prof pf("attn_f32", st);
    k_attn_rows_f32<<<grid, 256, max_len * sizeof(float), st>>>(
        (const float*)q, H * hd, (const float*)kc, (const float*)vc, pos, 1, 1, H, n_kv, hd,
        max_len, scale, (float*)out);
    return hipGetLastError();
  }
  float* part_o = part;
  float* part_ml = part + (size_t)B * H * p.splits * hd;
  dim3 grid(p.splits, n_kv, B);
  dim3 cgrid(H, B);
  {
    Prof pf("attn_decode", st);
    if (hd == 128)
      k_attn_decode_bf16<128><<<grid, 256, 0, st>>>((const bf16_t*)q, (const bf16_t*)kc,
                                                    (const bf16_t*)vc, pos, H, n_kv, max_len,
                                                    p.splits, scale, part_o, part_ml);
    else
      k_attn_decode_bf16<64><<<grid, 256, 0, st>>>((const bf16_t*)q, (const bf16_t*)kc,
                                                   (const bf16_t*)vc, pos, H, n_kv, max_len,
                                                   p.splits, scale, part_o, part_ml);
  }
  {
    Prof pf("attn_combine", st);
    if (hd == 128)
      k_attn_combine<128><<<cgrid, 128, 0, st>>>(part_o, part_ml, pos, H, max_len, p.splits,
                                                 (bf16_t*)out);
    else
      k_attn_combine<64><<<cgrid, 64, 0, st>>>(part_o, part_ml, pos, H, max_len, p.splits,
                                               (bf16_t*)out);
  }
  return hipGetLastError();
}

hipError_t attn_prefill(int dtype, const void* q, const void* k, const void* v_or_vt, int N,
                        int T, int H, int n_kv, int hd, int k_len, int k_seq_stride, void* out,
                        hipStream_t st) {
  if (N <= 0 || T <= 0) return hipSuccess;
  const float scale = 1.f / sqrtf((float)hd);
  if (dtype == 0) {
    dim3 grid(N * T, H);
    Prof pf("attn_f32", st);
    k_attn_rows_f32<<<grid, 256, T * sizeof(float), st>>>(
        (const float*)q, H * hd, (const float*)k, (const float*)v_or_vt, nullptr, T, k_seq_stride,
        H, n_kv, hd, k_len, scale, (float*)out);
    return hipGetLastError();
  }
  const int vt_len = (T + 7) / 8 * 8;
  dim3 grid((T + 63) / 64, H, N);
  Prof pf("flash_attn", st);
  if (hd == 128)
    k_flash_bf16<128><<<grid, 256, 0, st>>>((const bf16_t*)q, (const bf16_t*)k,
                                            (const bf16_t*)v_or_vt, T, H, n_kv, k_len,
                                            k_seq_stride, vt_len, scale, (bf16_t*)out);
  else
    k_flash_bf16<64><<<grid, 256, 0, st>>>((const bf16_t*)q, (const bf16_t*)k,
                                           (const bf16_t*)v_or_vt, T, H, n_kv, k_len, k_seq_stride,
                                           vt_len, scale, (bf16_t*)out);
  return hipGetLastError();
}

}  // namespace grpo
