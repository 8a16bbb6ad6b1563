// Decode attention against the per-sequence KV cache (split-K over the context).
//
// bf16: one workgroup per (context span, kv head, sequence); the span is the
// whole context unless there are too few (sequence, kv head) pairs to fill the
// chip.  Each of the 4 waves (2 for grids of twice the workgroups that fit on
// the chip at once) streams tiles of 32 positions (tiles w, w+4, ...)
// with the next tile's K and V loads in flight while the current tile is
// computed, and keeps an online softmax (running max, sum and unnormalised
// output per query head).  QK^T runs on MFMA with the K tile as the A operand
// (16 positions x head_dim) and the group's query heads as the B columns; P.V
// runs on the vector units (each lane owns 8 head-dim elements of one position,
// 16-byte coalesced V loads).  K and V are loaded non-temporally: every cached
// byte is read once per step.  The waves are merged through LDS at the end; a
// single-span launch writes the normalised bf16 output directly, otherwise each
// span writes (max, sum, unnormalised o) and a second kernel merges the spans in
// span order.
//
// Grouped rollouts (the G samples of a prompt in consecutive batch rows, their
// prompt K/V identical): the prompt positions are read once per group.  A
// prefix launch, one workgroup per (prompt chunk, kv head, group), copies the
// group leader's K and V tiles straight into a 4-stage LDS ring (one copy per
// workgroup, three tiles ahead, one barrier per tile).  Its query columns are
// the heads of up to 32 / GQ samples (all 8 samples x 4 heads at the 7B shape),
// and both products run on MFMA: every wave computes the scores and softmax of
// all the columns and P.V for a quarter of the head dimension; the (max, sum,
// o) of each column form one span.  The per-sequence launch then covers the
// generated positions only and merges the prompt chunks into its result when
// those are a single span (else a merge kernel takes the prompt chunks first,
// then the generated spans).
//
// fp32 models use the plain vector kernel of the prefill path.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace grpo {

namespace {

constexpr int DT = 32;            // decode positions per wave tile
constexpr int SPAN_Q = 4 * DT;    // span granularity: one tile per wave
constexpr int MAX_CHUNKS = 16;    // prompt chunks of a grouped step, at most

// Grouped rollout: G samples per group (0 = every row on its own), prompt
// positions shared below prefix_len, n_sub workgroups per group and chunk (each
// holding 32 / GQ samples), `chunks` prompt chunks of span_p positions.
struct DecodeGroup { int G, prefix_len, n_sub, chunks, span_p; };

// Positions the group of batch row b shares: prefix_len, cut to the context
// every member has reached (so a shared position exists for all of them).
// The members' positions are read eight at a time (indices past the group
// repeat its last member), all eight loads in flight together.
__device__ __forceinline__ int group_shared(const int32_t* __restrict__ pos, int grp,
                                            const DecodeGroup& ga, int max_len) {
  int pl = ga.prefix_len;
  const int32_t* pg = pos + grp * ga.G;
  for (int i0 = 0; i0 < ga.G; i0 += 8) {
    int v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = pg[min(i0 + u, ga.G - 1)];
#pragma unroll
    for (int u = 0; u < 8; ++u) pl = min(pl, min(v[u], max_len - 1) + 1);
  }
  return pl;
}

// Positions per span of a row with n positions past its shared length, cut
// into `spans` spans (the merge kernel recomputes it the same way).
__device__ __forceinline__ int row_span(int n, int spans) {
  return max(SPAN_Q, ((n + spans - 1) / spans + SPAN_Q - 1) / SPAN_Q * SPAN_Q);
}

template <int HD, int NG, int NVT>
struct KVTile {
  u32x4_t k[NG][HD / 32];
  u32x4_t v[NVT];
};

// ---------------------------------------------------------------- decode, bf16
// NW waves per workgroup (4; 2 when the grid holds at least twice the
// workgroups of 4 waves that fit on the chip at once).
// blockIdx = (span, kv head, batch row); the spans start at the group's shared
// length when ga.G > 0 and write partial row split_base + span of S.  A grouped
// step whose generated positions are one span (S = chunks + 1) merges the prompt
// chunks' partials here and writes the output (no merge kernel).
template <int HD, int MAXG, int NW>
__global__ __launch_bounds__(64 * NW) void k_attn_decode_bf16(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    const int32_t* __restrict__ pos, const int32_t* __restrict__ slots, int H, int n_kv,
    int max_len, int S, float scale, float* __restrict__ part_o,
    float* __restrict__ part_ml, bf16_t* __restrict__ out, int pack_nb, DecodeGroup ga,
    int split_base) {
  constexpr int QSTEPS = HD / 32;     // MFMA k-steps over the head dim
  constexpr int LPT = HD / 8;         // lanes per position in P.V
  constexpr int PPW = 64 / LPT;       // positions per V load instruction
  constexpr int NVT = DT / PPW;       // V load instructions per tile
  constexpr int NG = DT / 16;         // MFMA position groups per tile
  constexpr int NT = 64 * NW;         // threads
  using Tile = KVTile<HD, NG, NVT>;
  static_assert(MAX_CHUNKS * MAXG <= NT, "one thread per prompt chunk and head");
  __shared__ __attribute__((aligned(16))) float pw[NW][DT][MAXG];
  __shared__ __attribute__((aligned(16))) float pa[NW][MAXG];
  __shared__ float red[NW][MAXG * HD];
  __shared__ float wm[NW][MAXG], wl[NW][MAXG];

  const int split = blockIdx.x, g = blockIdx.y;
  const int GQ = H / n_kv;
  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64;
  const int lg = lane >> 4;           // MFMA k-group of this lane
  const int j = lane & 15;            // MFMA row (position) / column (query head)
  const int ts = lane / LPT, hg = lane % LPT;
  // positions [t0, t1) of this workgroup
  const int src = blockIdx.z;
  const int ctx = min(pos[src], max_len - 1) + 1;
  const int base = ga.G > 0 ? group_shared(pos, src / ga.G, ga, max_len) : 0;
  const bool fold = ga.G > 0 && S == ga.chunks + 1;
  // the row's positions past `base` cut evenly into the plan's spans (whole
  // 128-position units, one tile per wave), so that every span has work as the
  // context grows; the last span runs to the row's end
  const int rspan = row_span(ctx - base, S - split_base);
  const int t0 = base + split * rspan;
  if (t0 >= ctx && !fold) return;             // (folding still merges the prompt part)
  const int t1 = split == S - split_base - 1 ? ctx : min(t0 + rspan, ctx);
  const int ntiles = t1 > t0 ? (t1 - t0 + DT - 1) / DT : 0;
  const int nmine = ntiles > wave ? (ntiles - wave + NW - 1) / NW : 0;
  const int slot = slots ? slots[src] : src;          // the row's cache slot
  const size_t head_base = ((size_t)slot * n_kv + g) * max_len;
  const bf16_t* kb = kc + head_base * HD;
  const bf16_t* vb = vc + head_base * HD;

  // query fragments; head-dim chunk (st * 4 + lg) of 8 elements feeds MFMA step st,
  // so each K load instruction reads 64 contiguous bytes per position
  bf16x8_t qf[QSTEPS];
  {
    const bf16_t* qp = q + ((size_t)src * H + g * GQ + min(j, GQ - 1)) * HD + lg * 8;
#pragma unroll
    for (int st = 0; st < QSTEPS; ++st) {
      u32x4_t v = *(const u32x4_t*)(qp + st * 32);
      if (j >= GQ) v = (u32x4_t){0u, 0u, 0u, 0u};
      qf[st] = __builtin_bit_cast(bf16x8_t, v);
    }
  }

  auto load = [&](Tile& tl, int i) {
    const int tb = t0 + (wave + NW * i) * DT;
#pragma unroll
    for (int grp = 0; grp < NG; ++grp) {
      const int t = min(tb + grp * 16 + j, t1 - 1);
      const bf16_t* kp = kb + (size_t)t * HD + lg * 8;
#pragma unroll
      for (int st = 0; st < QSTEPS; ++st)
        tl.k[grp][st] = __builtin_nontemporal_load((const u32x4_t*)(kp + st * 32));
    }
#pragma unroll
    for (int iv = 0; iv < NVT; ++iv) {
      const int t = min(tb + iv * PPW + ts, t1 - 1);
      tl.v[iv] = __builtin_nontemporal_load((const u32x4_t*)(vb + (size_t)t * HD + hg * 8));
    }
  };

  float m = -1e30f, l = 0.f;          // running max / partial sum of head j (this lane's rows)
  float o[MAXG][8];
#pragma unroll
  for (int h = 0; h < MAXG; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[h][e] = 0.f;

  auto compute = [&](const Tile& tl, int i) {
    const int tb = t0 + (wave + NW * i) * DT;
    float sv[NG][4];
    float tmax = -INFINITY;
#pragma unroll
    for (int grp = 0; grp < NG; ++grp) {
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < QSTEPS; ++st)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, tl.k[grp][st]),
                                                      qf[st], acc, 0, 0, 0);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float sc = (tb + grp * 16 + lg * 4 + v < t1) ? acc[v] * scale : -INFINITY;
        sv[grp][v] = sc;
        tmax = fmaxf(tmax, sc);
      }
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float mnew = fmaxf(m, tmax);
    const float alpha = __expf(m - mnew);
    m = mnew;
    float ps = 0.f;
#pragma unroll
    for (int grp = 0; grp < NG; ++grp)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float p = __expf(sv[grp][v] - mnew);
        ps += p;
        if (j < MAXG) pw[wave][grp * 16 + lg * 4 + v][j] = p;
      }
    l = l * alpha + ps;
    if (lg == 0 && j < MAXG) pa[wave][j] = alpha;
    __builtin_amdgcn_wave_barrier();
    float al[MAXG];
#pragma unroll
    for (int h = 0; h < MAXG; h += 4) {
      const float4 a4 = *(const float4*)&pa[wave][h];
      al[h] = a4.x; al[h + 1] = a4.y; al[h + 2] = a4.z; al[h + 3] = a4.w;
    }
    // all MAXG columns are updated (no per-head branches in the loop); columns
    // past GQ hold products of a zero query and are never written out
#pragma unroll
    for (int h = 0; h < MAXG; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) o[h][e] *= al[h];
#pragma unroll
    for (int iv = 0; iv < NVT; ++iv) {
      const u32x4_t raw = tl.v[iv];
      float vv[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        vv[2 * e] = __uint_as_float(raw[e] << 16);
        vv[2 * e + 1] = __uint_as_float(raw[e] & 0xffff0000u);
      }
      float pp[MAXG];
#pragma unroll
      for (int h = 0; h < MAXG; h += 4) {
        const float4 p4 = *(const float4*)&pw[wave][iv * PPW + ts][h];
        pp[h] = p4.x; pp[h + 1] = p4.y; pp[h + 2] = p4.z; pp[h + 3] = p4.w;
      }
#pragma unroll
      for (int h = 0; h < MAXG; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] = fmaf(pp[h], vv[e], o[h][e]);
    }
    __builtin_amdgcn_wave_barrier();
  };

  // two tiles in registers: the next one loads while the current one is used.
  // Past the wave's last tile the loads still go out (no branch, so the waits
  // stay those of the steady state) but take tile index nmine, which starts at
  // or past t1: every lane's position clamps to t1 - 1, so such a load reads one
  // row of K and V instead of a whole tile (in bounds, results unused).
  if (nmine > 0) {
    Tile ta, tb;
    load(ta, 0);
    for (int i = 0; i < nmine; i += 2) {
      load(tb, min(i + 1, nmine));
      compute(ta, i);
      load(ta, min(i + 2, nmine));
      if (i + 1 < nmine) compute(tb, i + 1);
    }
  }

  // The prompt chunks' partials (folding): issued here, without branches, so
  // that their latency overlaps the reductions below.  Chunk c of the shared
  // length is used when c < nused; an unused chunk's loads re-read chunk 0 and
  // count as (max -inf, sum 0, output 0) in the merge.  Thread i < MAX_CHUNKS * MAXG
  // loads the (max, sum) pair of chunk i / MAXG, head i % MAXG (shared by every
  // head-dim element: kept in LDS); every thread loads the output elements of
  // its NIT (head, element) pairs.
  constexpr int NIT = (MAXG * HD + NT - 1) / NT;
  __shared__ __attribute__((aligned(8))) float2 fml[MAX_CHUNKS][MAXG];
  float co[NIT][MAX_CHUNKS];
  float2 cml = make_float2(-INFINITY, 0.f);
  const int nused = fold ? min(ga.chunks, (base + ga.span_p - 1) / ga.span_p) : 0;
  if (fold) {
    const size_t rh = ((size_t)src * H + g * GQ) * S;   // partial row of head 0, chunk 0
    if (tid < MAX_CHUNKS * MAXG) {
      const int c = tid / MAXG, h = tid % MAXG;
      const bool u = c < nused && h < GQ;
      const float2 v = *(const float2*)(part_ml + (rh + (size_t)min(h, GQ - 1) * S + (u ? c : 0)) * 2);
      cml = u ? v : make_float2(-INFINITY, 0.f);
    }
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const int i = min(tid + NT * it, GQ * HD - 1);
      const float* pr = part_o + (rh + (size_t)(i / HD) * S) * HD + i % HD;
#pragma unroll
      for (int c = 0; c < MAX_CHUNKS; ++c) co[it][c] = pr[(size_t)(c < nused ? c : 0) * HD];
    }
  }

  // wave totals: o over the positions of a load instruction, l over the k-groups
#pragma unroll
  for (int h = 0; h < MAXG; ++h)
    if (h < GQ) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float x = o[h][e];
#pragma unroll
        for (int off = LPT; off < 64; off <<= 1) x += __shfl_xor(x, off, 64);
        o[h][e] = x;
      }
    }
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (lg == 0 && j < MAXG) { wm[wave][j] = m; wl[wave][j] = l; }
  if (ts == 0) {
#pragma unroll
    for (int h = 0; h < MAXG; ++h)
      if (h < GQ) {
#pragma unroll
        for (int e = 0; e < 8; ++e) red[wave][h * HD + hg * 8 + e] = o[h][e];
      }
  }
  if (fold && tid < MAX_CHUNKS * MAXG) fml[tid / MAXG][tid % MAXG] = cml;
  __syncthreads();
  // merge the NW waves (fixed order)
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int i = tid + NT * it;
    if (i >= GQ * HD) break;
    const int h = i / HD, e = i % HD;
    float M = wm[0][h];
#pragma unroll
    for (int w = 1; w < NW; ++w) M = fmaxf(M, wm[w][h]);
    float x = 0.f, L = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float c = __expf(wm[w][h] - M);
      x = fmaf(c, red[w][i], x);
      L = fmaf(c, wl[w][h], L);
    }
    if (fold) {
      // the prompt chunks below the shared length (partial rows 0 .. chunks-1)
      float Mt = M;
#pragma unroll
      for (int c = 0; c < MAX_CHUNKS; ++c) Mt = fmaxf(Mt, fml[c][h].x);
      const float sc = __expf(M - Mt);
      x *= sc;
      L *= sc;
#pragma unroll
      for (int c = 0; c < MAX_CHUNKS; ++c) {
        const float2 ml = fml[c][h];
        const float w = __expf(ml.x - Mt);   // 0 for unused chunks
        x = fmaf(c < nused ? co[it][c] : 0.f, w, x);
        L = fmaf(ml.y, w, L);
      }
    }
    if (S == 1 || fold) {
      const int k = (g * GQ + h) * HD + e;
      out[pack_nb ? act_frag_index(src, k, pack_nb) : (size_t)src * H * HD + k] = f2bf(x / L);
    } else {
      const size_t row = ((size_t)src * H + g * GQ + h) * S + split_base + split;
      part_o[row * HD + e] = x;
      if (e == 0) { part_ml[row * 2] = M; part_ml[row * 2 + 1] = L; }
    }
  }
}

// ------------------------------------------------- grouped prompt chunks, bf16
// 16 bytes per lane global -> LDS (lds + 16 lane), non-temporal.
__device__ __forceinline__ void dma16_nt(const bf16_t* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off nt" ::"s"(lds), "v"(g)
               : "memory");
}
// Stage swizzles (16-byte pieces XOR-ed per row).  K: the 16 rows one fragment
// read touches, 8 (i >> 2) + 4 b + (i & 3) for lane row i, fall in 16 distinct
// bank groups (hd 128: 256-byte rows, the swizzle takes row bits 0-1 and 3-4;
// hd 64: 128-byte rows, bits 1 and 3-4).  V: the four position groups 8 g + e
// one transposed read touches sit 2 pieces apart (row bits 3-4).
template <int HD>
__device__ __forceinline__ int kstage_swz(int r) {
  return HD == 128 ? ((r & 3) | (((r >> 3) & 3) << 2)) : (((r >> 1) & 1) | (((r >> 3) & 3) << 1));
}
__device__ __forceinline__ int vstage_swz(int r) { return ((r >> 3) & 3) << 1; }

// blockIdx = (chunk, kv head, group x n_sub).  Sub-block u takes the 16 NCB / GQ
// samples u * (16 NCB / GQ) .. of the group: query column c (NCB MFMA blocks of
// 16: 2, or 3 when that keeps a whole group in one sub-block)
// is head g * GQ + c % GQ of sample c / GQ.  Every wave computes the scores and
// softmax of all the columns (the same values in each wave) and O^T for its
// quarter of the head dimension, so a wave reads a quarter of the V^T fragments.
// Per 32-position tile: S^T = K Q^T on MFMA with the K rows of each 16-row block
// permuted (block b, row i -> position 8 (i >> 2) + 4 b + (i & 3)), so a lane's
// eight scores of its column are positions 8 g .. 8 g + 7: exactly the B operand
// of O^T += V^T P^T, which takes P as two bf16 terms (hi + lo: no rounding point
// added) and V^T fragments read transposed from the stage.
template <int HD, int NCB>
__global__ __launch_bounds__(256) void k_attn_prefix_bf16(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    const int32_t* __restrict__ pos, const int32_t* __restrict__ slots, int H, int n_kv,
    int max_len, int S, int span, float scale, float* __restrict__ part_o,
    float* __restrict__ part_ml, DecodeGroup ga) {
  constexpr int QSTEPS = HD / 32;
  constexpr int HB = HD / 16;         // 16-row head-dim blocks of O^T
  constexpr int HBW = HB / 4;         // blocks per wave
  constexpr int PPR = HD / 8;         // 16-byte pieces per row
  constexpr int RPC = 64 / PPR;       // rows per 1 KB copy
  constexpr int NCP = DT / RPC;       // copies per K (and per V) tile
  constexpr int NSTG = 4;             // LDS ring stages
  constexpr int CPW = 2 * NCP / 4;    // copies per wave and tile
  static_assert(DT == 32 && NCP % 4 == 0 && HB % 4 == 0, "tile, copy and block split");
  __shared__ __attribute__((aligned(1024))) bf16_t ks[NSTG][DT * HD];
  __shared__ __attribute__((aligned(1024))) bf16_t vs[NSTG][DT * HD];

  const int split = blockIdx.x, g = blockIdx.y;
  const int GQ = H / n_kv;
  const int tid = threadIdx.x, lane = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
  const int lg = lane >> 4, j = lane & 15;
  const int group = blockIdx.z / ga.n_sub;
  const int spb = 16 * NCB / GQ;                             // samples per sub-block
  const int s0 = blockIdx.z % ga.n_sub * spb;                // its first sample
  const int ncols = min(spb, ga.G - s0) * GQ;                // valid columns (> 0)
  const int t0 = split * span;
  const int t1 = min(t0 + span, group_shared(pos, group, ga, max_len));
  if (t0 >= t1) return;                       // the whole workgroup
  const int ntiles = (t1 - t0 + DT - 1) / DT;
  const int src = group * ga.G;               // the group leader's batch row
  const size_t head_base = ((size_t)(slots ? slots[src] : src) * n_kv + g) * max_len;
  const bf16_t* kb = kc + head_base * HD;
  const bf16_t* vb = vc + head_base * HD;

  // Q as the B operand of column block cb: column j -> c = 16 cb + j (zero past
  // ncols); MFMA step st takes piece 4 st + lg
  bf16x8_t qf[NCB][QSTEPS];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    const int c = min(16 * cb + j, ncols - 1);
    const bf16_t* qp =
        q + ((size_t)(src + s0 + c / GQ) * H + g * GQ + c % GQ) * HD + lg * 8;
#pragma unroll
    for (int st = 0; st < QSTEPS; ++st) {
      u32x4_t v = *(const u32x4_t*)(qp + st * 32);
      if (16 * cb + j >= ncols) v = (u32x4_t){0u, 0u, 0u, 0u};
      qf[cb][st] = __builtin_bit_cast(bf16x8_t, v);
    }
  }
  // the query loads complete before the copies start (the copies are counted by
  // hand below): an empty use of the fragments holds them here
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int st = 0; st < QSTEPS; ++st) asm volatile("" ::"v"(qf[cb][st]));

  // Tile t into stage t % NSTG: copy c fills rows
  // RPC c .. RPC c + RPC - 1, lane l the 16-byte slot l % PPR of row RPC c + l / PPR
  // with source piece slot ^ swizzle.  Positions past t1 - 1 read position t1 - 1
  // (masked scores, finite values).
  auto copy_tile = [&](int t) __attribute__((always_inline)) {
    const int stg = t % NSTG, tb = t0 + t * DT;
#pragma unroll
    for (int c0 = 0; c0 < NCP; c0 += 4) {
      const int c = c0 + wave;
      const int row = c * RPC + lane / PPR, slot = lane % PPR;
      const size_t p = (size_t)min(tb + row, t1 - 1) * HD;
      dma16_nt(kb + p + (slot ^ kstage_swz<HD>(row)) * 8, lds_addr(&ks[stg][c * 512]));
      dma16_nt(vb + p + (slot ^ vstage_swz(row)) * 8, lds_addr(&vs[stg][c * 512]));
    }
  };

  float m[NCB], l[NCB];   // per column block: column j
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) { m[cb] = -1e30f; l[cb] = 0.f; }
  f32x4_t oacc[HBW][NCB];   // O^T rows 16 (HBW wave + hb) + 4 lg + v of column j of block cb
#pragma unroll
  for (int hb = 0; hb < HBW; ++hb)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) oacc[hb][cb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int stg, int t) __attribute__((always_inline)) {
    const int tb = t0 + t * DT;
    const bf16_t* ksb = &ks[stg][0];
    const uint16_t* vsb = (const uint16_t*)&vs[stg][0];
    f32x4_t sacc[2][NCB];   // [b][cb]
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int row = 8 * (j >> 2) + 4 * b + (j & 3);      // this lane's A row
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) sacc[b][cb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < QSTEPS; ++st) {
        const bf16x8_t kf =
            *(const bf16x8_t*)(ksb + row * HD + ((st * 4 + lg) ^ kstage_swz<HD>(row)) * 8);
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
          sacc[b][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[cb][st], sacc[b][cb], 0, 0, 0);
      }
    }
    // lane (j, lg): sacc[b][cb][v] is position 8 lg + 4 b + v of the tile
    float sv[NCB][8], mnew[NCB];
    bool moved = false;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      float tmax = -INFINITY;
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float sc = (tb + 8 * lg + 4 * b + v < t1) ? sacc[b][cb][v] * scale : -INFINITY;
          sv[cb][4 * b + v] = sc;
          tmax = fmaxf(tmax, sc);
        }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
      mnew[cb] = fmaxf(m[cb], tmax);
      moved |= mnew[cb] != m[cb];
    }
    // rescale only when some column's maximum moved (otherwise the factor is 1)
    if (__builtin_amdgcn_ballot_w64(moved)) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        const float alpha = __expf(m[cb] - mnew[cb]);
        l[cb] *= alpha;
#pragma unroll
        for (int hb = 0; hb < HBW; ++hb)
#pragma unroll
          for (int v = 0; v < 4; ++v) oacc[hb][cb][v] *= alpha;
      }
    }
    bf16x8_t ph[NCB], pl[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      m[cb] = mnew[cb];
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const float p0 = __expf(sv[cb][e] - mnew[cb]), p1 = __expf(sv[cb][e + 1] - mnew[cb]);
        l[cb] += p0;
        l[cb] += p1;
        const bf16x2_t hi = __builtin_convertvector((f32x2_t){p0, p1}, bf16x2_t);
        const bf16x2_t lo =
            __builtin_convertvector((f32x2_t){p0 - (float)hi[0], p1 - (float)hi[1]}, bf16x2_t);
        ph[cb][e] = hi[0]; ph[cb][e + 1] = hi[1];
        pl[cb][e] = lo[0]; pl[cb][e + 1] = lo[1];
      }
    }
    // V^T fragment of block HBW wave + hb: row 16 (HBW wave + hb) + j (a head
    // dimension), positions 8 lg .. 8 lg + 7, read as 2-byte elements
#pragma unroll
    for (int hb = 0; hb < HBW; ++hb) {
      const int d = (HBW * wave + hb) * 16 + j;
      u32x4_t w;
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const int r0 = 8 * lg + e, r1 = r0 + 1;
        const uint32_t a = vsb[r0 * HD + (((d >> 3) ^ vstage_swz(r0)) << 3) + (d & 7)];
        const uint32_t c = vsb[r1 * HD + (((d >> 3) ^ vstage_swz(r1)) << 3) + (d & 7)];
        w[e / 2] = a | (c << 16);
      }
      const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, w);
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        oacc[hb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, ph[cb], oacc[hb][cb], 0, 0, 0);
        oacc[hb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pl[cb], oacc[hb][cb], 0, 0, 0);
      }
    }
  };

  // ring: tiles t + 1 .. min(t + NSTG - 2, ntiles - 1) stay in flight while this
  // wave waits for its copies of tile t (copies complete in issue order)
#pragma unroll
  for (int t = 0; t < NSTG - 1; ++t)
    if (t < ntiles) copy_tile(t);
  static_assert(NSTG == 4, "the waits below count two tiles ahead");
  for (int t = 0; t < ntiles; ++t) {
    const int ahead = ntiles - 1 - t;
    if (ahead >= 2) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * CPW) : "memory");
    else if (ahead == 1) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(CPW) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();   // every wave's copies of t landed; every wave is done with tile t - 1
    if (t + NSTG - 1 < ntiles) copy_tile(t + NSTG - 1);           // into tile t - 1's stage
    compute(t % NSTG, t);
  }

  // column c = 16 cb + j: head g * GQ + c % GQ of batch row src + s0 + c / GQ
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    float lt = l[cb];
    lt += __shfl_xor(lt, 16, 64);
    lt += __shfl_xor(lt, 32, 64);
    const int c = 16 * cb + j;
    if (c < ncols) {
      const size_t row = ((size_t)(src + s0 + c / GQ) * H + g * GQ + c % GQ) * S + split;
#pragma unroll
      for (int hb = 0; hb < HBW; ++hb)
        *(f32x4_t*)(part_o + row * HD + (HBW * wave + hb) * 16 + 4 * lg) = oacc[hb][cb];
      if (wave == 0 && lg == 0) {
        part_ml[row * 2] = m[cb];
        part_ml[row * 2 + 1] = lt;
      }
    }
  }
}

// Merge of the spans of (row b, head h) in partial-row order.  Grouped: rows
// 0 .. chunks-1 are the prompt chunks of span_p positions below the group's
// shared length, then the spans of the generated positions from there.
template <int HD>
__global__ __launch_bounds__(HD) void k_attn_combine(const float* __restrict__ part_o,
                                                     const float* __restrict__ part_ml,
                                                     const int32_t* __restrict__ pos, int H,
                                                     int max_len, int S,
                                                     bf16_t* __restrict__ out, int pack_nb,
                                                     DecodeGroup ga, int chunks, int span_p) {
  const int h = blockIdx.x, b = blockIdx.y, e = threadIdx.x;
  const int ctx = min(pos[b], max_len - 1) + 1;
  const int base = ga.G > 0 ? group_shared(pos, b / ga.G, ga, max_len) : 0;
  const int rspan = row_span(ctx - base, S - chunks);
  auto used = [&](int s) { return s < chunks ? s * span_p < base : base + (s - chunks) * rspan < ctx; };
  const size_t row0 = ((size_t)b * H + h) * S;
  float M = -INFINITY;
  for (int s = 0; s < S; ++s)
    if (used(s)) M = fmaxf(M, part_ml[(row0 + s) * 2]);
  float L = 0.f, acc = 0.f;
  for (int s = 0; s < S; ++s) {
    if (!used(s)) continue;
    const float w = __expf(part_ml[(row0 + s) * 2] - M);
    L = fmaf(part_ml[(row0 + s) * 2 + 1], w, L);
    acc = fmaf(part_o[(row0 + s) * HD + e], w, acc);
  }
  const int k = h * HD + e;
  out[pack_nb ? act_frag_index(b, k, pack_nb) : (size_t)b * H * HD + k] = f2bf(acc / L);
}

}  // namespace

DecodeAttnPlan decode_attn_plan(int B, int H, int n_kv, int hd, int max_len, int G,
                                int prefix_len) {
  // enough spans for about two workgroups per compute unit; one span (and no
  // merge kernel) whenever the (sequence, kv head) pairs alone reach that
  constexpr int kTargetWGs = 512;
  const int pairs = std::max(1, B * n_kv);
  const int max_spans = (max_len + SPAN_Q - 1) / SPAN_Q;
  const int want = std::min(std::max(1, (kTargetWGs + pairs / 2) / pairs), max_spans);
  DecodeAttnPlan p{};
  p.tc = ((max_len + want - 1) / want + SPAN_Q - 1) / SPAN_Q * SPAN_Q;
  p.splits = (max_len + p.tc - 1) / p.tc;
  // two workgroups of 4 waves fit on a compute unit (registers); a grid of at
  // least twice that would run in two or more rounds, each paying the
  // workgroups' fixed start and merge, so it takes workgroups of 2 waves (four
  // per unit, the same 8 waves: 1B, 1024 workgroups, 35.0 -> 33.2 us per
  // launch).  Between one and two chips' worth (batch 96 at the 7B shape, 768
  // workgroups) 2 waves would leave 6 waves per unit: 76.1 -> 80.6 us.
  p.waves = (long)p.splits * n_kv * B >= 2 * kTargetWGs ? 2 : 4;
  p.part_floats = p.splits > 1 ? (size_t)B * H * p.splits * (hd + 2) : 0;
  if (G <= 0 || prefix_len <= 0) return p;
  // grouped: the prompt is cut into chunks of whole tiles, about kTargetWGs
  // prefix workgroups in all
  // samples per prefix workgroup: 2 column blocks of 16 (query heads of its
  // samples), 3 when that takes the whole group in one workgroup where 2 do not
  // (32B: 8 samples x 5 heads; the paper's K = 12 at 4 heads), so that the
  // group's prompt K/V is read once
  const int gq = std::max(1, H / n_kv);
  const int spb2 = 32 / gq, spb3 = 48 / gq;
  p.ncb = (G + spb3 - 1) / spb3 < (G + spb2 - 1) / spb2 ? 3 : 2;
  const int spb = 16 * p.ncb / gq;
  p.G = G;
  p.prefix_len = std::min(prefix_len, max_len);
  p.n_sub = (G + spb - 1) / spb;
  const int gpairs = std::max(1, B / G * n_kv * p.n_sub);
  const int max_chunks = std::min(MAX_CHUNKS, (p.prefix_len + DT - 1) / DT);
  const int wc = std::min(std::max(1, (kTargetWGs + gpairs / 2) / gpairs), max_chunks);
  p.span_p = ((p.prefix_len + wc - 1) / wc + DT - 1) / DT * DT;
  p.chunks = (p.prefix_len + p.span_p - 1) / p.span_p;
  // the per-row spans start at the shared length: sized on the positions past
  // the prompt (32B: 4095 of a 12287-position cache, two spans of 2048 instead
  // of one busy span of 6144 and one never reached), the last one open-ended
  const int gen = std::max(1, max_len - p.prefix_len);
  const int gspans = std::min(std::max(1, (kTargetWGs + pairs / 2) / pairs),
                              (gen + SPAN_Q - 1) / SPAN_Q);
  p.tc = ((gen + gspans - 1) / gspans + SPAN_Q - 1) / SPAN_Q * SPAN_Q;
  p.splits = (gen + p.tc - 1) / p.tc;
  p.waves = (long)p.splits * n_kv * B >= 2 * kTargetWGs ? 2 : 4;
  p.part_floats = (size_t)B * H * (p.chunks + p.splits) * (hd + 2);
  return p;
}

size_t decode_attn_part_floats_max(int B, int H, int n_kv, int hd, int max_len) {
  // grouped or not, a plan has at most `want` per-row spans (the count the
  // ungrouped plan aims at; its rounding can only lower it) and MAX_CHUNKS chunks
  const int pairs = std::max(1, B * n_kv);
  const int want = std::min(std::max(1, (512 + pairs / 2) / pairs), (max_len + SPAN_Q - 1) / SPAN_Q);
  const DecodeAttnPlan p = decode_attn_plan(B, H, n_kv, hd, max_len);
  return (size_t)B * H * (MAX_CHUNKS + std::max(p.splits, want)) * (hd + 2);
}

template <int HD, int MAXG>
static void launch_decode(dim3 grid, int waves, hipStream_t st, const void* q, const void* kc,
                          const void* vc, const int32_t* pos, const int32_t* slots, int H,
                          int n_kv, int max_len, int S, float scale, float* part_o,
                          float* part_ml, void* out, int pack_nb, DecodeGroup ga,
                          int split_base) {
  if (waves == 2)
    k_attn_decode_bf16<HD, MAXG, 2><<<grid, 128, 0, st>>>(
        (const bf16_t*)q, (const bf16_t*)kc, (const bf16_t*)vc, pos, slots, H, n_kv, max_len, S,
        scale, part_o, part_ml, (bf16_t*)out, pack_nb, ga, split_base);
  else
    k_attn_decode_bf16<HD, MAXG, 4><<<grid, 256, 0, st>>>(
        (const bf16_t*)q, (const bf16_t*)kc, (const bf16_t*)vc, pos, slots, H, n_kv, max_len, S,
        scale, part_o, part_ml, (bf16_t*)out, pack_nb, ga, split_base);
}

template <int HD>
static hipError_t attn_decode_hd(const void* q, const void* kc, const void* vc,
                                 const int32_t* pos, const int32_t* slots, int B, int H, int n_kv, int max_len,
                                 const DecodeAttnPlan& p, float* part, void* out, hipStream_t st,
                                 int pack_nb) {
  const float scale = 1.f / sqrtf((float)HD);
  const int gq = H / n_kv;
  const bool grouped = p.G > 0;
  const int S = p.chunks + p.splits;      // partial rows per (row, head)
  float* part_o = S > 1 ? part : nullptr;
  float* part_ml = S > 1 ? part + (size_t)B * H * S * HD : nullptr;
  const DecodeGroup ga{p.G, p.prefix_len, p.n_sub, p.chunks, p.span_p};
  if (grouped) {
    Prof pf("attn_prefix", st);
    dim3 grid(p.chunks, n_kv, B / p.G * p.n_sub);
    if (p.ncb == 3)
      k_attn_prefix_bf16<HD, 3><<<grid, 256, 0, st>>>(
          (const bf16_t*)q, (const bf16_t*)kc, (const bf16_t*)vc, pos, slots, H, n_kv, max_len,
          S, p.span_p, scale, part_o, part_ml, ga);
    else
      k_attn_prefix_bf16<HD, 2><<<grid, 256, 0, st>>>(
          (const bf16_t*)q, (const bf16_t*)kc, (const bf16_t*)vc, pos, slots, H, n_kv, max_len,
          S, p.span_p, scale, part_o, part_ml, ga);
  }
  {
    Prof pf("attn_decode", st);
    dim3 grid(p.splits, n_kv, B);
    if (gq <= 4)
      launch_decode<HD, 4>(grid, p.waves, st, q, kc, vc, pos, slots, H, n_kv, max_len, S, scale,
                           part_o, part_ml, out, pack_nb, ga, p.chunks);
    else
      launch_decode<HD, 8>(grid, p.waves, st, q, kc, vc, pos, slots, H, n_kv, max_len, S, scale,
                           part_o, part_ml, out, pack_nb, ga, p.chunks);
  }
  // grouped with one span of generated positions: merged by the per-row kernel
  if (S > 1 && !(grouped && p.splits == 1)) {
    Prof pf("attn_combine", st);
    k_attn_combine<HD><<<dim3(H, B), HD, 0, st>>>(part_o, part_ml, pos, H, max_len, S,
                                                  (bf16_t*)out, pack_nb, ga, p.chunks, p.span_p);
  }
  return hipGetLastError();
}

hipError_t attn_decode(int dtype, const void* q, const void* kc, const void* vc,
                       const int32_t* pos, const int32_t* slots, int B, int H, int n_kv, int hd, int n_seqs, int max_len,
                       const DecodeAttnPlan& p, float* part, void* out, hipStream_t st,
                       int pack_nb) {
  (void)n_seqs;
  if (B <= 0) return hipSuccess;
  if (pack_nb && (dtype == 0 || B > pack_nb || pack_nb % 16)) return hipErrorInvalidValue;
  if (dtype == 0)
    return attn_rows_f32((const float*)q, (const float*)kc, (const float*)vc, pos, slots, B, 1, 1,
                         H, n_kv, hd, max_len, (float*)out, st);
  if (H % n_kv || H / n_kv > 8 || (hd != 64 && hd != 128) || (p.waves != 2 && p.waves != 4))
    return hipErrorInvalidValue;
  if (p.G > 0 && (B % p.G || p.chunks < 1 || p.chunks > MAX_CHUNKS || p.n_sub < 1 ||
                  (p.ncb != 2 && p.ncb != 3) ||
                  (long)p.n_sub * (16 * p.ncb / (H / n_kv)) < p.G || p.prefix_len > max_len ||
                  (long)p.chunks * p.span_p < p.prefix_len))
    return hipErrorInvalidValue;
  return hd == 128 ? attn_decode_hd<128>(q, kc, vc, pos, slots, B, H, n_kv, max_len, p, part, out,
                                         st, pack_nb)
                   : attn_decode_hd<64>(q, kc, vc, pos, slots, B, H, n_kv, max_len, p, part, out,
                                        st, pack_nb);
}

}  // namespace grpo
