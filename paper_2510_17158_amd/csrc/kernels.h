// Host-side launchers of the HIP kernels (internal interface of libgrpo_hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace grpo {

// Kernel timing for benchmarks: while profiling is on (grpo_profile_begin),
// each launch is bracketed by HIP events on its stream and accumulated under
// its name.  Off, a Prof costs one relaxed flag read.
struct Prof {
  Prof(const char* name, hipStream_t st);
  ~Prof();
  const char* name;
  hipStream_t st;
  void* ev0;
};
bool profiling();

// STORE: out = X W^T;  RESID: out += X W^T;  SWIGLU: out = silu(gate) * up;
// PARTIAL (decode GEMM only): out[split] = this split's share of X W^T, the
// consumer adds the splits;  LSE (row-tile GEMMs, the scoring LM head): the
// product's log-sum-exp pieces per row instead of the product (LseArgs).
// SAMPLE (decode GEMM, the LM head): the sampler's pieces per row and output tile
// instead of the logits (DecSample).
enum Epi { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_PARTIAL = 3, EPI_LSE = 4,
           EPI_SAMPLE = 5 };
constexpr int kMaxSplits = 16;

// Up to three weight matrices stacked along the output dimension: output row r
// belongs to w[0] for r < n1, to w[1] for n1 <= r < n2, else to w[2].
struct WStack {
  const void* w[3];
  int n1, n2;
};

// A batch of products with the same shape: product b reads X + b sx, the
// weights + (b / wdiv) sw and writes out + b so (elements).  tri, for causal
// products whose output rows m pair with columns or k-indices n <= m: 1 = output
// tiles lying wholly above the diagonal (every column > every row) are not
// computed (nor written: their consumer never reads them); 2 = X[m][k] is zero
// for k > m, and each row tile's k loop ends after its last row; 3 = X[m][k] is
// zero for k < m, and each row tile's k loop starts at its first row.  The bf16
// row-tile kernel honours tri (its callers may leave X unwritten outside the
// band of kTiledRows rows its row tiles still read); the fp32 kernel ignores it
// (its callers write the zeros).
struct GemmBatch {
  int count = 1;
  size_t sx = 0, sw = 0, so = 0;
  int wdiv = 1;
  int tri = 0;
};
// Row-tile height of the bf16 row-tile kernel (batched products always run on
// it): with tri 2 or 3 a row tile reads X only inside this band around the
// diagonal.
constexpr int kTiledRows = 128;

// EPI_LSE: for product row r (logits z = X W^T of the row, scaled x = c z with
// c = log2(e) / temperature) and each 64-column slot s (columns 64 s .. 64 s + 63
// below N), the pair (max_n x_n, sum_n 2^(x_n - max)) at out_f32[(r ld_out + s) 2]
// (ld_out = lse_slots(N)); the row's target logit z_t at tgt_z[r], the target
// being tokens[(g / Ts) T + score_from + g % Ts] for g = i0 + r, clamped to
// [0, N) (the token that follows the row's position).
struct LseArgs {
  const int32_t* tokens = nullptr;
  int T = 0, Ts = 1, score_from = 0, i0 = 0;
  float c = 0.f;
  float* tgt_z = nullptr;
};
inline int lse_slots(int N) { return (N + 63) / 64; }

// EPI_SAMPLE: for batch row b and output tile s (weight rows = vocabulary ids
// 16 rb s .. 16 rb s + 16 rb - 1 below N) of logits x, at part[(b tiles + s) 8]:
//   0 m = max x,  1 sum exp(x / T - m / T),  2-3 arg-max of x (value, id bits),
//   4-6 Gumbel-max over the tile (key, id bits, its x), the key of id v being
//   gumbel_key(x_v, T, word v % 4 of Philox block (v / 4, step, pid, 0), key seed)
// with step = step + *step_ctr (if set) and pid = seq_ids[b] (NULL: b); greedy
// (temperature <= 0) skips the keys and reads T as 1.  out_f32, if set, also
// receives the logits [B][ld_out] (a trace).
struct DecSample {
  float temperature = 0.f;
  uint64_t seed = 0;
  int step = 0;
  const int32_t* step_ctr = nullptr;
  const int32_t* seq_ids = nullptr;
  float* part = nullptr;
};

struct EpiArgs {
  float* out_f32;       // EPI_STORE: [rows, ld_out] fp32;  EPI_RESID: residual [rows, ld_out]
                        // EPI_LSE: [rows, ld_out slots] (max, sum) pairs
  void* out_act;        // EPI_SWIGLU: [rows, ld_out] activation dtype
  int ld_out;
  const char* name = nullptr;  // kernel-timing label of a decode GEMM (a string literal)
  LseArgs lse = {};
  DecSample smp = {};
};

// ---- decode GEMM: Y[B, N] = X[B, K] . W[N, K]^T for B <= 128 (bf16 MFMA) ----
// Operands in fragment order: X [K/32][nb/16][64][8] (act_frag_index, nb =
// decode_nb(B)), W [K/32][N/16][64][8] (pack_frag).  epi is EPI_PARTIAL
// (out_f32 [splits][B][ld_out] row-major) or EPI_SWIGLU (W = pack_frag of
// (gate, up) interleaved, N = 2 d_ffn, out_act = silu(gate) * up
// in fragment order [nb][ld_out = d_ffn], never split).  N % 16 == 0, K % 128 == 0.
int decode_nb(int B);                                           // 16, 32, 64 or 128
struct DecodePlan {
  int nb;        // padded batch
  int rb;        // 16-row blocks per output tile (2 for nb = 128; else 4, 6, 7 or 8)
  int tiles;     // output tiles of 16 * rb weight rows
  int splits;    // split-K factor (partial products written)
};
DecodePlan decode_plan(int B, int N, int K, int epi, int target_wgs, int max_splits = kMaxSplits);
hipError_t gemm_decode_bf16(const uint16_t* Xf, int B, const uint16_t* Wf, int N, int K, int epi,
                            EpiArgs ep, const DecodePlan& p, hipStream_t st);
// Fragment-order copy [K/32][N/16][64][8] of N row-major bf16 rows of length K:
// row n from w[0] (n < n1), w[1] (n1 <= n < n2) or w[2]; with interleave, 16-row
// block i holds rows 8 i .. 8 i + 7 of w[0] and then the same rows of w[1].
struct PackSrc {
  const void* w[3];
  int n1, n2;
  int interleave;
};
hipError_t pack_frag(const PackSrc& s, int N, int K, uint16_t* dst, hipStream_t st);

// ---- tiled GEMM for many rows (prefill / scoring): bf16 MFMA -----------------
hipError_t gemm_tiled_bf16(const uint16_t* X, int ldx, int M, WStack W, int N, int K, int epi,
                           EpiArgs ep, hipStream_t st, GemmBatch bt = GemmBatch{});

// ---- fp32 GEMM (fp32 models; VALU) -------------------------------------------
hipError_t gemm_f32(const float* X, int ldx, int M, WStack W, int N, int K, int epi, EpiArgs ep,
                    hipStream_t st, GemmBatch bt = GemmBatch{});

// ---- elementwise ---------------------------------------------------------------
// x[m, :] = emb[tok[m]] (fp32).  tok ids clamped to [0, vocab).
// ctr (optional): thread 0 adds 1 to *ctr (the decode step counter of a replayed graph).
hipError_t embed(int dtype, const void* emb, const int32_t* tok, int M, int d, int vocab, float* x,
                 hipStream_t st, int32_t* ctr = nullptr);
// Source row of output row m: ((i0 + m) / per) * stride + off + (i0 + m) % per.
struct RowMap {
  int i0, per, stride, off;
  static RowMap identity() { return RowMap{0, 0x7fffffff, 0, 0}; }
};
// Pending split-K partial products of a residual GEMM: part[s*split_stride + row*ld + i].
struct Partials {
  const float* part;
  int splits;            // 0: nothing pending
  size_t split_stride;   // floats between splits
  int ld;
};
// With p.splits > 0, first x[src(m)] += sum_s part (split order, written back).
// Then, if g != NULL, out[m] = round(x[src(m)] / sqrt(mean(x^2) + eps) * g), row-major
// with row stride ldo, or (pack_nb > 0, bf16) in decode-GEMM fragment order [pack_nb][d].
hipError_t rmsnorm(int dtype, float* x, int ldx, RowMap rows, Partials p, const void* g, int M,
                   int d, float eps, void* out, int ldo, hipStream_t st, int pack_nb = 0);
hipError_t fill_i32(int32_t* p, size_t n, int32_t v, hipStream_t st);
// dst[i] = vals[i] for i < n (host values passed as launch arguments, 128 per launch)
hipError_t set_i32(int32_t* dst, const int32_t* host_vals, int n, hipStream_t st);

// Destination row of a traced row m (and copy r < dup of it):
// (m / per) * stride + off + m % per + r * dup_stride.
struct TraceMap {
  int per, stride, off, dup, dup_stride;
  static TraceMap rows(int off = 0) { return TraceMap{0x7fffffff, 0, off, 1, 0}; }
};
// Trace copy: dst[map(m) * width + i] = element (m, i) of src as fp32, for
// m < M, i < width.  src layout: TR_F32 fp32 row-major (row stride ld),
// TR_BF16 bf16 row-major (ld), TR_FRAG bf16 in decode-GEMM fragment order
// [width/32][ld/16][64][8] (ld = the padded batch).
enum TraceSrc { TR_F32 = 0, TR_BF16 = 1, TR_FRAG = 2 };
hipError_t trace_rows(const void* src, int layout, int ld, int M, int width, TraceMap map,
                      float* dst, hipStream_t st);
// cos / sin table of the rotary angles, [rows][hd / 2] float2: row r is position
// pos_arr[r] (device array) or, with pos_arr NULL, position r.
hipError_t rope_table(const int32_t* pos_arr, int rows, int hd, float theta, float2* cs,
                      hipStream_t st);
// V^T [b][n_kv][hd][vt_len] of cached sequences (slot slots[b]) for positions
// 0 .. pos0[b] + T - 1, zero beyond (device arrays slots, pos0 of B entries).
hipError_t cache_vt(const void* vc, const int32_t* slots, const int32_t* pos0, int B, int T,
                    int n_kv, int max_len, int hd, int vt_len, uint16_t* vt, hipStream_t st);
// row_pos[m] = pos0[m / T] + m % T, row_slot[m] = slots[m / T] for m < B * T.
hipError_t row_positions(const int32_t* pos0, const int32_t* slots, int B, int T,
                         int32_t* row_pos, int32_t* row_slot, hipStream_t st);
// Rotary embedding + cache write.  qkv fp32 [M, q_dim + 2 kv_dim], or the sum
// of `splits` such arrays split_stride floats apart (decode GEMM partials).  Row m is
// (seq, pos): mode 0: seq = m, pos = pos_arr[m];  mode 1: seq = m / T, pos =
// (pos_arr ? pos_arr[seq] : pos0) + m % T.  slots (optional): cache slot of seq.
// cs: rope_table rows of pos_arr (mode 0) or of positions 0..T-1 (mode 1).
// q_out: [M, q_dim] act.  K/V written to cache slots seq*G + g (g < G) at pos
// (positions >= max_len skipped).  vt (optional, mode 1, M a multiple of T) gets
// V transposed: [seq][n_kv][hd][vt_len] for the prefill/scoring attention,
// positions T..vt_len-1 zero.
struct RopeArgs {
  int mode, T, G;
  const int32_t* pos_arr;
  const int32_t* slots;         // cache slot of sequence seq (NULL: seq * G + g)
  int n_heads, n_kv, hd;
  float theta;
  void* kcache; void* vcache;   // layer base of K and V: [n_seqs][n_kv][max_len][hd]; V may be NULL
  int n_seqs, max_len;
  uint16_t* vt; int vt_len;
  int splits; size_t split_stride;
  const float2* cs;
  int pos0;    // mode 1: position of each sequence's first row (0: rows start at 0)
  int vt_G;    // V^T written to vt_G consecutive sequence slots per sequence (0 or 1: one)
  // trace (each optional): q [.][q_dim], k and v [.][kv_dim] fp32 rows at tmap(m)
  float* tq; float* tk; float* tv;
  TraceMap tmap;
};
hipError_t rope_kv(int dtype, const float* qkv, int M, void* q_out, const RopeArgs& a,
                   hipStream_t st);

// ---- attention -------------------------------------------------------------------
// Decode: q act [B, H, hd]; cache layer base K/V [n_seqs][n_kv][max_len][hd];
// row b reads cache slot slots[b] (NULL: b) and attends positions 0..pos[b].  out act [B, H*hd] row-major, or (pack_nb > 0) in
// decode-GEMM fragment order [pack_nb][H*hd].
// tc: context positions per span (a multiple of 128); splits: spans per (sequence,
// kv head); part_floats: fp32 scratch for the span merge (0 with a single span).
// tc positions per span, splits spans per row; grouped steps (G > 0) add
// `chunks` prompt chunks of span_p positions below prefix_len per group of G
// rows, n_sub prefix workgroups per group and chunk.  part_floats: the partial
// buffer the plan needs.
struct DecodeAttnPlan {
  int tc, splits;
  int waves;     // waves per workgroup of the per-row kernel (4, or 2 for large grids)
  int G, prefix_len, chunks, span_p, n_sub;
  int ncb;       // query column blocks of 16 per prefix workgroup (2 or 3)
  size_t part_floats;
};
DecodeAttnPlan decode_attn_plan(int B, int H, int n_kv, int hd, int max_len, int G = 0,
                                int prefix_len = 0);
// partial floats of any plan for these shapes, grouped or not
size_t decode_attn_part_floats_max(int B, int H, int n_kv, int hd, int max_len);
hipError_t attn_decode(int dtype, const void* q, const void* kc, const void* vc,
                       const int32_t* pos, const int32_t* slots, int B, int H, int n_kv, int hd, int n_seqs, int max_len,
                       const DecodeAttnPlan& p, float* part, void* out, hipStream_t st,
                       int pack_nb = 0);
// fp32 attention rows (decode rows when pos != NULL: row m is sequence m at
// position pos[m]; else row m is position m % T of sequence m / T at cache slot
// (m / T) * slot_mul); k_len positions of cache per sequence and kv head.
hipError_t attn_rows_f32(const float* q, const float* kc, const float* vc, const int32_t* pos,
                         const int32_t* slots, int rows, int T, int slot_mul, int H, int n_kv, int hd, int k_len,
                         float* out, hipStream_t st);
// Causal attention over N sequences of T rows: q act [N*T, H*hd]; K in cache
// layout [n][n_kv][k_len][hd] (sequence n at slot n*k_stride_seq), Vt
// [n][n_kv][hd][T] (bf16 path) or V in cache layout (fp32 path).  out act [N*T, H*hd].
// bf16 only: q_pos0 is the position of each sequence's first
// query row (keys 0 .. q_pos0 + T - 1 are attended), V^T of sequence n at slot
// n * vt_seq_stride with rows of vt_len positions (0: (q_pos0 + T) rounded up to 8).
// qpos (optional, bf16): per-sequence first query position (replaces q_pos0);
// kslots (optional, bf16): cache slot of sequence n's K (replaces n * k_seq_stride).
hipError_t attn_prefill(int dtype, const void* q, const void* k, const void* v_or_vt, int N,
                        int T, int H, int n_kv, int hd, int k_len, int k_seq_stride,
                        void* out, hipStream_t st, int q_pos0 = 0, int vt_seq_stride = 1,
                        int vt_len = 0, const int32_t* qpos = nullptr,
                        const int32_t* kslots = nullptr);

// ---- sampling / log-probs ---------------------------------------------------------
// logits fp32 [R, V] (row stride ld).  Row r makes G draws; draw g writes
// tok_out[q*out_stride], logp_out[q*out_stride] for q = r*G + g and uses Philox
// sequence id seq_ids[q] (NULL: q).
struct SampleArgs {
  float temperature; int top_k; uint64_t seed;
  int step;               // Philox step word
  int G;                  // draws per row (prefill: G samples per prompt)
  int32_t* tok_out; float* logp_out;  // [R*G], element stride out_stride
  int out_stride;
  int32_t* tok_state;     // optional [R*G]: also store token here
  int32_t* pos_state;     // optional [R*G]: pos += 1
  const int32_t* step_ctr;  // optional: Philox step = step + *step_ctr, outputs at column *step_ctr
  const int32_t* seq_ids;   // optional [R*G]: Philox sequence id of draw q
};
hipError_t sample(const float* logits, int R, int V, int ld, const SampleArgs& a, hipStream_t st);
// The same draw (no top-k cut, one draw per row) from the EPI_SAMPLE pieces of
// R rows over `tiles` output tiles: the token of the best Gumbel key (greedy:
// the arg-max), logp = x_tok / T - (M / T + log S) with M the largest tile
// maximum and S = sum over tiles s of sum_s exp(m_s / T - M / T); the same outputs and state
// updates as `sample`.
hipError_t sample_combine(const float* part, int tiles, int R, int V, const SampleArgs& a,
                          hipStream_t st);
// Teacher-forced log-prob of scored row r, log_softmax(z / temperature) at the
// row's target, from the LM head's EPI_LSE pieces:
// logp[r] = z_t[r] / temperature - ln2 (M + log2 S) with M = max_s m_s and
// S = sum_s s_s 2^(m_s - M) over the row's `slots` (max, sum) pairs.
hipError_t lse_combine(const float* part, int slots, const float* tgt_z, int R,
                       float temperature, float* logp, hipStream_t st);

// ---- GRPO ---------------------------------------------------------------------------
hipError_t advantages(const float* r, int P, int G, float eps, float* adv, hipStream_t st);
// Distillation loss -mean(logp) over the masked tokens (agg as token_loss) and its
// gradient; row_ws: 3 N doubles.
hipError_t sft_loss(const float* lp, const uint8_t* mask, int N, int Tr, int agg, float* loss,
                    float* dl, double* row_ws, hipStream_t st);
// kl[r] = KL(softmax(z[r] / T) || softmax(zr[r] / T)) over V entries, fp64 inside.
hipError_t exact_kl(const float* z, const float* zr, int R, int V, int ld, float temperature,
                    float* kl, hipStream_t st);
// Device address, on the current device, of the loss's static scratch
// (kLossStaticRows sequences x 9 doubles); looked up once per device.
constexpr int kLossStaticRows = 16384;
hipError_t loss_static_scratch(double** out);
hipError_t token_loss(const float* lp, const float* lo, const float* lr, const uint8_t* mask,
                      const float* adv, int N, int Tr, float clip_eps, float beta, int agg,
                      float* loss, float* tok_loss, float* dl, float* stats, double* row_ws,
                      hipStream_t st);

// ---- backward pass and optimizer (backward.hip) ---------------------------------
// dtype / tin / tout: 0 fp32, 1 bf16.  Transpose: out[c][r] = in[r][c] for r < R,
// c < C, out columns R .. Rpad-1 zero; batch element b reads in + b in_bs and
// writes out + (b / div) s1 + (b % div) s2.
hipError_t transpose(int tin, int tout, const void* in, int ldi, size_t in_bs, int R, int C,
                     void* out, int ldo, size_t s1, size_t s2, int div, int Rpad, int batch,
                     hipStream_t st);
hipError_t dlogits(int dtype, const float* z, int R, int V, int ldz, const int32_t* tgt,
                   int tstride, const float* g, float temperature, void* dz, int ldo,
                   hipStream_t st);
hipError_t rmsnorm_bwd(int dtype, const float* x, int ldx, const void* g, const float* dy, int ldy,
                       int T, int d, float eps, float* dres, void* dres_e, float* rr, float* part,
                       float* dg, hipStream_t st);
hipError_t swiglu_fwd(int dtype, const float* gu, int T, int F, void* a, hipStream_t st);
hipError_t swiglu_bwd(int dtype, const float* gu, const float* da, int T, int F, void* dgu,
                      hipStream_t st);
hipError_t rope_bwd(int dtype, float* dqkv, int T, int heads, int n_rot, int hd, const float2* cs,
                    void* out, hipStream_t st);
// fp32 models (dtype 0 only): softmax backward from the stored S and dP products
hipError_t attn_softmax_bwd(int dtype, const float* S, const float* dP, int T, int Tp, int batch,
                            float scale, float* stats, void* dS, void* dST, void* PT,
                            hipStream_t st);
// bf16 models: the same outputs as the score products and attn_softmax_bwd
// together, from q, dO ([T][ldq], head b at column b hd) and the batch's K and V
// ([batch / gq][Tp][hd], head b reading group b / gq), the scores formed on the
// matrix cores twice and never stored; above the diagonal only the band tiles
// the causal products read (kTiledRows) are written.
hipError_t attn_scores_bwd(const void* q, const void* dO, int ldq, const void* kb, const void* vb,
                          int gq, int T, int Tp, int batch, int hd, float scale, void* dS,
                          void* dST, void* PT, hipStream_t st);
hipError_t sum_heads(const float* tmp, int T, int hd, int gq, int groups, float* out, int ldo,
                     hipStream_t st);
// demb[tok[t]] += dx[t] for t < T <= 16384 (V <= 2^18), without atomics: the
// (token, t) keys are sorted into `keys` [T] and each token's rows summed in
// increasing t, then added to its embedding row.
hipError_t embed_bwd(const int32_t* tok, const float* dx, int T, int d, int V, uint32_t* keys,
                     float* demb, hipStream_t st);
hipError_t fill_f32(float* p, size_t n, float v, hipStream_t st);
hipError_t cast_f32(const float* in, size_t n, int dtype, void* out, hipStream_t st);
hipError_t adamw(int dtype, void* param, float* master, float* m, float* v, const float* grad,
                 size_t n, float lr, float b1, float b2, float eps, float wd, int step,
                 hipStream_t st);

}  // namespace grpo
