// libgrpo_hip: the C-ABI of include/grpo_hip.h.
//
// Host side only: argument validation (before anything is enqueued), workspace
// layout, and the order in which the kernels of kernels.h run for prefill,
// decode steps, scoring and the GRPO loss.  No device memory is allocated here.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "grpo_hip.h"
#include "kernels.h"

using namespace grpo;

// A decode step captured as a HIP graph, replayed n_steps times; recaptured
// when any argument of the call changes.
struct DecodeGraph {
  hipGraphExec_t exec = nullptr;
  hipStream_t capture = nullptr;
  std::vector<uint64_t> key;
};

// Fragment-order copies of the projections for the decode GEMM (bf16 models),
// in a caller-owned buffer written by grpo_model_pack_decode.
struct DecodeWeights {
  const void* base = nullptr;
  std::vector<const uint16_t*> qkv, o, gate_up, down;
  const uint16_t* lm_head = nullptr;
};

struct grpo_model {
  grpo_config cfg;
  const void* tok_emb;
  std::vector<const void*> attn_norm, wq, wk, wv, wo, mlp_norm, w_gate, w_up, w_down;
  const void* final_norm;
  const void* lm_head;
  DecodeWeights dec;
  DecodeGraph graph;
};

// ---- kernel timing (grpo_profile_begin / grpo_profile_end) ----
namespace {
struct ProfRec {
  const char* name;
  hipEvent_t e0, e1;
};
std::atomic<bool> g_prof{false};
std::mutex g_prof_mu;
std::deque<ProfRec> g_prof_pending;
std::vector<hipEvent_t> g_prof_free;
std::map<std::string, std::pair<long, double>> g_prof_acc;

hipEvent_t prof_event() {
  if (!g_prof_free.empty()) {
    hipEvent_t e = g_prof_free.back();
    g_prof_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// accumulate finished records until at most `keep` are pending (lock held)
void prof_drain(size_t keep) {
  while (g_prof_pending.size() > keep) {
    ProfRec r = g_prof_pending.front();
    g_prof_pending.pop_front();
    float ms = 0.f;
    if (hipEventSynchronize(r.e1) == hipSuccess && hipEventElapsedTime(&ms, r.e0, r.e1) == hipSuccess) {
      auto& a = g_prof_acc[r.name];
      a.first += 1;
      a.second += ms;
    }
    g_prof_free.push_back(r.e0);
    g_prof_free.push_back(r.e1);
  }
}
}  // namespace

namespace grpo {
bool profiling() { return g_prof.load(std::memory_order_relaxed); }

Prof::Prof(const char* n, hipStream_t s) : name(n), st(s), ev0(nullptr) {
  if (!profiling()) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  hipEvent_t e = prof_event();
  if (e && hipEventRecord(e, s) == hipSuccess) ev0 = e;
}

Prof::~Prof() {
  if (!ev0) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  hipEvent_t e1 = prof_event();
  if (!e1 || hipEventRecord(e1, st) != hipSuccess) return;
  g_prof_pending.push_back(ProfRec{name, (hipEvent_t)ev0, e1});
  if (g_prof_pending.size() > 8192) prof_drain(4096);
}
}  // namespace grpo

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIPCHK(expr)                                                                  \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess) return fail(GRPO_HIP_ERROR, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

// True while rocprofv3 collects hardware counters in this process (it exports
// ROCPROF_COUNTER_COLLECTION).  Counter collection rewrites every kernel dispatch
// on the intercepted queue; two combinations aborted under it (graph replay:
// "invalid AQL packet"; HIP-event bracketing of every launch: the process died
// on the host), so during such runs decode steps launch eagerly and kernel
// timing is refused.  Results are identical either way.
bool counter_collection() {
  static const bool on = getenv("ROCPROF_COUNTER_COLLECTION") != nullptr;
  return on;
}

// split-K target grid of the decode GEMM (GRPO_DECODE_WGS overrides, for tuning)
int decode_target() {
  static const int v = [] {
    const char* e = getenv("GRPO_DECODE_WGS");
    const int x = e ? atoi(e) : 0;
    return x > 0 ? x : 256;
  }();
  return v;
}
constexpr int kScoreTokens = 262144;   // rows per scoring chunk (sequences * T)
constexpr int kBackwardTokens = 16384; // longest sequence of the backward pass
constexpr size_t kHeadBytes = size_t(1) << 30;   // LM-head working set per scoring sub-chunk

// bump allocator over the caller's workspace; base == nullptr only measures
struct Bump {
  char* base;
  size_t off = 0;
  explicit Bump(void* b) : base((char*)b) {}
  template <class T>
  T* take(size_t n) {
    if (n == 0) return nullptr;
    off = (off + 255) & ~size_t(255);
    T* p = base ? (T*)(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
};

int esize(const grpo_config& c) { return c.dtype == GRPO_F32 ? 4 : 2; }
int qdim(const grpo_config& c) { return c.n_heads * c.head_dim; }
int kvdim(const grpo_config& c) { return c.n_kv_heads * c.head_dim; }

int check_config(const grpo_config* c) {
  if (!c) return fail(GRPO_INVALID_ARG, "config is NULL");
  if (c->n_layers < 1 || c->d_model < 1 || c->n_heads < 1 || c->n_kv_heads < 1 ||
      c->head_dim < 1 || c->d_ffn < 1 || c->vocab < 1)
    return fail(GRPO_INVALID_ARG, "config sizes must be positive");
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f))
    return fail(GRPO_INVALID_ARG, "rms_eps must be >= 0 and rope_theta > 0");
  if (c->dtype != GRPO_F32 && c->dtype != GRPO_BF16)
    return fail(GRPO_UNSUPPORTED, "dtype %d is neither GRPO_F32 nor GRPO_BF16", c->dtype);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(GRPO_UNSUPPORTED, "head_dim %d not in {64, 128}", c->head_dim);
  if (c->n_heads % c->n_kv_heads)
    return fail(GRPO_UNSUPPORTED, "n_heads %d not a multiple of n_kv_heads %d", c->n_heads,
                c->n_kv_heads);
  if (c->n_heads / c->n_kv_heads > 8)
    return fail(GRPO_UNSUPPORTED, "more than 8 query heads per kv head");
  if (c->d_model > 8192) return fail(GRPO_UNSUPPORTED, "d_model above 8192");
  if (c->dtype == GRPO_BF16 && c->vocab % 16)
    return fail(GRPO_UNSUPPORTED, "vocab %d of a bf16 model not a multiple of 16", c->vocab);
  const int mult = c->dtype == GRPO_F32 ? 32 : 128;
  if (c->d_model % mult || qdim(*c) % mult || c->d_ffn % mult)
    return fail(GRPO_UNSUPPORTED, "d_model, n_heads*head_dim and d_ffn must be multiples of %d",
                mult);
  return GRPO_OK;
}

struct Layer {
  void* k;
  void* v;
};
Layer kv_layer(const grpo_model* m, void* kv, int l, int n_seqs, int max_len) {
  const grpo_config& c = m->cfg;
  const size_t per = (size_t)n_seqs * c.n_kv_heads * max_len * c.head_dim * esize(c);
  char* base = (char*)kv + (size_t)l * 2 * per;
  return Layer{base, base + per};
}

// ---- GEMMs ----
// Many-row products (prefill, scoring) and every product of fp32 models read the
// row-major weights: fp32 on the vector units, bf16 on the tiled MFMA kernels.
// The decode steps of bf16 models run the decode GEMM on fragment-order operands
// and leave split-K partial products for the consuming kernel (RMSNorm adds
// residual partials, RoPE adds QKV partials).
struct GemmScratch {
  float* part;   // decode-GEMM partial products
};

int gemm_fail(hipError_t e) {
  return fail(GRPO_HIP_ERROR, "GEMM launch failed: %s", hipGetErrorString(e));
}

// out = X W^T (EPI_STORE), x += X W^T (EPI_RESID) or out_act = silu(gate) * up
// (EPI_SWIGLU, W = (gate, up) stack), row-major everything
int gemm_rows(const grpo_model* m, const void* X, int ldx, int M, WStack W, int N, int K, int epi,
              EpiArgs ep, hipStream_t st) {
  const hipError_t e =
      m->cfg.dtype == GRPO_F32
          ? gemm_f32((const float*)X, ldx, M, W, N, K, epi, ep, st)
          : gemm_tiled_bf16((const uint16_t*)X, ldx, M, W, N, K, epi, ep, st);
  return e == hipSuccess ? GRPO_OK : gemm_fail(e);
}

// Decode GEMM over fragment-order X [nb][K] and W: the product as *splits partial
// arrays *stride floats apart, the first at `out` when there is one split, else
// in the scratch.
int gemm_dec(const void* Xf, int B, const uint16_t* Wf, int N, int K, float* out, GemmScratch s,
             int max_splits, const float** res, int* splits, size_t* stride, hipStream_t st,
             const char* name) {
  const DecodePlan p = decode_plan(B, N, K, EPI_PARTIAL, decode_target(), max_splits);
  float* dst = p.splits == 1 ? out : s.part;
  const hipError_t e = gemm_decode_bf16((const uint16_t*)Xf, B, Wf, N, K, EPI_PARTIAL,
                                        EpiArgs{dst, nullptr, N, name}, p, st);
  *res = dst;
  *splits = p.splits;
  *stride = (size_t)B * N;
  return e == hipSuccess ? GRPO_OK : gemm_fail(e);
}

// The decode LM head with the sampling epilogue: per-tile pieces of the draw
// `sa` describes into part ([B][*tiles][8]); the logits into `logits` too if set.
int gemm_dec_sample(const void* Xf, int B, const uint16_t* Wf, int N, int K, const SampleArgs& sa,
                    float* part, float* logits, int* tiles, hipStream_t st) {
  const DecodePlan p = decode_plan(B, N, K, EPI_PARTIAL, decode_target(), 1);
  EpiArgs ep{logits, nullptr, N, "gemm_decode_lm_head"};
  ep.smp.temperature = sa.temperature;
  ep.smp.seed = sa.seed;
  ep.smp.step = sa.step;
  ep.smp.step_ctr = sa.step_ctr;
  ep.smp.seq_ids = sa.seq_ids;
  ep.smp.part = part;
  *tiles = p.tiles;
  const hipError_t e = gemm_decode_bf16((const uint16_t*)Xf, B, Wf, N, K, EPI_SAMPLE, ep, p, st);
  return e == hipSuccess ? GRPO_OK : gemm_fail(e);
}

// residual projection: the product is left in *pend for the next RMSNorm to add
int gemm_dec_resid(const void* Xf, int B, const uint16_t* Wf, int N, int K, GemmScratch s,
                   Partials* pend, hipStream_t st, const char* name) {
  const float* res;
  int splits;
  size_t stride;
  if (int rc = gemm_dec(Xf, B, Wf, N, K, s.part, s, kMaxSplits, &res, &splits, &stride, st, name))
    return rc;
  *pend = Partials{res, splits, stride, N};
  return GRPO_OK;
}

// a[nb][f] (fragment order) = silu(X Wg^T) * (X Wu^T)
int gemm_dec_swiglu(const void* Xf, int B, const uint16_t* Wf, int f, int K, void* a,
                    hipStream_t st) {
  const DecodePlan p = decode_plan(B, 2 * f, K, EPI_SWIGLU, decode_target());
  const hipError_t e = gemm_decode_bf16((const uint16_t*)Xf, B, Wf, 2 * f, K, EPI_SWIGLU,
                                        EpiArgs{nullptr, a, f, "gemm_decode_swiglu"}, p, st);
  return e == hipSuccess ? GRPO_OK : gemm_fail(e);
}

// partial-product scratch of the decode GEMM for B rows, over the split shapes
// of the model (QKV, O and down projections)
size_t decode_scratch(const grpo_config& c, int B) {
  if (c.dtype == GRPO_F32) return 0;
  const int d = c.d_model, f = c.d_ffn;
  const int shapes[3][2] = {{qdim(c) + 2 * kvdim(c), d}, {d, qdim(c)}, {d, f}};
  size_t part = 0;
  for (auto& sh : shapes) {
    const DecodePlan p = decode_plan(B, sh[0], sh[1], EPI_PARTIAL, decode_target());
    part = std::max(part, (size_t)p.splits * B * sh[0]);
  }
  return part;
}

// Byte offsets of the decode copy: per layer QKV (rows q, k, v), O, gate/up
// (8 gate rows then the same 8 up rows per 16-row block), down; then the LM head.
struct DecodeLayout {
  std::vector<size_t> qkv, o, gate_up, down;
  size_t lm_head = 0, total = 0;
};
DecodeLayout decode_layout(const grpo_config& c) {
  DecodeLayout L;
  const size_t d = c.d_model, qd = qdim(c), kvd = kvdim(c), f = c.d_ffn;
  size_t off = 0;
  auto take = [&](size_t rows, size_t cols) {
    const size_t at = off;
    off += (rows * cols * 2 + 255) & ~size_t(255);
    return at;
  };
  for (int l = 0; l < c.n_layers; ++l) {
    L.qkv.push_back(take(qd + 2 * kvd, d));
    L.o.push_back(take(d, qd));
    L.gate_up.push_back(take(2 * f, d));
    L.down.push_back(take(d, f));
  }
  L.lm_head = take(c.vocab, d);
  L.total = off;
  return L;
}

// ---- workspace layouts ----
struct StepWS {   // activations of `rows` token rows
  float* x; void* h; float* qkv; void* q; void* o; void* a;
  float2* cs;      // rotary cos / sin table
  GemmScratch g;
};

// act_rows: rows of the GEMM inputs h, o and a (the padded batch of a decode step);
// cs_rows: rows of the rotary table (decode: one per sequence; else one per position)
StepWS take_step(Bump& b, const grpo_config& c, int rows, int act_rows, size_t part_floats,
                 int cs_rows) {
  StepWS w;
  const int es = esize(c);
  w.x = b.take<float>((size_t)rows * c.d_model);
  w.h = b.take<char>((size_t)act_rows * c.d_model * es);
  w.qkv = b.take<float>((size_t)rows * (qdim(c) + 2 * kvdim(c)));
  w.q = b.take<char>((size_t)rows * qdim(c) * es);
  w.o = b.take<char>((size_t)act_rows * qdim(c) * es);
  w.a = b.take<char>((size_t)act_rows * c.d_ffn * es);
  w.cs = b.take<float2>((size_t)cs_rows * (c.head_dim / 2));
  w.g.part = b.take<float>(part_floats);
  return w;
}

struct RolloutWS {
  StepWS s;
  float* logits;       // the LM head's logits (sampling with a top-k cut, fp32 models)
  float* spart;        // the sampling epilogue's per-tile pieces [B][tiles][8] (bf16)
  float* attn_part;
  int32_t* step_ctr;   // decode steps done by the replayed graph
  int32_t* slots;      // [B] cache slot / Philox sequence id of each row (seq_ids)
};
RolloutWS take_rollout(Bump& b, const grpo_config& c, int B, int max_len) {
  RolloutWS w;
  w.s = take_step(b, c, B, c.dtype == GRPO_F32 ? B : decode_nb(B), decode_scratch(c, B), B);
  w.logits = b.take<float>((size_t)B * c.vocab);
  // tiles of at least 32 vocabulary rows (16 rb, rb >= 2)
  w.spart = b.take<float>(c.dtype == GRPO_F32 ? 0 : (size_t)B * ((c.vocab + 31) / 32) * 8);
  w.attn_part = b.take<float>(
      c.dtype == GRPO_F32 ? 0
                          : decode_attn_part_floats_max(B, c.n_heads, c.n_kv_heads, c.head_dim,
                                                        max_len));
  w.step_ctr = b.take<int32_t>(1);
  w.slots = b.take<int32_t>(B);
  return w;
}

struct PrefillWS {
  StepWS s;
  uint16_t* vt;
  void* hl;
  float* logits;
};
int round8(int t) { return (t + 7) / 8 * 8; }
PrefillWS take_prefill(Bump& b, const grpo_config& c, int P, int Tp) {
  PrefillWS w;
  const size_t M = (size_t)P * Tp;
  w.s = take_step(b, c, (int)M, (int)M, 0, Tp);
  w.vt = b.take<uint16_t>(c.dtype == GRPO_F32 ? 0 : (size_t)P * kvdim(c) * round8(Tp));
  w.hl = b.take<char>((size_t)P * c.d_model * esize(c));
  w.logits = b.take<float>((size_t)P * c.vocab);
  return w;
}

constexpr int kExtendChunk = GRPO_EXTEND_CHUNK;   // span rows per sequence and call

struct ExtendWS {
  StepWS s;
  uint16_t* vt;         // V^T of every sequence up to max_len (bf16)
  void* hl;
  float* logits;
  int32_t *slots, *pos0, *row_pos, *row_slot;
};
ExtendWS take_extend(Bump& b, const grpo_config& c, int B, int max_len) {
  ExtendWS w;
  const size_t M = (size_t)B * kExtendChunk;
  w.s = take_step(b, c, (int)M, (int)M, 0, max_len);
  w.vt = b.take<uint16_t>(c.dtype == GRPO_F32 ? 0 : (size_t)B * kvdim(c) * round8(max_len));
  w.hl = b.take<char>((size_t)B * c.d_model * esize(c));
  w.logits = b.take<float>((size_t)B * c.vocab);
  w.slots = b.take<int32_t>(B);
  w.pos0 = b.take<int32_t>(B);
  w.row_pos = b.take<int32_t>(M);
  w.row_slot = b.take<int32_t>(M);
  return w;
}

struct ScoreWS {
  int chunk;         // sequences per chunk
  int sub_rows;      // LM-head rows per sub-chunk, at most
  StepWS s;
  void* kbuf; void* vbuf; uint16_t* vt;
  void* hs;          // the sub-chunk's normed final hidden rows
  float* lse;        // its LM-head log-sum-exp pieces: [rows][lse_slots(V)] (max, sum)
  float* tgt_z;      // its target logits
};
ScoreWS take_score(Bump& b, const grpo_config& c, int N, int T) {
  ScoreWS w;
  w.chunk = std::max(1, std::min(N, kScoreTokens / std::max(T, 1)));
  const size_t M = (size_t)w.chunk * T;
  const size_t per_row = (size_t)c.d_model * esize(c) + (size_t)lse_slots(c.vocab) * 8 + 4;
  w.sub_rows = (int)std::min<size_t>(M, std::max<size_t>(256, kHeadBytes / per_row / 256 * 256));
  w.s = take_step(b, c, (int)M, (int)M, 0, T);
  const size_t kvn = (size_t)w.chunk * kvdim(c) * T;
  w.kbuf = b.take<char>(kvn * esize(c));
  w.vbuf = b.take<char>(c.dtype == GRPO_F32 ? kvn * 4 : 0);
  w.vt = b.take<uint16_t>(c.dtype == GRPO_F32 ? 0 : (size_t)w.chunk * kvdim(c) * round8(T));
  w.hs = b.take<char>((size_t)w.sub_rows * c.d_model * esize(c));
  w.lse = b.take<float>((size_t)w.sub_rows * lse_slots(c.vocab) * 2);
  w.tgt_z = b.take<float>((size_t)w.sub_rows);
  return w;
}
// Rows per LM-head sub-chunk for R scored rows: the fewest sub-chunks of at most
// sub_rows rows, of equal size in multiples of 256 (the last one shorter).
int head_step(const ScoreWS& w, int R) {
  const int n = (R + w.sub_rows - 1) / w.sub_rows;
  return std::min(w.sub_rows, ((R + n - 1) / n + 255) / 256 * 256);
}

WStack qkv_stack(const grpo_model* m, int l) {
  const grpo_config& c = m->cfg;
  return WStack{{m->wq[l], m->wk[l], m->wv[l]}, qdim(c), qdim(c) + kvdim(c)};
}
WStack one(const void* w) { return WStack{{w, w, w}, 0x7fffffff, 0x7fffffff}; }
WStack gate_up(const grpo_model* m, int l) {
  return WStack{{m->w_gate[l], m->w_up[l], m->w_up[l]}, m->cfg.d_ffn, 2 * m->cfg.d_ffn};
}

// Trace capture: rows of a forward buffer into layer l of a trace member
// ([layers][R][width] fp32); a NULL member is skipped.
int trace(float* member, int l, size_t R, int width, const void* src, int layout, int ld, int M,
          TraceMap map, hipStream_t st) {
  if (!member || M <= 0) return GRPO_OK;
  HIPCHK(trace_rows(src, layout, ld, M, width, map, member + (size_t)l * R * width, st));
  return GRPO_OK;
}
// trace member pointer or NULL
#define TRM(tr, f) ((tr) ? (tr)->f : nullptr)

// Layers of a many-row forward (prefill or scoring).  Rows are sequence-major
// (row = seq * T + t).  K/V go to kc/vc (cache layout with n_slots slots of
// k_len positions; sequence s at slot s * G) and V also transposed to vt.
// tr: trace of R rows, these rows at tmap.
int forward_rows(const grpo_model* m, StepWS& w, int M, int T, int G, int n_slots, int k_len,
                 void* kv_or_null, void* kbuf, void* vbuf, uint16_t* vt, const grpo_trace* tr,
                 size_t R, TraceMap tmap, hipStream_t st) {
  const grpo_config& c = m->cfg;
  const int d = c.d_model, qd = qdim(c), kvd = kvdim(c), f = c.d_ffn;
  const int N = M / T;
  const Partials none{nullptr, 0, 0, d};
  const int act = c.dtype == GRPO_F32 ? TR_F32 : TR_BF16;
  int rc;
  HIPCHK(rope_table(nullptr, T, c.head_dim, c.rope_theta, w.cs, st));
  for (int l = 0; l < c.n_layers; ++l) {
    void *kl = kbuf, *vl = vbuf;
    if (kv_or_null) {
      Layer L = kv_layer(m, kv_or_null, l, n_slots, k_len);
      kl = L.k;
      vl = L.v;
    }
    HIPCHK(rmsnorm(c.dtype, w.x, d, RowMap::identity(), none, m->attn_norm[l], M, d, c.rms_eps,
                   w.h, d, st));
    if ((rc = trace(TRM(tr, x), l, R, d, w.x, TR_F32, d, M, tmap, st)) ||
        (rc = trace(TRM(tr, h_attn), l, R, d, w.h, act, d, M, tmap, st)))
      return rc;
    if ((rc = gemm_rows(m, w.h, d, M, qkv_stack(m, l), qd + 2 * kvd, d, EPI_STORE,
                        EpiArgs{w.qkv, nullptr, qd + 2 * kvd}, st)))
      return rc;
    RopeArgs ra{};
    ra.mode = 1; ra.T = T; ra.G = G; ra.pos_arr = nullptr;
    ra.n_heads = c.n_heads; ra.n_kv = c.n_kv_heads; ra.hd = c.head_dim; ra.theta = c.rope_theta;
    ra.kcache = kl; ra.vcache = vl; ra.n_seqs = n_slots; ra.max_len = k_len;
    ra.vt = c.dtype == GRPO_F32 ? nullptr : vt; ra.vt_len = round8(T);
    ra.splits = 1; ra.split_stride = 0;
    ra.cs = w.cs;
    if (tr) {
      ra.tq = tr->q ? tr->q + (size_t)l * R * qd : nullptr;
      ra.tk = tr->k ? tr->k + (size_t)l * R * kvd : nullptr;
      ra.tv = tr->v ? tr->v + (size_t)l * R * kvd : nullptr;
      ra.tmap = tmap;
    }
    HIPCHK(rope_kv(c.dtype, w.qkv, M, w.q, ra, st));
    HIPCHK(attn_prefill(c.dtype, w.q, kl, c.dtype == GRPO_F32 ? vl : (const void*)vt, N, T,
                        c.n_heads, c.n_kv_heads, c.head_dim, k_len, G, w.o, st));
    if ((rc = trace(TRM(tr, o), l, R, qd, w.o, act, qd, M, tmap, st))) return rc;
    if ((rc = gemm_rows(m, w.o, qd, M, one(m->wo[l]), d, qd, EPI_RESID, EpiArgs{w.x, nullptr, d},
                        st)))
      return rc;
    HIPCHK(rmsnorm(c.dtype, w.x, d, RowMap::identity(), none, m->mlp_norm[l], M, d, c.rms_eps,
                   w.h, d, st));
    if ((rc = trace(TRM(tr, x_attn), l, R, d, w.x, TR_F32, d, M, tmap, st)) ||
        (rc = trace(TRM(tr, h_mlp), l, R, d, w.h, act, d, M, tmap, st)))
      return rc;
    if ((rc = gemm_rows(m, w.h, d, M, gate_up(m, l), f, d, EPI_SWIGLU, EpiArgs{nullptr, w.a, f},
                        st)))
      return rc;
    if ((rc = trace(TRM(tr, act), l, R, f, w.a, act, f, M, tmap, st))) return rc;
    if ((rc = gemm_rows(m, w.a, f, M, one(m->w_down[l]), d, f, EPI_RESID, EpiArgs{w.x, nullptr, d},
                        st)))
      return rc;
  }
  return trace(TRM(tr, x), c.n_layers, R, d, w.x, TR_F32, d, M, tmap, st);
}

// head rows [off, off + M) of a scoring trace: normed input and logits
// LM head of `rows` normed rows (w.hs) with the log-softmax at each row's
// target fused into the product (Alg. 1 scoring, log pi of the sampled token):
// the product's epilogue leaves per-row log-sum-exp pieces and the target
// logit, lse_combine turns them into logp; the [rows, V] logits are never
// stored.  Row r is scored row i0 + r of the chunk's tokens tk.  With a trace,
// the normed rows and (by a second product into the trace itself) the logits
// are recorded at trace rows off ...; R = the trace's rows.
int score_head(const grpo_model* m, const ScoreWS& w, int rows, const int32_t* tk, int T,
               int score_from, int Ts, int i0, float temperature, float* logp,
               const grpo_trace* tr, size_t R, int off, hipStream_t st) {
  const grpo_config& c = m->cfg;
  const int d = c.d_model, slots = lse_slots(c.vocab);
  const float t = temperature > 0.f ? temperature : 1.f;
  EpiArgs ep{w.lse, nullptr, slots};
  ep.lse = LseArgs{tk, T, Ts, score_from, i0, 1.44269504088896341f / t, w.tgt_z};
  if (int rc = gemm_rows(m, w.hs, d, rows, one(m->lm_head), c.vocab, d, EPI_LSE, ep, st)) return rc;
  HIPCHK(lse_combine(w.lse, slots, w.tgt_z, rows, t, logp, st));
  if (!tr) return GRPO_OK;
  if (int rc = trace(tr->h_final, 0, R, d, w.hs, c.dtype == GRPO_F32 ? TR_F32 : TR_BF16, d, rows,
                     TraceMap::rows(off), st))
    return rc;
  if (!tr->logits) return GRPO_OK;
  return gemm_rows(m, w.hs, d, rows, one(m->lm_head), c.vocab, d, EPI_STORE,
                   EpiArgs{tr->logits + (size_t)off * c.vocab, nullptr, c.vocab}, st);
}

int check_sampling(const grpo_sampling* s, int vocab) {
  if (!s) return fail(GRPO_INVALID_ARG, "sampling is NULL");
  if (!(s->temperature >= 0.f) || s->temperature == INFINITY)
    return fail(GRPO_INVALID_ARG, "temperature must be finite and >= 0");
  if (s->top_k < 0 || s->top_k > vocab) return fail(GRPO_INVALID_ARG, "top_k outside [0, vocab]");
  return GRPO_OK;
}

// ---- backward pass (grpo_policy_backward) ----------------------------------------
constexpr size_t kAttnBwdBytes = size_t(8) << 30;   // per-head attention scratch per batch
constexpr size_t kHeadBwdBytes = size_t(1) << 30;   // LM-head logits per row chunk
int round64(int t) { return (t + 63) / 64 * 64; }

struct BackwardWS {
  int Tp, hb, head_rows;
  float* X;                       // (L + 1) x [T, d] residual stream checkpoints
  void* h; float* qkv; void* q; void* kb; void* vb; uint16_t* vt; void* o;
  float* xa; void* h2; float* gu; void* a; float2* cs;
  float* dx; float* dxa; void* dxe; float* da; void* dgu; float* dh; float* dof; void* doe;
  float* dqkv; void* dqkve; float* rr; float* part;
  uint32_t* ekeys;                // the embedding gradient's sorted (token, position) keys
  void* tA; void* tB;             // transposed gradient / activation operands [rows][Tp]
  float* S; float* dP; float* stats; void* dS; void* PT; void* dST; void* qT; void* doT; void* kT;
  float* tk; float* tv;           // per-head dk, dv before the sum over each group
  void* hf; float* z; void* dz; void* dzT; void* hfT; float* dhf;
  std::vector<void*> WdT, WguT, WoT, WqkvT;
  void* WheadT;
};

BackwardWS take_backward(Bump& b, const grpo_config& c, int T) {
  BackwardWS w;
  const int es = esize(c), d = c.d_model, qd = qdim(c), kvd = kvdim(c), f = c.d_ffn;
  const int ldqkv = qd + 2 * kvd, hd = c.head_dim, V = c.vocab, L = c.n_layers;
  const int gq = c.n_heads / c.n_kv_heads;
  const int Tp = round64(T);
  w.Tp = Tp;
  const size_t TT = (size_t)T * Tp, PP = (size_t)Tp * Tp;
  // fp32 models keep S and dP (fp32) and the row statistics per head; bf16
  // models form the scores inside the fused kernel
  const bool fp32_scores = c.dtype == GRPO_F32;
  const size_t per_head = TT * ((fp32_scores ? 8 : 0) + es) + PP * 2 * es +
                          (size_t)hd * Tp * 2 * es + (size_t)T * hd * 8 +
                          (fp32_scores ? (size_t)T * 12 : 0);
  int groups = (int)std::max<size_t>(1, kAttnBwdBytes / (per_head * gq));
  groups = std::min(groups, c.n_kv_heads);
  while (c.n_kv_heads % groups) --groups;
  w.hb = groups * gq;
  w.head_rows = (int)std::max<size_t>(64, std::min<size_t>((size_t)T, kHeadBwdBytes / ((size_t)V * (4 + 2 * es))));
  w.head_rows = std::max(64, w.head_rows / 64 * 64);
  const int R = w.head_rows, Rp = round64(R);
  w.X = b.take<float>((size_t)(L + 1) * T * d);
  w.h = b.take<char>((size_t)T * d * es);
  w.qkv = b.take<float>((size_t)T * ldqkv);
  w.q = b.take<char>((size_t)T * qd * es);
  w.kb = b.take<char>((size_t)kvd * Tp * es);
  w.vb = b.take<char>((size_t)kvd * Tp * es);
  w.vt = b.take<uint16_t>(c.dtype == GRPO_F32 ? 0 : (size_t)kvd * round8(T));
  w.o = b.take<char>((size_t)T * qd * es);
  w.xa = b.take<float>((size_t)T * d);
  w.h2 = b.take<char>((size_t)T * d * es);
  w.gu = b.take<float>((size_t)T * 2 * f);
  w.a = b.take<char>((size_t)T * f * es);
  w.cs = b.take<float2>((size_t)T * (hd / 2));
  w.dx = b.take<float>((size_t)T * d);
  w.dxa = b.take<float>((size_t)T * d);
  w.dxe = b.take<char>((size_t)T * d * es);
  w.da = b.take<float>((size_t)T * f);
  w.dgu = b.take<char>((size_t)T * 2 * f * es);
  w.dh = b.take<float>((size_t)T * std::max(d, R > 0 ? d : d));
  w.dof = b.take<float>((size_t)T * qd);
  w.doe = b.take<char>((size_t)T * qd * es);
  w.dqkv = b.take<float>((size_t)T * ldqkv);
  w.dqkve = b.take<char>((size_t)T * ldqkv * es);
  w.rr = b.take<float>((size_t)std::max(T, R));
  w.part = b.take<float>((size_t)((std::max(T, R) + 63) / 64) * d);
  w.ekeys = b.take<uint32_t>((size_t)T);
  const int rowsA = std::max(std::max(2 * f, ldqkv), d);
  const int rowsB = std::max(std::max(f, d), qd);
  w.tA = b.take<char>((size_t)rowsA * Tp * es);
  w.tB = b.take<char>((size_t)rowsB * Tp * es);
  const int hb = w.hb;
  w.S = b.take<float>(fp32_scores ? hb * TT : 0);
  w.dP = b.take<float>(fp32_scores ? hb * TT : 0);
  w.stats = b.take<float>(fp32_scores ? (size_t)hb * T * 3 : 0);
  w.dS = b.take<char>(hb * TT * es);
  w.PT = b.take<char>(hb * PP * es);
  w.dST = b.take<char>(hb * PP * es);
  w.qT = b.take<char>((size_t)hb * hd * Tp * es);
  w.doT = b.take<char>((size_t)hb * hd * Tp * es);
  w.kT = b.take<char>((size_t)c.n_kv_heads * hd * Tp * es);
  w.tk = b.take<float>((size_t)hb * T * hd);
  w.tv = b.take<float>((size_t)hb * T * hd);
  w.hf = b.take<char>((size_t)R * d * es);
  w.z = b.take<float>((size_t)R * V);
  w.dz = b.take<char>((size_t)R * V * es);
  w.dzT = b.take<char>((size_t)V * Rp * es);
  w.hfT = b.take<char>((size_t)d * Rp * es);
  w.dhf = b.take<float>((size_t)R * d);
  for (int l = 0; l < L; ++l) {
    w.WdT.push_back(b.take<char>((size_t)f * d * es));
    w.WguT.push_back(b.take<char>((size_t)d * 2 * f * es));
    w.WoT.push_back(b.take<char>((size_t)qd * d * es));
    w.WqkvT.push_back(b.take<char>((size_t)d * ldqkv * es));
  }
  w.WheadT = b.take<char>((size_t)d * V * es);
  return w;
}

int gemm_bt(const grpo_model* m, const void* X, int ldx, int M, WStack W, int N, int K, int epi,
            EpiArgs ep, GemmBatch bt, hipStream_t st) {
  const hipError_t e =
      m->cfg.dtype == GRPO_F32
          ? gemm_f32((const float*)X, ldx, M, W, N, K, epi, ep, st, bt)
          : gemm_tiled_bf16((const uint16_t*)X, ldx, M, W, N, K, epi, ep, st, bt);
  return e == hipSuccess ? GRPO_OK : gemm_fail(e);
}

// transposed copy of rows [N, K] (the model dtype) as [K, N]
hipError_t transpose_w(const grpo_config& c, const void* w, int N, int K, void* out, int ldo,
                       hipStream_t st) {
  const int t = c.dtype == GRPO_F32 ? 0 : 1;
  return transpose(t, t, w, K, 0, N, K, out, ldo, 0, 0, 1, N, 1, st);
}

// one layer's forward over a sequence from its input x [T, d]: h, q, K/V (kb, vb
// [n_kv][Tp][hd]), o, xa, h2, gate|up (gu) and a; x_out (optional) = xa + a Wd^T
int layer_fwd(const grpo_model* m, BackwardWS& w, int l, const float* x, int T, float* x_out,
              hipStream_t st) {
  const grpo_config& c = m->cfg;
  const int d = c.d_model, qd = qdim(c), kvd = kvdim(c), f = c.d_ffn, ldqkv = qd + 2 * kvd;
  const Partials none{nullptr, 0, 0, d};
  int rc;
  HIPCHK(rmsnorm(c.dtype, const_cast<float*>(x), d, RowMap::identity(), none, m->attn_norm[l], T,
                 d, c.rms_eps, w.h, d, st));
  if ((rc = gemm_rows(m, w.h, d, T, qkv_stack(m, l), ldqkv, d, EPI_STORE,
                      EpiArgs{w.qkv, nullptr, ldqkv}, st)))
    return rc;
  RopeArgs ra{};
  ra.mode = 1; ra.T = T; ra.G = 1; ra.pos_arr = nullptr; ra.pos0 = 0;
  ra.n_heads = c.n_heads; ra.n_kv = c.n_kv_heads; ra.hd = c.head_dim; ra.theta = c.rope_theta;
  ra.kcache = w.kb; ra.vcache = w.vb; ra.n_seqs = 1; ra.max_len = w.Tp;
  ra.vt = c.dtype == GRPO_F32 ? nullptr : w.vt; ra.vt_len = round8(T);
  ra.splits = 1; ra.split_stride = 0; ra.cs = w.cs;
  HIPCHK(rope_kv(c.dtype, w.qkv, T, w.q, ra, st));
  HIPCHK(attn_prefill(c.dtype, w.q, w.kb, c.dtype == GRPO_F32 ? w.vb : (const void*)w.vt, 1, T,
                      c.n_heads, c.n_kv_heads, c.head_dim, w.Tp, 1, w.o, st, 0, 1, round8(T)));
  HIPCHK(hipMemcpyAsync(w.xa, x, (size_t)T * d * 4, hipMemcpyDeviceToDevice, st));
  if ((rc = gemm_rows(m, w.o, qd, T, one(m->wo[l]), d, qd, EPI_RESID, EpiArgs{w.xa, nullptr, d},
                      st)))
    return rc;
  HIPCHK(rmsnorm(c.dtype, w.xa, d, RowMap::identity(), none, m->mlp_norm[l], T, d, c.rms_eps,
                 w.h2, d, st));
  if ((rc = gemm_rows(m, w.h2, d, T, gate_up(m, l), 2 * f, d, EPI_STORE,
                      EpiArgs{w.gu, nullptr, 2 * f}, st)))
    return rc;
  HIPCHK(swiglu_fwd(c.dtype, w.gu, T, f, w.a, st));
  if (!x_out) return GRPO_OK;
  HIPCHK(hipMemcpyAsync(x_out, w.xa, (size_t)T * d * 4, hipMemcpyDeviceToDevice, st));
  return gemm_rows(m, w.a, f, T, one(m->w_down[l]), d, f, EPI_RESID, EpiArgs{x_out, nullptr, d}, st);
}

// dW[N, K] += dY^T X over T token rows: dY [T, N] (fp32 or the model dtype, ld
// ldy), X [T, K] (the model dtype, ld ldx); both transposed into [.][Tp] first
int wgrad(const grpo_model* m, BackwardWS& w, const void* dY, int dy_f32, int ldy, int N,
          const void* X, int ldx, int K, int T, float* dW, hipStream_t st) {
  const grpo_config& c = m->cfg;
  const int e = c.dtype == GRPO_F32 ? 0 : 1;
  HIPCHK(transpose(dy_f32 ? 0 : e, e, dY, ldy, 0, T, N, w.tA, w.Tp, 0, 0, 1, w.Tp, 1, st));
  HIPCHK(transpose(e, e, X, ldx, 0, T, K, w.tB, w.Tp, 0, 0, 1, w.Tp, 1, st));
  return gemm_rows(m, w.tA, w.Tp, N, one(w.tB), K, w.Tp, EPI_RESID, EpiArgs{dW, nullptr, K}, st);
}

// attention backward of one sequence: do (w.doe) -> dq, dk, dv in w.dqkv
int attn_bwd(const grpo_model* m, BackwardWS& w, int T, hipStream_t st) {
  const grpo_config& c = m->cfg;
  const int H = c.n_heads, Hk = c.n_kv_heads, hd = c.head_dim, gq = H / Hk;
  const int qd = qdim(c), kvd = kvdim(c), ldqkv = qd + 2 * kvd, Tp = w.Tp, es = esize(c);
  const int e = c.dtype == GRPO_F32 ? 0 : 1;
  const size_t TT = (size_t)T * Tp, PP = (size_t)Tp * Tp, hT = (size_t)hd * Tp;
  const float scale = 1.f / sqrtf((float)hd);
  char* kb = (char*)w.kb;
  char* vb = (char*)w.vb;
  int rc;
  // K^T of every kv head [n_kv][hd][Tp]
  HIPCHK(transpose(e, e, w.kb, hd, (size_t)Tp * hd, T, hd, w.kT, Tp, hT, 0, 1, Tp, Hk, st));
  for (int h0 = 0; h0 < H; h0 += w.hb) {
    const int nb = std::min(w.hb, H - h0), g0 = h0 / gq;
    if (c.dtype == GRPO_BF16) {
      // P and dS' straight from q, do, k and v (the scores formed twice, never stored)
      HIPCHK(attn_scores_bwd((char*)w.q + (size_t)h0 * hd * es, (char*)w.doe + (size_t)h0 * hd * es,
                             qd, kb + (size_t)g0 * Tp * hd * es, vb + (size_t)g0 * Tp * hd * es, gq,
                             T, Tp, nb, hd, scale, w.dS, w.dST, w.PT, st));
    } else {
      // S = q_h k_g^T, dP = do_h v_g^T (raw products, fp32)
      GemmBatch sb{nb, (size_t)hd, (size_t)Tp * hd, TT, gq, 1};   // causal: lower tiles only
      if ((rc = gemm_bt(m, (char*)w.q + (size_t)h0 * hd * es, qd, T,
                        one(kb + (size_t)g0 * Tp * hd * es), T, hd, EPI_STORE,
                        EpiArgs{w.S, nullptr, Tp}, sb, st)))
        return rc;
      if ((rc = gemm_bt(m, (char*)w.doe + (size_t)h0 * hd * es, qd, T,
                        one(vb + (size_t)g0 * Tp * hd * es), T, hd, EPI_STORE,
                        EpiArgs{w.dP, nullptr, Tp}, sb, st)))
        return rc;
      HIPCHK(attn_softmax_bwd(c.dtype, w.S, w.dP, T, Tp, nb, scale, w.stats, w.dS, w.dST, w.PT,
                              st));
    }
    // dq_h = dS'_h k_g (K = key positions)
    GemmBatch qb{nb, TT, hT, (size_t)hd, gq, 2};   // dS' is zero past each row
    if ((rc = gemm_bt(m, w.dS, Tp, T, one((char*)w.kT + (size_t)g0 * hT * es), hd, Tp, EPI_STORE,
                      EpiArgs{w.dqkv + (size_t)h0 * hd, nullptr, ldqkv}, qb, st)))
      return rc;
    // per head: dk_h = dS'_h^T q_h, dv_h = P_h^T do_h (K = query positions)
    HIPCHK(transpose(e, e, (char*)w.q + (size_t)h0 * hd * es, qd, hd, T, hd, w.qT, Tp, hT, 0, 1,
                     Tp, nb, st));
    HIPCHK(transpose(e, e, (char*)w.doe + (size_t)h0 * hd * es, qd, hd, T, hd, w.doT, Tp, hT, 0,
                     1, Tp, nb, st));
    GemmBatch kb2{nb, PP, hT, (size_t)T * hd, 1, 3};   // dS'^T, P^T zero before each row
    if ((rc = gemm_bt(m, w.dST, Tp, T, one(w.qT), hd, Tp, EPI_STORE, EpiArgs{w.tk, nullptr, hd},
                      kb2, st)) ||
        (rc = gemm_bt(m, w.PT, Tp, T, one(w.doT), hd, Tp, EPI_STORE, EpiArgs{w.tv, nullptr, hd},
                      kb2, st)))
      return rc;
    HIPCHK(sum_heads(w.tk, T, hd, gq, nb / gq, w.dqkv + qd + (size_t)g0 * hd, ldqkv, st));
    HIPCHK(sum_heads(w.tv, T, hd, gq, nb / gq, w.dqkv + qd + kvd + (size_t)g0 * hd, ldqkv, st));
  }
  return GRPO_OK;
}

}  // namespace

extern "C" {

const char* grpo_last_error(void) { return g_err.c_str(); }

int grpo_model_create(const grpo_config* cfg, const grpo_weights* w, grpo_model** out) {
  if (!out) return fail(GRPO_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (int rc = check_config(cfg)) return rc;
  if (!w) return fail(GRPO_INVALID_ARG, "weights is NULL");
  if (!w->tok_emb || !w->final_norm || !w->lm_head)
    return fail(GRPO_INVALID_ARG, "tok_emb, final_norm and lm_head must be set");
  const void* const* arrays[9] = {w->attn_norm, w->wq, w->wk, w->wv, w->wo,
                                  w->mlp_norm, w->w_gate, w->w_up, w->w_down};
  for (auto a : arrays) {
    if (!a) return fail(GRPO_INVALID_ARG, "a per-layer weight array is NULL");
    for (int l = 0; l < cfg->n_layers; ++l)
      if (!a[l]) return fail(GRPO_INVALID_ARG, "layer %d has a NULL weight pointer", l);
  }
  grpo_model* m = new grpo_model;
  m->cfg = *cfg;
  m->tok_emb = w->tok_emb;
  m->final_norm = w->final_norm;
  m->lm_head = w->lm_head;
  std::vector<const void*>* dst[9] = {&m->attn_norm, &m->wq, &m->wk, &m->wv, &m->wo,
                                      &m->mlp_norm, &m->w_gate, &m->w_up, &m->w_down};
  for (int i = 0; i < 9; ++i) dst[i]->assign(arrays[i], arrays[i] + cfg->n_layers);
  *out = m;
  g_err.clear();
  return GRPO_OK;
}

int grpo_model_destroy(grpo_model* m) {
  if (!m) return GRPO_OK;
  if (m->graph.exec) {
    (void)hipDeviceSynchronize();
    (void)hipGraphExecDestroy(m->graph.exec);
  }
  if (m->graph.capture) (void)hipStreamDestroy(m->graph.capture);
  delete m;
  return GRPO_OK;
}

size_t grpo_decode_weights_bytes(const grpo_config* cfg) {
  if (check_config(cfg) || cfg->dtype != GRPO_BF16) return 0;
  return decode_layout(*cfg).total;
}

int grpo_model_pack_decode(grpo_model* m, void* buf, size_t bytes, void* stream) {
  if (!m) return fail(GRPO_INVALID_ARG, "model is NULL");
  const grpo_config& c = m->cfg;
  if (c.dtype != GRPO_BF16) {
    g_err.clear();
    return GRPO_OK;   // fp32 models decode from the row-major weights
  }
  const DecodeLayout L = decode_layout(c);
  if (!buf) return fail(GRPO_INVALID_ARG, "buf is NULL");
  if (bytes < L.total)
    return fail(GRPO_INVALID_ARG, "decode weight buffer %zu bytes, need %zu", bytes, L.total);
  if ((uintptr_t)buf % 256) return fail(GRPO_INVALID_ARG, "buf must be 256-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  const int d = c.d_model, qd = qdim(c), kvd = kvdim(c), f = c.d_ffn;
  char* base = (char*)buf;
  auto at = [&](size_t off) { return (uint16_t*)(base + off); };
  for (int l = 0; l < c.n_layers; ++l) {
    HIPCHK(pack_frag(PackSrc{{m->wq[l], m->wk[l], m->wv[l]}, qd, qd + kvd, 0}, qd + 2 * kvd, d,
                     at(L.qkv[l]), st));
    HIPCHK(pack_frag(PackSrc{{m->wo[l], m->wo[l], m->wo[l]}, d, d, 0}, d, qd, at(L.o[l]), st));
    HIPCHK(pack_frag(PackSrc{{m->w_gate[l], m->w_up[l], m->w_up[l]}, 0, 0, 1}, 2 * f, d,
                     at(L.gate_up[l]), st));
    HIPCHK(pack_frag(PackSrc{{m->w_down[l], m->w_down[l], m->w_down[l]}, d, d, 0}, d, f,
                     at(L.down[l]), st));
  }
  HIPCHK(pack_frag(PackSrc{{m->lm_head, m->lm_head, m->lm_head}, c.vocab, c.vocab, 0}, c.vocab, d,
                   at(L.lm_head), st));
  DecodeWeights& D = m->dec;
  D.base = buf;
  D.qkv.assign(c.n_layers, nullptr);
  D.o.assign(c.n_layers, nullptr);
  D.gate_up.assign(c.n_layers, nullptr);
  D.down.assign(c.n_layers, nullptr);
  for (int l = 0; l < c.n_layers; ++l) {
    D.qkv[l] = at(L.qkv[l]);
    D.o[l] = at(L.o[l]);
    D.gate_up[l] = at(L.gate_up[l]);
    D.down[l] = at(L.down[l]);
  }
  D.lm_head = at(L.lm_head);
  g_err.clear();
  return GRPO_OK;
}

int grpo_decode_structure(const grpo_model* m, int32_t B, int32_t max_len, int32_t G,
                          int32_t prefix_len, int32_t* out) {
  if (!m || !out) return fail(GRPO_INVALID_ARG, "model and out must be set");
  if (B < 1 || B > 128 || max_len < 1 || G < 0 || (G > 0 && B % G) || prefix_len < 0 ||
      prefix_len > max_len)
    return fail(GRPO_INVALID_ARG, "sizes outside the decode step's ranges");
  for (int i = 0; i < 9; ++i) out[i] = 0;
  const grpo_config& c = m->cfg;
  if (c.dtype == GRPO_F32) {
    g_err.clear();
    return GRPO_OK;
  }
  const int d = c.d_model, qd = qdim(c), kvd = kvdim(c), f = c.d_ffn;
  out[0] = decode_plan(B, qd + 2 * kvd, d, EPI_PARTIAL, decode_target()).splits;
  out[1] = decode_plan(B, d, qd, EPI_PARTIAL, decode_target()).splits;
  out[2] = decode_plan(B, d, f, EPI_PARTIAL, decode_target()).splits;
  out[3] = decode_plan(B, c.vocab, d, EPI_PARTIAL, decode_target(), 1).splits;
  const bool grouped = G > 0 && prefix_len > 0;
  const DecodeAttnPlan ap = decode_attn_plan(B, c.n_heads, c.n_kv_heads, c.head_dim, max_len,
                                             grouped ? G : 0, grouped ? prefix_len : 0);
  out[4] = ap.tc;
  out[5] = ap.splits;
  out[6] = grouped ? ap.span_p : 0;
  out[7] = grouped ? ap.chunks : 0;
  out[8] = ap.waves;
  g_err.clear();
  return GRPO_OK;
}

int grpo_profile_begin(void) {
  if (counter_collection())
    return fail(GRPO_UNSUPPORTED, "kernel timing is off while hardware counters are collected");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_acc.clear();
  g_prof.store(true);
  return GRPO_OK;
}

int grpo_profile_end(char* json, size_t len) {
  std::string out = "{";
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof.store(false);
    prof_drain(0);
    bool first = true;
    for (auto& kv : g_prof_acc) {
      char buf[256];
      snprintf(buf, sizeof buf, "%s\"%s\": [%ld, %.6f]", first ? "" : ", ", kv.first.c_str(),
               kv.second.first, kv.second.second);
      out += buf;
      first = false;
    }
  }
  out += "}";
  if (!json || len == 0) return fail(GRPO_INVALID_ARG, "json buffer is NULL");
  if (out.size() + 1 > len) return fail(GRPO_INVALID_ARG, "json buffer too small (%zu)", out.size() + 1);
  memcpy(json, out.c_str(), out.size() + 1);
  return GRPO_OK;
}

size_t grpo_kv_cache_bytes(const grpo_config* cfg, int32_t n_seqs, int32_t max_len) {
  if (check_config(cfg) || n_seqs < 1 || max_len < 1) return 0;
  return (size_t)cfg->n_layers * 2 * n_seqs * cfg->n_kv_heads * max_len * cfg->head_dim *
         esize(*cfg);
}

size_t grpo_workspace_bytes(const grpo_model* m, int32_t op, int32_t n_rows, int32_t seq_len) {
  if (n_rows < 1 || seq_len < 1) return 0;
  Bump b(nullptr);
  if (op == GRPO_OP_LOSS) {
    b.take<double>((size_t)n_rows * 9);
    return b.off;
  }
  if (!m) return 0;
  switch (op) {
    case GRPO_OP_PREFILL: take_prefill(b, m->cfg, n_rows, seq_len); break;
    case GRPO_OP_ROLLOUT: take_rollout(b, m->cfg, n_rows, seq_len); break;
    case GRPO_OP_SCORE: take_score(b, m->cfg, n_rows, seq_len); break;
    case GRPO_OP_EXTEND: take_extend(b, m->cfg, n_rows, seq_len); break;
    case GRPO_OP_BACKWARD:
      if (seq_len < 2 || seq_len > kBackwardTokens) return 0;
      take_backward(b, m->cfg, seq_len);
      break;
    default: return 0;
  }
  return b.off;
}

int grpo_prefill(const grpo_model* m, void* kv, int32_t n_seqs, int32_t max_len,
                 const int32_t* prompts, int32_t P, int32_t Tp, int32_t G, const grpo_sampling* s,
                 int32_t* tok_out, float* logp_out, const grpo_trace* trace_out, void* ws,
                 size_t ws_bytes, void* stream) {
  if (!m) return fail(GRPO_INVALID_ARG, "model is NULL");
  const grpo_config& c = m->cfg;
  if (!kv || !prompts || !tok_out || !logp_out || !ws)
    return fail(GRPO_INVALID_ARG, "kv, prompts, tok_out, logp_out and ws must be set");
  if (P < 1 || Tp < 1 || G < 1) return fail(GRPO_INVALID_ARG, "P, Tp and G must be >= 1");
  if ((long)P * G > n_seqs) return fail(GRPO_INVALID_ARG, "P*G = %ld exceeds n_seqs %d", (long)P * G, n_seqs);
  if (Tp > max_len) return fail(GRPO_KV_CAPACITY, "prompt length %d exceeds max_len %d", Tp, max_len);
  if ((long)P * Tp > (1L << 30)) return fail(GRPO_UNSUPPORTED, "P*Tp too large");
  if (c.dtype == GRPO_F32 && Tp > 16384) return fail(GRPO_UNSUPPORTED, "fp32 prompts above 16384");
  if (int rc = check_sampling(s, c.vocab)) return rc;
  const size_t need = grpo_workspace_bytes(m, GRPO_OP_PREFILL, P, Tp);
  if (ws_bytes < need)
    return fail(GRPO_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes, need);
  hipStream_t st = (hipStream_t)stream;
  Bump b(ws);
  PrefillWS w = take_prefill(b, c, P, Tp);
  const int M = P * Tp, d = c.d_model;
  HIPCHK(embed(c.dtype, m->tok_emb, prompts, M, d, c.vocab, w.s.x, st));
  if (int rc = forward_rows(m, w.s, M, Tp, G, n_seqs, max_len, kv, nullptr, nullptr, w.vt,
                            trace_out, (size_t)M, TraceMap::rows(), st))
    return rc;
  const Partials none{nullptr, 0, 0, d};
  HIPCHK(rmsnorm(c.dtype, w.s.x, d, RowMap{0, 1, Tp, Tp - 1}, none, m->final_norm, P, d, c.rms_eps,
                 w.hl, d, st));
  if (int rc = gemm_rows(m, w.hl, d, P, one(m->lm_head), c.vocab, d, EPI_STORE,
                         EpiArgs{w.logits, nullptr, c.vocab}, st))
    return rc;
  if (int rc = trace(TRM(trace_out, h_final), 0, P, d, w.hl,
                     c.dtype == GRPO_F32 ? TR_F32 : TR_BF16, d, P, TraceMap::rows(), st))
    return rc;
  if (int rc = trace(TRM(trace_out, logits), 0, P, c.vocab, w.logits, TR_F32, c.vocab, P,
                     TraceMap::rows(), st))
    return rc;
  SampleArgs sa{};
  sa.temperature = s->temperature; sa.top_k = s->top_k; sa.seed = s->seed; sa.step = 0;
  sa.G = G; sa.tok_out = tok_out; sa.logp_out = logp_out; sa.out_stride = 1;
  HIPCHK(sample(w.logits, P, c.vocab, c.vocab, sa, st));
  g_err.clear();
  return GRPO_OK;
}

// Decode steps; G > 0: rows in groups of G sharing the cache below prefix_len.
static int rollout(const grpo_model* m, void* kv, int32_t n_seqs, int32_t max_len, int32_t B,
                   const int32_t* seq_ids, int32_t* pos, int32_t* tok, int32_t max_pos,
                   int32_t step0, int32_t n_steps, const grpo_sampling* s, int32_t* tok_out,
                   float* logp_out, const grpo_trace* trace_out, int32_t G, int32_t prefix_len,
                   void* ws, size_t ws_bytes, void* stream) {
  if (!m) return fail(GRPO_INVALID_ARG, "model is NULL");
  const grpo_config& c = m->cfg;
  if (!kv || !pos || !tok || !tok_out || !logp_out || !ws)
    return fail(GRPO_INVALID_ARG, "kv, pos, tok, tok_out, logp_out and ws must be set");
  if (B < 1 || n_steps < 1 || max_len < 1) return fail(GRPO_INVALID_ARG, "B, n_steps, max_len must be >= 1");
  if (B > n_seqs) return fail(GRPO_INVALID_ARG, "B %d exceeds n_seqs %d", B, n_seqs);
  if (c.dtype == GRPO_BF16 && B > 128) return fail(GRPO_UNSUPPORTED, "B %d above 128 for a bf16 model", B);
  if (max_pos < 0 || step0 < 0) return fail(GRPO_INVALID_ARG, "max_pos and step0 must be >= 0");
  if ((long)max_pos + n_steps > max_len)
    return fail(GRPO_KV_CAPACITY, "max_pos %d + n_steps %d exceeds max_len %d", max_pos, n_steps,
                max_len);
  if (c.dtype == GRPO_F32 && max_len > 16384) return fail(GRPO_UNSUPPORTED, "fp32 caches above 16384");
  if (int rc = check_sampling(s, c.vocab)) return rc;
  if (seq_ids) {
    std::vector<int32_t> sorted(seq_ids, seq_ids + B);
    for (int b = 0; b < B; ++b)
      if (sorted[b] < 0 || sorted[b] >= n_seqs)
        return fail(GRPO_INVALID_ARG, "seq_ids[%d] = %d outside [0, n_seqs %d)", b, sorted[b], n_seqs);
    std::sort(sorted.begin(), sorted.end());
    for (int b = 1; b < B; ++b)
      if (sorted[b] == sorted[b - 1])
        return fail(GRPO_INVALID_ARG, "seq_ids repeats sequence %d", sorted[b]);
  }
  const size_t need = grpo_workspace_bytes(m, GRPO_OP_ROLLOUT, B, max_len);
  if (ws_bytes < need)
    return fail(GRPO_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes, need);
  if (c.dtype == GRPO_BF16 && !m->dec.base)
    return fail(GRPO_INVALID_ARG, "bf16 model without decode weights (grpo_model_pack_decode)");
  hipStream_t st = (hipStream_t)stream;
  Bump b(ws);
  RolloutWS w = take_rollout(b, c, B, max_len);
  const int d = c.d_model, qd = qdim(c), kvd = kvdim(c), f = c.d_ffn;
  const bool pk = c.dtype == GRPO_BF16;
  const int nb = pk ? decode_nb(B) : 0;
  // GEMM inputs of bf16 decode sit in fragment order over the padded batch
  const int act = pk ? TR_FRAG : TR_F32;
  const int act_ld = pk ? nb : 0;
  // fp32 attention reads every row's own cache (the shared positions hold the
  // same values, so the results are those of a grouped step)
  const bool grouped = pk && G > 0 && prefix_len > 0;
  const DecodeAttnPlan ap = decode_attn_plan(B, c.n_heads, c.n_kv_heads, c.head_dim, max_len,
                                             grouped ? G : 0, grouped ? prefix_len : 0);
  // the rows' cache slots / Philox sequence ids, once per call
  const int32_t* slots = nullptr;
  if (seq_ids) {
    HIPCHK(set_i32(w.slots, seq_ids, B, st));
    slots = w.slots;
  }
  const TraceMap rows = TraceMap::rows();
  // One decode step on stream `ss`.  In graph mode the Philox step and the output
  // column come from the device step counter (advanced by the embedding kernel).
  auto enqueue_step = [&](hipStream_t ss, bool graph, int step) -> int {
    const grpo_trace* tr = step == n_steps - 1 ? trace_out : nullptr;
    int rc;
    hipStream_t st = ss;
    HIPCHK(embed(c.dtype, m->tok_emb, tok, B, d, c.vocab, w.s.x, st, graph ? w.step_ctr : nullptr));
    HIPCHK(rope_table(pos, B, c.head_dim, c.rope_theta, w.s.cs, st));
    // bf16: GEMM inputs in fragment order, products as split-K partials;
    // fp32: row-major, products straight into their destinations
    Partials pend{nullptr, 0, 0, d};
    const DecodeWeights& D = m->dec;
    for (int l = 0; l < c.n_layers; ++l) {
      Layer L = kv_layer(m, kv, l, n_seqs, max_len);
      HIPCHK(rmsnorm(c.dtype, w.s.x, d, RowMap::identity(), pend, m->attn_norm[l], B, d,
                     c.rms_eps, w.s.h, d, st, nb));
      if ((rc = trace(TRM(tr, x), l, B, d, w.s.x, TR_F32, d, B, rows, st)) ||
          (rc = trace(TRM(tr, h_attn), l, B, d, w.s.h, act, pk ? act_ld : d, B, rows, st)))
        return rc;
      const float* qsrc = w.s.qkv;
      int qs = 1;
      size_t qstride = 0;
      if (pk) {
        if ((rc = gemm_dec(w.s.h, B, D.qkv[l], qd + 2 * kvd, d, w.s.qkv, w.s.g, kMaxSplits, &qsrc,
                           &qs, &qstride, st, "gemm_decode_qkv")))
          return rc;
      } else if ((rc = gemm_rows(m, w.s.h, d, B, qkv_stack(m, l), qd + 2 * kvd, d, EPI_STORE,
                                 EpiArgs{w.s.qkv, nullptr, qd + 2 * kvd}, st))) {
        return rc;
      }
      RopeArgs ra{};
      ra.mode = 0; ra.T = 1; ra.G = 1; ra.pos_arr = pos; ra.slots = slots;
      ra.n_heads = c.n_heads; ra.n_kv = c.n_kv_heads; ra.hd = c.head_dim; ra.theta = c.rope_theta;
      ra.kcache = L.k; ra.vcache = L.v; ra.n_seqs = n_seqs; ra.max_len = max_len;
      ra.vt = nullptr; ra.vt_len = 0;
      ra.splits = qs; ra.split_stride = qstride;
      ra.cs = w.s.cs;
      if (tr) {
        ra.tq = tr->q ? tr->q + (size_t)l * B * qd : nullptr;
        ra.tk = tr->k ? tr->k + (size_t)l * B * kvd : nullptr;
        ra.tv = tr->v ? tr->v + (size_t)l * B * kvd : nullptr;
        ra.tmap = rows;
      }
      HIPCHK(rope_kv(c.dtype, qsrc, B, w.s.q, ra, st));
      HIPCHK(attn_decode(c.dtype, w.s.q, L.k, L.v, pos, slots, B, c.n_heads, c.n_kv_heads,
                         c.head_dim, n_seqs, max_len, ap, w.attn_part, w.s.o, st, nb));
      if ((rc = trace(TRM(tr, o), l, B, qd, w.s.o, act, pk ? act_ld : qd, B, rows, st))) return rc;
      if (pk) {
        if ((rc = gemm_dec_resid(w.s.o, B, D.o[l], d, qd, w.s.g, &pend, st, "gemm_decode_o")))
          return rc;
      } else if ((rc = gemm_rows(m, w.s.o, qd, B, one(m->wo[l]), d, qd, EPI_RESID,
                                 EpiArgs{w.s.x, nullptr, d}, st))) {
        return rc;
      }
      HIPCHK(rmsnorm(c.dtype, w.s.x, d, RowMap::identity(), pend, m->mlp_norm[l], B, d, c.rms_eps,
                     w.s.h, d, st, nb));
      if ((rc = trace(TRM(tr, x_attn), l, B, d, w.s.x, TR_F32, d, B, rows, st)) ||
          (rc = trace(TRM(tr, h_mlp), l, B, d, w.s.h, act, pk ? act_ld : d, B, rows, st)))
        return rc;
      if (pk) {
        if ((rc = gemm_dec_swiglu(w.s.h, B, D.gate_up[l], f, d, w.s.a, st))) return rc;
        if ((rc = trace(TRM(tr, act), l, B, f, w.s.a, act, act_ld, B, rows, st))) return rc;
        if ((rc = gemm_dec_resid(w.s.a, B, D.down[l], d, f, w.s.g, &pend, st, "gemm_decode_down")))
          return rc;
      } else {
        if ((rc = gemm_rows(m, w.s.h, d, B, gate_up(m, l), f, d, EPI_SWIGLU,
                            EpiArgs{nullptr, w.s.a, f}, st)))
          return rc;
        if ((rc = trace(TRM(tr, act), l, B, f, w.s.a, TR_F32, f, B, rows, st))) return rc;
        if ((rc = gemm_rows(m, w.s.a, f, B, one(m->w_down[l]), d, f, EPI_RESID,
                            EpiArgs{w.s.x, nullptr, d}, st)))
          return rc;
      }
    }
    HIPCHK(rmsnorm(c.dtype, w.s.x, d, RowMap::identity(), pend, m->final_norm, B, d, c.rms_eps,
                   w.s.h, d, st, nb));
    if ((rc = trace(TRM(tr, x), c.n_layers, B, d, w.s.x, TR_F32, d, B, rows, st)) ||
        (rc = trace(TRM(tr, h_final), 0, B, d, w.s.h, act, pk ? act_ld : d, B, rows, st)))
      return rc;
    SampleArgs sa{};
    sa.temperature = s->temperature; sa.top_k = s->top_k; sa.seed = s->seed;
    sa.G = 1; sa.out_stride = n_steps;
    sa.tok_state = tok; sa.pos_state = pos; sa.seq_ids = slots;
    if (graph) {
      sa.step = step0; sa.step_ctr = w.step_ctr;
      sa.tok_out = tok_out; sa.logp_out = logp_out;
    } else {
      sa.step = step0 + step; sa.step_ctr = nullptr;
      sa.tok_out = tok_out + step; sa.logp_out = logp_out + step;
    }
    // without a top-k cut the LM head's epilogue reduces its logits to the
    // sampler's per-tile pieces (the logits are stored only for a trace)
    if (pk && (s->top_k <= 0 || s->top_k >= c.vocab)) {
      float* lg = TRM(tr, logits) ? w.logits : nullptr;
      int tiles = 0;
      if ((rc = gemm_dec_sample(w.s.h, B, D.lm_head, c.vocab, d, sa, w.spart, lg, &tiles, st)))
        return rc;
      if ((rc = trace(TRM(tr, logits), 0, B, c.vocab, w.logits, TR_F32, c.vocab, B, rows, st)))
        return rc;
      HIPCHK(sample_combine(w.spart, tiles, B, c.vocab, sa, st));
      return GRPO_OK;
    }
    if (pk) {
      const float* res;
      int ns;
      size_t nst;
      if ((rc = gemm_dec(w.s.h, B, D.lm_head, c.vocab, d, w.logits, w.s.g, 1, &res, &ns, &nst, st,
                         "gemm_decode_lm_head")))
        return rc;
    } else if ((rc = gemm_rows(m, w.s.h, d, B, one(m->lm_head), c.vocab, d, EPI_STORE,
                               EpiArgs{w.logits, nullptr, c.vocab}, st))) {
      return rc;
    }
    if ((rc = trace(TRM(tr, logits), 0, B, c.vocab, w.logits, TR_F32, c.vocab, B, rows, st)))
      return rc;
    HIPCHK(sample(w.logits, B, c.vocab, c.vocab, sa, st));
    return GRPO_OK;
  };

  const bool use_graph = n_steps >= 2 && !trace_out && !profiling() && !getenv("GRPO_NO_GRAPH") &&
                         !counter_collection();
  if (!use_graph) {
    for (int step = 0; step < n_steps; ++step)
      if (int rc = enqueue_step(st, false, step)) return rc;
    g_err.clear();
    return GRPO_OK;
  }
  grpo_model* mm = const_cast<grpo_model*>(m);
  DecodeGraph& dg = mm->graph;
  const std::vector<uint64_t> key = {
      (uint64_t)(uintptr_t)kv, (uint64_t)n_seqs, (uint64_t)max_len, (uint64_t)B,
      (uint64_t)(uintptr_t)pos, (uint64_t)(uintptr_t)tok, (uint64_t)step0, (uint64_t)n_steps,
      (uint64_t)(uintptr_t)tok_out, (uint64_t)(uintptr_t)logp_out, (uint64_t)(uintptr_t)ws,
      (uint64_t)(uintptr_t)m->dec.base, (uint64_t)(slots != nullptr),
      (uint64_t)*(const uint32_t*)&s->temperature, (uint64_t)(uint32_t)s->top_k, s->seed,
      (uint64_t)(uint32_t)ap.G, (uint64_t)(uint32_t)ap.prefix_len};
  HIPCHK(fill_i32(w.step_ctr, 1, -1, st));   // the first replay's embedding makes it 0
  if (!dg.exec || dg.key != key) {
    if (dg.exec) {
      HIPCHK(hipStreamSynchronize(st));
      HIPCHK(hipGraphExecDestroy(dg.exec));
      dg.exec = nullptr;
    }
    if (!dg.capture) HIPCHK(hipStreamCreateWithFlags(&dg.capture, hipStreamNonBlocking));
    HIPCHK(hipStreamBeginCapture(dg.capture, hipStreamCaptureModeThreadLocal));
    const int rc = enqueue_step(dg.capture, true, 0);
    hipGraph_t graph = nullptr;
    const hipError_t ce = hipStreamEndCapture(dg.capture, &graph);
    if (rc) {
      if (graph) (void)hipGraphDestroy(graph);
      return rc;
    }
    if (ce != hipSuccess) return fail(GRPO_HIP_ERROR, "graph capture: %s", hipGetErrorString(ce));
    const hipError_t ie = hipGraphInstantiate(&dg.exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (ie != hipSuccess) {
      dg.exec = nullptr;
      return fail(GRPO_HIP_ERROR, "graph instantiate: %s", hipGetErrorString(ie));
    }
    dg.key = key;
  }
  for (int step = 0; step < n_steps; ++step) HIPCHK(hipGraphLaunch(dg.exec, st));
  g_err.clear();
  return GRPO_OK;
}

int grpo_rollout_step(const grpo_model* m, void* kv, int32_t n_seqs, int32_t max_len, int32_t B,
                      const int32_t* seq_ids, int32_t* pos, int32_t* tok, int32_t max_pos,
                      int32_t step0, int32_t n_steps, const grpo_sampling* s, int32_t* tok_out,
                      float* logp_out, const grpo_trace* trace, void* ws, size_t ws_bytes,
                      void* stream) {
  return rollout(m, kv, n_seqs, max_len, B, seq_ids, pos, tok, max_pos, step0, n_steps, s,
                 tok_out, logp_out, trace, 0, 0, ws, ws_bytes, stream);
}

int grpo_rollout_step_grouped(const grpo_model* m, void* kv, int32_t n_seqs, int32_t max_len,
                              int32_t B, int32_t G, int32_t prefix_len, const int32_t* seq_ids,
                              int32_t* pos, int32_t* tok, int32_t max_pos, int32_t step0,
                              int32_t n_steps, const grpo_sampling* s, int32_t* tok_out,
                              float* logp_out, const grpo_trace* trace, void* ws,
                              size_t ws_bytes, void* stream) {
  if (!m) return fail(GRPO_INVALID_ARG, "model is NULL");
  if (G < 1 || B < 1 || B % G)
    return fail(GRPO_INVALID_ARG, "G %d must be >= 1 and divide B %d", G, B);
  if (prefix_len < 0 || prefix_len > max_len)
    return fail(GRPO_INVALID_ARG, "prefix_len %d outside [0, max_len %d]", prefix_len, max_len);
  return rollout(m, kv, n_seqs, max_len, B, seq_ids, pos, tok, max_pos, step0, n_steps, s,
                 tok_out, logp_out, trace, G, prefix_len, ws, ws_bytes, stream);
}

int grpo_score_sequences(const grpo_model* m, const int32_t* tokens, int32_t N, int32_t T,
                         int32_t score_from, float temperature, float* logp_out,
                         const grpo_trace* trace_out, void* ws, size_t ws_bytes, void* stream) {
  if (!m) return fail(GRPO_INVALID_ARG, "model is NULL");
  const grpo_config& c = m->cfg;
  if (!tokens || !logp_out || !ws) return fail(GRPO_INVALID_ARG, "tokens, logp_out and ws must be set");
  if (N < 1 || T < 2) return fail(GRPO_INVALID_ARG, "N must be >= 1 and T >= 2");
  if (score_from < 1 || score_from >= T)
    return fail(GRPO_INVALID_ARG, "score_from %d outside [1, T)", score_from);
  if (!(temperature >= 0.f) || temperature == INFINITY)
    return fail(GRPO_INVALID_ARG, "temperature must be finite and >= 0");
  if (c.dtype == GRPO_F32 && T > 16384) return fail(GRPO_UNSUPPORTED, "fp32 sequences above 16384");
  if ((long)T > kScoreTokens) return fail(GRPO_UNSUPPORTED, "T above %d", kScoreTokens);
  const size_t need = grpo_workspace_bytes(m, GRPO_OP_SCORE, N, T);
  if (ws_bytes < need)
    return fail(GRPO_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes, need);
  hipStream_t st = (hipStream_t)stream;
  Bump b(ws);
  ScoreWS w = take_score(b, c, N, T);
  const int d = c.d_model, Ts = T - score_from;
  const Partials none{nullptr, 0, 0, d};
  for (int n0 = 0; n0 < N; n0 += w.chunk) {
    const int C = std::min(w.chunk, N - n0);
    const int M = C * T;
    const int32_t* tk = tokens + (size_t)n0 * T;
    HIPCHK(embed(c.dtype, m->tok_emb, tk, M, d, c.vocab, w.s.x, st));
    if (int rc = forward_rows(m, w.s, M, T, 1, C, T, nullptr, w.kbuf,
                              c.dtype == GRPO_F32 ? w.vbuf : nullptr, w.vt, trace_out,
                              (size_t)N * T, TraceMap::rows(n0 * T), st))
      return rc;
    const int R = C * Ts, step = head_step(w, R);
    for (int i0 = 0; i0 < R; i0 += step) {
      const int rc_rows = std::min(step, R - i0);
      HIPCHK(rmsnorm(c.dtype, w.s.x, d, RowMap{i0, Ts, T, score_from - 1}, none, m->final_norm,
                     rc_rows, d, c.rms_eps, w.hs, d, st));
      if (int rc = score_head(m, w, rc_rows, tk, T, score_from, Ts, i0, temperature,
                              logp_out + (size_t)n0 * Ts + i0, trace_out, (size_t)N * Ts,
                              n0 * Ts + i0, st))
        return rc;
    }
  }
  g_err.clear();
  return GRPO_OK;
}

int grpo_score_sequences_grouped(const grpo_model* m, const int32_t* tokens, int32_t N,
                                 int32_t T, int32_t score_from, float temperature, int32_t G,
                                 int32_t prefix_len, float* logp_out, const grpo_trace* trace_out,
                                 void* ws, size_t ws_bytes, void* stream) {
  if (!m) return fail(GRPO_INVALID_ARG, "model is NULL");
  if (G < 1 || N < 1 || N % G) return fail(GRPO_INVALID_ARG, "G %d must be >= 1 and divide N %d", G, N);
  if (prefix_len < 0 || prefix_len > score_from)
    return fail(GRPO_INVALID_ARG, "prefix_len %d outside [0, score_from %d]", prefix_len, score_from);
  const grpo_config& c = m->cfg;
  // every sequence's own rows start at the multiple of 32 at or below the last
  // shared position (its K/V recomputed per sequence: the same values)
  const int P0 = prefix_len > 0 ? (prefix_len - 1) / 32 * 32 : 0;
  const int chunk_seqs = std::max(1, std::min(N, kScoreTokens / std::max(T, 1)));
  const int C = chunk_seqs / G * G;
  if (c.dtype == GRPO_F32 || G == 1 || P0 == 0 || C == 0 || score_from < 1 || score_from >= T)
    return grpo_score_sequences(m, tokens, N, T, score_from, temperature, logp_out, trace_out,
                                ws, ws_bytes, stream);
  if (!tokens || !logp_out || !ws) return fail(GRPO_INVALID_ARG, "tokens, logp_out and ws must be set");
  if (!(temperature >= 0.f) || temperature == INFINITY)
    return fail(GRPO_INVALID_ARG, "temperature must be finite and >= 0");
  if ((long)T > kScoreTokens) return fail(GRPO_UNSUPPORTED, "T above %d", kScoreTokens);
  const size_t need = grpo_workspace_bytes(m, GRPO_OP_SCORE, N, T);
  if (ws_bytes < need)
    return fail(GRPO_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes, need);
  hipStream_t st = (hipStream_t)stream;
  Bump b(ws);
  ScoreWS w = take_score(b, c, N, T);
  const int d = c.d_model, qd = qdim(c), kvd = kvdim(c), f = c.d_ffn, Ts = T - score_from;
  const int Tb = T - 1 - P0;          // own rows per sequence: positions P0 .. T - 2
  const int ldqkv = qd + 2 * kvd, es = esize(c);
  const Partials none{nullptr, 0, 0, d};
  HIPCHK(rope_table(nullptr, T, c.head_dim, c.rope_theta, w.s.cs, st));
  for (int n0 = 0; n0 < N; n0 += C) {
    const int Cc = std::min(C, N - n0), Pc = Cc / G;
    // rows: the Pc groups' shared positions 0 .. prefix_len - 1 once each, then
    // every sequence's own rows
    const int M1 = Pc * prefix_len, M = M1 + Cc * Tb;
    const int32_t* tk = tokens + (size_t)n0 * T;
    for (int p = 0; p < Pc; ++p)
      HIPCHK(embed(c.dtype, m->tok_emb, tk + (size_t)p * G * T, prefix_len, d, c.vocab,
                   w.s.x + (size_t)p * prefix_len * d, st));
    for (int n = 0; n < Cc; ++n)
      HIPCHK(embed(c.dtype, m->tok_emb, tk + (size_t)n * T + P0, Tb, d, c.vocab,
                   w.s.x + ((size_t)M1 + (size_t)n * Tb) * d, st));
    char* q1 = (char*)w.s.q + (size_t)M1 * qd * es;
    char* o1 = (char*)w.s.o + (size_t)M1 * qd * es;
    int rc;
    // trace rows: each shared row to all G members' rows, own rows from P0
    const size_t RT = (size_t)N * T;
    const TraceMap tm_shared{prefix_len, G * T, n0 * T, G, T};
    const TraceMap tm_own{Tb, T, n0 * T + P0, 1, 0};
    auto tr2 = [&](float* member, int l, int width, const void* src, int layout, int ld,
                   int ebytes) -> int {
      if (int r = trace(member, l, RT, width, src, layout, ld, M1, tm_shared, st)) return r;
      return trace(member, l, RT, width, (const char*)src + (size_t)M1 * ld * ebytes, layout, ld,
                   Cc * Tb, tm_own, st);
    };
    const int act = c.dtype == GRPO_F32 ? TR_F32 : TR_BF16;
    for (int l = 0; l < c.n_layers; ++l) {
      HIPCHK(rmsnorm(c.dtype, w.s.x, d, RowMap::identity(), none, m->attn_norm[l], M, d,
                     c.rms_eps, w.s.h, d, st));
      if ((rc = tr2(TRM(trace_out, x), l, d, w.s.x, TR_F32, d, 4)) ||
          (rc = tr2(TRM(trace_out, h_attn), l, d, w.s.h, act, d, es)))
        return rc;
      if ((rc = gemm_rows(m, w.s.h, d, M, qkv_stack(m, l), ldqkv, d, EPI_STORE,
                          EpiArgs{w.s.qkv, nullptr, ldqkv}, st)))
        return rc;
      // shared rows: K and V^T into all G slots of the group; own rows from P0
      RopeArgs ra{};
      ra.mode = 1; ra.T = prefix_len; ra.G = G; ra.pos_arr = nullptr;
      ra.n_heads = c.n_heads; ra.n_kv = c.n_kv_heads; ra.hd = c.head_dim; ra.theta = c.rope_theta;
      ra.kcache = w.kbuf; ra.vcache = nullptr; ra.n_seqs = Cc; ra.max_len = T;
      ra.vt = w.vt; ra.vt_len = round8(T); ra.vt_G = G;
      ra.splits = 1; ra.split_stride = 0; ra.cs = w.s.cs; ra.pos0 = 0;
      if (trace_out) {
        const grpo_trace* t = trace_out;
        ra.tq = t->q ? t->q + (size_t)l * RT * qd : nullptr;
        ra.tk = t->k ? t->k + (size_t)l * RT * kvd : nullptr;
        ra.tv = t->v ? t->v + (size_t)l * RT * kvd : nullptr;
        ra.tmap = tm_shared;
      }
      HIPCHK(rope_kv(c.dtype, w.s.qkv, M1, w.s.q, ra, st));
      RopeArgs rb = ra;
      rb.T = Tb; rb.G = 1; rb.vt_G = 1; rb.pos0 = P0; rb.tmap = tm_own;
      HIPCHK(rope_kv(c.dtype, w.s.qkv + (size_t)M1 * ldqkv, Cc * Tb, q1, rb, st));
      HIPCHK(attn_prefill(c.dtype, w.s.q, w.kbuf, w.vt, Pc, prefix_len, c.n_heads, c.n_kv_heads,
                          c.head_dim, T, G, w.s.o, st, 0, G, round8(T)));
      HIPCHK(attn_prefill(c.dtype, q1, w.kbuf, w.vt, Cc, Tb, c.n_heads, c.n_kv_heads,
                          c.head_dim, T, 1, o1, st, P0, 1, round8(T)));
      if ((rc = tr2(TRM(trace_out, o), l, qd, w.s.o, act, qd, es))) return rc;
      if ((rc = gemm_rows(m, w.s.o, qd, M, one(m->wo[l]), d, qd, EPI_RESID,
                          EpiArgs{w.s.x, nullptr, d}, st)))
        return rc;
      HIPCHK(rmsnorm(c.dtype, w.s.x, d, RowMap::identity(), none, m->mlp_norm[l], M, d,
                     c.rms_eps, w.s.h, d, st));
      if ((rc = tr2(TRM(trace_out, x_attn), l, d, w.s.x, TR_F32, d, 4)) ||
          (rc = tr2(TRM(trace_out, h_mlp), l, d, w.s.h, act, d, es)))
        return rc;
      if ((rc = gemm_rows(m, w.s.h, d, M, gate_up(m, l), f, d, EPI_SWIGLU,
                          EpiArgs{nullptr, w.s.a, f}, st)))
        return rc;
      if ((rc = tr2(TRM(trace_out, act), l, f, w.s.a, act, f, es))) return rc;
      if ((rc = gemm_rows(m, w.s.a, f, M, one(m->w_down[l]), d, f, EPI_RESID,
                          EpiArgs{w.s.x, nullptr, d}, st)))
        return rc;
    }
    if ((rc = tr2(TRM(trace_out, x), c.n_layers, d, w.s.x, TR_F32, d, 4))) return rc;
    // logits of positions score_from - 1 .. T - 2: own rows of each sequence
    const int R = Cc * Ts, step = head_step(w, R);
    for (int i0 = 0; i0 < R; i0 += step) {
      const int rc_rows = std::min(step, R - i0);
      HIPCHK(rmsnorm(c.dtype, w.s.x, d, RowMap{i0, Ts, Tb, M1 + score_from - 1 - P0}, none,
                     m->final_norm, rc_rows, d, c.rms_eps, w.hs, d, st));
      if ((rc = score_head(m, w, rc_rows, tk, T, score_from, Ts, i0, temperature,
                           logp_out + (size_t)n0 * Ts + i0, trace_out, (size_t)N * Ts,
                           n0 * Ts + i0, st)))
        return rc;
    }
  }
  g_err.clear();
  return GRPO_OK;
}

int grpo_extend(const grpo_model* m, void* kv, int32_t n_seqs, int32_t max_len, int32_t B,
                const int32_t* seq_ids, const int32_t* pos0, const int32_t* tokens, int32_t Te,
                int32_t step, const grpo_sampling* s, int32_t* tok_out, float* logp_out,
                const grpo_trace* trace_out, void* ws, size_t ws_bytes, void* stream) {
  if (!m) return fail(GRPO_INVALID_ARG, "model is NULL");
  const grpo_config& c = m->cfg;
  if (!kv || !pos0 || !tokens || !tok_out || !logp_out || !ws)
    return fail(GRPO_INVALID_ARG, "kv, pos0, tokens, tok_out, logp_out and ws must be set");
  if (B < 1 || max_len < 1 || step < 0) return fail(GRPO_INVALID_ARG, "B, max_len >= 1, step >= 0");
  if (Te < 1 || Te > kExtendChunk)
    return fail(GRPO_INVALID_ARG, "span length %d outside [1, %d]: inject longer spans in chunks",
                Te, kExtendChunk);
  if (!seq_ids && B > n_seqs) return fail(GRPO_INVALID_ARG, "B %d exceeds n_seqs %d", B, n_seqs);
  if (c.dtype == GRPO_F32 && max_len > 16384) return fail(GRPO_UNSUPPORTED, "fp32 caches above 16384");
  if (int rc = check_sampling(s, c.vocab)) return rc;
  std::vector<int32_t> ids(B);
  for (int b = 0; b < B; ++b) ids[b] = seq_ids ? seq_ids[b] : b;
  {
    std::vector<int32_t> sorted(ids);
    for (int b = 0; b < B; ++b)
      if (sorted[b] < 0 || sorted[b] >= n_seqs)
        return fail(GRPO_INVALID_ARG, "seq_ids[%d] = %d outside [0, n_seqs %d)", b, sorted[b], n_seqs);
    std::sort(sorted.begin(), sorted.end());
    for (int b = 1; b < B; ++b)
      if (sorted[b] == sorted[b - 1]) return fail(GRPO_INVALID_ARG, "seq_ids repeats sequence %d", sorted[b]);
  }
  for (int b = 0; b < B; ++b) {
    if (pos0[b] < 0) return fail(GRPO_INVALID_ARG, "pos0[%d] = %d is negative", b, pos0[b]);
    if ((long)pos0[b] + Te > max_len)
      return fail(GRPO_KV_CAPACITY, "pos0[%d] %d + span %d exceeds max_len %d", b, pos0[b], Te,
                  max_len);
  }
  const size_t need = grpo_workspace_bytes(m, GRPO_OP_EXTEND, B, max_len);
  if (ws_bytes < need)
    return fail(GRPO_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes, need);
  hipStream_t st = (hipStream_t)stream;
  Bump bump(ws);
  ExtendWS w = take_extend(bump, c, B, max_len);
  const int d = c.d_model, qd = qdim(c), kvd = kvdim(c), f = c.d_ffn, M = B * Te;
  const Partials none{nullptr, 0, 0, d};
  const int act = c.dtype == GRPO_F32 ? TR_F32 : TR_BF16;
  const TraceMap rows = TraceMap::rows();
  const grpo_trace* tr = trace_out;
  int rc;
  HIPCHK(set_i32(w.slots, ids.data(), B, st));
  HIPCHK(set_i32(w.pos0, pos0, B, st));
  if (c.dtype == GRPO_F32) HIPCHK(row_positions(w.pos0, w.slots, B, Te, w.row_pos, w.row_slot, st));
  HIPCHK(embed(c.dtype, m->tok_emb, tokens, M, d, c.vocab, w.s.x, st));
  HIPCHK(rope_table(nullptr, max_len, c.head_dim, c.rope_theta, w.s.cs, st));
  const int vt_len = round8(max_len);
  for (int l = 0; l < c.n_layers; ++l) {
    Layer L = kv_layer(m, kv, l, n_seqs, max_len);
    HIPCHK(rmsnorm(c.dtype, w.s.x, d, RowMap::identity(), none, m->attn_norm[l], M, d, c.rms_eps,
                   w.s.h, d, st));
    if ((rc = trace(TRM(tr, x), l, M, d, w.s.x, TR_F32, d, M, rows, st)) ||
        (rc = trace(TRM(tr, h_attn), l, M, d, w.s.h, act, d, M, rows, st)))
      return rc;
    if ((rc = gemm_rows(m, w.s.h, d, M, qkv_stack(m, l), qd + 2 * kvd, d, EPI_STORE,
                        EpiArgs{w.s.qkv, nullptr, qd + 2 * kvd}, st)))
      return rc;
    // the span's K/V into each sequence's slot at pos0[b] + t
    RopeArgs ra{};
    ra.mode = 1; ra.T = Te; ra.G = 1; ra.pos_arr = w.pos0; ra.slots = w.slots;
    ra.n_heads = c.n_heads; ra.n_kv = c.n_kv_heads; ra.hd = c.head_dim; ra.theta = c.rope_theta;
    ra.kcache = L.k; ra.vcache = L.v; ra.n_seqs = n_seqs; ra.max_len = max_len;
    ra.vt = nullptr; ra.vt_len = 0; ra.splits = 1; ra.split_stride = 0; ra.cs = w.s.cs;
    if (tr) {
      ra.tq = tr->q ? tr->q + (size_t)l * M * qd : nullptr;
      ra.tk = tr->k ? tr->k + (size_t)l * M * kvd : nullptr;
      ra.tv = tr->v ? tr->v + (size_t)l * M * kvd : nullptr;
      ra.tmap = rows;
    }
    HIPCHK(rope_kv(c.dtype, w.s.qkv, M, w.s.q, ra, st));
    // causal attention of the span rows over each sequence's cache 0 .. pos0[b] + t
    if (c.dtype == GRPO_F32) {
      HIPCHK(attn_rows_f32((const float*)w.s.q, (const float*)L.k, (const float*)L.v, w.row_pos,
                           w.row_slot, M, 1, 1, c.n_heads, c.n_kv_heads, c.head_dim, max_len,
                           (float*)w.s.o, st));
    } else {
      HIPCHK(cache_vt(L.v, w.slots, w.pos0, B, Te, c.n_kv_heads, max_len, c.head_dim, vt_len,
                      w.vt, st));
      HIPCHK(attn_prefill(c.dtype, w.s.q, L.k, w.vt, B, Te, c.n_heads, c.n_kv_heads, c.head_dim,
                          max_len, 1, w.s.o, st, 0, 1, vt_len, w.pos0, w.slots));
    }
    if ((rc = trace(TRM(tr, o), l, M, qd, w.s.o, act, qd, M, rows, st))) return rc;
    if ((rc = gemm_rows(m, w.s.o, qd, M, one(m->wo[l]), d, qd, EPI_RESID,
                        EpiArgs{w.s.x, nullptr, d}, st)))
      return rc;
    HIPCHK(rmsnorm(c.dtype, w.s.x, d, RowMap::identity(), none, m->mlp_norm[l], M, d, c.rms_eps,
                   w.s.h, d, st));
    if ((rc = trace(TRM(tr, x_attn), l, M, d, w.s.x, TR_F32, d, M, rows, st)) ||
        (rc = trace(TRM(tr, h_mlp), l, M, d, w.s.h, act, d, M, rows, st)))
      return rc;
    if ((rc = gemm_rows(m, w.s.h, d, M, gate_up(m, l), f, d, EPI_SWIGLU,
                        EpiArgs{nullptr, w.s.a, f}, st)))
      return rc;
    if ((rc = trace(TRM(tr, act), l, M, f, w.s.a, act, f, M, rows, st))) return rc;
    if ((rc = gemm_rows(m, w.s.a, f, M, one(m->w_down[l]), d, f, EPI_RESID,
                        EpiArgs{w.s.x, nullptr, d}, st)))
      return rc;
  }
  if ((rc = trace(TRM(tr, x), c.n_layers, M, d, w.s.x, TR_F32, d, M, rows, st))) return rc;
  // the next token of each sequence, from the span's last row
  HIPCHK(rmsnorm(c.dtype, w.s.x, d, RowMap{0, 1, Te, Te - 1}, none, m->final_norm, B, d, c.rms_eps,
                 w.hl, d, st));
  if ((rc = gemm_rows(m, w.hl, d, B, one(m->lm_head), c.vocab, d, EPI_STORE,
                      EpiArgs{w.logits, nullptr, c.vocab}, st)))
    return rc;
  if ((rc = trace(TRM(tr, h_final), 0, B, d, w.hl, act, d, B, rows, st)) ||
      (rc = trace(TRM(tr, logits), 0, B, c.vocab, w.logits, TR_F32, c.vocab, B, rows, st)))
    return rc;
  SampleArgs sa{};
  sa.temperature = s->temperature; sa.top_k = s->top_k; sa.seed = s->seed; sa.step = step;
  sa.G = 1; sa.tok_out = tok_out; sa.logp_out = logp_out; sa.out_stride = 1;
  sa.seq_ids = w.slots;
  HIPCHK(sample(w.logits, B, c.vocab, c.vocab, sa, st));
  g_err.clear();
  return GRPO_OK;
}

int grpo_advantages(const float* rewards, int32_t P, int32_t G, float eps, float* adv_out,
                    void* stream) {
  if (!rewards || !adv_out) return fail(GRPO_INVALID_ARG, "rewards and adv_out must be set");
  if (P < 1) return fail(GRPO_INVALID_ARG, "P must be >= 1");
  if (G < 2) return fail(GRPO_INVALID_ARG, "a group needs G >= 2 samples");
  if (!(eps >= 0.f)) return fail(GRPO_INVALID_ARG, "eps must be >= 0");
  HIPCHK(advantages(rewards, P, G, eps, adv_out, (hipStream_t)stream));
  g_err.clear();
  return GRPO_OK;
}

int grpo_reward(const uint8_t* correct, const double* t_base, const double* t,
                const int32_t* tools_used, const int32_t* tools_avail, int32_t n, float* r_out) {
  if (!correct || !t_base || !t || !tools_used || !tools_avail || !r_out)
    return fail(GRPO_INVALID_ARG, "every array must be set");
  if (n < 1) return fail(GRPO_INVALID_ARG, "n must be >= 1");
  for (int i = 0; i < n; ++i) {
    if (!(t_base[i] > 0.0) || !(t[i] > 0.0) || t_base[i] == INFINITY || t[i] == INFINITY)
      return fail(GRPO_INVALID_ARG, "times of entry %d must be positive and finite", i);
    if (tools_avail[i] < 1 || tools_used[i] < 0 || tools_used[i] > tools_avail[i])
      return fail(GRPO_INVALID_ARG, "entry %d: need 0 <= tools_used <= tools_avail, avail >= 1", i);
  }
  for (int i = 0; i < n; ++i) {
    double perf;
    if (!correct[i]) perf = -2.0;
    else if (t[i] > t_base[i]) perf = -1.0;
    else perf = std::min(10.0, t_base[i] / t[i] - 1.0);
    r_out[i] = (float)(perf + 0.5 * (double)tools_used[i] / (double)tools_avail[i]);
  }
  g_err.clear();
  return GRPO_OK;
}

int grpo_sft_loss(const float* logp, const uint8_t* mask, int32_t N, int32_t Tr, int32_t agg,
                  float* loss_out, float* dloss_dlogp, void* ws, size_t ws_bytes, void* stream) {
  if (!logp || !mask || !loss_out || !ws)
    return fail(GRPO_INVALID_ARG, "logp, mask, loss_out and ws must be set");
  if (N < 1 || Tr < 1) return fail(GRPO_INVALID_ARG, "N and Tr must be >= 1");
  if (agg != 0 && agg != 1) return fail(GRPO_INVALID_ARG, "agg must be 0 or 1");
  const size_t need = grpo_workspace_bytes(nullptr, GRPO_OP_LOSS, N, Tr);
  if (ws_bytes < need)
    return fail(GRPO_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes, need);
  HIPCHK(sft_loss(logp, mask, N, Tr, agg, loss_out, dloss_dlogp, (double*)ws,
                  (hipStream_t)stream));
  g_err.clear();
  return GRPO_OK;
}

int grpo_exact_kl(const float* logits, const float* logits_ref, int32_t R, int32_t V, int32_t ld,
                  float temperature, float* kl_out, void* stream) {
  if (!logits || !logits_ref || !kl_out)
    return fail(GRPO_INVALID_ARG, "logits, logits_ref and kl_out must be set");
  if (R < 1 || V < 1 || ld < V) return fail(GRPO_INVALID_ARG, "need R, V >= 1 and ld >= V");
  if (!(temperature >= 0.f) || temperature == INFINITY)
    return fail(GRPO_INVALID_ARG, "temperature must be finite and >= 0");
  HIPCHK(exact_kl(logits, logits_ref, R, V, ld, temperature, kl_out, (hipStream_t)stream));
  g_err.clear();
  return GRPO_OK;
}

int grpo_token_loss(const float* logp, const float* logp_old, const float* logp_ref,
                    const uint8_t* mask, const float* adv, int32_t N, int32_t Tr, float clip_eps,
                    float beta, int32_t agg, float* loss_out, float* tok_loss, float* dloss_dlogp,
                    float* stats, void* ws, size_t ws_bytes, void* stream) {
  if (!logp || !logp_old || !logp_ref || !mask || !adv || !loss_out || !ws)
    return fail(GRPO_INVALID_ARG, "logp, logp_old, logp_ref, mask, adv, loss_out, ws must be set");
  if (N < 1 || Tr < 1) return fail(GRPO_INVALID_ARG, "N and Tr must be >= 1");
  if (!(clip_eps >= 0.f && clip_eps < 1.f)) return fail(GRPO_INVALID_ARG, "clip_eps outside [0, 1)");
  if (!(beta >= 0.f)) return fail(GRPO_INVALID_ARG, "beta must be >= 0");
  if (agg != 0 && agg != 1) return fail(GRPO_INVALID_ARG, "agg must be 0 or 1");
  const size_t need = grpo_workspace_bytes(nullptr, GRPO_OP_LOSS, N, Tr);
  if (ws_bytes < need)
    return fail(GRPO_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes, need);
  HIPCHK(token_loss(logp, logp_old, logp_ref, mask, adv, N, Tr, clip_eps, beta, agg, loss_out,
                    tok_loss, dloss_dlogp, stats, (double*)ws, (hipStream_t)stream));
  g_err.clear();
  return GRPO_OK;
}

int grpo_policy_backward(const grpo_model* m, const int32_t* tokens, int32_t N, int32_t T,
                         int32_t score_from, float temperature, const float* dlogp,
                         const grpo_grads* g, void* ws, size_t ws_bytes, void* stream) {
  if (!m) return fail(GRPO_INVALID_ARG, "model is NULL");
  const grpo_config& c = m->cfg;
  if (!tokens || !dlogp || !g || !ws) return fail(GRPO_INVALID_ARG, "tokens, dlogp, g and ws must be set");
  if (N < 1 || T < 2) return fail(GRPO_INVALID_ARG, "N must be >= 1 and T >= 2");
  if (score_from < 1 || score_from >= T)
    return fail(GRPO_INVALID_ARG, "score_from %d outside [1, T)", score_from);
  if (!(temperature >= 0.f) || temperature == INFINITY)
    return fail(GRPO_INVALID_ARG, "temperature must be finite and >= 0");
  if (T > kBackwardTokens) return fail(GRPO_UNSUPPORTED, "T above %d", kBackwardTokens);
  if (c.n_heads % c.n_kv_heads) return fail(GRPO_UNSUPPORTED, "n_heads not a multiple of n_kv_heads");
  if (!g->tok_emb || !g->final_norm || !g->lm_head || !g->attn_norm || !g->wq || !g->wk ||
      !g->wv || !g->wo || !g->mlp_norm || !g->w_gate || !g->w_up || !g->w_down)
    return fail(GRPO_INVALID_ARG, "every gradient buffer must be set");
  for (int l = 0; l < c.n_layers; ++l)
    if (!g->attn_norm[l] || !g->wq[l] || !g->wk[l] || !g->wv[l] || !g->wo[l] || !g->mlp_norm[l] ||
        !g->w_gate[l] || !g->w_up[l] || !g->w_down[l])
      return fail(GRPO_INVALID_ARG, "gradient buffers of layer %d must be set", l);
  const size_t need = grpo_workspace_bytes(m, GRPO_OP_BACKWARD, N, T);
  if (ws_bytes < need)
    return fail(GRPO_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes, need);
  hipStream_t st = (hipStream_t)stream;
  Bump b(ws);
  BackwardWS w = take_backward(b, c, T);
  const int d = c.d_model, qd = qdim(c), kvd = kvdim(c), f = c.d_ffn, ldqkv = qd + 2 * kvd;
  const int V = c.vocab, L = c.n_layers, Ts = T - score_from, Tp = w.Tp, es = esize(c);
  const int e = c.dtype == GRPO_F32 ? 0 : 1;
  const Partials none{nullptr, 0, 0, d};
  int rc;
  // transposed weights, once per call: the data gradients' W operands
  for (int l = 0; l < L; ++l) {
    HIPCHK(transpose_w(c, m->w_down[l], d, f, w.WdT[l], d, st));
    HIPCHK(transpose_w(c, m->w_gate[l], f, d, w.WguT[l], 2 * f, st));
    HIPCHK(transpose_w(c, m->w_up[l], f, d, (char*)w.WguT[l] + (size_t)f * es, 2 * f, st));
    HIPCHK(transpose_w(c, m->wo[l], d, qd, w.WoT[l], d, st));
    HIPCHK(transpose_w(c, m->wq[l], qd, d, w.WqkvT[l], ldqkv, st));
    HIPCHK(transpose_w(c, m->wk[l], kvd, d, (char*)w.WqkvT[l] + (size_t)qd * es, ldqkv, st));
    HIPCHK(transpose_w(c, m->wv[l], kvd, d, (char*)w.WqkvT[l] + (size_t)(qd + kvd) * es, ldqkv, st));
  }
  HIPCHK(transpose_w(c, m->lm_head, V, d, w.WheadT, V, st));
  HIPCHK(rope_table(nullptr, T, c.head_dim, c.rope_theta, w.cs, st));
  const size_t Td = (size_t)T * d;
  for (int n = 0; n < N; ++n) {
    const int32_t* tk = tokens + (size_t)n * T;
    const float* gn = dlogp + (size_t)n * Ts;
    // forward, keeping every layer's input
    HIPCHK(embed(c.dtype, m->tok_emb, tk, T, d, V, w.X, st));
    for (int l = 0; l < L; ++l)
      if ((rc = layer_fwd(m, w, l, w.X + l * Td, T, w.X + (l + 1) * Td, st))) return rc;
    // head: scored rows score_from - 1 .. T - 2 in chunks
    const float* xL = w.X + L * Td;
    HIPCHK(fill_f32(w.dx, Td, 0.f, st));
    for (int i0 = 0; i0 < Ts; i0 += w.head_rows) {
      const int R = std::min(w.head_rows, Ts - i0), Rp = round64(R), r0 = score_from - 1 + i0;
      HIPCHK(rmsnorm(c.dtype, const_cast<float*>(xL), d, RowMap{r0, 1, 1, 0}, none, m->final_norm,
                     R, d, c.rms_eps, w.hf, d, st));
      if ((rc = gemm_rows(m, w.hf, d, R, one(m->lm_head), V, d, EPI_STORE,
                          EpiArgs{w.z, nullptr, V}, st)))
        return rc;
      HIPCHK(dlogits(c.dtype, w.z, R, V, V, tk + score_from + i0, 1, gn + i0, temperature, w.dz,
                     V, st));
      HIPCHK(transpose(e, e, w.dz, V, 0, R, V, w.dzT, Rp, 0, 0, 1, Rp, 1, st));
      HIPCHK(transpose(e, e, w.hf, d, 0, R, d, w.hfT, Rp, 0, 0, 1, Rp, 1, st));
      if ((rc = gemm_rows(m, w.dzT, Rp, V, one(w.hfT), d, Rp, EPI_RESID,
                          EpiArgs{g->lm_head, nullptr, d}, st)))
        return rc;
      if ((rc = gemm_rows(m, w.dz, V, R, one(w.WheadT), d, V, EPI_STORE,
                          EpiArgs{w.dhf, nullptr, d}, st)))
        return rc;
      HIPCHK(rmsnorm_bwd(c.dtype, xL + (size_t)r0 * d, d, m->final_norm, w.dhf, d, R, d, c.rms_eps,
                         w.dx + (size_t)r0 * d, nullptr, w.rr, w.part, g->final_norm, st));
    }
    // layers in reverse; w.dx holds the gradient of the layer's output
    for (int l = L - 1; l >= 0; --l) {
      const float* x = w.X + l * Td;
      if ((rc = layer_fwd(m, w, l, x, T, nullptr, st))) return rc;
      // down projection: x_out = xa + a Wd^T
      if ((rc = wgrad(m, w, w.dx, 1, d, d, w.a, f, f, T, g->w_down[l], st))) return rc;
      HIPCHK(cast_f32(w.dx, Td, c.dtype, w.dxe, st));
      if ((rc = gemm_rows(m, w.dxe, d, T, one(w.WdT[l]), f, d, EPI_STORE,
                          EpiArgs{w.da, nullptr, f}, st)))
        return rc;
      HIPCHK(swiglu_bwd(c.dtype, w.gu, w.da, T, f, w.dgu, st));
      // gate / up: dgu^T h2 for each half, dh2 = dgu [Wg; Wu]
      HIPCHK(transpose(e, e, w.dgu, 2 * f, 0, T, 2 * f, w.tA, Tp, 0, 0, 1, Tp, 1, st));
      HIPCHK(transpose(e, e, w.h2, d, 0, T, d, w.tB, Tp, 0, 0, 1, Tp, 1, st));
      if (g->w_up[l] == g->w_gate[l] + (size_t)f * d) {   // adjacent: one product
        if ((rc = gemm_rows(m, w.tA, Tp, 2 * f, one(w.tB), d, Tp, EPI_RESID,
                            EpiArgs{g->w_gate[l], nullptr, d}, st)))
          return rc;
      } else if ((rc = gemm_rows(m, w.tA, Tp, f, one(w.tB), d, Tp, EPI_RESID,
                                 EpiArgs{g->w_gate[l], nullptr, d}, st)) ||
                 (rc = gemm_rows(m, (char*)w.tA + (size_t)f * Tp * es, Tp, f, one(w.tB), d, Tp,
                                 EPI_RESID, EpiArgs{g->w_up[l], nullptr, d}, st))) {
        return rc;
      }
      if ((rc = gemm_rows(m, w.dgu, 2 * f, T, one(w.WguT[l]), d, 2 * f, EPI_STORE,
                          EpiArgs{w.dh, nullptr, d}, st)))
        return rc;
      HIPCHK(hipMemcpyAsync(w.dxa, w.dx, Td * 4, hipMemcpyDeviceToDevice, st));
      HIPCHK(rmsnorm_bwd(c.dtype, w.xa, d, m->mlp_norm[l], w.dh, d, T, d, c.rms_eps, w.dxa, w.dxe,
                         w.rr, w.part, g->mlp_norm[l], st));
      // output projection: xa = x + o Wo^T
      if ((rc = wgrad(m, w, w.dxa, 1, d, d, w.o, qd, qd, T, g->wo[l], st))) return rc;
      if ((rc = gemm_rows(m, w.dxe, d, T, one(w.WoT[l]), qd, d, EPI_STORE,
                          EpiArgs{w.dof, nullptr, qd}, st)))
        return rc;
      HIPCHK(cast_f32(w.dof, (size_t)T * qd, c.dtype, w.doe, st));
      if ((rc = attn_bwd(m, w, T, st))) return rc;
      HIPCHK(rope_bwd(c.dtype, w.dqkv, T, c.n_heads + 2 * c.n_kv_heads, c.n_heads + c.n_kv_heads,
                      c.head_dim, w.cs, w.dqkve, st));
      // q, k, v projections: dqkv^T h into the three gradients, dh = dqkv [Wq; Wk; Wv]
      HIPCHK(transpose(e, e, w.dqkve, ldqkv, 0, T, ldqkv, w.tA, Tp, 0, 0, 1, Tp, 1, st));
      HIPCHK(transpose(e, e, w.h, d, 0, T, d, w.tB, Tp, 0, 0, 1, Tp, 1, st));
      if (g->wk[l] == g->wq[l] + (size_t)qd * d && g->wv[l] == g->wk[l] + (size_t)kvd * d) {
        if ((rc = gemm_rows(m, w.tA, Tp, ldqkv, one(w.tB), d, Tp, EPI_RESID,
                            EpiArgs{g->wq[l], nullptr, d}, st)))   // adjacent: one product
          return rc;
      } else if ((rc = gemm_rows(m, w.tA, Tp, qd, one(w.tB), d, Tp, EPI_RESID,
                                 EpiArgs{g->wq[l], nullptr, d}, st)) ||
                 (rc = gemm_rows(m, (char*)w.tA + (size_t)qd * Tp * es, Tp, kvd, one(w.tB), d, Tp,
                                 EPI_RESID, EpiArgs{g->wk[l], nullptr, d}, st)) ||
                 (rc = gemm_rows(m, (char*)w.tA + (size_t)(qd + kvd) * Tp * es, Tp, kvd,
                                 one(w.tB), d, Tp, EPI_RESID, EpiArgs{g->wv[l], nullptr, d}, st))) {
        return rc;
      }
      if ((rc = gemm_rows(m, w.dqkve, ldqkv, T, one(w.WqkvT[l]), d, ldqkv, EPI_STORE,
                          EpiArgs{w.dh, nullptr, d}, st)))
        return rc;
      HIPCHK(rmsnorm_bwd(c.dtype, x, d, m->attn_norm[l], w.dh, d, T, d, c.rms_eps, w.dxa, nullptr,
                         w.rr, w.part, g->attn_norm[l], st));
      std::swap(w.dx, w.dxa);
    }
    HIPCHK(embed_bwd(tk, w.dx, T, d, c.vocab, w.ekeys, g->tok_emb, st));
  }
  g_err.clear();
  return GRPO_OK;
}

int grpo_adamw_step(int32_t dtype, void* param, float* master, float* m1, float* m2,
                    const float* grad, size_t n, const grpo_adamw* hp, int32_t step, void* stream) {
  if (dtype != GRPO_F32 && dtype != GRPO_BF16) return fail(GRPO_INVALID_ARG, "dtype must be 0 or 1");
  if (!param || !m1 || !m2 || !grad || !hp) return fail(GRPO_INVALID_ARG, "param, m, v, grad and hp must be set");
  if (dtype == GRPO_BF16 && !master) return fail(GRPO_INVALID_ARG, "bf16 parameters need an fp32 master copy");
  if (step < 1) return fail(GRPO_INVALID_ARG, "step counts from 1");
  if (!(hp->lr >= 0.f) || !(hp->beta1 >= 0.f && hp->beta1 < 1.f) ||
      !(hp->beta2 >= 0.f && hp->beta2 < 1.f) || !(hp->eps > 0.f) || !(hp->weight_decay >= 0.f))
    return fail(GRPO_INVALID_ARG, "AdamW hyper-parameters out of range");
  HIPCHK(adamw(dtype, param, master, m1, m2, grad, n, hp->lr, hp->beta1, hp->beta2, hp->eps,
               hp->weight_decay, step, (hipStream_t)stream));
  g_err.clear();
  return GRPO_OK;
}

}  // extern "C"

static_assert(GRPO_LOSS_STATIC_ROWS == kLossStaticRows, "static loss scratch size");

extern "C" int grpo_token_loss_noalloc(const float* logp, const float* logp_old,
                                       const float* logp_ref, const uint8_t* mask,
                                       const float* adv, int32_t N, int32_t Tr, float clip_eps,
                                       float beta, int32_t agg, float* loss_out, float* tok_loss,
                                       float* dloss_dlogp, float* stats, void* stream) {
  if (!logp || !logp_old || !logp_ref || !mask || !adv || !loss_out)
    return fail(GRPO_INVALID_ARG, "logp, logp_old, logp_ref, mask, adv and loss_out must be set");
  if (N < 1 || Tr < 1) return fail(GRPO_INVALID_ARG, "N and Tr must be >= 1");
  if (N > kLossStaticRows)
    return fail(GRPO_INVALID_ARG, "N %d exceeds the %d sequences of the static scratch", N,
                kLossStaticRows);
  if (!(clip_eps >= 0.f && clip_eps < 1.f)) return fail(GRPO_INVALID_ARG, "clip_eps outside [0, 1)");
  if (!(beta >= 0.f)) return fail(GRPO_INVALID_ARG, "beta must be >= 0");
  if (agg != 0 && agg != 1) return fail(GRPO_INVALID_ARG, "agg must be 0 or 1");
  double* scr = nullptr;
  HIPCHK(loss_static_scratch(&scr));
  HIPCHK(token_loss(logp, logp_old, logp_ref, mask, adv, N, Tr, clip_eps, beta, agg, loss_out,
                    tok_loss, dloss_dlogp, stats, scr, (hipStream_t)stream));
  g_err.clear();
  return GRPO_OK;
}
