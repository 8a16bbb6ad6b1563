// GRPO group advantages and the clipped-ratio + KL token loss.
//
// Both are microsecond-scale next to rollout and scoring; they run in fp64
// internally so the per-token KL estimator exp(d) - d - 1 (a difference of
// nearly equal numbers when d is small) keeps its relative accuracy, and every
// reduction is a fixed-order tree: per-row sums, then one workgroup over rows.
#include <mutex>
#include <vector>

#include "common.h"
#include "kernels.h"

// Scratch of the allocation-free loss entry point: per sequence 8 partial sums
// and 1 gradient weight (fp64) for up to kLossStaticRows sequences.  Each GPU
// holds its own copy from the library's load until the process ends.  In host
// code the name stands for the host-side shadow, never the device memory:
// kernels get the address from loss_static_scratch().
static __device__ __align__(256) double scratch[(size_t)grpo::kLossStaticRows * 9];

namespace grpo {

namespace {

__global__ void k_advantages(const float* __restrict__ r, int P, int G, float eps,
                             float* __restrict__ adv) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= P) return;
  const float* rg = r + (size_t)p * G;
  double mean = 0.0, mx = -INFINITY, mn = INFINITY;
  for (int i = 0; i < G; ++i) {
    const double v = rg[i];
    mean += v;
    mx = fmax(mx, v);
    mn = fmin(mn, v);
  }
  mean /= G;
  double ss = 0.0;
  for (int i = 0; i < G; ++i) {
    const double dv = (double)rg[i] - mean;
    ss += dv * dv;
  }
  const double sd = sqrt(ss / (G - 1));
  const bool degenerate = (mx == mn);
  for (int i = 0; i < G; ++i)
    adv[(size_t)p * G + i] = degenerate ? 0.f : (float)(((double)rg[i] - mean) / (sd + (double)eps));
}

struct TokTerms {
  double ell, dl, kl, rho;
  bool clip_hit;
};

__device__ __forceinline__ TokTerms tok_terms(float lp, float lo, float lr, float A, float ceps,
                                              float beta) {
  TokTerms t;
  const double rho = exp((double)lp - (double)lo);
  const double a = A;
  const double clipped = fmin(fmax(rho, 1.0 - (double)ceps), 1.0 + (double)ceps);
  const double un = rho * a, cl = clipped * a;
  const bool unclipped = un <= cl;
  const double s = unclipped ? un : cl;
  const double d = (double)lr - (double)lp;
  const double em1 = expm1(d);
  t.kl = em1 - d;
  t.ell = -s + (double)beta * t.kl;
  t.dl = -(unclipped ? un : 0.0) - (double)beta * em1;
  t.rho = rho;
  t.clip_hit = !unclipped;
  return t;
}

// row sums: [sum m*l, count, sum m*kl, clip hits, sum m*rho, non-finite]
__global__ __launch_bounds__(256) void k_loss_rows(const float* lp, const float* lo,
                                                   const float* lr, const uint8_t* mask,
                                                   const float* adv, int Tr, float ceps,
                                                   float beta, float* tok_loss, double* row_ws) {
  __shared__ double sh[6][4];
  const int n = blockIdx.x;
  const float A = adv[n];
  double acc[6] = {0, 0, 0, 0, 0, 0};
  for (int t = threadIdx.x; t < Tr; t += 256) {
    const size_t i = (size_t)n * Tr + t;
    const bool m = mask[i] != 0;
    float out = 0.f;
    if (m) {
      const TokTerms tt = tok_terms(lp[i], lo[i], lr[i], A, ceps, beta);
      acc[0] += tt.ell;
      acc[1] += 1.0;
      acc[2] += tt.kl;
      acc[3] += tt.clip_hit ? 1.0 : 0.0;
      acc[4] += tt.rho;
      acc[5] += isfinite(tt.ell) ? 0.0 : 1.0;
      out = (float)tt.ell;
    }
    if (tok_loss) tok_loss[i] = out;
  }
  const int w = threadIdx.x / 64, l = threadIdx.x % 64;
#pragma unroll
  for (int k = 0; k < 6; ++k) {
    const double v = wave_sum_d(acc[k]);
    if (l == 0) sh[k][w] = v;
  }
  __syncthreads();
  if (threadIdx.x < 6) {
    const int k = threadIdx.x;
    row_ws[(size_t)n * 8 + k] = ((sh[k][0] + sh[k][1]) + sh[k][2]) + sh[k][3];
  }
}

// one workgroup: loss, statistics and the per-row gradient weights
__global__ __launch_bounds__(256) void k_loss_final(const double* row_ws, int N, int agg,
                                                    float* loss, float* stats, double* wts) {
  __shared__ double sh[6][4];
  __shared__ double s_tot[6];
  double acc[6] = {0, 0, 0, 0, 0, 0};
  for (int n = threadIdx.x; n < N; n += 256) {
    const double* r = row_ws + (size_t)n * 8;
    acc[0] += agg == 0 ? r[0] / fmax(1.0, r[1]) : r[0];
    for (int k = 1; k < 6; ++k) acc[k] += r[k];
  }
  const int w = threadIdx.x / 64, l = threadIdx.x % 64;
#pragma unroll
  for (int k = 0; k < 6; ++k) {
    const double v = wave_sum_d(acc[k]);
    if (l == 0) sh[k][w] = v;
  }
  __syncthreads();
  if (threadIdx.x < 6) {
    const int k = threadIdx.x;
    s_tot[k] = ((sh[k][0] + sh[k][1]) + sh[k][2]) + sh[k][3];
  }
  __syncthreads();
  const double ntok = fmax(1.0, s_tot[1]);
  if (threadIdx.x == 0) {
    loss[0] = (float)(agg == 0 ? s_tot[0] / (double)N : s_tot[0] / ntok);
    if (stats) {
      stats[0] = (float)(s_tot[2] / ntok);
      stats[1] = (float)(s_tot[3] / ntok);
      stats[2] = (float)(s_tot[4] / ntok);
      stats[3] = (float)s_tot[5];
    }
  }
  for (int n = threadIdx.x; n < N; n += 256)
    wts[n] = agg == 0 ? 1.0 / ((double)N * fmax(1.0, row_ws[(size_t)n * 8 + 1])) : 1.0 / ntok;
}

__global__ __launch_bounds__(256) void k_loss_grad(const float* lp, const float* lo,
                                                   const float* lr, const uint8_t* mask,
                                                   const float* adv, int Tr, float ceps,
                                                   float beta, const double* wts, float* dl) {
  const int n = blockIdx.x;
  const double w = wts[n];
  const float A = adv[n];
  for (int t = threadIdx.x; t < Tr; t += 256) {
    const size_t i = (size_t)n * Tr + t;
    float g = 0.f;
    if (mask[i]) g = (float)(tok_terms(lp[i], lo[i], lr[i], A, ceps, beta).dl * w);
    dl[i] = g;
  }
}

// distillation loss, row sums: [sum m*logp, count]
__global__ __launch_bounds__(256) void k_sft_rows(const float* lp, const uint8_t* mask, int Tr,
                                                  double* row_ws) {
  __shared__ double sh[2][4];
  const int n = blockIdx.x;
  double acc[2] = {0, 0};
  for (int t = threadIdx.x; t < Tr; t += 256) {
    const size_t i = (size_t)n * Tr + t;
    if (mask[i]) {
      acc[0] += lp[i];
      acc[1] += 1.0;
    }
  }
  const int w = threadIdx.x / 64, l = threadIdx.x % 64;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const double v = wave_sum_d(acc[k]);
    if (l == 0) sh[k][w] = v;
  }
  __syncthreads();
  if (threadIdx.x < 2) {
    const int k = threadIdx.x;
    row_ws[(size_t)n * 2 + k] = ((sh[k][0] + sh[k][1]) + sh[k][2]) + sh[k][3];
  }
}

// one workgroup: the loss and the per-row gradient weights
__global__ __launch_bounds__(256) void k_sft_final(const double* row_ws, int N, int agg,
                                                   float* loss, double* wts) {
  __shared__ double sh[2][4];
  __shared__ double s_tot[2];
  double acc[2] = {0, 0};
  for (int n = threadIdx.x; n < N; n += 256) {
    const double* r = row_ws + (size_t)n * 2;
    acc[0] += agg == 0 ? r[0] / fmax(1.0, r[1]) : r[0];
    acc[1] += r[1];
  }
  const int w = threadIdx.x / 64, l = threadIdx.x % 64;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const double v = wave_sum_d(acc[k]);
    if (l == 0) sh[k][w] = v;
  }
  __syncthreads();
  if (threadIdx.x < 2) {
    const int k = threadIdx.x;
    s_tot[k] = ((sh[k][0] + sh[k][1]) + sh[k][2]) + sh[k][3];
  }
  __syncthreads();
  const double ntok = fmax(1.0, s_tot[1]);
  if (threadIdx.x == 0) loss[0] = (float)(agg == 0 ? -s_tot[0] / (double)N : -s_tot[0] / ntok);
  for (int n = threadIdx.x; n < N; n += 256)
    wts[n] = agg == 0 ? 1.0 / ((double)N * fmax(1.0, row_ws[(size_t)n * 2 + 1])) : 1.0 / ntok;
}

__global__ __launch_bounds__(256) void k_sft_grad(const uint8_t* mask, int Tr, const double* wts,
                                                  float* dl) {
  const int n = blockIdx.x;
  const float g = (float)(-wts[n]);
  for (int t = threadIdx.x; t < Tr; t += 256) {
    const size_t i = (size_t)n * Tr + t;
    dl[i] = mask[i] ? g : 0.f;
  }
}

// Exact KL(softmax(a) || softmax(b)) of one row, a = z / T, b = z_ref / T, in fp64:
// KL = sum e^(a - ma) (a - b) / Sa - (ma + ln Sa) + (mb + ln Sb).
__global__ __launch_bounds__(256) void k_exact_kl(const float* z, const float* zr, int V, int ld,
                                                  double inv_t, float* kl) {
  __shared__ double sh[4];
  const int r = blockIdx.x;
  const float* a = z + (size_t)r * ld;
  const float* b = zr + (size_t)r * ld;
  double ma = -INFINITY, mb = -INFINITY;
  for (int i = threadIdx.x; i < V; i += 256) {
    ma = fmax(ma, (double)a[i] * inv_t);
    mb = fmax(mb, (double)b[i] * inv_t);
  }
  auto bmax = [&](double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
    __syncthreads();
    if (threadIdx.x % 64 == 0) sh[threadIdx.x / 64] = v;
    __syncthreads();
    return fmax(fmax(sh[0], sh[1]), fmax(sh[2], sh[3]));
  };
  auto bsum = [&](double v) {
    v = wave_sum_d(v);
    __syncthreads();
    if (threadIdx.x % 64 == 0) sh[threadIdx.x / 64] = v;
    __syncthreads();
    return ((sh[0] + sh[1]) + sh[2]) + sh[3];
  };
  ma = bmax(ma);
  mb = bmax(mb);
  double sa = 0.0, sb = 0.0, d = 0.0;
  for (int i = threadIdx.x; i < V; i += 256) {
    const double ai = (double)a[i] * inv_t, bi = (double)b[i] * inv_t;
    const double ea = exp(ai - ma);
    sa += ea;
    sb += exp(bi - mb);
    d += ea * (ai - bi);
  }
  sa = bsum(sa);
  sb = bsum(sb);
  d = bsum(d);
  if (threadIdx.x == 0) kl[r] = (float)(d / sa - (ma + log(sa)) + (mb + log(sb)));
}

}  // namespace

hipError_t sft_loss(const float* lp, const uint8_t* mask, int N, int Tr, int agg, float* loss,
                    float* dl, double* row_ws, hipStream_t st) {
  if (N <= 0) return hipSuccess;
  double* wts = row_ws + (size_t)N * 2;
  Prof pf("sft_loss", st);
  k_sft_rows<<<N, 256, 0, st>>>(lp, mask, Tr, row_ws);
  k_sft_final<<<1, 256, 0, st>>>(row_ws, N, agg, loss, wts);
  if (dl) k_sft_grad<<<N, 256, 0, st>>>(mask, Tr, wts, dl);
  return hipGetLastError();
}

hipError_t exact_kl(const float* z, const float* zr, int R, int V, int ld, float temperature,
                    float* kl, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  const double inv_t = 1.0 / (double)(temperature > 0.f ? temperature : 1.f);
  Prof pf("exact_kl", st);
  k_exact_kl<<<R, 256, 0, st>>>(z, zr, V, ld, inv_t, kl);
  return hipGetLastError();
}

hipError_t advantages(const float* r, int P, int G, float eps, float* adv, hipStream_t st) {
  if (P <= 0) return hipSuccess;
  Prof pf("advantages", st);
  k_advantages<<<(P + 63) / 64, 64, 0, st>>>(r, P, G, eps, adv);
  return hipGetLastError();
}

hipError_t loss_static_scratch(double** out) {
  static std::mutex mu;
  static std::vector<double*> by_device;   // device address of `scratch` per device
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(mu);
  if ((int)by_device.size() <= dev) by_device.resize(dev + 1, nullptr);
  if (!by_device[dev]) {
    // the current device is `dev`: the address of its copy
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    by_device[dev] = (double*)p;
  }
  *out = by_device[dev];
  return hipSuccess;
}

hipError_t token_loss(const float* lp, const float* lo, const float* lr, const uint8_t* mask,
                      const float* adv, int N, int Tr, float clip_eps, float beta, int agg,
                      float* loss, float* tok_loss, float* dl, float* stats, double* row_ws,
                      hipStream_t st) {
  if (N <= 0) return hipSuccess;
  double* wts = row_ws + (size_t)N * 8;
  Prof pf("token_loss", st);
  k_loss_rows<<<N, 256, 0, st>>>(lp, lo, lr, mask, adv, Tr, clip_eps, beta, tok_loss, row_ws);
  k_loss_final<<<1, 256, 0, st>>>(row_ws, N, agg, loss, stats, wts);
  if (dl) k_loss_grad<<<N, 256, 0, st>>>(lp, lo, lr, mask, adv, Tr, clip_eps, beta, wts, dl);
  return hipGetLastError();
}

}  // namespace grpo
