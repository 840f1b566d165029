// RL objective over a packed ragged batch: per-sequence log-ratio statistics
// and filter masks (Eq. 18-21), group-normalised advantages (Eq. 3 / 12), the
// sequence-masked clipped surrogate (Eq. 17) with an optional token-level
// truncation or drop of the ratio (Sec. 4.5.2) and an optional KL term, and
// its gradient with respect to the per-token log-probs.  One workgroup per group, one wave per
// sequence, wave-level reductions; all sums in fp64 and in a fixed order.
#include <hip/hip_runtime.h>

#include <mutex>

#include "mc_internal.hpp"

// Device scratch of the allocation-free loss entry point (mc_rl_loss_noalloc):
// one copy per GPU, held for the life of the process.  Host code never uses
// this name as an address (on the host it is a stand-in symbol); it takes
// the device address that hipGetSymbolAddress returns for the current GPU.
static __device__ __align__(256) char scratch[MC_RL_LOSS_NOALLOC_SCRATCH_BYTES];

namespace mc {

namespace {

constexpr int kLossThreads = 256;
constexpr int kLossWaves = kLossThreads / 64;

__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}
__device__ __forceinline__ int wave_sum(int x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}

// Bounds of sequence i clamped into [0, T]; flags inconsistent metadata.
__device__ __forceinline__ void seq_bounds(const int32_t* cu, int i, int B, int64_t T,
                                           int64_t& s, int64_t& e, bool& bad) {
  s = cu[i];
  e = cu[i + 1];
  if ((i == 0 && s != 0) || (i == B - 1 && e != T) || s < 0 || e > T || e < s) bad = true;
  s = s < 0 ? 0 : (s > T ? T : s);
  e = e < s ? s : (e > T ? T : e);
}

__device__ __forceinline__ void group_bounds(const int32_t* cg, int g, int NG, int B, int& a,
                                             int& b, bool& bad) {
  a = cg[g];
  b = cg[g + 1];
  if ((g == 0 && a != 0) || (g == NG - 1 && b != B) || a < 0 || b > B || b < a) bad = true;
  a = a < 0 ? 0 : (a > B ? B : a);
  b = b < a ? a : (b > B ? B : b);
}

struct SeqOut {
  uint8_t* seq_mask;
  int32_t* seq_len;
  float* adv;
  double* adv_d;
  float* stat_abs;
  float* stat_signed;
  long long* group_n;
  int32_t* err;
};

__global__ void k_loss_init(int32_t* err) {
  if (threadIdx.x == 0) *err = 0;
}

// Phase 1: per-sequence L_i, statistics and M_i; per-group advantages and
// N_g = sum_i M_i L_i.
__global__ __launch_bounds__(kLossThreads) void k_seq_stats(
    const float* __restrict__ logp, const float* __restrict__ lr,
    const uint8_t* __restrict__ mask, const int32_t* __restrict__ cu,
    const int32_t* __restrict__ cg, const float* __restrict__ rewards, int64_t T, int B,
    int NG, mc_rl_params_t p, SeqOut o) {
  __shared__ long long nsum[kLossWaves];
  __shared__ int bad_any;
  const int g = blockIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (threadIdx.x == 0) bad_any = 0;
  __syncthreads();
  bool bad = false;
  int a, b;
  group_bounds(cg, g, NG, B, a, b, bad);
  long long n_w = 0;
  for (int i = a + w; i < b; i += kLossWaves) {
    int64_t s, e;
    seq_bounds(cu, i, B, T, s, e, bad);
    int cnt = 0;
    double sa = 0.0, ss = 0.0;
    for (int64_t t = s + lane; t < e; t += 64) {
      const bool valid = mask ? mask[t] != 0 : true;
      if (valid) {
        const double ell = double(logp[t]) - double(lr[t]);
        cnt += 1;
        sa += fabs(ell);
        ss += ell;
      }
    }
    cnt = wave_sum(cnt);
    sa = wave_sum(sa);
    ss = wave_sum(ss);
    const double sabs = cnt > 0 ? sa / cnt : 0.0;
    const double ssig = cnt > 0 ? ss / cnt : 0.0;
    bool keep = cnt > 0;
    if (p.filter == MC_FILTER_MIRRORPOP) keep = keep && sabs <= double(p.delta);
    else if (p.filter == MC_FILTER_VANILLA) keep = keep && fabs(ssig) <= double(p.delta);
    if (lane == 0) {
      o.seq_len[i] = cnt;
      o.seq_mask[i] = keep ? 1 : 0;
      o.stat_abs[i] = float(sabs);
      o.stat_signed[i] = float(ssig);
    }
    n_w += keep ? cnt : 0;
  }
  if (lane == 0) nsum[w] = n_w;
  if (bad) bad_any = 1;
  __syncthreads();
  if (threadIdx.x == 0) {
    long long n = 0;
    for (int k = 0; k < kLossWaves; ++k) n += nsum[k];
    o.group_n[g] = n;
    const int G = b - a;
    if (G > 0) {
      double mean = 0.0;
      bool equal = true;
      for (int i = a; i < b; ++i) {
        mean += double(rewards[i]);
        equal = equal && rewards[i] == rewards[a];
      }
      mean /= G;
      double var = 0.0;
      for (int i = a; i < b; ++i) {
        const double dr = double(rewards[i]) - mean;
        var += dr * dr;
      }
      const int dof = G - p.std_ddof;
      var = dof > 0 ? var / dof : 0.0;
      const double den = sqrt(var) + double(p.adv_eps);
      for (int i = a; i < b; ++i) {
        const double num = double(rewards[i]) - mean;
        const double A = equal ? 0.0 : num / den;
        o.adv_d[i] = A;
        o.adv[i] = float(A);
      }
    }
    if (bad_any) *o.err = 1;
  }
}

// Phase 2: N = sum over groups (integer, fixed order).
__global__ __launch_bounds__(256) void k_count(const long long* __restrict__ group_n, int NG,
                                               long long* __restrict__ n_out) {
  __shared__ long long part[256];
  long long s = 0;
  for (int g = threadIdx.x; g < NG; g += 256) s += group_n[g];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (threadIdx.x < off) part[threadIdx.x] += part[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) *n_out = part[0];
}

// Phase 3: per-token surrogate and gradient (Eq. 17); per-sequence sums.
// With a reference policy, the KL term beta * k3 (k3 = e^r - r - 1,
// r = logp_ref - logp) joins the same token mean.  The token mode acts on
// the log-ratio ell: TIS scales the term of a token with ell > ln C by the
// constant C / rho (its gradient weight becomes C A), IcePop drops a token
// with ell outside [ln lo, ln hi] from the surrogate (it stays in N).
__global__ __launch_bounds__(kLossThreads) void k_surrogate(
    const float* __restrict__ logp, const float* __restrict__ lr,
    const float* __restrict__ lref, const uint8_t* __restrict__ mask,
    const int32_t* __restrict__ cu, const int32_t* __restrict__ cg, int64_t T, int B, int NG,
    mc_rl_params_t p, const uint8_t* __restrict__ seq_mask, const double* __restrict__ adv_d,
    const long long* __restrict__ n_valid, float* __restrict__ dlogp,
    double* __restrict__ seq_sum, int* __restrict__ seq_clip, double* __restrict__ seq_kl,
    int* __restrict__ seq_tok) {
  const int g = blockIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  bool bad = false;
  int a, b;
  group_bounds(cg, g, NG, B, a, b, bad);
  const long long N = *n_valid;
  const double invN = N > 0 ? 1.0 / double(N) : 0.0;
  const double lo = 1.0 - double(p.eps_low), hi = 1.0 + double(p.eps_high);
  const int mode = p.token_mode;
  const double log_cap = mode == MC_TOKEN_TIS ? log(double(p.tis_cap)) : 0.0;
  const double log_alo = mode == MC_TOKEN_ICEPOP ? log(double(p.icepop_lo)) : 0.0;
  const double log_ahi = mode == MC_TOKEN_ICEPOP ? log(double(p.icepop_hi)) : 0.0;
  for (int i = a + w; i < b; i += kLossWaves) {
    int64_t s, e;
    seq_bounds(cu, i, B, T, s, e, bad);
    const bool keep = seq_mask[i] != 0 && N > 0;
    const double A = adv_d[i];
    const double beta = double(p.kl_beta);
    const bool with_kl = lref != nullptr && beta != 0.0;
    double sum = 0.0, kl = 0.0;
    int nclip = 0, ntok = 0;
    for (int64_t t = s + lane; t < e; t += 64) {
      float out = 0.0f;
      const bool valid = mask ? mask[t] != 0 : true;
      if (keep && valid) {
        const double lp = double(logp[t]);
        const double ell = lp - double(lr[t]);
        double wgt = 1.0;
        bool dropped = false;
        if (mode == MC_TOKEN_TIS && ell > log_cap) {
          wgt = exp(log_cap - ell);
          ntok += 1;
        } else if (mode == MC_TOKEN_ICEPOP && !(ell >= log_alo && ell <= log_ahi)) {
          dropped = true;
          ntok += 1;
        }
        double g = 0.0;
        if (!dropped) {
          const double rho = exp(ell);
          const double un = rho * A;
          const double cl = fmin(fmax(rho, lo), hi) * A;
          sum += wgt * fmin(un, cl);
          if (un <= cl) g = -wgt * un;
          else nclip += 1;
        }
        if (with_kl) {
          const double r = double(lref[t]) - lp;
          const double er = exp(r);
          kl += er - r - 1.0;
          g += beta * (1.0 - er);
        }
        out = float(g * invN);
      }
      dlogp[t] = out;
    }
    sum = wave_sum(sum);
    kl = wave_sum(kl);
    nclip = wave_sum(nclip);
    ntok = wave_sum(ntok);
    if (lane == 0) {
      seq_sum[i] = sum;
      seq_clip[i] = nclip;
      seq_kl[i] = kl;
      seq_tok[i] = ntok;
    }
  }
}

// Phase 4: loss = -(1/N) sum_i seq_sum_i (+ beta * KL), the clip fraction,
// the token-mode fraction and the mean KL estimate.
__global__ __launch_bounds__(256) void k_finish(const double* __restrict__ seq_sum,
                                                const int* __restrict__ seq_clip,
                                                const double* __restrict__ seq_kl,
                                                const int* __restrict__ seq_tok, int B,
                                                float beta, const long long* __restrict__ n_valid,
                                                float* __restrict__ loss,
                                                float* __restrict__ clip_frac,
                                                float* __restrict__ kl_out,
                                                float* __restrict__ tok_frac) {
  __shared__ double ps[256], pk[256];
  __shared__ long long pc[256], pt[256];
  double s = 0.0, k = 0.0;
  long long c = 0, n = 0;
  for (int i = threadIdx.x; i < B; i += 256) {
    s += seq_sum[i];
    k += seq_kl[i];
    c += seq_clip[i];
    n += seq_tok[i];
  }
  ps[threadIdx.x] = s;
  pk[threadIdx.x] = k;
  pc[threadIdx.x] = c;
  pt[threadIdx.x] = n;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (threadIdx.x < off) {
      ps[threadIdx.x] += ps[threadIdx.x + off];
      pk[threadIdx.x] += pk[threadIdx.x + off];
      pc[threadIdx.x] += pc[threadIdx.x + off];
      pt[threadIdx.x] += pt[threadIdx.x + off];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const long long N = *n_valid;
    const double kl = N > 0 ? pk[0] / double(N) : 0.0;
    *loss = N > 0 ? float(-ps[0] / double(N) + double(beta) * kl) : 0.0f;
    if (clip_frac) *clip_frac = N > 0 ? float(double(pc[0]) / double(N)) : 0.0f;
    if (kl_out) *kl_out = float(kl);
    if (tok_frac) *tok_frac = N > 0 ? float(double(pt[0]) / double(N)) : 0.0f;
  }
}

// PrimeEcho trajectory reward (Eq. 9-10): R = alpha s_1 + (1 - alpha) max_k s_k
// + beta1 [success_1] + beta2 [not success_1 and success_2].  One thread per
// trajectory; K_i is clamped into [1, Kmax].
__global__ __launch_bounds__(256) void k_primeecho(const float* __restrict__ scores,
                                                   const uint8_t* __restrict__ success,
                                                   const int32_t* __restrict__ n_turns, int B,
                                                   int Kmax, float alpha, float beta1,
                                                   float beta2, float* __restrict__ rewards) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B) return;
  int K = n_turns ? n_turns[i] : Kmax;
  K = K < 1 ? 1 : (K > Kmax ? Kmax : K);
  const float* sc = scores + int64_t(i) * Kmax;
  const double first = double(sc[0]);
  double best = first;
  for (int k = 1; k < K; ++k) best = fmax(best, double(sc[k]));
  double b = 0.0;
  if (success) {
    const uint8_t* su = success + int64_t(i) * Kmax;
    if (su[0]) b = double(beta1);
    else if (K >= 2 && su[1]) b = double(beta2);
  }
  rewards[i] = float(double(alpha) * first + (1.0 - double(alpha)) * best + b);
}

}  // namespace

size_t loss_workspace(int64_t T, int32_t B, int32_t NG) {
  (void)T;
  const size_t b = size_t(B > 0 ? B : 1), g = size_t(NG > 0 ? NG : 1);
  size_t n = 0;
  n += align_up(b * 1, kWsAlign);                 // seq_mask
  n += align_up(b * 4, kWsAlign);                 // seq_len
  n += 3 * align_up(b * 4, kWsAlign);             // adv, stat_abs, stat_signed
  n += align_up(b * 8, kWsAlign);                 // adv_d
  n += align_up(b * 8, kWsAlign);                 // seq_sum
  n += align_up(b * 4, kWsAlign);                 // seq_clip
  n += align_up(b * 8, kWsAlign);                 // seq_kl
  n += align_up(b * 4, kWsAlign);                 // seq_tok
  n += align_up(g * 8, kWsAlign);                 // group_n
  n += align_up(8, kWsAlign);                     // n_valid
  n += align_up(4, kWsAlign);                     // err
  return n;
}

hipError_t launch_primeecho(const float* scores, const uint8_t* success, const int32_t* n_turns,
                            int32_t B, int32_t Kmax, float alpha, float beta1, float beta2,
                            float* rewards, hipStream_t s) {
  if (B == 0) return hipSuccess;
  hipLaunchKernelGGL(k_primeecho, dim3(cdiv(B, 256)), dim3(256), 0, s, scores, success, n_turns,
                     B, Kmax, alpha, beta1, beta2, rewards);
  return hipGetLastError();
}

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

// The current GPU's copy of `scratch`, looked up once per device with that
// device current; no allocation.
hipError_t loss_scratch(void** ptr, size_t* bytes) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  *bytes = MC_RL_LOSS_NOALLOC_SCRATCH_BYTES;
  return hipSuccess;
}

hipError_t launch_loss(const float* logp, const float* logp_rollout, const float* logp_ref,
                       const uint8_t* mask,
                       const int32_t* cu_seqlens, const int32_t* cu_groups,
                       const float* rewards, int64_t T, int32_t B, int32_t NG,
                       const mc_rl_params_t& p, const mc_rl_outputs_t& out, void* ws,
                       hipStream_t s, bool profile) {
  const size_t b = size_t(B > 0 ? B : 1), g = size_t(NG > 0 ? NG : 1);
  Carve cv(ws);
  uint8_t* w_mask = cv.take<uint8_t>(b);
  int32_t* w_len = cv.take<int32_t>(b);
  float* w_adv = cv.take<float>(b);
  float* w_sa = cv.take<float>(b);
  float* w_ss = cv.take<float>(b);
  double* adv_d = cv.take<double>(b);
  double* seq_sum = cv.take<double>(b);
  int* seq_clip = cv.take<int>(b);
  double* seq_kl = cv.take<double>(b);
  int* seq_tok = cv.take<int>(b);
  long long* group_n = cv.take<long long>(g);
  long long* w_n = cv.take<long long>(1);
  int32_t* w_err = cv.take<int32_t>(1);

  SeqOut o{out.seq_mask ? out.seq_mask : w_mask,
           out.seq_len ? out.seq_len : w_len,
           out.adv ? out.adv : w_adv,
           adv_d,
           out.stat_abs ? out.stat_abs : w_sa,
           out.stat_signed ? out.stat_signed : w_ss,
           group_n,
           out.error_flag ? out.error_flag : w_err};
  long long* n_valid = out.n_valid ? reinterpret_cast<long long*>(out.n_valid) : w_n;

  // (the profiler's events are created only when it is enabled and profile is set)
  ProfScope ps_(s, profile ? "rl_loss" : nullptr, 0.0,
                double(T) * (4 + 4 + (mask ? 1 : 0) + 4) + 16.0 * b);
  hipLaunchKernelGGL(k_loss_init, dim3(1), dim3(64), 0, s, o.err);
  if (NG > 0)
    hipLaunchKernelGGL(k_seq_stats, dim3(NG), dim3(kLossThreads), 0, s, logp, logp_rollout,
                       mask, cu_seqlens, cu_groups, rewards, T, B, NG, p, o);
  hipLaunchKernelGGL(k_count, dim3(1), dim3(256), 0, s, group_n, NG, n_valid);
  if (NG > 0)
    hipLaunchKernelGGL(k_surrogate, dim3(NG), dim3(kLossThreads), 0, s, logp, logp_rollout,
                       logp_ref, mask, cu_seqlens, cu_groups, T, B, NG, p, o.seq_mask, adv_d,
                       n_valid, out.dlogp, seq_sum, seq_clip, seq_kl, seq_tok);
  hipLaunchKernelGGL(k_finish, dim3(1), dim3(256), 0, s, seq_sum, seq_clip, seq_kl, seq_tok, B,
                     p.kl_beta, n_valid, out.loss, out.clip_frac, out.kl, out.token_frac);
  return hipGetLastError();
}

}  // namespace mc
