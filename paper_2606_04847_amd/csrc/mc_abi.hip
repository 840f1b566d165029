// extern "C" entry points of libmc.so: argument validation on the host (no
// HIP call on any error path), workspace checks, then the launches.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "mc_internal.hpp"

namespace {

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

constexpr int64_t kMaxDim = (int64_t(1) << 31) - 1;
constexpr int64_t kMaxD = int64_t(64) * 65535;   // transposes tile d over grid y

mc_status_t check_dims(int64_t T, int64_t d, int64_t V, mc_dtype_t dt) {
  if (T < 0 || d < 1 || V < 1) return MC_ERR_INVALID_ARG;
  if (dt != MC_F32 && dt != MC_BF16) return MC_ERR_UNSUPPORTED;
  if (d % 8 != 0) return MC_ERR_UNSUPPORTED;
  if (T > kMaxDim || V > kMaxDim - 256 || d > kMaxD) return MC_ERR_UNSUPPORTED;
  // one launch must stay below 2^31 workgroups
  if (mc::cdiv(T, 256) * mc::cdiv(V, 256) > kMaxDim) return MC_ERR_UNSUPPORTED;
  return MC_OK;
}

mc_status_t check_ws(void* ws, size_t bytes, size_t need) {
  if (need == 0) return MC_OK;
  if (ws == nullptr || bytes < need || !aligned(ws, mc::kWsAlign)) return MC_ERR_WORKSPACE;
  return MC_OK;
}

mc_status_t from_hip(hipError_t e) { return e == hipSuccess ? MC_OK : MC_ERR_HIP; }

bool finite(float x) { return std::isfinite(x); }

}  // namespace

extern "C" {

const char* mc_status_string(mc_status_t s) {
  switch (s) {
    case MC_OK: return "MC_OK";
    case MC_ERR_INVALID_ARG: return "MC_ERR_INVALID_ARG";
    case MC_ERR_UNSUPPORTED: return "MC_ERR_UNSUPPORTED";
    case MC_ERR_WORKSPACE: return "MC_ERR_WORKSPACE";
    case MC_ERR_HIP: return "MC_ERR_HIP";
  }
  return "MC_ERR_UNKNOWN";
}

const char* mc_version(void) { return "mc 0.1.0 gfx950"; }

size_t mc_logprob_fwd_workspace_size(int64_t T, int64_t d, int64_t V, mc_dtype_t dt) {
  if (check_dims(T, d, V, dt) != MC_OK) return 0;
  return mc::fwd_workspace(T, d, V, dt);
}

mc_status_t mc_logprob_fwd(const void* hidden, const void* weight, const int64_t* targets,
                           int64_t T, int64_t d, int64_t V, mc_dtype_t dt, float* logp,
                           float* lse, float* entropy, void* ws, size_t ws_bytes, void* stream) {
  mc_status_t st = check_dims(T, d, V, dt);
  if (st != MC_OK) return st;
  if (T == 0) return MC_OK;
  if (!hidden || !weight || !targets || !logp || !lse) return MC_ERR_INVALID_ARG;
  if (!aligned(hidden, 16) || !aligned(weight, 16) || !aligned(targets, 8) ||
      !aligned(logp, 4) || !aligned(lse, 4) || (entropy && !aligned(entropy, 4)))
    return MC_ERR_INVALID_ARG;
  st = check_ws(ws, ws_bytes, mc::fwd_workspace(T, d, V, dt));
  if (st != MC_OK) return st;
  return from_hip(mc::launch_fwd(hidden, weight, targets, T, d, V, 0, V, dt, logp, lse, entropy,
                                 nullptr, entropy != nullptr, ws,
                                 static_cast<hipStream_t>(stream)));
}

mc_status_t mc_logprob_fwd_shard(const void* hidden, const void* weight_shard,
                                 const int64_t* targets, int64_t T, int64_t d, int64_t V_shard,
                                 int64_t v_offset, int64_t V_total, mc_dtype_t dt,
                                 float* partial, void* ws, size_t ws_bytes, void* stream) {
  mc_status_t st = check_dims(T, d, V_shard, dt);
  if (st != MC_OK) return st;
  if (v_offset < 0 || V_total < V_shard || v_offset > V_total - V_shard || V_total > kMaxDim)
    return MC_ERR_INVALID_ARG;
  if (T == 0) return MC_OK;
  if (!hidden || !weight_shard || !targets || !partial) return MC_ERR_INVALID_ARG;
  if (!aligned(hidden, 16) || !aligned(weight_shard, 16) || !aligned(targets, 8) ||
      !aligned(partial, 4))
    return MC_ERR_INVALID_ARG;
  st = check_ws(ws, ws_bytes, mc::fwd_workspace(T, d, V_shard, dt));
  if (st != MC_OK) return st;
  return from_hip(mc::launch_fwd(hidden, weight_shard, targets, T, d, V_shard, v_offset, V_total,
                                 dt, nullptr, nullptr, nullptr, partial, true, ws,
                                 static_cast<hipStream_t>(stream)));
}

mc_status_t mc_logprob_merge_shards(const float* partials, int32_t S, const int64_t* targets,
                                    int64_t T, int64_t V_total, float* logp, float* lse,
                                    float* entropy, void* stream) {
  if (S < 1 || T < 0 || T > kMaxDim || V_total < 1) return MC_ERR_INVALID_ARG;
  if (T == 0) return MC_OK;
  if (!partials || !targets || !logp || !lse) return MC_ERR_INVALID_ARG;
  if (!aligned(partials, 4) || !aligned(targets, 8)) return MC_ERR_INVALID_ARG;
  return from_hip(mc::launch_merge(partials, S, targets, T, V_total, logp, lse, entropy,
                                   static_cast<hipStream_t>(stream)));
}

size_t mc_logprob_bwd_workspace_size(int64_t T, int64_t d, int64_t V, mc_dtype_t dt) {
  if (check_dims(T, d, V, dt) != MC_OK) return 0;
  return mc::bwd_workspace(T, d, V, dt);
}

size_t mc_logprob_cache_size(int64_t T, int64_t d, int64_t V, mc_dtype_t dt) {
  if (check_dims(T, d, V, dt) != MC_OK) return 0;
  return mc::cache_bytes(T, d, V, dt);
}

mc_status_t mc_logprob_fwd_cached(const void* hidden, const void* weight, const int64_t* targets,
                                  int64_t T, int64_t d, int64_t V, mc_dtype_t dt, float* logp,
                                  float* lse, float* entropy, void* cache, size_t cache_bytes,
                                  void* ws, size_t ws_bytes, void* stream) {
  mc_status_t st = check_dims(T, d, V, dt);
  if (st != MC_OK) return st;
  if (T == 0) return MC_OK;
  if (!hidden || !weight || !targets || !logp || !lse) return MC_ERR_INVALID_ARG;
  if (!aligned(hidden, 16) || !aligned(weight, 16) || !aligned(targets, 8) ||
      !aligned(logp, 4) || !aligned(lse, 4) || (entropy && !aligned(entropy, 4)))
    return MC_ERR_INVALID_ARG;
  st = check_ws(cache, cache_bytes, mc::cache_bytes(T, d, V, dt));
  if (st != MC_OK) return st;
  st = check_ws(ws, ws_bytes, mc::fwd_workspace(T, d, V, dt));
  if (st != MC_OK) return st;
  return from_hip(mc::launch_fwd_cache(hidden, weight, targets, T, d, V, dt, logp, lse, entropy,
                                       cache, ws, static_cast<hipStream_t>(stream)));
}

size_t mc_logprob_bwd_cached_workspace_size(int64_t T, int64_t d, int64_t V, mc_dtype_t dt) {
  if (check_dims(T, d, V, dt) != MC_OK) return 0;
  return mc::bwd_cache_workspace(T, d, V, dt);
}

mc_status_t mc_logprob_bwd_cached(const void* hidden, const void* weight, const int64_t* targets,
                                  const float* lse, const float* dlogp, int64_t T, int64_t d,
                                  int64_t V, mc_dtype_t dt, void* cache, size_t cache_bytes,
                                  float* dhidden, float* dweight, int32_t flags, void* ws,
                                  size_t ws_bytes, void* stream) {
  mc_status_t st = check_dims(T, d, V, dt);
  if (st != MC_OK) return st;
  if (flags & ~(MC_BWD_ACCUMULATE_DHIDDEN | MC_BWD_ACCUMULATE_DWEIGHT | MC_BWD_SKIP_DEAD_TOKENS))
    return MC_ERR_INVALID_ARG;
  if (!dhidden && !dweight) return MC_ERR_INVALID_ARG;
  if (!hidden || !weight) return MC_ERR_INVALID_ARG;
  if (!aligned(hidden, 16) || !aligned(weight, 16) || (dhidden && !aligned(dhidden, 16)) ||
      (dweight && !aligned(dweight, 16)))
    return MC_ERR_INVALID_ARG;
  if (T == 0) {
    if (dweight && !(flags & MC_BWD_ACCUMULATE_DWEIGHT))
      return from_hip(mc::launch_zero(dweight, V * d, static_cast<hipStream_t>(stream)));
    return MC_OK;
  }
  if (!targets || !lse || !dlogp) return MC_ERR_INVALID_ARG;
  if (!aligned(targets, 8) || !aligned(lse, 4) || !aligned(dlogp, 4)) return MC_ERR_INVALID_ARG;
  st = check_ws(cache, cache_bytes, mc::cache_bytes(T, d, V, dt));
  if (st != MC_OK) return st;
  st = check_ws(ws, ws_bytes, mc::bwd_cache_workspace(T, d, V, dt));
  if (st != MC_OK) return st;
  return from_hip(mc::launch_bwd_cache(hidden, weight, targets, lse, dlogp, T, d, V, dt, cache,
                                       dhidden, dweight, flags, ws,
                                       static_cast<hipStream_t>(stream)));
}

static mc_status_t bwd_common(const void* hidden, const void* weight, const int64_t* targets,
                              const float* lse, const float* dlogp, int64_t T, int64_t d,
                              int64_t V, int64_t v_offset, int64_t V_total, mc_dtype_t dt,
                              float* dhidden, float* dweight, int32_t flags, void* ws,
                              size_t ws_bytes, void* stream);

mc_status_t mc_logprob_bwd(const void* hidden, const void* weight, const int64_t* targets,
                           const float* lse, const float* dlogp, int64_t T, int64_t d, int64_t V,
                           mc_dtype_t dt, float* dhidden, float* dweight, int32_t flags,
                           void* ws, size_t ws_bytes, void* stream) {
  return bwd_common(hidden, weight, targets, lse, dlogp, T, d, V, 0, V, dt, dhidden, dweight,
                    flags, ws, ws_bytes, stream);
}

mc_status_t mc_logprob_bwd_shard(const void* hidden, const void* weight_shard,
                                 const int64_t* targets, const float* lse, const float* dlogp,
                                 int64_t T, int64_t d, int64_t V_shard, int64_t v_offset,
                                 int64_t V_total, mc_dtype_t dt, float* dhidden,
                                 float* dweight_shard, int32_t flags, void* ws, size_t ws_bytes,
                                 void* stream) {
  if (v_offset < 0 || V_total < V_shard || v_offset > V_total - V_shard || V_total > kMaxDim)
    return MC_ERR_INVALID_ARG;
  return bwd_common(hidden, weight_shard, targets, lse, dlogp, T, d, V_shard, v_offset, V_total,
                    dt, dhidden, dweight_shard, flags, ws, ws_bytes, stream);
}

static mc_status_t bwd_common(const void* hidden, const void* weight, const int64_t* targets,
                              const float* lse, const float* dlogp, int64_t T, int64_t d,
                              int64_t V, int64_t v_offset, int64_t V_total, mc_dtype_t dt,
                              float* dhidden, float* dweight, int32_t flags, void* ws,
                              size_t ws_bytes, void* stream) {
  mc_status_t st = check_dims(T, d, V, dt);
  if (st != MC_OK) return st;
  if (flags & ~(MC_BWD_ACCUMULATE_DHIDDEN | MC_BWD_ACCUMULATE_DWEIGHT | MC_BWD_SKIP_DEAD_TOKENS))
    return MC_ERR_INVALID_ARG;
  if (!dhidden && !dweight) return MC_ERR_INVALID_ARG;
  if (!hidden || !weight) return MC_ERR_INVALID_ARG;
  if (!aligned(hidden, 16) || !aligned(weight, 16) || (dhidden && !aligned(dhidden, 16)) ||
      (dweight && !aligned(dweight, 16)))
    return MC_ERR_INVALID_ARG;
  if (T == 0) {
    // no tokens: dhidden is empty; dweight receives a zero gradient
    if (dweight && !(flags & MC_BWD_ACCUMULATE_DWEIGHT))
      return from_hip(mc::launch_zero(dweight, V * d, static_cast<hipStream_t>(stream)));
    return MC_OK;
  }
  if (!targets || !lse || !dlogp) return MC_ERR_INVALID_ARG;
  if (!aligned(targets, 8) || !aligned(lse, 4) || !aligned(dlogp, 4)) return MC_ERR_INVALID_ARG;
  st = check_ws(ws, ws_bytes, mc::bwd_workspace(T, d, V, dt));
  if (st != MC_OK) return st;
  return from_hip(mc::launch_bwd(hidden, weight, targets, lse, dlogp, T, d, V, v_offset, V_total,
                                 dt, dhidden, dweight, flags, ws,
                                 static_cast<hipStream_t>(stream)));
}

size_t mc_rl_loss_workspace_size(int64_t T, int32_t B, int32_t NG) {
  if (T < 0 || B < 0 || NG < 0) return 0;
  return mc::loss_workspace(T, B, NG);
}

// Argument checks shared by mc_rl_loss and mc_rl_loss_noalloc.
static mc_status_t check_loss_args(const float* logp, const float* logp_rollout,
                                   const int32_t* cu_seqlens, const int32_t* cu_groups,
                                   const float* rewards, int64_t T, int32_t B, int32_t NG,
                                   const mc_rl_params_t* params, const mc_rl_outputs_t* out) {
  if (T < 0 || B < 0 || NG < 0 || T > kMaxDim) return MC_ERR_INVALID_ARG;
  if (!params || !out || !out->loss) return MC_ERR_INVALID_ARG;
  if (B == 0 && T > 0) return MC_ERR_INVALID_ARG;   // tokens outside every sequence
  if (NG == 0 && B > 0) return MC_ERR_INVALID_ARG;  // sequences outside every group
  const mc_rl_params_t& p = *params;
  if (!finite(p.eps_low) || !finite(p.eps_high) || !finite(p.delta) || !finite(p.adv_eps) ||
      !finite(p.kl_beta) || p.kl_beta < 0.0f)
    return MC_ERR_INVALID_ARG;
  if (p.eps_low < 0.0f || p.eps_low >= 1.0f || p.eps_high < 0.0f || p.delta < 0.0f ||
      p.adv_eps < 0.0f)
    return MC_ERR_INVALID_ARG;
  if (p.std_ddof != 0 && p.std_ddof != 1) return MC_ERR_INVALID_ARG;
  if (p.filter != MC_FILTER_NONE && p.filter != MC_FILTER_VANILLA &&
      p.filter != MC_FILTER_MIRRORPOP)
    return MC_ERR_INVALID_ARG;
  if (p.token_mode != MC_TOKEN_NONE && p.token_mode != MC_TOKEN_TIS &&
      p.token_mode != MC_TOKEN_ICEPOP)
    return MC_ERR_INVALID_ARG;
  if (p.token_mode == MC_TOKEN_TIS && !(finite(p.tis_cap) && p.tis_cap > 0.0f))
    return MC_ERR_INVALID_ARG;
  if (p.token_mode == MC_TOKEN_ICEPOP &&
      !(finite(p.icepop_lo) && finite(p.icepop_hi) && p.icepop_lo > 0.0f &&
        p.icepop_lo <= p.icepop_hi))
    return MC_ERR_INVALID_ARG;
  if (!cu_seqlens || !cu_groups || (B > 0 && !rewards)) return MC_ERR_INVALID_ARG;
  if (T > 0 && (!logp || !logp_rollout || !out->dlogp)) return MC_ERR_INVALID_ARG;
  if (!aligned(cu_seqlens, 4) || !aligned(cu_groups, 4) || !aligned(out->loss, 4) ||
      (out->n_valid && !aligned(out->n_valid, 8)))
    return MC_ERR_INVALID_ARG;
  return MC_OK;
}

mc_status_t mc_rl_loss(const float* logp, const float* logp_rollout, const float* logp_ref,
                       const uint8_t* loss_mask, const int32_t* cu_seqlens,
                       const int32_t* cu_groups, const float* rewards, int64_t T, int32_t B,
                       int32_t NG, const mc_rl_params_t* params, const mc_rl_outputs_t* out,
                       void* ws, size_t ws_bytes, void* stream) {
  mc_status_t st = check_loss_args(logp, logp_rollout, cu_seqlens, cu_groups, rewards, T, B, NG,
                                   params, out);
  if (st != MC_OK) return st;
  st = check_ws(ws, ws_bytes, mc::loss_workspace(T, B, NG));
  if (st != MC_OK) return st;
  return from_hip(mc::launch_loss(logp, logp_rollout, logp_ref, loss_mask, cu_seqlens, cu_groups,
                                  rewards, T, B, NG, *params, *out, ws,
                                  static_cast<hipStream_t>(stream)));
}

size_t mc_rl_loss_noalloc_max_bytes(void) { return MC_RL_LOSS_NOALLOC_SCRATCH_BYTES; }

mc_status_t mc_rl_loss_noalloc(const float* logp, const float* logp_rollout,
                               const float* logp_ref, const uint8_t* loss_mask,
                               const int32_t* cu_seqlens, const int32_t* cu_groups,
                               const float* rewards, int64_t T, int32_t B, int32_t NG,
                               const mc_rl_params_t* params, const mc_rl_outputs_t* out,
                               void* stream) {
  mc_status_t st = check_loss_args(logp, logp_rollout, cu_seqlens, cu_groups, rewards, T, B, NG,
                                   params, out);
  if (st != MC_OK) return st;
  if (mc::loss_workspace(T, B, NG) > MC_RL_LOSS_NOALLOC_SCRATCH_BYTES) return MC_ERR_UNSUPPORTED;
  // the scratch is per GPU: the stream must belong to the current device
  const hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return MC_ERR_HIP;
  if (s != nullptr) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(s, &sdev) != hipSuccess) return MC_ERR_HIP;
    if (int(sdev) != dev) return MC_ERR_INVALID_ARG;
  }
  void* ws = nullptr;
  size_t ws_bytes = 0;
  if (mc::loss_scratch(&ws, &ws_bytes) != hipSuccess) return MC_ERR_HIP;
  return from_hip(mc::launch_loss(logp, logp_rollout, logp_ref, loss_mask, cu_seqlens, cu_groups,
                                  rewards, T, B, NG, *params, *out, ws, s, false));
}

mc_status_t mc_primeecho_rewards(const float* scores, const uint8_t* success,
                                 const int32_t* n_turns, int32_t B, int32_t Kmax, float alpha,
                                 float beta1, float beta2, float* rewards, void* stream) {
  if (B < 0 || Kmax < 1) return MC_ERR_INVALID_ARG;
  if (!finite(alpha) || alpha < 0.0f || alpha > 1.0f || !finite(beta1) || !finite(beta2))
    return MC_ERR_INVALID_ARG;
  if (B == 0) return MC_OK;
  if (!scores || !rewards) return MC_ERR_INVALID_ARG;
  return from_hip(mc::launch_primeecho(scores, success, n_turns, B, Kmax, alpha, beta1, beta2,
                                       rewards, static_cast<hipStream_t>(stream)));
}

mc_status_t mc_check_packing(const int32_t* cu, int32_t B, const int32_t* cg, int32_t NG,
                             int64_t T) {
  if (!cu || !cg || B < 0 || NG < 0 || T < 0) return MC_ERR_INVALID_ARG;
  if (cu[0] != 0 || int64_t(cu[B]) != T) return MC_ERR_INVALID_ARG;
  for (int32_t i = 0; i < B; ++i)
    if (cu[i + 1] < cu[i]) return MC_ERR_INVALID_ARG;
  if (cg[0] != 0 || cg[NG] != B) return MC_ERR_INVALID_ARG;
  for (int32_t g = 0; g < NG; ++g)
    if (cg[g + 1] < cg[g]) return MC_ERR_INVALID_ARG;
  return MC_OK;
}

}  // extern "C"
