// Internal launch interface between the C ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "mc.h"

namespace mc {

constexpr size_t kWsAlign = 256;

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Bump allocator over the caller's workspace.
struct Carve {
  char* base;
  size_t used = 0;
  explicit Carve(void* p) : base(static_cast<char*>(p)) {}
  template <typename U> U* take(size_t n) {
    U* p = reinterpret_cast<U*>(base ? base + used : nullptr);
    used = align_up(used + n * sizeof(U), kWsAlign);
    return p;
  }
};

// Vocabulary chunk width of the backward: the transient [T x chunk] softmax
// operand stays within kBwdChunkBytes (sized for 288 GB of HBM: the
// 16384 x 151936 bf16 operand of the headline shape is one 5 GB chunk);
// larger problems are split into equal chunks, multiples of 256 columns.
constexpr size_t kBwdChunkBytes = size_t(8) << 30;
int64_t bwd_chunk_cols(int64_t T, int64_t V, size_t esize);

// RAII timing scope around one or more launches on `s` (see mc_profiler_*);
// a null name records nothing.
class ProfScope {
 public:
  ProfScope(hipStream_t s, const char* name, double flops, double bytes);
  ~ProfScope();
  ProfScope(const ProfScope&) = delete;
  ProfScope& operator=(const ProfScope&) = delete;

 private:
  hipStream_t stream_;
  const char* name_;
  double flops_, bytes_;
  hipEvent_t start_ = nullptr, stop_ = nullptr;
  bool active_ = false;
};

size_t fwd_workspace(int64_t T, int64_t d, int64_t V, mc_dtype_t dt);
size_t bwd_workspace(int64_t T, int64_t d, int64_t V, mc_dtype_t dt);
size_t cache_bytes(int64_t T, int64_t d, int64_t V, mc_dtype_t dt);
size_t bwd_cache_workspace(int64_t T, int64_t d, int64_t V, mc_dtype_t dt);
size_t loss_workspace(int64_t T, int32_t B, int32_t NG);

// Forward over the vocabulary shard [v_off, v_off + Vs) of V entries.  With
// part == null: final logp, lse (and entropy if non-null); otherwise the
// shard's partial [4][T] = (max, sum exp, sum exp * z, target logit or -inf).
hipError_t launch_fwd(const void* H, const void* W, const int64_t* y, int64_t T, int64_t d,
                      int64_t Vs, int64_t v_off, int64_t V, mc_dtype_t dt, float* logp,
                      float* lse, float* entropy, float* part, bool with_u, void* ws,
                      hipStream_t s);
hipError_t launch_merge(const float* parts, int S, const int64_t* y, int64_t T, int64_t V,
                        float* logp, float* lse, float* entropy, hipStream_t s);
hipError_t launch_bwd(const void* H, const void* W, const int64_t* y, const float* lse,
                      const float* dlogp, int64_t T, int64_t d, int64_t Vs, int64_t v_off,
                      int64_t V, mc_dtype_t dt, float* dH, float* dW, int flags, void* ws,
                      hipStream_t s);
hipError_t launch_fwd_cache(const void* H, const void* W, const int64_t* y, int64_t T, int64_t d,
                            int64_t V, mc_dtype_t dt, float* logp, float* lse, float* entropy,
                            void* cache, void* ws, hipStream_t s);
// p[0 .. n) = 0 with a kernel (not a memset, so that a captured graph holds
// only kernel nodes).
hipError_t launch_zero(float* p, int64_t n, hipStream_t s);
hipError_t launch_bwd_cache(const void* H, const void* W, const int64_t* y, const float* lse,
                            const float* dlogp, int64_t T, int64_t d, int64_t V, mc_dtype_t dt,
                            void* cache, float* dH, float* dW, int flags, void* ws,
                            hipStream_t s);
hipError_t launch_primeecho(const float* scores, const uint8_t* success, const int32_t* n_turns,
                            int32_t B, int32_t Kmax, float alpha, float beta1, float beta2,
                            float* rewards, hipStream_t s);
hipError_t launch_loss(const float* logp, const float* logp_rollout, const float* logp_ref,
                       const uint8_t* mask,
                       const int32_t* cu_seqlens, const int32_t* cu_groups,
                       const float* rewards, int64_t T, int32_t B, int32_t NG,
                       const mc_rl_params_t& p, const mc_rl_outputs_t& out, void* ws,
                       hipStream_t s, bool profile = true);
// Device address and size of the current GPU's fixed loss scratch (no
// allocation; looked up once per device).
hipError_t loss_scratch(void** ptr, size_t* bytes);

}  // namespace mc
