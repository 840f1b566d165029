/*
 * mc.h -- C ABI of the fused RL log-prob library (libmc.so) for AMD MI355X
 * (gfx950).
 *
 * The library computes, on one GPU:
 *   - the trainer-side per-token log-probability log pi_theta(o_t | x, o_<t)
 *     over the full vocabulary (the numerator of the importance ratio of
 *     Eq. 4): logits z = hidden . weight^T are reduced in the GEMM epilogue by
 *     an online log-sum-exp and a gather of the target logit.  In the plain
 *     pair (mc_logprob_fwd / mc_logprob_bwd) the logits are never written to
 *     memory: the forward keeps only per-row partials and the backward
 *     recomputes the logits, writing their gradient (a 2-byte transient per
 *     vocabulary chunk) as the operand of its two contractions.  The cached
 *     pair (mc_logprob_fwd_cached / mc_logprob_bwd_cached) trades memory for
 *     that recomputation: its forward writes a [T, V] softmax cache;
 *   - its backward (chain rule through the log-softmax);
 *   - the RL objective on top of it: log importance ratios (Eq. 4), the
 *     MirrorPop sequence statistic and mask (Eq. 19-21) or the signed one
 *     (Eq. 18), optional token-level truncation or dropping of the ratio
 *     (Sec. 4.5.2), group-normalised advantages (Eq. 3 / Eq. 12), the
 *     sequence-masked clipped surrogate and the KL term beta D_KL of Eq. 17
 *     (beta a parameter, 0 unless a reference policy's log-probs are passed;
 *     the paper names no estimator, this library uses k3), with its gradient
 *     with respect to the per-token log-probs.
 *
 * Conventions shared by every entry point
 *   Memory      Every array argument is caller-owned DEVICE memory unless a
 *               comment says "host".  The library allocates nothing and keeps
 *               no pointer after a call returns.
 *   Workspace   Each entry point takes a device workspace of at least the size
 *               its *_workspace_size query returns, aligned to 256 bytes.  Its
 *               contents on entry do not matter; on return they are undefined.
 *   Streams     `stream` is a hipStream_t (NULL = the default stream).  Work is
 *               enqueued on it and the call returns without waiting; buffers
 *               must stay valid until the stream has finished the work.
 *   Layout      Matrices are row-major and contiguous, 16-byte aligned.
 *               d must be a multiple of 8 and at most 4194240 (64 x 65535).
 *   Errors      Scalar and pointer arguments are checked on the host before any
 *               launch; a bad argument returns an error code and enqueues
 *               nothing.  A launch failure returns MC_ERR_HIP.  No exception or
 *               abort crosses the ABI.
 *   Threads     Re-entrant; no mutable global state apart from the opt-in
 *               profiler at the end of this header.
 *   Determinism Results are bit-identical from run to run for the same
 *               inputs, shapes and device: no floating-point atomics are used.
 */
#ifndef MC_H_
#define MC_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MC_OK = 0,
  MC_ERR_INVALID_ARG = 1,   /* null pointer, negative size, bad parameter */
  MC_ERR_UNSUPPORTED = 2,   /* valid but not supported (d % 8 != 0, dtype) */
  MC_ERR_WORKSPACE = 3,     /* workspace too small or misaligned */
  MC_ERR_HIP = 4            /* a HIP launch or runtime call failed */
} mc_status_t;

typedef enum {
  MC_F32 = 0,               /* fp32 hidden/weight, fp32 MFMA */
  MC_BF16 = 1               /* bf16 hidden/weight, bf16 MFMA, fp32 accumulate */
} mc_dtype_t;

typedef enum {
  MC_FILTER_NONE = 0,       /* keep every sequence with a valid token (Eq. 5) */
  MC_FILTER_VANILLA = 1,    /* |(1/L_i) sum_t log rho_t| <= delta (Eq. 18) */
  MC_FILTER_MIRRORPOP = 2   /* (1/L_i) sum_t |log rho_t| <= delta (Eq. 21) */
} mc_filter_t;

/* Token-level treatment of the importance ratio, the alternatives to
 * sequence masking that Sec. 4.5.2 names (truncated importance sampling and
 * IcePop) without giving formulas; the definitions below are this library's
 * readings.  Both combine with any mc_filter_t and act on retained tokens
 * (loss mask set, M_i = 1) only. */
typedef enum {
  MC_TOKEN_NONE = 0,        /* plain Eq. 17 */
  MC_TOKEN_TIS = 1,         /* a token with rho_t > tis_cap has its term scaled by the
                               stop-gradient factor tis_cap / rho_t: its gradient
                               weight rho_t A_i is truncated to tis_cap A_i */
  MC_TOKEN_ICEPOP = 2       /* a token with rho_t outside [icepop_lo, icepop_hi] adds
                               nothing to the loss or the gradient (it still counts in N) */
} mc_token_mode_t;

/* Parameters of the objective (host struct). */
typedef struct {
  float eps_low;            /* lower clip width of Eq. 5/17; ratio >= 1-eps_low, 0 <= eps_low < 1 */
  float eps_high;           /* upper clip width; ratio <= 1+eps_high, eps_high >= 0 */
  float delta;              /* filter threshold in log-ratio space (Eq. 21), >= 0 */
  float adv_eps;            /* epsilon added to the group std (Eq. 3), >= 0 */
  int32_t std_ddof;         /* 0: population std, 1: sample std */
  int32_t filter;           /* an mc_filter_t */
  float kl_beta;            /* weight beta of the KL term of Eq. 5/17 (>= 0); used only
                               when a reference log-prob array is passed */
  int32_t token_mode;       /* an mc_token_mode_t */
  float tis_cap;            /* MC_TOKEN_TIS: cap C > 0 of the ratio (default 2) */
  float icepop_lo;          /* MC_TOKEN_ICEPOP: 0 < icepop_lo <= icepop_hi (defaults 0.5, 2); */
  float icepop_hi;          /*   ratios are compared in log space, bounds inclusive */
} mc_rl_params_t;

/* Outputs of mc_rl_loss (host struct holding device pointers).  `loss` and
 * `dlogp` are required; any other member may be NULL. */
typedef struct {
  float* loss;              /* [1]  -(1/N) sum_i M_i sum_t min(rho A_i, clip(rho) A_i) */
  float* dlogp;             /* [T]  d loss / d logp_t */
  uint8_t* seq_mask;        /* [B]  M_i */
  int32_t* seq_len;         /* [B]  L_i = number of loss-mask tokens of sequence i */
  int64_t* n_valid;         /* [1]  N = sum_i M_i L_i */
  float* adv;               /* [B]  A_i */
  float* stat_abs;          /* [B]  (1/L_i) sum_t |log rho_t|  (log of Eq. 20's statistic) */
  float* stat_signed;       /* [B]  (1/L_i) sum_t log rho_t    (log of Eq. 18's statistic) */
  float* clip_frac;         /* [1]  share of the N tokens on the clipped branch */
  int32_t* error_flag;      /* [1]  set to 1 when cu_seqlens/cu_groups are inconsistent */
  float* kl;                /* [1]  (1/N) sum_i M_i sum_t k3_t (0 without a reference) */
  float* token_frac;        /* [1]  share of the N tokens the token mode truncated (TIS)
                                    or dropped (IcePop); 0 for MC_TOKEN_NONE */
} mc_rl_outputs_t;

/* Flags of mc_logprob_bwd, mc_logprob_bwd_shard and mc_logprob_bwd_cached. */
#define MC_BWD_ACCUMULATE_DHIDDEN 1   /* dhidden += gradient instead of = */
#define MC_BWD_ACCUMULATE_DWEIGHT 2   /* dweight += gradient instead of = */
/* The two gradient contractions also leave out the products of the tokens
 * whose gradient row is zero (dlogp_t == 0 or an ignored target), which
 * are exact zeros, so the work of the whole backward scales with the
 * live tokens instead of T.  dweight is bit-identical to the result without
 * the flag; dhidden is the same up to the order of fp32 sums (a last round
 * of tiles that would leave compute units idle is split along the
 * vocabulary), still deterministic; dead tokens' rows are identical. */
#define MC_BWD_SKIP_DEAD_TOKENS 4

/* Human-readable name of a status code (static string). */
const char* mc_status_string(mc_status_t status);

/* Library version string (static). */
const char* mc_version(void);

/* ------------------------------------------------------------------------
 * Forward: per-token log-prob over the full vocabulary.
 *   logp[t] = z[t, y_t] - lse[t],  lse[t] = log sum_v exp(z[t, v]),
 *   z = hidden . weight^T,
 * i.e. log pi_theta(o_t | x, o_<t) of Eq. 4, for the token y_t the rollout
 * sampled at row t (the caller applies the next-token shift).
 *   hidden   [T, d]  dtype         activations entering the LM head
 *   weight   [V, d]  dtype         LM-head weight (one row per vocabulary entry)
 *   targets  [T]     int64         y_t; a value outside [0, V) marks an ignored
 *                                  token: logp = 0 there and it gets no gradient
 *   logp     [T]     fp32 (out)
 *   lse      [T]     fp32 (out)    kept for the backward
 *   entropy  [T]     fp32 (out)    optional (NULL to skip): -sum_v p log p of the
 *                                  row's softmax, the entropy diagnostic of the
 *                                  MirrorPop ablation (Sec. 5.4), from one extra
 *                                  running sum in the same epilogue
 * T = 0 is a valid no-op.  T >= 0, d >= 8, d % 8 == 0, V >= 1.
 * ------------------------------------------------------------------------ */
size_t mc_logprob_fwd_workspace_size(int64_t T, int64_t d, int64_t V, mc_dtype_t dtype);
mc_status_t mc_logprob_fwd(const void* hidden, const void* weight, const int64_t* targets,
                           int64_t T, int64_t d, int64_t V, mc_dtype_t dtype,
                           float* logp, float* lse, float* entropy,
                           void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Vocabulary-sharded forward (the one-GPU part of a tensor-parallel LM head,
 * Sec. 5.1): this call sees the shard weight[V_shard, d] holding vocabulary
 * entries [v_offset, v_offset + V_shard) and writes, per row, the shard's
 * partial[4][T] = (max_v z, sum_v exp(z - max), sum_v exp(z - max) z,
 * z[t, y_t] if y_t is in the shard else -inf), fp32.  Targets are global
 * indices.  Workspace: mc_logprob_fwd_workspace_size(T, d, V_shard, dtype).
 * mc_logprob_merge_shards folds S such partials (partials[S][4][T], shard
 * order; gathered from the shards by the caller) into logp, lse and
 * (optionally) entropy, exactly as the unsharded forward defines them;
 * V_total is the full vocabulary size (targets outside it are ignored).
 * ------------------------------------------------------------------------ */
mc_status_t mc_logprob_fwd_shard(const void* hidden, const void* weight_shard,
                                 const int64_t* targets, int64_t T, int64_t d, int64_t V_shard,
                                 int64_t v_offset, int64_t V_total, mc_dtype_t dtype,
                                 float* partial, void* workspace, size_t workspace_bytes,
                                 void* stream);
mc_status_t mc_logprob_merge_shards(const float* partials, int32_t S, const int64_t* targets,
                                    int64_t T, int64_t V_total, float* logp, float* lse,
                                    float* entropy, void* stream);

/* ------------------------------------------------------------------------
 * Backward of the forward above for an upstream gradient dlogp[t]:
 *   G[t, v]  = dlogp_t (1[v = y_t] - exp(z[t, v] - lse_t))   (0 for ignored t)
 *   dhidden  = G . weight      [T, d] fp32
 *   dweight  = G^T . hidden    [V, d] fp32
 *   lse      [T] fp32          as returned by mc_logprob_fwd for the same inputs
 *   dlogp    [T] fp32
 *   dhidden / dweight may be NULL to skip that gradient (not both).
 *   flags    MC_BWD_ACCUMULATE_* bits: accumulate into the outputs;
 *            MC_BWD_SKIP_DEAD_TOKENS: see its definition.
 * The softmax part is formed per vocabulary chunk as a transient operand in
 * the workspace; logits are recomputed, never stored.  They are recomputed
 * only where the gradient row can be nonzero: the tokens with dlogp_t != 0
 * and a target in [0, V) are ordered first, and the operand rows of the
 * others are read as zeros without being formed, so this step costs in
 * proportion to the live tokens (the results are the same; both gradient
 * contractions still run over all T tokens).  For MC_BF16 inputs
 * that operand and the transposed hidden and weight rows the contractions
 * read are fp16, each scaled by a power of two chosen from its magnitude
 * bound and unscaled exactly in fp32: each element of the softmax part is
 * within 2^-11 relative of its exact value (elements far below the largest
 * aside), against 2^-8 for a bf16 operand.  MC_F32 inputs use fp32
 * operands.
 * ------------------------------------------------------------------------ */
size_t mc_logprob_bwd_workspace_size(int64_t T, int64_t d, int64_t V, mc_dtype_t dtype);
mc_status_t mc_logprob_bwd(const void* hidden, const void* weight, const int64_t* targets,
                           const float* lse, const float* dlogp,
                           int64_t T, int64_t d, int64_t V, mc_dtype_t dtype,
                           float* dhidden, float* dweight, int32_t flags,
                           void* workspace, size_t workspace_bytes, void* stream);

/* Backward on a vocabulary shard (see mc_logprob_fwd_shard): with the global
 * lse of the merged forward, dhidden receives this shard's part of G . W
 * (the shards' parts sum to the full dhidden) and dweight_shard[V_shard, d]
 * the shard's rows of dW.  Workspace:
 * mc_logprob_bwd_workspace_size(T, d, V_shard, dtype). */
mc_status_t mc_logprob_bwd_shard(const void* hidden, const void* weight_shard,
                                 const int64_t* targets, const float* lse, const float* dlogp,
                                 int64_t T, int64_t d, int64_t V_shard, int64_t v_offset,
                                 int64_t V_total, mc_dtype_t dtype, float* dhidden,
                                 float* dweight_shard, int32_t flags, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Forward and backward with a softmax cache: the same quantities as
 * mc_logprob_fwd / mc_logprob_bwd (the numerator of Eq. 4 and its
 * gradient), with the backward reading what the forward kept instead of
 * recomputing the logits.  The forward stores, in `cache`,
 *   E[t, v] = exp(z[t, v] - c_b[t])   (vocabulary panels; fp16 for MC_BF16
 *                                      inputs: E lies in (0, 1] and the
 *                                      block maximum is exactly 1; fp32
 *                                      for MC_F32)
 *   c_b[t]  = max of z[t, .] over block b of 128 vocabulary entries (fp32)
 * and the backward gathers from E the softmax part of G for the tokens whose
 * gradient row can be nonzero (for MC_BF16 the recompute pair's fp16
 * operand, scaled by the same power of two) into its workspace and runs the
 * two contractions on it as mc_logprob_bwd does.  E adds one rounding before
 * the operand's own: each element of the operand is within about 2^-10
 * relative of its exact value, against 2^-11 for the recompute pair.
 *   cache     device, 256-byte aligned, at least mc_logprob_cache_size bytes;
 *             owned by the caller; written by mc_logprob_fwd_cached and
 *             read (not modified) by mc_logprob_bwd_cached calls with the
 *             same hidden, weight, targets and shapes, any number of them
 *             (several upstream gradients of one forward).
 *   The forward takes the workspace of mc_logprob_fwd
 *   (mc_logprob_fwd_workspace_size); the backward takes
 *   mc_logprob_bwd_cached_workspace_size bytes (it holds the gathered
 *   operand: about the cache's size).  Flags as for mc_logprob_bwd.  Errors
 *   as for the plain entry points; a missing or short cache returns
 *   MC_ERR_WORKSPACE.
 * ------------------------------------------------------------------------ */
size_t mc_logprob_cache_size(int64_t T, int64_t d, int64_t V, mc_dtype_t dtype);
mc_status_t mc_logprob_fwd_cached(const void* hidden, const void* weight,
                                  const int64_t* targets, int64_t T, int64_t d, int64_t V,
                                  mc_dtype_t dtype, float* logp, float* lse, float* entropy,
                                  void* cache, size_t cache_bytes, void* workspace,
                                  size_t workspace_bytes, void* stream);
size_t mc_logprob_bwd_cached_workspace_size(int64_t T, int64_t d, int64_t V, mc_dtype_t dtype);
mc_status_t mc_logprob_bwd_cached(const void* hidden, const void* weight,
                                  const int64_t* targets, const float* lse, const float* dlogp,
                                  int64_t T, int64_t d, int64_t V, mc_dtype_t dtype,
                                  void* cache, size_t cache_bytes, float* dhidden,
                                  float* dweight, int32_t flags, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * RL objective over a packed ragged batch (Eq. 3/12, 4, 17-21).
 *   logp          [T]    fp32   trainer log-probs (from mc_logprob_fwd)
 *   logp_rollout  [T]    fp32   rollout log-probs of the same tokens
 *                               (ignored where loss_mask is 0)
 *   logp_ref      [T]    fp32   reference-policy log-probs for the KL term of
 *                               Eq. 5/17, or NULL for beta = 0.  The paper
 *                               names no estimator; the term is
 *                               kl_beta * (1/N) sum_i M_i sum_t k3_t with
 *                               k3 = exp(r) - r - 1, r = logp_ref - logp
 *   loss_mask     [T]    u8     1 = token counts (e.g. first-turn response
 *                               tokens); NULL = all tokens count
 *   cu_seqlens    [B+1]  int32  sequence i is rows [cu_seqlens[i], cu_seqlens[i+1]);
 *                               cu_seqlens[0] = 0, non-decreasing, cu_seqlens[B] = T
 *   cu_groups     [NG+1] int32  group g is sequences [cu_groups[g], cu_groups[g+1]);
 *                               cu_groups[0] = 0, non-decreasing, cu_groups[NG] = B
 *   rewards       [B]    fp32   r_i (or a trajectory reward, Eq. 9)
 * The loss is one token mean over the whole batch, N = sum_i M_i L_i; N = 0
 * gives loss 0 and dlogp 0.  A sequence with L_i = 0 has M_i = 0.  The packing
 * arrays live on the device and are checked there: inconsistent values never
 * cause an out-of-bounds access; they set *error_flag (when given) and the
 * outputs are then unspecified.  mc_check_packing validates host copies.
 * ------------------------------------------------------------------------ */
size_t mc_rl_loss_workspace_size(int64_t T, int32_t B, int32_t NG);
mc_status_t mc_rl_loss(const float* logp, const float* logp_rollout, const float* logp_ref,
                       const uint8_t* loss_mask,
                       const int32_t* cu_seqlens, const int32_t* cu_groups,
                       const float* rewards, int64_t T, int32_t B, int32_t NG,
                       const mc_rl_params_t* params, const mc_rl_outputs_t* out,
                       void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * mc_rl_loss without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation).  Same arguments, outputs and results as
 * mc_rl_loss (the same kernels), but its scratch is a fixed device array of
 * MC_RL_LOSS_NOALLOC_SCRATCH_BYTES (4 MiB) inside the library, one copy per
 * GPU, held until the process ends; the call itself allocates nothing.
 *   Limit     mc_rl_loss_workspace_size(T, B, NG) must not exceed
 *             mc_rl_loss_noalloc_max_bytes() (= the array size; it fits
 *             B <= 65536 sequences in at most 65536 groups, any T);
 *             larger batches return MC_ERR_UNSUPPORTED and enqueue nothing.
 *   Stream    must belong to the current device (else MC_ERR_INVALID_ARG).
 *   Races     every call on one GPU shares that GPU's array: calls whose
 *             work may overlap on one GPU (other host threads, other
 *             streams) race and must be serialised by the caller.  The
 *             array keeps the last call's contents; every value the kernels
 *             read is written earlier in the same call.
 * ------------------------------------------------------------------------ */
#define MC_RL_LOSS_NOALLOC_SCRATCH_BYTES ((size_t)4 << 20)
size_t mc_rl_loss_noalloc_max_bytes(void);
mc_status_t mc_rl_loss_noalloc(const float* logp, const float* logp_rollout,
                               const float* logp_ref, const uint8_t* loss_mask,
                               const int32_t* cu_seqlens, const int32_t* cu_groups,
                               const float* rewards, int64_t T, int32_t B, int32_t NG,
                               const mc_rl_params_t* params, const mc_rl_outputs_t* out,
                               void* stream);

/* PrimeEcho trajectory rewards (Sec. 4.4.3, Eq. 9-10), one per trajectory:
 *   R_i = alpha s_i1 + (1 - alpha) max_{k <= K_i} s_ik
 *         + beta1 [success_i1] + beta2 [not success_i1 and success_i2]
 *   scores   [B][Kmax] fp32   turn scores s_ik
 *   success  [B][Kmax] u8     turn verified (NULL: no early-success bonus)
 *   n_turns  [B]       int32  K_i, clamped into [1, Kmax] (NULL: all Kmax)
 *   rewards  [B]       fp32 (out), to pass to mc_rl_loss (Eq. 12)
 * 0 <= alpha <= 1 (the paper's default is 0.75), beta1, beta2 finite. */
mc_status_t mc_primeecho_rewards(const float* scores, const uint8_t* success,
                                 const int32_t* n_turns, int32_t B, int32_t Kmax, float alpha,
                                 float beta1, float beta2, float* rewards, void* stream);

/* Host-side check of packing metadata (host arrays): MC_OK when cu_seqlens and
 * cu_groups satisfy the rules stated for mc_rl_loss, MC_ERR_INVALID_ARG
 * otherwise.  Makes no HIP call. */
mc_status_t mc_check_packing(const int32_t* cu_seqlens_host, int32_t B,
                             const int32_t* cu_groups_host, int32_t NG, int64_t T);

/* ------------------------------------------------------------------------
 * Per-kernel timing, a measurement aid (the one piece of global state).
 * mc_profiler_enable(1) makes every later launch record a pair of hipEvents
 * on its own stream, tagged with the kernel name and its algorithmic FLOPs
 * and bytes (what the method must compute and move, not what the
 * implementation moves).  mc_profiler_read waits for the recorded events,
 * adds them into per-name totals and copies up to `cap` totals into `out`
 * (host array); it returns the number of names.  mc_profiler_reset clears
 * the totals.  Thread-safe; enabling costs one event pair per launch.
 * ------------------------------------------------------------------------ */
typedef struct {
  char name[48];
  int64_t launches;
  double total_ms;
  double total_flops;
  double total_bytes;
} mc_kernel_time_t;

void mc_profiler_enable(int32_t on);
void mc_profiler_reset(void);
int32_t mc_profiler_read(mc_kernel_time_t* out, int32_t cap);

#ifdef __cplusplus
}
#endif

#endif /* MC_H_ */
