// Fused LM-head log-prob on gfx950: forward (GEMM + online log-sum-exp +
// target gather in the epilogue, optionally keeping a softmax cache), the
// partial merge, and the backward: the scaled softmax operand (from the cache,
// normalised in place, or from recomputed logits) -> two contractions, plus
// the exact one-hot terms in fp32 (dH's in its contraction's epilogue, dW's
// by a deterministic bucketed scatter).
#include <hip/hip_runtime.h>

#include <numeric>
#include <type_traits>

#include "mc_internal.hpp"
#include "mc_tile.hpp"

namespace mc {

namespace {

constexpr float kLog2e = 1.4426950408889634f;

// Integer clamp (the device min/max overloads of int64 go through fp64).
__device__ __forceinline__ int clamp_rows(int64_t n, int hi) {
  return n <= 0 ? 0 : (n >= hi ? hi : int(n));
}
constexpr float kNegInf = -__builtin_huge_valf();

// Combine x over the four lanes l % 16 + 16 g (g = 0..3): the four 16-lane
// groups of a 16 x 16 accumulator block hold rows 4 g .. 4 g + 3 of the same
// column.  With both operands equal, v_permlane32_swap leaves
// (x[l % 32], x[l % 32 + 32]) in every lane, and v_permlane16_swap the pair
// (x[l], x[l ^ 16]) ordered by row parity.
__device__ __forceinline__ float quad_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x),
                                                  __builtin_bit_cast(uint32_t, x), false, false);
  const float y = fmaxf(__builtin_bit_cast(float, uint32_t(r[0])),
                        __builtin_bit_cast(float, uint32_t(r[1])));
  const auto q = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, y),
                                                  __builtin_bit_cast(uint32_t, y), false, false);
  return fmaxf(__builtin_bit_cast(float, uint32_t(q[0])), __builtin_bit_cast(float, uint32_t(q[1])));
}
__device__ __forceinline__ float quad_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x),
                                                  __builtin_bit_cast(uint32_t, x), false, false);
  const float y = __builtin_bit_cast(float, uint32_t(r[0])) + __builtin_bit_cast(float, uint32_t(r[1]));
  const auto q = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, y),
                                                  __builtin_bit_cast(uint32_t, y), false, false);
  return __builtin_bit_cast(float, uint32_t(q[0])) + __builtin_bit_cast(float, uint32_t(q[1]));
}

// Row (within the wave's kWaveRows) of accumulator element e of block i in
// this lane.
__device__ __forceinline__ int wrow(int i, int e, int lane) {
  return i * 16 + 4 * (lane >> 4) + e;
}

// ---------------------------------------------------------------------------
// A 256 x 256 bf16 tile (rows: 256 vocabulary entries of a chunk, columns:
// 256 tokens) staged in the workgroup's LDS operand buffers for stores of
// whole panel rows: four 32 KiB panels (64 vocabulary entries each) of 256
// token rows x 128 bytes.  A lane stages 4 consecutive vocabulary entries of
// one token (8 bytes, half of a 16-byte chunk); the 16 lanes of one such
// write hold 16 consecutive tokens.  The chunk index is XOR-ed with
// (t >> 1) & 7 and the chunk's two 8-byte halves are swapped when
// (t ^ (t >> 1)) & 1: the 16 tokens of a lane group then cover 16 distinct
// (chunk, half) slots, i.e. all 32 banks of a 128-byte row pair, and the 32
// lanes of two groups all 64 banks of the two rows they touch (XOR-ing the
// chunk with t & 7 alone put tokens t and t + 8 on the same banks, and
// (t >> 1) & 7 alone tokens t and t ^ 1: 1023 conflict cycles per tile
// counted).  The reader swaps the halves back.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int panel_swz(int t) { return (t >> 1) & 7; }
__device__ __forceinline__ int panel_half(int t) { return (t ^ (t >> 1)) & 1; }
__device__ __forceinline__ int panel_stage_off(int v, int t) {
  return (v >> 6) * 32768 + t * 128 + ((((v & 63) >> 3) ^ panel_swz(t)) << 4) +
         ((((v >> 2) & 1) ^ panel_half(t)) << 3) + ((v & 3) << 1);
}

// Each panel's 256 token rows are 32 KiB of contiguous memory: 16-byte
// stores, eight lanes per 128-byte row, non-temporal (the operand is far
// larger than the caches and next read by another kernel).  Rows t >= Tn
// and chunk columns >= ld are skipped.  The caller has synchronised after
// staging.  A thread's chunks are all read from the LDS first and then
// stored, from one base address per thread: as a loop of read, wait, store
// (with 64-bit address arithmetic in each step) this took most of the
// cache's cost in the forward.
template <typename TP>   // a 2-byte element type
__device__ __forceinline__ void store_staged_panels(const char* lds, TP* P, int64_t m0,
                                                    int64_t n0, int64_t Tn, int64_t ld,
                                                    int64_t pld) {
  constexpr int64_t kPanel = 64;
  constexpr int kRows = kThreads / 8;            // token rows per round
  constexpr int kRounds = 256 / kRows;           // rounds per panel
  constexpr int kIters = 4 * kRounds;
  static_assert(kRows % 16 == 0, "the swizzle of row r0 + kRows k is that of r0");
  const int ch = threadIdx.x & 7, r0 = threadIdx.x >> 3;
  const int sw = (ch ^ panel_swz(r0)) << 4;
  const bool swap = panel_half(r0) != 0;
  u32x4 v[kIters];
#pragma unroll
  for (int it = 0; it < kIters; ++it) {
    const u32x4 x = *reinterpret_cast<const u32x4*>(lds + (it / kRounds) * 32768 +
                                                    ((it % kRounds) * kRows + r0) * 128 + sw);
    v[it] = swap ? u32x4{x[2], x[3], x[0], x[1]} : x;
  }
  TP* const base = P + (m0 / kPanel) * pld * kPanel + (n0 + r0) * kPanel + ch * 8;
#pragma unroll
  for (int it = 0; it < kIters; ++it) {
    const int pn = it / kRounds, tl = (it % kRounds) * kRows + r0;
    if (n0 + tl < Tn && m0 + pn * kPanel < ld)
      __builtin_nontemporal_store(
          v[it], reinterpret_cast<u32x4*>(base + pn * pld * kPanel +
                                          int64_t((it % kRounds) * kRows) * kPanel));
  }
}

// ---------------------------------------------------------------------------
// Forward epilogue.  The tile's rows are vocabulary entries (M) and its
// columns tokens (N), so each lane holds, for each of its kTN token columns,
// 32 of the wave's 128 vocabulary rows and the three lanes l ^ 16, l ^ 32,
// l ^ 48 the other 96.  Per token: max, sum of exp and (optionally) sum of exp * z over the
// tile's valid rows -> one (m, s, u) partial per (vocab tile, token); the
// target logit z[t, y_t] is written by the one lane that holds it.  The
// weight may be a vocabulary shard: row r of this launch is vocabulary entry
// v_off + r.
// With a softmax cache (E non-null) the epilogue also keeps what the
// backward needs instead of recomputing the logits: E[t, v] =
// exp(z_tv - cm[b][t]) in TE (fp16 for bf16 inputs: the values lie in
// (0, 1], the block maximum is exactly 1, and fp16 keeps 11 significant bits
// against bf16's 8; fp32 for fp32 inputs), in the panel layout of the
// backward operand, where cm[b][t] is the max over the wave's block b of 128
// vocabulary rows (zero for rows >= Vs).
// ---------------------------------------------------------------------------
template <typename T, typename TE = T>   // TE: the softmax cache's element type
struct EpiFwd {
  const int64_t* y;
  int64_t Tn, Vs, v_off;  // tokens, shard width, shard offset
  float* part_m;          // [nTv][Tn]
  float* part_s;          // [nTv][Tn]
  float* part_u;          // [nTv][Tn] or null (no entropy)
  float* zy;              // [Tn]: receives z[t, y_t] for targets inside the shard
  TE* E;                  // softmax cache: panels [ldE / BV][pld][BV], or null
  float* cm;              // [2 nTv][Tn] block maxima (with E)
  int64_t pld, ldE;       // padded token count, padded vocabulary width
  static constexpr int kLdsExtra = 3 * kWavesM * 256 * 4;
  static constexpr int64_t kPanel = 128 / sizeof(TE);

  // this lane's targets (shard-local, -1 outside the shard) of its kTN
  // token columns
  struct Pre {
    int y[kTN];
  };
  __device__ __forceinline__ Pre prologue(int64_t, int64_t n0) const {
    Pre p;
    const int lane = threadIdx.x & 63, wn = wave_n();
#pragma unroll
    for (int j = 0; j < kTN; ++j) {
      const int64_t t = n0 + wn * kWaveCols + j * 16 + (lane & 15);
      p.y[j] = -1;
      if (t < Tn) {
        const int64_t yl = y[t] - v_off;
        if (yl >= 0 && yl < Vs) p.y[j] = int(yl);
      }
    }
    return p;
  }

  // max / sum exp / sum exp z of block column j over this lane's rows; kFull:
  // all rows of the wave are valid (no per-element mask); kStore: also the
  // softmax cache values of these rows (staged in LDS for a 2-byte cache)
  template <bool kFull, bool kStore>
  __device__ __forceinline__ void column(const Acc& acc, int j, int vlim, int lane, bool with_u,
                                         float& mx, float& s, float& u, char* lds, int wm,
                                         int tl, int64_t m0, int64_t t) const {
    mx = kNegInf;
#pragma unroll
    for (int i = 0; i < kTM; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (kFull || wrow(i, e, lane) < vlim) mx = fmaxf(mx, acc[i][j][e]);
    mx = quad_max(mx);
    const float mb = mx * kLog2e;
    s = 0.0f;
    u = 0.0f;
#pragma unroll
    for (int i = 0; i < kTM; ++i) {
      f32x4 xs;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        xs[e] = 0.0f;
        if (kFull || wrow(i, e, lane) < vlim) {
          const float x = __builtin_amdgcn_exp2f(fmaf(acc[i][j][e], kLog2e, -mb));
          s += x;
          if (with_u) u = fmaf(x, acc[i][j][e], u);
          xs[e] = x;
        }
      }
      if constexpr (kStore) {
        const int vr = wm * kWaveRows + wrow(i, 0, lane);   // tile row of element 0
        if constexpr (sizeof(TE) == 2) {
          typedef TE te4 __attribute__((ext_vector_type(4)));
          *reinterpret_cast<u32x2*>(lds + panel_stage_off(vr, tl)) =
              __builtin_bit_cast(u32x2, __builtin_convertvector(xs, te4));
        } else {
          const int64_t c = m0 + vr;
          if (t < Tn && c < ldE)
            *reinterpret_cast<f32x4*>(E + (c / kPanel) * pld * kPanel + t * kPanel + c % kPanel) =
                xs;
        }
      }
    }
    s = quad_sum(s);
    if (with_u) u = quad_sum(u);
  }

  __device__ __forceinline__ void epilogue(Acc& acc, int tm, int, int64_t m0, int64_t n0,
                                          char* lds, char* extra, const Pre& pre) const {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wm = wave_m(), wn = wave_n();
    float* red = reinterpret_cast<float*>(extra);   // [m|s|u][wm][token]
    const int64_t rbase = m0 + wm * kWaveRows;              // first vocab row of this wave
    const int vlim = clamp_rows(Vs - rbase, kWaveRows);
    const bool with_u = part_u != nullptr;
#pragma unroll
    for (int j = 0; j < kTN; ++j) {
      const int tl = wn * kWaveCols + j * 16 + (lane & 15);   // token within the tile
      const int64_t t = n0 + tl;
      float mx, s, u;
      if (E != nullptr) {
        if (vlim >= kWaveRows)
          column<true, true>(acc, j, vlim, lane, with_u, mx, s, u, lds, wm, tl, m0, t);
        else
          column<false, true>(acc, j, vlim, lane, with_u, mx, s, u, lds, wm, tl, m0, t);
        if (lane < 16 && t < Tn) cm[(int64_t(tm) * kWavesM + wm) * Tn + t] = mx;
      } else {
        if (vlim >= kWaveRows)
          column<true, false>(acc, j, vlim, lane, with_u, mx, s, u, lds, wm, tl, m0, t);
        else
          column<false, false>(acc, j, vlim, lane, with_u, mx, s, u, lds, wm, tl, m0, t);
      }
      // target logit: row yw of this wave, held by the lane of group (yw >> 2) & 3
      const int yw = pre.y[j] - int(rbase);
      if (yw >= 0 && yw < kWaveRows && ((yw >> 2) & 3) == (lane >> 4)) {
        const int ii = yw >> 4, ee = yw & 3;
        float z = 0.0f;
#pragma unroll
        for (int i = 0; i < kTM; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (i == ii && e == ee) z = acc[i][j][e];
        zy[n0 + tl] = z;
      }
      if (lane < 16) {
        red[(0 * kWavesM + wm) * 256 + tl] = mx;
        red[(1 * kWavesM + wm) * 256 + tl] = s;
        red[(2 * kWavesM + wm) * 256 + tl] = u;
      }
    }
    __syncthreads();
    if constexpr (sizeof(TE) == 2)
      if (E != nullptr) store_staged_panels(lds, E, m0, n0, Tn, ldE, pld);
    for (int tl = tid; tl < kBN; tl += kThreads) {
      const int64_t t = n0 + tl;
      if (t >= Tn) continue;
      float M = red[tl];
#pragma unroll
      for (int w = 1; w < kWavesM; ++w) M = fmaxf(M, red[w * 256 + tl]);
      float S = 0.0f, U = 0.0f;
#pragma unroll
      for (int w = 0; w < kWavesM; ++w) {
        const float mw = red[w * 256 + tl];
        if (mw != kNegInf) {
          const float f = __builtin_amdgcn_exp2f((mw - M) * kLog2e);
          S += red[(kWavesM + w) * 256 + tl] * f;
          U += red[(2 * kWavesM + w) * 256 + tl] * f;
        }
      }
      part_m[int64_t(tm) * Tn + t] = M;
      part_s[int64_t(tm) * Tn + t] = S;
      if (with_u) part_u[int64_t(tm) * Tn + t] = U;
    }
  }
};

// Running (max, sum exp, sum exp * z) triple, folded in a fixed order.
struct Lse3 {
  float m = kNegInf, s = 0.0f, u = 0.0f;
  __device__ void add(float m2, float s2, float u2) {
    if (m2 == kNegInf) return;
    if (m2 > m) {
      const float f = expf(m - m2);
      s = s * f + s2;
      u = u * f + u2;
      m = m2;
    } else {
      const float f = expf(m2 - m);
      s += s2 * f;
      u += u2 * f;
    }
  }
};

// Fold the per-vocab-tile partials of 64 rows in tile order: 8 waves stride
// over the tiles, then wave 0 folds the 8 running triples in order.
__device__ __forceinline__ Lse3 fold_tiles(const float* __restrict__ pm,
                                           const float* __restrict__ ps,
                                           const float* __restrict__ pu, int nT, int64_t T,
                                           int64_t t, float (*sh)[8][64]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  Lse3 acc;
  if (t < T) {
    // four tiles' partials are loaded before they are folded (same order)
    int j = w;
    for (; j + 24 < nT; j += 32) {
      float m4[4], s4[4], u4[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t o = int64_t(j + 8 * q) * T + t;
        m4[q] = pm[o];
        s4[q] = ps[o];
        u4[q] = pu ? pu[o] : 0.0f;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) acc.add(m4[q], s4[q], u4[q]);
    }
    for (; j < nT; j += 8) {
      const int64_t o = int64_t(j) * T + t;
      acc.add(pm[o], ps[o], pu ? pu[o] : 0.0f);
    }
  }
  sh[0][w][lane] = acc.m;
  sh[1][w][lane] = acc.s;
  sh[2][w][lane] = acc.u;
  __syncthreads();
  Lse3 out;
  if (w == 0)
    for (int k = 0; k < 8; ++k) out.add(sh[0][k][lane], sh[1][k][lane], sh[2][k][lane]);
  return out;
}

// Final merge: lse = m + log s, logp = z_y - lse (0 for an ignored target),
// entropy = lse - u / s (the expectation of z under the softmax).
__global__ __launch_bounds__(512) void k_lse_merge(const float* __restrict__ pm,
                                                   const float* __restrict__ ps,
                                                   const float* __restrict__ pu, int nT,
                                                   int64_t T, const int64_t* __restrict__ y,
                                                   int64_t V, float* __restrict__ logp,
                                                   float* __restrict__ lse,
                                                   float* __restrict__ entropy) {
  __shared__ float sh[3][8][64];
  const int64_t t = int64_t(blockIdx.x) * 64 + (threadIdx.x & 63);
  const Lse3 r = fold_tiles(pm, ps, pu, nT, T, t, sh);
  if ((threadIdx.x >> 6) == 0 && t < T) {
    const float l = r.m + logf(r.s);
    lse[t] = l;
    const int64_t yy = y[t];
    logp[t] = (yy >= 0 && yy < V) ? logp[t] - l : 0.0f;
    if (entropy) entropy[t] = l - r.u / r.s;
  }
}

// Shard partial: (m, s, u, z_y or -inf) of this vocabulary shard per row,
// part = [4][T]; z_y was written into part[3] by the GEMM epilogue.
__global__ __launch_bounds__(512) void k_shard_partial(const float* __restrict__ pm,
                                                       const float* __restrict__ ps,
                                                       const float* __restrict__ pu, int nT,
                                                       int64_t T, const int64_t* __restrict__ y,
                                                       int64_t v_off, int64_t Vs,
                                                       float* __restrict__ part) {
  __shared__ float sh[3][8][64];
  const int64_t t = int64_t(blockIdx.x) * 64 + (threadIdx.x & 63);
  const Lse3 r = fold_tiles(pm, ps, pu, nT, T, t, sh);
  if ((threadIdx.x >> 6) == 0 && t < T) {
    part[t] = r.m;
    part[T + t] = r.s;
    part[2 * T + t] = r.u;
    const int64_t yl = y[t] - v_off;
    if (!(yl >= 0 && yl < Vs)) part[3 * T + t] = kNegInf;
  }
}

// Merge of S shard partials (shard order) into lse, logp and entropy.
__global__ __launch_bounds__(256) void k_shard_merge(const float* __restrict__ parts, int S,
                                                     int64_t T, const int64_t* __restrict__ y,
                                                     int64_t V, float* __restrict__ logp,
                                                     float* __restrict__ lse,
                                                     float* __restrict__ entropy) {
  const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= T) return;
  Lse3 r;
  float zy = kNegInf;
  for (int k = 0; k < S; ++k) {
    const float* p = parts + int64_t(k) * 4 * T;
    r.add(p[t], p[T + t], p[2 * T + t]);
    zy = fmaxf(zy, p[3 * T + t]);
  }
  const float l = r.m + logf(r.s);
  lse[t] = l;
  const int64_t yy = y[t];
  logp[t] = (yy >= 0 && yy < V) ? zy - l : 0.0f;
  if (entropy) entropy[t] = l - r.u / r.s;
}

// ---------------------------------------------------------------------------
// Power-of-two scales of the recompute backward's fp16 operands.  The
// transient operand and the transposed W and H are fp16 there (11 significant
// bits against bf16's 8), so each needs its magnitudes inside fp16's range;
// scaling by a power of two (ldexp: exact for any finite value that stays in
// range) loses nothing, and the contractions' epilogues undo it exactly.  A
// magnitude bound travels as the bits of a non-negative float in an unsigned
// word (atomicMax orders them like the floats); a scale travels as its
// exponent, since the one dlogp near fp32's smallest values needs is beyond
// fp32's largest.
// ---------------------------------------------------------------------------
// e with bound = m 2^e, 0.5 <= m < 1, from the bits alone (subnormal bounds
// included, whatever the denormal mode); bits != 0.
__device__ __forceinline__ int bound_exponent(unsigned bits) {
  const int ef = int(bits >> 23);
  if (ef > 0) return ef - 126;
  return (32 - __builtin_clz(bits)) - 149;   // m 2^-149 with m < 2^23
}
// -dlogp * softmax: magnitudes up to max |dlogp|, scaled below 2^14.
__device__ __forceinline__ int probs_shift(unsigned bits) {
  return (bits == 0u || bits >= 0x7f800000u) ? 0 : 14 - bound_exponent(bits);
}
// W and H: left unscaled while their bound lies in [2^-4, 2^15) (so the largest
// converts to a finite fp16 value and values down to 2^-10 of it stay normal),
// else scaled below 2^14.
__device__ __forceinline__ int operand_shift(unsigned bits) {
  if (bits == 0u || bits >= 0x7f800000u) return 0;
  const int e = bound_exponent(bits);
  return (e >= -3 && e <= 15) ? 0 : 14 - e;
}
// Undoes the shifts probs_shift(*bp) and operand_shift(*bo), one at a time
// (their sum alone can leave fp32's exponent range while the result does
// not).  Null bp: nothing to undo.
struct Unscale {
  int a, b;
  __device__ __forceinline__ Unscale(const unsigned* bp, const unsigned* bo) {
    a = bp != nullptr ? -probs_shift(*bp) : 0;
    b = bp != nullptr ? -operand_shift(*bo) : 0;
  }
  __device__ __forceinline__ f32x4 operator()(f32x4 v) const {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = ldexpf(ldexpf(v[e], a), b);
    return v;
  }
};
// Raise *bound to x (>= 0) unless it is already at least x: after a few
// workgroups the bound is rarely exceeded, so few atomics reach memory.
__device__ __forceinline__ void raise_bound(unsigned* bound, float x) {
  const unsigned b = __float_as_uint(x);
  if (b > *reinterpret_cast<volatile unsigned*>(bound)) atomicMax(bound, b);
}
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x = fmaxf(x, __shfl_xor(x, m));
  return x;
}

// ---------------------------------------------------------------------------
// Backward, step 1: recompute the logits of a vocabulary chunk (tile rows =
// chunk columns v, tile columns = tokens t) and write the transient operand
// P~[t, v] = -dlogp_t exp(z_tv - lse_t) (zero for ignored tokens and for the
// padding columns [width, ld)) in the panel layout.  A lane holds 4
// consecutive v of one token per accumulator block.  bf16: the tile is staged in
// the (then idle) LDS operand buffers and written as whole 128-byte panel
// rows; fp32: 4-element stores straight to memory.
// ---------------------------------------------------------------------------
// TP: the operand's type (fp16 for bf16 inputs, shifted by probs_shift of the
// max |dlogp| bound when `bound` is set; the input type otherwise).
template <typename T, typename TP = T>
struct EpiProbs {
  const int64_t* y;
  const float* lse;
  const float* dlogp;
  int64_t Tn, V, width, ld, pld;   // V: full vocabulary (target validity); ld: padded chunk
                                   // width; pld: padded token count
  TP* P;                           // panel layout (see Lay::TileTK)
  const unsigned* bound;           // max |dlogp| (fp16 operand) or null
  // Tile columns, and P~'s rows, are positions in the live-first token
  // order (k_live_perm): the B operand holds the row of token perm[j] at
  // position j.  The tiles of positions from *nlive on hold no live token
  // and are not computed (k_bwd_probs): the contractions that read P~ read
  // its rows from *nlive on as zeros.  Null: positions are tokens.
  const int* perm;
  const int* nlive;
  static constexpr int64_t kPanel = 128 / sizeof(TP);

  __device__ __forceinline__ int64_t token(int64_t j) const {
    return perm != nullptr ? int64_t(perm[j]) : j;
  }

  // lse_t log2(e) and -dlogp_t (0 for ignored tokens) of the tokens of this
  // lane's kTN columns
  struct Pre {
    float l2[kTN], g[kTN];
  };
  __device__ __forceinline__ Pre prologue(int64_t, int64_t n0) const {
    Pre p;
    const int lane = threadIdx.x & 63, wn = wave_n();
    const int sh = bound != nullptr ? probs_shift(*bound) : 0;
#pragma unroll
    for (int j = 0; j < kTN; ++j) {
      const int64_t pos = n0 + wn * kWaveCols + j * 16 + (lane & 15);
      p.l2[j] = 0.0f;
      p.g[j] = 0.0f;
      if (pos < Tn) {
        const int64_t t = token(pos), yy = y[t];
        p.l2[j] = lse[t] * kLog2e;
        p.g[j] = (yy >= 0 && yy < V) ? ldexpf(-dlogp[t], sh) : 0.0f;
      }
    }
    return p;
  }

  // P~ of this lane's elements.  vlim: valid rows (v < width) of the wave,
  // llim: rows below ld (a multiple of 4); kFull: all kWaveRows rows valid.
  template <bool kFull>
  __device__ __forceinline__ void values(const Acc& acc, char* lds, int lane, int wm, int wn,
                                         const Pre& pre, int vlim, int llim, int64_t m0,
                                         int64_t n0) const {
#pragma unroll
    for (int j = 0; j < kTN; ++j) {
      const int tl = wn * kWaveCols + j * 16 + (lane & 15);
      const int64_t pos = n0 + tl;   // position of the column's token
      const float lb = pre.l2[j], gs = pre.g[j];
      // Whether any of the column block's 16 tokens has a nonzero factor
      // (wave-uniform).  A block of tokens with zero dlogp (outside the loss
      // mask, filtered, clipped, ignored) has an all-zero operand: its zeros
      // are written without evaluating the exponentials.
      const bool live = __builtin_amdgcn_ballot_w64(pos < Tn && gs != 0.0f) != 0;
      if (pos >= Tn) continue;
#pragma unroll
      for (int i = 0; i < kTM; ++i) {
        {
          const int r = wrow(i, 0, lane);   // first of the 4 consecutive rows of block i
          if (!kFull && r >= llim) continue;
          f32x4 p = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
          if (live) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              p[e] = gs * __builtin_amdgcn_exp2f(fmaf(acc[i][j][e], kLog2e, -lb));
              if (!kFull && r + e >= vlim) p[e] = 0.0f;
            }
          }
          const int vr = wm * kWaveRows + r;   // row of the tile
          if constexpr (sizeof(TP) == 2) {
            typedef TP tp4 __attribute__((ext_vector_type(4)));
            *reinterpret_cast<u32x2*>(lds + panel_stage_off(vr, tl)) =
                __builtin_bit_cast(u32x2, __builtin_convertvector(p, tp4));
          } else {
            const int64_t c = m0 + vr;
            TP* dst = P + (c / kPanel) * pld * kPanel + pos * kPanel + c % kPanel;
            *reinterpret_cast<f32x4*>(dst) = p;
          }
        }
      }
    }
  }

  __device__ __forceinline__ void epilogue(Acc& acc, int, int, int64_t m0, int64_t n0,
                                          char* lds, char*, const Pre& pre) const {
    const int lane = threadIdx.x & 63;
    const int wm = wave_m(), wn = wave_n();
    const int64_t rb = m0 + wm * kWaveRows;
    const int vlim = clamp_rows(width - rb, kWaveRows);
    const int llim = clamp_rows(ld - rb, kWaveRows);
    if (vlim == kWaveRows)
      values<true>(acc, lds, lane, wm, wn, pre, vlim, llim, m0, n0);
    else
      values<false>(acc, lds, lane, wm, wn, pre, vlim, llim, m0, n0);
    if constexpr (sizeof(TP) == 2) {
      __syncthreads();
      store_staged_panels(lds, P, m0, n0, Tn, ld, pld);
    }
  }
};

// dH tile epilogue (rows: tokens, columns: hidden dimensions): stores (or
// adds) the tile, plus the one-hot part of G W when W is set:
//   dH[t, c] (+)= tile[t, c] + dlogp_t W[y_t - v_off, c]   (y_t in the shard)
// in that order, all in fp32.
template <typename T>
struct EpiDH {
  float* C;
  int64_t ldc, rows, cols;
  int accumulate;
  const T* W;   // [Vs x ldc] weight shard, or null: no one-hot part here
  const int64_t* y;
  const float* dlogp;
  int64_t v_off, Vs;
  // fp16 operands: bounds of max |dlogp| and of this chunk's W rows; the
  // tile's shifts (probs_shift, operand_shift) are undone first (powers of
  // two: exact).  Null: unscaled operands.
  const unsigned* bound_p;
  const unsigned* bound_w;
  // Tile rows are positions in the live-first token order: row r of the tile
  // is dH's row perm[r].  Null: rows are tokens.
  const int* perm;

  struct Pre {};
  __device__ __forceinline__ Pre prologue(int64_t, int64_t) const { return Pre{}; }
  // The tile goes out through the LDS in kWavesM passes of one wave row
  // (128 token rows x 256 columns of fp32, 128 KiB): the waves of that row
  // write their values to it (the 16-byte chunk index XOR-ed with the row, so
  // the rows 4 apart that one write instruction touches hit distinct banks),
  // then every wave stores whole 1 KiB row segments of dH, adding the stored
  // value and the one-hot part in the same order as before (0.2 ms of dH's
  // time went to its 4-byte stores).
  __device__ __forceinline__ void epilogue(Acc& acc, int, int, int64_t m0, int64_t n0, char* lds,
                                          char*, const Pre& = Pre{}) const {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wm = wave_m(), wn = wave_n();
    const Unscale us(bound_p, bound_w);
    constexpr int kChunks = kBN / 4;               // 16-byte chunks per staged row
    constexpr int kIters = kWaveRows * kChunks / kThreads;
    static_assert(kWaveRows * kChunks * 16 <= kLdsGemm, "staging");
    static_assert(kIters * kThreads == kWaveRows * kChunks, "whole rounds");
#pragma unroll
    for (int h = 0; h < kWavesM; ++h) {
      if (wm == h) {
#pragma unroll
        for (int i = 0; i < kTM; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int rl = i * 16 + 4 * (lane >> 4) + e;
#pragma unroll
            for (int j = 0; j < kTN; ++j) {
              const int cl = wn * kWaveCols + j * 16 + (lane & 15);
              *reinterpret_cast<float*>(lds + rl * (kChunks * 16) +
                                        (((cl >> 2) ^ (rl & 15)) << 4) + ((cl & 3) << 2)) =
                  acc[i][j][e];
            }
          }
      }
      __syncthreads();
#pragma unroll
      for (int it = 0; it < kIters; ++it) {
        const int q = tid + it * kThreads, rl = q / kChunks, c4 = q % kChunks;
        const int64_t r = m0 + h * kWaveRows + rl, c = n0 + 4 * c4;
        if (r >= rows || c >= cols) continue;   // cols and ldc are multiples of 4
        f32x4 v = *reinterpret_cast<const f32x4*>(lds + rl * (kChunks * 16) +
                                                  ((c4 ^ (rl & 15)) << 4));
        v = us(v);
        const int64_t t = perm != nullptr ? int64_t(perm[r]) : r;
        float* o = C + t * ldc + c;
        if (accumulate) v += *reinterpret_cast<const f32x4*>(o);
        if (W != nullptr) {
          const int64_t yy = y[t] - v_off;
          if (yy >= 0 && yy < Vs) {
            const float g = dlogp[t];
            const T* w = W + yy * ldc + c;
#pragma unroll
            for (int k = 0; k < 4; ++k) v[k] += g * float(w[k]);
          }
        }
        *reinterpret_cast<f32x4*>(o) = v;
      }
      if (h + 1 < kWavesM) __syncthreads();   // the next pass reuses the staging
    }
  }
};

// fp32 store (or accumulate) of a tile whose rows are C's columns and whose
// columns are C's rows (C[c, r] = tile[r, c], C is [cols x ldc]): each lane's
// four consecutive tile rows are 16 contiguous bytes of one row of C.
struct EpiStoreT {
  float* C;
  int64_t ldc, rows, cols;
  int accumulate;
  // fp16 operands: bounds of max |dlogp| and of H; the tile's shifts are
  // undone (exact).  Null: unscaled.
  const unsigned* bound_p = nullptr;
  const unsigned* bound_h = nullptr;

  struct Pre {};
  __device__ __forceinline__ Pre prologue(int64_t, int64_t) const { return Pre{}; }
  // The tile goes out through the LDS in two halves of 128 columns (128 KiB
  // of fp32 each): the waves holding a half write their blocks to it, a
  // 16-byte chunk per row of 4, chunk index XOR-ed with the column so the 16
  // columns of a write hit distinct banks; then every wave stores whole
  // 1 KiB row segments of C (0.67 ms of dW's epilogue went to stores of
  // 64 bytes into 16 rows each before).
  __device__ __forceinline__ void epilogue(Acc& acc, int, int, int64_t m0, int64_t n0, char* lds,
                                          char*, const Pre& = Pre{}) const {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wm = wave_m(), wn = wave_n();
    const Unscale us(bound_p, bound_h);
    constexpr int kHalf = kBN / 2;                 // columns per pass
    constexpr int kRowChunks = kBM / 4;            // 16-byte chunks per staged column
    static_assert(kHalf * kRowChunks * 16 <= kLdsGemm, "staging");
    static_assert(kWavesN % 2 == 0, "a half of the columns per pair of wave columns");
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (wn / (kWavesN / 2) == h) {
#pragma unroll
        for (int j = 0; j < kTN; ++j) {
          const int cl = (wn % (kWavesN / 2)) * kWaveCols + j * 16 + (lane & 15);
#pragma unroll
          for (int i = 0; i < kTM; ++i) {
            const int ch = (wm * kWaveRows + i * 16 + 4 * (lane >> 4)) >> 2;
            *reinterpret_cast<f32x4*>(lds + cl * (kRowChunks * 16) + ((ch ^ (cl & 15)) << 4)) =
                acc[i][j];
          }
        }
      }
      __syncthreads();
      for (int q = tid; q < kHalf * kRowChunks; q += kThreads) {
        const int cl = q / kRowChunks, ch = q % kRowChunks;
        const int64_t c = n0 + h * kHalf + cl, r = m0 + 4 * ch;
        if (c < cols && r < rows) {   // rows, ldc and r are multiples of 4
          f32x4 v = *reinterpret_cast<const f32x4*>(lds + cl * (kRowChunks * 16) +
                                                    ((ch ^ (cl & 15)) << 4));
          v = us(v);
          f32x4* o = reinterpret_cast<f32x4*>(C + c * ldc + r);
          if (accumulate) v += *o;
          *o = v;
        }
      }
      if (h == 0) __syncthreads();   // the second half reuses the staging
    }
  }
};


// bound = max |x| over n values (one wave per 64 values of a block).
__global__ __launch_bounds__(256) void k_bound_abs(const float* __restrict__ x, int64_t n,
                                                   unsigned* __restrict__ bound) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const float m = wave_max(i < n ? fabsf(x[i]) : 0.0f);
  if ((threadIdx.x & 63) == 0) raise_bound(bound, m);
}

// out[c][r] = in[r][c] for r < rows, c < cols, and out[c][r] = 0 for
// rows <= r < 64 ceil(rows / 64) (ld_out covers that padding; cols, ld_in and
// ld_out are multiples of 8).  The zero padding matters: a K-contiguous
// operand is copied in 16-byte chunks, so up to the next multiple of 8 (bf16)
// past K is read.  One wave per 64 x 64 tile (grid x over groups of 4
// column tiles, y over row tiles: consecutive workgroups read whole input
// rows; 6% faster than row tiles first), no LDS: lane (a, b) loads rows 8a .. 8a+7 of
// column chunk b (CE elements per 16 bytes), transposes the CE x CE block in
// registers and stores it as rows 8b .. of output chunk a; every 8 lanes
// cover one whole 128-byte row in each access.  Gives the backward's
// contractions over the vocabulary and over tokens operands that run along K.
// TO != TI (bf16 -> fp16): the values are converted; with `bound` the first
// pass (rescale = 0) converts unscaled and raises *bound to max |in|, and a
// second launch (rescale = 1, row tiles strided over grid y) converts again
// shifted by operand_shift(*bound) when that is not 0, and returns at once
// otherwise.
// grid y of the rescaling launch: when no rescaling is needed its
// workgroups only read the bound and return
constexpr int64_t kRescaleRows = 64;
template <typename TI, typename TO>
__global__ __launch_bounds__(256) void k_transpose(const TI* __restrict__ in, int64_t rows,
                                                   int64_t cols, int64_t ld_in,
                                                   TO* __restrict__ out, int64_t ld_out,
                                                   unsigned* __restrict__ bound, int rescale) {
  static_assert(sizeof(TI) == sizeof(TO), "same element size");
  constexpr bool kConvert = !std::is_same<TI, TO>::value;
  constexpr int CE = 16 / sizeof(TI);  // elements per 16-byte access
  constexpr int S = 64 / CE;           // lanes per 64-element row: 8 (bf16) or 16 (fp32)
  int shift = 0;
  if (rescale) {
    shift = operand_shift(*bound);
    if (shift == 0) return;
  }
  const int lane = threadIdx.x & 63;
  const int64_t c0 = (int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6)) * 64;
  if (c0 >= cols) return;
  const int64_t nby = (rows + 63) / 64;
  constexpr int kPasses = (64 / CE) * (64 / CE) / 64;   // bf16: 1, fp32: 4
  float mx = 0.0f;
  for (int64_t by = blockIdx.y; by < nby; by += gridDim.y) {
    const int64_t r0 = by * 64;
#pragma unroll
    for (int pass = 0; pass < kPasses; ++pass) {
      const int blk = pass * 64 + lane;          // CE x CE block index within the tile
      const int a = blk / S, b = blk % S;        // row block, column chunk
      const int64_t c = c0 + int64_t(b) * CE;    // first input column of the chunk
      TI v[CE][CE];
#pragma unroll
      for (int j = 0; j < CE; ++j) {
        const int64_t r = r0 + int64_t(a) * CE + j;
        u32x4 raw = {0u, 0u, 0u, 0u};
        if (r < rows && c < cols) raw = *reinterpret_cast<const u32x4*>(in + r * ld_in + c);
        *reinterpret_cast<u32x4*>(v[j]) = raw;
      }
      if (c >= cols) continue;
#pragma unroll
      for (int i = 0; i < CE; ++i) {
        TO o[CE];
#pragma unroll
        for (int j = 0; j < CE; ++j) {
          if constexpr (kConvert) {
            const float x = float(v[j][i]);
            mx = fmaxf(mx, fabsf(x));
            o[j] = TO(ldexpf(x, shift));
          } else {
            o[j] = v[j][i];
          }
        }
        *reinterpret_cast<u32x4*>(out + (c + i) * ld_out + r0 + int64_t(a) * CE) =
            *reinterpret_cast<const u32x4*>(o);
      }
    }
  }
  if constexpr (kConvert) {
    if (bound != nullptr && !rescale) {
      mx = wave_max(mx);
      if (lane == 0) raise_bound(bound, mx);
    }
  }
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o, 64);
    if (lane >= o) v += u;
  }
  return v;
}

// A token whose row of the softmax operand can be nonzero: dlogp_t != 0
// and a target in [0, V).
__device__ __forceinline__ bool token_live(int64_t yy, float g, int64_t V) {
  return g != 0.0f && yy >= 0 && yy < V;
}

// Hm[t] = H[t] for the tokens whose rows of the softmax operand can be
// nonzero (dlogp_t != 0 and a target in [0, V)), a zero row otherwise.  The
// backward's softmax contraction and the H^T operand of dW read Hm instead
// of H: every result stays the same (the operand is exactly zero on those
// tokens, so z there only feeds products by zero), while the MFMAs on the
// zero rows draw less power, and these contractions run power-limited.
//
// With `perm` set (the recompute backward), row j of Hm is that of the token
// perm[j] at position j of the live-first order (k_live_perm).
template <typename T>
__global__ __launch_bounds__(256) void k_live_rows(const T* __restrict__ H,
                                                   const int64_t* __restrict__ y,
                                                   const float* __restrict__ dlogp, int64_t Tn,
                                                   int64_t d, int64_t V,
                                                   const int* __restrict__ perm,
                                                   T* __restrict__ Hm) {
  constexpr int CE = 16 / sizeof(T);   // elements per 16-byte chunk (d is a multiple)
  const int64_t cpr = d / CE;
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= Tn * cpr) return;
  const int64_t j = i / cpr, c = i - j * cpr;
  const int64_t t = perm != nullptr ? int64_t(perm[j]) : j;
  u32x4 v = {0u, 0u, 0u, 0u};
  if (token_live(y[t], dlogp[t], V)) v = reinterpret_cast<const u32x4*>(H)[t * cpr + c];
  reinterpret_cast<u32x4*>(Hm)[i] = v;
}

// Live-first order of the tokens for the recompute backward: the live tokens
// (a nonzero row of the softmax operand) in index order, then the others in
// index order.  perm[j] = the token at position j; nlive[0] = the number of
// live tokens.  Two passes over blocks of kLiveBlock tokens (256 threads x 4
// consecutive tokens): k_live_count writes each block's live count, and
// k_live_perm adds the counts of the blocks before its own to an in-block
// scan (integer sums: exact, the order is deterministic).
constexpr int kLiveBlock = 1024;

__global__ __launch_bounds__(256) void k_live_count(const int64_t* __restrict__ y,
                                                    const float* __restrict__ dlogp, int64_t Tn,
                                                    int64_t V, int* __restrict__ blk) {
  __shared__ int part[4];
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t t0 = int64_t(blockIdx.x) * kLiveBlock + tid * 4;
  int v = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (t0 + q < Tn) v += token_live(y[t0 + q], dlogp[t0 + q], V) ? 1 : 0;
  v = wave_incl_scan(v, lane);
  if (lane == 63) part[tid >> 6] = v;
  __syncthreads();
  if (tid == 0) blk[blockIdx.x] = part[0] + part[1] + part[2] + part[3];
}

__global__ __launch_bounds__(256) void k_live_perm(const int64_t* __restrict__ y,
                                                   const float* __restrict__ dlogp, int64_t Tn,
                                                   int64_t V, const int* __restrict__ blk,
                                                   int nblk, int* __restrict__ perm,
                                                   int* __restrict__ nlive) {
  __shared__ int part[4], before[4], total[4];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // live tokens in the blocks before this one, and in all blocks
  int pre = 0, all = 0;
  for (int k = tid; k < nblk; k += 256) {
    const int c = blk[k];
    all += c;
    if (k < int(blockIdx.x)) pre += c;
  }
  pre = wave_incl_scan(pre, lane);
  all = wave_incl_scan(all, lane);
  if (lane == 63) {
    before[w] = pre;
    total[w] = all;
  }
  const int64_t t0 = int64_t(blockIdx.x) * kLiveBlock + tid * 4;
  bool lv[4];
  int own = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    lv[q] = t0 + q < Tn && token_live(y[t0 + q], dlogp[t0 + q], V);
    own += lv[q] ? 1 : 0;
  }
  const int incl = wave_incl_scan(own, lane);
  if (lane == 63) part[w] = incl;
  __syncthreads();
  const int n_live = total[0] + total[1] + total[2] + total[3];
  const int live_before = before[0] + before[1] + before[2] + before[3];
  int run = live_before + incl - own;          // live tokens before t0
  for (int k = 0; k < w; ++k) run += part[k];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t t = t0 + q;
    if (t < Tn) {
      // a dead token goes after all live ones, behind the dead tokens before it
      const int64_t pos = lv[q] ? int64_t(run) : int64_t(n_live) + (t - run);
      perm[pos] = int(t);
    }
    run += lv[q] ? 1 : 0;
  }
  if (blockIdx.x == 0 && tid == 0) nlive[0] = n_live;
}

// Zeros, grid-stride (the grid is capped; n may exceed 2^31 elements).
__global__ __launch_bounds__(256) void k_zero_f32(float* __restrict__ p, int64_t n) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride)
    p[i] = 0.0f;
}

// --- deterministic bucketing of tokens by target (for the one-hot part of dW)
__global__ void k_fill_i32(int* __restrict__ p, int64_t n, int v) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// Also counts into counts[V] the tokens whose gradient row is live (a
// target in range and a nonzero dlogp): one atomic per workgroup of 256.
__global__ __launch_bounds__(256) void k_hist(const int64_t* __restrict__ y,
                                              const float* __restrict__ dlogp, int64_t T,
                                              int64_t v_off, int64_t V, int* __restrict__ counts) {
  __shared__ int wave_live[4];
  const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t yy = t < T ? y[t] - v_off : -1;
  const bool in = yy >= 0 && yy < V;
  const uint64_t live = __ballot(in && dlogp[t] != 0.0f);
  if ((threadIdx.x & 63) == 0) wave_live[threadIdx.x >> 6] = int(__popcll(live));
  if (in) atomicAdd(counts + yy, 1);
  __syncthreads();
  if (threadIdx.x == 0) {
    const int n = wave_live[0] + wave_live[1] + wave_live[2] + wave_live[3];
    if (n) atomicAdd(counts + V, n);
  }
}

// A bucket of more than kRankDirect tokens is ordered through a bitmap in
// slot offsets[v] / kRankDirect (see k_bucket_rank): large buckets start at
// least kRankDirect positions apart, so the slots are distinct.
constexpr int kRankDirect = 256;
__host__ __device__ inline int64_t rank_slots(int64_t T) { return T / kRankDirect + 1; }
__host__ __device__ inline int64_t rank_words(int64_t T) { return (T + 31) / 32; }

// Exclusive scan of counts[V] into offsets[V + 1] in two passes over blocks
// of kScanBlock entries (256 threads x 4 consecutive entries, coalesced):
// k_scan_sums writes each block's total, k_scan_apply adds the totals of the
// blocks before its own to an in-block scan.  Integer sums: exact.
constexpr int kScanBlock = 1024;

__global__ __launch_bounds__(256) void k_scan_sums(const int* __restrict__ counts, int64_t V,
                                                   int* __restrict__ sums) {
  __shared__ int part[4];
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t i0 = int64_t(blockIdx.x) * kScanBlock + tid * 4;
  int v = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (i0 + q < V) v += counts[i0 + q];
  v = wave_incl_scan(v, lane);
  if (lane == 63) part[tid >> 6] = v;
  __syncthreads();
  if (tid == 0) sums[blockIdx.x] = part[0] + part[1] + part[2] + part[3];
}

// k_scan_apply also records each large bucket's range [b, e) in its slot of
// `meta` (zeroed beforehand).
__global__ __launch_bounds__(256) void k_scan_apply(const int* __restrict__ counts, int64_t V,
                                                    const int* __restrict__ sums,
                                                    int* __restrict__ offsets,
                                                    int* __restrict__ meta) {
  __shared__ int part[4];
  __shared__ int base[4];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // total of the blocks before this one
  int pre = 0;
  for (int k = tid; k < int(blockIdx.x); k += 256) pre += sums[k];
  pre = wave_incl_scan(pre, lane);
  if (lane == 63) base[w] = pre;
  // in-block exclusive scan
  const int64_t i0 = int64_t(blockIdx.x) * kScanBlock + tid * 4;
  int c[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) c[q] = i0 + q < V ? counts[i0 + q] : 0;
  const int own = c[0] + c[1] + c[2] + c[3];
  const int incl = wave_incl_scan(own, lane);
  if (lane == 63) part[w] = incl;
  __syncthreads();
  int run = base[0] + base[1] + base[2] + base[3] + incl - own;
  for (int k = 0; k < w; ++k) run += part[k];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (i0 + q < V) {
      offsets[i0 + q] = run;
      if (c[q] > kRankDirect) {
        meta[2 * (run / kRankDirect)] = run;
        meta[2 * (run / kRankDirect) + 1] = run + c[q];
      }
    }
    run += c[q];
  }
  if (i0 < V && i0 + 4 >= V) offsets[V] = run;   // the thread holding entry V - 1
}

// Buckets larger than kRankDirect are ordered through a bitmap (see
// k_bucket_rank); the (unordered) list is filled for the others only.
__global__ void k_bucket_fill(const int64_t* __restrict__ y, int64_t T, int64_t v_off,
                              int64_t V, const int* __restrict__ offsets,
                              int* __restrict__ cursor, int* __restrict__ unsorted) {
  const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= T) return;
  const int64_t yy = y[t] - v_off;
  if (yy < 0 || yy >= V) return;
  const int b = offsets[yy];
  if (offsets[yy + 1] - b > kRankDirect) return;
  unsorted[b + atomicAdd(cursor + yy, 1)] = int(t);
}

// Place each token at its rank among the tokens of its bucket (ascending t).
// A bucket of at most kRankDirect tokens: each token counts the smaller
// token indices in the bucket's (unordered) list.  A larger bucket: each
// token sets its bit in the bucket's bitmap of T bits (in the bucket's
// slot), and k_bucket_rank_large writes the set bits out in order, so no
// bucket costs more than O(size + T / 32).
__global__ void k_bucket_rank(const int64_t* __restrict__ y, int64_t T, int64_t v_off,
                              int64_t V, const int* __restrict__ offsets,
                              const int* __restrict__ unsorted, int* __restrict__ sorted,
                              unsigned* __restrict__ bits) {
  const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= T) return;
  const int64_t yy = y[t] - v_off;
  if (yy < 0 || yy >= V) return;
  const int b = offsets[yy], e = offsets[yy + 1];
  if (e - b > kRankDirect) {
    const int64_t slot = b / kRankDirect;
    atomicOr(bits + slot * rank_words(T) + (t >> 5), 1u << (t & 31));
    return;
  }
  // 16 independent loads per step: a bucket's scan is not one load latency
  // per entry
  int rank = 0, p = b;
  for (; p + 16 <= e; p += 16) {
    int u[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) u[i] = unsorted[p + i];
#pragma unroll
    for (int i = 0; i < 16; ++i) rank += u[i] < int(t);
  }
  for (; p < e; ++p) rank += unsorted[p] < int(t);
  sorted[b + rank] = int(t);
}

// One workgroup per slot: the set bits of a large bucket's bitmap in
// ascending order are its tokens in ascending order; 256 words per round,
// each word's bits placed after the popcounts of the words before it.
__global__ __launch_bounds__(256) void k_bucket_rank_large(const unsigned* __restrict__ bits,
                                                           const int* __restrict__ meta,
                                                           int64_t T, int* __restrict__ sorted) {
  __shared__ int part[4];
  const int64_t slot = blockIdx.x;
  const int b = meta[2 * slot], e = meta[2 * slot + 1];
  if (e - b <= kRankDirect) return;   // unused slot (zeroed) or a direct bucket
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t nw = rank_words(T);
  const unsigned* wb = bits + slot * nw;
  int base = b;
  for (int64_t w0 = 0; w0 < nw; w0 += 256) {
    const unsigned word = w0 + tid < nw ? wb[w0 + tid] : 0u;
    const int c = __popc(word);
    const int incl = wave_incl_scan(c, lane);
    if (lane == 63) part[w] = incl;
    __syncthreads();
    int pos = base + incl - c;
    for (int k = 0; k < w; ++k) pos += part[k];
    const int total = part[0] + part[1] + part[2] + part[3];
    for (unsigned x = word; x != 0u; x &= x - 1u)
      sorted[pos++] = int((w0 + tid) * 32 + __builtin_ctz(x));
    base += total;
    __syncthreads();   // part[] is rewritten in the next round
  }
}

// dW[v, :] += sum over tokens t with y_t = v (ascending t) of dlogp_t h_t,
// over the bucketed token list `sorted` (tokens grouped by target, ascending
// t within a bucket) cut into segments of kSeg positions.  k_onehot_seg:
// one workgroup per (segment, block of 1024 columns); it walks the segment's
// positions in order and, for each run of one bucket, sums dlogp_t h_t over
// the run's tokens with a nonzero dlogp (4 columns per thread).  A bucket
// that lies wholly inside the segment is added to its row of dW at once; a
// run of a bucket that crosses the segment's edge goes to a slot of the
// segment (slot 0: the bucket began in an earlier segment, slot 1: it
// continues past this one).  k_onehot_join adds each crossing bucket's
// slots to its row in segment order.  So a large bucket is spread over many
// workgroups, and every row's sum has a fixed order (run order, then
// segment order): bit-identical from run to run.  A bucket whose tokens all
// have zero dlogp (outside the loss mask, filtered, clipped) leaves its row
// as it is.
constexpr int kSeg = 16;
constexpr int kOnehotAhead = 8;
template <typename T>
__global__ __launch_bounds__(256) void k_onehot_seg(const T* __restrict__ H,
                                                    const int64_t* __restrict__ y,
                                                    const float* __restrict__ dlogp,
                                                    const int* __restrict__ offsets,
                                                    const int* __restrict__ sorted, int64_t d,
                                                    int64_t v_off, int64_t V,
                                                    float* __restrict__ dW,
                                                    float* __restrict__ slots,
                                                    int* __restrict__ slot_live) {
  __shared__ int s_t[kSeg], s_v[kSeg];
  __shared__ float s_g[kSeg];
  const int n_pos = offsets[V];
  const int x = blockIdx.x;
  const int p0 = x * kSeg;
  if (p0 >= n_pos) return;                                   // uniform
  const int p1 = min(p0 + kSeg, n_pos), n = p1 - p0;
  if (int(threadIdx.x) < n) {
    const int t = sorted[p0 + threadIdx.x];
    s_t[threadIdx.x] = t;
    s_g[threadIdx.x] = dlogp[t];
    s_v[threadIdx.x] = int(y[t] - v_off);
  }
  __syncthreads();
  const int64_t k = (int64_t(blockIdx.y) * blockDim.x + threadIdx.x) * 4;
  const bool act = k < d;                                    // d is a multiple of 8
  for (int q = 0; q < n;) {
    const int v = s_v[q];
    int r = q + 1;
    while (r < n && s_v[r] == v) ++r;                        // run [q, r) of bucket v
    bool live = false;                                       // a token with nonzero dlogp
    for (int u = q; u < r && !live; ++u) live = s_g[u] != 0.0f;
    const int b = offsets[v], e = offsets[v + 1];
    const bool from_here = b >= p0, to_here = e <= p1;
    // a live bucket wholly in this segment: its row of dW is loaded together
    // with the rows of H (one memory latency per run, not two)
    f32x4* const row = reinterpret_cast<f32x4*>(dW + int64_t(v) * d + k);
    f32x4 cur = {0.0f, 0.0f, 0.0f, 0.0f};
    if (from_here && to_here && live && act) cur = *row;
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int u0 = q; u0 < r; u0 += kOnehotAhead) {
      float g[kOnehotAhead];
      T h[kOnehotAhead][4];
#pragma unroll
      for (int u = 0; u < kOnehotAhead; ++u) {
        g[u] = u0 + u < r ? s_g[u0 + u] : 0.0f;
        if (g[u] != 0.0f && act) {
          const T* hp = H + int64_t(s_t[u0 + u]) * d + k;
#pragma unroll
          for (int c = 0; c < 4; ++c) h[u][c] = hp[c];
        }
      }
#pragma unroll
      for (int u = 0; u < kOnehotAhead; ++u) {
        if (g[u] == 0.0f) continue;
        if (act) {
#pragma unroll
          for (int c = 0; c < 4; ++c) acc[c] += g[u] * float(h[u][c]);
        }
      }
    }
    if (from_here && to_here) {
      if (live && act) *row = cur + acc;
    } else {
      const int slot = 2 * x + (from_here ? 1 : 0);
      if (act) *reinterpret_cast<f32x4*>(slots + int64_t(slot) * d + k) = acc;
      if (threadIdx.x == 0) slot_live[slot] = live ? 1 : 0;
    }
    q = r;
  }
}

// The buckets that begin in segment x and continue past it: their slots (1
// of segment x, 0 of the later segments they reach) summed in segment order
// and added to their rows of dW.
__global__ __launch_bounds__(256) void k_onehot_join(const int64_t* __restrict__ y,
                                                     const int* __restrict__ offsets,
                                                     const int* __restrict__ sorted, int64_t d,
                                                     int64_t v_off, int64_t V,
                                                     const float* __restrict__ slots,
                                                     const int* __restrict__ slot_live,
                                                     float* __restrict__ dW) {
  const int n_pos = offsets[V];
  const int x = blockIdx.x;
  const int p0 = x * kSeg;
  if (p0 >= n_pos) return;
  const int p1 = min(p0 + kSeg, n_pos);
  const int v = int(y[sorted[p1 - 1]] - v_off);
  const int b = offsets[v], e = offsets[v + 1];
  if (!(b >= p0 && e > p1)) return;
  const int xl = (e - 1) / kSeg;                             // the bucket's last segment
  bool live = slot_live[2 * x + 1] != 0;
  for (int c = x + 1; c <= xl && !live; ++c) live = slot_live[2 * c] != 0;
  if (!live) return;
  const int64_t k = (int64_t(blockIdx.y) * blockDim.x + threadIdx.x) * 4;
  if (k >= d) return;
  f32x4 acc = *reinterpret_cast<const f32x4*>(slots + int64_t(2 * x + 1) * d + k);
  int c = x + 1;
  for (; c + 8 <= xl + 1; c += 8) {                          // 8 slot loads in flight
    f32x4 w[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) w[i] = *reinterpret_cast<const f32x4*>(slots + int64_t(2 * (c + i)) * d + k);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc += w[i];
  }
  for (; c <= xl; ++c) acc += *reinterpret_cast<const f32x4*>(slots + int64_t(2 * c) * d + k);
  f32x4* o = reinterpret_cast<f32x4*>(dW + int64_t(v) * d + k);
  f32x4 cur = *o;
  cur += acc;
  *o = cur;
}

// Named kernels, one per role of the shared tile core.
// Softmax cache -> backward operand, in place: P~[t, v] = -dlogp_t
// exp(cm[v / kWaveRows][t] - lse_t) E[t, v] (0 for ignored tokens).
// The cached pair's operand: P~ = -dlogp_t exp(c_b - lse_t) E[t] for the live
// tokens, written to row j of the workspace operand for the token t =
// perm[j] at position j of the live-first order; rows past the live tokens
// are not written (the contractions read them as zeros), and the cache is
// only read.  Workgroup = one group of kCachePanels consecutive panels x one
// block of 32 positions; thread = one 16-byte chunk of one row of each of
// those panels (8 lanes per 128-byte row).  With at most half of the tokens
// live the panels of one block go first, otherwise the blocks of one panel
// group (every token live at T = 65536, V = 248320: 12.9 against 14.1 ms).  4 panels per thread (1, 2, 3, 6 or 8 measured slower for the
// in-place pass this replaces).  Touched once: non-temporal loads and
// stores.  Where the factor is exactly zero (a vocabulary block past V, or
// a factor that underflows) the chunk is written as zeros without reading
// it: the cached values are finite.
constexpr int kCachePanels = 4;
template <typename T>
__global__ __launch_bounds__(256) void k_cache_gather(const T* __restrict__ E,
                                                      const float* __restrict__ cm,
                                                      const float* __restrict__ lse,
                                                      const float* __restrict__ dlogp,
                                                      const int64_t* __restrict__ y,
                                                      const int* __restrict__ perm,
                                                      const int* __restrict__ nlive,
                                                      int64_t Tn, int64_t V, int64_t pld,
                                                      int64_t npanels, uint32_t ngroups,
                                                      const unsigned* __restrict__ bound,
                                                      T* __restrict__ P) {
  constexpr int BV = 128 / sizeof(T);   // panel width
  constexpr int CE = 16 / sizeof(T);    // entries per chunk
  const uint32_t nblocks = uint32_t((Tn + 31) / 32);
  const bool dense = 2 * int64_t(*nlive) > Tn;
  const uint32_t gi = dense ? blockIdx.x / nblocks : blockIdx.x % ngroups;
  const uint32_t jb = dense ? blockIdx.x % nblocks : blockIdx.x / ngroups;
  const int64_t j = int64_t(jb) * 32 + (threadIdx.x >> 3);
  if (j >= int64_t(*nlive)) return;
  const int64_t t = perm[j];
  const int ch = threadIdx.x & 7;
  const int64_t yy = y[t];
  const int sh = bound != nullptr ? probs_shift(*bound) : 0;
  const float g = (yy >= 0 && yy < V) ? ldexpf(-dlogp[t], sh) : 0.0f;
  const float l = lse[t];
  const int64_t p0 = int64_t(gi) * kCachePanels;
  u32x4 raw[kCachePanels];
  float f[kCachePanels];
#pragma unroll
  for (int q = 0; q < kCachePanels; ++q) {
    const int64_t pn = p0 + q;
    raw[q] = u32x4{0u, 0u, 0u, 0u};
    f[q] = 0.0f;
    if (pn < npanels && g != 0.0f) {
      const float m = cm[((pn * BV + ch * CE) / kWaveRows) * Tn + t];
      if (m != kNegInf) f[q] = g * __expf(m - l);
      if (f[q] != 0.0f)
        raw[q] = __builtin_nontemporal_load(
            reinterpret_cast<const u32x4*>(E + (pn * pld + t) * BV + ch * CE));
    }
  }
#pragma unroll
  for (int q = 0; q < kCachePanels; ++q) {
    const int64_t pn = p0 + q;
    if (pn < npanels) {
      T vals[CE];
      *reinterpret_cast<u32x4*>(vals) = raw[q];
#pragma unroll
      for (int e = 0; e < CE; ++e) vals[e] = T(float(vals[e]) * f[q]);
      __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(vals),
                                  reinterpret_cast<u32x4*>(P + (pn * pld + j) * BV + ch * CE));
    }
  }
}

// Vocabulary x token contractions (forward, softmax): tiles of 4 vocabulary
// rows walk the tokens together (0.4 ms faster than 8 for the forward at the
// headline shape; the backward's dH keeps 8).
constexpr int kGroupVT = 4;
// Which operand takes the 3-stage side of the loop's ring (measured).
constexpr bool kDeepFwdA = true;    // forward / softmax: W (A) over H (B)
constexpr bool kDeepDhA = true;     // dH: the operand panels (A) over W^T (B)
constexpr bool kDeepDwA = false;    // dW^T: the operand panels (B) over H^T (A)
template <typename T, typename TE = T>
__global__ __launch_bounds__(kThreads, 1) void k_fwd_logits_lse(Operand A, Operand B, int64_t K,
                                                                int nTm, int nTn,
                                                                EpiFwd<T, TE> epi) {
  static_assert(kLdsGemm + EpiFwd<T, TE>::kLdsExtra <= kLdsRing, "epilogue LDS");
  __shared__ __attribute__((aligned(16))) char lds[kLdsRing];
  gemm_body<T, Lay::KMajor, Lay::KMajor, EpiFwd<T, TE>, 2, kDeepFwdA>(A, B, K, nTm, nTn, epi,
                                                                      lds, kGroupVT);
}
// T: the inputs' type, TP: the operand's (see EpiProbs)
// With the live-first order, the first nTm x ntn workgroups take the tiles
// of the ntn token tiles that hold a live token, in the XCD-aware order of
// that smaller grid; the rest (tiles of dead tokens only) exit at once, after
// all of them.
template <typename T, typename TP>
__global__ __launch_bounds__(kThreads, 1) void k_bwd_probs(Operand A, Operand B, int64_t K,
                                                           int nTm, int nTn,
                                                           EpiProbs<T, TP> epi) {
  __shared__ __attribute__((aligned(16))) char lds[kLdsRing];
  int tm, tn;
  int ntn = nTn;
  if (epi.nlive != nullptr) {
    const int64_t nl = *epi.nlive;
    ntn = int((nl + kBN - 1) / kBN);
    if (int64_t(blockIdx.x) >= int64_t(nTm) * ntn) return;
  }
  tile_of(blockIdx.x, nTm, ntn, kGroupVT, tm, tn);
  const int64_t m0 = int64_t(tm) * kBM, n0 = int64_t(tn) * kBN;
  const auto pre = epi.prologue(m0, n0);
  Acc acc;
  gemm_mainloop<T, Lay::KMajor, Lay::KMajor, 2, kDeepFwdA>(A, B, m0, n0, K, lds, acc);
  epi.epilogue(acc, tm, tn, m0, n0, lds, lds + kLdsGemm, pre);
}
// TG: the contraction's operand type (the operand panels and W^T), T: the
// weight's, read by the one-hot part.  Groups of 4 token tile rows walk the
// hidden dimensions (measured against 8 and 16 with the current copy
// schedule: 0.18 ms faster than 8).
constexpr int kGroupDH = 4;
// With `nlive` set (the live-first order), the operand's rows from *nlive on
// are read as zeros (the copies take the out-of-range offset): they belong
// to tokens with zero gradient rows and were never written.  Every tile and
// every MFMA still runs.  The live rows then sit in the first token tile
// rows, which the XCD-aware map would hand to the first XCDs alone (each XCD
// takes a contiguous run of tile rows); token tile rows are therefore
// visited as tm * stride mod nTm (stride coprime to nTm), which deals the
// live rows out to every XCD and every round.  With `skip` set as well, a
// tile of dead tokens only runs its epilogue (zero rows), without the loop,
// and the live tiles come first in a grid of their own (the strided order
// measured 10.4 ms against 6.4 there: it left live tiles waiting for CUs
// behind others).  When the live tiles' last round would fill at most half
// of the CUs, its tiles are split along K (plan_tail, computed here from the
// live count) into fp32 slots that k_dh_tail_reduce sums in split order.
// The grid then has up to kTailSlots workgroups more than tiles; the spare
// ones exit.
template <typename TG, typename T>
__global__ __launch_bounds__(kThreads, 1) void k_bwd_dhidden(Operand A, Operand B, int64_t K,
                                                             int nTm, int nTn, EpiDH<T> epi,
                                                             const int* nlive, int stride,
                                                             int skip, int ncu, float* slots,
                                                             int cap) {
  __shared__ __attribute__((aligned(16))) char lds[kLdsRing];
  int tm, tn;
  int j = -1;   // the K slice of a split tile, or -1
  Operand a = A, b = B;
  int64_t k = K;
  if (skip && nlive != nullptr) {
    // the live token tile rows' tiles first, in the XCD-aware order of that
    // smaller grid; then the split tiles' slices; then the tiles of dead
    // tokens (no loop: zero rows)
    const int ntl = int((int64_t(*nlive) + kBM - 1) / kBM);
    const TailSplit ts = plan_tail(ntl * nTn, K, ncu, cap);
    const int nsp = ts.rem * ts.splits;
    const int bid = blockIdx.x;
    if (bid < ts.full) {
      tile_of(bid, ntl, nTn, kGroupDH, tm, tn, ts.full);
    } else if (bid < ts.full + nsp) {
      j = bid - ts.full;
      tile_of_logical(ts.full + j / ts.splits, ntl, nTn, kGroupDH, tm, tn);
      const int64_t k0 = int64_t(j % ts.splits) * ts.ks;
      k = K - k0 < ts.ks ? K - k0 : ts.ks;
      a = k_slice<TG, Lay::TileTK>(A, k0, k);
      b = k_slice<TG, Lay::KMajor>(B, k0, k);
    } else {
      const int r = bid - ts.full - nsp;
      tm = ntl + r / nTn;
      tn = r % nTn;
      if (tm >= nTm) return;   // spare workgroup
    }
  } else {
    tile_of(blockIdx.x, nTm, nTn, kGroupDH, tm, tn);
    tm = int((int64_t(tm) * stride) % nTm);
  }
  const int64_t m0 = int64_t(tm) * kBM, n0 = int64_t(tn) * kBN;
  if (nlive != nullptr) {
    const int64_t nl = *nlive;
    if (nl < a.rows) a.rows = nl;
    if (skip && m0 >= nl) k = 0;
  }
  Acc acc;
  gemm_mainloop<TG, Lay::TileTK, Lay::KMajor, 2, kDeepDhA>(a, b, m0, n0, k, lds, acc);
  if (j < 0) {
    epi.epilogue(acc, tm, tn, m0, n0, lds, lds + kLdsGemm);
  } else {
    const EpiStoreT slot{slots + int64_t(j) * (kBM * kBN), kBM, kBM, kBN, 0};
    slot.epilogue(acc, tm, tn, 0, 0, lds, nullptr);
  }
}

// The split tiles of k_bwd_dhidden (same plan, from the live count): each
// element is the sum of its slots in split order (slot[c][r]), then what
// EpiDH does to a tile element: unscale, add the stored value when
// accumulating, add the one-hot part, store to dH's row perm[r].  Grid x:
// split tiles (spare workgroups exit), y: groups of 4 columns; thread: one
// row, 4 consecutive columns.
template <typename T>
__global__ __launch_bounds__(256) void k_dh_tail_reduce(const float* __restrict__ slots,
                                                        const int* __restrict__ nlive, int nTn,
                                                        int64_t K, int ncu, int cap,
                                                        EpiDH<T> epi) {
  const int ntl = int((int64_t(*nlive) + kBM - 1) / kBM);
  const TailSplit ts = plan_tail(ntl * nTn, K, ncu, cap);
  if (int(blockIdx.x) >= ts.rem) return;
  int tm, tn;
  tile_of_logical(ts.full + int(blockIdx.x), ntl, nTn, kGroupDH, tm, tn);
  const int r = threadIdx.x, c4 = int(blockIdx.y) * 4;
  const int64_t pos = int64_t(tm) * kBM + r, c = int64_t(tn) * kBN + c4;
  if (pos >= epi.rows || c >= epi.cols) return;   // cols and ldc are multiples of 4
  f32x4 v = {0.0f, 0.0f, 0.0f, 0.0f};
  const float* sl = slots + int64_t(blockIdx.x) * ts.splits * (kBM * kBN);
  for (int q = 0; q < ts.splits; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] += sl[int64_t(q) * (kBM * kBN) + (c4 + e) * kBM + r];
  v = Unscale(epi.bound_p, epi.bound_w)(v);
  const int64_t t = epi.perm != nullptr ? int64_t(epi.perm[pos]) : pos;
  float* o = epi.C + t * epi.ldc + c;
  if (epi.accumulate) v += *reinterpret_cast<const f32x4*>(o);
  if (epi.W != nullptr) {
    const int64_t yy = epi.y[t] - epi.v_off;
    if (yy >= 0 && yy < epi.Vs) {
      const float g = epi.dlogp[t];
      const T* w = epi.W + yy * epi.ldc + c;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] += g * float(w[e]);
    }
  }
  *reinterpret_cast<f32x4*>(o) = v;
}
// dW^T = H^T P~ : tile rows are hidden dimensions (A = H^T, along the
// tokens), tile columns vocabulary entries (B = the operand panels read
// across, with the transposing LDS read on the operand with fewer blocks per
// wave), stored transposed into dW.
// Tiles of 4 hidden-dimension rows walk the vocabulary together: the 32
// workgroups of an XCD then share 4 H^T and 8 operand panels (measured best
// of 1, 2, 4, 8 at the headline shape).
constexpr int kGroupDW = 4;
// Workgroups past ts.full compute K slices of the last ts.rem tiles into
// 256 x 256 fp32 slots (stored [column][row]) for k_tail_reduce.
// With `nlive` set, both operands' K (token positions) from *nlive on is
// read as zeros, as in k_bwd_dhidden; the K loop still covers every token,
// unless `skip` is set: then it stops at the last stage holding a live
// token (the products it leaves out are exact zeros).
template <typename T>
__global__ __launch_bounds__(kThreads, 1) void k_bwd_dweight(Operand A, Operand B, int64_t K,
                                                             int nTm, int nTn, EpiStoreT epi,
                                                             TailSplit ts, float* slots,
                                                             const int* nlive, int skip) {
  __shared__ __attribute__((aligned(16))) char lds[kLdsRing];
  const int bid = blockIdx.x;
  int tm, tn, j = -1;
  Operand a = A, b = B;
  int64_t k = K;
  if (bid < ts.full) {
    tile_of(bid, nTm, nTn, kGroupDW, tm, tn, ts.full);
  } else {
    j = bid - ts.full;
    tile_of_logical(ts.full + j / ts.splits, nTm, nTn, kGroupDW, tm, tn);
    const int64_t k0 = int64_t(j % ts.splits) * ts.ks;
    k = K - k0 < ts.ks ? K - k0 : ts.ks;
    a = k_slice<T, Lay::KMajor>(A, k0, k);
    b = k_slice<T, Lay::TileVT>(B, k0, k);
  }
  if (nlive != nullptr) {
    const int64_t k0 = j < 0 ? 0 : int64_t(j % ts.splits) * ts.ks;
    const int64_t nl = int64_t(*nlive) - k0;
    const int64_t lim = nl < 0 ? 0 : (nl < k ? nl : k);
    a.K = lim;
    b.K = lim;
    if (skip) k = lim;
  }
  const int64_t m0 = int64_t(tm) * kBM, n0 = int64_t(tn) * kBN;
  Acc acc;
  gemm_mainloop<T, Lay::KMajor, Lay::TileVT, 1, kDeepDwA>(a, b, m0, n0, k, lds, acc);
  if (j < 0) {
    epi.epilogue(acc, tm, tn, m0, n0, lds, nullptr);
  } else {
    const EpiStoreT slot{slots + int64_t(j) * (kBM * kBN), kBM, kBM, kBN, 0};
    slot.epilogue(acc, tm, tn, 0, 0, lds, nullptr);
  }
}

// dW[n0 + c, m0 + r] (+)= sum over the splits, in split order, of
// slot[c][r] for each split tile (grid x: tiles, y: groups of 4 columns;
// thread: 4 consecutive rows of one column).
__global__ __launch_bounds__(256) void k_tail_reduce(const float* __restrict__ slots,
                                                     TailSplit ts, int nTm, int nTn,
                                                     float* __restrict__ C, int64_t ldc,
                                                     int64_t rows, int64_t cols, int accumulate,
                                                     const unsigned* bound_p,
                                                     const unsigned* bound_h) {
  int tm, tn;
  tile_of_logical(ts.full + int(blockIdx.x), nTm, nTn, kGroupDW, tm, tn);
  const int cl = int(blockIdx.y) * 4 + (threadIdx.x >> 6), rl = (threadIdx.x & 63) * 4;
  const int64_t c = int64_t(tn) * kBN + cl, r = int64_t(tm) * kBM + rl;
  if (c >= cols || r >= rows) return;   // rows, ldc and r are multiples of 4
  const float* src = slots + int64_t(blockIdx.x) * ts.splits * (kBM * kBN) + cl * kBM + rl;
  f32x4 v = *reinterpret_cast<const f32x4*>(src);
  for (int q = 1; q < ts.splits; ++q) v += *reinterpret_cast<const f32x4*>(src + q * (kBM * kBN));
  v = Unscale(bound_p, bound_h)(v);
  f32x4* o = reinterpret_cast<f32x4*>(C + c * ldc + r);
  if (accumulate) v += *o;
  *o = v;
}

// Slot floats the tail split of one dW launch over `width` vocabulary columns
// can use: at most 8 splits of each of its tiles, and at most kTailSlots.
size_t tail_slot_floats(int64_t d, int64_t width) {
  const int64_t tiles = cdiv(d, int64_t(kBM)) * cdiv(width, int64_t(kBN));
  return size_t(std::min<int64_t>(kTailSlots, 8 * tiles)) * kBM * kBN;
}

// Forward over a vocabulary shard [v_off, v_off + Vs) of a V-entry vocabulary
// (the whole vocabulary when v_off = 0, Vs = V).  part == null: final lse,
// logp (and entropy when given); otherwise the shard's partial [4][T].
// cacheE: the softmax cache (element type TE), or null.
template <typename T, typename TE = T>
hipError_t fwd_impl(const T* H, const T* W, const int64_t* y, int64_t Tn, int64_t d, int64_t Vs,
                    int64_t v_off, int64_t V, float* logp, float* lse, float* entropy,
                    float* part, bool with_u, void* ws, hipStream_t s, TE* cacheE = nullptr,
                    float* cacheM = nullptr) {
  // tile rows: vocabulary (the weight's rows), tile columns: tokens
  const int nTv = int(cdiv(Vs, kBM)), nTt = int(cdiv(Tn, kBN));
  Carve cv(ws);
  float* pm = cv.take<float>(size_t(nTv) * Tn);
  float* ps = cv.take<float>(size_t(nTv) * Tn);
  float* pu = cv.take<float>(size_t(nTv) * Tn);
  if (!with_u) pu = nullptr;
  const double es = sizeof(T);
  Operand A{W, d, Vs, d}, B{H, d, Tn, d};
  if (!operand_in_bounds<T, Lay::KMajor>(A, size_t(Vs) * d * sizeof(T)) ||
      !operand_in_bounds<T, Lay::KMajor>(B, size_t(Tn) * d * sizeof(T)))
    return hipErrorInvalidValue;
  const int64_t pld = cdiv(Tn, 64) * 64, ldE = int64_t(align_up(size_t(Vs), 64));
  EpiFwd<T, TE> epi{y,  Tn,     Vs,     v_off,  pm,  ps, pu, part ? part + 3 * Tn : logp,
                    cacheE, cacheM, pld, ldE};
  {
    ProfScope ps_(s, "logprob_fwd_gemm", 2.0 * Tn * d * Vs,
                  es * (double(Tn) * d + double(Vs) * d) + 12.0 * Tn +
                      (cacheE ? es * double(Tn) * Vs + 8.0 * nTv * Tn : 0.0));
    hipLaunchKernelGGL((k_fwd_logits_lse<T, TE>), dim3(nTv * nTt), dim3(kThreads), 0,
                       s, A, B, d, nTv, nTt, epi);
  }
  {
    ProfScope ps_(s, "logprob_fwd_merge", 0.0, (with_u ? 12.0 : 8.0) * nTv * Tn + 24.0 * Tn);
    if (part)
      hipLaunchKernelGGL(k_shard_partial, dim3(cdiv(Tn, 64)), dim3(512), 0, s, pm, ps, pu, nTv,
                         Tn, y, v_off, Vs, part);
    else
      hipLaunchKernelGGL(k_lse_merge, dim3(cdiv(Tn, 64)), dim3(512), 0, s, pm, ps, pu, nTv, Tn,
                         y, V, logp, lse, entropy);
  }
  return hipGetLastError();
}

// Backward over a vocabulary shard [v_off, v_off + Vs) of a V-entry
// vocabulary: dH receives this shard's part of G W (the shards' parts sum to
// dH), dW the shard's rows.  A target outside [0, V) is an ignored token; a
// target outside the shard contributes only the softmax part here.
// T: the inputs' type; TP: the type of the operand and of the transposes,
// fp16 (power-of-two scaled, see probs_shift) for bf16 inputs, with or
// without a cache (the cache is then fp16 too), T otherwise.
// A stride near n / kXcds that is coprime to n (so tm -> tm * stride mod n
// permutes the tile rows), 1 for n below 2 kXcds.
inline int row_stride(int n) {
  if (n < 2 * kXcds) return 1;
  int st = n / kXcds;
  while (std::gcd(st, n) != 1) ++st;
  return st;
}

template <typename T, typename TP>
hipError_t bwd_impl(const T* H, const T* W, const int64_t* y, const float* lse,
                    const float* dlogp, int64_t Tn, int64_t d, int64_t Vs, int64_t v_off,
                    int64_t V, float* dH, float* dW, int flags, void* ws, hipStream_t s,
                    TP* cacheE = nullptr, const float* cacheM = nullptr) {
  static_assert(sizeof(T) == sizeof(TP), "the operand keeps the input's element size");
  constexpr bool kScaled = !std::is_same<T, TP>::value;
  // With a softmax cache the whole vocabulary is one chunk and the operand is
  // gathered from the cache; otherwise the logits of each chunk are
  // recomputed.
  const int64_t chunk = cacheE ? Vs : bwd_chunk_cols(Tn, Vs, sizeof(T));
  const int64_t ld = int64_t(align_up(size_t(min(chunk, Vs)), 64));
  const int64_t pld = cdiv(Tn, 64) * 64;
  const int64_t nchunks = cdiv(Vs, chunk);
  Carve cv(ws);
  TP* P = cv.take<TP>(size_t(pld) * ld);
  TP* Wt = cv.take<TP>(size_t(d) * ld);    // [d x chunk] transpose of W's chunk rows
  TP* Ht = cv.take<TP>(size_t(d) * pld);   // [d x T] transpose of H
  // H with the dead tokens' rows zeroed, in the live-first order (recompute
  // pair) or in token order (cached pair)
  T* Hm = cv.take<T>(size_t(Tn) * d);
  int* counts = cv.take<int>(Vs + 1);   // counts[Vs]: live tokens
  int* cursor = cv.take<int>(Vs);
  unsigned* rank_bits = cv.take<unsigned>(size_t(rank_slots(Tn) * rank_words(Tn)));
  int* rank_meta = cv.take<int>(size_t(2 * rank_slots(Tn)));
  int* offsets = cv.take<int>(Vs + 1);
  int* unsorted = cv.take<int>(Tn);
  int* sorted = cv.take<int>(Tn);
  int* scan_sums = cv.take<int>(cdiv(Vs, kScanBlock));
  float* slots = cv.take<float>(tail_slot_floats(d, min(chunk, Vs)));
  float* seg_slots = cv.take<float>(size_t(2) * cdiv(Tn, kSeg) * d);
  int* seg_live = cv.take<int>(size_t(2) * cdiv(Tn, kSeg));
  // magnitude bounds of the scaled operands: [0] max |dlogp|, [1] max |H|,
  // [2 + c] max |W| over chunk c
  unsigned* bounds = kScaled ? cv.take<unsigned>(size_t(2 + nchunks)) : nullptr;
  // the live-first token order (position -> token) and the live counts of
  // its blocks, followed by the number of live tokens
  const int nlb = int(cdiv(Tn, kLiveBlock));
  int* perm = cv.take<int>(Tn);
  int* live_blk = cv.take<int>(size_t(nlb) + 1);
  const int* nlive = live_blk + nlb;
  // the gradient contractions also skip the dead tokens' MFMAs
  const bool skip = (flags & MC_BWD_SKIP_DEAD_TOKENS) != 0;
  int ncu = 0, dev = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    ncu = 0;   // no tail split
  const int nTm = int(cdiv(Tn, kBM));
  const int nTd = int(cdiv(d, kBN));

  const double es = sizeof(T);
  {
    ProfScope ps_(s, "logprob_bwd_live_order", 0.0, 24.0 * Tn);
    hipLaunchKernelGGL(k_live_count, dim3(nlb), dim3(256), 0, s, y, dlogp, Tn, V, live_blk);
    hipLaunchKernelGGL(k_live_perm, dim3(nlb), dim3(256), 0, s, y, dlogp, Tn, V, live_blk, nlb,
                       perm, live_blk + nlb);
  }
  if (!cacheE || dW) {   // read by the softmax contraction and by H^T
    ProfScope ps_(s, "logprob_bwd_live_rows", 0.0, 2.0 * es * double(Tn) * d + 12.0 * Tn);
    const int64_t chunks = Tn * d / (16 / int64_t(sizeof(T)));
    if (cdiv(chunks, int64_t(256)) > int64_t(0x7fffffff)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_live_rows<T>, dim3(unsigned(cdiv(chunks, int64_t(256)))), dim3(256), 0,
                       s, H, y, dlogp, Tn, d, V, perm, Hm);
  }
  if (kScaled) {
    ProfScope ps_(s, "logprob_bwd_bounds", 0.0, 4.0 * Tn);
    hipLaunchKernelGGL(k_fill_i32, dim3(cdiv(2 + nchunks, 256)), dim3(256), 0, s,
                       reinterpret_cast<int*>(bounds), 2 + nchunks, 0);
    hipLaunchKernelGGL(k_bound_abs, dim3(cdiv(Tn, 256)), dim3(256), 0, s, dlogp, Tn, bounds);
  }
  if (dW) {
    ProfScope ps_(s, "logprob_bwd_bucket", 0.0, 32.0 * Tn + 16.0 * Vs);
    const int nb = int(cdiv(Vs, 256)), tb = int(cdiv(Tn, 256));
    hipLaunchKernelGGL(k_fill_i32, dim3(nb + 1), dim3(256), 0, s, counts, Vs + 1, 0);
    // cursor, the large buckets' bitmaps and their slots: one zero fill
    const int64_t zspan = reinterpret_cast<int*>(rank_meta + 2 * rank_slots(Tn)) - cursor;
    if (cdiv(zspan, int64_t(256)) > int64_t(0x7fffffff)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_fill_i32, dim3(unsigned(cdiv(zspan, int64_t(256)))), dim3(256), 0, s,
                       cursor, zspan, 0);
    hipLaunchKernelGGL(k_hist, dim3(tb), dim3(256), 0, s, y, dlogp, Tn, v_off, Vs, counts);
    const int nsb = int(cdiv(Vs, kScanBlock));
    hipLaunchKernelGGL(k_scan_sums, dim3(nsb), dim3(256), 0, s, counts, Vs, scan_sums);
    hipLaunchKernelGGL(k_scan_apply, dim3(nsb), dim3(256), 0, s, counts, Vs, scan_sums, offsets,
                       rank_meta);
    hipLaunchKernelGGL(k_bucket_fill, dim3(tb), dim3(256), 0, s, y, Tn, v_off, Vs, offsets,
                       cursor, unsorted);
    hipLaunchKernelGGL(k_bucket_rank, dim3(tb), dim3(256), 0, s, y, Tn, v_off, Vs, offsets,
                       unsorted, sorted, rank_bits);
    hipLaunchKernelGGL(k_bucket_rank_large, dim3(unsigned(rank_slots(Tn))), dim3(256), 0, s,
                       rank_bits, rank_meta, Tn, sorted);
  }
  for (int64_t v0 = 0; v0 < Vs; v0 += chunk) {
    const int64_t width = min(chunk, Vs - v0);
    unsigned* const bound_w = kScaled ? bounds + 2 + v0 / chunk : nullptr;
    const int64_t ldc = int64_t(align_up(size_t(width), 64));   // padded width of this chunk
    const T* Wc = W + v0 * d;
    const size_t wc_bytes = size_t(Vs - v0) * d * sizeof(T);
    const size_t p_bytes = size_t(pld) * ld * sizeof(TP);
    if (cacheE) {
      // algorithmic bytes: per-token values (the live tokens' reads and
      // writes depend on dlogp and are not counted)
      ProfScope ps_(s, "logprob_bwd_cache_probs", 0.0, 4.0 * Tn * 6);
      const int64_t panels = ldc / (128 / int64_t(sizeof(T)));
      const int64_t groups = cdiv(panels, kCachePanels), blocks = cdiv(Tn, 32);
      if (groups * blocks > int64_t(0x7fffffff) || ldc > ld) return hipErrorInvalidValue;
      hipLaunchKernelGGL(k_cache_gather<TP>, dim3(unsigned(groups * blocks)), dim3(256), 0, s,
                         cacheE, cacheM, lse, dlogp, y, perm, nlive, Tn, V, pld, panels,
                         uint32_t(groups), bounds, P);
    } else {
      // tile rows: chunk columns (up to the padded width ldc), tile columns: tokens
      Operand A{Wc, d, width, d}, B{Hm, d, Tn, d};   // B: H's rows in the live-first order
      if (!operand_in_bounds<T, Lay::KMajor>(A, wc_bytes) ||
          !operand_in_bounds<T, Lay::KMajor>(B, size_t(Tn) * d * sizeof(T)) || ldc > ld)
        return hipErrorInvalidValue;
      EpiProbs<T, TP> epi{y, lse, dlogp, Tn, V, width, ldc, pld, P, bounds, perm, nlive};
      const int nTv = int(cdiv(ldc, kBM)), nTt = int(cdiv(Tn, kBN));
      ProfScope ps_(s, "logprob_bwd_probs", 2.0 * Tn * d * width,
                    es * (double(Tn) * d + double(width) * d + double(Tn) * width) + 16.0 * Tn);
      hipLaunchKernelGGL((k_bwd_probs<T, TP>), dim3(nTv * nTt),
                         dim3(kThreads), 0, s, A, B, d, nTv, nTt, epi);
    }
    if (dH) {
      // dH (+)= P~ Wc : M = T, N = d, K = chunk columns, with Wc^T [d x ldc]
      // so that both operands run along K
      {
        ProfScope ps_(s, "logprob_bwd_transpose", 0.0, 2.0 * es * double(width) * d);
        hipLaunchKernelGGL((k_transpose<T, TP>), dim3(cdiv(d, 256), cdiv(width, 64)), dim3(256),
                           0, s, Wc, width, d, d, Wt, ldc, bound_w, 0);
        if (kScaled)   // converts again, scaled, only when the bound asks for it
          hipLaunchKernelGGL((k_transpose<T, TP>),
                             dim3(cdiv(d, 256), std::min<int64_t>(cdiv(width, 64), kRescaleRows)),
                             dim3(256), 0, s, Wc, width, d, d, Wt, ldc, bound_w, 1);
      }
      Operand A{P, pld, Tn, ldc}, B{Wt, ldc, d, width};   // ldc = 64 ceil(width / 64)
      if (!operand_in_bounds<TP, Lay::TileTK>(A, p_bytes) ||
          !operand_in_bounds<TP, Lay::KMajor>(B, size_t(d) * ldc * sizeof(TP)) ||
          width > ldc || size_t(d) * ldc > size_t(d) * ld)
        return hipErrorInvalidValue;
      // the one-hot part goes into the last chunk's epilogue
      const bool last = v0 + chunk >= Vs;
      EpiDH<T> epi{dH,      d,     Tn,    d, (v0 > 0 || (flags & MC_BWD_ACCUMULATE_DHIDDEN)) ? 1 : 0,
                   last ? W : nullptr, y, dlogp, v_off, Vs, bounds, bound_w, perm};
      ProfScope ps_(s, "logprob_bwd_dhidden", 2.0 * Tn * d * (width + (last ? 1 : 0)),
                    es * (double(Tn) * width + double(width) * d) +
                        4.0 * Tn * d * (epi.accumulate ? 2 : 1) +
                        (last ? es * double(Tn) * d + 16.0 * Tn : 0.0));
      // skipping: up to kTailSlots spare workgroups for the split tiles'
      // slices (dW's tail slots, free until dW runs)
      const int cap = int(tail_slot_floats(d, min(chunk, Vs)) / (kBM * kBN));
      hipLaunchKernelGGL((k_bwd_dhidden<TP, T>), dim3(nTm * nTd + (skip ? kTailSlots : 0)),
                         dim3(kThreads), 0, s, A, B, ldc, nTm, nTd, epi, nlive,
                         nlive != nullptr ? row_stride(nTm) : 1, skip ? 1 : 0, ncu, slots, cap);
      if (skip)
        hipLaunchKernelGGL(k_dh_tail_reduce<T>, dim3(kTailSlots / 2, kBN / 4), dim3(256), 0, s,
                           slots, nlive, nTd, ldc, ncu, cap, epi);
    }
    if (dW) {
      // dW[chunk]^T (+)= H^T P~ : M = d, N = chunk columns, K = T (the
      // positions of P~'s rows), with H^T [d x pld] (made once, from Hm: in
      // the same order as P~'s rows) so that the M operand runs along K
      if (v0 == 0) {
        ProfScope ps_(s, "logprob_bwd_transpose", 0.0, 2.0 * es * double(Tn) * d);
        unsigned* const bound_h = kScaled ? bounds + 1 : nullptr;
        hipLaunchKernelGGL((k_transpose<T, TP>), dim3(cdiv(d, 256), cdiv(Tn, 64)), dim3(256), 0,
                           s, Hm, Tn, d, d, Ht, pld, bound_h, 0);
        if (kScaled)
          hipLaunchKernelGGL((k_transpose<T, TP>),
                             dim3(cdiv(d, 256), std::min<int64_t>(cdiv(Tn, 64), kRescaleRows)),
                             dim3(256), 0, s, Hm, Tn, d, d, Ht, pld, bound_h, 1);
      }
      Operand A{Ht, pld, d, Tn}, B{P, pld, ldc, Tn};   // pld = 64 ceil(Tn / 64)
      if (!operand_in_bounds<TP, Lay::KMajor>(A, size_t(d) * pld * sizeof(TP)) ||
          !operand_in_bounds<TP, Lay::TileVT>(B, p_bytes))
        return hipErrorInvalidValue;
      EpiStoreT epi{dW + v0 * d, d, d, width, (flags & MC_BWD_ACCUMULATE_DWEIGHT) ? 1 : 0,
                    kScaled ? bounds : nullptr, kScaled ? bounds + 1 : nullptr};
      const int nTv = int(cdiv(width, kBM));
      ProfScope ps_(s, "logprob_bwd_dweight", 2.0 * Tn * d * width,
                    es * (double(Tn) * width + double(Tn) * d) +
                        4.0 * width * d * (epi.accumulate ? 2 : 1));
      const TailSplit ts = plan_tail(nTd * nTv, Tn, ncu);
      hipLaunchKernelGGL(k_bwd_dweight<TP>, dim3(ts.full + ts.rem * ts.splits), dim3(kThreads),
                         0, s, A, B, Tn, nTd, nTv, epi, ts, slots, nlive, skip ? 1 : 0);
      if (ts.rem > 0)
        hipLaunchKernelGGL(k_tail_reduce, dim3(ts.rem, kBN / 4), dim3(256), 0, s, slots, ts, nTd,
                           nTv, epi.C, epi.ldc, epi.rows, epi.cols, epi.accumulate, epi.bound_p,
                           epi.bound_h);
    }
  }
  if (dW) {
    ProfScope ps_(s, "logprob_bwd_onehot_dw", 2.0 * Tn * d, (es + 8.0) * Tn * d);
    const dim3 grid(unsigned(cdiv(Tn, kSeg)), unsigned(cdiv(d, 1024)));
    hipLaunchKernelGGL(k_onehot_seg<T>, grid, dim3(256), 0, s, H, y, dlogp, offsets, sorted, d,
                       v_off, Vs, dW, seg_slots, seg_live);
    hipLaunchKernelGGL(k_onehot_join, grid, dim3(256), 0, s, y, offsets, sorted, d, v_off, Vs,
                       seg_slots, seg_live, dW);
  }
  return hipGetLastError();
}

}  // namespace

int64_t bwd_chunk_cols(int64_t T, int64_t V, size_t esize) {
  const int64_t per_col = std::max<int64_t>(1, T) * int64_t(esize);
  int64_t cap = int64_t(kBwdChunkBytes) / per_col;
  cap = std::max<int64_t>(kBN, cap / kBN * kBN);
  if (cap >= V) return V;
  const int64_t n = cdiv(V, cap);
  return std::min(cap, cdiv(cdiv(V, n), kBN) * kBN);
}

// Segment slots of the one-hot scatter: 2 rows of d floats and 2 flags per
// segment of kSeg bucketed positions.
static size_t onehot_seg_bytes(int64_t T, int64_t d) {
  const size_t nseg = size_t(cdiv(std::max<int64_t>(T, 1), kSeg));
  return align_up(2 * nseg * size_t(d) * 4, kWsAlign) + align_up(2 * nseg * 4, kWsAlign);
}

size_t fwd_workspace(int64_t T, int64_t, int64_t V, mc_dtype_t) {
  const size_t n = size_t(cdiv(V, kBN)) * size_t(T);
  return 3 * align_up(n * sizeof(float), kWsAlign);
}

size_t cache_bytes(int64_t T, int64_t, int64_t V, mc_dtype_t dt) {
  const size_t es = dt == MC_BF16 ? 2 : 4;
  const size_t pld = size_t(cdiv(T, 64)) * 64, ldE = align_up(size_t(V), 64);
  return align_up(pld * ldE * es, kWsAlign) +
         align_up(size_t(cdiv(V, kBM)) * kWavesM * size_t(T) * 4, kWsAlign);
}

size_t bwd_cache_workspace(int64_t T, int64_t d, int64_t V, mc_dtype_t dt) {
  const size_t es = dt == MC_BF16 ? 2 : 4;
  const size_t ld = align_up(size_t(V), 64);
  const size_t pld = size_t(cdiv(T, 64)) * 64;
  size_t n = align_up(pld * ld * es, kWsAlign);   // the operand, gathered from the cache
  n += align_up(size_t(d) * ld * es, kWsAlign);
  n += align_up(size_t(d) * pld * es, kWsAlign);
  n += align_up(size_t(T) * size_t(d) * es, kWsAlign);   // H with dead rows zeroed
  n += align_up(size_t(V + 1) * 4, kWsAlign) + align_up(size_t(V) * 4, kWsAlign);
  n += align_up(size_t(rank_slots(T) * rank_words(T)) * 4, kWsAlign) +
       align_up(size_t(2 * rank_slots(T)) * 4, kWsAlign);   // large buckets' bitmaps
  n += align_up(size_t(V + 1) * 4, kWsAlign);
  n += 2 * align_up(size_t(T) * 4, kWsAlign);
  n += align_up(size_t(cdiv(V, kScanBlock)) * 4, kWsAlign);
  n += align_up(tail_slot_floats(d, V) * 4, kWsAlign);
  n += onehot_seg_bytes(T, d);
  if (dt == MC_BF16) n += align_up(size_t(3) * 4, kWsAlign);   // bounds (one chunk)
  n += align_up(size_t(T) * 4, kWsAlign);                         // order
  n += align_up(size_t(cdiv(T, kLiveBlock) + 1) * 4, kWsAlign);   // its counts
  return n;
}

size_t bwd_workspace(int64_t T, int64_t d, int64_t V, mc_dtype_t dt) {
  const size_t es = dt == MC_BF16 ? 2 : 4;
  const int64_t chunk = bwd_chunk_cols(T, V, es);
  const size_t ld = align_up(size_t(std::min(chunk, V)), 64);
  const size_t pld = size_t(cdiv(T, 64)) * 64;
  size_t n = align_up(pld * ld * es, kWsAlign);
  n += align_up(size_t(d) * ld * es, kWsAlign);
  n += align_up(size_t(d) * pld * es, kWsAlign);
  n += align_up(size_t(T) * size_t(d) * es, kWsAlign);   // H with dead rows zeroed
  n += align_up(size_t(V + 1) * 4, kWsAlign) + align_up(size_t(V) * 4, kWsAlign);
  n += align_up(size_t(rank_slots(T) * rank_words(T)) * 4, kWsAlign) +
       align_up(size_t(2 * rank_slots(T)) * 4, kWsAlign);   // large buckets' bitmaps
  n += align_up(size_t(V + 1) * 4, kWsAlign);
  n += 2 * align_up(size_t(T) * 4, kWsAlign);
  n += align_up(size_t(cdiv(V, kScanBlock)) * 4, kWsAlign);
  n += align_up(tail_slot_floats(d, std::min(chunk, V)) * 4, kWsAlign);
  n += onehot_seg_bytes(T, d);
  if (dt == MC_BF16) n += align_up(size_t(2 + cdiv(V, chunk)) * 4, kWsAlign);   // bounds
  n += align_up(size_t(T) * 4, kWsAlign);                                      // order
  n += align_up(size_t(cdiv(T, kLiveBlock) + 1) * 4, kWsAlign);                // its counts
  return n;
}

hipError_t launch_fwd(const void* H, const void* W, const int64_t* y, int64_t T, int64_t d,
                      int64_t Vs, int64_t v_off, int64_t V, mc_dtype_t dt, float* logp,
                      float* lse, float* entropy, float* part, bool with_u, void* ws,
                      hipStream_t s) {
  if (dt == MC_BF16)
    return fwd_impl(static_cast<const bf16_t*>(H), static_cast<const bf16_t*>(W), y, T, d, Vs,
                    v_off, V, logp, lse, entropy, part, with_u, ws, s);
  return fwd_impl(static_cast<const float*>(H), static_cast<const float*>(W), y, T, d, Vs, v_off,
                  V, logp, lse, entropy, part, with_u, ws, s);
}

hipError_t launch_zero(float* p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>(cdiv(n, int64_t(256)), int64_t(1) << 16);
  hipLaunchKernelGGL(k_zero_f32, dim3(unsigned(blocks)), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_merge(const float* parts, int S, const int64_t* y, int64_t T, int64_t V,
                        float* logp, float* lse, float* entropy, hipStream_t s) {
  ProfScope ps_(s, "logprob_merge_shards", 0.0, 16.0 * S * T + 20.0 * T);
  hipLaunchKernelGGL(k_shard_merge, dim3(cdiv(T, 256)), dim3(256), 0, s, parts, S, T, y, V, logp,
                     lse, entropy);
  return hipGetLastError();
}

hipError_t launch_bwd(const void* H, const void* W, const int64_t* y, const float* lse,
                      const float* dlogp, int64_t T, int64_t d, int64_t Vs, int64_t v_off,
                      int64_t V, mc_dtype_t dt, float* dH, float* dW, int flags, void* ws,
                      hipStream_t s) {
  if (dt == MC_BF16)
    return bwd_impl<bf16_t, half_t>(static_cast<const bf16_t*>(H), static_cast<const bf16_t*>(W),
                                    y, lse, dlogp, T, d, Vs, v_off, V, dH, dW, flags, ws, s);
  return bwd_impl<float, float>(static_cast<const float*>(H), static_cast<const float*>(W), y, lse,
                                dlogp, T, d, Vs, v_off, V, dH, dW, flags, ws, s);
}

// Softmax cache layout: E panels [ldE / BV][pld][BV] (fp16 for bf16 inputs,
// fp32 for fp32), then the block maxima [2 nTv][T] fp32.
template <typename T>
static void carve_cache(void* cache, int64_t T_, int64_t V, T*& E, float*& cm) {
  Carve cv(cache);
  const size_t pld = size_t(cdiv(T_, 64)) * 64, ldE = align_up(size_t(V), 64);
  E = cv.take<T>(pld * ldE);
  cm = cv.take<float>(size_t(cdiv(V, kBM)) * kWavesM * size_t(T_));
}

hipError_t launch_fwd_cache(const void* H, const void* W, const int64_t* y, int64_t T, int64_t d,
                            int64_t V, mc_dtype_t dt, float* logp, float* lse, float* entropy,
                            void* cache, void* ws, hipStream_t s) {
  if (dt == MC_BF16) {   // fp16 cache (see launch_bwd_cache)
    half_t* E;
    float* cm;
    carve_cache(cache, T, V, E, cm);
    return fwd_impl(static_cast<const bf16_t*>(H), static_cast<const bf16_t*>(W), y, T, d, V,
                    int64_t(0), V, logp, lse, entropy, nullptr, entropy != nullptr, ws, s, E, cm);
  }
  float* E;
  float* cm;
  carve_cache(cache, T, V, E, cm);
  return fwd_impl(static_cast<const float*>(H), static_cast<const float*>(W), y, T, d, V,
                  int64_t(0), V, logp, lse, entropy, nullptr, entropy != nullptr, ws, s, E, cm);
}

hipError_t launch_bwd_cache(const void* H, const void* W, const int64_t* y, const float* lse,
                            const float* dlogp, int64_t T, int64_t d, int64_t V, mc_dtype_t dt,
                            void* cache, float* dH, float* dW, int flags, void* ws,
                            hipStream_t s) {
  if (dt == MC_BF16) {
    // The cache holds exp(z - c_b) in (0, 1] as fp16 (11 significant bits);
    // the backward rescales it in place into the power-of-two scaled fp16
    // operand of the recompute pair and runs the same fp16 contractions.
    half_t* E;
    float* cm;
    carve_cache(cache, T, V, E, cm);
    return bwd_impl<bf16_t, half_t>(static_cast<const bf16_t*>(H), static_cast<const bf16_t*>(W),
                                    y, lse, dlogp, T, d, V, int64_t(0), V, dH, dW, flags, ws, s,
                                    E, cm);
  }
  float* E;
  float* cm;
  carve_cache(cache, T, V, E, cm);
  return bwd_impl<float, float>(static_cast<const float*>(H), static_cast<const float*>(W), y, lse,
                                dlogp, T, d, V, int64_t(0), V, dH, dW, flags, ws, s, E, cm);
}

}  // namespace mc
