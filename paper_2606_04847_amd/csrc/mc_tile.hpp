// MFMA tile core for gfx950 (CDNA4): a 256 x 256 output tile per workgroup of
// kWavesM x kWavesN wave64s (two waves per SIMD), each owning a
// kWaveRows x kWaveCols sub-tile held as 16 x 16 fp32 accumulator blocks
// (v_mfma_f32_16x16x32_bf16: at equal issue rate it sustains a markedly
// higher throughput than the 32 x 32 form on realistic data on this part).
// With two waves per SIMD, one wave's MFMAs run while the other waits on
// memory or a barrier.
//
// Operands are staged through LDS in a K-contiguous layout: each tile row
// holds 128 bytes of K (64 bf16 or 32 fp32) as eight 16-byte chunks, and the
// chunk index is XOR-swizzled with the row so that the 16-byte writes of the
// global->LDS copy and the 16-byte fragment reads of the MFMA loop avoid bank
// conflicts.  An operand that is contiguous along M/N in memory is transposed
// in registers on its way to LDS (fp32), or copied as is and read back with
// the transposing LDS read (bf16).  Direct global->LDS copies fill a ring of
// 3 + 2 operand stages (all 160 KiB of LDS), keeping one operand's copies two
// steps and the other's one step ahead of the MFMAs; the register-staged
// copies (fp32 M/N-contiguous operands) use two stages and keep step k+2 in
// registers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace mc {

typedef __bf16 bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 half_t;
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBM = 256;                       // tile rows (M)
constexpr int kBN = 256;                       // tile columns (N)
constexpr int kRowBytes = 128;                 // K bytes per tile row per stage
#ifndef MC_WAVES_M
#define MC_WAVES_M 2
#endif
#ifndef MC_WAVES_N
#define MC_WAVES_N 4
#endif
constexpr int kWavesM = MC_WAVES_M;            // waves along M
constexpr int kWavesN = MC_WAVES_N;            // waves along N
constexpr int kThreads = 64 * kWavesM * kWavesN;
constexpr int kWaves = kWavesM * kWavesN;
constexpr int kWaveRows = kBM / kWavesM;       // 128
constexpr int kWaveCols = kBN / kWavesN;       // 64
constexpr int kTM = kWaveRows / 16;            // 16-row accumulator blocks per wave
constexpr int kTN = kWaveCols / 16;            // 16-column accumulator blocks per wave
constexpr int kStageBytes = kBM * kRowBytes;   // 32 KiB per operand per stage
constexpr int kLdsGemm = 4 * kStageBytes;      // 2 operands x 2 stages
// The ring of the two-K-contiguous-operand loop: 3 stages of one operand and
// 2 of the other, all of gfx950's 160 KiB.  Epilogues may use the bytes past
// kLdsGemm once the loop is over.
constexpr int kLdsRing = 5 * kStageBytes;
constexpr int kGroupM = 8;                     // tile rows per scheduling group
// Copies (of a wave's 4) of each deep stage that go out in the first half of
// the step two before their use instead of right after the barrier that
// freed their slot (see gemm_mainloop_dma).  All 4: the copy issues then
// alternate between the two halves of a step, 4 each; measured 0.3 ms faster
// per recompute step than 0 (forward -0.13 ms, softmax contraction -0.15,
// dH -0.2), while 1 and 2 were slower than 0.
constexpr int kDeepLate = 4;
// The same for the loop with inline-asm copies (dW; all of a stage's deep
// copies or none): measured 0.1-0.3 ms faster for dW.
constexpr bool kDeepLateAsm = true;
constexpr int kXcds = 8;                       // MI355X: 8 XCDs, workgroup i -> XCD i % 8

typedef f32x4 Acc[kTM][kTN];

template <typename T> struct Elem;
template <> struct Elem<bf16_t> { static constexpr int kChunk = 8; };
template <> struct Elem<half_t> { static constexpr int kChunk = 8; };
template <> struct Elem<float> { static constexpr int kChunk = 4; };

// Operand of a contraction C[m][n] = sum_k A[m][k] B[n][k].  For A the "rows"
// are M, for B they are N.  Rows >= rows and k >= K read as zero, at the
// granularity of a 16-byte chunk: a K-contiguous operand's chunk is copied
// whole when its first element is below K, so up to the next multiple of the
// chunk (8 bf16, 4 fp32) past K must be readable and hold zeros (or K be a
// multiple of it); an M/N-contiguous operand's chunk is taken whole when its
// first row is below `rows`, with the same rule along the rows.  The layout
// is a template policy of the copy (see below); `ld` is its stride parameter.
struct Operand {
  const void* ptr;
  int64_t ld;
  int64_t rows;
  int64_t K;
};

// Layout policies.  A 16-byte chunk runs along k for the K-contiguous kinds
// and along r for the M/N-contiguous ones.
//   KMajor   (r, k) at r * ld + k
//   MNMajor  (r, k) at k * ld + r
//   TileTK   panel buffer read with r = token, k = vocab
//   TileVT   the same buffer read with r = vocab, k = token
// The panel buffer (the backward's transient operand) holds the vocabulary
// in panels of BV = 128 bytes of elements; panel j is a row-major
// [ld x BV] matrix (ld = padded token count), panels stored one after the
// other: element (t, v) at (v / BV) * ld * BV + t * BV + v % BV.  Every
// 128-byte run either contraction reads is contiguous.
enum class Lay { KMajor, MNMajor, TileTK, TileVT };

template <Lay L> struct KContig {
  static constexpr bool value = (L == Lay::KMajor || L == Lay::TileTK);
};

// Byte offsets: base of the tile starting at row r0 (stage 0), the advance of
// one K stage, and the offset of (r0 + dr, k0 + dk) relative to the stage base.
template <typename T, Lay L> struct LayMath {
  static constexpr int64_t es = sizeof(T);
  static constexpr int64_t BV = 128 / sizeof(T);
  static constexpr int64_t KT = 128 / sizeof(T);
  __host__ __device__ static int64_t tile_base(const Operand& op, int64_t r0) {
    if constexpr (L == Lay::KMajor) return r0 * op.ld * es;
    else if constexpr (L == Lay::MNMajor) return r0 * es;
    else if constexpr (L == Lay::TileTK) return r0 * BV * es;
    else return (r0 / BV) * op.ld * BV * es;
  }
  __host__ __device__ static int64_t stage_step(const Operand& op) {
    if constexpr (L == Lay::KMajor) return KT * es;
    else if constexpr (L == Lay::MNMajor) return KT * op.ld * es;
    else if constexpr (L == Lay::TileTK) return op.ld * BV * es;
    else return KT * BV * es;
  }
  __host__ __device__ static uint32_t rel(const Operand& op, int dr, int dk) {
    if constexpr (L == Lay::KMajor) return uint32_t((int64_t(dr) * op.ld + dk) * es);
    else if constexpr (L == Lay::MNMajor) return uint32_t((int64_t(dk) * op.ld + dr) * es);
    else if constexpr (L == Lay::TileTK) return uint32_t((int64_t(dr) * BV + dk) * es);
    else return uint32_t(((dr / BV) * op.ld * BV + int64_t(dk) * BV + dr % BV) * es);
  }
};

constexpr uint32_t kBufRange = 0x7ffffff0u;   // records of every operand resource
constexpr uint32_t kBufOut = 0x80000000u;     // an offset past the range: reads zero

// Host-side check used before every launch: the last in-range chunk of the
// operand (offsets grow with r and k in every layout) lies inside `bytes`,
// the per-thread 32-bit offsets of one tile cannot overflow, and K fits the
// copies' 32-bit K bounds.
template <typename T, Lay L>
inline bool operand_in_bounds(const Operand& op, size_t bytes) {
  using M = LayMath<T, L>;
  constexpr int64_t E = Elem<T>::kChunk;
  if (op.rows < 1 || op.K < 1 || op.K > int64_t(0x7fffffff) - 2 * M::KT) return false;
  int64_t r = op.rows - 1, k = op.K - 1;
  if (KContig<L>::value) k = k / E * E; else r = r / E * E;
  const int64_t last = M::tile_base(op, r / 256 * 256) + (k / M::KT) * M::stage_step(op) +
                       int64_t(M::rel(op, int(r % 256), int(k % M::KT)));
  const int64_t span = (L == Lay::KMajor) ? 256 * op.ld * M::es
                       : (L == Lay::MNMajor) ? M::KT * op.ld * M::es
                       : (L == Lay::TileVT) ? 256 * op.ld * M::es : 256 * M::BV * M::es;
  return last >= 0 && size_t(last) + 16 <= bytes && span + 16 <= int64_t(kBufRange);
}

__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 2)) & 7; }
__device__ __forceinline__ int lds_off(int r, int c) {
  return r * kRowBytes + ((c ^ swz(r)) << 4);
}

// Workgroup id -> (tile row, tile column).  The first 8*floor(n/8) ids are
// regrouped so that each XCD receives a contiguous run of logical tiles; the
// logical order walks group_m tile rows before moving to the next tile column,
// so the 32 workgroups resident on one XCD share a few operand panels in its L2.
// With `count` < nTm nTn only the first `count` logical tiles are regrouped
// and handed out (the rest are covered by another launch shape).
__device__ __forceinline__ void tile_of_logical(int L, int nTm, int nTn, int group_m, int& tm,
                                                int& tn) {
  const int group = group_m * nTn;
  const int g = L / group;
  const int first = g * group_m;
  const int gm = min(nTm - first, group_m);
  const int r = L - g * group;
  tm = first + r % gm;
  tn = r / gm;
}
__device__ __forceinline__ void tile_of(int bid, int nTm, int nTn, int group_m, int& tm, int& tn,
                                        int count = -1) {
  const int total = count < 0 ? nTm * nTn : count;
  const int q = total / kXcds;
  int L = bid;
  if (bid < q * kXcds) L = (bid % kXcds) * q + bid / kXcds;
  tile_of_logical(L, nTm, nTn, group_m, tm, tn);
}

// The operand restricted to K columns [k0, k0 + len): k0 is a multiple of the
// stage depth, so the slice starts at a stage boundary of every layout.
template <typename T, Lay L>
__host__ __device__ inline Operand k_slice(const Operand& op, int64_t k0, int64_t len) {
  using M = LayMath<T, L>;
  Operand o = op;
  o.ptr = static_cast<const char*>(op.ptr) + (k0 / M::KT) * M::stage_step(op);
  o.K = len;
  return o;
}

// Tail split: when the last round of tiles fills at most half of the CUs,
// its `rem` tiles are each split into `splits` K ranges of `ks` columns
// (whole stages), computed by rem * splits workgroups into fp32 slots and
// summed in split order by a second kernel.  full = the tiles computed
// whole.  At most kTailSlots slots.
constexpr int kTailSlots = 256;
struct TailSplit {
  int full, rem, splits;
  int64_t ks;
};
// `cap`: the slots available.  Host and device (a kernel may plan from a
// tile count it reads from device memory).
__host__ __device__ inline TailSplit plan_tail(int total, int64_t K, int ncu,
                                               int cap = kTailSlots) {
  constexpr int64_t kStage = 64;   // K columns of one bf16 stage (32 for fp32; a multiple works)
  TailSplit t{total, 0, 1, K};
  if (ncu <= 0) return t;
  const int rem = total % ncu;
  if (rem == 0 || 2 * rem > ncu) return t;
  const int room = ncu < cap ? ncu : cap;
  int splits = 1;
  while (splits < 8 && rem * splits * 2 <= room && K >= int64_t(splits) * 2 * 4 * kStage)
    splits *= 2;
  const int64_t nst = (K + kStage - 1) / kStage;
  int64_t ks = (nst + splits - 1) / splits * kStage;
  while (splits > 1 && int64_t(splits - 1) * ks >= K) {   // every split non-empty
    splits /= 2;
    ks = (nst + splits - 1) / splits * kStage;
  }
  if (splits == 1) return t;
  t.full = total - rem;
  t.rem = rem;
  t.splits = splits;
  t.ks = ks;
  return t;
}

// ---------------------------------------------------------------------------
// Global -> register -> LDS copy of one 256-row x 128-byte operand stage.
// Every copy keeps a uniform 64-bit tile base and per-thread 32-bit offsets
// computed once per tile, and reads through a buffer resource rebased at
// each K stage.  An out-of-range chunk gets an offset past the resource's
// range, which the hardware's range check turns into zeros without touching
// memory: only the 32-bit offset is selected, never the loaded value, so
// nothing waits on a load before its data is needed in LDS.
// ---------------------------------------------------------------------------

__device__ __forceinline__ __amdgpu_buffer_rsrc_t stage_rsrc(const char* base) {
  // raw (stride 0) resource; 0x00020000 is the gfx9 untyped-buffer word 3
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), (short)0, int(kBufRange),
                                           0x00020000);
}

__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

template <typename T, Lay L, bool KC = KContig<L>::value> struct StageCopy;

// K-contiguous: thread owns chunk (tid & 7) of rows (tid >> 3) + kPass * i.
template <typename T, Lay L> struct StageCopy<T, L, true> {
  using M = LayMath<T, L>;
  static constexpr int E = Elem<T>::kChunk;
  static constexpr int kPass = kThreads / 8;   // rows per pass
  static constexpr int NL = kBM / kPass;       // loads per thread
  u32x4 r[NL];
  const char* tb;
  int64_t step, K;
  uint32_t off[NL];
  uint32_t rowok;
  int kc;
  __device__ __forceinline__ void init(const Operand& op, int64_t r0, int tid) {
    tb = static_cast<const char*>(op.ptr) + M::tile_base(op, r0);
    step = M::stage_step(op);
    K = op.K;
    kc = (tid & 7) * E;
    rowok = 0;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int dr = (tid >> 3) + kPass * i;
      off[i] = M::rel(op, dr, kc);
      if (r0 + dr < op.rows) rowok |= 1u << i;
    }
  }
  __device__ __forceinline__ void load(int64_t kt) {
    const __amdgpu_buffer_rsrc_t rs = stage_rsrc(tb + kt * step);
    const bool kok = kt * M::KT + kc < K;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const bool ok = kok && ((rowok >> i) & 1u);
      r[i] = buf_load16(rs, ok ? off[i] : kBufOut);
    }
  }
  __device__ __forceinline__ void store(char* lds, int tid) const {
    const int c = tid & 7;
#pragma unroll
    for (int i = 0; i < NL; ++i)
      *reinterpret_cast<u32x4*>(lds + lds_off((tid >> 3) + kPass * i, c)) = r[i];
  }
};

// M/N-contiguous fp32: 4(k) x 4(mn) blocks (mn-block b & 63, k-block b >> 6),
// kThreads/... per thread, transposed by register moves.
template <Lay L> struct StageCopy<float, L, false> {
  using M = LayMath<float, L>;
  static constexpr int NB = 512 / kThreads;   // blocks per thread
  u32x4 r[4 * NB];
  const char* tb;
  int64_t step, K;
  uint32_t off0[NB], dk_bytes;
  int kb[NB];
  bool mnok[NB];
  __device__ __forceinline__ void init(const Operand& op, int64_t r0, int tid) {
    tb = static_cast<const char*>(op.ptr) + M::tile_base(op, r0);
    step = M::stage_step(op);
    K = op.K;
#pragma unroll
    for (int h = 0; h < NB; ++h) {
      const int b = tid + kThreads * h;
      kb[h] = (b >> 6) * 4;
      off0[h] = M::rel(op, (b & 63) * 4, kb[h]);
      mnok[h] = r0 + (b & 63) * 4 < op.rows;
    }
    dk_bytes = M::rel(op, (tid & 63) * 4, kb[0] + 1) - off0[0];
  }
  __device__ __forceinline__ void load(int64_t kt) {
    const __amdgpu_buffer_rsrc_t rs = stage_rsrc(tb + kt * step);
#pragma unroll
    for (int h = 0; h < NB; ++h) {
      const int64_t k0 = kt * M::KT + kb[h];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool ok = mnok[h] && (k0 + i < K);
        r[4 * h + i] = buf_load16(rs, ok ? off0[h] + i * dk_bytes : kBufOut);
      }
    }
  }
  __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
    for (int h = 0; h < NB; ++h) {
      const int b = tid + kThreads * h;
      const int row0 = (b & 63) * 4;
      const int c = b >> 6;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        u32x4 out{r[4 * h + 0][j], r[4 * h + 1][j], r[4 * h + 2][j], r[4 * h + 3][j]};
        *reinterpret_cast<u32x4*>(lds + lds_off(row0 + j, c)) = out;
      }
    }
  }
};

// ---------------------------------------------------------------------------
// One 128-byte K stage of MFMA work for this wave's sub-tile.  Lane l
// supplies row (l & 31) of each 32-row block and K-chunk (l >> 5) of each
// 32-byte K slice; A and B use the same lane -> k assignment.
// ---------------------------------------------------------------------------
// Compile-time loop: f(integral_constant<int, i>) for i = b .. e-1.
template <int V> struct IntC {
  static constexpr int value = V;
};
template <int b, int e, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (b < e) {
    f(IntC<b>{});
    static_for<b + 1, e>(f);
  }
}

template <bool c, class X, class Y>
__device__ __forceinline__ auto& pick(X& x, Y& y) {
  if constexpr (c) return x; else return y;
}

template <typename T> struct Mfma;

// Issue order: the 8 row blocks of one column block, then the next column
// block, so that consecutive MFMAs of a wave share their B operand (the
// forward measured 0.1 ms faster than row blocks first; the part is
// power-limited, and fewer operand changes toggle fewer bits).  Each
// accumulator block sees the same K order either way.
template <> struct Mfma<bf16_t> {
  __device__ __forceinline__ static void step(Acc& acc, const u32x4 (&a)[kTM],
                                              const u32x4 (&b)[kTN]) {
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
      for (int i = 0; i < kTM; ++i)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8, a[i]), __builtin_bit_cast(bf16x8, b[j]), acc[i][j], 0, 0, 0);
  }
  // the MFMAs r0 .. r1-1 of step()'s order (r = j kTM + i)
  template <int r0, int r1>
  __device__ __forceinline__ static void range(Acc& acc, const u32x4 (&a)[kTM],
                                               const u32x4 (&b)[kTN]) {
#pragma unroll
    for (int r = r0; r < r1; ++r)
      acc[r % kTM][r / kTM] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
          __builtin_bit_cast(bf16x8, a[r % kTM]), __builtin_bit_cast(bf16x8, b[r / kTM]),
          acc[r % kTM][r / kTM], 0, 0, 0);
  }
};

// fp16 operands (the backward's scaled transient operand and transposes):
// the same 16 x 16 x 32 shape and rate as bf16, with 11 significant bits.
template <> struct Mfma<half_t> {
  __device__ __forceinline__ static void step(Acc& acc, const u32x4 (&a)[kTM],
                                              const u32x4 (&b)[kTN]) {
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
      for (int i = 0; i < kTM; ++i)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
            __builtin_bit_cast(f16x8, a[i]), __builtin_bit_cast(f16x8, b[j]), acc[i][j], 0, 0, 0);
  }
  // the MFMAs r0 .. r1-1 of step()'s order (r = j kTM + i)
  template <int r0, int r1>
  __device__ __forceinline__ static void range(Acc& acc, const u32x4 (&a)[kTM],
                                               const u32x4 (&b)[kTN]) {
#pragma unroll
    for (int r = r0; r < r1; ++r)
      acc[r % kTM][r / kTM] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
          __builtin_bit_cast(f16x8, a[r % kTM]), __builtin_bit_cast(f16x8, b[r / kTM]),
          acc[r % kTM][r / kTM], 0, 0, 0);
  }
};

// fp32: each 16-byte chunk holds 4 K values, consumed by 4 MFMAs of K = 4
// (element e of lane group g is k = 4 g + e of the step; A and B agree).
// (The chunks are bit-cast to float vectors as a whole: bit-casting a single
// element of an integer vector compiles to element 0 with this toolchain.)
template <> struct Mfma<float> {
  __device__ __forceinline__ static void step(Acc& acc, const u32x4 (&a)[kTM],
                                              const u32x4 (&b)[kTN]) {
    f32x4 af[kTM], bf[kTN];
#pragma unroll
    for (int i = 0; i < kTM; ++i) af[i] = __builtin_bit_cast(f32x4, a[i]);
#pragma unroll
    for (int j = 0; j < kTN; ++j) bf[j] = __builtin_bit_cast(f32x4, b[j]);
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int i = 0; i < kTM; ++i)
#pragma unroll
        for (int j = 0; j < kTN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i][e], bf[j][e], acc[i][j], 0, 0, 0);
  }
};

// LDS format of one operand stage.  K: 256 rows of 128 bytes of K (the
// register-staged copies and the direct copies of K-contiguous operands).
// MN (bf16 only): 64 K rows of 256 elements along M/N, 512 bytes each, the
// 16-byte chunk index XOR-ed with mn_swz(k); fragments are read with the
// transposing LDS read.
enum class Stg { K, MN };

// The 8 K rows one half-wave of a transposing fragment read touches
// (k0 + {0..3, 8..11}) get 8 distinct chunk offsets, so its 16 chunks fall
// in distinct bank groups.
__device__ __forceinline__ int mn_swz(int k) { return ((k & 3) << 2) | (((k >> 3) & 1) << 1); }

__device__ __forceinline__ int lds_off_mn(int k, int m) {
  return k * (kBM * 2) + (((m >> 3) ^ mn_swz(k)) << 4) + ((m & 7) << 1);
}

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4_t;

// One 16 x 32 MFMA operand fragment (lane l: row l % 16, k = 8 (l / 16) + 0..7
// of K step ks) from an MN stage.  ds_read_b64_tr_b16 hands lane i of each
// 16-lane group element i % 4 of the 8-byte pieces loaded by lanes
// 4 e + i / 4 (e = 0..3) of that group; so lane s loads 4 consecutive rows at
// one k, and after the exchange each lane holds 4 consecutive k of one row.
// Two reads give 8.
__device__ __forceinline__ u32x4 read_frag_mn(const char* base, int row0, int ks, int lane) {
  const int g = lane >> 4, s = lane & 15;
  const int k = 32 * ks + 8 * g + (s >> 2);
  const int m = row0 + 4 * (s & 3);
  const char* p = base + lds_off_mn(k, m);
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)p);
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(p + 4 * kBM * 2));
  const u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
  return u32x4{a[0], a[1], b[0], b[1]};
}

// Fragment of K step ks (32 bf16 or 16 fp32 of the stage's 128 bytes):
// lane l reads row row0 + l % 16, 16-byte chunk 4 ks + l / 16.
// For a K stage the lane's part of the address depends only on ks and on
// the parity of the 16-row block (rows 32 apart share the swizzle), so the
// blocks of a wave differ by compile-time offsets.
__device__ __forceinline__ int kfrag_lane_off(int ks, int par, int lane) {
  const int x = lane & 15, c = 4 * ks + (lane >> 4);
  const int sw = ((x & 7) ^ ((4 * par + (x >> 2)) & 7)) & 7;   // swz(32 q + 16 par + x)
  return x * kRowBytes + ((c ^ sw) << 4);
}

// row0 (a multiple of 16): first row of the block; wave bases are multiples
// of 32.
template <Stg S>
__device__ __forceinline__ u32x4 read_frag(const char* base, int row0, int ks, int lane) {
  if constexpr (S == Stg::K)
    return *reinterpret_cast<const u32x4*>(base + row0 * kRowBytes +
                                           kfrag_lane_off(ks, (row0 >> 4) & 1, lane));
  else
    return read_frag_mn(base, row0, ks, lane);
}

template <typename T, Stg SA, Stg SB>
__device__ __forceinline__ void read_frags(u32x4 (&a)[kTM], u32x4 (&b)[kTN], const char* ldsA,
                                           const char* ldsB, int wm, int wn, int lane, int ks) {
#pragma unroll
  for (int i = 0; i < kTM; ++i) a[i] = read_frag<SA>(ldsA, wm * kWaveRows + i * 16, ks, lane);
#pragma unroll
  for (int j = 0; j < kTN; ++j) b[j] = read_frag<SB>(ldsB, wn * kWaveCols + j * 16, ks, lane);
}

// The two K steps of one stage; the fragments of step 1 are requested
// behind the MFMAs of step 0.
template <typename T, Stg SA = Stg::K, Stg SB = Stg::K>
__device__ __forceinline__ void mfma_stage(Acc& acc, const char* ldsA, const char* ldsB, int wm,
                                           int wn, int lane) {
  u32x4 a0[kTM], b0[kTN], a1[kTM], b1[kTN];
  read_frags<T, SA, SB>(a0, b0, ldsA, ldsB, wm, wn, lane, 0);
  Mfma<T>::step(acc, a0, b0);
  read_frags<T, SA, SB>(a1, b1, ldsA, ldsB, wm, wn, lane, 1);
  Mfma<T>::step(acc, a1, b1);
}

// ---------------------------------------------------------------------------
// Direct global->LDS copy (buffer_load ... lds) of one K-contiguous operand
// stage.  One wave instruction fills 1 KiB of LDS (8 tile rows of 128 bytes),
// lane i writing the 16 bytes at offset 16 i; each lane therefore loads the
// global chunk that the swizzle assigns to its slot.  No registers hold the
// data, and the copy of stage k+1 overlaps the MFMAs of stage k.
// ---------------------------------------------------------------------------
typedef int i32x4 __attribute__((ext_vector_type(4)));

// Buffer resource words of a raw (stride 0) view starting at `base`, forced
// into scalar registers (the base is uniform across the wave by construction).
__device__ __forceinline__ i32x4 dma_rsrc(const char* base) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane(int(uint32_t(a)));
  r[1] = __builtin_amdgcn_readfirstlane(int(uint32_t(a >> 32) & 0xffffu));
  r[2] = int(kBufRange);
  r[3] = 0x00020000;
  return r;
}

// LDS byte address of a (wave-uniform) pointer into the workgroup's LDS.
__device__ __forceinline__ uint32_t lds_addr(const char* p) {
  return __builtin_amdgcn_readfirstlane(
      uint32_t(uintptr_t((__attribute__((address_space(3))) const char*)p)));
}

// One 16-byte-per-lane direct load into LDS: lane i's chunk lands at
// m0 + 16 i.  Issued from inline asm so that the compiler's wait insertion
// does not serialise later LDS reads behind the copy; the loops that issue
// these wait for them explicitly (vmcnt) before their barrier, and no
// compiler-generated vector-memory load is outstanding meanwhile.
// The compiler inserts no hazard padding before an asm statement, so the
// statement carries its own: a VALU write of an SGPR (the readfirstlane of
// the resource words) needs 5 wait states before a vector-memory
// instruction reads that SGPR, and an SALU write of m0 needs 1 before the
// LDS-direct load.
__device__ __forceinline__ void dma16(const i32x4& rs, uint32_t voff, uint32_t m0) {
  asm volatile("s_nop 4\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :: "v"(voff), "s"(rs), "{m0}"(m0) : "memory");
}

// The same base pointer with both halves forced into scalar registers.
__device__ __forceinline__ const char* uniform_ptr(const char* p) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  const uint64_t lo = uint32_t(__builtin_amdgcn_readfirstlane(int(uint32_t(a))));
  const uint64_t hi = uint32_t(__builtin_amdgcn_readfirstlane(int(uint32_t(a >> 32))));
  return reinterpret_cast<const char*>((hi << 32) | lo);
}

// kAsm: issue through dma16 (loops that also use the transposing LDS read,
// which the compiler would otherwise order behind every copy in flight);
// otherwise through the compiler builtin.
// Wave w copies the 1 KiB groups w + kWaves i (i = 0..NI-1).  Groups kWaves
// apart are 8 kWaves = 64 rows apart, where both swizzles repeat, so every
// group of a wave has the same lane -> chunk pattern: one offset register,
// a constant stride per group, one K bound.
template <typename T, Lay L, bool kAsm> struct DmaCopy {
  using M = LayMath<T, L>;
  static constexpr int E = Elem<T>::kChunk;
  static constexpr int NI = kBM / 8 / kWaves;   // 1 KiB groups per wave
  static_assert(8 * kWaves % 32 == 0, "group stride must keep the row swizzle");
  const char* tb;
  int64_t step;
  uint32_t off0, istride;
  int klim;   // K - (this lane's chunk column): the chunk of step kt is in range iff kt KT < klim
  uint32_t rowok;
  int grp;
  __device__ __forceinline__ void init(const Operand& op, int64_t r0, int tid) {
    tb = static_cast<const char*>(op.ptr) + M::tile_base(op, r0);
    step = M::stage_step(op);
    const int lane = tid & 63;
    grp = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int row = 8 * grp + (lane >> 3);
    const int kc = ((lane & 7) ^ swz(row)) * E;
    klim = int(op.K) - kc;
    off0 = M::rel(op, row, kc);
    istride = M::rel(op, row + 8 * kWaves, kc) - off0;
    rowok = 0;
#pragma unroll
    for (int i = 0; i < NI; ++i)
      if (r0 + row + 8 * kWaves * i < op.rows) rowok |= 1u << i;
  }
  // one copy at a time (inline-asm path): prep() once per step, then one(i)
  struct Step {
    i32x4 rs;
    uint32_t m0;
    bool kok;
  };
  __device__ __forceinline__ Step prep(int64_t kt, char* lds) const {
    return Step{dma_rsrc(tb + kt * step), lds_addr(lds) + grp * 1024,
                int(kt) * int(M::KT) < klim};
  }
  __device__ __forceinline__ void one(const Step& h, int i) const {
    const bool ok = h.kok && ((rowok >> i) & 1u);
    dma16(h.rs, ok ? off0 + i * istride : kBufOut, h.m0 + i * kWaves * 1024);
  }
  // the copies i0 .. i1-1 of one stage (builtin path)
  template <int i0, int i1>
  __device__ __forceinline__ void issue_part(int64_t kt, char* lds) const {
    static_assert(!kAsm, "builtin copies");
    const bool kok = int(kt) * int(M::KT) < klim;
    const __amdgpu_buffer_rsrc_t rs = stage_rsrc(uniform_ptr(tb + kt * step));
#pragma unroll
    for (int i = i0; i < i1; ++i) {
      const bool ok = kok && ((rowok >> i) & 1u);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rs, (__attribute__((address_space(3))) void*)(lds + (grp + i * kWaves) * 1024), 16,
          ok ? off0 + i * istride : kBufOut, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void issue(int64_t kt, char* lds) const {
    const bool kok = int(kt) * int(M::KT) < klim;
    if constexpr (kAsm) {
      const i32x4 rs = dma_rsrc(tb + kt * step);
      const uint32_t m0 = lds_addr(lds) + grp * 1024;
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const bool ok = kok && ((rowok >> i) & 1u);
        dma16(rs, ok ? off0 + i * istride : kBufOut, m0 + i * kWaves * 1024);
      }
    } else {
      const __amdgpu_buffer_rsrc_t rs = stage_rsrc(uniform_ptr(tb + kt * step));
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const bool ok = kok && ((rowok >> i) & 1u);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rs, (__attribute__((address_space(3))) void*)(lds + (grp + i * kWaves) * 1024), 16,
            ok ? off0 + i * istride : kBufOut, 0, 0, 0);
      }
    }
  }
};

// Direct copy of one M/N-contiguous bf16 operand stage into the MN format:
// one wave instruction fills 1 KiB (two K rows of 256 elements); lane i
// writes slot i % 32 of K row 2 g + i / 32 and loads the 8-element chunk
// that the swizzle assigns to that slot.  Wave w takes the groups
// w + kWaves i: K rows 16 i apart, where mn_swz repeats.
template <Lay L> struct DmaCopyMN {
  using M = LayMath<bf16_t, L>;
  static constexpr int NI = kStageBytes / 1024 / kWaves;   // 1 KiB groups per wave
  static_assert(2 * kWaves % 16 == 0, "group stride must keep the K-row swizzle");
  const char* tb;
  int64_t step;
  uint32_t off0, istride;
  int klim;   // K - (this lane's first K row): group i of step kt is in range iff kt KT + 2 kWaves i < klim
  bool mok;
  int grp;
  __device__ __forceinline__ void init(const Operand& op, int64_t r0, int tid) {
    tb = static_cast<const char*>(op.ptr) + M::tile_base(op, r0);
    step = M::stage_step(op);
    const int lane = tid & 63;
    grp = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int k0 = 2 * grp + (lane >> 5);
    klim = int(op.K) - k0;
    const int c = (lane & 31) ^ mn_swz(k0);
    off0 = M::rel(op, 8 * c, k0);
    istride = M::rel(op, 8 * c, k0 + 2 * kWaves) - off0;
    mok = r0 + 8 * c < op.rows;
  }
  struct Step {
    i32x4 rs;
    uint32_t m0;
    int kk;
  };
  __device__ __forceinline__ Step prep(int64_t kt, char* lds) const {
    return Step{dma_rsrc(tb + kt * step), lds_addr(lds) + grp * 1024, int(kt) * int(M::KT)};
  }
  __device__ __forceinline__ void one(const Step& h, int i) const {
    const bool ok = mok && (h.kk + 2 * kWaves * i < klim);
    dma16(h.rs, ok ? off0 + i * istride : kBufOut, h.m0 + i * kWaves * 1024);
  }
  __device__ __forceinline__ void issue(int64_t kt, char* lds) const {
    const Step h = prep(kt, lds);
#pragma unroll
    for (int i = 0; i < NI; ++i) one(h, i);
  }
};

template <typename T, Lay L> struct DmaOf {
  static constexpr Stg stg = KContig<L>::value ? Stg::K : Stg::MN;
};
template <typename T, Lay L, bool kAsm, bool KC = KContig<L>::value> struct DmaSel;
template <typename T, Lay L, bool kAsm> struct DmaSel<T, L, kAsm, true> {
  typedef DmaCopy<T, L, kAsm> type;
};
template <Lay L, bool kAsm> struct DmaSel<bf16_t, L, kAsm, false> { typedef DmaCopyMN<L> type; };
template <Lay L, bool kAsm> struct DmaSel<half_t, L, kAsm, false> { typedef DmaCopyMN<L> type; };

// All of this wave's direct copies have landed, then a workgroup barrier.
// The barrier carries no memory fence (the fence of __syncthreads would wait
// for every copy in flight); the empty asm statements keep the compiler from
// moving LDS accesses across it.
__device__ __forceinline__ void dma_wait_barrier() {
  __builtin_amdgcn_s_waitcnt(0x3f70);   // vmcnt(0), other counters unconstrained
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Direct-copy K loop.  Two LDS stages, copies two steps ahead, one barrier
// per step placed between the two K sub-steps of a stage:
//   read sub-step 1 of stage k | MFMAs of sub-step 0 of stage k |
//   wait (this wave's copies of stage k+1 landed, its reads of stage k done),
//   barrier | copy stage k+2 into stage k's buffer | read sub-step 0 of
//   stage k+1 | MFMAs of sub-step 1 of stage k
// so the MFMAs after the barrier already have their fragments in registers
// while the next stage's first reads are in flight.
// kSpread: MFMAs between consecutive copy issues after the barrier of the
// cross-barrier loop (2 for the forward and dH: measured).  kDeepA: operand
// A gets the 3-stage side of the ring (else B).
template <typename T, Lay LA, Lay LB, int kSpread = 1, bool kDeepA = true>
__device__ __forceinline__ void gemm_mainloop_dma(const Operand& A, const Operand& B, int64_t m0,
                                                  int64_t n0, int64_t K, char* lds, Acc& acc) {
  constexpr int KT = kRowBytes / sizeof(T);
  constexpr Stg SA = DmaOf<T, LA>::stg, SB = DmaOf<T, LB>::stg;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % kWavesM, wn = wave / kWavesM;
  const int64_t nk = (K + KT - 1) / KT;

#pragma unroll
  for (int i = 0; i < kTM; ++i)
#pragma unroll
    for (int j = 0; j < kTN; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  if (nk <= 0) return;

  constexpr bool kAsm = !(KContig<LA>::value && KContig<LB>::value);
  using CA = typename DmaSel<T, LA, kAsm>::type;
  using CB = typename DmaSel<T, LB, kAsm>::type;
  CA ca;
  CB cb;
  ca.init(A, m0, tid);
  cb.init(B, n0, tid);
  if constexpr (SA == Stg::MN) {
    ca.issue(0, lds);
    cb.issue(0, lds + kStageBytes);
    // A transposing-read A operand needs per-block fragment addresses for its
    // kTM blocks; without the spare registers for the cross-barrier
    // prefetch, one barrier at the top of each step: it publishes step k and
    // releases step k-1's buffer.  (With the transposing reads on B, kTN
    // blocks, the cross-barrier loop below fits and is faster.)
    constexpr int kReads = (SA == Stg::MN ? 2 : 1) * kTM + (SB == Stg::MN ? 2 : 1) * kTN;
    for (int64_t kt = 0; kt < nk; ++kt) {
      char* cur = lds + (kt & 1) * (2 * kStageBytes);
      char* nxt = lds + ((kt + 1) & 1) * (2 * kStageBytes);
      dma_wait_barrier();
      __builtin_amdgcn_sched_barrier(0);
      // past the end: zero-filling copies into the released buffer
      ca.issue(kt + 1, nxt);
      cb.issue(kt + 1, nxt + kStageBytes);
      u32x4 a0[kTM], b0[kTN], a1[kTM], b1[kTN];
      read_frags<T, SA, SB>(a0, b0, cur, cur + kStageBytes, wm, wn, lane, 0);
      Mfma<T>::step(acc, a0, b0);
      read_frags<T, SA, SB>(a1, b1, cur, cur + kStageBytes, wm, wn, lane, 1);
      Mfma<T>::step(acc, a1, b1);
      // the step-1 reads go out one per MFMA of step 0
      __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);   // step-0 reads
#pragma unroll
      for (int r = 0; r < kReads; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);     // step-1 read
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2 * kTM * kTN - kReads, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_s_waitcnt(0x0070);
    __syncthreads();
    return;
  }
  // Cross-barrier loop over a ring of kNA stages of A and kNB of B (one of
  // them 3 deep): stage k of A lives in slot k % kNA at ldsA, of B in slot
  // k % kNB at ldsB.  After the barrier of step k the slots of step k are
  // free; the shallow operand's copy of step k + 2 is issued first, then the
  // deep operand's of step k + 3, so the wait for step k + 1 before the next
  // barrier may leave exactly the deep operand's newest copies in flight.
  constexpr int kNA = kDeepA ? 3 : 2, kNB = kDeepA ? 2 : 3;
  // LDS reads per sub-step: one per block, two per transposed block
  constexpr int kRd = (SA == Stg::MN ? 2 : 1) * kTM + (SB == Stg::MN ? 2 : 1) * kTN;
  static_assert(kRd <= kTM * kTN, "read slots");
  static_assert((kNA + kNB) * kStageBytes <= kLdsRing, "ring");
  constexpr int kNID = kDeepA ? CA::NI : CB::NI;                // deep copies per step
  constexpr int kNIS = kDeepA ? CB::NI : CA::NI;                // shallow copies per step
  static_assert(kNIS + 2 * kNID <= 15, "vmcnt field");
  char* const ldsA = lds;
  char* const ldsB = lds + kNA * kStageBytes;
  // prologue: steps 0 and 1 of both, step 2 of the deep operand (past the
  // end: zero-filled); wait for step 0
  ca.issue(0, ldsA);
  cb.issue(0, ldsB);
  // builtin path: the last kLate copies of each deep stage k + 2 go out in
  // the first half of step k (before its barrier) rather than with the rest
  // after the barrier of step k - 1, so that fewer copies leave at once
  // (the slot was freed at that barrier; the wait before the barrier of
  // step k + 1 still leaves exactly the deep stage k + 3's copies in flight)
  // (inline-asm path: all of a stage's deep copies or none)
  constexpr int kLate = kAsm ? (kDeepLateAsm ? kNID : 0) : kDeepLate;
  static_assert(kLate >= 0 && kLate <= kNID, "late copies");
  constexpr int kCopyGap = 2;   // inline-asm path: MFMAs after each copy
  if constexpr (kDeepA) {
    cb.issue(1, ldsB + kStageBytes);
    ca.issue(1, ldsA + kStageBytes);
    if constexpr (kLate == 0)
      ca.issue(2, ldsA + 2 * kStageBytes);
    else if constexpr (kLate < kNID)
      ca.template issue_part<0, kNID - kLate>(2, ldsA + 2 * kStageBytes);
  } else {
    ca.issue(1, ldsA + kStageBytes);
    cb.issue(1, ldsB + kStageBytes);
    if constexpr (kLate == 0)
      cb.issue(2, ldsB + 2 * kStageBytes);
    else if constexpr (kLate < kNID)
      cb.template issue_part<0, kNID - kLate>(2, ldsB + 2 * kStageBytes);
  }
  __builtin_amdgcn_s_waitcnt(0x3f70 | (kNIS + 2 * kNID - kLate));
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  u32x4 a0[kTM], b0[kTN], a1[kTM], b1[kTN];
  read_frags<T, SA, SB>(a0, b0, ldsA, ldsB, wm, wn, lane, 0);
  int sa = 0, sb = 0;   // slots of step kt
  for (int64_t kt = 0; kt < nk; ++kt) {
    char* const curA = ldsA + sa * kStageBytes;
    char* const curB = ldsB + sb * kStageBytes;
    const int na = sa + 1 == kNA ? 0 : sa + 1, nb = sb + 1 == kNB ? 0 : sb + 1;
    // the slot of deep step kt+2 (freed at the barrier of step kt-1)
    char* const deep2 = kDeepA ? ldsA + (sa + 2 < kNA ? sa + 2 : sa + 2 - kNA) * kStageBytes
                               : ldsB + (sb + 2 < kNB ? sb + 2 : sb + 2 - kNB) * kStageBytes;
    if constexpr (kAsm && kLate > 0) {
      // one late copy, then kCopyGap MFMAs, each pair fenced; then the
      // fragment reads of the second half interleaved with the rest
      static_assert(kCopyGap * kLate + kRd <= kTM * kTN, "issue slots");
      const auto& cd = pick<kDeepA>(ca, cb);
      const auto hd = cd.prep(kt + 2, deep2);
      static_for<0, kLate>([&](auto c) {
        constexpr int r = decltype(c)::value;
        cd.one(hd, r);
        Mfma<T>::template range<kCopyGap * r, kCopyGap * (r + 1)>(acc, a0, b0);
        __builtin_amdgcn_sched_barrier(0);
      });
      read_frags<T, SA, SB>(a1, b1, curA, curB, wm, wn, lane, 1);
      Mfma<T>::template range<kCopyGap * kLate, kTM * kTN>(acc, a0, b0);
#pragma unroll
      for (int r = 0; r < kRd; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
      }
      __builtin_amdgcn_sched_group_barrier(0x008, kTM * kTN - kCopyGap * kLate - kRd, 0);
    } else {
      read_frags<T, SA, SB>(a1, b1, curA, curB, wm, wn, lane, 1);
      if constexpr (kLate > 0) {
        // the late copies of deep step kt+2
        if constexpr (kDeepA)
          ca.template issue_part<kNID - kLate, kNID>(kt + 2, deep2);
        else
          cb.template issue_part<kNID - kLate, kNID>(kt + 2, deep2);
      }
      Mfma<T>::step(acc, a0, b0);
      // issue order: one MFMA, one fragment read, ... so that the reads go out
      // while the MFMA pipe is busy
#pragma unroll
      for (int r = 0; r < kRd; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
      }
#pragma unroll
      for (int r = 0; r < kLate; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x008, kSpread, 0);   // MFMA
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);         // copy issue
      }
      static_assert(kRd + kSpread * kLate <= kTM * kTN, "issue slots");
      __builtin_amdgcn_sched_group_barrier(0x008, kTM * kTN - kRd - kSpread * kLate, 0);
    }
    // this wave: step kt+1 landed (only the deep operand's step kt+2 may be
    // in flight), reads of step kt returned; nothing is scheduled across the
    // barrier
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0x0070 | kNID);   // vmcnt(kNID) lgkmcnt(0)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    // the freed slots: shallow step kt+2, deep step kt+3 (past the end: every
    // chunk out of K, zero-filled, harmless in a free slot); the first
    // fragments of step kt+1 (past the end: unused)
    if constexpr (kAsm) {
      // the scheduler does not see inline-asm copies: one copy, then kCopyGap
      // MFMAs, in program order, each pair fenced (the deep copies only when
      // they do not go out late)
      constexpr int kNow = kNIS + kNID - kLate;
      static_assert(kCopyGap * kNow + kRd <= kTM * kTN, "issue slots");
      const auto& cs = pick<kDeepA>(cb, ca);   // shallow
      const auto& cd = pick<kDeepA>(ca, cb);   // deep
      const auto hs = cs.prep(kt + 2, kDeepA ? curB : curA);
      const auto hd = cd.prep(kt + 3, kDeepA ? curA : curB);
      static_for<0, kNow>([&](auto c) {
        constexpr int r = decltype(c)::value;
        if constexpr (r < kNIS)
          cs.one(hs, r);
        else
          cd.one(hd, r - kNIS);
        Mfma<T>::template range<kCopyGap * r, kCopyGap * (r + 1)>(acc, a1, b1);
        __builtin_amdgcn_sched_barrier(0);
      });
      read_frags<T, SA, SB>(a0, b0, ldsA + na * kStageBytes, ldsB + nb * kStageBytes, wm, wn,
                            lane, 0);
      Mfma<T>::template range<kCopyGap * kNow, kTM * kTN>(acc, a1, b1);
#pragma unroll
      for (int r = 0; r < kRd; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
      }
      sa = na;
      sb = nb;
      continue;
    }
    // (the inline-asm path has continued above)
    if constexpr (kDeepA) {
      cb.issue(kt + 2, curB);
      if constexpr (kLate == 0 || kAsm)
        ca.issue(kt + 3, curA);
      else
        ca.template issue_part<0, kNID - kLate>(kt + 3, curA);
    } else {
      ca.issue(kt + 2, curA);
      if constexpr (kLate == 0 || kAsm)
        cb.issue(kt + 3, curB);
      else
        cb.template issue_part<0, kNID - kLate>(kt + 3, curB);
    }
    read_frags<T, SA, SB>(a0, b0, ldsA + na * kStageBytes, ldsB + nb * kStageBytes, wm, wn,
                          lane, 0);
    Mfma<T>::step(acc, a1, b1);
    constexpr int kNow = CA::NI + CB::NI - kLate;   // copies after the barrier
    static_assert(kSpread * kNow + kRd <= kTM * kTN, "issue slots");
#pragma unroll
    for (int r = 0; r < kNow; ++r) {
      __builtin_amdgcn_sched_group_barrier(0x008, kSpread, 0);   // MFMA
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);         // copy issue
    }
#pragma unroll
    for (int r = 0; r < kRd; ++r) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kTM * kTN - kSpread * kNow - kRd, 0);
    sa = na;
    sb = nb;
  }
  // the zero-filling copies issued by the last steps land before the LDS is
  // reused
  __builtin_amdgcn_s_waitcnt(0x0070);
  __syncthreads();
}

// Full K loop with register-staged copies (loads of step k+2 in flight).
template <typename T, Lay LA, Lay LB>
__device__ __forceinline__ void gemm_mainloop_reg(const Operand& A, const Operand& B, int64_t m0,
                                                  int64_t n0, int64_t K, char* lds, Acc& acc) {
  constexpr int KT = kRowBytes / sizeof(T);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % kWavesM, wn = wave / kWavesM;
  const int64_t nk = (K + KT - 1) / KT;

#pragma unroll
  for (int i = 0; i < kTM; ++i)
#pragma unroll
    for (int j = 0; j < kTN; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  StageCopy<T, LA> ca;
  StageCopy<T, LB> cb;
  ca.init(A, m0, tid);
  cb.init(B, n0, tid);
  ca.load(0);
  cb.load(0);
  ca.store(lds, tid);
  cb.store(lds + kStageBytes, tid);
  if (nk > 1) {
    ca.load(1);
    cb.load(1);
  }
  __syncthreads();
  for (int64_t kt = 0; kt < nk; ++kt) {
    char* cur = lds + (kt & 1) * (2 * kStageBytes);
    char* nxt = lds + ((kt + 1) & 1) * (2 * kStageBytes);
    mfma_stage<T>(acc, cur, cur + kStageBytes, wm, wn, lane);
    if (kt + 1 < nk) {
      ca.store(nxt, tid);
      cb.store(nxt + kStageBytes, tid);
    }
    if (kt + 2 < nk) {
      ca.load(kt + 2);
      cb.load(kt + 2);
    }
    __syncthreads();
  }
}

// Full K loop for the tile at (m0, n0).  `lds` holds kLdsGemm bytes.  bf16,
// or fp32 with both operands K-contiguous: direct copies; otherwise (fp32
// M/N-contiguous operands) register-staged copies.
template <typename T, Lay LA, Lay LB, int kSpread = 1, bool kDeepA = true>
__device__ __forceinline__ void gemm_mainloop(const Operand& A, const Operand& B, int64_t m0,
                                              int64_t n0, int64_t K, char* lds, Acc& acc) {
  if constexpr ((KContig<LA>::value && KContig<LB>::value) || sizeof(T) == 2)
    gemm_mainloop_dma<T, LA, LB, kSpread, kDeepA>(A, B, m0, n0, K, lds, acc);
  else
    gemm_mainloop_reg<T, LA, LB>(A, B, m0, n0, K, lds, acc);
}

// This lane's wave coordinates, and the row / column (within the tile) of
// accumulator element e of block (i, j).
__device__ __forceinline__ int wave_m() { return (threadIdx.x >> 6) % kWavesM; }
__device__ __forceinline__ int wave_n() { return (threadIdx.x >> 6) / kWavesM; }
__device__ __forceinline__ int acc_row(int wm, int i, int e, int lane) {
  return wm * kWaveRows + i * 16 + 4 * (lane >> 4) + e;
}
__device__ __forceinline__ int acc_col(int wn, int j, int lane) {
  return wn * kWaveCols + j * 16 + (lane & 15);
}

// Body of every tiled contraction kernel.  Epi provides prologue(m0, n0),
// which loads the few per-lane values its epilogue needs into registers
// before the loop (the loop owns all of the LDS), and epilogue(acc, tm, tn,
// m0, n0, lds, extra, pre), which may use the LDS once the loop is over:
// the stage buffers from `lds` and kLdsRing - kLdsGemm bytes from `extra`.
// Each use is wrapped in a __global__ function of its own name (so profiles
// name the role), whose LDS array is kLdsRing bytes.
template <typename T, Lay LA, Lay LB, class Epi, int kSpread = 1, bool kDeepA = true>
__device__ __forceinline__ void gemm_body(const Operand& A, const Operand& B, int64_t K, int nTm,
                                          int nTn, const Epi& epi, char* lds,
                                          int group_m = kGroupM) {
  int tm, tn;
  tile_of(blockIdx.x, nTm, nTn, group_m, tm, tn);
  const int64_t m0 = int64_t(tm) * kBM, n0 = int64_t(tn) * kBN;
  const auto pre = epi.prologue(m0, n0);
  Acc acc;
  gemm_mainloop<T, LA, LB, kSpread, kDeepA>(A, B, m0, n0, K, lds, acc);
  epi.epilogue(acc, tm, tn, m0, n0, lds, lds + kLdsGemm, pre);
}

}  // namespace mc
