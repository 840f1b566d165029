// MFMA tile core for gfx950 (CDNA4): a 256 x 256 output tile per workgroup,
// four wave64s in a 2 x 2 arrangement, each owning 128 x 128 outputs held as
// 4 x 4 blocks of 32 x 32 fp32 accumulators.
//
// Operands are staged through LDS in a K-contiguous layout: each tile row
// holds 128 bytes of K (64 bf16 or 32 fp32) as eight 16-byte chunks, and the
// chunk index is XOR-swizzled with the row so that both the 16-byte writes of
// the global->LDS copy and the 16-byte fragment reads of the MFMA loop are free
// of bank conflicts.  An operand that is contiguous along M/N in memory is
// transposed in registers (8 x 8 bf16 or 4 x 4 fp32 blocks) on its way to LDS,
// so every contraction runs the same inner loop.  Two LDS stages: the global
// loads of step k+2 are in flight while step k is multiplied.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mc {

typedef __bf16 bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBM = 256;                       // tile rows (M)
constexpr int kBN = 256;                       // tile columns (N)
constexpr int kRowBytes = 128;                 // K bytes per tile row per stage
constexpr int kThreads = 256;                  // 4 waves
constexpr int kStageBytes = kBM * kRowBytes;   // 32 KiB per operand per stage
constexpr int kLdsGemm = 4 * kStageBytes;      // 2 operands x 2 stages
constexpr int kGroupM = 8;                     // tile rows per scheduling group
constexpr int kXcds = 8;                       // MI355X: 8 XCDs, workgroup i -> XCD i % 8

template <typename T> struct Elem;
template <> struct Elem<bf16_t> { static constexpr int kChunk = 8; };
template <> struct Elem<float> { static constexpr int kChunk = 4; };

// Operand of a contraction C[m][n] = sum_k A[m][k] B[n][k].  For A the "rows"
// are M, for B they are N.  K-major: element (r, k) at ptr[r * ld + k];
// MN-major: element (r, k) at ptr[k * ld + r].  Rows >= rows and k >= K read
// as zero.  K-major needs K % chunk == 0; MN-major needs rows % chunk == 0.
struct Operand {
  const void* ptr;
  int64_t ld;
  int64_t rows;
  int64_t K;
};

__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & 7; }
__device__ __forceinline__ int lds_off(int r, int c) {
  return r * kRowBytes + ((c ^ swz(r)) << 4);
}

// Workgroup id -> (tile row, tile column).  The first 8*floor(n/8) ids are
// regrouped so that each XCD receives a contiguous run of logical tiles; the
// logical order walks kGroupM tile rows before moving to the next tile column,
// so the 32 workgroups resident on one XCD share a few operand panels in its L2.
__device__ __forceinline__ void tile_of(int bid, int nTm, int nTn, int& tm, int& tn) {
  const int total = nTm * nTn;
  const int q = total / kXcds;
  int L = bid;
  if (bid < q * kXcds) L = (bid % kXcds) * q + bid / kXcds;
  const int group = kGroupM * nTn;
  const int g = L / group;
  const int first = g * kGroupM;
  const int gm = min(nTm - first, kGroupM);
  const int r = L - g * group;
  tm = first + r % gm;
  tn = r / gm;
}

// ---------------------------------------------------------------------------
// Global -> register -> LDS copy of one 256-row x 128-byte operand stage.
// ---------------------------------------------------------------------------
template <typename T, bool KMajor> struct StageCopy;

// K-contiguous: thread owns chunk (tid & 7) of rows (tid >> 3) + 32 i.
template <typename T> struct StageCopy<T, true> {
  static constexpr int E = Elem<T>::kChunk;
  u32x4 r[8];
  __device__ __forceinline__ void load(const Operand& op, int64_t r0, int64_t k0, int tid) {
    const int c = tid & 7;
    const int64_t kk = k0 + c * E;
    const T* base = static_cast<const T*>(op.ptr);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t row = r0 + (tid >> 3) + 32 * i;
      if (row < op.rows && kk < op.K)
        r[i] = *reinterpret_cast<const u32x4*>(base + row * op.ld + kk);
      else
        r[i] = u32x4{0u, 0u, 0u, 0u};
    }
  }
  __device__ __forceinline__ void store(char* lds, int tid) const {
    const int c = tid & 7;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      *reinterpret_cast<u32x4*>(lds + lds_off((tid >> 3) + 32 * i, c)) = r[i];
  }
};

// M/N-contiguous bf16: thread owns one 8(k) x 8(mn) block, mn-block tid & 31,
// k-block tid >> 5; transposed with byte permutes before the LDS write.
template <> struct StageCopy<bf16_t, false> {
  u32x4 r[8];
  __device__ __forceinline__ void load(const Operand& op, int64_t r0, int64_t k0, int tid) {
    const int64_t mn = r0 + (tid & 31) * 8;
    const int64_t kb = k0 + (tid >> 5) * 8;
    const bf16_t* base = static_cast<const bf16_t*>(op.ptr);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t k = kb + i;
      if (mn < op.rows && k < op.K)
        r[i] = *reinterpret_cast<const u32x4*>(base + k * op.ld + mn);
      else
        r[i] = u32x4{0u, 0u, 0u, 0u};
    }
  }
  __device__ __forceinline__ void store(char* lds, int tid) const {
    const int row0 = (tid & 31) * 8;
    const int c = tid >> 5;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      // out[q] packs (k = 2q, k = 2q+1) of column j: low halves for even j,
      // high halves for odd j.
      const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
      u32x4 out;
      out[0] = __builtin_amdgcn_perm(r[1][j >> 1], r[0][j >> 1], sel);
      out[1] = __builtin_amdgcn_perm(r[3][j >> 1], r[2][j >> 1], sel);
      out[2] = __builtin_amdgcn_perm(r[5][j >> 1], r[4][j >> 1], sel);
      out[3] = __builtin_amdgcn_perm(r[7][j >> 1], r[6][j >> 1], sel);
      *reinterpret_cast<u32x4*>(lds + lds_off(row0 + j, c)) = out;
    }
  }
};

// M/N-contiguous fp32: two 4(k) x 4(mn) blocks per thread, transposed by
// register moves.
template <> struct StageCopy<float, false> {
  u32x4 r[8];
  __device__ __forceinline__ void load(const Operand& op, int64_t r0, int64_t k0, int tid) {
    const float* base = static_cast<const float*>(op.ptr);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int b = tid + 256 * h;
      const int64_t mn = r0 + (b & 63) * 4;
      const int64_t kb = k0 + (b >> 6) * 4;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t k = kb + i;
        if (mn < op.rows && k < op.K)
          r[4 * h + i] = *reinterpret_cast<const u32x4*>(base + k * op.ld + mn);
        else
          r[4 * h + i] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  }
  __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int b = tid + 256 * h;
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
// One 128-byte K stage of MFMA work for this wave's 128 x 128 sub-tile.
// Lane l supplies row (l & 31) of each 32-row block and K-chunk (l >> 5) of
// each 32-byte K slice; A and B use the same lane -> k assignment.
// ---------------------------------------------------------------------------
template <typename T> struct Mfma;

template <> struct Mfma<bf16_t> {
  __device__ __forceinline__ static void step(f32x16 (&acc)[4][4], const u32x4 (&a)[4],
                                              const u32x4 (&b)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8, a[i]), __builtin_bit_cast(bf16x8, b[j]), acc[i][j], 0, 0, 0);
  }
};

// fp32: each 16-byte chunk holds 4 K values, consumed by 4 MFMAs of K = 2.
// (The chunks are bit-cast to float vectors as a whole: bit-casting a single
// element of an integer vector compiles to element 0 with this toolchain.)
template <> struct Mfma<float> {
  __device__ __forceinline__ static void step(f32x16 (&acc)[4][4], const u32x4 (&a)[4],
                                              const u32x4 (&b)[4]) {
    f32x4 af[4], bf[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      af[i] = __builtin_bit_cast(f32x4, a[i]);
      bf[i] = __builtin_bit_cast(f32x4, b[i]);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i][e], bf[j][e], acc[i][j], 0, 0, 0);
  }
};

template <typename T>
__device__ __forceinline__ void mfma_stage(f32x16 (&acc)[4][4], const char* ldsA,
                                           const char* ldsB, int wm, int wn, int lane) {
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    u32x4 a[4], b[4];
    const int c = 2 * kk + (lane >> 5);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      a[i] = *reinterpret_cast<const u32x4*>(ldsA + lds_off(wm * 128 + i * 32 + (lane & 31), c));
#pragma unroll
    for (int j = 0; j < 4; ++j)
      b[j] = *reinterpret_cast<const u32x4*>(ldsB + lds_off(wn * 128 + j * 32 + (lane & 31), c));
    Mfma<T>::step(acc, a, b);
  }
}

// Full K loop for the tile at (m0, n0).  `lds` holds kLdsGemm bytes.
template <typename T, bool AK, bool BK>
__device__ __forceinline__ void gemm_mainloop(const Operand& A, const Operand& B, int64_t m0,
                                              int64_t n0, int64_t K, char* lds,
                                              f32x16 (&acc)[4][4]) {
  constexpr int KT = kRowBytes / sizeof(T);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int64_t nk = (K + KT - 1) / KT;

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  StageCopy<T, AK> ca;
  StageCopy<T, BK> cb;
  ca.load(A, m0, 0, tid);
  cb.load(B, n0, 0, tid);
  ca.store(lds, tid);
  cb.store(lds + kStageBytes, tid);
  if (nk > 1) {
    ca.load(A, m0, KT, tid);
    cb.load(B, n0, KT, tid);
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
      ca.load(A, m0, (kt + 2) * KT, tid);
      cb.load(B, n0, (kt + 2) * KT, tid);
    }
    __syncthreads();
  }
}

// Row / column of accumulator element e of block (i, j) held by this lane.
__device__ __forceinline__ int acc_row(int wm, int i, int e, int lane) {
  return wm * 128 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
}
__device__ __forceinline__ int acc_col(int wn, int j, int lane) {
  return wn * 128 + j * 32 + (lane & 31);
}

// Generic tiled contraction kernel: Epi provides prologue(m0, n0, extra) to
// stage per-row data into `extra` LDS before the loop and
// epilogue(acc, tm, tn, m0, n0, lds, extra) after it.
template <typename T, bool AK, bool BK, class Epi>
__global__ __launch_bounds__(kThreads, 1) void gemm_kernel(Operand A, Operand B, int64_t K,
                                                           int nTm, int nTn, Epi epi) {
  __shared__ __attribute__((aligned(16))) char lds[kLdsGemm + Epi::kLdsExtra];
  int tm, tn;
  tile_of(blockIdx.x, nTm, nTn, tm, tn);
  const int64_t m0 = int64_t(tm) * kBM, n0 = int64_t(tn) * kBN;
  char* extra = lds + kLdsGemm;
  epi.prologue(m0, n0, extra);
  f32x16 acc[4][4];
  gemm_mainloop<T, AK, BK>(A, B, m0, n0, K, lds, acc);
  epi.epilogue(acc, tm, tn, m0, n0, lds, extra);
}

}  // namespace mc
