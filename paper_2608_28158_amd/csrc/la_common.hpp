// Device building blocks for the packed chunkwise linear-attention kernels
// (gfx950 / CDNA4, wave64): MFMA tile products on LDS operands, chunk row
// resolution (replay rows by index, own rows contiguous, zero padding) and
// the in-chunk prefix sum of the log-decay.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "plan.hpp"

namespace harts {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int CB = 64;        // execution chunk (rows); equals the wave size
constexpr int NTHREADS = 256;  // four waves per workgroup
constexpr int NWAVES = NTHREADS / 64;
constexpr int DVT = 32;        // state columns per workgroup in the scan kernels

// Row kinds inside a packed chunk.
enum : int { ROW_PAD = 0, ROW_REPLAY = 1, ROW_OWN = 2 };

template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int PAD = 4;  // 16 bytes of row padding in LDS
  __device__ static inline float to_f(float x) { return x; }
  __device__ static inline float from_f(float x) { return x; }
};
template <> struct Elem<bf16> {
  static constexpr int PAD = 8;
  __device__ static inline float to_f(bf16 x) { return static_cast<float>(x); }
  __device__ static inline bf16 from_f(float x) { return static_cast<bf16>(x); }  // RNE
};

// C[16x16] += sum_k A[m][k] * Bt[n][k] for one tile.  A and Bt point at the
// tile's first row in LDS (row-major, K contiguous); K is a multiple of the
// instruction depth.  Lane l supplies row (l % 16) of both operands.
template <typename T> struct Mma;
template <> struct Mma<bf16> {
  __device__ static inline void tile(f32x4& c, const bf16* A, int lda, const bf16* Bt, int ldb,
                                     int K, int lane) {
    const bf16* a = A + (lane & 15) * lda + (lane >> 4) * 8;
    const bf16* b = Bt + (lane & 15) * ldb + (lane >> 4) * 8;
#pragma unroll 4
    for (int k = 0; k < K; k += 32) {
      const bf16x8 av = *reinterpret_cast<const bf16x8*>(a + k);
      const bf16x8 bv = *reinterpret_cast<const bf16x8*>(b + k);
      c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, c, 0, 0, 0);
    }
  }
};
template <> struct Mma<float> {
  __device__ static inline void tile(f32x4& c, const float* A, int lda, const float* Bt, int ldb,
                                     int K, int lane) {
    const float* a = A + (lane & 15) * lda + (lane >> 4);
    const float* b = Bt + (lane & 15) * ldb + (lane >> 4);
#pragma unroll 8
    for (int k = 0; k < K; k += 4) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[k], b[k], c, 0, 0, 0);
  }
};

// acc += A[16 x 16] * B[16 x 16] where A is read from LDS (A points at the
// tile's first row and column, row stride lda) and B is a 16x16 float32
// accumulator tile held in registers (C layout: lane l, element r holds
// B[4*(l/16) + r][l % 16]).  The C layout of a tile is exactly the B-operand
// layout of the 16x16x16 bf16 instruction; the float32 path issues four
// 16x16x4 instructions over the k indices {4g + j}, g = lane / 16.
template <typename T> struct MmaRegB;
template <> struct MmaRegB<bf16> {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  __device__ static inline void step(f32x4& c, const bf16* A, int lda, const f32x4& B, int lane) {
    const bf16x4 a = *reinterpret_cast<const bf16x4*>(A + (lane & 15) * lda + (lane >> 4) * 4);
    bf16x4 b;
    b[0] = static_cast<bf16>(B[0]);
    b[1] = static_cast<bf16>(B[1]);
    b[2] = static_cast<bf16>(B[2]);
    b[3] = static_cast<bf16>(B[3]);
    c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
  }
};
template <> struct MmaRegB<float> {
  __device__ static inline void step(f32x4& c, const float* A, int lda, const f32x4& B, int lane) {
    const float* a = A + (lane & 15) * lda + (lane >> 4) * 4;
#pragma unroll
    for (int j = 0; j < 4; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], B[j], c, 0, 0, 0);
  }
};

// Accumulator element r of lane l in a 16x16 tile sits at
// row 4*(l/16) + r, column l % 16.
__device__ inline int acc_row(int lane, int r) { return 4 * (lane >> 4) + r; }
__device__ inline int acc_col(int lane) { return lane & 15; }

// Per-chunk row table: global row, kind and (for replay rows) replay index.
struct ChunkRows {
  int row[CB];
  int kind[CB];
  int rep[CB];
};

// Resolve the 64 packed positions of chunk c of a sequence (threads < 64).
__device__ inline void resolve_rows(ChunkRows& cr, const int32_t* seq, int c,
                                    const int32_t* replay_row, int t) {
  if (t < CB) {
    const int p = c * CB + t;
    const int n_rep = seq[SEQ_N_REPLAY];
    const int n_tok = seq[SEQ_N_TOK];
    if (p < n_rep) {
      const int j = seq[SEQ_REPLAY_OFF] + p;
      cr.row[t] = replay_row[j];
      cr.kind[t] = ROW_REPLAY;
      cr.rep[t] = j;
    } else if (p < n_tok) {
      cr.row[t] = seq[SEQ_OWN_ROW] + (p - n_rep);
      cr.kind[t] = ROW_OWN;
      cr.rep[t] = -1;
    } else {
      cr.row[t] = 0;
      cr.kind[t] = ROW_PAD;
      cr.rep[t] = -1;
    }
  }
}

// Inclusive prefix sum of g over the chunk (wave 0, one row per lane); pad
// rows contribute 0.  G[t] = g_0 + ... + g_t.
__device__ inline void chunk_cumsum(float* G, const ChunkRows& cr, const float* g, int H, int h,
                                    int t) {
  if (t < CB) {
    float x = cr.kind[t] != ROW_PAD ? g[static_cast<int64_t>(cr.row[t]) * H + h] : 0.f;
#pragma unroll
    for (int off = 1; off < CB; off <<= 1) {
      const float y = __shfl_up(x, off, CB);
      if (t >= off) x += y;
    }
    G[t] = x;
  }
}

// Sum over the 16 lanes that share the same accumulator rows.
__device__ inline float sum16(float x) {
  x += __shfl_xor(x, 1, 64);
  x += __shfl_xor(x, 2, 64);
  x += __shfl_xor(x, 4, 64);
  x += __shfl_xor(x, 8, 64);
  return x;
}

}  // namespace harts
