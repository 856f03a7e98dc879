// Device building blocks for the packed chunkwise linear-attention kernels
// (gfx950 / CDNA4, wave64).
//
// Operand staging.  Every chunk tile lives in LDS exactly as it is stored in
// HBM: token-major [64][d] (or [64][64] for the masked score tiles), written
// with 16-byte vector stores.  MFMA operands whose contraction index is the
// token index are read "k-major" with the gfx950 LDS transpose read
// (ds_read_b64_tr_b16): within each group of 16 lanes, lane i, slot j
// receives element i % 4 of the 4-element read issued by lane 4j + i / 4, so
// lane L of group g reading &X[4g + L/4][4*(L%4)] obtains X[4g + e][L],
// e = 0..3 -- the 16x16x16 operand layout; two such reads form the 16x16x32
// one.  The float32 path reads single elements and needs no transpose.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "plan.hpp"

namespace harts {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int CB = 64;  // execution chunk (rows); equals the wave size

// Row kinds inside a packed chunk (ordered: pad < replay < own).
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

// Launch shape and LDS strides for element type T and head dimension D.
template <typename T, int D>
struct Cfg {
  static constexpr int NW = D == 128 ? 8 : 4;          // waves per workgroup
  static constexpr int NTHR = 64 * NW;
  static constexpr int VE = 16 / sizeof(T);            // elements per 16-byte vector
  static constexpr int VPR = D / VE;                   // vectors per row
  static constexpr int NV = CB * VPR / NTHR;           // vectors per thread per tile
  static constexpr int NT = D / 16;                    // 16-wide tiles along d
  static constexpr int LDR = D + Elem<T>::PAD;         // [64][D] tiles
  static constexpr int LDA = CB + Elem<T>::PAD;        // [64][64] tiles
  static constexpr int ATPW = 16 / NW;                 // score tiles per wave
  static_assert(NT == NW, "one 16-column state tile per wave");
};

// 16x16 MFMA tile products.  C[m][n] += sum_k A[m][k] B[k][n] with each
// operand either k-contiguous ("kc": A stored [m][k], B stored [n][k]) or
// k-major ("km": A stored [k][m], B stored [k][n]).  Pointers address the
// tile origin (row m0 / n0 for kc, column m0 / n0 for km) at k = 0.
template <typename T> struct Frag;
template <> struct Frag<bf16> {
  static constexpr int KSTEP = 32;
  typedef bf16x8 V;
  __device__ static inline V kc(const bf16* p, int ld, int lane) {
    return *reinterpret_cast<const bf16x8*>(p + (lane & 15) * ld + (lane >> 4) * 8);
  }
  __device__ static inline V km(const bf16* p, int ld, int lane) {
    const bf16* base = p + ((lane >> 4) * 8 + ((lane & 15) >> 2)) * ld + 4 * (lane & 3);
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + 4 * ld));
    V r;
    const bf16x4 a = __builtin_bit_cast(bf16x4, lo), b = __builtin_bit_cast(bf16x4, hi);
    r[0] = a[0]; r[1] = a[1]; r[2] = a[2]; r[3] = a[3];
    r[4] = b[0]; r[5] = b[1]; r[6] = b[2]; r[7] = b[3];
    return r;
  }
  __device__ static inline void mma(f32x4& c, const V& a, const V& b) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Frag<float> {
  static constexpr int KSTEP = 4;
  typedef float V;
  __device__ static inline V kc(const float* p, int ld, int lane) {
    return p[(lane & 15) * ld + (lane >> 4)];
  }
  __device__ static inline V km(const float* p, int ld, int lane) {
    return p[(lane >> 4) * ld + (lane & 15)];
  }
  __device__ static inline void mma(f32x4& c, const V& a, const V& b) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

template <typename T, bool A_KM, bool B_KM>
__device__ inline void tile(f32x4& c, const T* A, int lda, const T* B, int ldb, int K, int lane) {
  using F = Frag<T>;
#pragma unroll
  for (int k = 0; k < K; k += F::KSTEP) {
    const typename F::V a = A_KM ? F::km(A + k * lda, lda, lane) : F::kc(A + k, lda, lane);
    const typename F::V b = B_KM ? F::km(B + k * ldb, ldb, lane) : F::kc(B + k, ldb, lane);
    F::mma(c, a, b);
  }
}

// acc += A[16 x 16] * B where A is k-contiguous in LDS (A points at the tile
// origin, row stride lda) and B is a 16x16 float32 accumulator tile held in
// registers (C layout: lane l, element r holds B[4*(l/16) + r][l % 16]).
// The C layout is exactly the B-operand layout of the 16x16x16 bf16
// instruction; the float32 path issues four 16x16x4 instructions over the k
// indices {4g + j}, g = lane / 16.
template <typename T> struct MmaRegB;
template <> struct MmaRegB<bf16> {
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

// Accumulator element r of lane l in a 16x16 tile sits at row 4*(l/16) + r,
// column l % 16.
__device__ inline int acc_row(int lane, int r) { return 4 * (lane >> 4) + r; }
__device__ inline int acc_col(int lane) { return lane & 15; }

// Packed position p of a sequence -> (global row, kind, replay index).
struct RowRef {
  int row, kind, rep;
};
__device__ inline RowRef pos_row(const int32_t* seq, int p, const int32_t* replay_row) {
  const int n_rep = seq[SEQ_N_REPLAY];
  if (p < n_rep) {
    const int j = seq[SEQ_REPLAY_OFF] + p;
    return RowRef{replay_row[j], ROW_REPLAY, j};
  }
  if (p < seq[SEQ_N_TOK]) return RowRef{seq[SEQ_OWN_ROW] + (p - n_rep), ROW_OWN, -1};
  return RowRef{0, ROW_PAD, -1};
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
