// Device building blocks for the packed chunkwise linear-attention kernels
// (gfx950 / CDNA4, wave64).
//
// Operand staging.  Every chunk tile lives in LDS exactly as it is stored in
// HBM: token-major [64][d] (or [64][64] for the masked score tiles), written
// with 16-byte vector stores.  MFMA operands whose contraction index is the
// token index are read "k-major" with the gfx950 LDS transpose read
// (ds_read_b64_tr_b16): within each group of 16 lanes, lane i, slot j
// receives element i % 4 of the 4-element read issued by lane 4j + i / 4, so
// lane L of group g reading &X[R + L/4][C + 4*(L%4)] obtains X[R + e][C + L],
// e = 0..3; with R = 4g this is the 16x16x16 operand layout.  The float32
// path reads single elements and needs no transpose.
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
  __device__ static inline float to_f(float x) { return x; }
  __device__ static inline float from_f(float x) { return x; }
};
template <> struct Elem<bf16> {
  __device__ static inline float to_f(bf16 x) { return static_cast<float>(x); }
  __device__ static inline bf16 from_f(float x) { return static_cast<bf16>(x); }  // RNE
};

// Four consecutive elements as one float32x4 (one 8-byte bf16 or 16-byte
// float access; the address must be aligned to that size).
template <typename T> struct Vec4;
template <> struct Vec4<float> {
  __device__ static inline f32x4 load(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
  __device__ static inline void store(float* p, const f32x4& v) { *reinterpret_cast<f32x4*>(p) = v; }
};
template <> struct Vec4<bf16> {
  __device__ static inline f32x4 load(const bf16* p) {
    const bf16x4 b = *reinterpret_cast<const bf16x4*>(p);
    return f32x4{static_cast<float>(b[0]), static_cast<float>(b[1]), static_cast<float>(b[2]),
                 static_cast<float>(b[3])};
  }
  __device__ static inline void store(bf16* p, const f32x4& v) {
    bf16x4 b;
#pragma unroll
    for (int e = 0; e < 4; ++e) b[e] = static_cast<bf16>(v[e]);
    *reinterpret_cast<bf16x4*>(p) = b;
  }
};

// Four consecutive elements read in their storage type, widened later (so
// that the read can be issued well before the value is needed).
template <typename T> struct Vec4Raw;
template <> struct Vec4Raw<float> {
  typedef f32x4 V;
  __device__ static inline V load(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
  __device__ static inline f32x4 widen(const V& v) { return v; }
};
template <> struct Vec4Raw<bf16> {
  typedef bf16x4 V;
  __device__ static inline V load(const bf16* p) { return *reinterpret_cast<const bf16x4*>(p); }
  __device__ static inline f32x4 widen(const V& b) {
    return f32x4{static_cast<float>(b[0]), static_cast<float>(b[1]), static_cast<float>(b[2]),
                 static_cast<float>(b[3])};
  }
};

// Stores through a buffer resource (raw, byte offsets): a lane whose offset
// lies at or past the resource's size stores nothing, so a store can be
// issued by every lane instead of inside a branch.
constexpr uint32_t BUF_DROP = 0x80000000u;  // an offset past any resource here
__device__ inline __amdgpu_buffer_rsrc_t buffer_rsrc(void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, static_cast<short>(0), static_cast<int>(bytes), 0x00020000);
}
template <typename T> struct BufVec4;
template <> struct BufVec4<bf16> {
  __device__ static inline void store(__amdgpu_buffer_rsrc_t r, uint32_t off, const f32x4& v) {
    bf16x4 b;
#pragma unroll
    for (int e = 0; e < 4; ++e) b[e] = static_cast<bf16>(v[e]);
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, b), r, static_cast<int>(off), 0, 0);
  }
};
template <> struct BufVec4<float> {
  __device__ static inline void store(__amdgpu_buffer_rsrc_t r, uint32_t off, const f32x4& v) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, static_cast<int>(off), 0, 0);
  }
};

// LDS tile layout: 64 rows of COLS elements, row-major, each row padded by
// 16 bytes.  Addresses are affine in (r, c), so every fragment read is a
// per-lane base plus an immediate offset.  With the padding, 16-byte row
// writes, 2-byte accumulator-layout writes and the k-contiguous 8-byte
// fragment reads below are free of bank conflicts; the transpose reads take
// twice their minimum time (measured on gfx950, whose LDS serves 256 bytes a
// clock to reads).
//
// XS (bf16 rows of 128 elements only): rows padded by 32 bytes, and in rows
// 8..15 of every 16-row group the 8-byte units swap in pairs of pairs
// (element bit 3 flipped).  Then both the k-contiguous fragment reads and
// the transpose reads are conflict-free: a half-wave's 32 lanes hit 32
// distinct bank pairs (the plain 32-byte pad serves the transpose reads but
// doubles the fragment reads).  16-byte units stay contiguous.  Fragment
// reads with origins (r0, c0) that are multiples of 16 address
// base(r0, c0) + lane(ri, ci): an affine part plus a lane constant.
template <typename T, int COLS, bool XS = false, int PADB = (XS ? 32 : 16)>
struct Tile {
  static_assert(!XS || (sizeof(T) == 2 && COLS == 128), "swizzled rows are bf16 x 128");
  static constexpr int LD = COLS + PADB / static_cast<int>(sizeof(T));  // row stride (elements)
  static constexpr int SIZE = CB * LD;
  __device__ static inline int swz(int r) { return XS ? ((r >> 3) & 1) << 3 : 0; }
  __device__ static inline int at(int r, int c) { return r * LD + (c ^ swz(r)); }
  __device__ static inline int base(int r0, int c0) { return r0 * LD + c0; }
  __device__ static inline int lane(int ri, int ci) { return ri * LD + (ci ^ swz(ri)); }
};

// The swizzled layout where the element type and head dimension allow it,
// else the plain one.
template <typename T, int D>
using TileX = Tile<T, D, sizeof(T) == 2 && D == 128>;

// Launch shape for element type T and head dimension D.  Four waves per
// workgroup; wave w owns the state columns 16 CPW w .. 16 CPW (w + 1) - 1 (CPW
// 16-column strips) and all NT 16-row tiles of them.  Chunk kernels are built
// for two resident workgroups per CU (two waves per SIMD).
template <typename T, int D>
struct Cfg {
  static constexpr int NW = 4;                         // waves per workgroup
  static constexpr int NTHR = 64 * NW;
  static constexpr int VE = 16 / sizeof(T);            // elements per 16-byte vector
  static constexpr int VPR = D / VE;                   // vectors per row
  static constexpr int NV = CB * VPR / NTHR;           // vectors per thread per tile
  static constexpr int NT = D / 16;                    // 16-row tiles of a state
  static constexpr int CPW = D / 16 / NW;              // 16-column strips per wave
  static constexpr int WPE = 2;                        // waves per SIMD
  using TD = Tile<T, D>;                               // [64][D] tiles
  using TX = TileX<T, D>;                              // [64][D] tiles read transposed
  using TA = Tile<T, CB>;                              // [64][64] tiles
  static_assert(CPW >= 1 && NT == NW * CPW, "state split into column strips");
};

// 16x16 MFMA tile products.  C[m][n] += sum_k A[m][k] B[k][n] with each
// operand either k-contiguous ("kc": A stored as rows m, B stored as rows n)
// or k-major ("km": A stored as rows k with m along the row, B as rows k with
// n along the row).  An operand is (tile base, tile layout, origin): for kc
// the origin is (row m0 or n0, column k = 0); for km it is (row k = 0,
// column m0 or n0).
template <typename T> struct Frag;
// bf16: one 16x16x32 instruction per 32-deep k step.  Lane (g, i), g = lane /
// 16, holds k in {4g..4g+3} u {16+4g..16+4g+3} for both operands (the same
// permutation of k on both sides leaves the product unchanged), so every
// fragment is two non-adjacent 8-byte LDS reads.
template <> struct Frag<bf16> {
  static constexpr int KSTEP = 32;
  typedef bf16x8 V;
  __device__ static inline V join(const bf16x4& a, const bf16x4& b) {
    V v;
    v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
    v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
    return v;
  }
  // (r0, c0 multiples of 16: the lane parts stay inside one 16 x 16 block)
  // The two halves are read as separate 8-byte LDS loads: merged into one
  // two-address load (ds_read2_b64), this lane pattern takes 16 clocks
  // instead of 2 x 2 on gfx950 (measured), so the loads are marked volatile,
  // which keeps the compiler from pairing them.
  template <typename L>
  __device__ static inline V kc(const bf16* t, int r0, int c0, int lane) {
    typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
    const bf16* p = t + L::base(r0, c0) + L::lane(lane & 15, (lane >> 4) * 4);
    const bf16x4 lo = *(volatile lds_bf16x4*)p;
    const bf16x4 hi = *(volatile lds_bf16x4*)(p + 16);
    return join(lo, hi);
  }
  template <typename L>
  __device__ static inline V km(const bf16* t, int r0, int c0, int lane) {
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    const bf16* p = t + L::base(r0, c0) + L::lane((lane >> 4) * 4 + ((lane & 15) >> 2), 4 * (lane & 3));
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 16 * L::LD));
    return join(__builtin_bit_cast(bf16x4, lo), __builtin_bit_cast(bf16x4, hi));
  }
  // km fragment with row k of the tile (the contraction index) scaled by
  // s[k]: slot e holds k = r0 + 4g + e, slot 4 + e holds k = r0 + 16 + 4g + e.
  template <typename L>
  __device__ static inline V km_scaled(const bf16* t, int r0, int c0, const float* s, int lane) {
    const V x = km<L>(t, r0, c0, lane);
    const int k4 = r0 + (lane >> 4) * 4;
    const f32x4 lo = *reinterpret_cast<const f32x4*>(s + k4);
    const f32x4 hi = *reinterpret_cast<const f32x4*>(s + k4 + 16);
    V y;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      y[e] = static_cast<bf16>(static_cast<float>(x[e]) * lo[e]);
      y[4 + e] = static_cast<bf16>(static_cast<float>(x[4 + e]) * hi[e]);
    }
    return y;
  }
  __device__ static inline void mma(f32x4& c, const V& a, const V& b) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Frag<float> {
  static constexpr int KSTEP = 4;
  typedef float V;
  template <typename L>
  __device__ static inline V kc(const float* t, int r0, int c0, int lane) {
    return t[L::at(r0 + (lane & 15), c0 + (lane >> 4))];
  }
  template <typename L>
  __device__ static inline V km(const float* t, int r0, int c0, int lane) {
    return t[L::at(r0 + (lane >> 4), c0 + (lane & 15))];
  }
  template <typename L>
  __device__ static inline V km_scaled(const float* t, int r0, int c0, const float* s, int lane) {
    return km<L>(t, r0, c0, lane) * s[r0 + (lane >> 4)];
  }
  __device__ static inline void mma(f32x4& c, const V& a, const V& b) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

// c[j] += A * B_j for the NJ output tiles of one row block (origins bn + 16 j),
// the A fragment shared; B is k-major.  k runs over [k0, K).
// With SWAP the operands of each product trade places, which leaves the
// transposed tile (B_j^T A^T) in c[j]: lane (g, i) then holds row i, columns
// 4g..4g+3 of A B_j.  With EAGER all fragments of a step are requested before
// its first product (more registers live, no wait per product).
template <typename T, typename LA, bool A_KM, typename LB, int NJ, bool SWAP = false, bool EAGER = false>
__device__ inline void tile_cols(f32x4* c, const T* A, int am, const T* B, int bn, int k0, int K,
                                 int lane) {
  using F = Frag<T>;
#pragma unroll 1
  for (int k = k0; k < K; k += F::KSTEP) {
    const typename F::V a = A_KM ? F::template km<LA>(A, k, am, lane) : F::template kc<LA>(A, am, k, lane);
    if constexpr (EAGER) {
      typename F::V b[NJ];
#pragma unroll
      for (int j = 0; j < NJ; ++j) b[j] = F::template km<LB>(B, k, bn + 16 * j, lane);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        if (SWAP) F::mma(c[j], b[j], a);
        else F::mma(c[j], a, b[j]);
      }
    } else {
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const typename F::V b = F::template km<LB>(B, k, bn + 16 * j, lane);
        if (SWAP) F::mma(c[j], b, a);
        else F::mma(c[j], a, b);
      }
    }
  }
}

// S[j NT + i] += A_i * diag(s) * B_j for the state tiles of a wave: A_i is
// k-major with origin column 16 i, B_j k-major with origin column bn + 16 j
// and its row k scaled by s[k]; each fragment is loaded once per k step.
template <typename T, typename LA, typename LB, int NT, int CPW, bool EAGER = false>
__device__ inline void state_update(f32x4* S, const T* A, const T* B, int bn, const float* s, int lane) {
  using F = Frag<T>;
#pragma unroll 1
  for (int k = 0; k < CB; k += F::KSTEP) {
    typename F::V b[CPW];
    if constexpr (EAGER) {
      // all fragments of the step are requested before its first product
      typename F::V a[NT];
#pragma unroll
      for (int i = 0; i < NT; ++i) a[i] = F::template km<LA>(A, k, i * 16, lane);
#pragma unroll
      for (int j = 0; j < CPW; ++j) b[j] = F::template km_scaled<LB>(B, k, bn + 16 * j, s, lane);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < NT; ++i)
#pragma unroll
        for (int j = 0; j < CPW; ++j) F::mma(S[j * NT + i], a[i], b[j]);
    } else {
#pragma unroll
      for (int j = 0; j < CPW; ++j) b[j] = F::template km_scaled<LB>(B, k, bn + 16 * j, s, lane);
#pragma unroll
      for (int i = 0; i < NT; ++i) {
        const typename F::V a = F::template km<LA>(A, k, i * 16, lane);
#pragma unroll
        for (int j = 0; j < CPW; ++j) F::mma(S[j * NT + i], a, b[j]);
      }
    }
  }
}

// acc[j] += A * B_j where A is k-contiguous in LDS (rows m0.., columns k of a
// tile with layout L) and B_j is the wave's state strip j held in registers
// in the accumulator layout (lane l, element r of state tile kt holds
// B[16 kt + 4 (l / 16) + r][l % 16]), pre-converted by RegB<T>::pack.  For
// bf16 two state tiles kt, kt + 1 form the B operand of one 16x16x32
// instruction: lane group g then holds k = 16 kt + {4g..4g+3} and
// 16 (kt + 1) + {4g..4g+3}, which is exactly the k set of the k-contiguous A
// fragment read at column 16 kt.  The float32 path issues four 16x16x4
// instructions per state tile over k = 16 kt + 4g + e.
template <typename T> struct RegB;
template <> struct RegB<bf16> {
  static constexpr int KT = 2;  // state tiles per B operand
  typedef bf16x8 P;
  typedef bf16x8 A;
  __device__ static inline P pack(const f32x4* B) {
    P b;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      b[r] = static_cast<bf16>(B[0][r]);
      b[4 + r] = static_cast<bf16>(B[1][r]);
    }
    return b;
  }
  template <typename L>
  __device__ static inline A load(const bf16* t, int m0, int k0, int lane) {
    return Frag<bf16>::kc<L>(t, m0, k0, lane);
  }
  __device__ static inline void mma(f32x4& c, const A& a, const P& b) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct RegB<float> {
  static constexpr int KT = 1;
  typedef f32x4 P;
  typedef f32x4 A;
  __device__ static inline P pack(const f32x4* B) { return B[0]; }
  template <typename L>
  __device__ static inline A load(const float* t, int m0, int k0, int lane) {
    const int r = m0 + (lane & 15), c4 = k0 + (lane >> 4) * 4;
    return f32x4{t[L::at(r, c4)], t[L::at(r, c4 + 1)], t[L::at(r, c4 + 2)], t[L::at(r, c4 + 3)]};
  }
  __device__ static inline void mma(f32x4& c, const A& a, const P& b) {
#pragma unroll
    for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b[e], c, 0, 0, 0);
  }
};

// acc[j] += A[m0.., :] * B_j over the whole state dimension, B_j being the
// wave's float32 state strip j (tiles S[j NT + kt]), converted per use.
// With SWAP the products leave the transposed tiles in acc, EAGER as in
// tile_cols.
template <typename T, typename L, int NT, int CPW, bool SWAP = false, bool EAGER = false>
__device__ inline void regb_rows(f32x4* acc, const T* A, int m0, const f32x4* S, int lane) {
  using R = RegB<T>;
  if constexpr (EAGER) {
    typename R::A a[NT / R::KT];
#pragma unroll
    for (int kt = 0; kt < NT; kt += R::KT) a[kt / R::KT] = R::template load<L>(A, m0, kt * 16, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kt = 0; kt < NT; kt += R::KT)
#pragma unroll
      for (int j = 0; j < CPW; ++j) {
        if (SWAP) R::mma(acc[j], R::pack(S + j * NT + kt), a[kt / R::KT]);
        else R::mma(acc[j], a[kt / R::KT], R::pack(S + j * NT + kt));
      }
  } else {
#pragma unroll
    for (int kt = 0; kt < NT; kt += R::KT) {
      const typename R::A a = R::template load<L>(A, m0, kt * 16, lane);
#pragma unroll
      for (int j = 0; j < CPW; ++j) {
        if (SWAP) R::mma(acc[j], R::pack(S + j * NT + kt), a);
        else R::mma(acc[j], a, R::pack(S + j * NT + kt));
      }
    }
  }
}

// A wave's state strips converted once to B operands (for bf16 two state
// tiles per operand), for several regb_rows_packed calls on an unchanged
// state.  The converted values are hidden from the optimiser, so that the
// conversion is not repeated at each use.
template <typename T, int NT, int CPW>
struct PackedState {
  typename RegB<T>::P p[CPW][NT / RegB<T>::KT];
  __device__ inline void pack(const f32x4* S) {
    using R = RegB<T>;
#pragma unroll
    for (int j = 0; j < CPW; ++j)
#pragma unroll
      for (int kt = 0; kt < NT; kt += R::KT) {
        p[j][kt / R::KT] = R::pack(S + j * NT + kt);
        asm volatile("" : "+v"(p[j][kt / R::KT]));
      }
  }
};

// regb_rows on a packed state (SWAP, EAGER as there).
template <typename T, typename L, int NT, int CPW, bool SWAP = false, bool EAGER = false>
__device__ inline void regb_rows_packed(f32x4* acc, const T* A, int m0, const PackedState<T, NT, CPW>& ps,
                                        int lane) {
  using R = RegB<T>;
  typename R::A a[NT / R::KT];
#pragma unroll
  for (int kt = 0; kt < NT; kt += R::KT) a[kt / R::KT] = R::template load<L>(A, m0, kt * 16, lane);
  if (EAGER) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int kt = 0; kt < NT; kt += R::KT)
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      if (SWAP) R::mma(acc[j], ps.p[j][kt / R::KT], a[kt / R::KT]);
      else R::mma(acc[j], a[kt / R::KT], ps.p[j][kt / R::KT]);
    }
}

// Hides the values of a state from the optimiser (no instructions): values
// derived from it inside a loop stay inside the loop.
template <int N>
__device__ inline void opaque_state(f32x4* S) {
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(S[i]));
}

// Four consecutive floats of a per-row vector at rows r0 + 4g .. + 3 (lane group g).
__device__ inline f32x4 row_vec(const float* v, int r0, int lane) {
  return *reinterpret_cast<const f32x4*>(v + r0 + (lane >> 4) * 4);
}

// Accumulator element r of lane l in a 16x16 tile sits at row 4*(l/16) + r,
// column l % 16.
__device__ inline int acc_row(int lane, int r) { return 4 * (lane >> 4) + r; }
__device__ inline int acc_col(int lane) { return lane & 15; }

// The sequence-table fields the chunk kernels use, read once per workgroup
// (uniform, kept in scalar registers).
struct SeqInfo {
  int n_rep;       // replay rows (< chunk)
  int n_tok;       // replay + own rows
  int replay_off;  // global replay index of the first replay row
  int own_row;     // physical row of the first own row
  int chunk_off;   // first chunk of the sequence within the round
};
__device__ inline SeqInfo seq_info(const int32_t* seq) {
  return SeqInfo{seq[SEQ_N_REPLAY], seq[SEQ_N_TOK], seq[SEQ_REPLAY_OFF], seq[SEQ_OWN_ROW],
                 seq[SEQ_CHUNK_OFF]};
}

// A block kernel workgroup's unit of work: one entry of the round's launch
// table (uniform, kept in scalar registers).
struct BlkInfo {
  int b;           // block id
  int li;          // sequence (local index within the round)
  int c0, nc;      // first chunk of the block (within the sequence), chunks
  int idx, n_blk;  // block index within the sequence, blocks of the sequence
  int final_leaf;  // leaf index receiving the sequence's final state
  int init_bank;   // bank entry of the sequence's initial state, or -1
  SeqInfo sq;
};
__device__ inline BlkInfo blk_info(const int32_t* launch, int j) {
  const int32_t* e = launch + j * LCH_WORDS;
  BlkInfo bl;
  bl.b = e[LCH_BLK];
  bl.li = e[LCH_SEQ];
  bl.c0 = e[LCH_C0];
  bl.nc = e[LCH_NC];
  bl.idx = e[LCH_IDX];
  bl.n_blk = e[LCH_N_BLK];
  bl.final_leaf = e[LCH_FINAL_LEAF];
  bl.init_bank = e[LCH_INIT_BANK];
  bl.sq = SeqInfo{e[LCH_N_REPLAY], e[LCH_N_TOK], e[LCH_REPLAY_OFF], e[LCH_OWN_ROW], e[LCH_CHUNK_OFF]};
  return bl;
}

// Packed position p of a sequence -> (global row, kind, replay index).
struct RowRef {
  int row, kind, rep;
};
__device__ inline RowRef pos_row(const SeqInfo& sq, int p, const int32_t* replay_row) {
  if (p < sq.n_rep) {
    const int j = sq.replay_off + p;
    return RowRef{replay_row[j], ROW_REPLAY, j};
  }
  if (p < sq.n_tok) return RowRef{sq.own_row + (p - sq.n_rep), ROW_OWN, -1};
  return RowRef{0, ROW_PAD, -1};
}

// The wave index of thread t, as a value the compiler knows to be uniform
// over the wave (so that branches on it are scalar branches and values
// derived from it live in scalar registers).
__device__ inline int wave_id(int t) { return __builtin_amdgcn_readfirstlane(t >> 6); }

// Cross-lane steps on DPP (data-parallel primitives: a VALU operand modifier
// moving data between lanes of a 16-lane row), so that no step goes through
// the LDS queue.  Lanes without a source read 0.
template <int CTRL>
__device__ inline float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL,
                                                               0xF, 0xF, true));
}
constexpr int DPP_ROW_SHL = 0x100;       // + n: lane i reads lane i + n of its row
constexpr int DPP_ROW_SHR = 0x110;       // + n: lane i reads lane i - n of its row


// Inclusive prefix sum over the 64 lanes of a wave (lane order).
__device__ inline float wave_prefix_sum(float x, int lane) {
  x += dpp<DPP_ROW_SHR + 1>(x);
  x += dpp<DPP_ROW_SHR + 2>(x);
  x += dpp<DPP_ROW_SHR + 4>(x);
  x += dpp<DPP_ROW_SHR + 8>(x);
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 15));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 31));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 47));
  const int row = lane >> 4;
  return x + (row >= 1 ? r0 : 0.f) + (row >= 2 ? r1 : 0.f) + (row >= 3 ? r2 : 0.f);
}

// Inclusive suffix sum over the 64 lanes of a wave (lane order).
__device__ inline float wave_suffix_sum(float x, int lane) {
  x += dpp<DPP_ROW_SHL + 1>(x);
  x += dpp<DPP_ROW_SHL + 2>(x);
  x += dpp<DPP_ROW_SHL + 4>(x);
  x += dpp<DPP_ROW_SHL + 8>(x);
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 48));
  const int row = lane >> 4;
  return x + (row <= 0 ? r1 : 0.f) + (row <= 1 ? r2 : 0.f) + (row <= 2 ? r3 : 0.f);
}

// Value of lane l (uniform).
__device__ inline float lane_value(float x, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), l));
}

// Sum over the four 16-lane groups of a wave (lanes i, i + 16, i + 32,
// i + 48), returned to every lane.  v_permlane32_swap exchanges the upper
// half of its first operand with the lower half of its second; applied to two
// copies of x, the pair then holds x[l] and x[l ^ 32] in every lane (and
// likewise for v_permlane16_swap with rows of 16).  Both results of the swap
// are needed, hence inline asm with two tied operands; the nops keep the
// swap clear of any VALU read/write hazard.
__device__ inline float group_sum4(float x) {
  float a = x, b = x;
  asm volatile("s_nop 4\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 4" : "+v"(a), "+v"(b));
  const float y = a + b;
  float c = y, d = y;
  asm volatile("s_nop 4\n\tv_permlane16_swap_b32 %0, %1\n\ts_nop 4" : "+v"(c), "+v"(d));
  return c + d;
}

}  // namespace harts
