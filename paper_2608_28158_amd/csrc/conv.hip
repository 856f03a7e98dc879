// Causal depthwise convolution over compact rows with true-ancestor context
// (HARTS, Sec. 4.2, "KDA state reuse and causal convolution"), for gfx950.
//
// Along every trajectory, y_t[c] = sum_{i < w} W[c, i] x_{t-i}[c], zero
// before the trajectory's first token.  In the compact layout a row's i-th
// predecessor on its trajectory is unique (a row has one ancestor path): the
// row i above it inside its segment, else a row of an ancestor segment,
// never a row of an adjacent packed sequence.  harts_conv_context (host,
// semantic.cpp) writes that predecessor table once per plan, and the
// transposed table of consumers, which the backward walks to gather each
// row's gradient.
//   k_conv_fwd      one thread per (4 channels, run of 32 rows);
//   k_conv_bwd      runs of 64 rows: dx of each row (its own term plus
//                   every consumer's, in (tap, row) order) and the run's
//                   tap sums x[pred_i(r)] dy[r], in row order;
//   k_conv_dw_sum   per (channel, tap), the runs' partials in a fixed order.
// Arithmetic in float32; no atomics, so reruns are bitwise identical.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <new>
#include <string>
#include <vector>

#include "harts.h"
#include "plan.hpp"

namespace harts {
namespace {

typedef __bf16 bf16;
constexpr int CV_THR = 256;
constexpr int CV_MAXW = 8;
constexpr int CV_RUN = 32;     // rows per thread in the forward
constexpr int CV_RUN_B = 64;   // rows per thread in the backward (one partial dW per run)
constexpr int CV_SUCC = 2048;  // consumer entries of a backward run staged in LDS

template <typename T> struct CV;
template <> struct CV<bf16> {
  static constexpr int N = 4;  // 8-byte pieces: half the registers of 16-byte ones
  using Raw = uint2;           // a piece as loaded, widened where it is used
  __device__ static inline Raw raw(const bf16* p) { return *reinterpret_cast<const uint2*>(p); }
  __device__ static inline void cvt(const Raw u, float* x) {
    x[0] = __uint_as_float(u.x << 16);
    x[1] = __uint_as_float(u.x & 0xffff0000u);
    x[2] = __uint_as_float(u.y << 16);
    x[3] = __uint_as_float(u.y & 0xffff0000u);
  }
  __device__ static inline void load(const bf16* p, float* x) { cvt(raw(p), x); }
  __device__ static inline void store(bf16* p, const float* x) {
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    bf16x4 b;
#pragma unroll
    for (int i = 0; i < 4; ++i) b[i] = static_cast<bf16>(x[i]);
    *reinterpret_cast<bf16x4*>(p) = b;
  }
};
template <> struct CV<float> {
  static constexpr int N = 4;
  using Raw = float4;
  __device__ static inline Raw raw(const float* p) { return *reinterpret_cast<const float4*>(p); }
  __device__ static inline void cvt(const Raw u, float* x) {
    x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
  }
  __device__ static inline void load(const float* p, float* x) { cvt(raw(p), x); }
  __device__ static inline void store(float* p, const float* x) {
    *reinterpret_cast<float4*>(p) = float4{x[0], x[1], x[2], x[3]};
  }
};

// Threads own 4 channels each (consecutive threads,
// consecutive vectors of the same rows: coalesced) and walk a run of rows,
// with their W taps in registers.  Inside a segment a row's predecessors
// are the rows just before it, so the activations of the previous rows are
// kept in registers and reloaded only where the table points elsewhere
// (a segment's first rows, whose window reaches into an ancestor).
template <typename T, int W>
__device__ inline void load_taps(const float* __restrict__ Wt, int c0, float (&wt)[W][CV<T>::N]) {
#pragma unroll
  for (int e = 0; e < CV<T>::N; ++e) {
    const float4* src = reinterpret_cast<const float4*>(Wt + (c0 + e) * W);
    if constexpr (W % 4 == 0) {
#pragma unroll
      for (int q = 0; q < W / 4; ++q) {
        const float4 u = src[q];
        wt[4 * q][e] = u.x; wt[4 * q + 1][e] = u.y; wt[4 * q + 2][e] = u.z; wt[4 * q + 3][e] = u.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < W; ++i) wt[i][e] = Wt[(c0 + e) * W + i];
    }
  }
}

// v <- x[pred_i(r)] (tap i >= 1): from the registers of the previous rows
// when the predecessor is the row i above in this thread's run, else loaded
// (zero before the trajectory start or for an invalid entry).
// hist[j] = x[r - 1 - j].
template <typename T, int W>
__device__ inline void tap_value(const T* __restrict__ x, int64_t C, int Cch, int c0, int64_t r,
                                 int64_t run0, int i, int32_t p, const float (&hist)[W - 1][CV<T>::N],
                                 float (&v)[CV<T>::N]) {
  if (p == r - i && r - i >= run0) {
#pragma unroll
    for (int e = 0; e < CV<T>::N; ++e) v[e] = hist[i - 1][e];
  } else if (p >= 0 && p < C) {
    CV<T>::load(x + static_cast<int64_t>(p) * Cch + c0, v);
  } else {
#pragma unroll
    for (int e = 0; e < CV<T>::N; ++e) v[e] = 0.f;
  }
}

template <typename T, int W>
__device__ inline void shift_hist(float (&hist)[W - 1][CV<T>::N], const float (&cur)[CV<T>::N]) {
#pragma unroll
  for (int j = W - 2; j > 0; --j)
#pragma unroll
    for (int e = 0; e < CV<T>::N; ++e) hist[j][e] = hist[j - 1][e];
#pragma unroll
  for (int e = 0; e < CV<T>::N; ++e) hist[0][e] = cur[e];
}

template <typename T, int W>
__global__ __launch_bounds__(CV_THR) void k_conv_fwd(int64_t C, int Cch, const T* __restrict__ x,
                                                     const float* __restrict__ Wt,
                                                     const int32_t* __restrict__ pred, T* __restrict__ y) {
  using V = CV<T>;
  const int vec = blockIdx.x * CV_THR + threadIdx.x;
  const int c0 = vec * V::N;
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * CV_RUN;
  const int64_t r1 = r0 + CV_RUN < C ? r0 + CV_RUN : C;
  // the run's predecessor table, staged in LDS (one global round trip per
  // workgroup instead of one per row)
  __shared__ int32_t s_pred[CV_RUN * (W - 1)];
  for (int j = threadIdx.x; j < (r1 - r0) * (W - 1); j += CV_THR) s_pred[j] = pred[r0 * (W - 1) + j];
  __syncthreads();
  if (vec >= Cch / V::N) return;
  float wt[W][V::N], hist[W - 1][V::N];
  load_taps<T, W>(Wt, c0, wt);
  for (int64_t r = r0; r < r1; ++r) {
    float cur[V::N], v[V::N], acc[V::N];
    V::load(x + r * Cch + c0, cur);
#pragma unroll
    for (int e = 0; e < V::N; ++e) acc[e] = wt[0][e] * cur[e];
#pragma unroll
    for (int i = 1; i < W; ++i) {
      tap_value<T, W>(x, C, Cch, c0, r, r0, i, s_pred[(r - r0) * (W - 1) + i - 1], hist, v);
#pragma unroll
      for (int e = 0; e < V::N; ++e) acc[e] += wt[i][e] * v[e];
    }
    V::store(y + r * Cch + c0, acc);
    shift_hist<T, W>(hist, cur);
  }
}

// dx of a run of rows, and the run's partial weight gradient:
// part[run][c][i] = sum over the run's rows r of x[pred_i(r)][c] dy[r][c].
// Inside a segment the consumers of row r through tap i are the rows r + i,
// so dy of the next W - 1 rows rides along in registers (one new row
// loaded per step) and only consumers elsewhere (the first rows of child
// segments) are loaded through the table.
template <typename T, int W>
__global__ __launch_bounds__(CV_THR) void k_conv_bwd(int64_t C, int Cch, const T* __restrict__ x,
                                                     const float* __restrict__ Wt,
                                                     const int32_t* __restrict__ pred,
                                                     const int64_t* __restrict__ succ_off,
                                                     const int32_t* __restrict__ succ, int64_t n_succ,
                                                     const T* __restrict__ dy, T* __restrict__ dx,
                                                     float* __restrict__ part) {
  using V = CV<T>;
  const int vec = blockIdx.x * CV_THR + threadIdx.x;
  const int c0 = vec * V::N;
  const int64_t r0 = static_cast<int64_t>(blockIdx.y) * CV_RUN_B;
  const int64_t r1 = r0 + CV_RUN_B < C ? r0 + CV_RUN_B : C;
  // the run's tables, staged in LDS: predecessors, consumer offsets
  // (relative to the run's first entry) and up to CV_SUCC consumer entries;
  // entries beyond that (rows feeding very many children) are read from
  // global memory
  __shared__ int32_t s_pred[CV_RUN_B * (W - 1)];
  __shared__ int32_t s_off[CV_RUN_B + 1];
  __shared__ int32_t s_succ[CV_SUCC];
  const int64_t nr = r1 - r0;
  const int64_t b0 = succ_off[r0] < 0 ? 0 : (succ_off[r0] > n_succ ? n_succ : succ_off[r0]);
  for (int j = threadIdx.x; j < nr * (W - 1); j += CV_THR) s_pred[j] = pred[r0 * (W - 1) + j];
  for (int j = threadIdx.x; j <= nr; j += CV_THR) {
    int64_t o = succ_off[r0 + j];
    o = o < b0 ? b0 : (o > n_succ ? n_succ : o);
    s_off[j] = static_cast<int32_t>(o - b0 < INT32_MAX ? o - b0 : INT32_MAX);
  }
  __syncthreads();
  const int32_t n_run_succ = s_off[nr];
  for (int j = threadIdx.x; j < n_run_succ && j < CV_SUCC; j += CV_THR) s_succ[j] = succ[b0 + j];
  __syncthreads();
  if (vec >= Cch / V::N) return;
  float wt[W][V::N], hist[W - 1][V::N], gw[W][V::N];
  load_taps<T, W>(Wt, c0, wt);
#pragma unroll
  for (int i = 0; i < W; ++i)
#pragma unroll
    for (int e = 0; e < V::N; ++e) gw[i][e] = 0.f;
  // dr[i] = dy[r + i] as loaded, one row beyond the window, so that the
  // window's rows are widened at the top of a row while only the row beyond
  // it and the next row's x are in flight.  Every load is unconditional:
  // past the last row the last row is requested again, an entry never used
  // (the consumers of a row are rows of the table).
  using Raw = typename V::Raw;
  Raw dr[W + 1];
#pragma unroll
  for (int i = 0; i <= W; ++i) dr[i] = V::raw(dy + (r0 + i < C ? r0 + i : C - 1) * Cch + c0);
  Raw xr = V::raw(x + r0 * Cch + c0);   // x of the row, requested a row ahead
  for (int64_t r = r0; r < r1; ++r) {
    float cur[V::N], dwin[W][V::N], v[V::N], acc[V::N];
    V::cvt(xr, cur);
#pragma unroll
    for (int k = 0; k < W; ++k) V::cvt(dr[k], dwin[k]);
    xr = V::raw(x + (r + 1 < C ? r + 1 : C - 1) * Cch + c0);
#pragma unroll
    for (int e = 0; e < V::N; ++e) {
      acc[e] = wt[0][e] * dwin[0][e];
      gw[0][e] += cur[e] * dwin[0][e];
    }
#pragma unroll
    for (int i = 1; i < W; ++i) {
      tap_value<T, W>(x, C, Cch, c0, r, r0, i, s_pred[(r - r0) * (W - 1) + i - 1], hist, v);
#pragma unroll
      for (int e = 0; e < V::N; ++e) gw[i][e] += v[e] * dwin[0][e];
    }
    // consumers in table order: the staged entries from LDS, any beyond
    // them from global memory (two loops, so that neither read goes through
    // a flat address that would wait for every outstanding load)
    const auto consume = [&](int32_t code) __attribute__((always_inline)) {
      const int32_t sr = code >> 3, i = code & 7;  // consumer row, tap
      if (sr < 0 || sr >= C || i < 1 || i >= W) return;
      if (sr == r + i) {  // the row i below: already in registers
#pragma unroll
        for (int k = 1; k < W; ++k)
          if (k == i) {
#pragma unroll
            for (int e = 0; e < V::N; ++e) acc[e] += wt[k][e] * dwin[k][e];
          }
      } else {
        V::load(dy + static_cast<int64_t>(sr) * Cch + c0, v);
#pragma unroll
        for (int k = 1; k < W; ++k)
          if (k == i) {
#pragma unroll
            for (int e = 0; e < V::N; ++e) acc[e] += wt[k][e] * v[e];
          }
      }
    };
    const int32_t jb = s_off[r - r0], je = s_off[r - r0 + 1];
    const int32_t jl = je < CV_SUCC ? je : CV_SUCC;
    for (int32_t j = jb; j < jl; ++j) consume(s_succ[j]);
    for (int32_t j = jb > CV_SUCC ? jb : CV_SUCC; j < je; ++j) consume(succ[b0 + j]);
    V::store(dx + r * Cch + c0, acc);
    shift_hist<T, W>(hist, cur);
#pragma unroll
    for (int k = 0; k < W; ++k) dr[k] = dr[k + 1];
    dr[W] = V::raw(dy + (r + W + 1 < C ? r + W + 1 : C - 1) * Cch + c0);
  }
  // partials tap-major ([run][tap][channel]): every store is a coalesced
  // 16- or 32-byte piece of one tap's channel row
  float* out = part + static_cast<int64_t>(blockIdx.y) * Cch * W;
#pragma unroll
  for (int i = 0; i < W; ++i)
#pragma unroll
    for (int e = 0; e < V::N; e += 4)
      *reinterpret_cast<float4*>(out + static_cast<int64_t>(i) * Cch + c0 + e) =
          float4{gw[i][e], gw[i][e + 1], gw[i][e + 2], gw[i][e + 3]};
}

// dW[c][i] = sum over runs of part[run][i][c]: a workgroup takes 32
// consecutive (tap, channel) entries; its 8 groups of 32 threads sum every
// 8th run (group g takes runs g, g + 8, ...), and the 8 group sums are
// added in group order: a fixed association, independent of scheduling.
constexpr int DW_K = 32, DW_G = CV_THR / DW_K;
__global__ __launch_bounds__(CV_THR) void k_conv_dw_sum(int64_t n_run, int Cch, int W,
                                                        const float* __restrict__ part,
                                                        float* __restrict__ dW) {
  __shared__ float red[DW_G][DW_K];
  const int lk = threadIdx.x % DW_K, g = threadIdx.x / DW_K;
  const int64_t n = static_cast<int64_t>(Cch) * W;
  const int64_t k = static_cast<int64_t>(blockIdx.x) * DW_K + lk;  // i * Cch + c
  float acc = 0.f;
  if (k < n)
    for (int64_t b = g; b < n_run; b += DW_G) acc += part[b * n + k];
  red[g][lk] = acc;
  __syncthreads();
  if (g == 0 && k < n) {
    float sum = red[0][lk];
#pragma unroll
    for (int j = 1; j < DW_G; ++j) sum += red[j][lk];
    const int64_t i = k / Cch, c = k % Cch;
    dW[c * W + i] = sum;
  }
}

int conv_status(const char* where) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error(std::string(where) + ": " + hipGetErrorString(e));
    return HARTS_EHIP;
  }
  return HARTS_OK;
}

int check_conv(int32_t dtype, int64_t C, int32_t Cch, int32_t w, const char* where) {
  const std::string s(where);
  if (dtype != HARTS_F32 && dtype != HARTS_BF16) { set_error(s + ": unknown dtype"); return HARTS_EUNSUPPORTED; }
  if (w < 2 || w > CV_MAXW) { set_error(s + ": width must be in [2, 8]"); return HARTS_EUNSUPPORTED; }
  if (Cch < 8 || Cch % 8 || Cch > (1 << 20)) {
    set_error(s + ": channels must be a positive multiple of 8, at most 2^20");
    return HARTS_EUNSUPPORTED;
  }
  if (C < 0 || C >= (int64_t{1} << 28)) { set_error(s + ": need 0 <= C < 2^28 rows"); return HARTS_EUNSUPPORTED; }
  return HARTS_OK;
}

bool a16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

template <typename T>
int launch_fwd(int w, int64_t C, int Cch, const void* x, const float* Wt, const int32_t* pred, void* y,
               hipStream_t s) {
  const int nvec = Cch / CV<T>::N;
  const dim3 grid(static_cast<uint32_t>((nvec + CV_THR - 1) / CV_THR),
                  static_cast<uint32_t>((C + CV_RUN - 1) / CV_RUN));
  const T* xx = static_cast<const T*>(x);
  T* yy = static_cast<T*>(y);
  switch (w) {
#define HARTS_CONV_FWD(WW) \
  case WW: hipLaunchKernelGGL((k_conv_fwd<T, WW>), grid, dim3(CV_THR), 0, s, C, Cch, xx, Wt, pred, yy); break;
    HARTS_CONV_FWD(2) HARTS_CONV_FWD(3) HARTS_CONV_FWD(4) HARTS_CONV_FWD(5)
    HARTS_CONV_FWD(6) HARTS_CONV_FWD(7) HARTS_CONV_FWD(8)
#undef HARTS_CONV_FWD
  }
  return conv_status("k_conv_fwd");
}

template <typename T>
int launch_bwd(int w, int64_t C, int Cch, const void* x, const float* Wt, const int32_t* pred,
               const int64_t* succ_off, const int32_t* succ, int64_t n_succ, const void* dy, void* dx,
               float* dW, float* part, hipStream_t s) {
  const int nvec = Cch / CV<T>::N;
  const int64_t n_run = (C + CV_RUN_B - 1) / CV_RUN_B;
  const dim3 grid(static_cast<uint32_t>((nvec + CV_THR - 1) / CV_THR), static_cast<uint32_t>(n_run));
  const T* xx = static_cast<const T*>(x);
  const T* gy = static_cast<const T*>(dy);
  T* gx = static_cast<T*>(dx);
  switch (w) {
#define HARTS_CONV_BWD(WW)                                                                            \
  case WW:                                                                                            \
    hipLaunchKernelGGL((k_conv_bwd<T, WW>), grid, dim3(CV_THR), 0, s, C, Cch, xx, Wt, pred, succ_off, \
                       succ, n_succ, gy, gx, part);                                                   \
    break;
    HARTS_CONV_BWD(2) HARTS_CONV_BWD(3) HARTS_CONV_BWD(4) HARTS_CONV_BWD(5)
    HARTS_CONV_BWD(6) HARTS_CONV_BWD(7) HARTS_CONV_BWD(8)
#undef HARTS_CONV_BWD
  }
  if (int rc = conv_status("k_conv_bwd")) return rc;
  const int64_t n = static_cast<int64_t>(Cch) * w;
  hipLaunchKernelGGL(k_conv_dw_sum, dim3(static_cast<uint32_t>((n + DW_K - 1) / DW_K)), dim3(CV_THR), 0,
                     s, n_run, Cch, w, part, dW);
  return conv_status("k_conv_dw_sum");
}

}  // namespace
}  // namespace harts

using namespace harts;

extern "C" int harts_conv_workspace_size(int64_t C, int32_t Cch, int32_t w, size_t* bytes) {
  if (int rc = check_conv(HARTS_F32, C, Cch, w, "harts_conv_workspace_size")) return rc;
  if (!bytes) { set_error("harts_conv_workspace_size: NULL bytes"); return HARTS_EINVAL; }
  const int64_t n_run = (C + CV_RUN_B - 1) / CV_RUN_B;
  *bytes = static_cast<size_t>(std::max<int64_t>(n_run, 1)) * Cch * w * sizeof(float);
  return HARTS_OK;
}

extern "C" int harts_conv_fwd(int32_t dtype, int64_t C, int32_t Cch, int32_t w, const void* x, const float* Wt,
                              const int32_t* pred, void* y, void* stream) {
  if (int rc = check_conv(dtype, C, Cch, w, "harts_conv_fwd")) return rc;
  if (C == 0) return HARTS_OK;
  if (!x || !Wt || !pred || !y || !a16(x) || !a16(y) || !a16(Wt)) {
    set_error("harts_conv_fwd: NULL or misaligned (16 bytes) pointer");
    return HARTS_EINVAL;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  return dtype == HARTS_BF16 ? launch_fwd<bf16>(w, C, Cch, x, Wt, pred, y, s)
                             : launch_fwd<float>(w, C, Cch, x, Wt, pred, y, s);
}

extern "C" int harts_conv_bwd(int32_t dtype, int64_t C, int32_t Cch, int32_t w, const void* x, const float* Wt,
                              const int32_t* pred, const int64_t* succ_off, const int32_t* succ,
                              int64_t n_succ, const void* dy, void* dx, float* dW, void* ws,
                              size_t ws_bytes, void* stream) {
  if (int rc = check_conv(dtype, C, Cch, w, "harts_conv_bwd")) return rc;
  if (C == 0) return HARTS_OK;
  if (!x || !Wt || !pred || !succ_off || (!succ && n_succ > 0) || n_succ < 0 || !dy || !dx || !dW || !ws ||
      !a16(x) || !a16(dy) || !a16(dx) || !a16(Wt)) {
    set_error("harts_conv_bwd: NULL or misaligned (16 bytes) pointer, or n_succ < 0");
    return HARTS_EINVAL;
  }
  size_t need = 0;
  harts_conv_workspace_size(C, Cch, w, &need);
  if (ws_bytes < need) {
    set_error("harts_conv_bwd: workspace too small (see harts_conv_workspace_size)");
    return HARTS_EINVAL;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  float* part = static_cast<float*>(ws);
  return dtype == HARTS_BF16
             ? launch_bwd<bf16>(w, C, Cch, x, Wt, pred, succ_off, succ, n_succ, dy, dx, dW, part, s)
             : launch_bwd<float>(w, C, Cch, x, Wt, pred, succ_off, succ, n_succ, dy, dx, dW, part, s);
}
