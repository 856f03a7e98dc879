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
//   k_conv_fwd      one thread per (row, 16-byte channel vector);
//   k_conv_dx       one thread per (row, vector): its own term plus every
//                   consumer's, in (tap, row) order;
//   k_conv_dw_part  per block of 512 rows and channel vector, the tap sums
//                   x[pred_i(r)] dy[r] over the block's rows, in row order;
//   k_conv_dw_sum   per (channel, tap), the block partials in block order.
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
constexpr int CV_ROWS = 512;  // rows per weight-gradient block

template <typename T> struct CV;
template <> struct CV<bf16> {
  static constexpr int N = 8;
  __device__ static inline void load(const bf16* p, float* x) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  __device__ static inline void store(bf16* p, const float* x) {
    typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
    bf16x8 b;
#pragma unroll
    for (int i = 0; i < 8; ++i) b[i] = static_cast<bf16>(x[i]);
    *reinterpret_cast<bf16x8*>(p) = b;
  }
};
template <> struct CV<float> {
  static constexpr int N = 4;
  __device__ static inline void load(const float* p, float* x) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
  }
  __device__ static inline void store(float* p, const float* x) {
    *reinterpret_cast<float4*>(p) = float4{x[0], x[1], x[2], x[3]};
  }
};

template <typename T, int W>
__global__ __launch_bounds__(CV_THR) void k_conv_fwd(int64_t C, int Cch, const T* __restrict__ x,
                                                     const float* __restrict__ Wt,
                                                     const int32_t* __restrict__ pred, T* __restrict__ y) {
  using V = CV<T>;
  const int nvec = Cch / V::N;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * CV_THR + threadIdx.x;
  const int64_t row = idx / nvec;
  if (row >= C) return;
  const int c0 = static_cast<int>(idx % nvec) * V::N;
  float acc[V::N], v[V::N];
  V::load(x + row * Cch + c0, v);
#pragma unroll
  for (int e = 0; e < V::N; ++e) acc[e] = Wt[(c0 + e) * W] * v[e];
#pragma unroll
  for (int i = 1; i < W; ++i) {
    const int32_t p = pred[row * (W - 1) + i - 1];
    if (p < 0 || p >= C) continue;  // before the trajectory start (or invalid): zero
    V::load(x + static_cast<int64_t>(p) * Cch + c0, v);
#pragma unroll
    for (int e = 0; e < V::N; ++e) acc[e] += Wt[(c0 + e) * W + i] * v[e];
  }
  V::store(y + row * Cch + c0, acc);
}

template <typename T, int W>
__global__ __launch_bounds__(CV_THR) void k_conv_dx(int64_t C, int Cch, const float* __restrict__ Wt,
                                                    const int64_t* __restrict__ succ_off,
                                                    const int32_t* __restrict__ succ, int64_t n_succ,
                                                    const T* __restrict__ dy, T* __restrict__ dx) {
  using V = CV<T>;
  const int nvec = Cch / V::N;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * CV_THR + threadIdx.x;
  const int64_t row = idx / nvec;
  if (row >= C) return;
  const int c0 = static_cast<int>(idx % nvec) * V::N;
  float acc[V::N], v[V::N];
  V::load(dy + row * Cch + c0, v);
#pragma unroll
  for (int e = 0; e < V::N; ++e) acc[e] = Wt[(c0 + e) * W] * v[e];
  const int64_t b = succ_off[row] < 0 ? 0 : succ_off[row];
  const int64_t end = succ_off[row + 1] > n_succ ? n_succ : succ_off[row + 1];
  for (int64_t j = b; j < end; ++j) {
    const int32_t code = succ[j];
    const int32_t s = code >> 3, i = code & 7;  // consumer row, tap
    if (s < 0 || s >= C || i < 1 || i >= W) continue;
    V::load(dy + static_cast<int64_t>(s) * Cch + c0, v);
#pragma unroll
    for (int e = 0; e < V::N; ++e) acc[e] += Wt[(c0 + e) * W + i] * v[e];
  }
  V::store(dx + row * Cch + c0, acc);
}

// partial[blk][c][i] = sum over the block's rows r of x[pred_i(r)][c] dy[r][c]
template <typename T, int W>
__global__ __launch_bounds__(CV_THR) void k_conv_dw_part(int64_t C, int Cch, const T* __restrict__ x,
                                                         const int32_t* __restrict__ pred,
                                                         const T* __restrict__ dy,
                                                         float* __restrict__ part) {
  using V = CV<T>;
  const int nvec = Cch / V::N;
  const int vec = blockIdx.y * CV_THR + threadIdx.x;
  if (vec >= nvec) return;
  const int c0 = vec * V::N;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * CV_ROWS;
  const int64_t r1 = r0 + CV_ROWS < C ? r0 + CV_ROWS : C;
  float acc[W][V::N];
#pragma unroll
  for (int i = 0; i < W; ++i)
#pragma unroll
    for (int e = 0; e < V::N; ++e) acc[i][e] = 0.f;
  for (int64_t r = r0; r < r1; ++r) {
    float g[V::N], v[V::N];
    V::load(dy + r * Cch + c0, g);
    V::load(x + r * Cch + c0, v);
#pragma unroll
    for (int e = 0; e < V::N; ++e) acc[0][e] += v[e] * g[e];
#pragma unroll
    for (int i = 1; i < W; ++i) {
      const int32_t p = pred[r * (W - 1) + i - 1];
      if (p < 0 || p >= C) continue;
      V::load(x + static_cast<int64_t>(p) * Cch + c0, v);
#pragma unroll
      for (int e = 0; e < V::N; ++e) acc[i][e] += v[e] * g[e];
    }
  }
  float* out = part + static_cast<int64_t>(blockIdx.x) * Cch * W;
#pragma unroll
  for (int e = 0; e < V::N; ++e)
#pragma unroll
    for (int i = 0; i < W; ++i) out[(c0 + e) * W + i] = acc[i][e];
}

__global__ __launch_bounds__(CV_THR) void k_conv_dw_sum(int64_t n_blk, int64_t n, const float* __restrict__ part,
                                                        float* __restrict__ dW) {
  const int64_t k = static_cast<int64_t>(blockIdx.x) * CV_THR + threadIdx.x;
  if (k >= n) return;
  float acc = 0.f;
  for (int64_t b = 0; b < n_blk; ++b) acc += part[b * n + k];
  dW[k] = acc;
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
  const int64_t threads = C * (Cch / CV<T>::N);
  const dim3 grid(static_cast<uint32_t>((threads + CV_THR - 1) / CV_THR));
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
  const int64_t threads = C * (Cch / CV<T>::N);
  const dim3 grid(static_cast<uint32_t>((threads + CV_THR - 1) / CV_THR));
  const int64_t n_blk = (C + CV_ROWS - 1) / CV_ROWS;
  const int nvec = Cch / CV<T>::N;
  const dim3 pgrid(static_cast<uint32_t>(n_blk), static_cast<uint32_t>((nvec + CV_THR - 1) / CV_THR));
  const T* xx = static_cast<const T*>(x);
  const T* gy = static_cast<const T*>(dy);
  T* gx = static_cast<T*>(dx);
  switch (w) {
#define HARTS_CONV_BWD(WW)                                                                              \
  case WW:                                                                                              \
    hipLaunchKernelGGL((k_conv_dx<T, WW>), grid, dim3(CV_THR), 0, s, C, Cch, Wt, succ_off, succ, n_succ, \
                       gy, gx);                                                                         \
    if (int rc = conv_status("k_conv_dx")) return rc;                                                   \
    hipLaunchKernelGGL((k_conv_dw_part<T, WW>), pgrid, dim3(CV_THR), 0, s, C, Cch, xx, pred, gy, part); \
    break;
    HARTS_CONV_BWD(2) HARTS_CONV_BWD(3) HARTS_CONV_BWD(4) HARTS_CONV_BWD(5)
    HARTS_CONV_BWD(6) HARTS_CONV_BWD(7) HARTS_CONV_BWD(8)
#undef HARTS_CONV_BWD
  }
  if (int rc = conv_status("k_conv_dw_part")) return rc;
  const int64_t n = static_cast<int64_t>(Cch) * w;
  hipLaunchKernelGGL(k_conv_dw_sum, dim3(static_cast<uint32_t>((n + CV_THR - 1) / CV_THR)), dim3(CV_THR), 0,
                     s, n_blk, n, part, dW);
  return conv_status("k_conv_dw_sum");
}

}  // namespace
}  // namespace harts

using namespace harts;

extern "C" int harts_conv_workspace_size(int64_t C, int32_t Cch, int32_t w, size_t* bytes) {
  if (int rc = check_conv(HARTS_F32, C, Cch, w, "harts_conv_workspace_size")) return rc;
  if (!bytes) { set_error("harts_conv_workspace_size: NULL bytes"); return HARTS_EINVAL; }
  const int64_t n_blk = (C + CV_ROWS - 1) / CV_ROWS;
  *bytes = static_cast<size_t>(std::max<int64_t>(n_blk, 1)) * Cch * w * sizeof(float);
  return HARTS_OK;
}

extern "C" int harts_conv_fwd(int32_t dtype, int64_t C, int32_t Cch, int32_t w, const void* x, const float* Wt,
                              const int32_t* pred, void* y, void* stream) {
  if (int rc = check_conv(dtype, C, Cch, w, "harts_conv_fwd")) return rc;
  if (C == 0) return HARTS_OK;
  if (!x || !Wt || !pred || !y || !a16(x) || !a16(y)) {
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
      !a16(x) || !a16(dy) || !a16(dx)) {
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
