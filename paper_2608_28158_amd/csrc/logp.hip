// Compact-to-semantic log-probabilities for gfx950 (HARTS, Sec. 3.5).
//
// Vocabulary-wide work runs once per compact logit row, scalar work once
// per semantic position (eq. mapped-logp):
//   k_logp_lse     one workgroup per compact row c streams z[c, :] and keeps
//                  a running (max, sum of exponentials) per thread, then
//                  combines them: lse_c = log sum_v exp z[c, v];
//   k_logp_gather  one thread per position s: lambda_s = z[m(s), y_s] - lse.
// Backward (eq. mapped-logp-grad), for upstream gradients g_s:
//   k_logp_rowsum  one thread per row: G_c = sum of g_s over the row's
//                  positions, in the row's (target, position) order;
//   k_logp_grad    one workgroup per row writes dz[c, v] = -G_c p_{c,v},
//                  p = exp(z - lse), over the whole vocabulary;
//   k_logp_onehot  one thread per row rewrites the row's target columns:
//                  dz[c, y] = -G_c p_{c,y} + (sum of g_s over the row's
//                  positions with y_s = y), one rounding from float32.
// Rows are streamed as 16-byte vectors (8 bf16 or 4 float32 logits per
// load, four loads in flight per thread); exponentials are base 2 of
// log2(e)-scaled logits.  No atomics: every output is written by one thread.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "harts.h"
#include "plan.hpp"

namespace harts {
namespace {

typedef __bf16 bf16;
constexpr int LP_THR = 256;   // threads per row workgroup
constexpr int LP_UNROLL = 4;  // 16-byte loads in flight per thread
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <typename T> struct LV;
template <> struct LV<bf16> {
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
    for (int i = 0; i < 8; ++i) b[i] = static_cast<bf16>(x[i]);  // round to nearest even
    *reinterpret_cast<bf16x8*>(p) = b;
  }
  __device__ static inline float one(const bf16* p) { return static_cast<float>(*p); }
  __device__ static inline void put(bf16* p, float x) { *p = static_cast<bf16>(x); }
};
template <> struct LV<float> {
  static constexpr int N = 4;
  __device__ static inline void load(const float* p, float* x) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    x[0] = u.x; x[1] = u.y; x[2] = u.z; x[3] = u.w;
  }
  __device__ static inline void store(float* p, const float* x) {
    *reinterpret_cast<float4*>(p) = float4{x[0], x[1], x[2], x[3]};
  }
  __device__ static inline float one(const float* p) { return *p; }
  __device__ static inline void put(float* p, float x) { *p = x; }
};

__device__ inline float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

// (m, s) with s = sum 2^(x - m): merge two partial results
__device__ inline void lse_merge(float& m, float& s, float m2, float s2) {
  const float n = fmaxf(m, m2);
  s = (m == -INFINITY ? 0.f : s * ex2(m - n)) + (m2 == -INFINITY ? 0.f : s2 * ex2(m2 - n));
  m = n;
}

template <typename T>
__global__ __launch_bounds__(LP_THR) void k_logp_lse(const T* __restrict__ z, int64_t V,
                                                     float* __restrict__ lse) {
  using L = LV<T>;
  const int64_t c = blockIdx.x;
  const int t = threadIdx.x;
  const T* row = z + c * V;
  const int64_t nvec = V / L::N;
  float m = -INFINITY, s = 0.f;
  for (int64_t i0 = t; i0 < nvec; i0 += static_cast<int64_t>(LP_THR) * LP_UNROLL) {
    float x[LP_UNROLL][L::N];
#pragma unroll
    for (int u = 0; u < LP_UNROLL; ++u) {
      const int64_t i = i0 + static_cast<int64_t>(u) * LP_THR;
      if (i < nvec) {
        L::load(row + i * L::N, x[u]);
      } else {
#pragma unroll
        for (int e = 0; e < L::N; ++e) x[u][e] = -INFINITY;
      }
    }
#pragma unroll
    for (int u = 0; u < LP_UNROLL; ++u) {
      float vm = -INFINITY;
#pragma unroll
      for (int e = 0; e < L::N; ++e) {
        x[u][e] *= kLog2e;
        vm = fmaxf(vm, x[u][e]);
      }
      if (vm == -INFINITY) continue;  // a vector past the row's end
      const float n = fmaxf(m, vm);
      float acc = m == -INFINITY ? 0.f : s * ex2(m - n);
#pragma unroll
      for (int e = 0; e < L::N; ++e) acc += ex2(x[u][e] - n);
      m = n;
      s = acc;
    }
  }
  // wave, then workgroup
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float m2 = __shfl_xor(m, off);
    const float s2 = __shfl_xor(s, off);
    lse_merge(m, s, m2, s2);
  }
  __shared__ float ms[LP_THR / 64], ss[LP_THR / 64];
  if ((t & 63) == 0) {
    ms[t >> 6] = m;
    ss[t >> 6] = s;
  }
  __syncthreads();
  if (t == 0) {
    float mm = ms[0], sa = ss[0];
    for (int w = 1; w < LP_THR / 64; ++w) lse_merge(mm, sa, ms[w], ss[w]);
    lse[c] = (mm + log2f(sa)) * kLn2;
  }
}

template <typename T>
__global__ __launch_bounds__(LP_THR) void k_logp_gather(const T* __restrict__ z, int64_t C, int64_t V,
                                                        const float* __restrict__ lse,
                                                        const int32_t* __restrict__ m,
                                                        const int32_t* __restrict__ y, int64_t n_pos,
                                                        float* __restrict__ logp) {
  const int64_t s = static_cast<int64_t>(blockIdx.x) * LP_THR + threadIdx.x;
  if (s >= n_pos) return;
  const int32_t c = m[s], v = y[s];
  // an index outside the logits yields NaN instead of a read out of bounds
  if (c < 0 || c >= C || v < 0 || v >= V) {
    logp[s] = __builtin_nanf("");
    return;
  }
  logp[s] = LV<T>::one(z + static_cast<int64_t>(c) * V + v) - lse[c];
}

__global__ __launch_bounds__(LP_THR) void k_logp_rowsum(const int64_t* __restrict__ row_off,
                                                        const int32_t* __restrict__ row_pos,
                                                        const float* __restrict__ g, int64_t C,
                                                        int64_t n_pos, float* __restrict__ G) {
  const int64_t c = static_cast<int64_t>(blockIdx.x) * LP_THR + threadIdx.x;
  if (c >= C) return;
  const int64_t b = row_off[c] < 0 ? 0 : row_off[c];
  const int64_t e = row_off[c + 1] > n_pos ? n_pos : row_off[c + 1];
  float acc = 0.f;
  for (int64_t j = b; j < e; ++j) {
    const int32_t s = row_pos[j];
    if (s >= 0 && s < n_pos) acc += g[s];
  }
  G[c] = acc;
}

template <typename T>
__global__ __launch_bounds__(LP_THR) void k_logp_grad(const T* __restrict__ z, int64_t V,
                                                      const float* __restrict__ lse,
                                                      const float* __restrict__ G, T* __restrict__ dz) {
  using L = LV<T>;
  const int64_t c = blockIdx.x;
  const int t = threadIdx.x;
  const T* row = z + c * V;
  T* out = dz + c * V;
  const int64_t nvec = V / L::N;
  const float l2 = lse[c] * kLog2e;
  const float ng = -G[c];
  for (int64_t i0 = t; i0 < nvec; i0 += static_cast<int64_t>(LP_THR) * LP_UNROLL) {
    float x[LP_UNROLL][L::N];
#pragma unroll
    for (int u = 0; u < LP_UNROLL; ++u) {
      const int64_t i = i0 + static_cast<int64_t>(u) * LP_THR;
      if (i < nvec) L::load(row + i * L::N, x[u]);
    }
#pragma unroll
    for (int u = 0; u < LP_UNROLL; ++u) {
      const int64_t i = i0 + static_cast<int64_t>(u) * LP_THR;
      if (i < nvec) {
#pragma unroll
        for (int e = 0; e < L::N; ++e) x[u][e] = ng * ex2(x[u][e] * kLog2e - l2);
        L::store(out + i * L::N, x[u]);
      }
    }
  }
}

template <typename T>
__global__ __launch_bounds__(LP_THR) void k_logp_onehot(const T* __restrict__ z, int64_t C, int64_t V,
                                                        const float* __restrict__ lse,
                                                        const float* __restrict__ G,
                                                        const int64_t* __restrict__ row_off,
                                                        const int32_t* __restrict__ row_pos,
                                                        const int32_t* __restrict__ y,
                                                        const float* __restrict__ g, int64_t n_pos,
                                                        T* __restrict__ dz) {
  const int64_t c = static_cast<int64_t>(blockIdx.x) * LP_THR + threadIdx.x;
  if (c >= C) return;
  const int64_t b = row_off[c] < 0 ? 0 : row_off[c];
  const int64_t e = row_off[c + 1] > n_pos ? n_pos : row_off[c + 1];
  const float l2 = lse[c] * kLog2e;
  const float ng = -G[c];
  int64_t j = b;
  while (j < e) {
    const int32_t s0 = row_pos[j];
    if (s0 < 0 || s0 >= n_pos) {  // an invalid entry: skipped
      ++j;
      continue;
    }
    const int32_t v = y[s0];
    float acc = 0.f;
    // the run of positions with this target, in position order (it holds
    // at least the entry at j)
    for (; j < e; ++j) {
      const int32_t s = row_pos[j];
      if (s < 0 || s >= n_pos || y[s] != v) break;
      acc += g[s];
    }
    if (v < 0 || v >= V) continue;  // a target outside the vocabulary: skipped
    const int64_t at = c * V + v;
    const float p = ex2(LV<T>::one(z + at) * kLog2e - l2);
    LV<T>::put(dz + at, ng * p + acc);
  }
}

int hip_status(const char* where) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error(std::string(where) + ": " + hipGetErrorString(e));
    return HARTS_EHIP;
  }
  return HARTS_OK;
}

bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_logits(int32_t dtype, int64_t C, int64_t V, const char* where) {
  const std::string w(where);
  if (dtype != HARTS_F32 && dtype != HARTS_BF16) {
    set_error(w + ": unknown dtype");
    return HARTS_EUNSUPPORTED;
  }
  if (C < 0 || C > INT32_MAX) { set_error(w + ": need 0 <= C <= 2^31 - 1"); return HARTS_EINVAL; }
  if (V < 8 || V % 8 != 0 || V > INT32_MAX) {
    set_error(w + ": the vocabulary size must be a positive multiple of 8, below 2^31");
    return HARTS_EUNSUPPORTED;
  }
  return HARTS_OK;
}

}  // namespace
}  // namespace harts

using namespace harts;

extern "C" int harts_logp_fwd(int32_t dtype, int64_t C, int64_t V, const void* logits, int64_t n_pos,
                              const int32_t* m, const int32_t* y, float* lse, float* logp,
                              void* stream) {
  if (int rc = check_logits(dtype, C, V, "harts_logp_fwd")) return rc;
  if (n_pos < 0 || (C > 0 && (!logits || !lse)) || (n_pos > 0 && (!m || !y || !logp))) {
    set_error("harts_logp_fwd: NULL required pointer or n_pos < 0");
    return HARTS_EINVAL;
  }
  if (!al16(logits)) { set_error("harts_logp_fwd: logits must be 16-byte aligned"); return HARTS_EINVAL; }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (C > 0) {
    if (dtype == HARTS_BF16)
      hipLaunchKernelGGL((k_logp_lse<bf16>), dim3(static_cast<uint32_t>(C)), dim3(LP_THR), 0, s,
                         static_cast<const bf16*>(logits), V, lse);
    else
      hipLaunchKernelGGL((k_logp_lse<float>), dim3(static_cast<uint32_t>(C)), dim3(LP_THR), 0, s,
                         static_cast<const float*>(logits), V, lse);
    if (int rc = hip_status("k_logp_lse")) return rc;
  }
  if (n_pos > 0) {
    const dim3 grid(static_cast<uint32_t>((n_pos + LP_THR - 1) / LP_THR));
    if (dtype == HARTS_BF16)
      hipLaunchKernelGGL((k_logp_gather<bf16>), grid, dim3(LP_THR), 0, s,
                         static_cast<const bf16*>(logits), C, V, lse, m, y, n_pos, logp);
    else
      hipLaunchKernelGGL((k_logp_gather<float>), grid, dim3(LP_THR), 0, s,
                         static_cast<const float*>(logits), C, V, lse, m, y, n_pos, logp);
    if (int rc = hip_status("k_logp_gather")) return rc;
  }
  return HARTS_OK;
}

extern "C" int harts_logp_bwd(int32_t dtype, int64_t C, int64_t V, const void* logits,
                              const float* lse, int64_t n_pos, const int64_t* row_off,
                              const int32_t* row_pos, const int32_t* y, const float* dlogp,
                              float* row_g, void* dlogits, void* stream) {
  if (int rc = check_logits(dtype, C, V, "harts_logp_bwd")) return rc;
  if (n_pos < 0 || (C > 0 && (!logits || !lse || !row_off || !row_g || !dlogits)) ||
      (n_pos > 0 && (!row_pos || !y || !dlogp))) {
    set_error("harts_logp_bwd: NULL required pointer or n_pos < 0");
    return HARTS_EINVAL;
  }
  if (!al16(logits) || !al16(dlogits)) {
    set_error("harts_logp_bwd: logits and dlogits must be 16-byte aligned");
    return HARTS_EINVAL;
  }
  if (C == 0) return HARTS_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 rows(static_cast<uint32_t>((C + LP_THR - 1) / LP_THR));
  hipLaunchKernelGGL(k_logp_rowsum, rows, dim3(LP_THR), 0, s, row_off, row_pos, dlogp, C, n_pos, row_g);
  if (int rc = hip_status("k_logp_rowsum")) return rc;
  if (dtype == HARTS_BF16) {
    hipLaunchKernelGGL((k_logp_grad<bf16>), dim3(static_cast<uint32_t>(C)), dim3(LP_THR), 0, s,
                       static_cast<const bf16*>(logits), V, lse, row_g, static_cast<bf16*>(dlogits));
    if (int rc = hip_status("k_logp_grad")) return rc;
    hipLaunchKernelGGL((k_logp_onehot<bf16>), rows, dim3(LP_THR), 0, s, static_cast<const bf16*>(logits),
                       C, V, lse, row_g, row_off, row_pos, y, dlogp, n_pos, static_cast<bf16*>(dlogits));
  } else {
    hipLaunchKernelGGL((k_logp_grad<float>), dim3(static_cast<uint32_t>(C)), dim3(LP_THR), 0, s,
                       static_cast<const float*>(logits), V, lse, row_g, static_cast<float*>(dlogits));
    if (int rc = hip_status("k_logp_grad")) return rc;
    hipLaunchKernelGGL((k_logp_onehot<float>), rows, dim3(LP_THR), 0, s, static_cast<const float*>(logits),
                       C, V, lse, row_g, row_off, row_pos, y, dlogp, n_pos, static_cast<float*>(dlogits));
  }
  return hip_status("k_logp_onehot");
}
