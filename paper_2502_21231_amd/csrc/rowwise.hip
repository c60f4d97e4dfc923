// Bandwidth-bound row kernels: LSE merge, backward preprocess, dQ finalize.
//
// Each (token, head) row of head_dim elements is handled by a group of
// head_dim/8 (bf16) or head_dim/4 (fp32) lanes, one 16-byte vector per lane,
// so every row is read and written with fully coalesced 16-byte accesses.
#include "attn.hpp"

namespace bs {
namespace {

template <typename T> struct Vec;
template <> struct Vec<bf16> { typedef bf16x8 type; static constexpr int N = 8; };
template <> struct Vec<float> { typedef f32x4 type; static constexpr int N = 4; };

template <typename T>
__device__ __forceinline__ float to_f(T x) { return (float)x; }
template <typename T>
__device__ __forceinline__ T from_f(float x);
template <> __device__ __forceinline__ bf16 from_f<bf16>(float x) { return f2bf(x); }
template <> __device__ __forceinline__ float from_f<float>(float x) { return x; }

// Combination of the partial results of one query row over n disjoint key
// sets (the steps of a context-parallel ring):
//   LSE = m + log(sum_c exp(LSE_c - m)),   O = sum_c exp(LSE_c - LSE) O_c,
// m = max_c LSE_c; partials at -inf weigh 0; all -inf gives O = 0, LSE = -inf.
template <typename T, int D, int U>
__global__ __launch_bounds__(256) void lse_merge_kernel(const T* __restrict__ parts,
                                                        const float* __restrict__ lse_parts,
                                                        int32_t n, int64_t rows, int32_t hq,
                                                        int64_t total_q, T* __restrict__ out,
                                                        float* __restrict__ lse) {
  typedef typename Vec<T>::type V;
  constexpr int LPR = D / Vec<T>::N;  // lanes per row
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = gid / LPR;      // row = t * hq + h
  const int part = gid % LPR;
  if (row >= rows) return;
  const int64_t t = row / hq;
  const int h = row % hq;
  const float* lp = lse_parts + (int64_t)h * total_q + t;
  const int64_t lstride = (int64_t)hq * total_q;
  const int64_t pstride = rows * D;
  const T* src = parts + row * D + part * Vec<T>::N;
  float acc[Vec<T>::N];
#pragma unroll
  for (int i = 0; i < Vec<T>::N; ++i) acc[i] = 0.f;
  float m = -INFINITY, wsum = 0.f;
  // partials in groups of U: every load of a group is issued before any of it is used, so
  // that each lane keeps U row reads in flight (one at a time is latency-bound); the sum is
  // rescaled when a group raises the running maximum
  for (int c0 = 0; c0 < n; c0 += U) {
    float l[U];
    V x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (c0 + u < n) {
        l[u] = lp[(c0 + u) * lstride];
        x[u] = __builtin_nontemporal_load(reinterpret_cast<const V*>(src + (c0 + u) * pstride));
      } else {
        l[u] = -INFINITY;
        x[u] = V{};
      }
    }
    float mg = m;
#pragma unroll
    for (int u = 0; u < U; ++u) mg = fmaxf(mg, l[u]);
    if (mg == -INFINITY) continue;
    const float r = expf(m - mg);  // 0 while nothing was added (m = -inf)
    wsum *= r;
#pragma unroll
    for (int i = 0; i < Vec<T>::N; ++i) acc[i] *= r;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float wgt = expf(l[u] - mg);  // exp(-inf) = 0
      wsum += wgt;
#pragma unroll
      for (int i = 0; i < Vec<T>::N; ++i) acc[i] += wgt * to_f(x[u][i]);
    }
    m = mg;
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  V y;
#pragma unroll
  for (int i = 0; i < Vec<T>::N; ++i) y[i] = from_f<T>(acc[i] * inv);
  *reinterpret_cast<V*>(out + row * D + part * Vec<T>::N) = y;
  if (part == 0) lse[(int64_t)h * total_q + t] = m == -INFINITY ? -INFINITY : m + logf(wsum);
}

// D = rowsum(dO * O) in fp32, stored [hq, T]; optionally zeroes a dQ accumulator.
template <typename T, int D>
__global__ __launch_bounds__(256) void preprocess_kernel(const T* __restrict__ o,
                                                         const T* __restrict__ dout, int64_t rows,
                                                         int32_t hq, int64_t total_q,
                                                         float* __restrict__ dvec,
                                                         float* __restrict__ dq_acc,
                                                         const WsHeader* __restrict__ hdr) {
  typedef typename Vec<T>::type V;
  if (hdr != nullptr && hdr->status != BS_DEV_OK) return;  // planner rejected the input
  constexpr int LPR = D / Vec<T>::N;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = gid / LPR;
  const int part = gid % LPR;
  const bool live = row < rows;
  float s = 0.f;
  if (live) {
    const V a = *reinterpret_cast<const V*>(o + row * D + part * Vec<T>::N);
    const V b = *reinterpret_cast<const V*>(dout + row * D + part * Vec<T>::N);
#pragma unroll
    for (int i = 0; i < Vec<T>::N; ++i) s += to_f(a[i]) * to_f(b[i]);
    if (dq_acc != nullptr) {
      f32x4* z = reinterpret_cast<f32x4*>(dq_acc + row * D + part * Vec<T>::N);
#pragma unroll
      for (int i = 0; i < Vec<T>::N / 4; ++i) z[i] = f32x4{};
    }
  }
  // reduce over the LPR lanes of the row (LPR is a power of two <= 32, aligned)
#pragma unroll
  for (int off = LPR / 2; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (live && part == 0) dvec[(int64_t)(row % hq) * total_q + row / hq] = s;
}

template <typename T>
__global__ __launch_bounds__(256) void dq_finalize_kernel(const float* __restrict__ acc,
                                                          T* __restrict__ dq, int64_t n4,
                                                          const WsHeader* __restrict__ hdr) {
  if (hdr != nullptr && hdr->status != BS_DEV_OK) return;  // planner rejected the input
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  const f32x4 x = reinterpret_cast<const f32x4*>(acc)[i];
  T y[4] __attribute__((aligned(16)));
#pragma unroll
  for (int j = 0; j < 4; ++j) y[j] = from_f<T>(x[j]);
  if constexpr (sizeof(T) == 2)
    *reinterpret_cast<bf16x4*>(dq + i * 4) = *reinterpret_cast<const bf16x4*>(y);
  else
    *reinterpret_cast<f32x4*>(dq + i * 4) = *reinterpret_cast<const f32x4*>(y);
}

inline unsigned blocks_for(int64_t threads) { return (unsigned)((threads + 255) / 256); }

}  // namespace

hipError_t launch_lse_merge(const bs_dims& dims, const void* out_parts, const float* lse_parts,
                            int32_t n, void* out, float* lse, hipStream_t stream) {
  const int64_t rows = dims.total_q * dims.hq;
  if (rows == 0) return hipSuccess;
  const int vec = dims.dtype == BS_BF16 ? 8 : 4;
  const unsigned grid = blocks_for(rows * (dims.head_dim / vec));
#define BS_MERGE_U(T, D, U)                                                                   \
  hipLaunchKernelGGL((lse_merge_kernel<T, D, U>), dim3(grid), dim3(256), 0, stream,          \
                     static_cast<const T*>(out_parts), lse_parts, n, rows, dims.hq,           \
                     dims.total_q, static_cast<T*>(out), lse)
#define BS_MERGE(T, D)                                                                        \
  do {                                                                                        \
    if (n <= 2) BS_MERGE_U(T, D, 2);                                                          \
    else if (n <= 4) BS_MERGE_U(T, D, 4);                                                     \
    else BS_MERGE_U(T, D, 8);                                                                 \
  } while (0)
  if (dims.dtype == BS_BF16) {
    if (dims.head_dim == 128) BS_MERGE(bf16, 128); else BS_MERGE(bf16, 64);
  } else {
    if (dims.head_dim == 128) BS_MERGE(float, 128); else BS_MERGE(float, 64);
  }
#undef BS_MERGE
#undef BS_MERGE_U
  return hipGetLastError();
}

hipError_t launch_bwd_preprocess(const bs_dims& dims, const void* out, const void* dout,
                                 float* dvec, float* dq_acc_to_zero, const void* ws,
                                 hipStream_t stream) {
  const int64_t rows = dims.total_q * dims.hq;
  if (rows == 0) return hipSuccess;
  const int vec = dims.dtype == BS_BF16 ? 8 : 4;
  const unsigned grid = blocks_for(rows * (dims.head_dim / vec));
#define BS_PRE(T, D)                                                                          \
  hipLaunchKernelGGL((preprocess_kernel<T, D>), dim3(grid), dim3(256), 0, stream,            \
                     static_cast<const T*>(out), static_cast<const T*>(dout), rows, dims.hq,  \
                     dims.total_q, dvec, dq_acc_to_zero,             \
                     static_cast<const WsHeader*>(ws))
  if (dims.dtype == BS_BF16) {
    if (dims.head_dim == 128) BS_PRE(bf16, 128); else BS_PRE(bf16, 64);
  } else {
    if (dims.head_dim == 128) BS_PRE(float, 128); else BS_PRE(float, 64);
  }
#undef BS_PRE
  return hipGetLastError();
}

hipError_t launch_dq_finalize(const bs_dims& dims, const float* dq_acc, void* dq,
                              const void* ws, hipStream_t stream) {
  const WsHeader* hdr = static_cast<const WsHeader*>(ws);
  const int64_t n4 = dims.total_q * dims.hq * dims.head_dim / 4;
  if (n4 == 0) return hipSuccess;
  if (dims.dtype == BS_BF16)
    hipLaunchKernelGGL(dq_finalize_kernel<bf16>, dim3(blocks_for(n4)), dim3(256), 0, stream,
                       dq_acc, static_cast<bf16*>(dq), n4, hdr);
  else
    hipLaunchKernelGGL(dq_finalize_kernel<float>, dim3(blocks_for(n4)), dim3(256), 0, stream,
                       dq_acc, static_cast<float*>(dq), n4, hdr);
  return hipGetLastError();
}

}  // namespace bs
