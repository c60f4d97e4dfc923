// Softmax cross-entropy over a large vocabulary with its gradient fused in (Sec. 7,
// Fused SoftmaxCrossEntropy): bf16 (or fp32) logits in, fp32 arithmetic, per-token loss and
// log-sum-exp out, and the gradient g (softmax - onehot) written in the logits' dtype, in
// place over the logits if the caller wants.  No fp32 copy of the logits is ever made.
//
// Bandwidth-bound, one workgroup per row, in two forms.  bf16 rows of 16K..128K entries (the
// vocabularies of current LLMs up to LLaMA3's) use the register-resident form below: the row is read from HBM
// once into registers and its gradient written from there.  Other rows are streamed twice by a
// persistent grid that keeps one row per CU in flight, so that the second pass finds the row in
// the caches.  Streaming form: pass 1 streams the row with 16-byte loads and keeps
// a running (max, sum of 2^(x - max)) per lane in the log2 domain; the max is raised only when a
// chunk exceeds it by 2^8, so the sum is rescaled almost never and its terms stay below 2^8.
// The lanes' pairs are combined in a fixed order (wave shuffles, then the waves through LDS),
// so every run gives the same bits.  Pass 2 reads the row again (it is still in the XCD's L2 or
// the last-level cache: the same workgroup read it microseconds before), forms
// g * (2^(x - lse) - [j == label]) and writes it.  HBM traffic per element: the logit read once
// and the gradient written once.
#include "common.hpp"

namespace bs {
namespace {

constexpr int kXentThreads = 1024;
constexpr float kXentRescale = 8.0f;  // log2 units

struct XentParams {
  const void* logits;
  const int64_t* labels;
  void* dlogits;
  float* loss;
  float* lse;
  int64_t vocab;
  int64_t ignore_index;
  float grad_scale;
};

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <typename T> struct XVec;
template <> struct XVec<bf16> { typedef bf16x8 type; static constexpr int N = 8; };
template <> struct XVec<float> { typedef f32x4 type; static constexpr int N = 4; };

// (m, s) <- the pair that represents both: s 2^m = s 2^m + s2 2^m2 (log2 domain)
__device__ __forceinline__ void combine(float& m, float& s, float m2, float s2) {
  const float M = fmaxf(m, m2);
  if (M == -INFINITY) return;  // both still empty
  s = s * fast_exp2(m - M) + s2 * fast_exp2(m2 - M);  // 2^-inf = 0
  m = M;
}

// Adds N logits (raw values z; x = z log2 e) to the lane's running pair.
template <int N>
__device__ __forceinline__ void accumulate(const float (&z)[N], float& m, float& s) {
  float zc = z[0];
#pragma unroll
  for (int k = 1; k < N; ++k) zc = fmaxf(zc, z[k]);
  const float mc = zc * kLog2e;
  if (mc > m + kXentRescale) {  // first chunk (m = -inf), or a new max well above the old
    s *= fast_exp2(m - mc);
    m = mc;
  }
  const float b = m == -INFINITY ? 0.f : m;  // a row that so far holds only -inf
#pragma unroll
  for (int k = 0; k < N; ++k) s += fast_exp2(fmaf(z[k], kLog2e, -b));
}

template <typename T, int N>
__device__ __forceinline__ void load_f(const T* src, float (&z)[N]) {
  if constexpr (N == 1) {
    z[0] = (float)src[0];
  } else {
    const typename XVec<T>::type v = *reinterpret_cast<const typename XVec<T>::type*>(src);
#pragma unroll
    for (int k = 0; k < N; ++k) z[k] = (float)v[k];
  }
}

template <typename T, int N>
__device__ __forceinline__ void store_f(T* dst, const float (&g)[N]) {
  if constexpr (N == 1) {
    if constexpr (sizeof(T) == 2) dst[0] = f2bf(g[0]);
    else dst[0] = g[0];
  } else {
    typename XVec<T>::type v;
#pragma unroll
    for (int k = 0; k < N; ++k) {
      if constexpr (sizeof(T) == 2) v[k] = f2bf(g[k]);
      else v[k] = g[k];
    }
    *reinterpret_cast<typename XVec<T>::type*>(dst) = v;
  }
}

// VEC: 16-byte chunks (vocab a multiple of the vector width, rows 16-byte aligned); otherwise
// one element per lane and step.  Persistent: one workgroup of kXentThreads lanes per CU walks
// the rows strided by the grid, so that only one row per CU is in flight and the second pass
// finds it in the caches (a row is read from HBM once as long as the rows in flight, CUs x row
// bytes, fit the last-level cache).
template <typename T, bool VEC>
__global__ __launch_bounds__(kXentThreads) void xent_kernel(const XentParams p, int64_t rows) {
  constexpr int N = VEC ? XVec<T>::N : 1;
  constexpr int U = VEC ? 4 : 8;  // chunks in flight per lane
  constexpr int NW = kXentThreads / 64;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t nch = p.vocab / N;
  __shared__ float red_m[2][NW], red_s[2][NW];
  int it = 0;
  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x, ++it) {
    const T* zr = static_cast<const T*>(p.logits) + row * p.vocab;
    const int64_t y = p.labels[row];
    const bool ignored = y == p.ignore_index;
    const bool in_range = y >= 0 && y < p.vocab;

    // pass 1: running (max, sum) per lane
    float m = -INFINITY, s = 0.f;
    int64_t c = tid;
    for (; c + (U - 1) * kXentThreads < nch; c += U * kXentThreads) {
      float z[U][N];
#pragma unroll
      for (int u = 0; u < U; ++u) load_f<T, N>(zr + (c + u * kXentThreads) * N, z[u]);
#pragma unroll
      for (int u = 0; u < U; ++u) accumulate<N>(z[u], m, s);
    }
    for (; c < nch; c += kXentThreads) {
      float z[N];
      load_f<T, N>(zr + c * N, z);
      accumulate<N>(z, m, s);
    }
    // the label's logit, read before any gradient can overwrite it (in-place use)
    float zy = 0.f;
    if (tid == 0 && !ignored && in_range) zy = (float)zr[y];

    // fixed-order reduction: within the wave, then the waves (two buffers, alternating by row)
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const float m2 = __shfl_xor(m, off), s2 = __shfl_xor(s, off);
      combine(m, s, m2, s2);
    }
    const int rb = it & 1;
    if (lane == 0) {
      red_m[rb][w] = m;
      red_s[rb][w] = s;
    }
    __syncthreads();
    m = red_m[rb][0];
    s = red_s[rb][0];
#pragma unroll
    for (int i = 1; i < NW; ++i) combine(m, s, red_m[rb][i], red_s[rb][i]);
    const float lse2 = m == -INFINITY ? -INFINITY : m + log2f(s);
    if (tid == 0) {
      if (p.lse != nullptr) p.lse[row] = lse2 * kLn2;
      p.loss[row] = ignored ? 0.f : (in_range ? lse2 * kLn2 - zy : NAN);
    }
    if (p.dlogits == nullptr) continue;

    // pass 2: gradient g (2^(x - lse2) - [j == label]); an ignored row is written as zeros
    T* dr = static_cast<T*>(p.dlogits) + row * p.vocab;
    const float g = p.grad_scale;
    const int64_t cy = in_range && !ignored ? y / N : -1;
    const int ky = (int)(y - cy * N);
    auto grad = [&](int64_t cc, const float (&z)[N]) {
      float o[N];
#pragma unroll
      for (int k = 0; k < N; ++k) o[k] = fast_exp2(fmaf(z[k], kLog2e, -lse2)) * g;
      if (cc == cy) {
#pragma unroll
        for (int k = 0; k < N; ++k) o[k] = k == ky ? o[k] - g : o[k];
      }
      store_f<T, N>(dr + cc * N, o);
    };
    c = tid;
    if (ignored) {
      const float zero[N] = {};
      for (; c < nch; c += kXentThreads) store_f<T, N>(dr + c * N, zero);
      continue;
    }
    for (; c + (U - 1) * kXentThreads < nch; c += U * kXentThreads) {
      float z[U][N];
#pragma unroll
      for (int u = 0; u < U; ++u) load_f<T, N>(zr + (c + u * kXentThreads) * N, z[u]);
#pragma unroll
      for (int u = 0; u < U; ++u) grad(c + u * kXentThreads, z[u]);
    }
    for (; c < nch; c += kXentThreads) {
      float z[N];
      load_f<T, N>(zr + c * N, z);
      grad(c, z);
    }
  }
}

// Register-resident form (bf16, vocab a multiple of 8 and at most 8 * 1024 * CPT): 1024 lanes
// per row, each holding its CPT 16-byte chunks of the row in registers from the one read of
// the row to the write of its gradient, so the row is read from HBM exactly once whatever the
// caches hold.  The grid is persistent (one workgroup per CU, rows strided by the grid): as a
// chunk's gradient is stored, the same registers load that chunk of the workgroup's next row,
// so the next row's reads overlap this row's writes and arithmetic without extra registers.
// Each lane folds its chunks into a running (max, sum) as the streamed form does, and the 16
// waves combine their pairs in a fixed order through LDS (two buffers, alternating by row).
constexpr int kXentRegThreads = 1024;

template <int CPT>
__global__ __launch_bounds__(kXentRegThreads) void xent_reg_kernel(const XentParams p,
                                                                   int64_t rows) {
  constexpr int NW = kXentRegThreads / 64;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nch = (int)(p.vocab / 8);
  const bf16* z0 = static_cast<const bf16*>(p.logits);
  __shared__ float red_m[2][NW], red_s[2][NW];

  // buffer descriptors of one row (bases in scalar registers): chunk i of the lane is at byte
  // tid * 16 + i * 16 KB, so no per-chunk address occupies vector registers
  const uint32_t row_bytes = (uint32_t)(p.vocab * 2);
  auto rsrc_of = [&](const void* base) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, row_bytes, 0x00020000);
  };
  auto load_row = [&](int64_t r, bf16x8 (&dst)[CPT]) {
    const __amdgpu_buffer_rsrc_t rs = rsrc_of(z0 + r * p.vocab);
#pragma unroll
    for (int i = 0; i < CPT; ++i)
      if (tid + i * kXentRegThreads < nch)
        dst[i] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(
                                                rs, tid * 16, i * kXentRegThreads * 16, 0));
  };

  int64_t row = blockIdx.x;
  bf16x8 buf[CPT];
  if (row < rows) load_row(row, buf);
  for (int it = 0; row < rows; ++it, row += gridDim.x) {
    const int64_t next = row + gridDim.x;
    const bf16* zr = z0 + row * p.vocab;
    const int64_t y = p.labels[row];
    const bool ignored = y == p.ignore_index;
    const bool in_range = y >= 0 && y < p.vocab;
    float zy = 0.f;
    if (tid == 0 && !ignored && in_range) zy = (float)zr[y];  // before any in-place write

    float m = -INFINITY, s = 0.f;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      if (tid + i * kXentRegThreads < nch) {
        float z[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) z[k] = (float)buf[i][k];
        accumulate<8>(z, m, s);
      }
    }
    // the gradient below converts the chunks afresh: fp32 copies kept from here would double
    // the registers the row occupies
#pragma unroll
    for (int i = 0; i < CPT; ++i) asm volatile("" : "+v"(buf[i]));
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const float m2 = __shfl_xor(m, off), s2 = __shfl_xor(s, off);
      combine(m, s, m2, s2);
    }
    const int rb = it & 1;  // the other buffer may still be read for the previous row
    if (lane == 0) {
      red_m[rb][w] = m;
      red_s[rb][w] = s;
    }
    __syncthreads();
    m = red_m[rb][0];
    s = red_s[rb][0];
#pragma unroll
    for (int i = 1; i < NW; ++i) combine(m, s, red_m[rb][i], red_s[rb][i]);
    const float lse2 = m == -INFINITY ? -INFINITY : m + log2f(s);
    if (tid == 0) {
      if (p.lse != nullptr) p.lse[row] = lse2 * kLn2;
      p.loss[row] = ignored ? 0.f : (in_range ? lse2 * kLn2 - zy : NAN);
    }
    const bool grad = p.dlogits != nullptr;
    const __amdgpu_buffer_rsrc_t ws =
        rsrc_of(grad ? static_cast<bf16*>(p.dlogits) + row * p.vocab : static_cast<bf16*>(nullptr));
    const __amdgpu_buffer_rsrc_t rs_next = rsrc_of(z0 + (next < rows ? next : row) * p.vocab);
    const float g = ignored ? 0.f : p.grad_scale;
    const int64_t cy = in_range && !ignored ? y / 8 : -1;
    const int ky = (int)(y & 7);
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + i * kXentRegThreads;
      if (c < nch) {
        if (grad) {
          bf16x8 o;
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            float v = fast_exp2(fmaf((float)buf[i][k], kLog2e, -lse2)) * g;
            if (c == cy && k == ky) v -= g;
            o[k] = f2bf(v);
          }
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, o), ws, tid * 16,
                                                 i * kXentRegThreads * 16, 0);
        }
        // the same registers take this chunk of the next row (its read overlaps these writes)
        if (next < rows)
          buf[i] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(
                                                  rs_next, tid * 16, i * kXentRegThreads * 16, 0));
      }
    }
  }
}

}  // namespace

hipError_t launch_softmax_xent(int64_t rows, int64_t vocab, int dtype, const void* logits,
                               const int64_t* labels, int64_t ignore_index, float grad_scale,
                               float* loss, float* lse, void* dlogits, hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  XentParams p;
  p.logits = logits;
  p.labels = labels;
  p.dlogits = dlogits;
  p.loss = loss;
  p.lse = lse;
  p.vocab = vocab;
  p.ignore_index = ignore_index;
  p.grad_scale = grad_scale;
  const int esize = dtype == BS_BF16 ? 2 : 4;
  const int vw = 16 / esize;
  const bool aligned = reinterpret_cast<uintptr_t>(logits) % 16 == 0 &&
                       (dlogits == nullptr || reinterpret_cast<uintptr_t>(dlogits) % 16 == 0);
  const bool vec = aligned && vocab % vw == 0;
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess)
    hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  const dim3 grid((unsigned)(rows < cus ? rows : cus));  // persistent: one workgroup per CU
  const dim3 block(kXentThreads);
  // bf16 rows of 16K..128K entries: the register-resident form (one HBM read per element; 24
  // chunks per lane would spill under the 1024-lane register budget)
  if (dtype == BS_BF16 && vec && vocab > 16384 && vocab <= 8 * kXentRegThreads * 16) {
    const dim3 rblock(kXentRegThreads);
    const int64_t per = (vocab / 8 + kXentRegThreads - 1) / kXentRegThreads;  // chunks per lane
    if (per <= 4) hipLaunchKernelGGL(xent_reg_kernel<4>, grid, rblock, 0, stream, p, rows);
    else if (per <= 8) hipLaunchKernelGGL(xent_reg_kernel<8>, grid, rblock, 0, stream, p, rows);
    else hipLaunchKernelGGL(xent_reg_kernel<16>, grid, rblock, 0, stream, p, rows);
    return hipGetLastError();
  }
  if (dtype == BS_BF16) {
    if (vec) hipLaunchKernelGGL((xent_kernel<bf16, true>), grid, block, 0, stream, p, rows);
    else hipLaunchKernelGGL((xent_kernel<bf16, false>), grid, block, 0, stream, p, rows);
  } else {
    if (vec) hipLaunchKernelGGL((xent_kernel<float, true>), grid, block, 0, stream, p, rows);
    else hipLaunchKernelGGL((xent_kernel<float, false>), grid, block, 0, stream, p, rows);
  }
  return hipGetLastError();
}

}  // namespace bs
