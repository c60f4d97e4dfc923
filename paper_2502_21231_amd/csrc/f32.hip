// float32 attention kernels (forward, dQ, dK/dV) for full-precision checks.
//
// They walk the same planner work lists as the bf16 path (kF32BM x kF32BN
// tiles, FULL tiles without a mask, MASKED ones with it) but compute on the
// vector ALUs, one thread per query row (forward, dQ) or per key row (dK/dV),
// with the shared key (or query) tile staged in LDS.  Exact-order fp32 dot
// products, no MFMA: they exist so that float32 inputs are answered with
// float32 accuracy.
#include "attn.hpp"

namespace bs {
namespace {

struct F32Params {
  const float* q;
  const float* k;
  const float* v;
  const float* dout;
  const float* lse;
  const float* dvec;
  float* o;
  float* lse_out;
  float* o_run;    // forward running-merge mode (non-null): running output
  float* lse_run;  // and its running LSE
  int32_t accumulate;
  float* dq_acc;
  float* dk;
  float* dv;
  const WsHeader* hdr;
  const WorkItem* items;
  int64_t total_q;
  int32_t hq, hkv, group;
  int32_t causal;
  int32_t kv_accumulate;  // dK, dV added into (not written over) the outputs
  float scale, scale_log2;
};

constexpr int BM = kF32BM, BN = kF32BN;

// Stages rows [row0, row0 + BN) of a [*, heads, D] tensor (head `hd`) into LDS,
// zero-filling rows at or past `limit`.
template <int D>
__device__ __forceinline__ void stage_rows(float* dst, const float* src, int64_t row0, int valid,
                                           int64_t stride, int hd) {
  for (int u = threadIdx.x; u < BN * D / 4; u += blockDim.x) {
    const int r = u / (D / 4), c4 = u % (D / 4);
    f32x4 x = f32x4{};
    if (r < valid) x = *reinterpret_cast<const f32x4*>(src + (row0 + r) * stride + (int64_t)hd * D + c4 * 4);
    *reinterpret_cast<f32x4*>(dst + r * D + c4 * 4) = x;
  }
}

template <int D>
__global__ __launch_bounds__(BM) void fwd_f32_kernel(const F32Params p) {
  __shared__ __attribute__((aligned(16))) float Ks[BN * D];
  __shared__ __attribute__((aligned(16))) float Vs[BN * D];
  const int item_idx = blockIdx.x / p.hq;
  if (item_idx >= p.hdr->n_items) return;
  const WorkItem it = p.items[item_idx];
  const int h = blockIdx.x % p.hq, hk = h / p.group;
  const int r = threadIdx.x;
  const bool valid = r < it.a_rows;
  const int64_t qs = (int64_t)p.hq * D, ks = (int64_t)p.hkv * D;
  float qv[D], acc[D];
  const float* qp = p.q + (int64_t)(it.a_start + (valid ? r : 0)) * qs + (int64_t)h * D;
#pragma unroll
  for (int i = 0; i < D; ++i) { qv[i] = valid ? qp[i] : 0.f; acc[i] = 0.f; }
  float m = -INFINITY, l = 0.f;
  const int q_rel = it.tile * BM + r;
  for (int t = 0; t < it.n1; ++t) {
    __syncthreads();
    const int k0 = t * BN;
    const int nvalid = it.b_len - k0 < BN ? it.b_len - k0 : BN;
    stage_rows<D>(Ks, p.k, it.b_start + k0, nvalid, ks, hk);
    stage_rows<D>(Vs, p.v, it.b_start + k0, nvalid, ks, hk);
    __syncthreads();
    const bool masked = t >= it.n0;
    // score of key j of the tile in the base-2 domain (-inf when not visible)
    auto score = [&](int j) {
      float d = 0.f;
#pragma unroll
      for (int i = 0; i < D; ++i) d = fmaf(qv[i], Ks[j * D + i], d);
      d *= p.scale_log2;
      if (masked) {
        const int key = k0 + j;
        const bool vis = key < it.b_len && (!p.causal || key - q_rel <= it.diag);
        d = vis ? d : -INFINITY;
      }
      return d;
    };
    float mx = -INFINITY;
    for (int j = 0; j < BN; ++j) mx = fmaxf(mx, score(j));
    const float m_new = fmaxf(m, mx);
    const float base = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m - base);
    m = m_new;
    l *= alpha;
#pragma unroll
    for (int i = 0; i < D; ++i) acc[i] *= alpha;
    for (int j = 0; j < BN; ++j) {
      const float e = fast_exp2(score(j) - base);
      l += e;
#pragma unroll
      for (int i = 0; i < D; ++i) acc[i] = fmaf(e, Vs[j * D + i], acc[i]);
    }
  }
  if (!valid) return;
  const float inv = l > 0.f ? 1.f / l : 0.f;
  const int64_t row = it.a_start + r;
  const float lse2 = l > 0.f ? m + log2f(l) : -INFINITY;  // log2 domain
  if (p.o_run == nullptr) {
    float* op = p.o + row * qs + (int64_t)h * D;
#pragma unroll
    for (int i = 0; i < D; ++i) op[i] = acc[i] * inv;
    p.lse_out[(int64_t)h * p.total_q + row] = lse2 * kLn2;
    return;
  }
  // running merge: log-sum-exp weights of the running state and of this step
  float* lr = p.lse_run + (int64_t)h * p.total_q + row;
  const float old2 = p.accumulate ? *lr * kLog2e : -INFINITY;
  const float mx = fmaxf(old2, lse2);
  float w_old = 0.f, w_new = 0.f, lse_m = -INFINITY;
  if (mx != -INFINITY) {
    const float eo = fast_exp2(old2 - mx), en = fast_exp2(lse2 - mx);
    w_old = eo / (eo + en);
    w_new = en / (eo + en) * inv;
    lse_m = (mx + log2f(eo + en)) * kLn2;
  }
  float* orun = p.o_run + row * qs + (int64_t)h * D;
  float* dst = p.o != nullptr ? p.o + row * qs + (int64_t)h * D : orun;
#pragma unroll
  for (int i = 0; i < D; ++i) dst[i] = (w_old != 0.f ? orun[i] * w_old : 0.f) + acc[i] * w_new;
  *lr = lse_m;
}

// dQ row of one query: sum over visible keys of dS_ij k_j, dS = P (dO.v_j - D).
template <int D>
__global__ __launch_bounds__(BM) void bwd_dq_f32_kernel(const F32Params p) {
  __shared__ __attribute__((aligned(16))) float Ks[BN * D];
  __shared__ __attribute__((aligned(16))) float Vs[BN * D];
  const int item_idx = blockIdx.x / p.hq;
  if (item_idx >= p.hdr->n_items) return;
  const WorkItem it = p.items[item_idx];
  const int h = blockIdx.x % p.hq, hk = h / p.group;
  const int r = threadIdx.x;
  const bool valid = r < it.a_rows;
  const int64_t qs = (int64_t)p.hq * D, ks = (int64_t)p.hkv * D;
  const int64_t row = it.a_start + (valid ? r : 0);
  float qv[D], dov[D], acc[D];
#pragma unroll
  for (int i = 0; i < D; ++i) {
    qv[i] = valid ? p.q[row * qs + (int64_t)h * D + i] : 0.f;
    dov[i] = valid ? p.dout[row * qs + (int64_t)h * D + i] : 0.f;
    acc[i] = 0.f;
  }
  float lse2 = valid ? p.lse[(int64_t)h * p.total_q + row] : INFINITY;
  lse2 = lse2 == -INFINITY ? INFINITY : lse2 * kLog2e;
  const float dval = valid ? p.dvec[(int64_t)h * p.total_q + row] : 0.f;
  const int q_rel = it.tile * BM + r;
  for (int t = 0; t < it.n1; ++t) {
    __syncthreads();
    const int k0 = t * BN;
    const int nvalid = it.b_len - k0 < BN ? it.b_len - k0 : BN;
    stage_rows<D>(Ks, p.k, it.b_start + k0, nvalid, ks, hk);
    stage_rows<D>(Vs, p.v, it.b_start + k0, nvalid, ks, hk);
    __syncthreads();
    const bool masked = t >= it.n0;
    for (int j = 0; j < BN; ++j) {
      float s = 0.f, dp = 0.f;
#pragma unroll
      for (int i = 0; i < D; ++i) {
        s = fmaf(qv[i], Ks[j * D + i], s);
        dp = fmaf(dov[i], Vs[j * D + i], dp);
      }
      float pr = fast_exp2(s * p.scale_log2 - lse2);
      if (masked) {
        const int key = k0 + j;
        const bool vis = key < it.b_len && (!p.causal || key - q_rel <= it.diag);
        pr = vis ? pr : 0.f;
      }
      const float ds = pr * (dp - dval);
#pragma unroll
      for (int i = 0; i < D; ++i) acc[i] = fmaf(ds, Ks[j * D + i], acc[i]);
    }
  }
  if (valid) {
    float* dst = p.dq_acc + row * qs + (int64_t)h * D;
#pragma unroll
    for (int i = 0; i < D; ++i) dst[i] += acc[i] * p.scale;
  }
}

// dK, dV rows of one key, summed over the query heads of its group.
template <int D>
__global__ __launch_bounds__(BN) void bwd_dkdv_f32_kernel(const F32Params p) {
  __shared__ __attribute__((aligned(16))) float Qs[BM * D];
  __shared__ __attribute__((aligned(16))) float dOs[BM * D];
  __shared__ float ls[BM], dl[BM];
  const int item_idx = blockIdx.x / p.hkv;
  if (item_idx >= p.hdr->n_items) return;
  const WorkItem it = p.items[item_idx];
  const int hk = blockIdx.x % p.hkv;
  const int r = threadIdx.x;
  const bool valid = r < it.a_rows;
  const int64_t qs = (int64_t)p.hq * D, ks = (int64_t)p.hkv * D;
  const int64_t row = it.a_start + (valid ? r : 0);
  float kv[D], vv[D], dka[D], dva[D];
#pragma unroll
  for (int i = 0; i < D; ++i) {
    kv[i] = valid ? p.k[row * ks + (int64_t)hk * D + i] : 0.f;
    vv[i] = valid ? p.v[row * ks + (int64_t)hk * D + i] : 0.f;
    dka[i] = 0.f;
    dva[i] = 0.f;
  }
  const int key_rel = it.tile * BN + r;
  for (int hg = 0; hg < p.group; ++hg) {
    const int h = hk * p.group + hg;
    for (int jt = 0; jt < it.n2; ++jt) {
      const int qt = it.n0 + jt;
      const int q0 = qt * BM;
      const int nvalid = it.b_len - q0 < BM ? it.b_len - q0 : BM;
      __syncthreads();
      stage_rows<D>(Qs, p.q, it.b_start + q0, nvalid, qs, h);
      stage_rows<D>(dOs, p.dout, it.b_start + q0, nvalid, qs, h);
      if (r < BM) {
        float l = r < nvalid ? p.lse[(int64_t)h * p.total_q + it.b_start + q0 + r] : INFINITY;
        ls[r] = l == -INFINITY ? INFINITY : l * kLog2e;
        dl[r] = r < nvalid ? p.dvec[(int64_t)h * p.total_q + it.b_start + q0 + r] : 0.f;
      }
      __syncthreads();
      const bool masked = jt < it.n1;
      for (int i = 0; i < BM; ++i) {
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int x = 0; x < D; ++x) {
          s = fmaf(Qs[i * D + x], kv[x], s);
          dp = fmaf(dOs[i * D + x], vv[x], dp);
        }
        float pr = fast_exp2(s * p.scale_log2 - ls[i]);
        if (masked) {
          const bool vis = key_rel < it.tile * BN + it.a_rows && (!p.causal || key_rel - (q0 + i) <= it.diag);
          pr = vis ? pr : 0.f;
        }
        const float ds = pr * (dp - dl[i]);
#pragma unroll
        for (int x = 0; x < D; ++x) {
          dva[x] = fmaf(pr, dOs[i * D + x], dva[x]);
          dka[x] = fmaf(ds, Qs[i * D + x], dka[x]);
        }
      }
    }
  }
  if (valid) {
    float* dkp = p.dk + row * ks + (int64_t)hk * D;
    float* dvp = p.dv + row * ks + (int64_t)hk * D;
#pragma unroll
    for (int i = 0; i < D; ++i) {
      dkp[i] = (p.kv_accumulate ? dkp[i] : 0.f) + dka[i] * p.scale;
      dvp[i] = (p.kv_accumulate ? dvp[i] : 0.f) + dva[i];
    }
  }
}

F32Params make_params(const bs_dims& dims, const void* ws, const WsLayout& L, int causal,
                      float scale) {
  F32Params p = {};
  p.hdr = static_cast<const WsHeader*>(ws);
  p.items = reinterpret_cast<const WorkItem*>(static_cast<const char*>(ws) + L.sorted);
  p.total_q = dims.total_q;
  p.hq = dims.hq;
  p.hkv = dims.hkv;
  p.group = dims.hq / dims.hkv;
  p.causal = causal;
  p.scale = scale;
  p.scale_log2 = scale * kLog2e;
  return p;
}

}  // namespace

hipError_t launch_fwd_f32(const bs_dims& dims, const void* q, const void* k, const void* v,
                          int causal, float scale, void* out, float* lse, const FwdMerge* merge,
                          const void* ws, const WsLayout& L, hipStream_t stream) {
  if (L.max_items == 0 || dims.hq == 0) return hipSuccess;
  F32Params p = make_params(dims, ws, L, causal, scale);
  p.q = static_cast<const float*>(q);
  p.k = static_cast<const float*>(k);
  p.v = static_cast<const float*>(v);
  p.o = static_cast<float*>(out);
  p.lse_out = lse;
  p.o_run = merge ? merge->o_run : nullptr;
  p.lse_run = merge ? merge->lse_run : nullptr;
  p.accumulate = merge ? merge->accumulate : 0;
  const dim3 grid((unsigned)(L.max_items * dims.hq));
  if (dims.head_dim == 128) hipLaunchKernelGGL(fwd_f32_kernel<128>, grid, dim3(BM), 0, stream, p);
  else hipLaunchKernelGGL(fwd_f32_kernel<64>, grid, dim3(BM), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_bwd_f32_dq(const bs_dims& dims, const void* q, const void* k, const void* v,
                             const float* lse, const void* dout, const float* dvec, int causal,
                             float scale, float* dq_acc, const void* ws, const WsLayout& L,
                             hipStream_t stream) {
  if (L.max_items == 0 || dims.hq == 0) return hipSuccess;
  F32Params p = make_params(dims, ws, L, causal, scale);
  p.q = static_cast<const float*>(q);
  p.k = static_cast<const float*>(k);
  p.v = static_cast<const float*>(v);
  p.dout = static_cast<const float*>(dout);
  p.lse = lse;
  p.dvec = dvec;
  p.dq_acc = dq_acc;
  const dim3 grid((unsigned)(L.max_items * dims.hq));
  if (dims.head_dim == 128) hipLaunchKernelGGL(bwd_dq_f32_kernel<128>, grid, dim3(BM), 0, stream, p);
  else hipLaunchKernelGGL(bwd_dq_f32_kernel<64>, grid, dim3(BM), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_bwd_f32_dkdv(const bs_dims& dims, const void* q, const void* k, const void* v,
                               const float* lse, const void* dout, const float* dvec, int causal,
                               float scale, void* dk, void* dv, int kv_accumulate,
                               const void* ws, const WsLayout& L, hipStream_t stream) {
  if (L.max_items == 0 || dims.hkv == 0) return hipSuccess;
  F32Params p = make_params(dims, ws, L, causal, scale);
  p.kv_accumulate = kv_accumulate;
  p.q = static_cast<const float*>(q);
  p.k = static_cast<const float*>(k);
  p.v = static_cast<const float*>(v);
  p.dout = static_cast<const float*>(dout);
  p.lse = lse;
  p.dvec = dvec;
  p.dk = static_cast<float*>(dk);
  p.dv = static_cast<float*>(dv);
  const dim3 grid((unsigned)(L.max_items * dims.hkv));
  if (dims.head_dim == 128) hipLaunchKernelGGL(bwd_dkdv_f32_kernel<128>, grid, dim3(BN), 0, stream, p);
  else hipLaunchKernelGGL(bwd_dkdv_f32_kernel<64>, grid, dim3(BN), 0, stream, p);
  return hipGetLastError();
}

}  // namespace bs
