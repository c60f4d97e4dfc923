// bf16 attention backward for gfx950, dQ (recomputes P from the saved LSE; no atomics).
//
// dq_bf16_kernel (query-major, walks the forward work list: 128-row query tiles over
// 64-key tiles).  Like the forward it keeps one query per lane, computing S^T = K Q^T and
// dP^T = V dO^T with Q and dO resident in registers (B operands) and K, V tiles in LDS
// (A operands, row reads); P = exp2(S*scale*log2e - LSE*log2e), dS = P (dP - D) are
// per-lane fp32 math; dQ^T += K^T dS^T takes dS^T straight from registers as the B operand
// and K^T from the same K tile through transposing LDS reads (ds_read_b64_tr_b16), which
// deliver the keys in the register order of dS^T.  dQ is finished in registers and written
// once (bf16), or added to a float32 accumulator for the context-parallel steps.  Its
// prologue also forms D = rowsum(dO * O) of its rows for the dK/dV kernel.
//
// The kernel copies its tiles from HBM straight into LDS (buffer_load ... lds, no
// staging registers) into XOR-swizzled row-major tiles (conflict-free for row reads and
// transposing reads alike), double-buffered in distinct arrays: the copy of the next tile
// is issued before the current one is consumed and waited for after it, one full barrier
// per tile.  Rows past a segment are fetched from its last valid row and never contribute.
//
// This file is compiled with the backend's max-ILP scheduling strategy (build.py), which
// schedules this kernel's loop about 2-3% faster than the default; the other kernels keep
// the default.
#include "bwd_common.hpp"

namespace bs {
namespace {

template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void dq_bf16_kernel(const BwdParams p) {
  constexpr int BM = kFwdBM, BN = kFwdBN;
  constexpr int TILE = BN * D;   // swizzled [BN][D]
  constexpr int KK = D / 16, DB = D / 32;
  static_assert(BM == 128 && BN == 64, "tile shape");

  __shared__ __attribute__((aligned(16))) bf16 K0[TILE];
  __shared__ __attribute__((aligned(16))) bf16 K1[TILE];
  __shared__ __attribute__((aligned(16))) bf16 V0[TILE];
  __shared__ __attribute__((aligned(16))) bf16 V1[TILE];

  WorkItem it;
  int h;  // query head; the query heads of one KV group share its K/V stream
  if (!block_work(p.hdr, p.items, p.hq, p.group, 0, it, h)) return;
  const int hk = h / p.group;

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, c = lane & 31, hh = lane >> 5;
  const int qrow = w * 32 + c;
  const bool qvalid = qrow < it.a_rows;
  const int64_t qstride = (int64_t)p.hq * D;
  const int kvstride = p.hkv * D;
  const int64_t qoff = (int64_t)(it.a_start + (qvalid ? qrow : 0)) * qstride + (int64_t)h * D;

  // Q and dO of this lane's row (its half of head_dim), and D = rowsum(dO * O) of the row
  // (the two lanes of a row each sum their half; the dK/dV kernel reads D from dvec_out)
  bf16x8 qf[KK], dof[KK];
  float dpart = 0.f;
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    qf[kk] = *reinterpret_cast<const bf16x8*>(p.q + qoff + kk * 16 + hh * 8);
    dof[kk] = *reinterpret_cast<const bf16x8*>(p.dout + qoff + kk * 16 + hh * 8);
    const bf16x8 ov = *reinterpret_cast<const bf16x8*>(p.o + qoff + kk * 16 + hh * 8);
#pragma unroll
    for (int i = 0; i < 8; ++i) dpart = fmaf(bf2f(dof[kk][i]), bf2f(ov[i]), dpart);
  }
  const float drow = half_sum(dpart);
  float lse2 = INFINITY, dval = 0.f;
  if (qvalid) {
    const int64_t ri = (int64_t)h * p.total_q + it.a_start + qrow;
    const float l = p.lse[ri];
    lse2 = l == -INFINITY ? INFINITY : l * kLog2e;
    dval = drow;
    if (hh == 0) p.dvec_out[ri] = drow;
  }

  const bf16* kbase = p.k + (int64_t)it.b_start * kvstride + (int64_t)hk * D;
  const bf16* vbase = p.v + (int64_t)it.b_start * kvstride + (int64_t)hk * D;
  const int k_len = it.b_len;
  const int n_tiles = it.n1, n_full = it.n0;

  auto copy_tile = [&](int t, bf16* Kd, bf16* Vd) {
    const int k0 = t * BN;
    const int last = k_len - 1 - k0;
    dma_tile<D, BN, 4>(Kd, kbase + (int64_t)k0 * kvstride, kvstride, last, w, lane);
    dma_tile<D, BN, 4>(Vd, vbase + (int64_t)k0 * kvstride, kvstride, last, w, lane);
  };

  f32x16 dqacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) dqacc[db] = f32x16{};
  const float c2 = p.scale_log2;
  const int q_rel = it.tile * BM + qrow;
  int lim_base = k_len;
  if (p.causal) lim_base = min(k_len, q_rel + it.diag + 1);
  lim_base -= hh * 4;

  // lane bases of the row reads of K and V and the transposing reads of K
  const int rbase = swz_row_base<D>(lane), tbase = swz_tr_base<D>(lane);
  if (n_tiles > 0) copy_tile(0, K0, V0);
  wait_vmem_all();  // Q, dO fragments and tile 0
  __syncthreads();

  auto step = [&](int t, const bf16* Kb, const bf16* Vb, bf16* Kn, bf16* Vn) {
    // copy of tile t+1, without a branch (the last tile copies itself again into the
    // idle buffer), one instruction after each group of score products
    copy_tile(min(t + 1, n_tiles - 1), Kn, Vn);

    f32x16 sacc[2] = {f32x16{}, f32x16{}};
    f32x16 dpacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int off = (rbase ^ (kk << 5)) + kb * 64 * D;
        const bf16x8 a = lds_row16(Kb, off);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], sacc[kb], 0, 0, 0);
        const bf16x8 b = lds_row16(Vb, off);
        dpacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, dof[kk], dpacc[kb], 0, 0, 0);
      }
    }
    // K and V reads one contraction step ahead of the products, one copy instruction
    // after each group of four products
    __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 4, 0);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, 4, 0);
      __builtin_amdgcn_sched_group_barrier(kSchedVmem, 1, 0);
      if (kk + 1 < KK) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 4, 0);
    }
    if (t >= n_full) {
      const int lim = lim_base - t * BN;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sacc[kb][r] = (kb * 32 + (r >> 2) * 8 + (r & 3)) < lim ? sacc[kb][r] : -INFINITY;
    }
    bf16x8 dsb[4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float pr = fast_exp2(fmaf(sacc[kb][r], c2, -lse2));
        dsb[kb * 2 + (r >> 3)][r & 7] = f2bf(pr * (dpacc[kb][r] - dval));
      }
    }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const bf16x8 a = lds_tr16(Kb, (tbase ^ (db << 6)) + ks * 32 * D,
                                  (tbase ^ ((db << 6) | 32)) + ks * 32 * D + 16 * D);
        dqacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, dsb[ks], dqacc[db], 0, 0, 0);
      }
    }
    wait_vmem_all();  // this wave's copies of tile t+1
    __syncthreads();
  };
  for (int t = 0; t < n_tiles; t += 2) {
    step(t, K0, V0, K1, V1);
    if (t + 1 < n_tiles) step(t + 1, K1, V1, K0, V0);
  }

  if (qvalid) {
    const int64_t off = (int64_t)(it.a_start + qrow) * qstride + (int64_t)h * D + hh * 4;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int col = db * 32 + a * 8;
        if (p.dq != nullptr) {
          bf16x4 x = {f2bf(dqacc[db][a * 4 + 0] * p.scale), f2bf(dqacc[db][a * 4 + 1] * p.scale),
                      f2bf(dqacc[db][a * 4 + 2] * p.scale), f2bf(dqacc[db][a * 4 + 3] * p.scale)};
          *reinterpret_cast<bf16x4*>(p.dq + off + col) = x;
        } else {
          f32x4* dst = reinterpret_cast<f32x4*>(p.dq_acc + off + col);
          f32x4 y = *dst;
#pragma unroll
          for (int i = 0; i < 4; ++i) y[i] += dqacc[db][a * 4 + i] * p.scale;
          *dst = y;
        }
      }
    }
  }
}


}  // namespace

hipError_t launch_dq_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                          const void* out, const void* dout, const float* lse, float* dvec,
                          int causal, float scale, void* dq, float* dq_acc, const void* ws,
                          const WsLayout& L, hipStream_t stream) {
  if (L.max_items == 0 || dims.hq == 0) return hipSuccess;
  BwdParams p = make_params(dims, q, k, v, dout, lse, dvec, causal, scale, ws, L);
  p.o = static_cast<const bf16*>(out);
  p.dvec_out = dvec;
  p.dq = static_cast<bf16*>(dq);
  p.dq_acc = dq_acc;
  const dim3 grid((unsigned)(L.max_items * dims.hq));
  if (dims.head_dim == 128)
    hipLaunchKernelGGL(dq_bf16_kernel<128>, grid, dim3(256), 0, stream, p);
  else
    hipLaunchKernelGGL(dq_bf16_kernel<64>, grid, dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace bs
