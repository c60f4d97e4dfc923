// bf16 attention backward for gfx950 (recomputes P from the saved LSE).
//
// One workgroup = one key tile of the backward work list (kBwdBN = 128 keys)
// for one KV head; 4 waves, wave w owning keys 32w .. 32w+31, whose K and V
// rows it keeps in registers and whose dK, dV it accumulates in registers over
// all query heads of the KV group and all visible query tiles (kBwdBM = 64
// rows), the MASKED (diagonal) query tiles first.  Per query tile:
//
//   S  = Q K^T            (MFMA, A = Q from LDS, B = K from registers)
//   dP = dO V^T           (MFMA, A = dO from LDS, B = V from registers)
//   P  = exp2(S*scale*log2e - LSE*log2e),  dS = P (dP - D)        (fp32)
//   dV^T += dO^T P        (A = dO^T from LDS, B = P straight from registers)
//   dK^T += Q^T dS        (A = Q^T from LDS,  B = dS straight from registers)
//   dQ  += dS K           (dS through LDS, K^T from LDS), fp32 atomics to HBM
//
// The MFMA result layout (lane = one column, 16 rows) lets P and dS serve as
// the B operand of the q-contractions directly; the matching permutation of the
// q index inside each 16-group is applied when Q^T and dO^T are written to LDS.
// Query rows past the segment load as zeros with LSE = +inf (P = 0); rows whose
// LSE is -inf (no visible key) also get P = 0.  Keys past the segment load as
// zeros, so they add nothing to dQ; their dK, dV are never stored.
#include "common.hpp"

namespace bs {
namespace {

struct BwdParams {
  const bf16* q;
  const bf16* k;
  const bf16* v;
  const bf16* dout;
  const float* lse;
  const float* dvec;
  float* dq_acc;
  bf16* dk;
  bf16* dv;
  const WsHeader* hdr;
  const WorkItem* items;
  int64_t total_q;
  int32_t hq, hkv, group;
  int32_t causal;
  float scale, scale_log2;
};

__device__ __forceinline__ int qperm4(int g4) { return (g4 == 1) ? 2 : (g4 == 2 ? 1 : g4); }

__device__ __forceinline__ int kvhead_of(int slot, int hkv) {
  return (hkv & 7) == 0 ? (slot & 7) * (hkv >> 3) + (slot >> 3) : slot;
}

template <int D>
__global__ __launch_bounds__(256) void bwd_bf16_kernel(const BwdParams p) {
  constexpr int BM = kBwdBM, BN = kBwdBN;
  constexpr int KK = D / 16, DB = D / 32;
  constexpr int NSTR = D + 8;      // row-major [row][d] tiles
  constexpr int TSTR = BM + 8;     // transposed [d][q] tiles
  constexpr int SSTR = BN + 8;     // dS [q][key]
  constexpr int KTSTR = BN + 8;    // K^T [d][key]
  constexpr int QUNITS = (BM / 4) * (D / 8);   // (4 rows x 8 dims) units per Q/dO tile
  constexpr int KUNITS = (BN / 4) * (D / 8);
  static_assert(BM == 64 && BN == 128, "tile shape");

  __shared__ __attribute__((aligned(16))) bf16 Qs[BM * NSTR];
  __shared__ __attribute__((aligned(16))) bf16 dOs[BM * NSTR];
  __shared__ __attribute__((aligned(16))) bf16 Qt[D * TSTR];
  __shared__ __attribute__((aligned(16))) bf16 dOt[D * TSTR];
  __shared__ __attribute__((aligned(16))) bf16 dSs[BM * SSTR];
  __shared__ __attribute__((aligned(16))) bf16 Kt[D * KTSTR];
  __shared__ __attribute__((aligned(16))) float lse_s[BM];
  __shared__ __attribute__((aligned(16))) float dvec_s[BM];

  const int item_idx = blockIdx.x / p.hkv;
  if (item_idx >= p.hdr->n_items) return;
  const WorkItem it = p.items[item_idx];
  const int hk = kvhead_of(blockIdx.x % p.hkv, p.hkv);

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, c = lane & 31, hh = lane >> 5;
  const int64_t qstride = (int64_t)p.hq * D;
  const int64_t kvstride = (int64_t)p.hkv * D;
  const int k_rows = it.a_rows;
  const int key_loc = w * 32 + c;                  // this lane's key inside the tile
  const bool kvalid = key_loc < k_rows;
  const int key_rel = it.tile * BN + key_loc;      // key index inside its segment
  const int k_len_seg = it.tile * BN + k_rows;     // keys before the end of this tile's segment part

  // this lane's K and V rows (B operands of S = Q K^T and dP = dO V^T)
  bf16x8 kf[KK], vf[KK];
  {
    const int64_t row = it.a_start + (kvalid ? key_loc : 0);
    const bf16* kp = p.k + row * kvstride + (int64_t)hk * D;
    const bf16* vp = p.v + row * kvstride + (int64_t)hk * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      bf16x8 a = *reinterpret_cast<const bf16x8*>(kp + kk * 16 + hh * 8);
      bf16x8 b = *reinterpret_cast<const bf16x8*>(vp + kk * 16 + hh * 8);
      kf[kk] = kvalid ? a : bf16x8{};
      vf[kk] = kvalid ? b : bf16x8{};
    }
  }
  // K^T of the whole tile in LDS (natural key order), B operand of dQ = dS K
  for (int u = tid; u < KUNITS; u += 256) {
    const int g = u % (BN / 4), ch = u / (BN / 4);
    bf16x8 r[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = g * 4 + i;
      const bool ok = row < k_rows;
      bf16x8 x = *reinterpret_cast<const bf16x8*>(p.k + (int64_t)(it.a_start + (ok ? row : 0)) * kvstride +
                                                  (int64_t)hk * D + ch * 8);
      r[i] = ok ? x : bf16x8{};
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      bf16x4 col = {r[0][e], r[1][e], r[2][e], r[3][e]};
      *reinterpret_cast<bf16x4*>(&Kt[(ch * 8 + e) * KTSTR + g * 4]) = col;
    }
  }

  f32x16 dvacc[DB], dkacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) { dvacc[db] = f32x16{}; dkacc[db] = f32x16{}; }

  const int q_len = it.b_len;
  const int qt_first = it.n0, n_masked = it.n1, n_vis = it.n2;
  const int diag = it.diag;
  // dQ block of this wave: query block qb_w, head-dim blocks dbw0 .. dbw0 + DBW - 1
  constexpr int DBW = DB / 2;
  const int qb_w = w & 1, dbw0 = (w >> 1) * DBW;

  for (int hg = 0; hg < p.group; ++hg) {
    const int h = hk * p.group + hg;
    for (int j = 0; j < n_vis; ++j) {
      const int qt = qt_first + j;
      const int q_rel0 = qt * BM;
      const int64_t q_glob0 = (int64_t)it.b_start + q_rel0;
      const bool masked = j < n_masked;

      __syncthreads();  // previous tile fully consumed
      // Q and dO tiles: row-major and transposed (q permuted in 16-groups)
      for (int u = tid; u < QUNITS; u += 256) {
        const int g = u / (D / 8), ch = u % (D / 8);
        bf16x8 rq[4], rd[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = g * 4 + i;
          const bool ok = q_rel0 + row < q_len;
          const int64_t off = (q_glob0 + (ok ? row : 0)) * qstride + (int64_t)h * D + ch * 8;
          bf16x8 a = *reinterpret_cast<const bf16x8*>(p.q + off);
          bf16x8 b = *reinterpret_cast<const bf16x8*>(p.dout + off);
          rq[i] = ok ? a : bf16x8{};
          rd[i] = ok ? b : bf16x8{};
          *reinterpret_cast<bf16x8*>(&Qs[row * NSTR + ch * 8]) = rq[i];
          *reinterpret_cast<bf16x8*>(&dOs[row * NSTR + ch * 8]) = rd[i];
        }
        const int pcol = (g >> 2) * 16 + qperm4(g & 3) * 4;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          bf16x4 cq = {rq[0][e], rq[1][e], rq[2][e], rq[3][e]};
          bf16x4 cd = {rd[0][e], rd[1][e], rd[2][e], rd[3][e]};
          *reinterpret_cast<bf16x4*>(&Qt[(ch * 8 + e) * TSTR + pcol]) = cq;
          *reinterpret_cast<bf16x4*>(&dOt[(ch * 8 + e) * TSTR + pcol]) = cd;
        }
      }
      if (tid < BM) {
        const bool ok = q_rel0 + tid < q_len;
        float l = ok ? p.lse[(int64_t)h * p.total_q + q_glob0 + tid] : INFINITY;
        lse_s[tid] = l == -INFINITY ? INFINITY : l * kLog2e;
        dvec_s[tid] = ok ? p.dvec[(int64_t)h * p.total_q + q_glob0 + tid] : 0.f;
      }
      __syncthreads();

      f32x16 sacc[2], dpacc[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        sacc[qb] = f32x16{};
        dpacc[qb] = f32x16{};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          bf16x8 a = *reinterpret_cast<const bf16x8*>(&Qs[(qb * 32 + c) * NSTR + kk * 16 + hh * 8]);
          sacc[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, kf[kk], sacc[qb], 0, 0, 0);
          bf16x8 b = *reinterpret_cast<const bf16x8*>(&dOs[(qb * 32 + c) * NSTR + kk * 16 + hh * 8]);
          dpacc[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, vf[kk], dpacc[qb], 0, 0, 0);
        }
      }

      bf16x8 pb[4], dsb[4];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
          const int ql = qb * 32 + a4 * 8 + hh * 4;  // 4 consecutive query rows
          const f32x4 l4 = *reinterpret_cast<const f32x4*>(&lse_s[ql]);
          const f32x4 d4 = *reinterpret_cast<const f32x4*>(&dvec_s[ql]);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int r = a4 * 4 + i;
            float pr = fast_exp2(sacc[qb][r] * p.scale_log2 - l4[i]);
            if (masked) {
              const int qrel = q_rel0 + ql + i;
              const bool vis = key_rel < k_len_seg && (!p.causal || key_rel - qrel <= diag);
              pr = vis ? pr : 0.f;
            }
            const float ds = pr * (dpacc[qb][r] - d4[i]);
            pb[qb * 2 + (r >> 3)][r & 7] = f2bf(pr);
            const bf16 dsh = f2bf(ds);
            dsb[qb * 2 + (r >> 3)][r & 7] = dsh;
            dSs[(ql + i) * SSTR + key_loc] = dsh;
          }
        }
      }

#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int qs = 0; qs < 4; ++qs) {
          bf16x8 a = *reinterpret_cast<const bf16x8*>(&dOt[(db * 32 + c) * TSTR + qs * 16 + hh * 8]);
          dvacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[qs], dvacc[db], 0, 0, 0);
          bf16x8 b = *reinterpret_cast<const bf16x8*>(&Qt[(db * 32 + c) * TSTR + qs * 16 + hh * 8]);
          dkacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, dsb[qs], dkacc[db], 0, 0, 0);
        }
      }
      __syncthreads();  // dS tile complete

      f32x16 dqacc[DBW];
#pragma unroll
      for (int i = 0; i < DBW; ++i) dqacc[i] = f32x16{};
#pragma unroll
      for (int kk = 0; kk < BN / 16; ++kk) {
        bf16x8 a = *reinterpret_cast<const bf16x8*>(&dSs[(qb_w * 32 + c) * SSTR + kk * 16 + hh * 8]);
#pragma unroll
        for (int i = 0; i < DBW; ++i) {
          bf16x8 b = *reinterpret_cast<const bf16x8*>(&Kt[((dbw0 + i) * 32 + c) * KTSTR + kk * 16 + hh * 8]);
          dqacc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, dqacc[i], 0, 0, 0);
        }
      }
#pragma unroll
      for (int i = 0; i < DBW; ++i) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int ql = qb_w * 32 + (r >> 2) * 8 + hh * 4 + (r & 3);
          if (q_rel0 + ql < q_len) {
            float* dst = p.dq_acc + (q_glob0 + ql) * qstride + (int64_t)h * D + (dbw0 + i) * 32 + c;
            unsafeAtomicAdd(dst, dqacc[i][r] * p.scale);
          }
        }
      }
    }
  }

  if (kvalid) {
    const int64_t row = it.a_start + key_loc;
    bf16* dkp = p.dk + row * kvstride + (int64_t)hk * D;
    bf16* dvp = p.dv + row * kvstride + (int64_t)hk * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        bf16x4 xk = {f2bf(dkacc[db][a * 4 + 0] * p.scale), f2bf(dkacc[db][a * 4 + 1] * p.scale),
                     f2bf(dkacc[db][a * 4 + 2] * p.scale), f2bf(dkacc[db][a * 4 + 3] * p.scale)};
        bf16x4 xv = {f2bf(dvacc[db][a * 4 + 0]), f2bf(dvacc[db][a * 4 + 1]),
                     f2bf(dvacc[db][a * 4 + 2]), f2bf(dvacc[db][a * 4 + 3])};
        *reinterpret_cast<bf16x4*>(dkp + db * 32 + a * 8 + hh * 4) = xk;
        *reinterpret_cast<bf16x4*>(dvp + db * 32 + a * 8 + hh * 4) = xv;
      }
    }
  }
}

}  // namespace

hipError_t launch_bwd_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                           const void* dout, const float* lse, const float* dvec, float* dq_acc,
                           int causal, float scale, void* dk, void* dv, const void* ws,
                           const WsLayout& L, hipStream_t stream) {
  if (L.max_items == 0 || dims.hkv == 0) return hipSuccess;
  BwdParams p;
  p.q = static_cast<const bf16*>(q);
  p.k = static_cast<const bf16*>(k);
  p.v = static_cast<const bf16*>(v);
  p.dout = static_cast<const bf16*>(dout);
  p.lse = lse;
  p.dvec = dvec;
  p.dq_acc = dq_acc;
  p.dk = static_cast<bf16*>(dk);
  p.dv = static_cast<bf16*>(dv);
  p.hdr = static_cast<const WsHeader*>(ws);
  p.items = reinterpret_cast<const WorkItem*>(static_cast<const char*>(ws) + L.sorted);
  p.total_q = dims.total_q;
  p.hq = dims.hq;
  p.hkv = dims.hkv;
  p.group = dims.hq / dims.hkv;
  p.causal = causal;
  p.scale = scale;
  p.scale_log2 = scale * kLog2e;
  const dim3 grid((unsigned)(L.max_items * dims.hkv));
  if (dims.head_dim == 128)
    hipLaunchKernelGGL(bwd_bf16_kernel<128>, grid, dim3(256), 0, stream, p);
  else
    hipLaunchKernelGGL(bwd_bf16_kernel<64>, grid, dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace bs
