// bf16 attention backward for gfx950 (recomputes P from the saved LSE).
//
// Two kernels, neither of which needs atomics:
//
// dq_bf16_kernel (query-major, walks the forward work list: 128-row query
//   tiles over 64-key tiles).  Like the forward it keeps one query per lane,
//   computing S^T = K Q^T and dP^T = V dO^T with Q and dO resident in
//   registers (B operands) and K, V tiles in LDS (A operands, row reads);
//   P = exp2(S*scale*log2e - LSE*log2e), dS = P (dP - D) are per-lane fp32
//   math; dQ^T += K^T dS^T takes dS^T straight from registers as the B operand
//   and K^T from the same K tile through transposing LDS reads
//   (ds_read_b64_tr_b16), which deliver the keys in the register order of dS^T.
//   dQ is finished in registers and written once (bf16), or added to a float32
//   accumulator for the context-parallel steps.
//
// dkdv_bf16_kernel (key-major, walks the backward work list: 128-key tiles
//   over 64-row query tiles).  8 waves, 2 per SIMD: wave w owns the 32-key
//   block w%4 of the tile and the query-row half w/4 of every query tile, and
//   accumulates dK, dV of its keys in registers over all query heads of the KV
//   group and all visible query tiles (MASKED diagonal tiles first):
//     S  = Q K^T,  dP = dO V^T     (A = Q, dO rows; B = K, V rows; all from LDS)
//     P, dS                         (lane = one key, 16 query rows)
//     dV^T += dO^T P,  dK^T += Q^T dS   (A = transposing reads of the same Q, dO
//                                       tiles; B = P, dS straight from registers)
//   K and V of the key tile stay in LDS (row-major, padded) for the whole item;
//   query tiles are XOR-swizzled (they are read both as rows and transposed)
//   and double-buffered: the next one is fetched into registers and written to
//   the other buffer while the current one is consumed, one barrier per tile.
//   At the end the two waves of each key block add their partial sums through
//   LDS.  Query rows past the segment use LSE = +inf (P = 0), rows whose LSE is
//   -inf (no visible key) also get P = 0.
//
// The dQ kernel copies its tiles from HBM straight into LDS
// (global_load_lds_dwordx4, no staging registers) into XOR-swizzled row-major
// tiles (conflict-free for row reads and transposing reads alike), double-
// buffered in distinct arrays: the copy of the next tile is issued before the
// current one is consumed and waited for after it, one barrier per tile.  (The
// dK/dV kernel keeps register staging: its accumulators leave no room for the
// per-buffer LDS addresses that the direct copies need.)  Rows past a segment
// are fetched from its last valid row and never contribute.
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
  bf16* dq;          // varlen: dQ written directly
  float* dq_acc;     // chunk: dQ added into a float32 accumulator (dq == nullptr)
  bf16* dk;
  bf16* dv;
  float* dk_acc;     // when set, dK and dV are added into float32 accumulators
  float* dv_acc;
  const WsHeader* hdr;
  const WorkItem* items;
  int64_t total_q;
  int32_t hq, hkv, group;
  int32_t causal;
  float scale, scale_log2;
};

__device__ __forceinline__ int spread_head(int slot, int n) {
  return (n & 7) == 0 ? (slot & 7) * (n >> 3) + (slot >> 3) : slot;
}

// ----------------------------------------------------------------------------- dQ
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

  const int item_idx = blockIdx.x / p.hq;
  if (item_idx >= p.hdr->n_items) return;
  const WorkItem it = p.items[item_idx];
  const int h = spread_head(blockIdx.x % p.hq, p.hq);
  const int hk = h / p.group;

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, c = lane & 31, hh = lane >> 5;
  const int qrow = w * 32 + c;
  const bool qvalid = qrow < it.a_rows;
  const int64_t qstride = (int64_t)p.hq * D;
  const int kvstride = p.hkv * D;
  const int64_t qoff = (int64_t)(it.a_start + (qvalid ? qrow : 0)) * qstride + (int64_t)h * D;

  bf16x8 qf[KK], dof[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    qf[kk] = *reinterpret_cast<const bf16x8*>(p.q + qoff + kk * 16 + hh * 8);
    dof[kk] = *reinterpret_cast<const bf16x8*>(p.dout + qoff + kk * 16 + hh * 8);
  }
  float lse2 = INFINITY, dval = 0.f;
  if (qvalid) {
    const float l = p.lse[(int64_t)h * p.total_q + it.a_start + qrow];
    lse2 = l == -INFINITY ? INFINITY : l * kLog2e;
    dval = p.dvec[(int64_t)h * p.total_q + it.a_start + qrow];
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

  if (n_tiles > 0) copy_tile(0, K0, V0);
  wait_vmem_all();  // Q, dO fragments and tile 0
  __syncthreads();

  auto step = [&](int t, const bf16* Kb, const bf16* Vb, bf16* Kn, bf16* Vn) {
    if (t + 1 < n_tiles) copy_tile(t + 1, Kn, Vn);
    __builtin_amdgcn_sched_barrier(0);  // issue the copy before the reads below

    f32x16 sacc[2] = {f32x16{}, f32x16{}};
    f32x16 dpacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int off = swz_off<D>(kb * 32 + c, kk * 2 + hh);
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&Kb[off]);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], sacc[kb], 0, 0, 0);
        const bf16x8 b = *reinterpret_cast<const bf16x8*>(&Vb[off]);
        dpacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, dof[kk], dpacc[kb], 0, 0, 0);
      }
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
        const bf16x8 a = lds_read_tr2(Kb + swz_tr_off<D>(ks * 16, db * 32, 0, lane),
                                      Kb + swz_tr_off<D>(ks * 16, db * 32, 1, lane));
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

// --------------------------------------------------------------------------- dK, dV
template <int D>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void dkdv_bf16_kernel(const BwdParams p) {
  constexpr int BM = kBwdBM, BN = kBwdBN;
  constexpr int KK = D / 16, DB = D / 32;
  constexpr int NSTR = D + 8;                 // K, V row-major tiles (padded)
  constexpr int QTILE = BM * D;               // Q, dO tiles: swizzled (read both ways)
  constexpr int KTILE = BN * NSTR;
  constexpr int NT = 512;
  constexpr int QUNITS = BM * D / 8 / NT;     // 16-byte loads per thread per Q/dO tile
  constexpr int KUNITS = BN * D / 8 / NT;     // 16-byte loads per thread per K/V tile
  static_assert(BM == 64 && BN == 128 && QUNITS >= 1, "tile shape");
  // LDS: K, V of the key tile (resident), Q and dO query tiles (double-buffered),
  // LSE / D rows.  After the loop the same space holds the partial dK, dV of
  // the waves that own the second half of each query tile.
  constexpr int KV_BYTES = 2 * KTILE * 2;
  constexpr int Q_BYTES = 2 * 2 * QTILE * 2;
  constexpr int ROW_BYTES = 2 * 2 * BM * 4;
  constexpr int RED_BYTES = 4 * 64 * 2 * DB * 16 * 4;
  constexpr int SMEM = (KV_BYTES + Q_BYTES + ROW_BYTES) > RED_BYTES ? (KV_BYTES + Q_BYTES + ROW_BYTES)
                                                                    : RED_BYTES;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  bf16* Ks = reinterpret_cast<bf16*>(smem);
  bf16* Vs = Ks + KTILE;
  bf16* Qs = Vs + KTILE;            // [2][QTILE]
  bf16* dOs = Qs + 2 * QTILE;       // [2][QTILE]
  float* lse_s = reinterpret_cast<float*>(dOs + 2 * QTILE);  // [2][BM]
  float* dvec_s = lse_s + 2 * BM;                            // [2][BM]

  const int item_idx = blockIdx.x / p.hkv;
  if (item_idx >= p.hdr->n_items) return;
  const WorkItem it = p.items[item_idx];
  const int hk = spread_head(blockIdx.x % p.hkv, p.hkv);

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, c = lane & 31, hh = lane >> 5;
  const int kbw = w & 3;           // this wave's 32-key block of the tile
  const int qh = w >> 2;           // this wave's 32-row half of every query tile
  const int64_t qstride = (int64_t)p.hq * D;
  const int kvstride = p.hkv * D;
  const int k_rows = it.a_rows;
  const int key_loc = kbw * 32 + c;
  const int key_rel = it.tile * BN + key_loc;   // key index inside its segment

  // K, V of the key tile, row-major (rows past the segment repeat its last key)
  {
    const bf16* kb = p.k + (int64_t)it.a_start * kvstride + (int64_t)hk * D;
    const bf16* vb = p.v + (int64_t)it.a_start * kvstride + (int64_t)hk * D;
#pragma unroll
    for (int u = 0; u < KUNITS; ++u) {
      const int idx = u * NT + tid;
      const int row = idx / (D / 8), ch = idx % (D / 8);
      const int r = row < k_rows - 1 ? row : k_rows - 1;
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(kb + r * kvstride + ch * 8);
      const bf16x8 b = *reinterpret_cast<const bf16x8*>(vb + r * kvstride + ch * 8);
      *reinterpret_cast<bf16x8*>(&Ks[row * NSTR + ch * 8]) = a;
      *reinterpret_cast<bf16x8*>(&Vs[row * NSTR + ch * 8]) = b;
    }
  }

  f32x16 dvacc[DB], dkacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) { dvacc[db] = f32x16{}; dkacc[db] = f32x16{}; }

  const int q_len = it.b_len;
  const int qt_first = it.n0, n_masked = it.n1, n_vis = it.n2;
  const int diag = it.diag;
  const int n_iter = n_vis * p.group;

  bf16x8 rq[QUNITS], rd[QUNITS];
  float lse_r = INFINITY, dv_r = 0.f;
  auto load_tile = [&](int i) {
    const int hg = i / n_vis, j = i - hg * n_vis;
    const int h = hk * p.group + hg;
    const int q_rel0 = (qt_first + j) * BM;
    const int64_t q_glob0 = (int64_t)it.b_start + q_rel0;
    const int last = q_len - 1 - q_rel0;
    const bf16* qp = p.q + q_glob0 * qstride + (int64_t)h * D;
    const bf16* dp = p.dout + q_glob0 * qstride + (int64_t)h * D;
#pragma unroll
    for (int u = 0; u < QUNITS; ++u) {
      const int idx = u * NT + tid;
      const int row = idx / (D / 8), ch = idx % (D / 8);
      const int64_t ro = (int64_t)(row < last ? row : last) * qstride + ch * 8;
      rq[u] = *reinterpret_cast<const bf16x8*>(qp + ro);
      rd[u] = *reinterpret_cast<const bf16x8*>(dp + ro);
    }
    if (tid < BM) {
      const bool ok = tid <= last;
      const int64_t li = (int64_t)h * p.total_q + q_glob0 + (ok ? tid : 0);
      const float l = p.lse[li];
      lse_r = (!ok || l == -INFINITY) ? INFINITY : l * kLog2e;
      dv_r = ok ? p.dvec[li] : 0.f;
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int u = 0; u < QUNITS; ++u) {
      const int idx = u * NT + tid;
      const int row = idx / (D / 8), ch = idx % (D / 8);
      *reinterpret_cast<bf16x8*>(&Qs[buf * QTILE + swz_off<D>(row, ch)]) = rq[u];
      *reinterpret_cast<bf16x8*>(&dOs[buf * QTILE + swz_off<D>(row, ch)]) = rd[u];
    }
    if (tid < BM) {
      lse_s[buf * BM + tid] = lse_r;
      dvec_s[buf * BM + tid] = dv_r;
    }
  };
  // per-lane LDS offsets: rows of this wave's query half, its key block, and the
  // transposing reads of the query half
  const int qrow0 = qh * 32;
  const int koff = key_loc * NSTR + hh * 8;

  if (n_iter > 0) {
    load_tile(0);
    store_tile(0);
    if (n_iter > 1) load_tile(1);
  }
  __syncthreads();

  for (int i = 0; i < n_iter; ++i) {
    const int buf = i & 1;
    const int hg = i / n_vis, j = i - hg * n_vis;
    const int q_rel0 = (qt_first + j) * BM;
    const bool masked = j < n_masked;
    const bf16* Qb = Qs + buf * QTILE;
    const bf16* dOb = dOs + buf * QTILE;

    f32x16 sacc = f32x16{}, dpacc = f32x16{};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Ks[koff + kk * 16]);
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(&Qb[swz_off<D>(qrow0 + c, kk * 2 + hh)]);
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, kf, sacc, 0, 0, 0);
      const bf16x8 vf = *reinterpret_cast<const bf16x8*>(&Vs[koff + kk * 16]);
      const bf16x8 b = *reinterpret_cast<const bf16x8*>(&dOb[swz_off<D>(qrow0 + c, kk * 2 + hh)]);
      dpacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, vf, dpacc, 0, 0, 0);
    }

    bf16x8 pb[2], dsb[2];
    // lane = key key_loc, rows q = qrow0 + a4*8 + hh*4 + e
    const int vis_lim = key_rel - diag - q_rel0 - hh * 4;  // visible iff row >= vis_lim
#pragma unroll
    for (int a4 = 0; a4 < 4; ++a4) {
      const int ql = qrow0 + a4 * 8 + hh * 4;
      const f32x4 l4 = *reinterpret_cast<const f32x4*>(&lse_s[buf * BM + ql]);
      const f32x4 d4 = *reinterpret_cast<const f32x4*>(&dvec_s[buf * BM + ql]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = a4 * 4 + e;
        float pr = fast_exp2(fmaf(sacc[r], p.scale_log2, -l4[e]));
        if (masked && p.causal) pr = (qrow0 + a4 * 8 + e) >= vis_lim ? pr : 0.f;
        pb[r >> 3][r & 7] = f2bf(pr);
        dsb[r >> 3][r & 7] = f2bf(pr * (dpacc[r] - d4[e]));
      }
    }

#pragma unroll
    for (int qs = 0; qs < 2; ++qs) {
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int o0 = swz_tr_off<D>(qrow0 + qs * 16, db * 32, 0, lane);
        const int o1 = swz_tr_off<D>(qrow0 + qs * 16, db * 32, 1, lane);
        const bf16x8 a = lds_read_tr2(dOb + o0, dOb + o1);
        dvacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[qs], dvacc[db], 0, 0, 0);
        const bf16x8 b = lds_read_tr2(Qb + o0, Qb + o1);
        dkacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, dsb[qs], dkacc[db], 0, 0, 0);
      }
    }

    if (i + 1 < n_iter) {
      store_tile(buf ^ 1);  // buffer buf^1 was last read in iteration i-1
      if (i + 2 < n_iter) load_tile(i + 2);
    }
    __syncthreads();
  }

  // sum the two query halves: waves 4..7 hand their partials to waves 0..3
  // [kbw][2*DB*4 vectors][lane]: lane-minor, so a wave's accesses are contiguous
  f32x4* red = reinterpret_cast<f32x4*>(smem) + kbw * (2 * DB * 4) * 64 + lane;
  if (qh == 1) {
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        red[(db * 4 + a) * 64] =
            f32x4{dvacc[db][a * 4], dvacc[db][a * 4 + 1], dvacc[db][a * 4 + 2], dvacc[db][a * 4 + 3]};
        red[((DB + db) * 4 + a) * 64] =
            f32x4{dkacc[db][a * 4], dkacc[db][a * 4 + 1], dkacc[db][a * 4 + 2], dkacc[db][a * 4 + 3]};
      }
  }
  __syncthreads();
  if (qh == 0 && key_loc < k_rows) {
    const int64_t off = (int64_t)(it.a_start + key_loc) * kvstride + (int64_t)hk * D + hh * 4;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const f32x4 ov = red[(db * 4 + a) * 64];
        const f32x4 ok = red[((DB + db) * 4 + a) * 64];
        f32x4 gk, gv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          gk[e] = (dkacc[db][a * 4 + e] + ok[e]) * p.scale;
          gv[e] = dvacc[db][a * 4 + e] + ov[e];
        }
        const int col = db * 32 + a * 8;
        if (p.dk_acc != nullptr) {  // add into float32 accumulators
          f32x4* dk4 = reinterpret_cast<f32x4*>(p.dk_acc + off + col);
          f32x4* dv4 = reinterpret_cast<f32x4*>(p.dv_acc + off + col);
          *dk4 = *dk4 + gk;
          *dv4 = *dv4 + gv;
        } else {
          const bf16x4 xk = {f2bf(gk[0]), f2bf(gk[1]), f2bf(gk[2]), f2bf(gk[3])};
          const bf16x4 xv = {f2bf(gv[0]), f2bf(gv[1]), f2bf(gv[2]), f2bf(gv[3])};
          *reinterpret_cast<bf16x4*>(p.dk + off + col) = xk;
          *reinterpret_cast<bf16x4*>(p.dv + off + col) = xv;
        }
      }
    }
  }
}

BwdParams make_params(const bs_dims& dims, const void* q, const void* k, const void* v,
                      const void* dout, const float* lse, const float* dvec, int causal,
                      float scale, const void* ws, const WsLayout& L) {
  BwdParams p = {};
  p.q = static_cast<const bf16*>(q);
  p.k = static_cast<const bf16*>(k);
  p.v = static_cast<const bf16*>(v);
  p.dout = static_cast<const bf16*>(dout);
  p.lse = lse;
  p.dvec = dvec;
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

hipError_t launch_dq_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                          const void* dout, const float* lse, const float* dvec, int causal,
                          float scale, void* dq, float* dq_acc, const void* ws, const WsLayout& L,
                          hipStream_t stream) {
  if (L.max_items == 0 || dims.hq == 0) return hipSuccess;
  BwdParams p = make_params(dims, q, k, v, dout, lse, dvec, causal, scale, ws, L);
  p.dq = static_cast<bf16*>(dq);
  p.dq_acc = dq_acc;
  const dim3 grid((unsigned)(L.max_items * dims.hq));
  if (dims.head_dim == 128)
    hipLaunchKernelGGL(dq_bf16_kernel<128>, grid, dim3(256), 0, stream, p);
  else
    hipLaunchKernelGGL(dq_bf16_kernel<64>, grid, dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_dkdv_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                            const void* dout, const float* lse, const float* dvec, int causal,
                            float scale, void* dk, void* dv, int kv_accumulate, const void* ws,
                            const WsLayout& L, hipStream_t stream) {
  if (L.max_items == 0 || dims.hkv == 0) return hipSuccess;
  BwdParams p = make_params(dims, q, k, v, dout, lse, dvec, causal, scale, ws, L);
  if (kv_accumulate) {
    p.dk_acc = static_cast<float*>(dk);
    p.dv_acc = static_cast<float*>(dv);
  } else {
    p.dk = static_cast<bf16*>(dk);
    p.dv = static_cast<bf16*>(dv);
  }
  const dim3 grid((unsigned)(L.max_items * dims.hkv));
  if (dims.head_dim == 128)
    hipLaunchKernelGGL(dkdv_bf16_kernel<128>, grid, dim3(512), 0, stream, p);
  else
    hipLaunchKernelGGL(dkdv_bf16_kernel<64>, grid, dim3(512), 0, stream, p);
  return hipGetLastError();
}

}  // namespace bs
