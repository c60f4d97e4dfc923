// bf16 attention backward for gfx950, dK and dV (recomputes P from the saved LSE; no
// atomics).
//
// dkdv_bf16_kernel (key-major, walks the backward work list: 128-key tiles
//   over query tiles of 96 rows at head_dim 128, 64 at head_dim 64).  8 waves,
//   2 per SIMD, in pairs: both waves of
//   pair b own the 32-key block b of the tile, and split the work by role.
//     S wave  (holds K of its keys): S = Q K^T, P = exp2(S*c - LSE*log2e)
//                                    (lane = one key, the tile's query rows), hands the
//                                    bf16 P that feeds its own products to its
//                                    partner through LDS, and accumulates
//                                    dV^T += dO^T P.
//     dP wave (holds V of its keys): dP = dO V^T, then dP - D while the S wave
//                                    is still on its exponentials; dS = P (dP - D)
//                                    with that bf16 P, dK^T += Q^T dS.
//   Row operands (Q for S, dO for dP) are row reads of the query tiles, the
//   transposed ones (dO^T, Q^T) transposing LDS reads of the same tiles; P and
//   dS feed the MFMA straight from registers.  Each wave keeps only one of the
//   two fragments and one of the two accumulators, which leaves registers for
//   reading LDS operands several products ahead.  The S wave runs at raised
//   priority through its products, so that its exponentials overlap the dP
//   wave's products; the P hand-off is one LDS-only barrier per query tile,
//   at which the copy of the next tile stays in flight.  dK, dV of every key are
//   accumulated over all query heads of the KV group and all visible query
//   tiles and written once.  With one query head per KV head the query tiles
//   are walked from the diagonal (MASKED tiles first) to the end of the segment.
//   With a group of several, from the last tile of the segment down to the
//   diagonal, the heads of the group innermost: the workgroups of one segment's
//   key tiles for one KV head that run together on an XCD then read the same
//   query tile of the same head at about the same time, once from HBM into that
//   XCD's L2; walked upwards, each starts at its own diagonal, and its head
//   changes at its own time.  Which key tile and KV head a workgroup takes, and
//   how the XCDs share them, is block_work's (attn.hpp).
//   Query rows past the segment use LSE = +inf (P = 0), rows whose LSE is
//   -inf (no visible key) also get P = 0.
//
// The kernel copies its tiles from HBM straight into LDS (buffer_load ... lds, no
// staging registers) into XOR-swizzled row-major tiles (conflict-free for row reads and
// transposing reads alike), double-buffered in distinct arrays: the copy of the next tile
// is issued before the current one is consumed and waited for after it, one full barrier
// per tile.  Rows past a segment are fetched from its last valid row and never contribute.
#include <type_traits>

#include "bwd_common.hpp"

namespace bs {
namespace {

template <int D, bool kGroupOrder>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void dkdv_bf16_kernel(const BwdParams p) {
  constexpr int BM = bwd_bm(D), BN = kBwdBN;
  constexpr int KK = D / 16, DB = D / 32;
  constexpr int MB = BM / 32;                 // 32-row blocks of a query tile
  constexpr int QS = BM / 16;                 // 16-row contraction steps of a query tile
  constexpr int QTILE = BM * D;               // swizzled [BM][D] query tile
  constexpr int NW = 8;
  static_assert((BM == 64 || BM == 96) && BN == 128, "tile shape");
  // Q and dO tiles, double-buffered; each buffer is its own array (Q tile, then
  // dO tile), so that the compiler can tell the copy into one from the reads of
  // the other
  __shared__ __attribute__((aligned(16))) bf16 QD0[2 * QTILE];
  __shared__ __attribute__((aligned(16))) bf16 QD1[2 * QTILE];
  // LSE (log2 units) then D rows of the query tile, double-buffered
  __shared__ __attribute__((aligned(16))) float R0[2 * BM];
  __shared__ __attribute__((aligned(16))) float R1[2 * BM];
  // bf16 P handed from the S wave to the dP wave of each key block: [block][step][lane]
  __shared__ __attribute__((aligned(16))) bf16x8 Ps[4 * QS * 64];

  WorkItem it;
  int hk;  // KV head; each reads the Q/dO stream of its own query heads
  if (!block_work(p.hdr, p.items, p.hkv, 1, kHeadMajorRowsDkdv, it, hk)) return;

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, c = lane & 31, hh = lane >> 5;
  const int kb = w & 3;     // this wave's 32-key block of the tile
  const int role = w >> 2;  // 0: S, P, dV (holds K)    1: dP, dS, dK (holds V)
  const int64_t qstride = (int64_t)p.hq * D;
  const int kvstride = p.hkv * D;
  const int k_rows = it.a_rows;
  const int key_loc = kb * 32 + c;
  const bool kvalid = key_loc < k_rows;
  const int key_rel = it.tile * BN + key_loc;   // key index inside its segment

  // this lane's K row (role 0) or V row (role 1): B operand of S = Q K^T, dP = dO V^T
  bf16x8 frag[KK];
  {
    const bf16* src = role == 0 ? p.k : p.v;
    const bf16* rp = src + (int64_t)(it.a_start + (kvalid ? key_loc : 0)) * kvstride +
                     (int64_t)hk * D + hh * 8;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) frag[kk] = *reinterpret_cast<const bf16x8*>(rp + kk * 16);
  }
  // dV^T (role 0) or unscaled dK^T (role 1) of this lane's key: column c, rows d
  f32x16 acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x16{};

  const int q_len = it.b_len;
  const int qt_first = it.n0, n_masked = it.n1, n_vis = it.n2;
  const int diag = it.diag;
  const int n_iter = n_vis * p.group;
  // step i: query tile j (relative to qt_first) of query head hg of the group
  auto tile_of = [&](int i, int& hg, int& j) {
    if constexpr (kGroupOrder) {  // last tile first, heads innermost
      const int s = i / p.group;
      hg = i - s * p.group;
      j = n_vis - 1 - s;
    } else {                      // diagonal first, heads outermost
      hg = i / n_vis;
      j = i - hg * n_vis;
    }
  };

  // All eight waves copy query tile i (head, rows) into QDd; the first S wave fetches its
  // LSE rows, the second its D rows, and the S waves store them at the end of the step,
  // where they wait for the dP waves anyway (the other waves load a row too, unused, so
  // that the copy has no branch and can be scheduled among the products).
  const int ct = tid;  // thread index among the role-0 waves
  float row_r = 0.f;   // raw LSE / D value of one row (converted when stored)
  bool row_ok = false;  // the row lies inside the segment
  auto copy_tile = [&](int i, bf16* QDd) {
    int hg, j;
    tile_of(i, hg, j);
    const int h = hk * p.group + hg;
    const int q_rel0 = (qt_first + j) * BM;
    const int64_t q_glob0 = (int64_t)it.b_start + q_rel0;
    const int last = q_len - 1 - q_rel0;
    const int64_t qo = q_glob0 * qstride + (int64_t)h * D;
    dma_tile<D, BM, NW>(QDd, p.q + qo, (int)qstride, last, w, lane);
    dma_tile<D, BM, NW>(QDd + QTILE, p.dout + qo, (int)qstride, last, w, lane);
    {
      const int r = ct % BM;
      row_ok = r <= last;
      const int64_t li = (int64_t)h * p.total_q + q_glob0 + (row_ok ? r : 0);
      row_r = (ct < BM ? p.lse : p.dvec)[li];
    }
  };
  // LSE rows in log2 units, +inf (P = 0) past the segment and where no key is visible
  auto store_rows = [&](float* Rd) {
    if (ct < BM)
      Rd[ct] = (!row_ok || row_r == -INFINITY) ? INFINITY : row_r * kLog2e;
    else if (ct < 2 * BM)
      Rd[ct] = row_ok ? row_r : 0.f;
  };

  if (n_iter > 0) copy_tile(0, QD0);
  wait_vmem_all();  // K / V row, tile 0 and its rows
  if (role == 0 && n_iter > 0) store_rows(R0);
  __syncthreads();

  // phase 1 reads rows of Q (role 0) or dO (role 1); phase 2 reads dO (role 0)
  // or Q (role 1) transposed
  const int base1 = role * QTILE, base2 = (1 - role) * QTILE;
  // lane bases of the row reads and the transposing reads (the XOR form of the swizzle)
  const int rbase = swz_row_base<D>(lane), tbase = swz_tr_base<D>(lane);
  bf16x8* pslot = Ps + kb * QS * 64 + lane;

  // one query tile: consume (QDb, Rb) while tile i+1 is copied into (QDn, Rn),
  // which were last read one tile earlier, before the barrier that ended it
  auto step = [&](int i, const bf16* QDb, const float* Rb, bf16* QDn, float* Rn) {
    int hg, j;
    tile_of(i, hg, j);
    const int q_rel0 = (qt_first + j) * BM;
    const bool masked = j < n_masked;
    const bf16* A1 = QDb + base1;
    const bf16* A2 = QDb + base2;

    // S = Q K^T (role 0) or dP = dO V^T (role 1): lane = key, rows q = mb*32 + (r/4)*8 + hh*4 + r%4
    // (the S wave goes first on the matrix unit, so that its exponentials overlap
    // the dP wave's products)
    if (role == 0) __builtin_amdgcn_s_setprio(1);
    // the copy of tile i+1 (the last step copies its own tile again, into the idle
    // buffer: no branch, so the copy instructions can go among the products below
    // instead of queueing behind one another at the top of the step)
    copy_tile(min(i + 1, n_iter - 1), QDn);
    f32x16 s[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) s[mb] = f32x16{};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const bf16x8 a = lds_row16(A1, (rbase ^ (kk << 5)) + mb * 64 * D);
        s[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, frag[kk], s[mb], 0, 0, 0);
      }
    }
    // keep the row reads two contraction steps ahead of the products, with one copy
    // instruction after each of the first product pairs
    __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2 * MB, 0);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, MB, 0);
      if (kk < 6) __builtin_amdgcn_sched_group_barrier(kSchedVmem, 1, 0);
      if (kk + 2 < KK) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, MB, 0);
    }

    // B operand of phase 2: P (role 0) or dS (role 1), 16-row step qs = mb*2 + r/8
    bf16x8 ob[QS];
    if (role == 0) {
      __builtin_amdgcn_s_setprio(0);
      // P = exp2(S * scale * log2(e) - LSE * log2(e)); on MASKED tiles of a causal
      // pass, rows above the diagonal (row < vis_lim) are zeroed
      auto softmax = [&](auto use_mask) {
        const int vis_lim = key_rel - diag - q_rel0 - hh * 4;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
          for (int a4 = 0; a4 < 4; ++a4) {
            const f32x4 l4 = *reinterpret_cast<const f32x4*>(&Rb[mb * 32 + a4 * 8 + hh * 4]);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int r = a4 * 4 + e;
              float pr = fast_exp2(fmaf(s[mb][r], p.scale_log2, -l4[e]));
              if (decltype(use_mask)::value) pr = (mb * 32 + a4 * 8 + e) >= vis_lim ? pr : 0.f;
              ob[mb * 2 + (r >> 3)][r & 7] = f2bf(pr);
            }
          }
        }
      };
      if (masked && p.causal)
        softmax(std::true_type{});
      else
        softmax(std::false_type{});
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) pslot[qs * 64] = ob[qs];  // the bf16 P that feeds dV
    }
    if (role == 1) {
      // dP - D while the S wave is still on its exponentials (kept before the barrier)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
          const f32x4 d4 = *reinterpret_cast<const f32x4*>(&Rb[BM + mb * 32 + a4 * 8 + hh * 4]);
#pragma unroll
          for (int e = 0; e < 4; ++e) s[mb][a4 * 4 + e] -= d4[e];
        }
        asm volatile("" : "+v"(s[mb]));
      }
    }
    barrier_lds();  // P of every key block is in LDS (the copies of tile i+1 stay in flight)
    if (role == 1) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const bf16x8 p0 = pslot[(mb * 2) * 64], p1 = pslot[(mb * 2 + 1) * 64];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pr = bf2f((r >> 3) == 0 ? p0[r & 7] : p1[r & 7]);
          ob[mb * 2 + (r >> 3)][r & 7] = f2bf(pr * s[mb][r]);
        }
      }
    }

    // dV^T += dO^T P (role 0) or dK^T += Q^T dS (role 1)
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) {
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const bf16x8 a = lds_tr16(A2, (tbase ^ (db << 6)) + qs * 32 * D,
                                  (tbase ^ ((db << 6) | 32)) + qs * 32 * D + 16 * D);
        acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, ob[qs], acc[db], 0, 0, 0);
      }
    }
    // keep the transposing reads three products ahead
    __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 6, 1);
#pragma unroll
    for (int m = 0; m < QS * DB; ++m) {
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 1);
      if (m + 3 < QS * DB) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 1);
    }
    wait_vmem_all();  // this wave's copies of tile i+1 and its rows
    if (role == 0 && i + 1 < n_iter) store_rows(Rn);
    __syncthreads();
  };
  for (int i = 0; i < n_iter; i += 2) {
    step(i, QD0, R0, QD1, R1);
    if (i + 1 < n_iter) step(i + 1, QD1, R1, QD0, R0);
  }

  if (kvalid) {
    const int64_t off = (int64_t)(it.a_start + key_loc) * kvstride + (int64_t)hk * D + hh * 4;
    const float mul = role == 0 ? 1.f : p.scale;
    float* gacc = role == 0 ? p.dv_acc : p.dk_acc;
    bf16* gout = role == 0 ? p.dv : p.dk;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        f32x4 g;
#pragma unroll
        for (int e = 0; e < 4; ++e) g[e] = acc[db][a * 4 + e] * mul;
        const int col = db * 32 + a * 8;
        if (gacc != nullptr) {  // add into float32 accumulators
          f32x4* dst = reinterpret_cast<f32x4*>(gacc + off + col);
          *dst = *dst + g;
        } else {
          const bf16x4 x = {f2bf(g[0]), f2bf(g[1]), f2bf(g[2]), f2bf(g[3])};
          *reinterpret_cast<bf16x4*>(gout + off + col) = x;
        }
      }
    }
  }
}


}  // namespace

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
  const bool group_order = p.group > 1;
  if (dims.head_dim == 128) {
    if (group_order)
      hipLaunchKernelGGL((dkdv_bf16_kernel<128, true>), grid, dim3(512), 0, stream, p);
    else
      hipLaunchKernelGGL((dkdv_bf16_kernel<128, false>), grid, dim3(512), 0, stream, p);
  } else {
    if (group_order)
      hipLaunchKernelGGL((dkdv_bf16_kernel<64, true>), grid, dim3(512), 0, stream, p);
    else
      hipLaunchKernelGGL((dkdv_bf16_kernel<64, false>), grid, dim3(512), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace bs
