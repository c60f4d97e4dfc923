// bf16 attention forward for gfx950: tiled online softmax on MFMA.
//
// One workgroup = one query tile of the work list (kFwdBM = 128 rows) for one
// query head (which ones, and how the XCDs share them: block_work in attn.hpp);
// 4 waves, each owning 32 query rows.  The key loop walks the
// tile's visible key tiles (kFwdBN = 64 keys): the FULL ones first without any
// score mask, then the MASKED ones (causal diagonal / ragged key tail).
//
// Orientation.  The 32x32x16 bf16 MFMA leaves lane l holding column l%32 of its
// 32x32 result and 16 of the 32 rows.  The kernel therefore computes the
// transposed scores S^T = K Q^T, so that every lane owns ONE query (column) and
// 32 of the 64 keys of the tile: the softmax row max / row sum is a reduction
// over the lane's own registers plus one exchange with lane l^32, and the
// output O^T = V^T P^T lands in the same "one query per lane" layout, so the
// online-softmax rescale of O is a per-lane multiply.  P^T is fed back to the
// MFMA straight from registers as the B operand; V^T comes from transposing LDS
// reads (ds_read_b64_tr_b16), which hand out the keys in exactly the order in
// which the P^T registers hold them.
//
// Pipeline.  K and V tiles are copied from HBM straight into LDS
// (buffer_load_dwordx4 ... lds, no staging registers), into row-major tiles whose
// 16-byte chunks are XOR-swizzled so that both the row reads of K and the
// transposing reads of V are free of bank conflicts.  Both are double-buffered:
// the copy of tile t+1 is issued while tile t is consumed, its instructions placed
// one after each pair of score products (issued back to back at the top of the
// step, every wave's copies queue behind one another), and waited for after it, one
// barrier per key tile.  The last tile copies itself again into the idle buffer, so
// that the copy needs no branch.  Key rows past the segment are copied from the
// last valid row and removed by the score mask, which every ragged tile has.
//
// Softmax.  Scores stay raw; the scale is folded into one FMA,
// p = exp2(s * scale*log2(e) - m).  The running max m is only raised when a
// tile's max exceeds it by more than 2^8 (in the exponent), so the O rescale
// is skipped on almost every tile; p then stays below 2^8, which neither the
// bf16 P nor the fp32 sums mind, and O = acc / l, LSE = (m + log2 l) ln 2 use
// the same m.
#include "attn.hpp"

namespace bs {
namespace {

struct FwdParams {
  const bf16* q;
  const bf16* k;
  const bf16* v;
  bf16* o;
  float* lse;
  float* o_run;    // running-merge mode (non-null): float32 running output
  float* lse_run;  // and its running LSE
  int32_t accumulate;
  const WsHeader* hdr;
  const WorkItem* items;
  int64_t total_q;
  int32_t hq, hkv, group;
  int32_t causal;
  float scale_log2;  // scale * log2(e)
};

constexpr float kRescaleThreshold = 8.0f;  // log2 units

template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void fwd_bf16_kernel(const FwdParams p) {
  constexpr int BM = kFwdBM, BN = kFwdBN;
  constexpr int TILE = BN * D;      // swizzled [BN][D] tile
  constexpr int KK = D / 16;        // MFMA k-steps over head_dim
  constexpr int DB = D / 32;        // 32-wide blocks of head_dim
  static_assert(BM == 128 && BN == 64, "tile shape");

  // two buffers as distinct arrays, so that the compiler can tell the copy into one
  // from the reads of the other and does not wait for the copy before reading
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

  // Q fragment of this lane's query row, B operand of S^T = K Q^T
  bf16x8 qf[KK];
  {
    const bf16* qp = p.q + (int64_t)(it.a_start + (qvalid ? qrow : 0)) * qstride + (int64_t)h * D + hh * 8;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) qf[kk] = *reinterpret_cast<const bf16x8*>(qp + kk * 16);
  }

  const bf16* kbase = p.k + (int64_t)it.b_start * kvstride + (int64_t)hk * D;
  const bf16* vbase = p.v + (int64_t)it.b_start * kvstride + (int64_t)hk * D;
  const int k_len = it.b_len;
  const int n_tiles = it.n1, n_full = it.n0;

  auto copy_tile = [&](int t, bf16* Kd, bf16* Vd) {
    const int k0 = t * BN;
    const int last = k_len - 1 - k0;  // last valid row inside the tile (>= 0)
    dma_tile<D, BN, 4>(Kd, kbase + (int64_t)k0 * kvstride, kvstride, last, w, lane);
    dma_tile<D, BN, 4>(Vd, vbase + (int64_t)k0 * kvstride, kvstride, last, w, lane);
  };

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
  float m2 = -INFINITY;  // running max, log2 domain
  float l_run = 0.f;     // this lane's partial row sum (its 32 keys of every tile)
  const float c2 = p.scale_log2;
  // keys of tile t visible to this lane's query: local index < lim_base - t*BN
  const int q_rel = it.tile * BM + qrow;
  int lim_base = k_len;
  if (p.causal) lim_base = min(k_len, q_rel + it.diag + 1);
  lim_base -= hh * 4;  // fold the lane-half offset of the key index

  if (n_tiles > 0) copy_tile(0, K0, V0);
  wait_vmem_all();  // Q fragment and tile 0
  __syncthreads();

  // one key tile: consume (Kb, Vb) while tile t+1 is copied into (Kn, Vn), which
  // were last read one tile earlier, before the barrier that ended it
  auto step = [&](int t, const bf16* Kb, const bf16* Vb, bf16* Kn, bf16* Vn) {
    copy_tile(min(t + 1, n_tiles - 1), Kn, Vn);

    f32x16 sacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&Kb[swz_off<D>(kb * 32 + c, kk * 2 + hh)]);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], sacc[kb], 0, 0, 0);
      }
    }
    // K reads two contraction steps ahead of the products, one copy instruction after
    // each pair of products
    __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 4, 0);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, 2, 0);
      __builtin_amdgcn_sched_group_barrier(kSchedVmem, 1, 0);
      if (kk + 2 < KK) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
    }

    // mask (MASKED tiles only): key local index kb*32 + (r/4)*8 + hh*4 + r%4
    if (t >= n_full) {
      const int lim = lim_base - t * BN;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sacc[kb][r] = (kb * 32 + (r >> 2) * 8 + (r & 3)) < lim ? sacc[kb][r] : -INFINITY;
    }
    float mx = sacc[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][r]);
    mx = half_max(mx) * c2;
    if (__any(mx > m2 + kRescaleThreshold)) {
      const float m_new = fmaxf(m2, mx);
      const float alpha = fast_exp2(m2 - (m_new == -INFINITY ? 0.f : m_new));
      m2 = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
    }
    const float base = m2 == -INFINITY ? 0.f : m2;
    bf16x8 pb[4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = fast_exp2(fmaf(sacc[kb][r], c2, -base));
        l_run += e;
        pb[kb * 2 + (r >> 3)][r & 7] = f2bf(e);
      }
    }

#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const bf16x8 a = lds_read_tr2(Vb + swz_tr_off<D>(ks * 16, db * 32, 0, lane),
                                      Vb + swz_tr_off<D>(ks * 16, db * 32, 1, lane));
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[ks], oacc[db], 0, 0, 0);
      }
    }

    wait_vmem_all();  // this wave's copies of tile t+1
    __syncthreads();  // everyone's copies landed; everyone is done with (Kb, Vb)
  };
  for (int t = 0; t < n_tiles; t += 2) {
    step(t, K0, V0, K1, V1);
    if (t + 1 < n_tiles) step(t + 1, K1, V1, K0, V0);
  }

  const float l_tot = half_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (!qvalid) return;
  const int64_t row = it.a_start + qrow;
  const int64_t oidx = row * qstride + (int64_t)h * D + hh * 4;  // this lane's first column
  const float lse2 = l_tot > 0.f ? m2 + log2f(l_tot) : -INFINITY;  // log2 domain
  if (p.o_run == nullptr) {
    bf16* op = p.o + oidx;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        bf16x4 x = {f2bf(oacc[db][a * 4 + 0] * inv), f2bf(oacc[db][a * 4 + 1] * inv),
                    f2bf(oacc[db][a * 4 + 2] * inv), f2bf(oacc[db][a * 4 + 3] * inv)};
        *reinterpret_cast<bf16x4*>(op + db * 32 + a * 8) = x;
      }
    }
    if (hh == 0) p.lse[(int64_t)h * p.total_q + row] = lse2 * kLn2;
    return;
  }
  // Running merge: weights exp(LSE_old - LSE_new) and exp(LSE_step - LSE_new), which sum
  // to one; a running LSE of -inf gives its O weight 0 without reading it.
  float* lr = p.lse_run + (int64_t)h * p.total_q + row;
  const float old2 = p.accumulate ? *lr * kLog2e : -INFINITY;
  const float mx = fmaxf(old2, lse2);
  float w_old = 0.f, w_new = 0.f, lse_m = -INFINITY;
  if (mx != -INFINITY) {
    const float eo = fast_exp2(old2 - mx), en = fast_exp2(lse2 - mx);
    const float rs = 1.f / (eo + en);
    w_old = eo * rs;
    w_new = en * rs * inv;
    lse_m = (mx + log2f(eo + en)) * kLn2;
  }
  float* orun = p.o_run + oidx;
#pragma unroll
  for (int db = 0; db < DB; ++db) {
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      f32x4 x = {oacc[db][a * 4 + 0] * w_new, oacc[db][a * 4 + 1] * w_new,
                 oacc[db][a * 4 + 2] * w_new, oacc[db][a * 4 + 3] * w_new};
      if (w_old != 0.f) {
        const f32x4 prev = *reinterpret_cast<const f32x4*>(orun + db * 32 + a * 8);
        x = prev * w_old + x;
      }
      if (p.o != nullptr)
        *reinterpret_cast<bf16x4*>(p.o + oidx + db * 32 + a * 8) =
            bf16x4{f2bf(x[0]), f2bf(x[1]), f2bf(x[2]), f2bf(x[3])};
      else
        *reinterpret_cast<f32x4*>(orun + db * 32 + a * 8) = x;
    }
  }
  if (hh == 0) *lr = lse_m;
}

}  // namespace

hipError_t launch_fwd_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                           int causal, float scale, void* out, float* lse,
                           const FwdMerge* merge, const void* ws, const WsLayout& L,
                           hipStream_t stream) {
  if (L.max_items == 0 || dims.hq == 0) return hipSuccess;
  FwdParams p;
  p.q = static_cast<const bf16*>(q);
  p.k = static_cast<const bf16*>(k);
  p.v = static_cast<const bf16*>(v);
  p.o = static_cast<bf16*>(out);
  p.lse = lse;
  p.o_run = merge ? merge->o_run : nullptr;
  p.lse_run = merge ? merge->lse_run : nullptr;
  p.accumulate = merge ? merge->accumulate : 0;
  p.hdr = static_cast<const WsHeader*>(ws);
  p.items = reinterpret_cast<const WorkItem*>(static_cast<const char*>(ws) + L.sorted);
  p.total_q = dims.total_q;
  p.hq = dims.hq;
  p.hkv = dims.hkv;
  p.group = dims.hq / dims.hkv;
  p.causal = causal;
  p.scale_log2 = scale * kLog2e;
  const dim3 grid((unsigned)(L.max_items * dims.hq));
  if (dims.head_dim == 128)
    hipLaunchKernelGGL(fwd_bf16_kernel<128>, grid, dim3(256), 0, stream, p);
  else
    hipLaunchKernelGGL(fwd_bf16_kernel<64>, grid, dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace bs
