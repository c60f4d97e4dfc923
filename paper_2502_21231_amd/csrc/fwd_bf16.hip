// bf16 attention forward for gfx950: tiled online softmax on MFMA.
//
// One workgroup = one query tile of the work list (kFwdBM = 128 rows) for one
// query head; 4 waves, each owning 32 query rows.  The key loop walks the
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
// MFMA straight from registers as the B operand; the contraction index order
// that the register layout implies (within 16 keys: 0-3, 8-11 for lanes 0-31,
// 4-7, 12-15 for lanes 32-63) is matched by storing V^T in LDS with the keys of
// each 16-group permuted accordingly, so each A-operand read is one 16-byte
// LDS load.
//
// Pipeline.  K and V tiles are staged row-major in LDS ([key][d]; K padded by 8
// elements for the row reads of S^T = K Q^T, V by 32 for the transposing reads
// (ds_read_b64_tr_b16) that hand out V^T in the permuted key order of P^T),
// both double-buffered: while
// tile t is consumed from one buffer, tile t+1 (already in registers) is
// written to the other and tile t+2 is fetched from HBM, so there is one
// barrier per key tile.  Key rows past the segment are fetched from the last
// valid row (no zero-fill, so the global loads never have to be waited on
// early) and are removed by the score mask, which every ragged tile has.
//
// Softmax.  Scores stay raw; the scale is folded into one FMA,
// p = exp2(s * scale*log2(e) - m).  The running max m is only raised when a
// tile's max exceeds it by more than 2^8 (in the exponent), so the O rescale
// is skipped on almost every tile; p then stays below 2^8, which neither the
// bf16 P nor the fp32 sums mind, and O = acc / l, LSE = (m + log2 l) ln 2 use
// the same m.  All staging is row-contiguous 16-byte traffic (no bank conflicts).
#include "common.hpp"

namespace bs {
namespace {

struct FwdParams {
  const bf16* q;
  const bf16* k;
  const bf16* v;
  bf16* o;
  float* lse;
  const WsHeader* hdr;
  const WorkItem* items;
  int64_t total_q;
  int32_t hq, hkv, group;
  int32_t causal;
  float scale_log2;  // scale * log2(e)
};

constexpr float kRescaleThreshold = 8.0f;  // log2 units

// Query head handled by a block: heads are spread so that all blocks of one
// head (and of one KV group) fall on the same XCD when hq is a multiple of 8
// (blocks are dealt to the 8 XCDs round-robin by block index).
__device__ __forceinline__ int head_of(int slot, int hq) {
  return (hq & 7) == 0 ? (slot & 7) * (hq >> 3) + (slot >> 3) : slot;
}

template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void fwd_bf16_kernel(const FwdParams p) {
  constexpr int BM = kFwdBM, BN = kFwdBN;
  constexpr int KSTR = D + 8;       // K tile row stride (elements)
  constexpr int VSTR = D + 32;      // V tile row stride (transposing reads)
  constexpr int KK = D / 16;        // MFMA k-steps over head_dim
  constexpr int DB = D / 32;        // 32-wide blocks of head_dim
  constexpr int KUNITS = BN * D / 8 / 256;    // 16-byte K (and V) loads per thread
  static_assert(BM == 128 && BN == 64, "tile shape");
  static_assert(KUNITS >= 1, "K staging");

  __shared__ __attribute__((aligned(16))) bf16 Ks[2][BN * KSTR];
  __shared__ __attribute__((aligned(16))) bf16 Vs[2][BN * VSTR];

  const int item_idx = blockIdx.x / p.hq;
  if (item_idx >= p.hdr->n_items) return;
  const WorkItem it = p.items[item_idx];
  const int h = head_of(blockIdx.x % p.hq, p.hq);
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
    // Q must be resident before the key pipeline starts: otherwise the wait for it
    // is merged, on the loop back-edge, with the wait for the tile being prefetched
    wait_vmem_all();
  }

  const bf16* kbase = p.k + (int64_t)it.b_start * kvstride + (int64_t)hk * D;
  const bf16* vbase = p.v + (int64_t)it.b_start * kvstride + (int64_t)hk * D;
  const int k_len = it.b_len;
  const int n_tiles = it.n1, n_full = it.n0;

  bf16x8 kreg[KUNITS], vreg[KUNITS];
  auto load_tile = [&](int t) {
    const int k0 = t * BN;
    const int last = k_len - 1 - k0;  // last valid row inside the tile (>= 0)
    const bf16* kt = kbase + (int64_t)k0 * kvstride;
    const bf16* vt = vbase + (int64_t)k0 * kvstride;
#pragma unroll
    for (int i = 0; i < KUNITS; ++i) {
      const int idx = i * 256 + tid;
      const int row = idx / (D / 8), ch = idx % (D / 8);
      const int r = row < last ? row : last;
      kreg[i] = *reinterpret_cast<const bf16x8*>(kt + r * kvstride + ch * 8);
      vreg[i] = *reinterpret_cast<const bf16x8*>(vt + r * kvstride + ch * 8);
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KUNITS; ++i) {
      const int idx = i * 256 + tid;
      const int row = idx / (D / 8), ch = idx % (D / 8);
      *reinterpret_cast<bf16x8*>(&Ks[buf][row * KSTR + ch * 8]) = kreg[i];
      *reinterpret_cast<bf16x8*>(&Vs[buf][row * VSTR + ch * 8]) = vreg[i];
    }
  };
  const int vtr = tr_lane_ptr(Vs[0], VSTR, 0, 0, lane) - Vs[0];  // this lane's V^T read offset

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

  if (n_tiles > 0) {
    load_tile(0);
    store_tile(0);
    if (n_tiles > 1) load_tile(1);
  }
  __syncthreads();

  for (int t = 0; t < n_tiles; ++t) {
    const int buf = t & 1;
    const bf16* Kb = Ks[buf];
    const bf16* Vb = Vs[buf] + vtr;

    f32x16 sacc[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        bf16x8 a = *reinterpret_cast<const bf16x8*>(&Kb[(kb * 32 + c) * KSTR + kk * 16 + hh * 8]);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], sacc[kb], 0, 0, 0);
      }
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
    mx = fmaxf(mx, __shfl_xor(mx, 32)) * c2;
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
        const bf16x8 a = lds_read_tr(Vb + ks * 16 * VSTR + db * 32, VSTR);
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[ks], oacc[db], 0, 0, 0);
      }
    }

    if (t + 1 < n_tiles) {
      store_tile(buf ^ 1);  // buffer buf^1 was last read in iteration t-1
      if (t + 2 < n_tiles) load_tile(t + 2);
    }
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (qvalid) {
    bf16* op = p.o + (int64_t)(it.a_start + qrow) * qstride + (int64_t)h * D + hh * 4;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        bf16x4 x = {f2bf(oacc[db][a * 4 + 0] * inv), f2bf(oacc[db][a * 4 + 1] * inv),
                    f2bf(oacc[db][a * 4 + 2] * inv), f2bf(oacc[db][a * 4 + 3] * inv)};
        *reinterpret_cast<bf16x4*>(op + db * 32 + a * 8) = x;
      }
    }
    if (hh == 0)
      p.lse[(int64_t)h * p.total_q + it.a_start + qrow] =
          l_tot > 0.f ? (m2 + log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

}  // namespace

hipError_t launch_fwd_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                           int causal, float scale, void* out, float* lse, const void* ws,
                           const WsLayout& L, hipStream_t stream) {
  if (L.max_items == 0 || dims.hq == 0) return hipSuccess;
  FwdParams p;
  p.q = static_cast<const bf16*>(q);
  p.k = static_cast<const bf16*>(k);
  p.v = static_cast<const bf16*>(v);
  p.o = static_cast<bf16*>(out);
  p.lse = lse;
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
