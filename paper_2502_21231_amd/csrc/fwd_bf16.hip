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
// K tiles are staged in LDS row-major ([key][d], +8 element pad), V tiles
// transposed ([d][key], permuted, +8 pad); the next tile is prefetched into
// registers while the current one is consumed.
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
  float scale_log2;  // scale * log2(e): scores are kept in the base-2 domain
};

// Physical position, inside its 16-key group, of key kk of that group in the
// transposed V tile: groups of four keys 4-7 and 8-11 trade places.
__device__ __forceinline__ int vperm4(int g4) { return (g4 == 1) ? 2 : (g4 == 2 ? 1 : g4); }

// Query head handled by a block: heads are spread so that all blocks of one
// head (and of one KV group) fall on the same XCD when hq is a multiple of 8
// (blocks are dealt to the 8 XCDs round-robin by block index).
__device__ __forceinline__ int head_of(int slot, int hq) {
  return (hq & 7) == 0 ? (slot & 7) * (hq >> 3) + (slot >> 3) : slot;
}

template <int D>
__global__ __launch_bounds__(256) void fwd_bf16_kernel(const FwdParams p) {
  constexpr int BM = kFwdBM, BN = kFwdBN;
  constexpr int KSTR = D + 8;       // K tile row stride (elements)
  constexpr int VSTR = BN + 8;      // V^T tile row stride
  constexpr int KK = D / 16;        // MFMA k-steps over head_dim
  constexpr int DB = D / 32;        // 32-wide blocks of head_dim
  constexpr int KUNITS = BN * D / 8 / 256;  // 16-byte K loads per thread
  constexpr int VUNITS = (BN / 4) * (D / 8);  // (4 keys x 8 dims) V units per tile
  static_assert(BM == 128 && BN == 64, "tile shape");
  static_assert(KUNITS >= 1, "K staging");

  __shared__ __attribute__((aligned(16))) bf16 Ks[BN * KSTR];
  __shared__ __attribute__((aligned(16))) bf16 Vt[D * VSTR];

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
  const int64_t kvstride = (int64_t)p.hkv * D;

  // Q fragment of this lane's query row, B operand of S^T = K Q^T
  bf16x8 qf[KK];
  {
    const bf16* qp = p.q + (int64_t)(it.a_start + (qvalid ? qrow : 0)) * qstride + (int64_t)h * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      bf16x8 x = *reinterpret_cast<const bf16x8*>(qp + kk * 16 + hh * 8);
      qf[kk] = qvalid ? x : bf16x8{};
    }
  }

  const bf16* kbase = p.k + (int64_t)it.b_start * kvstride + (int64_t)hk * D;
  const bf16* vbase = p.v + (int64_t)it.b_start * kvstride + (int64_t)hk * D;
  const int k_len = it.b_len;

  bf16x8 kreg[KUNITS];
  bf16x8 vreg[4];
  auto load_tile = [&](int t) {
    const int k0 = t * BN;
#pragma unroll
    for (int i = 0; i < KUNITS; ++i) {
      const int idx = i * 256 + tid;
      const int row = idx / (D / 8), ch = idx % (D / 8);
      const bool ok = k0 + row < k_len;
      bf16x8 x = *reinterpret_cast<const bf16x8*>(kbase + (int64_t)(ok ? k0 + row : 0) * kvstride + ch * 8);
      kreg[i] = ok ? x : bf16x8{};
    }
    if (tid < VUNITS) {
      const int g = tid % (BN / 4), ch = tid / (BN / 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = g * 4 + i;
        const bool ok = k0 + row < k_len;
        bf16x8 x = *reinterpret_cast<const bf16x8*>(vbase + (int64_t)(ok ? k0 + row : 0) * kvstride + ch * 8);
        vreg[i] = ok ? x : bf16x8{};
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < KUNITS; ++i) {
      const int idx = i * 256 + tid;
      const int row = idx / (D / 8), ch = idx % (D / 8);
      *reinterpret_cast<bf16x8*>(&Ks[row * KSTR + ch * 8]) = kreg[i];
    }
    if (tid < VUNITS) {
      const int g = tid % (BN / 4), ch = tid / (BN / 4);
      const int pcol = (g >> 2) * 16 + vperm4(g & 3) * 4;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bf16x4 col = {vreg[0][e], vreg[1][e], vreg[2][e], vreg[3][e]};
        *reinterpret_cast<bf16x4*>(&Vt[(ch * 8 + e) * VSTR + pcol]) = col;
      }
    }
  };

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  const int n_tiles = it.n1, n_full = it.n0;
  const int q_rel = it.tile * BM + qrow;  // query index inside its segment
  const int diag = it.diag;

  if (n_tiles > 0) load_tile(0);
  for (int t = 0; t < n_tiles; ++t) {
    __syncthreads();
    store_tile();
    __syncthreads();
    if (t + 1 < n_tiles) load_tile(t + 1);

    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sacc[kb] = f32x16{};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        bf16x8 a = *reinterpret_cast<const bf16x8*>(&Ks[(kb * 32 + c) * KSTR + kk * 16 + hh * 8]);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], sacc[kb], 0, 0, 0);
      }
    }

    // scores of this lane's query against its 32 keys, base-2 domain
    float mx = -INFINITY;
    const bool masked = t >= n_full;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float s = sacc[kb][r] * p.scale_log2;
        if (masked) {
          const int key = t * BN + kb * 32 + (r >> 2) * 8 + hh * 4 + (r & 3);
          const bool vis = key < k_len && (!p.causal || key - q_rel <= diag);
          s = vis ? s : -INFINITY;
        }
        sacc[kb][r] = s;
        mx = fmaxf(mx, s);
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float base = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - base);
    m_run = m_new;
    float psum = 0.f;
    bf16x8 pb[4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = fast_exp2(sacc[kb][r] - base);
        psum += e;
        pb[kb * 2 + (r >> 3)][r & 7] = f2bf(e);
      }
    }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] *= alpha;

#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        bf16x8 a = *reinterpret_cast<const bf16x8*>(&Vt[(db * 32 + c) * VSTR + ks * 16 + hh * 8]);
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[ks], oacc[db], 0, 0, 0);
      }
    }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (qvalid) {
    bf16* op = p.o + (int64_t)(it.a_start + qrow) * qstride + (int64_t)h * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        bf16x4 x = {f2bf(oacc[db][a * 4 + 0] * inv), f2bf(oacc[db][a * 4 + 1] * inv),
                    f2bf(oacc[db][a * 4 + 2] * inv), f2bf(oacc[db][a * 4 + 3] * inv)};
        *reinterpret_cast<bf16x4*>(op + db * 32 + a * 8 + hh * 4) = x;
      }
    }
    if (hh == 0)
      p.lse[(int64_t)h * p.total_q + it.a_start + qrow] =
          l_tot > 0.f ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
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
