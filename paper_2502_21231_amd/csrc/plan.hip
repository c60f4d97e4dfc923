// Device work planner: cu_seqlens (or chunk offsets) -> ordered list of tiles.
//
// The paper observes that the work of a packed micro-batch is proportional to
// the area of its attention mask, not to its token count (Sec. 3.3, Imbalanced
// FLOPs; Sec. 7, Dist-attn with packing).  The planner enumerates, per segment,
// the query tiles (forward) or key tiles (backward), counts the tiles of the
// other side that carry visible pairs, separates the FULL ones (no score mask
// needed) from the MASKED ones (causal diagonal or ragged key tail), and orders
// the list so that a grid walking it in block order starts the largest work
// first (longest-processing-time-first balancing of the long-tailed length mix)
// while the tiles of one segment run side by side and share its K/V (forward)
// or Q/dO (backward) tiles in L2:
//   segments by size (len_q + len_k) descending, ties by segment index;
//   inside a segment by descending cost, which is a closed form: a query tile
//   sees no fewer key tiles than the one above it (forward: descending tile
//   index), a key tile is seen by no more query tiles than the one before it
//   (backward: ascending tile index).
// Tiles with no visible pair are never listed.
//
// Three kernels, all on the caller's stream and without host synchronisation:
//   plan_count : validate cu_seqlens, per-segment tile counts, exclusive scan
//   plan_rank  : one thread per segment: its first slot in the ordered list
//   plan_emit  : one thread per list entry, fills its fields at its slot
// or, for up to 1024 segments, the same three steps in one workgroup (plan_fused).
#include "attn.hpp"

namespace bs {
namespace {

constexpr int kCountThreads = 1024;

__device__ __forceinline__ void set_status(int32_t* st, int code) {
  atomicCAS(st, 0, code);  // keeps the first error seen
}

// Segment b of the problem: query start/length, key start/length, diagonal.
struct Seg {
  int64_t q0, lq, k0, lk;
  int32_t diag;
};

__device__ __forceinline__ int32_t clamp_diag(int64_t d) {
  return (int32_t)(d < -kDiagClamp ? -kDiagClamp : (d > kDiagClamp ? kDiagClamp : d));
}

// Diagonal: key j visible to query i iff j - i <= diag.  Varlen segments are
// aligned bottom-right (diag = len_k - len_q); packed chunk segments and single
// chunks take it from the global positions of their first query and key.
__device__ __forceinline__ Seg load_seg(const int32_t* cu_q, const int32_t* cu_k,
                                        const int64_t* q_pos, const int64_t* k_pos, int32_t b,
                                        int64_t total_q, int64_t total_k, int32_t diag_chunk) {
  Seg s;
  if (cu_q == nullptr) {  // chunk mode: one segment, diagonal from the offsets
    s.q0 = 0; s.lq = total_q; s.k0 = 0; s.lk = total_k; s.diag = diag_chunk;
  } else {
    s.q0 = cu_q[b]; s.lq = (int64_t)cu_q[b + 1] - cu_q[b];
    s.k0 = cu_k[b]; s.lk = (int64_t)cu_k[b + 1] - cu_k[b];
    s.diag = q_pos == nullptr ? clamp_diag(s.lk - s.lq) : clamp_diag(q_pos[b] - k_pos[b]);
  }
  return s;
}

// Validates cu_seqlens, computes items per segment and their exclusive prefix into seg_off
// (nseg + 1 entries), and the status word and item count into the header.  One workgroup
// of kCountThreads threads; scan, carry and status are its LDS.
__device__ __forceinline__ void count_body(const int32_t* __restrict__ cu_q,
                                           const int32_t* __restrict__ cu_k, int32_t num_seqs,
                                           int64_t total_q, int64_t total_k, int32_t max_seqlen,
                                           int kind, int tile_a, WsHeader* __restrict__ hdr,
                                           int32_t* seg_off, int32_t* scan, int32_t& carry,
                                           int32_t& status) {
  const int t = threadIdx.x;
  if (t == 0) { carry = 0; status = 0; }
  __syncthreads();
  const int32_t nseg = cu_q == nullptr ? 1 : num_seqs;
  if (cu_q != nullptr && t == 0) {
    if (cu_q[0] != 0 || cu_k[0] != 0) set_status(&status, BS_DEV_BAD_FIRST);
    if (cu_q[num_seqs] != total_q || cu_k[num_seqs] != total_k) set_status(&status, BS_DEV_BAD_TOTAL);
  }
  for (int32_t base = 0; base < nseg; base += kCountThreads) {
    const int32_t b = base + t;
    int32_t cnt = 0;
    if (b < nseg) {
      Seg s = load_seg(cu_q, cu_k, nullptr, nullptr, b, total_q, total_k, 0);
      if (s.lq < 0 || s.lk < 0) set_status(&status, BS_DEV_NOT_MONOTONE);
      else if (cu_q != nullptr && (s.lq > max_seqlen || s.lk > max_seqlen)) set_status(&status, BS_DEV_TOO_LONG);
      else {
        const int64_t la = kind == kPlanFwd ? s.lq : s.lk;
        cnt = (int32_t)((la + tile_a - 1) / tile_a);
      }
    }
    scan[t] = cnt;
    __syncthreads();
    for (int off = 1; off < kCountThreads; off <<= 1) {  // inclusive Hillis-Steele scan
      int32_t x = t >= off ? scan[t - off] : 0;
      __syncthreads();
      scan[t] += x;
      __syncthreads();
    }
    if (b < nseg) seg_off[b] = carry + scan[t] - cnt;
    __syncthreads();
    if (t == kCountThreads - 1) carry += scan[t];
    __syncthreads();
  }
  if (t == 0) {
    seg_off[nseg] = carry;
    hdr->status = status;
    hdr->n_items = status == 0 ? carry : 0;
  }
}

__global__ __launch_bounds__(kCountThreads) void plan_count(
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_k, int32_t num_seqs,
    int64_t total_q, int64_t total_k, int32_t max_seqlen, int kind, int tile_a,
    WsHeader* __restrict__ hdr, int32_t* __restrict__ seg_off) {
  __shared__ int32_t scan[kCountThreads];
  __shared__ int32_t carry;
  __shared__ int32_t status;
  count_body(cu_q, cu_k, num_seqs, total_q, total_k, max_seqlen, kind, tile_a, hdr, seg_off, scan,
             carry, status);
}

// List entry i (0 <= i < the item count): its segment, tile and counts, written at its slot.
__device__ __forceinline__ void emit_body(
    int64_t i, const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_k,
    const int64_t* __restrict__ q_pos, const int64_t* __restrict__ k_pos, int32_t num_seqs,
    int64_t total_q, int64_t total_k, int32_t diag_chunk, int causal, int kind, int tile_a,
    int tile_b, const int32_t* seg_off, const int32_t* seg_dst, WorkItem* __restrict__ items) {
  const int32_t nseg = cu_q == nullptr ? 1 : num_seqs;
  // segment b with seg_off[b] <= i < seg_off[b+1] (skipping empty segments)
  int32_t lo = 0, hi = nseg - 1;
  while (lo < hi) {
    int32_t mid = (lo + hi + 1) >> 1;
    if (seg_off[mid] <= i) lo = mid; else hi = mid - 1;
  }
  const int32_t b = lo;
  const Seg s = load_seg(cu_q, cu_k, q_pos, k_pos, b, total_q, total_k, diag_chunk);
  const int64_t tile = i - seg_off[b];
  const int64_t diag = s.diag;
  WorkItem w;
  w.seg = b; w.tile = (int32_t)tile; w.diag = s.diag; w.run0 = seg_dst[b]; w.nrun = (int32_t)(seg_off[b + 1] - seg_off[b]);
  if (kind == kPlanFwd) {
    const int64_t BM = tile_a, BN = tile_b;
    const int64_t q_first = tile * BM;
    const int64_t q_last = (q_first + BM < s.lq ? q_first + BM : s.lq) - 1;
    const int64_t nkt = (s.lk + BN - 1) / BN;
    int64_t n_tiles, n_full;
    if (causal) {
      const int64_t lim = q_last + diag;
      n_tiles = lim < 0 ? 0 : (lim / BN + 1 < nkt ? lim / BN + 1 : nkt);
      int64_t f = q_first + diag + 1;
      f = f < s.lk ? f : s.lk;
      n_full = f > 0 ? f / BN : 0;
    } else {
      n_tiles = nkt;
      n_full = s.lk / BN;
    }
    w.a_start = (int32_t)(s.q0 + q_first);
    w.a_rows = (int32_t)(q_last - q_first + 1);
    w.b_start = (int32_t)s.k0;
    w.b_len = (int32_t)s.lk;
    w.n0 = (int32_t)n_full;
    w.n1 = (int32_t)n_tiles;
    w.n2 = (int32_t)n_tiles;
  } else {
    const int64_t BM = tile_b, BN = tile_a;
    const int64_t k_first = tile * BN;
    const int64_t nqt = (s.lq + BM - 1) / BM;
    const bool in_range = k_first + BN <= s.lk;
    int64_t first, ffirst;
    if (causal) {
      const int64_t r = k_first - diag;  // first query row that sees key k_first
      first = r > s.lq - 1 ? nqt : (r > 0 ? r / BM : 0);
      if (!in_range) {
        ffirst = nqt;
      } else {
        const int64_t t = k_first + BN - 1 - diag;  // FULL needs q_first >= t
        ffirst = t <= 0 ? 0 : (t + BM - 1) / BM;
        ffirst = ffirst < nqt ? ffirst : nqt;
      }
    } else {
      first = 0;
      ffirst = in_range ? 0 : nqt;
    }
    const int64_t n_vis = nqt - first;
    const int64_t n_masked = ffirst - first > 0 ? ffirst - first : 0;
    w.a_start = (int32_t)(s.k0 + k_first);
    w.a_rows = (int32_t)(s.lk - k_first < BN ? s.lk - k_first : BN);
    w.b_start = (int32_t)s.q0;
    w.b_len = (int32_t)s.lq;
    w.n0 = (int32_t)first;
    w.n1 = (int32_t)n_masked;
    w.n2 = (int32_t)n_vis;
  }
  const int64_t cnt = seg_off[b + 1] - seg_off[b];
  items[seg_dst[b] + (kind == kPlanFwd ? cnt - 1 - tile : tile)] = w;
}

__global__ __launch_bounds__(256) void plan_emit(
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_k,
    const int64_t* __restrict__ q_pos, const int64_t* __restrict__ k_pos, int32_t num_seqs,
    int64_t total_q, int64_t total_k, int32_t diag_chunk, int causal, int kind, int tile_a,
    int tile_b, int64_t max_items, const WsHeader* __restrict__ hdr,
    const int32_t* __restrict__ seg_off, const int32_t* __restrict__ seg_dst,
    WorkItem* __restrict__ items) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= max_items || i >= hdr->n_items) return;
  emit_body(i, cu_q, cu_k, q_pos, k_pos, num_seqs, total_q, total_k, diag_chunk, causal, kind,
            tile_a, tile_b, seg_off, seg_dst, items);
}

// First slot of each segment in the ordered list: the items of every segment that
// comes before it (larger len_q + len_k, or equal size and a lower index).
constexpr int kRankChunk = 1024;

__global__ __launch_bounds__(256) void plan_rank(const int32_t* __restrict__ cu_q,
                                                 const int32_t* __restrict__ cu_k, int32_t num_seqs,
                                                 const WsHeader* __restrict__ hdr,
                                                 const int32_t* __restrict__ seg_off,
                                                 int32_t* __restrict__ seg_dst) {
  __shared__ int64_t ssz[kRankChunk];
  __shared__ int32_t scnt[kRankChunk];
  if (hdr->status != 0) return;  // uniform: the list is empty
  const int32_t nseg = cu_q == nullptr ? 1 : num_seqs;
  const int32_t b = blockIdx.x * blockDim.x + threadIdx.x;
  auto size_of = [&](int32_t x) -> int64_t {
    return cu_q == nullptr ? 0 : ((int64_t)cu_q[x + 1] - cu_q[x]) + ((int64_t)cu_k[x + 1] - cu_k[x]);
  };
  const int64_t mine = b < nseg ? size_of(b) : 0;
  int64_t dst = 0;
  for (int32_t base = 0; base < nseg; base += kRankChunk) {
    for (int j = threadIdx.x; j < kRankChunk; j += blockDim.x) {
      const bool ok = base + j < nseg;
      ssz[j] = ok ? size_of(base + j) : 0;
      scnt[j] = ok ? seg_off[base + j + 1] - seg_off[base + j] : 0;
    }
    __syncthreads();
    const int32_t lim = nseg - base < kRankChunk ? nseg - base : kRankChunk;
    for (int32_t j = 0; j < lim; ++j) {
      const bool before = ssz[j] > mine || (ssz[j] == mine && base + j < b);
      dst += before ? scnt[j] : 0;
    }
    __syncthreads();
  }
  if (b < nseg) seg_dst[b] = (int32_t)dst;
}

// All three steps in one workgroup, for up to kCountThreads segments (one thread per segment
// in the ranking): the per-segment offsets and first slots stay in LDS, and the list
// entries are filled in a loop over the workgroup.  Same list as the three kernels.
__global__ __launch_bounds__(kCountThreads) void plan_fused(
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_k,
    const int64_t* __restrict__ q_pos, const int64_t* __restrict__ k_pos, int32_t num_seqs,
    int64_t total_q, int64_t total_k, int32_t max_seqlen, int32_t diag_chunk, int causal,
    int kind, int tile_a, int tile_b, int64_t max_items, WsHeader* __restrict__ hdr,
    WorkItem* __restrict__ items) {
  __shared__ int32_t scan[kCountThreads];
  __shared__ int32_t soff[kCountThreads + 1];
  __shared__ int32_t sdst[kCountThreads];
  __shared__ int64_t ssz[kCountThreads];
  __shared__ int32_t carry;
  __shared__ int32_t status;
  count_body(cu_q, cu_k, num_seqs, total_q, total_k, max_seqlen, kind, tile_a, hdr, soff, scan,
             carry, status);
  __syncthreads();
  if (status != 0 || max_items == 0) return;  // uniform: the list is empty
  const int32_t nseg = cu_q == nullptr ? 1 : num_seqs;
  const int t = threadIdx.x;
  // first slot of segment t: the items of every segment that comes before it (larger
  // len_q + len_k, or equal size and a lower index)
  const int64_t mine =
      (cu_q != nullptr && t < nseg) ? ((int64_t)cu_q[t + 1] - cu_q[t]) + ((int64_t)cu_k[t + 1] - cu_k[t]) : 0;
  ssz[t] = mine;
  __syncthreads();
  if (t < nseg) {
    int32_t dst = 0;
    for (int32_t j = 0; j < nseg; ++j) {
      const bool before = ssz[j] > mine || (ssz[j] == mine && j < t);
      dst += before ? soff[j + 1] - soff[j] : 0;
    }
    sdst[t] = dst;
  }
  __syncthreads();
  const int64_t n = carry < max_items ? carry : max_items;
  for (int64_t i = t; i < n; i += kCountThreads)
    emit_body(i, cu_q, cu_k, q_pos, k_pos, num_seqs, total_q, total_k, diag_chunk, causal, kind,
              tile_a, tile_b, soff, sdst, items);
}

}  // namespace

hipError_t launch_plan(PlanKind kind, const int32_t* cu_q, const int32_t* cu_k,
                       const int64_t* q_pos, const int64_t* k_pos, int32_t num_seqs,
                       int64_t total_q, int64_t total_k, int32_t max_seqlen, int32_t diag_chunk,
                       int causal, int tile_a, int tile_b, int64_t max_items, void* ws,
                       const WsLayout& L, hipStream_t stream) {
  char* base = static_cast<char*>(ws);
  WsHeader* hdr = reinterpret_cast<WsHeader*>(base);
  int32_t* seg_off = reinterpret_cast<int32_t*>(base + L.seg_off);
  int32_t* seg_dst = reinterpret_cast<int32_t*>(base + L.seg_dst);
  WorkItem* sorted = reinterpret_cast<WorkItem*>(base + L.sorted);
  const int32_t nsegs = cu_q == nullptr ? 1 : num_seqs;
  if (nsegs <= kCountThreads) {
    hipLaunchKernelGGL(plan_fused, dim3(1), dim3(kCountThreads), 0, stream, cu_q, cu_k, q_pos,
                       k_pos, num_seqs, total_q, total_k, max_seqlen, diag_chunk, causal, (int)kind,
                       tile_a, tile_b, max_items, hdr, sorted);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(plan_count, dim3(1), dim3(kCountThreads), 0, stream, cu_q, cu_k, num_seqs,
                     total_q, total_k, max_seqlen, (int)kind, tile_a, hdr, seg_off);
  if (max_items > 0) {
    const int32_t nseg = cu_q == nullptr ? 1 : num_seqs;
    hipLaunchKernelGGL(plan_rank, dim3((unsigned)((nseg + 255) / 256)), dim3(256), 0, stream, cu_q,
                       cu_k, num_seqs, hdr, seg_off, seg_dst);
    const unsigned blocks = (unsigned)((max_items + 255) / 256);
    hipLaunchKernelGGL(plan_emit, dim3(blocks), dim3(256), 0, stream, cu_q, cu_k, q_pos, k_pos,
                       num_seqs, total_q, total_k, diag_chunk, causal, (int)kind, tile_a, tile_b,
                       max_items, hdr, seg_off, seg_dst, sorted);
  }
  return hipGetLastError();
}

}  // namespace bs
