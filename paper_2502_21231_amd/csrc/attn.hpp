// Definitions of the attention path of libbs_attn.so (gfx950 only): the ordered work
// list and its workspace, tile shapes, the placement of blocks on the XCDs, the
// swizzled LDS tiles with their copy and transposing reads, and the host launchers.
#pragma once

#include "common.hpp"

namespace bs {

constexpr int kDiagClamp = 1 << 30;

// One entry of the ordered work list (12 int32 = 48 bytes).
// Forward (query tile):  seg, tile=qtile, a_start=q_start, a_rows=q_rows,
//                        b_start=k_start, b_len=k_len, n0=n_full, n1=n_tiles, diag.
// Backward (key tile):   seg, tile=ktile, a_start=k_start, a_rows=k_rows,
//                        b_start=q_start, b_len=q_len, n0=qt_first, n1=n_masked,
//                        n2=n_vis, diag.
// Both: run0 = list slot of the first item of the segment, nrun = the segment's item
// count (the items of a segment are contiguous in the list).
struct WorkItem {
  int32_t seg, tile, a_start, a_rows, b_start, b_len, n0, n1, n2, diag, run0, nrun;
};
static_assert(sizeof(WorkItem) == 48, "work item is 12 int32");

enum PlanKind { kPlanFwd = 0, kPlanBwd = 1 };

// Tile sizes of each kernel family.  The forward walks query tiles of kFwdBM rows
// over key tiles of kFwdBN keys; the backward walks key tiles of kBwdBN keys over
// query tiles of bwd_bm(head_dim) rows: 96 at head_dim 128, 64 at head_dim 64 (a
// 96-row tile of 64-wide rows is 12 copy instructions, which 8 waves cannot share
// evenly).  The float32 kernels use their own sizes.
constexpr int kFwdBM = 128, kFwdBN = 64;
constexpr int kBwdBN = 128;
__host__ __device__ constexpr int bwd_bm(int head_dim) { return head_dim == 128 ? 96 : 64; }
constexpr int kF32BM = 64, kF32BN = 64;

// Workspace header: status word and item count, then the per-segment item
// offsets (segment order) and first slots (list order), the ordered work list,
// then op-specific float buffers.
struct WsHeader {
  int32_t status;
  int32_t n_items;
  int32_t pad[62];
};

// The dK/dV kernel walks a segment one head at a time from this many streamed rows (b_len)
// on; the forward and dQ kernels do so for every segment.
constexpr int kHeadMajorRowsDkdv = 16384;

// Work item and head of this workgroup in a grid of n_items * n_heads blocks; false when it
// has none.  Blocks are dealt to the 8 XCDs round-robin (block b runs on XCD b % 8), so with
// n_heads a multiple of 8 each XCD owns the hx = n_heads / 8 heads x*hx .. x*hx+hx-1 and walks
// the list segment by segment.  Inside a segment's run its heads are interleaved item by
// item, except where the segment streams at least min_rows rows and the XCD's heads read
// more than one stream (hx > heads_per_stream: heads that share a KV head share its K/V
// stream): there the XCD walks one head's items at a time, so that the workgroups resident
// on it read one stream, not hx / heads_per_stream, and each tile of it comes into the
// XCD's L2 that many times less often.
__device__ __forceinline__ bool block_work(const WsHeader* __restrict__ hdr,
                                           const WorkItem* __restrict__ items, int n_heads,
                                           int heads_per_stream, int min_rows, WorkItem& it,
                                           int& head) {
  const int b = blockIdx.x;
  const int n_items = hdr->n_items;
  if ((n_heads & 7) != 0) {
    const int i = b / n_heads;
    if (i >= n_items) return false;
    it = items[i];
    head = b - i * n_heads;
    return true;
  }
  const int hx = n_heads >> 3, jb = b >> 3;
  const int g = jb / hx;
  if (g >= n_items) return false;
  const WorkItem gi = items[g];
  const int r = jb - gi.run0 * hx;  // 0 <= r < nrun * hx: this block's place in the run
  int i, hl;
  if (hx > heads_per_stream && gi.b_len >= min_rows) {
    hl = r / gi.nrun;
    i = gi.run0 + (r - hl * gi.nrun);
  } else {
    i = g;
    hl = r - (g - gi.run0) * hx;
  }
  it = i == g ? gi : items[i];
  head = (b & 7) * hx + hl;
  return true;
}

struct WsLayout {
  size_t seg_off;     // int32[num_seqs + 1]
  size_t seg_dst;     // int32[num_seqs]
  size_t sorted;      // WorkItem[max_items]
  size_t dvec;        // float[hq * T]      (backward: rowsum(dO * O))
  size_t dq_acc;      // float[T * hq * d]  (varlen backward only)
  size_t total;
  int64_t max_items;
};

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Operand of a 32x32x16 bf16 MFMA that is the TRANSPOSE of a row-major LDS tile.
//
// X is a row-major bf16 tile in LDS (`stride` elements per row) whose rows run
// along the MFMA contraction index and whose columns run along the MFMA row
// (A operand) / column (B operand) index.  Lane l = 32*hh + c receives
// X[k0 + (e/4)*8 + hh*4 + e%4][m0 + c] as element e (e = 0..7): inside every
// 16-step of the contraction, lanes 0-31 take rows 0-3 and 8-11, lanes 32-63
// rows 4-7 and 12-15.  That is exactly the contraction order in which a lane
// holds the rows of a 32x32 MFMA result, so a result kept in registers (P, dS)
// can be fed as the other operand without reshuffling.
//
// Built from two ds_read_b64_tr_b16: inside each 16-lane group, output lane i
// gets element (i % 4) of the 8-byte chunk addressed by lane 4e + i/4, for
// e = 0..3; so lane s addresses row k0 + r*8 + hh*4 + (s%16)/4, columns
// m0 + 16*((s/16)%2) + 4*(s%4) .. +3, in read r = 0, 1.
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

__device__ __forceinline__ const bf16* tr_lane_ptr(const bf16* tile, int stride, int k0, int m0,
                                                   int lane) {
  const int i = lane & 15;
  return tile + (k0 + (lane >> 5) * 4 + (i >> 2)) * stride + m0 + ((lane >> 4) & 1) * 16 + (i & 3) * 4;
}

// The operand from two lane addresses: rows k0 + hh*4 + (i/4) and the row 8 below.
__device__ __forceinline__ bf16x8 lds_read_tr2(const bf16* p0, const bf16* p1) {
  const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p0));
  const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p1));
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  const i16x8 v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// `p` is tr_lane_ptr(tile, stride, k0, m0, lane) of a padded tile.
__device__ __forceinline__ bf16x8 lds_read_tr(const bf16* p, int stride) {
  return lds_read_tr2(p, p + 8 * stride);
}

// Swizzled row-major LDS tile with D bf16 per row (no padding) for tiles that are
// read both ways: row reads (16 consecutive rows, one 16-byte chunk each) and
// transposing reads (4 consecutive rows, 4 consecutive chunks each, per half
// wave).  Chunk c of row r is stored at chunk c ^ g(r).  With 64 banks of 4
// bytes, g makes both patterns conflict-free:
//   D = 128 (16 chunks = one bank line per row): g(r) = ((r&3) << 2) | ((r>>2)&3)
//     - any 16 consecutive rows: g is a bijection of r mod 16;
//     - 4 aligned rows: (r&3) moves each row's 4-chunk group to a different quarter.
//   D = 64 (8 chunks = half a bank line per row): g(r) = (((r>>1)&1) << 2) | ((r>>2)&3)
//     - rows of equal parity share a half line, and g is a bijection over them;
//     - of 4 aligned rows, the two of equal parity land in different 4-chunk groups.
// g depends on r mod 16 only, so tiles may be addressed from any 16-row boundary.
template <int D>
__device__ __forceinline__ int swz_g(int r) {
  static_assert(D == 64 || D == 128, "head_dim");
  return D == 128 ? (((r & 3) << 2) | ((r >> 2) & 3)) : ((((r >> 1) & 1) << 2) | ((r >> 2) & 3));
}

// Element offset of 16-byte chunk `c` of row `r`.
template <int D>
__device__ __forceinline__ int swz_off(int r, int c) {
  return r * D + ((c ^ swz_g<D>(r)) << 3);
}

// The swizzle only moves bits 4..7 of a byte offset inside a row (it XORs the chunk
// index), so a lane's reads of a tile differ by a lane-independent XOR plus a multiple of
// a row: one lane base per access pattern gives every address with one v_xor_b32, and the
// row part (and the tile's own LDS address) go into the instruction's immediate offset.
//   row read of chunk (2 kk + hh) of row (32 kb + c), lane = 32 hh + c:
//     swz_off(32 kb + c, 2 kk + hh) * 2 == (swz_row_base(lane) ^ (kk << 5)) + kb * 64 * D
//   transposing read r of contraction rows k0 = 16 ks, columns m0 = 32 db:
//     swz_tr_off(16 ks, 32 db, r, lane) * 2
//         == (swz_tr_base(lane) ^ ((db << 6) | (r << 5))) + ks * 32 * D + r * 16 * D
template <int D>
__device__ __forceinline__ int swz_row_base(int lane) {
  return swz_off<D>(lane & 31, lane >> 5) * 2;
}
template <int D>
__device__ __forceinline__ int swz_tr_base(int lane);

// One wave's share of copying rows 0..R-1 of a swizzled [R][D] bf16 tile from global
// memory straight into LDS (buffer_load_dwordx4 ... lds: lane l of an instruction
// writes 16 bytes at LDS base + offset + 16*l, so an instruction fills 64/(D/8) whole
// rows, 1 KB, and each lane fetches the global chunk that the swizzle places at its
// LDS position).  Row r of the tile comes from src + min(r, last) * gstride elements:
// rows past the end repeat the last valid one.  Completion is waited for with
// wait_vmem_all().
//
// Each wave copies a contiguous run of PER instructions from one LDS base (M0): the
// instruction offset (0, 1 KB, 2 KB, 3 KB) moves both the LDS and the global address,
// so the per-lane global offsets subtract it, and the buffer starts 4 KB before `src`
// to keep them non-negative (only src + row offsets are ever accessed).
//
// The buffer form (MUBUF) rather than global_load_lds (FLAT): the compiler treats a
// pending FLAT copy into LDS as a possible LDS access of unknown order and then
// waits for all LDS reads (lgkmcnt(0)) before every use, which defeats reading LDS
// operands ahead.  Byte offsets (R rows x gstride x 2 + 4 KB) stay below 2^31 for
// the head counts the C API accepts.
template <int K, int PER, int D>
struct DmaRun {
  static __device__ __forceinline__ void issue(__amdgpu_buffer_rsrc_t rs, bf16* lds, int row0,
                                               int sub, int phys, int gstride, int last) {
    constexpr int RPI = 64 / (D / 8);
    const int row = row0 + K * RPI + sub;
    const int r = row < last ? row : last;
    const int voff = (r * gstride + ((phys ^ swz_g<D>(row)) << 3)) * 2 + 4096 - K * 1024;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)lds, 16,
                                             voff, 0, K * 1024, 0);
    DmaRun<K + 1, PER, D>::issue(rs, lds, row0, sub, phys, gstride, last);
  }
};
template <int PER, int D>
struct DmaRun<PER, PER, D> {
  static __device__ __forceinline__ void issue(__amdgpu_buffer_rsrc_t, bf16*, int, int, int, int,
                                               int) {}
};

template <int D, int R, int NWAVES>
__device__ __forceinline__ void dma_tile(bf16* lds_tile, const bf16* src, int gstride, int last,
                                         int wave, int lane) {
  constexpr int CPR = D / 8, RPI = 64 / CPR, NI = R / RPI, PER = NI / NWAVES;
  static_assert(NI % NWAVES == 0, "whole instructions per wave");
  static_assert(PER >= 1 && PER <= 4, "instruction offsets of one run fit in 12 bits");
  const int sub = lane / CPR, phys = lane % CPR;
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(reinterpret_cast<const char*>(src) - 4096), 0, 0x7fffffff, 0x00020000);
  const int u0 = wave * PER;  // first instruction (1 KB of LDS) of this wave's run
  DmaRun<0, PER, D>::issue(rsrc, lds_tile + u0 * RPI * D, u0 * RPI, sub, phys, gstride, last);
}

// Element offset, in a swizzled tile, of this lane's 8-byte piece of the transposing
// read r (0 or 1) at contraction row k0 (a multiple of 16) and column m0 (a multiple
// of 32): row k0 + 8r + 4hh + i/4, column m0 + 16*((lane/16)%2) + 4*(i%4).
template <int D>
__device__ __forceinline__ int swz_tr_off(int k0, int m0, int r, int lane) {
  const int i = lane & 15;
  const int row = k0 + 8 * r + 4 * (lane >> 5) + (i >> 2);
  const int col = m0 + ((lane >> 4) & 1) * 16 + (i & 3) * 4;
  return swz_off<D>(row, col >> 3) + (col & 7);
}
template <int D>
__device__ __forceinline__ int swz_tr_base(int lane) {
  return swz_tr_off<D>(0, 0, 0, lane) * 2;
}
// Byte-addressed LDS views used with the bases above.
__device__ __forceinline__ bf16x8 lds_row16(const bf16* tile, int byte_off) {
  return *reinterpret_cast<const bf16x8*>(reinterpret_cast<const char*>(tile) + byte_off);
}
__device__ __forceinline__ bf16x8 lds_tr16(const bf16* tile, int off0, int off1) {
  const char* t = reinterpret_cast<const char*>(tile);
  return lds_read_tr2(reinterpret_cast<const bf16*>(t + off0), reinterpret_cast<const bf16*>(t + off1));
}

}  // namespace bs

// Host-side launchers implemented in the .hip files (all enqueue on `stream`).
namespace bs {
// Segments: cu_q/cu_k (NULL: one chunk with diagonal diag_chunk); q_pos/k_pos
// (NULL: diagonal len_k - len_q of each segment, else q_pos[b] - k_pos[b]).
hipError_t launch_plan(PlanKind kind, const int32_t* cu_q, const int32_t* cu_k,
                       const int64_t* q_pos, const int64_t* k_pos, int32_t num_seqs,
                       int64_t total_q, int64_t total_k, int32_t max_seqlen, int32_t diag_chunk,
                       int causal, int tile_a, int tile_b, int64_t max_items, void* ws,
                       const WsLayout& L, hipStream_t stream);

// Forward epilogue that folds the step into a running result instead of writing
// a partial (ring steps merged as they arrive): o_run float32 [T, hq, d], lse_run
// [hq, T] natural log; accumulate = 0 replaces the running state, otherwise the
// two are combined by their log-sum-exp weights.  With `out` non-null the merged
// output goes there in the input dtype and o_run is not written.
struct FwdMerge {
  float* o_run;
  float* lse_run;
  int accumulate;
};

// merge == NULL: plain forward writing (out, lse)
hipError_t launch_fwd_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                           int causal, float scale, void* out, float* lse,
                           const FwdMerge* merge, const void* ws, const WsLayout& L,
                           hipStream_t stream);
// The bf16 dQ kernel also forms D = rowsum(dO * O) and stores it in dvec for the dK/dV
// kernel (the float32 path computes D in launch_bwd_preprocess).
hipError_t launch_dq_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                          const void* out, const void* dout, const float* lse, float* dvec,
                          int causal, float scale, void* dq, float* dq_acc, const void* ws,
                          const WsLayout& L, hipStream_t stream);
hipError_t launch_dkdv_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                            const void* dout, const float* lse, const float* dvec, int causal,
                            float scale, void* dk, void* dv, int kv_accumulate, const void* ws,
                            const WsLayout& L, hipStream_t stream);

hipError_t launch_fwd_f32(const bs_dims& dims, const void* q, const void* k, const void* v,
                          int causal, float scale, void* out, float* lse, const FwdMerge* merge,
                          const void* ws, const WsLayout& L, hipStream_t stream);
hipError_t launch_bwd_f32_dq(const bs_dims& dims, const void* q, const void* k, const void* v,
                             const float* lse, const void* dout, const float* dvec, int causal,
                             float scale, float* dq_acc, const void* ws, const WsLayout& L,
                             hipStream_t stream);
hipError_t launch_bwd_f32_dkdv(const bs_dims& dims, const void* q, const void* k, const void* v,
                               const float* lse, const void* dout, const float* dvec, int causal,
                               float scale, void* dk, void* dv, int kv_accumulate,
                               const void* ws, const WsLayout& L, hipStream_t stream);

hipError_t launch_bwd_preprocess(const bs_dims& dims, const void* out, const void* dout,
                                 float* dvec, float* dq_acc_to_zero, const void* ws,
                                 hipStream_t stream);
hipError_t launch_dq_finalize(const bs_dims& dims, const float* dq_acc, void* dq,
                              const void* ws, hipStream_t stream);
hipError_t launch_lse_merge(const bs_dims& dims, const void* out_parts, const float* lse_parts,
                            int32_t n, void* out, float* lse, hipStream_t stream);
}  // namespace bs
