// Internal definitions shared by the HIP sources of libbs_attn.so (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/bs_attn.h"

namespace bs {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kDiagClamp = 1 << 30;

// One entry of the ordered work list (12 int32 = 48 bytes).
// Forward (query tile):  seg, tile=qtile, a_start=q_start, a_rows=q_rows,
//                        b_start=k_start, b_len=k_len, n0=n_full, n1=n_tiles, diag.
// Backward (key tile):   seg, tile=ktile, a_start=k_start, a_rows=k_rows,
//                        b_start=q_start, b_len=q_len, n0=qt_first, n1=n_masked,
//                        n2=n_vis, diag.
struct WorkItem {
  int32_t seg, tile, a_start, a_rows, b_start, b_len, n0, n1, n2, diag, pad0, pad1;
};
static_assert(sizeof(WorkItem) == 48, "work item is 12 int32");

enum PlanKind { kPlanFwd = 0, kPlanBwd = 1 };

// Tile sizes of each kernel family.  The forward walks query tiles of kFwdBM rows
// over key tiles of kFwdBN keys; the backward walks key tiles of kBwdBN keys over
// query tiles of kBwdBM rows.  The float32 kernels use their own sizes.
constexpr int kFwdBM = 128, kFwdBN = 64;
constexpr int kBwdBM = 64, kBwdBN = 128;
constexpr int kF32BM = 64, kF32BN = 64;

// Workspace header: status word and item count, then the per-segment item
// offsets, the unsorted and sorted work lists, then op-specific float buffers.
struct WsHeader {
  int32_t status;
  int32_t n_items;
  int32_t pad[62];
};

struct WsLayout {
  size_t seg_off;     // int32[num_seqs + 1]
  size_t unsorted;    // WorkItem[max_items]
  size_t sorted;      // WorkItem[max_items]
  size_t dvec;        // float[hq * T]      (backward: rowsum(dO * O))
  size_t dq_acc;      // float[T * hq * d]  (varlen backward only)
  size_t total;
  int64_t max_items;
};

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Device-side helpers --------------------------------------------------------

__device__ __forceinline__ float bf2f(bf16 x) { return (float)x; }
__device__ __forceinline__ bf16 f2bf(float x) { return (bf16)x; }  // RNE on gfx950

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// s_waitcnt vmcnt(0) (expcnt and lgkmcnt left unconstrained): all of this
// wave's outstanding vector-memory loads have returned.
__device__ __forceinline__ void wait_vmem_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

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

// `p` is tr_lane_ptr(tile, stride, k0, m0, lane); the second read is 8 rows below.
__device__ __forceinline__ bf16x8 lds_read_tr(const bf16* p, int stride) {
  const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
  const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 8 * stride));
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  const i16x8 v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_bit_cast(bf16x8, v);
}

}  // namespace bs

// Host-side launchers implemented in the .hip files (all enqueue on `stream`).
namespace bs {
hipError_t launch_plan(PlanKind kind, const int32_t* cu_q, const int32_t* cu_k, int32_t num_seqs,
                       int64_t total_q, int64_t total_k, int32_t max_seqlen, int32_t diag_chunk,
                       int causal, int tile_a, int tile_b, int64_t max_items, void* ws,
                       const WsLayout& L, hipStream_t stream);

hipError_t launch_fwd_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                           int causal, float scale, void* out, float* lse, const void* ws,
                           const WsLayout& L, hipStream_t stream);
hipError_t launch_dq_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                          const void* dout, const float* lse, const float* dvec, int causal,
                          float scale, void* dq, float* dq_acc, const void* ws, const WsLayout& L,
                          hipStream_t stream);
hipError_t launch_dkdv_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                            const void* dout, const float* lse, const float* dvec, int causal,
                            float scale, void* dk, void* dv, int kv_accumulate, const void* ws,
                            const WsLayout& L, hipStream_t stream);

hipError_t launch_fwd_f32(const bs_dims& dims, const void* q, const void* k, const void* v,
                          int causal, float scale, void* out, float* lse, const void* ws,
                          const WsLayout& L, hipStream_t stream);
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
