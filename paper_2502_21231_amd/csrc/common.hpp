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
hipError_t launch_bwd_bf16(const bs_dims& dims, const void* q, const void* k, const void* v,
                           const void* dout, const float* lse, const float* dvec, float* dq_acc,
                           int causal, float scale, void* dk, void* dv, const void* ws,
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
                               float scale, void* dk, void* dv, const void* ws,
                               const WsLayout& L, hipStream_t stream);

hipError_t launch_bwd_preprocess(const bs_dims& dims, const void* out, const void* dout,
                                 float* dvec, float* dq_acc_to_zero, const void* ws,
                                 hipStream_t stream);
hipError_t launch_dq_finalize(const bs_dims& dims, const float* dq_acc, void* dq,
                              const void* ws, hipStream_t stream);
hipError_t launch_lse_merge(const bs_dims& dims, const void* out_parts, const float* lse_parts,
                            int32_t n, void* out, float* lse, hipStream_t stream);
}  // namespace bs
