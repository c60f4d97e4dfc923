// Definitions shared by every HIP source of libbs_attn.so (gfx950 only): vector types,
// constants and device helpers.  The attention kernels' work list, tile shapes, LDS
// layouts and launchers are in attn.hpp.
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
// Device-side helpers --------------------------------------------------------

__device__ __forceinline__ float bf2f(bf16 x) { return (float)x; }
__device__ __forceinline__ bf16 f2bf(float x) { return (bf16)x; }  // RNE on gfx950

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Max / sum of this lane's value and lane (l ^ 32)'s: v_permlane32_swap exchanges the two
// 32-lane halves of a register pair in the vector unit (a shuffle would go through LDS and
// wait for every outstanding LDS read).  Both lanes of a pair get the same bits.
__device__ __forceinline__ float half_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// s_waitcnt vmcnt(0) (expcnt and lgkmcnt left unconstrained): all of this
// wave's outstanding vector-memory loads have returned.
__device__ __forceinline__ void wait_vmem_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Workgroup barrier that orders LDS traffic only: waits for this wave's LDS
// operations (lgkmcnt) but not for its outstanding global loads, so that copies
// into another buffer stay in flight across it.  The memory clobber keeps the
// compiler from moving memory operations across it.
__device__ __forceinline__ void barrier_lds() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Instruction classes of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedMfma = 0x008, kSchedVmem = 0x010, kSchedDsRead = 0x100;

// Fused softmax cross-entropy (xent.hip).
hipError_t launch_softmax_xent(int64_t rows, int64_t vocab, int dtype, const void* logits,
                               const int64_t* labels, int64_t ignore_index, float grad_scale,
                               float* loss, float* lse, void* dlogits, hipStream_t stream);

}  // namespace bs
