// Parameters shared by the two bf16 backward kernels (dq_bf16.hip, dkdv_bf16.hip), which
// recompute P from the saved LSE and need no atomics: the dQ kernel walks query tiles, the
// dK/dV kernel key tiles.
#pragma once

#include "attn.hpp"

namespace bs {

struct BwdParams {
  const bf16* q;
  const bf16* k;
  const bf16* v;
  const bf16* dout;
  const bf16* o;     // dQ kernel: the forward's output, for D = rowsum(dO * O)
  const float* lse;
  const float* dvec;
  float* dvec_out;   // dQ kernel: where it stores D for the dK/dV kernel
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

inline BwdParams make_params(const bs_dims& dims, const void* q, const void* k, const void* v,
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


}  // namespace bs
