// C ABI of libbs_attn.so: argument validation, workspace layout, launch order.
// The declarations and the contract of every entry point are in bs_attn.h.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <vector>

#include "attn.hpp"

// Scratch of the allocation-free forward (bs_attn_varlen_fwd_noalloc): the plan that the
// forward kernel walks (header, per-segment offsets, work list).  Each device holds its own
// copy from the time the library's code is loaded on it until the process ends.  Host code
// never uses this name as an address: the device address comes from hipGetSymbolAddress.
constexpr size_t kNoAllocScratchBytes = BS_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace bs {
namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return BS_OK;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(BS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int64_t kMaxTokens = int64_t(1) << 30;
// query heads: keeps the byte offsets inside one tile of rows below 2^31
constexpr int32_t kMaxHeads = 4096;

// Profiling: pairs of HIP events recorded around each kernel launch while enabled.
struct Profiler {
  std::mutex mu;
  std::atomic<bool> on{false};
  std::vector<std::pair<hipEvent_t, hipEvent_t>> recs[BS_KERNEL_COUNT];
  std::vector<hipEvent_t> spare;
};

Profiler& prof() {
  static Profiler* p = new Profiler();  // never destroyed: events may outlive static teardown
  return *p;
}

hipEvent_t take_event() {
  Profiler& P = prof();
  std::lock_guard<std::mutex> g(P.mu);
  if (!P.spare.empty()) {
    hipEvent_t e = P.spare.back();
    P.spare.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void give_back(hipEvent_t e) {
  if (e == nullptr) return;
  Profiler& P = prof();
  std::lock_guard<std::mutex> g(P.mu);
  P.spare.push_back(e);
}

// Records an event pair around the launches made during its lifetime (none when an event
// cannot be had: the one that was is returned to the pool).
class ProfScope {
 public:
  ProfScope(int kind, hipStream_t s) : kind_(kind), s_(s) {
    if (!prof().on.load(std::memory_order_relaxed)) return;
    a_ = take_event();
    b_ = take_event();
    if (a_ && b_) {
      hipEventRecord(a_, s_);
    } else {
      give_back(a_);
      give_back(b_);
      a_ = b_ = nullptr;
    }
  }
  ~ProfScope() {
    if (!a_ || !b_) return;
    hipEventRecord(b_, s_);
    Profiler& P = prof();
    std::lock_guard<std::mutex> g(P.mu);
    P.recs[kind_].emplace_back(a_, b_);
  }

 private:
  int kind_;
  hipStream_t s_;
  hipEvent_t a_ = nullptr, b_ = nullptr;
};

struct PlanCfg {
  PlanKind kind;
  int tile_a, tile_b;
};

bool is_bwd(int op) {
  return op == BS_OP_VARLEN_BWD || op == BS_OP_CHUNK_BWD || op == BS_OP_PACKED_CHUNK_BWD;
}
// ops whose problem is a list of segments (cu_seqlens)
bool is_varlen(int op) {
  return op == BS_OP_VARLEN_FWD || op == BS_OP_VARLEN_BWD || op == BS_OP_PACKED_CHUNK_FWD ||
         op == BS_OP_PACKED_CHUNK_BWD;
}
// segment ops whose diagonals come from per-segment global positions
bool is_packed(int op) { return op == BS_OP_PACKED_CHUNK_FWD || op == BS_OP_PACKED_CHUNK_BWD; }
// the backward that writes dQ itself (the others add into the caller's fp32 dq_accum)
bool writes_dq(int op) { return op == BS_OP_VARLEN_BWD; }
bool valid_op(int op) { return op >= BS_OP_VARLEN_FWD && op <= BS_OP_PACKED_CHUNK_BWD; }

// Plans an op runs, in launch order: the forward walks query tiles; the
// backward plans twice, query tiles for its dQ kernel, then key tiles for its
// dK/dV kernel.
int plans_of(int op, const bs_dims& d, PlanCfg out[2]) {
  if (d.dtype == BS_BF16) {
    out[0] = PlanCfg{kPlanFwd, kFwdBM, kFwdBN};
    out[1] = PlanCfg{kPlanBwd, kBwdBN, bwd_bm(d.head_dim)};
  } else {
    out[0] = PlanCfg{kPlanFwd, kF32BM, kF32BN};
    out[1] = PlanCfg{kPlanBwd, kF32BN, kF32BM};
  }
  return is_bwd(op) ? 2 : 1;
}

int64_t max_items_of(const PlanCfg& c, const bs_dims& d, int64_t nseg, bool varlen) {
  const int64_t ta = c.kind == kPlanFwd ? d.total_q : d.total_k;
  return (ta + c.tile_a - 1) / c.tile_a + (varlen ? nseg : 0);
}

int check_dims(const bs_dims* d, bool need_kv) {
  if (d == nullptr) return fail(BS_ERR_INVALID_ARG, "dims is NULL");
  if (d->dtype != BS_F32 && d->dtype != BS_BF16)
    return fail(BS_ERR_UNSUPPORTED, "dtype %d is not BS_F32 or BS_BF16", d->dtype);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(BS_ERR_UNSUPPORTED, "head_dim %d is not 64 or 128", d->head_dim);
  if (d->hq < 1 || d->hq > kMaxHeads)
    return fail(BS_ERR_INVALID_ARG, "hq = %d out of [1, %d]", d->hq, kMaxHeads);
  if (d->total_q < 0 || d->total_q >= kMaxTokens)
    return fail(BS_ERR_INVALID_ARG, "total_q = %lld out of [0, 2^30)", (long long)d->total_q);
  if (need_kv) {
    if (d->hkv < 1 || d->hq % d->hkv != 0)
      return fail(BS_ERR_INVALID_ARG, "hq = %d must be a positive multiple of hkv = %d", d->hq, d->hkv);
    if (d->total_k < 0 || d->total_k >= kMaxTokens)
      return fail(BS_ERR_INVALID_ARG, "total_k = %lld out of [0, 2^30)", (long long)d->total_k);
  }
  return BS_OK;
}

int check_ptr(const void* p, int64_t count, const char* name) {
  if (count == 0) return BS_OK;
  if (p == nullptr) return fail(BS_ERR_INVALID_ARG, "%s is NULL", name);
  if (reinterpret_cast<uintptr_t>(p) % 16 != 0)
    return fail(BS_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return BS_OK;
}

int check_scale(float s) {
  if (!isfinite(s) || !(s > 0.f)) return fail(BS_ERR_INVALID_ARG, "scale must be finite and > 0");
  return BS_OK;
}

WsLayout layout_of(int op, const bs_dims& d, int64_t nseg) {
  WsLayout L = {};
  PlanCfg cfg[2];
  const int np = plans_of(op, d, cfg);
  const bool varlen = is_varlen(op);
  int64_t mi = 0;
  for (int i = 0; i < np; ++i) {
    const int64_t m = max_items_of(cfg[i], d, nseg, varlen);
    mi = m > mi ? m : mi;
  }
  size_t off = align256(sizeof(WsHeader));
  L.seg_off = off;
  off += align256(sizeof(int32_t) * (size_t)(nseg + 2));
  L.seg_dst = off;
  off += align256(sizeof(int32_t) * (size_t)(nseg + 1));
  L.sorted = off;
  off += align256(sizeof(WorkItem) * (size_t)mi);
  if (is_bwd(op)) {
    L.dvec = off;
    off += align256(sizeof(float) * (size_t)(d.hq * d.total_q));
    if (writes_dq(op) && d.dtype == BS_F32) {  // the float32 dQ kernel accumulates
      L.dq_acc = off;
      off += align256(sizeof(float) * (size_t)(d.total_q * d.hq * d.head_dim));
    }
  }
  L.total = off;
  L.max_items = mi;
  return L;
}

int check_ws(const WsLayout& L, const void* ws, size_t bytes) {
  if (ws == nullptr) return fail(BS_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % 256 != 0)
    return fail(BS_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (bytes < L.total)
    return fail(BS_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", bytes,
                L.total);
  return BS_OK;
}

// Runs plan `i` of the op; returns the layout with max_items set for that plan.
hipError_t run_plan(int op, const bs_dims& d, int i, const int32_t* cu_q, const int32_t* cu_k,
                    const int64_t* q_pos, const int64_t* k_pos, int32_t num_seqs,
                    int32_t max_seqlen, int64_t q_off, int64_t k_off, int causal, void* ws,
                    const WsLayout& L, WsLayout* Lp, hipStream_t s) {
  PlanCfg cfg[2];
  plans_of(op, d, cfg);
  const bool varlen = is_varlen(op);
  *Lp = L;
  Lp->max_items = max_items_of(cfg[i], d, varlen ? num_seqs : 1, varlen);
  int64_t diag = q_off - k_off;
  diag = diag < -kDiagClamp ? -kDiagClamp : (diag > kDiagClamp ? kDiagClamp : diag);
  const bool packed = is_packed(op);
  return launch_plan(cfg[i].kind, varlen ? cu_q : nullptr, varlen ? cu_k : nullptr,
                     packed ? q_pos : nullptr, packed ? k_pos : nullptr,
                     varlen ? num_seqs : 1, d.total_q, d.total_k, max_seqlen, (int32_t)diag,
                     causal, cfg[i].tile_a, cfg[i].tile_b, Lp->max_items, ws, *Lp, s);
}

int check_varlen_args(int op, const int32_t* cu_q, const int32_t* cu_k, const int64_t* q_pos,
                      const int64_t* k_pos, int32_t num_seqs, int32_t max_seqlen) {
  if (num_seqs < 0) return fail(BS_ERR_INVALID_ARG, "num_seqs = %d < 0", num_seqs);
  if (max_seqlen < 0) return fail(BS_ERR_INVALID_ARG, "max_seqlen = %d < 0", max_seqlen);
  if (cu_q == nullptr || cu_k == nullptr) return fail(BS_ERR_INVALID_ARG, "cu_seqlens is NULL");
  if (is_packed(op) && num_seqs > 0 && (q_pos == nullptr || k_pos == nullptr))
    return fail(BS_ERR_INVALID_ARG, "q_pos / k_pos is NULL");
  return BS_OK;
}

#define BS_TRY(x)                 \
  do {                            \
    int rc__ = (x);               \
    if (rc__ != BS_OK) return rc__; \
  } while (0)
#define BS_HIP(x, what)                        \
  do {                                         \
    hipError_t e__ = (x);                      \
    if (e__ != hipSuccess) return hip_fail(e__, what); \
  } while (0)

// True when the byte ranges [a, a + na) and [b, b + nb) intersect.
bool overlaps(const void* a, int64_t na, const void* b, int64_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return na > 0 && nb > 0 && x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

// merge == NULL: writes the step's (out, lse).  Otherwise folds the step into the
// running (merge->o_run, merge->lse_run); out is then optional (the final output).
int fwd_common(int op, const bs_dims* dims, const void* q, const void* k, const void* v,
               const int32_t* cu_q, const int32_t* cu_k, const int64_t* q_pos,
               const int64_t* k_pos, int32_t num_seqs, int32_t max_seqlen, int64_t q_off,
               int64_t k_off, int causal, float scale, void* out, float* lse,
               const FwdMerge* merge, void* ws, size_t ws_bytes, void* stream) {
  BS_TRY(check_dims(dims, true));
  const bs_dims& d = *dims;
  const int64_t qn = d.total_q * d.hq * d.head_dim, kn = d.total_k * d.hkv * d.head_dim;
  BS_TRY(check_ptr(q, qn, "q"));
  BS_TRY(check_ptr(k, kn, "k"));
  BS_TRY(check_ptr(v, kn, "v"));
  if (merge == nullptr) {
    BS_TRY(check_ptr(out, qn, "out"));
    BS_TRY(check_ptr(lse, d.total_q * d.hq, "lse"));
  } else {
    BS_TRY(check_ptr(merge->o_run, qn, "o_run"));
    BS_TRY(check_ptr(merge->lse_run, d.total_q * d.hq, "lse_run"));
    if (out != nullptr) {
      BS_TRY(check_ptr(out, qn, "out"));
      if (overlaps(out, qn * (d.dtype == BS_BF16 ? 2 : 4), merge->o_run, qn * 4))
        return fail(BS_ERR_INVALID_ARG, "out overlaps o_run");
    }
  }
  BS_TRY(check_scale(scale));
  if (is_varlen(op)) BS_TRY(check_varlen_args(op, cu_q, cu_k, q_pos, k_pos, num_seqs, max_seqlen));
  const WsLayout L = layout_of(op, d, is_varlen(op) ? num_seqs : 1);
  BS_TRY(check_ws(L, ws, ws_bytes));
  hipStream_t s = static_cast<hipStream_t>(stream);
  WsLayout Lp;
  {
    ProfScope ps(BS_KERNEL_PLAN, s);
    BS_HIP(run_plan(op, d, 0, cu_q, cu_k, q_pos, k_pos, num_seqs, max_seqlen, q_off, k_off,
                    causal, ws, L, &Lp, s),
           "planner launch");
  }
  ProfScope ps(BS_KERNEL_FWD, s);
  if (d.dtype == BS_BF16)
    BS_HIP(launch_fwd_bf16(d, q, k, v, causal, scale, out, lse, merge, ws, Lp, s),
           "forward launch");
  else
    BS_HIP(launch_fwd_f32(d, q, k, v, causal, scale, out, lse, merge, ws, Lp, s),
           "forward launch");
  return ok();
}

int bwd_common(int op, const bs_dims* dims, const void* q, const void* k, const void* v,
               const void* out, const float* lse, const void* dout, const int32_t* cu_q,
               const int32_t* cu_k, const int64_t* q_pos, const int64_t* k_pos,
               int32_t num_seqs, int32_t max_seqlen, int64_t q_off, int64_t k_off, int causal,
               float scale, float* dq_accum, void* dq, void* dk, void* dv, int kv_accumulate,
               void* ws, size_t ws_bytes, void* stream) {
  BS_TRY(check_dims(dims, true));
  const bs_dims& d = *dims;
  const int64_t qn = d.total_q * d.hq * d.head_dim, kn = d.total_k * d.hkv * d.head_dim;
  BS_TRY(check_ptr(q, qn, "q"));
  BS_TRY(check_ptr(k, kn, "k"));
  BS_TRY(check_ptr(v, kn, "v"));
  BS_TRY(check_ptr(out, qn, "out"));
  BS_TRY(check_ptr(lse, d.total_q * d.hq, "lse"));
  BS_TRY(check_ptr(dout, qn, "dout"));
  BS_TRY(check_ptr(dk, kn, "dk"));
  BS_TRY(check_ptr(dv, kn, "dv"));
  const bool varlen = is_varlen(op), direct = writes_dq(op);
  if (direct) BS_TRY(check_ptr(dq, qn, "dq"));
  else BS_TRY(check_ptr(dq_accum, qn, "dq_accum"));
  BS_TRY(check_scale(scale));
  if (varlen) BS_TRY(check_varlen_args(op, cu_q, cu_k, q_pos, k_pos, num_seqs, max_seqlen));
  const WsLayout L = layout_of(op, d, varlen ? num_seqs : 1);
  BS_TRY(check_ws(L, ws, ws_bytes));
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* base = static_cast<char*>(ws);
  float* dvec = reinterpret_cast<float*>(base + L.dvec);
  const bool f32 = d.dtype == BS_F32;
  float* acc = direct ? (f32 ? reinterpret_cast<float*>(base + L.dq_acc) : nullptr) : dq_accum;
  WsLayout Lp;
  {
    ProfScope ps(BS_KERNEL_PLAN, s);
    BS_HIP(run_plan(op, d, 0, cu_q, cu_k, q_pos, k_pos, num_seqs, max_seqlen, q_off, k_off,
                    causal, ws, L, &Lp, s),
           "planner launch");
  }
  if (f32) {  // the bf16 dQ kernel forms D itself
    ProfScope ps(BS_KERNEL_PREPROCESS, s);
    BS_HIP(launch_bwd_preprocess(d, out, dout, dvec, direct ? acc : nullptr, ws, s),
           "preprocess launch");
  }
  {
    ProfScope ps(BS_KERNEL_BWD_DQ, s);
    if (f32)
      BS_HIP(launch_bwd_f32_dq(d, q, k, v, lse, dout, dvec, causal, scale, acc, ws, Lp, s),
             "backward dQ launch");
    else
      BS_HIP(launch_dq_bf16(d, q, k, v, out, dout, lse, dvec, causal, scale, direct ? dq : nullptr,
                            acc, ws, Lp, s),
             "backward dQ launch");
  }
  {
    ProfScope ps(BS_KERNEL_PLAN, s);
    BS_HIP(run_plan(op, d, 1, cu_q, cu_k, q_pos, k_pos, num_seqs, max_seqlen, q_off, k_off,
                    causal, ws, L, &Lp, s),
           "planner launch");
  }
  {
    ProfScope ps(BS_KERNEL_BWD_DKDV, s);
    if (f32)
      BS_HIP(launch_bwd_f32_dkdv(d, q, k, v, lse, dout, dvec, causal, scale, dk, dv, kv_accumulate,
                                 ws, Lp, s),
             "backward dK/dV launch");
    else
      BS_HIP(launch_dkdv_bf16(d, q, k, v, dout, lse, dvec, causal, scale, dk, dv, kv_accumulate,
                              ws, Lp, s),
             "backward dK/dV launch");
  }
  if (direct && f32) {
    ProfScope ps(BS_KERNEL_FINALIZE, s);
    BS_HIP(launch_dq_finalize(d, acc, dq, ws, s), "dQ finalize launch");
  }
  return ok();
}

// Device address of `scratch` on each device, looked up once per device (with that device
// current) on the first allocation-free call made there.
constexpr int kMaxScratchDevices = 256;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxScratchDevices] = {};

int noalloc_scratch(void* stream, void** addr) {
  int dev = -1;
  BS_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (stream != nullptr) {
    int sdev = -1;
    BS_HIP(hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev), "hipStreamGetDevice");
    if (sdev != dev)
      return fail(BS_ERR_INVALID_ARG, "stream belongs to device %d but device %d is current", sdev,
                  dev);
  }
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(BS_ERR_UNSUPPORTED, "device %d is beyond the %d devices with scratch slots", dev,
                kMaxScratchDevices);
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (g_scratch_addr[dev] == nullptr) {
    void* p = nullptr;
    BS_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (p == nullptr) return fail(BS_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_addr[dev] = p;
  }
  *addr = g_scratch_addr[dev];
  return BS_OK;
}

}  // namespace
}  // namespace bs

using namespace bs;

extern "C" {

size_t bs_attn_workspace_size(int op, const bs_dims* dims, int32_t num_seqs, int32_t max_seqlen) {
  if (!valid_op(op)) {
    fail(BS_ERR_UNSUPPORTED, "unknown op %d", op);
    return 0;
  }
  if (check_dims(dims, true) != BS_OK) return 0;
  if (is_varlen(op) && (num_seqs < 0 || max_seqlen < 0)) {
    fail(BS_ERR_INVALID_ARG, "num_seqs and max_seqlen must be >= 0");
    return 0;
  }
  ok();
  return layout_of(op, *dims, is_varlen(op) ? num_seqs : 1).total;
}

int bs_attn_varlen_fwd(const bs_dims* dims, const void* q, const void* k, const void* v,
                       const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k, int32_t num_seqs,
                       int32_t max_seqlen, int causal, float scale, void* out, float* lse,
                       void* workspace, size_t workspace_bytes, void* stream) {
  return fwd_common(BS_OP_VARLEN_FWD, dims, q, k, v, cu_seqlens_q, cu_seqlens_k, nullptr, nullptr,
                    num_seqs, max_seqlen, 0, 0, causal, scale, out, lse, nullptr, workspace,
                    workspace_bytes, stream);
}

int bs_attn_varlen_fwd_noalloc(const bs_dims* dims, const void* q, const void* k, const void* v,
                               const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                               int32_t num_seqs, int32_t max_seqlen, int causal, float scale,
                               void* out, float* lse, void* stream) {
  BS_TRY(check_dims(dims, true));
  BS_TRY(check_varlen_args(BS_OP_VARLEN_FWD, cu_seqlens_q, cu_seqlens_k, nullptr, nullptr,
                           num_seqs, max_seqlen));
  const size_t need = layout_of(BS_OP_VARLEN_FWD, *dims, num_seqs).total;
  if (need > kNoAllocScratchBytes)
    return fail(BS_ERR_WORKSPACE,
                "these sizes need %zu bytes of plan scratch, more than the %zu bytes of the "
                "allocation-free forward (use bs_attn_varlen_fwd with a workspace)",
                need, kNoAllocScratchBytes);
  void* ws = nullptr;
  BS_TRY(noalloc_scratch(stream, &ws));
  return fwd_common(BS_OP_VARLEN_FWD, dims, q, k, v, cu_seqlens_q, cu_seqlens_k, nullptr, nullptr,
                    num_seqs, max_seqlen, 0, 0, causal, scale, out, lse, nullptr, ws,
                    kNoAllocScratchBytes, stream);
}

int bs_attn_varlen_bwd(const bs_dims* dims, const void* q, const void* k, const void* v,
                       const void* out, const float* lse, const void* dout,
                       const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k, int32_t num_seqs,
                       int32_t max_seqlen, int causal, float scale, void* dq, void* dk, void* dv,
                       void* workspace, size_t workspace_bytes, void* stream) {
  return bwd_common(BS_OP_VARLEN_BWD, dims, q, k, v, out, lse, dout, cu_seqlens_q, cu_seqlens_k,
                    nullptr, nullptr, num_seqs, max_seqlen, 0, 0, causal, scale, nullptr, dq, dk,
                    dv, 0, workspace, workspace_bytes, stream);
}

int bs_attn_chunk_fwd(const bs_dims* dims, const void* q, const void* k, const void* v,
                      int64_t q_pos_offset, int64_t k_pos_offset, int causal, float scale,
                      void* out, float* lse, void* workspace, size_t workspace_bytes,
                      void* stream) {
  return fwd_common(BS_OP_CHUNK_FWD, dims, q, k, v, nullptr, nullptr, nullptr, nullptr, 1, 0,
                    q_pos_offset, k_pos_offset, causal, scale, out, lse, nullptr, workspace,
                    workspace_bytes, stream);
}

int bs_attn_chunk_fwd_merge(const bs_dims* dims, const void* q, const void* k, const void* v,
                            int64_t q_pos_offset, int64_t k_pos_offset, int causal, float scale,
                            float* o_run, float* lse_run, int accumulate, void* out,
                            void* workspace, size_t workspace_bytes, void* stream) {
  const FwdMerge m{o_run, lse_run, accumulate != 0};
  return fwd_common(BS_OP_CHUNK_FWD, dims, q, k, v, nullptr, nullptr, nullptr, nullptr, 1, 0,
                    q_pos_offset, k_pos_offset, causal, scale, out, nullptr, &m, workspace,
                    workspace_bytes, stream);
}

int bs_attn_chunk_bwd(const bs_dims* dims, const void* q, const void* k, const void* v,
                      const void* out_merged, const float* lse_merged, const void* dout,
                      int64_t q_pos_offset, int64_t k_pos_offset, int causal, float scale,
                      float* dq_accum, void* dk, void* dv, int kv_accumulate, void* workspace,
                      size_t workspace_bytes, void* stream) {
  return bwd_common(BS_OP_CHUNK_BWD, dims, q, k, v, out_merged, lse_merged, dout, nullptr, nullptr,
                    nullptr, nullptr, 1, 0, q_pos_offset, k_pos_offset, causal, scale, dq_accum,
                    nullptr, dk, dv, kv_accumulate != 0, workspace, workspace_bytes, stream);
}

int bs_attn_packed_chunk_fwd(const bs_dims* dims, const void* q, const void* k, const void* v,
                             const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                             const int64_t* q_pos, const int64_t* k_pos, int32_t num_seqs,
                             int32_t max_seqlen, int causal, float scale, void* out, float* lse,
                             void* workspace, size_t workspace_bytes, void* stream) {
  return fwd_common(BS_OP_PACKED_CHUNK_FWD, dims, q, k, v, cu_seqlens_q, cu_seqlens_k, q_pos,
                    k_pos, num_seqs, max_seqlen, 0, 0, causal, scale, out, lse, nullptr,
                    workspace, workspace_bytes, stream);
}

int bs_attn_packed_chunk_fwd_merge(const bs_dims* dims, const void* q, const void* k,
                                   const void* v, const int32_t* cu_seqlens_q,
                                   const int32_t* cu_seqlens_k, const int64_t* q_pos,
                                   const int64_t* k_pos, int32_t num_seqs, int32_t max_seqlen,
                                   int causal, float scale, float* o_run, float* lse_run,
                                   int accumulate, void* out, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  const FwdMerge m{o_run, lse_run, accumulate != 0};
  return fwd_common(BS_OP_PACKED_CHUNK_FWD, dims, q, k, v, cu_seqlens_q, cu_seqlens_k, q_pos,
                    k_pos, num_seqs, max_seqlen, 0, 0, causal, scale, out, nullptr, &m,
                    workspace, workspace_bytes, stream);
}

int bs_attn_packed_chunk_bwd(const bs_dims* dims, const void* q, const void* k, const void* v,
                             const void* out_merged, const float* lse_merged, const void* dout,
                             const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                             const int64_t* q_pos, const int64_t* k_pos, int32_t num_seqs,
                             int32_t max_seqlen, int causal, float scale, float* dq_accum,
                             void* dk, void* dv, int kv_accumulate, void* workspace,
                             size_t workspace_bytes, void* stream) {
  return bwd_common(BS_OP_PACKED_CHUNK_BWD, dims, q, k, v, out_merged, lse_merged, dout,
                    cu_seqlens_q, cu_seqlens_k, q_pos, k_pos, num_seqs, max_seqlen, 0, 0, causal,
                    scale, dq_accum, nullptr, dk, dv, kv_accumulate != 0, workspace,
                    workspace_bytes, stream);
}

int bs_dq_finalize(const bs_dims* dims, const float* dq_accum, void* dq, void* stream) {
  BS_TRY(check_dims(dims, false));
  const int64_t qn = dims->total_q * dims->hq * dims->head_dim;
  BS_TRY(check_ptr(dq_accum, qn, "dq_accum"));
  BS_TRY(check_ptr(dq, qn, "dq"));
  ProfScope ps(BS_KERNEL_FINALIZE, static_cast<hipStream_t>(stream));
  BS_HIP(launch_dq_finalize(*dims, dq_accum, dq, nullptr, static_cast<hipStream_t>(stream)),
         "dQ finalize launch");
  return ok();
}

int bs_lse_merge(const bs_dims* dims, const void* out_partials, const float* lse_partials,
                 int32_t n, void* out, float* lse, void* stream) {
  BS_TRY(check_dims(dims, false));
  if (n < 1) return fail(BS_ERR_INVALID_ARG, "n = %d must be >= 1", n);
  const int64_t qn = dims->total_q * dims->hq * dims->head_dim;
  BS_TRY(check_ptr(out_partials, qn * n, "out_partials"));
  BS_TRY(check_ptr(lse_partials, dims->total_q * dims->hq * n, "lse_partials"));
  BS_TRY(check_ptr(out, qn, "out"));
  BS_TRY(check_ptr(lse, dims->total_q * dims->hq, "lse"));
  ProfScope ps(BS_KERNEL_MERGE, static_cast<hipStream_t>(stream));
  BS_HIP(launch_lse_merge(*dims, out_partials, lse_partials, n, out, lse,
                          static_cast<hipStream_t>(stream)),
         "merge launch");
  return ok();
}

int bs_copy_async(void* dst, const void* src, size_t bytes, void* stream) {
  if (bytes == 0) return ok();
  if (dst == nullptr || src == nullptr) return fail(BS_ERR_INVALID_ARG, "dst or src is NULL");
  if (bytes > (size_t)INT64_MAX || overlaps(dst, (int64_t)bytes, src, (int64_t)bytes))
    return fail(BS_ERR_INVALID_ARG, "dst and src overlap");
  BS_HIP(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDeviceNoCU,
                        static_cast<hipStream_t>(stream)),
         "DMA copy");
  return ok();
}

int bs_softmax_xent(int64_t rows, int64_t vocab, int dtype, const void* logits,
                    const int64_t* labels, int64_t ignore_index, float grad_scale, float* loss,
                    float* lse, void* dlogits, void* stream) {
  if (dtype != BS_F32 && dtype != BS_BF16)
    return fail(BS_ERR_UNSUPPORTED, "dtype %d is not BS_F32 or BS_BF16", dtype);
  if (rows < 0 || rows >= kMaxTokens)
    return fail(BS_ERR_INVALID_ARG, "rows = %lld out of [0, 2^30)", (long long)rows);
  if (vocab < 1 || vocab > INT32_MAX)
    return fail(BS_ERR_INVALID_ARG, "vocab = %lld out of [1, 2^31)", (long long)vocab);
  if (!isfinite(grad_scale)) return fail(BS_ERR_INVALID_ARG, "grad_scale must be finite");
  if (rows == 0) return ok();
  if (logits == nullptr || labels == nullptr || loss == nullptr)
    return fail(BS_ERR_INVALID_ARG, "logits, labels or loss is NULL");
  const int64_t esize = dtype == BS_BF16 ? 2 : 4;
  if (reinterpret_cast<uintptr_t>(logits) % esize != 0 ||
      (dlogits != nullptr && reinterpret_cast<uintptr_t>(dlogits) % esize != 0))
    return fail(BS_ERR_INVALID_ARG, "logits / dlogits not aligned to their element size");
  if (reinterpret_cast<uintptr_t>(labels) % 8 != 0 || reinterpret_cast<uintptr_t>(loss) % 4 != 0 ||
      (lse != nullptr && reinterpret_cast<uintptr_t>(lse) % 4 != 0))
    return fail(BS_ERR_INVALID_ARG, "labels / loss / lse not aligned to their element size");
  if (rows > INT64_MAX / esize / vocab)
    return fail(BS_ERR_INVALID_ARG, "rows * vocab elements exceed the address range");
  const int64_t nbytes = rows * vocab * esize;
  if (dlogits != nullptr && dlogits != logits && overlaps(dlogits, nbytes, logits, nbytes))
    return fail(BS_ERR_INVALID_ARG, "dlogits overlaps logits without being equal to it");
  ProfScope ps(BS_KERNEL_XENT, static_cast<hipStream_t>(stream));
  BS_HIP(launch_softmax_xent(rows, vocab, dtype, logits, labels, ignore_index, grad_scale, loss,
                             lse, dlogits, static_cast<hipStream_t>(stream)),
         "cross-entropy launch");
  return ok();
}

int bs_read_device_status(const void* workspace, void* stream) {
  if (workspace == nullptr) return fail(BS_ERR_WORKSPACE, "workspace is NULL");
  WsHeader h;
  hipStream_t s = static_cast<hipStream_t>(stream);
  BS_HIP(hipMemcpyAsync(&h, workspace, sizeof(h), hipMemcpyDeviceToHost, s), "status copy");
  BS_HIP(hipStreamSynchronize(s), "status sync");
  if (h.status != BS_DEV_OK)
    return fail(BS_ERR_DEVICE_STATUS, "device planner rejected cu_seqlens: code %d", h.status);
  return ok();
}

int bs_attn_plan_export(int op, const bs_dims* dims, const int32_t* cu_seqlens_q,
                        const int32_t* cu_seqlens_k, int32_t num_seqs, int32_t max_seqlen,
                        int64_t q_pos_offset, int64_t k_pos_offset, const int64_t* q_pos,
                        const int64_t* k_pos, int causal, void* workspace,
                        size_t workspace_bytes, int32_t* host_items, size_t capacity,
                        size_t* count, int32_t* tile_m, int32_t* tile_n, void* stream) {
  if (!valid_op(op)) return fail(BS_ERR_UNSUPPORTED, "unknown op %d", op);
  BS_TRY(check_dims(dims, true));
  if (count == nullptr || (capacity > 0 && host_items == nullptr))
    return fail(BS_ERR_INVALID_ARG, "count / host_items is NULL");
  const bool varlen = is_varlen(op);
  if (varlen)
    BS_TRY(check_varlen_args(op, cu_seqlens_q, cu_seqlens_k, q_pos, k_pos, num_seqs, max_seqlen));
  const WsLayout L = layout_of(op, *dims, varlen ? num_seqs : 1);
  BS_TRY(check_ws(L, workspace, workspace_bytes));
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the plan the op's main kernel walks: the last one of the op
  PlanCfg cfg[2];
  const int np = plans_of(op, *dims, cfg);
  WsLayout Lp;
  BS_HIP(run_plan(op, *dims, np - 1, cu_seqlens_q, cu_seqlens_k, q_pos, k_pos, num_seqs,
                  max_seqlen, q_pos_offset, k_pos_offset, causal, workspace, L, &Lp, s),
         "planner launch");
  WsHeader h;
  BS_HIP(hipMemcpyAsync(&h, workspace, sizeof(h), hipMemcpyDeviceToHost, s), "plan copy");
  BS_HIP(hipStreamSynchronize(s), "plan sync");
  if (h.status != BS_DEV_OK)
    return fail(BS_ERR_DEVICE_STATUS, "device planner rejected cu_seqlens: code %d", h.status);
  const size_t n = (size_t)h.n_items;
  *count = n;
  if (tile_m) *tile_m = cfg[np - 1].kind == kPlanFwd ? cfg[np - 1].tile_a : cfg[np - 1].tile_b;
  if (tile_n) *tile_n = cfg[np - 1].kind == kPlanFwd ? cfg[np - 1].tile_b : cfg[np - 1].tile_a;
  const size_t m = n < capacity ? n : capacity;
  if (m > 0) {
    std::vector<WorkItem> items(m);
    BS_HIP(hipMemcpyAsync(items.data(), static_cast<char*>(workspace) + L.sorted,
                          m * sizeof(WorkItem), hipMemcpyDeviceToHost, s),
           "plan copy");
    BS_HIP(hipStreamSynchronize(s), "plan sync");
    for (size_t i = 0; i < m; ++i) {
      const WorkItem& w = items[i];
      int32_t* o = host_items + 12 * i;
      const int32_t common[6] = {w.seg, w.tile, w.a_start, w.a_rows, w.b_start, w.b_len};
      memcpy(o, common, sizeof(common));
      if (cfg[np - 1].kind == kPlanFwd) {
        o[6] = w.n0; o[7] = w.n1; o[8] = w.diag; o[9] = 0;
      } else {
        o[6] = w.n0; o[7] = w.n1; o[8] = w.n2; o[9] = w.diag;
      }
      o[10] = 0;
      o[11] = 0;
    }
  }
  return ok();
}

int bs_set_profiling(int enable) {
  Profiler& P = prof();
  std::lock_guard<std::mutex> g(P.mu);
  for (auto& v : P.recs) {
    for (auto& pr : v) {
      hipEventSynchronize(pr.second);
      P.spare.push_back(pr.first);
      P.spare.push_back(pr.second);
    }
    v.clear();
  }
  P.on.store(enable != 0);
  return ok();
}

int bs_profile_read(int kind, double* total_ms, int64_t* launches) {
  if (kind < 0 || kind >= BS_KERNEL_COUNT) return fail(BS_ERR_INVALID_ARG, "unknown kernel kind %d", kind);
  if (total_ms == nullptr || launches == nullptr) return fail(BS_ERR_INVALID_ARG, "NULL output");
  Profiler& P = prof();
  std::lock_guard<std::mutex> g(P.mu);
  double sum = 0.0;
  for (auto& pr : P.recs[kind]) {
    BS_HIP(hipEventSynchronize(pr.second), "event sync");
    float ms = 0.f;
    BS_HIP(hipEventElapsedTime(&ms, pr.first, pr.second), "event elapsed");
    sum += ms;
  }
  *total_ms = sum;
  *launches = (int64_t)P.recs[kind].size();
  return ok();
}

const char* bs_last_error(void) { return g_err; }

}  // extern "C"
