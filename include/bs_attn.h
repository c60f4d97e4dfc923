/*
 * bs_attn.h -- C ABI of libbs_attn.so, the per-device attention of ByteScale's
 * Hybrid Data Parallelism (HDP), arXiv 2502.21231, for AMD Instinct MI355X (gfx950).
 *
 * Under HDP every device ends up running causal self-attention in one of two
 * forms (Sec. 5.1, Hybrid Data Parallelism: some ranks hold whole short
 * sequences and compute locally, others hold a slice of a long sequence and
 * join a ring):
 *   - a varlen pass over whole sequences packed into one buffer without padding
 *     and separated by a segmented causal mask (Sec. 2.3, Padding and Packing);
 *   - one context-parallel (CP) step: a Q shard of a long sequence against one
 *     KV shard, masked by global token positions, returning O and the
 *     log-sum-exp so that the steps of a ring can be combined (Sec. 2.4, Long
 *     Context Training; Sec. 7, Dist-attn with packing).
 * Query heads share KV heads in contiguous groups (Sec. 7, GQA): query head h
 * reads KV head h / (hq / hkv).
 *
 * What is computed (softmax attention; the paper cites FlashAttention for it
 * and prints no formula of its own), per segment or chunk and query head:
 *   S = scale * Q K^T over the visible keys,  LSE = log sum_j exp(S_ij),
 *   P = exp(S - LSE),  O = P V.
 * A query row with no visible key gets O = 0 and LSE = -inf.
 * Backward, for the upstream gradient dO:
 *   D = rowsum(dO * O),  dS = P * (dO V^T - D),
 *   dQ = scale dS K,  dK = scale dS^T Q,  dV = P^T dO,
 * with dK and dV summed over the query heads of each KV group.
 *
 * Conventions for every entry point
 *   - All tensor pointers are DEVICE pointers, contiguous, owned by the caller.
 *     The library never allocates device memory on a call; scratch space comes
 *     from a caller-provided workspace sized by bs_attn_workspace_size(), except
 *     for bs_attn_varlen_fwd_noalloc(), which plans into a fixed device array.
 *   - Layouts (row-major):  Q, O, dO, dQ: [T, hq, head_dim];
 *     K, V, dK, dV: [Tk, hkv, head_dim];  LSE and D: float32 [hq, T];
 *     merge partials: O [n, T, hq, head_dim], LSE [n, hq, T]; running merge
 *     state: o_run float32 [T, hq, head_dim], lse_run float32 [hq, T].
 *   - Element type of Q/K/V/O/dO/dQ/dK/dV is dims->dtype: BS_BF16 (bf16 in,
 *     fp32 accumulation, round-to-nearest-even on every bf16 store) or BS_F32.
 *     LSE is always float32 (natural log).
 *   - head_dim must be 64 or 128; 1 <= hq <= 4096 and hq must be a multiple
 *     of hkv.
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL = default
 *     stream) and never synchronises the host, except the two test helpers
 *     bs_read_device_status() and bs_attn_plan_export().
 *   - Host-checkable errors (null pointer, bad sizes, unsupported head_dim,
 *     non-finite or non-positive scale, small workspace) return a status
 *     synchronously, enqueue nothing, and set a thread-local message readable
 *     with bs_last_error().  Data-dependent errors in cu_seqlens (first entry
 *     not 0, decreasing entries, last entry not equal to the total, a segment
 *     longer than max_seqlen) are detected on the device: the planning kernel
 *     writes a status word into the workspace and the compute kernels then
 *     write nothing; bs_read_device_status() reports it.
 *   - Calls that share a workspace must be ordered on one stream.
 */
#ifndef BS_ATTN_H
#define BS_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BS_OK = 0,
  BS_ERR_INVALID_ARG = 1,   /* null pointer, negative size, hq out of range, hq % hkv != 0,
                               bad scale, n < 1 */
  BS_ERR_UNSUPPORTED = 2,   /* head_dim not in {64, 128}, unknown dtype or op */
  BS_ERR_WORKSPACE = 3,     /* workspace pointer null or smaller than required */
  BS_ERR_HIP = 4,           /* a HIP runtime call failed (message names it) */
  BS_ERR_DEVICE_STATUS = 5  /* the device planner rejected cu_seqlens */
} bs_status;

typedef enum { BS_F32 = 0, BS_BF16 = 1 } bs_dtype;

/* Problem sizes shared by every call.  total_q / total_k are the token counts
 * T and Tk of the Q-side and K-side buffers. */
typedef struct {
  int64_t total_q;
  int64_t total_k;
  int32_t hq;
  int32_t hkv;
  int32_t head_dim;
  int32_t dtype; /* bs_dtype */
} bs_dims;

/* Operation codes for bs_attn_workspace_size() and bs_attn_plan_export(). */
enum {
  BS_OP_VARLEN_FWD = 0,
  BS_OP_VARLEN_BWD = 1,
  BS_OP_CHUNK_FWD = 2,
  BS_OP_CHUNK_BWD = 3,
  BS_OP_PACKED_CHUNK_FWD = 4,
  BS_OP_PACKED_CHUNK_BWD = 5
};

/* Device status word values (bs_read_device_status). */
enum {
  BS_DEV_OK = 0,
  BS_DEV_BAD_FIRST = 1,     /* cu_seqlens_[qk][0] != 0 */
  BS_DEV_NOT_MONOTONE = 2,  /* a segment length is negative */
  BS_DEV_BAD_TOTAL = 3,     /* last entry != total_q / total_k */
  BS_DEV_TOO_LONG = 4       /* a segment longer than max_seqlen */
};

/* Bytes of workspace that `op` needs for these sizes (num_seqs, max_seqlen are
 * ignored by the two single-chunk ops).  Returns 0 when the arguments are invalid (then
 * bs_last_error() says why).  The workspace needs no initialisation and holds
 * nothing across calls except what bs_read_device_status() reads. */
size_t bs_attn_workspace_size(int op, const bs_dims* dims, int32_t num_seqs, int32_t max_seqlen);

/* Varlen (packed) forward, Sec. 2.3 Padding and Packing: segment b holds queries
 * cu_seqlens_q[b] .. cu_seqlens_q[b+1]-1 and keys cu_seqlens_k[b] ..
 * cu_seqlens_k[b+1]-1 (int32 device arrays of num_seqs+1 entries).  With
 * causal != 0 key j of a segment is visible to query i iff j <= i + len_k - len_q
 * (diagonal aligned bottom-right; len_q == len_k for self-attention).  Empty
 * segments are legal.  max_seqlen bounds every segment length (validated on
 * the device).  Writes out [T, hq, d] and lse [hq, T]. */
int bs_attn_varlen_fwd(const bs_dims* dims, const void* q, const void* k, const void* v,
                       const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                       int32_t num_seqs, int32_t max_seqlen, int causal, float scale,
                       void* out, float* lse, void* workspace, size_t workspace_bytes,
                       void* stream);

/* Bytes of the per-device scratch array behind bs_attn_varlen_fwd_noalloc(). */
#define BS_NOALLOC_SCRATCH_BYTES ((size_t)4 << 20)

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): bs_attn_varlen_fwd without the
 * workspace arguments.  Same computation, arguments, layouts and results as
 * bs_attn_varlen_fwd; the plan that the forward kernel walks goes into a file-scope
 * device array of BS_NOALLOC_SCRATCH_BYTES (4 MiB) that the library holds on every
 * device it runs on until the process ends.  No hipMalloc or hipFree, and no allocating
 * library routine, is called.
 *   - Limit: the plan takes 256 B + 4 (2 num_seqs + 3) B (each part rounded up to 256 B)
 *     + 48 B per work item, with ceil(total_q / 128) + num_seqs items (bf16) or
 *     ceil(total_q / 64) + num_seqs items (float32); sizes beyond the array return
 *     BS_ERR_WORKSPACE (for example about 11M bf16 query tokens in 20 segments) and
 *     enqueue nothing.
 *   - `stream` must belong to the current device (BS_ERR_INVALID_ARG otherwise); the
 *     first call on a device looks up the array's address there (hipGetSymbolAddress).
 *   - Every call on one device uses that device's one array: calls that can overlap on
 *     a device (different streams, or other host threads) race and must be ordered by
 *     the caller.  The array keeps the last call's plan; nothing in it needs clearing.
 *   - A cu_seqlens error found on the device is written into the array's status word,
 *     which no helper reads: out and lse are then left unwritten. */
int bs_attn_varlen_fwd_noalloc(const bs_dims* dims, const void* q, const void* k, const void* v,
                               const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                               int32_t num_seqs, int32_t max_seqlen, int causal, float scale,
                               void* out, float* lse, void* stream);

/* Varlen backward: given the forward's out and lse and the upstream gradient
 * dout, writes dq [T, hq, d], dk and dv [Tk, hkv, d] (overwritten, not added).
 * Every gradient is accumulated in float32 and rounded once. */
int bs_attn_varlen_bwd(const bs_dims* dims, const void* q, const void* k, const void* v,
                       const void* out, const float* lse, const void* dout,
                       const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                       int32_t num_seqs, int32_t max_seqlen, int causal, float scale,
                       void* dq, void* dk, void* dv, void* workspace, size_t workspace_bytes,
                       void* stream);

/* One context-parallel step (Sec. 2.4; Sec. 7, Dist-attn with packing): the Q
 * shard of total_q tokens whose first token sits at global position
 * q_pos_offset, against a KV shard of total_k tokens at k_pos_offset.  With
 * causal != 0 key j is visible to query i iff k_pos_offset + j <= q_pos_offset + i.
 * Writes this step's partial out [T, hq, d] and lse [hq, T]; rows that see no
 * key get out = 0, lse = -inf.  Combine the steps with bs_lse_merge(), or use
 * bs_attn_chunk_fwd_merge() to combine each step as it is computed. */
int bs_attn_chunk_fwd(const bs_dims* dims, const void* q, const void* k, const void* v,
                      int64_t q_pos_offset, int64_t k_pos_offset, int causal, float scale,
                      void* out, float* lse, void* workspace, size_t workspace_bytes,
                      void* stream);

/* One context-parallel step folded into a running result as it arrives (the ring
 * steps of Sec. 2.4 overlap the key exchange with compute, so each step's output
 * can be combined at once instead of stored and merged at the end).  The mask and
 * the positions are those of bs_attn_chunk_fwd; workspace as for BS_OP_CHUNK_FWD.
 * Running state, owned by the caller: o_run float32 [T, hq, d] and lse_run
 * float32 [hq, T] (natural log).  With accumulate == 0 the running state is
 * replaced by this step's result (rows that see no key: o 0, lse -inf); with
 * accumulate != 0 it is combined with it by the rule of bs_lse_merge(),
 *   LSE' = log(exp(LSE) + exp(LSE_step)),
 *   O'   = exp(LSE - LSE') O + exp(LSE_step - LSE') O_step,
 * computed in float32 without rounding O_step to dims->dtype; a row whose running
 * LSE is -inf ignores its o_run contents.  out: NULL, or [T, hq, d] of
 * dims->dtype, not overlapping o_run; when given, the combined O is written there
 * (rounded once) instead of into o_run, which this call then leaves as it was
 * (pass it on a ring's last step); lse_run is updated either way.  Every query
 * row is written on every call, including rows that see no key of this step. */
int bs_attn_chunk_fwd_merge(const bs_dims* dims, const void* q, const void* k, const void* v,
                            int64_t q_pos_offset, int64_t k_pos_offset, int causal, float scale,
                            float* o_run, float* lse_run, int accumulate, void* out,
                            void* workspace, size_t workspace_bytes, void* stream);

/* Backward of one context-parallel step.  out_merged / lse_merged are the
 * final (merged over all steps) forward results.  Adds this step's dQ
 * contribution into dq_accum (float32 [T, hq, d], caller-zeroed before the
 * first step).  This KV shard's dK, dV [Tk, hkv, d]: with kv_accumulate == 0,
 * dk and dv are outputs of dims->dtype, overwritten; with kv_accumulate != 0
 * they are float32 accumulators (caller-zeroed) to which this step's
 * contribution is added, for a KV shard that several Q shards attend to (the
 * symmetric 2N-way split of Sec. 7, Dist-attn with packing).  bs_dq_finalize()
 * rounds any such float32 accumulator into dims->dtype. */
int bs_attn_chunk_bwd(const bs_dims* dims, const void* q, const void* k, const void* v,
                      const void* out_merged, const float* lse_merged, const void* dout,
                      int64_t q_pos_offset, int64_t k_pos_offset, int causal, float scale,
                      float* dq_accum, void* dk, void* dv, int kv_accumulate, void* workspace,
                      size_t workspace_bytes, void* stream);

/* Packed context-parallel step (Sec. 7, Dist-attn with packing: every
 * subsequence of a packed micro-batch is split into 2N parts, device i holds
 * parts i and 2N-1-i of each, and the ring passes the KV parts around).  One call
 * covers the part pairs of many subsequences: segment b holds queries
 * cu_seqlens_q[b] .. cu_seqlens_q[b+1]-1 whose first token sits at global
 * position q_pos[b] of its subsequence, and keys cu_seqlens_k[b] ..
 * cu_seqlens_k[b+1]-1 whose first token sits at k_pos[b] (cu_seqlens: int32,
 * num_seqs+1 entries, validated as for the varlen ops; q_pos, k_pos: int64 device
 * arrays of num_seqs entries).  With causal != 0 key j of segment b is visible to
 * query i iff k_pos[b] + j <= q_pos[b] + i.  Empty segments, and segments whose
 * keys are all in the future, are legal.  Writes this step's partial out
 * [T, hq, d] and lse [hq, T] with the conventions of bs_attn_chunk_fwd (rows that
 * see no key: out = 0, lse = -inf); combine the partials with bs_lse_merge().
 * A zig-zag ring step is two calls: the "straight" pairs (query part i with key
 * part j, part 2N-1-i with part 2N-1-j) and the "crossed" ones (part i with part
 * 2N-1-j, part 2N-1-i with part j, the key buffer holding the parts in that
 * order). */
int bs_attn_packed_chunk_fwd(const bs_dims* dims, const void* q, const void* k, const void* v,
                             const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                             const int64_t* q_pos, const int64_t* k_pos, int32_t num_seqs,
                             int32_t max_seqlen, int causal, float scale, void* out, float* lse,
                             void* workspace, size_t workspace_bytes, void* stream);

/* Packed context-parallel step folded into a running result: the segments, mask
 * and positions of bs_attn_packed_chunk_fwd with the running state (o_run, lse_run,
 * accumulate, out) of bs_attn_chunk_fwd_merge; workspace as for
 * BS_OP_PACKED_CHUNK_FWD. */
int bs_attn_packed_chunk_fwd_merge(const bs_dims* dims, const void* q, const void* k,
                                   const void* v, const int32_t* cu_seqlens_q,
                                   const int32_t* cu_seqlens_k, const int64_t* q_pos,
                                   const int64_t* k_pos, int32_t num_seqs, int32_t max_seqlen,
                                   int causal, float scale, float* o_run, float* lse_run,
                                   int accumulate, void* out, void* workspace,
                                   size_t workspace_bytes, void* stream);

/* Backward of one packed context-parallel step, with the conventions of
 * bs_attn_chunk_bwd: out_merged / lse_merged are the final forward results of
 * these query rows, this step's dQ is added into dq_accum (float32 [T, hq, d]),
 * and dk, dv are overwritten (kv_accumulate == 0) or float32 accumulators
 * (kv_accumulate != 0).  Each key row belongs to one segment of the call. */
int bs_attn_packed_chunk_bwd(const bs_dims* dims, const void* q, const void* k, const void* v,
                             const void* out_merged, const float* lse_merged, const void* dout,
                             const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                             const int64_t* q_pos, const int64_t* k_pos, int32_t num_seqs,
                             int32_t max_seqlen, int causal, float scale, float* dq_accum,
                             void* dk, void* dv, int kv_accumulate, void* workspace,
                             size_t workspace_bytes, void* stream);

/* Rounds a float32 dQ accumulator [T, hq, d] into dq of dims->dtype (RNE). */
int bs_dq_finalize(const bs_dims* dims, const float* dq_accum, void* dq, void* stream);

/* Combines n partial results of the same queries over disjoint key sets (the
 * ring steps of Sec. 2.4):  LSE = log sum_c exp(LSE_c),
 * O = sum_c exp(LSE_c - LSE) O_c.  A partial with LSE_c = -inf has weight 0; a
 * row where every partial is -inf gets O = 0, LSE = -inf.  Sizes come from
 * dims->total_q, hq, head_dim, dtype (hkv and total_k are not used).
 * out_partials [n, T, hq, d], lse_partials float [n, hq, T]; writes out
 * [T, hq, d] and lse [hq, T].  n must be >= 1. */
int bs_lse_merge(const bs_dims* dims, const void* out_partials, const float* lse_partials,
                 int32_t n, void* out, float* lse, void* stream);

/* Device-to-device copy of `bytes` on `stream` by the GPU's DMA engines, leaving
 * the compute units to the attention kernels that it overlaps (the copies that
 * Sec. 5.2, Selective Offloading, overlaps with compute run on DMA engines rather
 * than on the streaming multiprocessors for the same reason).  It stands in for
 * the transfer of a KV shard or of its gradients between ring neighbours when
 * one GPU rehearses a device's ring (Sec. 2.4).  dst and src: device pointers of
 * at least `bytes` bytes, not overlapping (BS_ERR_INVALID_ARG); bytes == 0
 * enqueues nothing. */
int bs_copy_async(void* dst, const void* src, size_t bytes, void* stream);

/* Softmax cross-entropy of next-token prediction with its gradient fused in (Sec. 7,
 * Fused SoftmaxCrossEntropy: bf16 logits over a vocabulary of ~128K entries, the
 * arithmetic in fp32, no fp32 copy of the logits).  logits: [rows, vocab] of `dtype`
 * (BS_BF16 or BS_F32), row-major; labels: int64 [rows].  Per row i:
 *   lse_i  = log sum_j exp(z_ij)                      (float32, natural log)
 *   loss_i = lse_i - z_i,label_i                      (float32; 0 if label_i == ignore_index)
 *   dlogits_ij = grad_scale * (exp(z_ij - lse_i) - [j == label_i])   (in `dtype`, RNE)
 * grad_scale is the upstream gradient of every token's loss (1/N for the token-level loss of
 * Sec. 5.1, Loss and Model Update).  An ignored row's gradient is all zero; its lse is still
 * written.  A label outside [0, vocab) that is not ignore_index gives loss NaN and the row's
 * gradient without the one-hot term (nothing is read or written outside the row).  A row
 * whose logits are all -inf gives lse -inf and loss NaN.  lse may be NULL (not written);
 * dlogits may be NULL (loss only), may equal logits (gradient written in place), and must not
 * otherwise overlap it.  1 <= vocab < 2^31 and 0 <= rows < 2^30.  The result is bitwise
 * deterministic. */
int bs_softmax_xent(int64_t rows, int64_t vocab, int dtype, const void* logits,
                    const int64_t* labels, int64_t ignore_index, float grad_scale, float* loss,
                    float* lse, void* dlogits, void* stream);

/* TEST HELPER (synchronises `stream`): the device status word left in the
 * workspace by the last planning kernel; BS_OK, or BS_ERR_DEVICE_STATUS with
 * the BS_DEV_* code in bs_last_error(). */
int bs_read_device_status(const void* workspace, void* stream);

/* TEST HELPER (synchronises `stream`): runs the device planner of `op` on the
 * given segment description and copies the ordered work list back to
 * host_items, 12 int32 per item, up to `capacity` items; *count receives the
 * item count and tile_m / tile_n (may be NULL) the tile sizes it used.
 * Forward items: seg, qtile, q_start, q_rows, k_start, k_len, n_full, n_tiles,
 * diag, 0, 0, 0.  Backward items: seg, ktile, k_start, k_rows, q_start, q_len,
 * qt_first, n_masked, n_vis, diag, 0, 0.  For the single-chunk ops cu_seqlens
 * are ignored and q_pos_offset / k_pos_offset are used; the packed chunk ops use
 * cu_seqlens and the per-segment device arrays q_pos / k_pos (NULL otherwise). */
int bs_attn_plan_export(int op, const bs_dims* dims, const int32_t* cu_seqlens_q,
                        const int32_t* cu_seqlens_k, int32_t num_seqs, int32_t max_seqlen,
                        int64_t q_pos_offset, int64_t k_pos_offset, const int64_t* q_pos,
                        const int64_t* k_pos, int causal, void* workspace,
                        size_t workspace_bytes, int32_t* host_items, size_t capacity,
                        size_t* count, int32_t* tile_m, int32_t* tile_n, void* stream);

/* Kernel classes timed by the profiling hooks below. */
enum {
  BS_KERNEL_PLAN = 0,       /* the three planning kernels of a plan */
  BS_KERNEL_FWD = 1,        /* forward attention kernel */
  BS_KERNEL_PREPROCESS = 2, /* backward preprocess (D = rowsum(dO * O)) */
  BS_KERNEL_BWD_DQ = 3,     /* backward kernel producing dQ */
  BS_KERNEL_BWD_DKDV = 4,   /* backward kernel producing dK and dV */
  BS_KERNEL_FINALIZE = 5,   /* float32 dQ accumulator -> dq */
  BS_KERNEL_MERGE = 6,      /* LSE merge */
  BS_KERNEL_XENT = 7,       /* softmax cross-entropy */
  BS_KERNEL_COUNT = 8
};

/* Profiling (off by default, process-wide).  While enabled, every call
 * records a pair of HIP events on its stream immediately around each of its
 * kernels, so the durations measured are those of the kernels alone, on the
 * stream they ran on.  Enabling or disabling clears what was recorded. */
int bs_set_profiling(int enable);

/* Synchronises the recorded events and returns, for kernel class `kind`, the
 * summed duration in milliseconds and the number of launches timed since
 * profiling was enabled.  BS_ERR_INVALID_ARG for an unknown kind or NULL
 * outputs. */
int bs_profile_read(int kind, double* total_ms, int64_t* launches);

/* Thread-local message of the last failed call on this thread ("" if none). */
const char* bs_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* BS_ATTN_H */
