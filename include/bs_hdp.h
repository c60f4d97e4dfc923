/*
 * bs_hdp.h -- C ABI of libbs_hdp.so, the host-side planners of ByteScale's Hybrid Data
 * Parallelism (HDP), arXiv 2502.21231: the data-aware selective offloading rule (Sec. 5.2,
 * Eq. 3), the naive HDP solution (Alg. 1) and the balance strategy (Sec. 6, Alg. 2).  They turn
 * one global batch of sequence lengths into micro-batches for d_hdp ranks; the per-rank
 * attention those micro-batches need is what libbs_attn.so computes.
 *
 * Cost model, per transformer layer (Sec. 4 profiles it; Eq. 3 states it):
 *   T(s)   = alpha1 s^2 + beta1 s + gamma   seconds of forward + backward for s tokens
 *   Act(s) = alpha2 s + beta2               bytes of activations for s tokens
 * A sequence of s <= capacity tokens fits one rank: such sequences are packed into
 * micro-batches of at most `capacity` tokens, which one rank runs in sum T(s_j).  A longer
 * sequence is a context-parallel unit on D(s) ranks (Eq. 3), each of which spends T(s) / D on it;
 * the D ranks start it together, when the last of them is free.
 *
 * Conventions: host pointers, owned by the caller; no call keeps a pointer after it returns.
 * Every call is synchronous and thread-safe (no shared state besides the thread-local error
 * message).  A status other than BS_HDP_OK writes nothing to the outputs and sets a message
 * readable with bs_hdp_last_error().  Results are deterministic: the same inputs give the same
 * plan bit for bit (IEEE double arithmetic in a fixed order).
 */
#ifndef BS_HDP_H
#define BS_HDP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BS_HDP_OK = 0,
  BS_HDP_ERR_INVALID_ARG = 1, /* null pointer, non-positive size, non-finite or negative cost */
  BS_HDP_ERR_INFEASIBLE = 2,  /* a sequence needs more ranks than d_hdp */
  BS_HDP_ERR_CAPACITY = 3     /* an output array is smaller than the plan */
} bs_hdp_status;

typedef enum { BS_HDP_NAIVE = 0, BS_HDP_DP_BALANCE = 1, BS_HDP_PP_BALANCE = 2 } bs_hdp_algorithm;

typedef struct {
  double alpha1, beta1, gamma; /* T(s), seconds per layer; all >= 0 */
  double alpha2, beta2;        /* Act(s), bytes per layer; Act(s) > 0 for s >= 1 */
  int32_t layers;              /* l, transformer layers per rank; >= 3 */
  double bw_d2h, bw_h2d;       /* host-link bandwidths, bytes per second; >= 0 */
} bs_hdp_cost;

typedef struct {
  int32_t seq_offset, n_seqs;   /* its sequences: seqs[seq_offset .. seq_offset + n_seqs) */
  int32_t rank_offset, n_ranks; /* the ranks that run it: ranks[rank_offset .. + n_ranks) */
  double offload_ratio;         /* r of Eq. 3 (0 for a packed micro-batch) */
  double start, time;           /* modelled start, and duration on each of its ranks */
} bs_hdp_microbatch;

/* Eq. 3 for one sequence of s tokens: the offload ratio r and the rank count D(s) =
 * ceil((2 Act(s) + (1 - r)(l - 2) Act(s)) / (l Act(C))).  D falls as r grows, so r is the
 * largest admissible ratio: min(1, T(s) min(B_d2h, B_h2d) / Act(s)) (the offload must hide
 * under the compute), unless that is below min(1, l Act(C) / ((l - 2) Act(s))), the ratio
 * below which offloading saves no rank, in which case r = 0.  s <= capacity gives r = 0,
 * D = 1.  s >= 1, capacity >= 1. */
int bs_hdp_offload_ratio(const bs_hdp_cost* cost, int64_t s, int64_t capacity, double* ratio,
                         int32_t* ranks);

/* Plans one global batch of n sequences (lengths[i] >= 1 tokens) on d_hdp ranks of `capacity`
 * tokens (delta >= 0 seconds, 1 <= n_buckets <= 2^20 for the balance strategies).
 *   BS_HDP_NAIVE (Alg. 1): the short sequences are packed by best fit, largest first (each
 *     into the open micro-batch with the least room that holds it, ties to the earlier one);
 *     the units (long sequences in batch order, then the packed micro-batches in the order
 *     they were opened) are dealt as data parallelism deals micro-batches: each to the
 *     ranks holding the fewest micro-batches (ties to the lower rank).  delta and n_buckets
 *     are not used.
 *   BS_HDP_DP_BALANCE / BS_HDP_PP_BALANCE (Alg. 2): the batch in order of decreasing length
 *     (ties: lower index first) is cut into n_buckets runs of about equal total T(s) (a
 *     sequence goes to bucket floor(cost before it * n_buckets / total cost)).  Rounds until
 *     every bucket is empty: max_time = the latest finish time; while a rank finishes more
 *     than delta before it, the earliest-finishing such rank receives one unit and the
 *     lagging set is re-derived; a round with no lagging rank gives one unit to the
 *     earliest-finishing rank.  A unit is the head of the bucket when that is a long
 *     sequence (on the D earliest-finishing ranks), else the bucket's short sequences that
 *     still fit, taken in order.  DP-Balance takes every unit from the first bucket (all ranks
 *     work on one length level at a time); PP-Balance takes rank g's from bucket
 *     (g mod #buckets) (each pipeline keeps to one length level).
 * Outputs: mbs[0 .. *n_mbs) in assignment order (max_mbs >= n always suffices); seqs, n
 * entries, each sequence exactly once, grouped by micro-batch; ranks[0 .. max_ranks), the
 * ranks of each micro-batch in the order chosen; rank_time[d_hdp], every rank's modelled
 * finish time.  BS_HDP_ERR_CAPACITY if max_mbs or max_ranks is too small. */
int bs_hdp_plan(int algorithm, const bs_hdp_cost* cost, const int64_t* lengths, int32_t n,
                int64_t capacity, int32_t d_hdp, double delta, int32_t n_buckets,
                bs_hdp_microbatch* mbs, int32_t max_mbs, int32_t* seqs, int32_t* ranks,
                int64_t max_ranks, int32_t* n_mbs, double* rank_time);

/* Thread-local message of the last failed call on this thread ("" if none). */
const char* bs_hdp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* BS_HDP_H */
