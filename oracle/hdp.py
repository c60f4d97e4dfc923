"""Hybrid Data Parallelism planners (Sec. 5 and Sec. 6): the oracle.

TEST INFRASTRUCTURE.  Only tests/, the smoke check and the benchmark's CPU-baseline leg may
import this module; the library never does.  Plain Python, the steps in the paper's order, no
code shared with the native planner.

Cost model (Sec. 4 profiles it; Eq. 3 states it), per transformer layer:
  T(s)   = alpha1 s^2 + beta1 s + gamma      seconds of forward + backward for s tokens
  Act(s) = alpha2 s + beta2                  bytes of activations for s tokens
with l layers per rank, rank capacity C tokens and host-link bandwidths B_d2h, B_h2d.

Work units.  A sequence of s <= C tokens fits one rank; short sequences are packed into
micro-batches of at most C tokens that one rank runs in sum_j T(s_j).  A longer sequence is a
context-parallel unit: D ranks hold it (Eq. 3) and each of them spends T(s) / D on it (the
zig-zag split of Sec. 7 gives every rank of the group the same share of the mask area); the D
ranks start it together, when the last of them is free.

Floating point: every quantity is an IEEE double computed by the expressions below in the order
written (left to right), so that another implementation doing the same operations in the same
order reproduces each decision bit for bit.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

ALG_NAIVE, ALG_DP_BALANCE, ALG_PP_BALANCE = 0, 1, 2


@dataclass(frozen=True)
class Cost:
    alpha1: float
    beta1: float
    gamma: float
    alpha2: float
    beta2: float
    layers: int
    bw_d2h: float
    bw_h2d: float

    def T(self, s) -> float:
        s = float(s)
        return self.alpha1 * s * s + self.beta1 * s + self.gamma

    def act(self, s) -> float:
        return self.alpha2 * float(s) + self.beta2


def offload_ratio(s: int, C: int, cost: Cost):
    """Eq. 3: the offload ratio r and rank count D(s) of a sequence of s tokens.

    D(r) = ceil((2 Act(s) + (1 - r)(l - 2) Act(s)) / (l Act(C))) falls as r grows, so the
    smallest D within the constraints is reached at the largest admissible r: the bandwidth
    constraint T(s) >= Act(s) r / min(B_d2h, B_h2d) caps r at T(s) min(B) / Act(s), and r <= 1.
    The lower bound r >= min(1, l Act(C) / ((l - 2) Act(s))) is the ratio below which offloading
    saves no rank at all; when the cap lies below it, the sequence is not offloaded (r = 0).
    A sequence that fits one rank (s <= C) has r = 0 and D = 1."""
    if s <= C:
        return 0.0, 1
    l = cost.layers
    a_s = cost.act(s)
    a_c = cost.act(C)
    r_lo = min(1.0, (l * a_c) / ((l - 2) * a_s))
    bw = min(cost.bw_d2h, cost.bw_h2d)
    r_hi = min(1.0, cost.T(s) * bw / a_s)
    r = r_hi if r_hi >= r_lo else 0.0
    D = math.ceil((2.0 * a_s + (1.0 - r) * (l - 2) * a_s) / (l * a_c))
    return r, int(D)


def best_fit_pack(seqs, lengths, C: int):
    """Alg. 1, the packing of the short sequences: best fit, largest first.  Sequences in order
    of decreasing length (ties: lower index first); each goes into the open micro-batch with the
    least room left that still holds it (ties: the earlier one), or opens a new one.  Returns
    the micro-batches as lists of sequence indices, in the order they were opened."""
    order = sorted(seqs, key=lambda i: (-lengths[i], i))
    bins, room = [], []
    for i in order:
        best = -1
        for b in range(len(bins)):
            if room[b] >= lengths[i] and (best < 0 or room[b] < room[best]):
                best = b
        if best < 0:
            bins.append([i])
            room.append(C - lengths[i])
        else:
            bins[best].append(i)
            room[best] -= lengths[i]
    return bins


def _place(exec_t, ranks, t):
    """The ranks start the unit together when the last of them is free; each spends t on it."""
    start = max(exec_t[g] for g in ranks)
    for g in ranks:
        exec_t[g] = start + t
    return start


def naive_hdp(lengths, C: int, d_hdp: int, cost: Cost):
    """Alg. 1.  Long sequences get (r, D) from Eq. 3; the short ones are packed by best fit; the
    units (the long sequences in batch order, then the packed micro-batches in the order they
    were opened) are dealt to ranks as data parallelism deals micro-batches, by count: a unit
    of D ranks goes to the D ranks that hold the fewest micro-batches so far (ties: lower rank).

    Returns (micro_batches, rank_time): micro_batches in assignment order as tuples
    (seqs, ranks, r, start, time), rank_time the modelled finish time of every rank."""
    n = len(lengths)
    pack_list, units = [], []
    for i in range(n):
        r, D = offload_ratio(lengths[i], C, cost)
        if lengths[i] <= C:
            pack_list.append(i)
        else:
            if D > d_hdp:
                raise ValueError(f"sequence {i} needs {D} ranks, more than d_hdp = {d_hdp}")
            units.append(([i], D, r, cost.T(lengths[i]) / D))
    for b in best_fit_pack(pack_list, lengths, C):
        t = 0.0
        for i in b:
            t += cost.T(lengths[i])
        units.append((b, 1, 0.0, t))
    count = [0] * d_hdp
    exec_t = [0.0] * d_hdp
    out = []
    for seqs, D, r, t in units:
        ranks = sorted(range(d_hdp), key=lambda g: (count[g], g))[:D]
        start = _place(exec_t, ranks, t)
        for g in ranks:
            count[g] += 1
        out.append((tuple(seqs), tuple(ranks), r, start, t))
    return out, exec_t


def _buckets(lengths, cost: Cost, n_buckets: int):
    """Alg. 2, step 1: the batch in order of decreasing length (ties: lower index first), cut
    into n_buckets runs of about equal total cost T(s): a sequence goes to the bucket in which
    the cost of everything before it falls.  Empty buckets are dropped."""
    order = sorted(range(len(lengths)), key=lambda i: (-lengths[i], i))
    costs = [cost.T(lengths[i]) for i in order]
    total = 0.0
    for c in costs:
        total += c
    buckets = [[] for _ in range(n_buckets)]
    cum = 0.0
    for i, c in zip(order, costs):
        b = min(n_buckets - 1, int(cum * n_buckets / total)) if total > 0.0 else 0
        buckets[b].append(i)
        cum += c
    return [b for b in buckets if b]


def _take(bucket, lengths, C: int):
    """One unit from the head of a bucket: a long sequence alone, or else the bucket's short
    sequences taken in order whenever they still fit in C tokens (first fit over the bucket)."""
    if lengths[bucket[0]] > C:
        return [bucket.pop(0)]
    room, picked, rest = C, [], []
    for i in bucket:
        if lengths[i] <= C and lengths[i] <= room:
            picked.append(i)
            room -= lengths[i]
        else:
            rest.append(i)
    bucket[:] = rest
    return picked


def balance(lengths, C: int, d_hdp: int, cost: Cost, delta: float, strategy: int,
            n_buckets: int):
    """Alg. 2 (balance strategy; it replaces the dealing step of Alg. 1).

    Rounds until every bucket is empty.  A round fixes max_time, the latest rank's finish time;
    while some rank finishes more than delta before it (the target ranks), the target that
    finishes first receives one unit and the targets are re-derived from the new finish times.
    A unit comes from the first bucket under DP-Balance (at any time all ranks run sequences of
    one length level, Sec. 6.3) and from bucket (rank mod #buckets) under PP-Balance (each
    pipeline keeps to one length level, Sec. 6.2).  A context-parallel unit of D ranks goes to
    the D ranks that finish first (the target among them) and starts when the last of them is
    free.  A round in which no rank lags (all within delta, as at the start) gives one unit to
    the rank that finishes first.  Ranks that finish early thus receive more micro-batches
    (Sec. 6.1).  Ties between ranks go to the lower rank.  Returns (micro_batches, rank_time)
    as naive_hdp does."""
    for i in range(len(lengths)):
        if lengths[i] > C and offload_ratio(lengths[i], C, cost)[1] > d_hdp:
            raise ValueError(f"sequence {i} needs more than d_hdp = {d_hdp} ranks")
    buckets = _buckets(lengths, cost, n_buckets)
    exec_t = [0.0] * d_hdp
    out = []

    def by_finish():
        return sorted(range(d_hdp), key=lambda g: (exec_t[g], g))

    def give(g):
        bi = 0 if strategy == ALG_DP_BALANCE else g % len(buckets)
        seqs = _take(buckets[bi], lengths, C)
        if not buckets[bi]:
            del buckets[bi]
        if len(seqs) == 1 and lengths[seqs[0]] > C:
            s = lengths[seqs[0]]
            r, D = offload_ratio(s, C, cost)
            ranks = by_finish()[:D]
            t = cost.T(s) / D
        else:
            r, ranks = 0.0, [g]
            t = 0.0
            for i in seqs:
                t += cost.T(lengths[i])
        start = _place(exec_t, ranks, t)
        out.append((tuple(seqs), tuple(ranks), r, start, t))

    while buckets:
        max_t = max(exec_t)
        targets = [g for g in by_finish() if max_t - exec_t[g] > delta]
        if not targets:
            give(by_finish()[0])
            continue
        while targets and buckets:
            give(targets[0])
            targets = [g for g in by_finish() if max_t - exec_t[g] > delta]
    return out, exec_t


def plan(algorithm: int, lengths, C: int, d_hdp: int, cost: Cost, delta: float = 0.0,
         n_buckets: int = 4):
    if algorithm == ALG_NAIVE:
        return naive_hdp(lengths, C, d_hdp, cost)
    return balance(lengths, C, d_hdp, cost, delta, algorithm, n_buckets)
