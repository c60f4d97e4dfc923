"""Pins of the HDP planner oracle (Sec. 5, Sec. 6) against what the paper and the mathematics fix:
the rank counts the paper works out, closed forms of Eq. 3 at r = 0, r = 1 and an exact
intermediate ratio, a brute-force argmin of Eq. 3, a hand-worked best-fit packing, the any-fit
property and brute-force optimal bin counts, Alg. 2 traced by hand (the equal-FLOPs bucket cut,
DP-Balance and PP-Balance plans unit by unit, a context-parallel unit), Insight 1's one length
level per pipeline, and the invariants of every assignment."""
import itertools
import math

import numpy as np
import pytest

from oracle import hdp as H

K = 1024


def cost(alpha1=1e-12, beta1=1e-7, gamma=1e-5, alpha2=1.0e5, beta2=0.0, layers=32,
         bw=0.0):
    return H.Cost(alpha1, beta1, gamma, alpha2, beta2, layers, bw, bw)


def test_paper_rank_counts_without_offloading():
    """Sec. 5.2: 1M tokens need 128 ranks of 8K; Sec. 5.1: 512K use 64 of them and 768K need 96.
    With no host bandwidth nothing can be offloaded (r = 0) and D = ceil(Act(s) / Act(C))."""
    c = cost(bw=0.0)
    for s, want in ((1024 * K, 128), (512 * K, 64), (768 * K, 96)):
        r, D = H.offload_ratio(s, 8 * K, c)
        assert r == 0.0 and D == want, (s, r, D)
    assert H.offload_ratio(8 * K, 8 * K, c) == (0.0, 1)  # fits one rank
    assert H.offload_ratio(8 * K + 1, 8 * K, c)[1] == 2


def test_full_offload_and_an_exact_intermediate_ratio():
    # unlimited bandwidth: r = 1 and D = ceil(2 Act(s) / (l Act(C))) = ceil(2 * 128 / 32) = 8
    r, D = H.offload_ratio(1024 * K, 8 * K, cost(bw=1e30))
    assert r == 1.0 and D == 8
    # bandwidth chosen so that T(s) min(B) / Act(s) = 1/2 exactly: alpha1 = 0 and beta1 = gamma = 0
    # give T(s) = 0 ... instead T(s) = beta1 s, Act(s) = alpha2 s: ratio = beta1 B / alpha2
    c = cost(alpha1=0.0, beta1=2.0 ** -20, gamma=0.0, alpha2=2.0 ** 10, bw=2.0 ** 29)
    r, D = H.offload_ratio(1024 * K, 8 * K, c)
    assert r == 0.5
    assert D == math.ceil((2 + 0.5 * 30) * 128 / 32) == 68


def test_no_offload_when_the_cap_cannot_save_a_rank():
    """The lower bound of r is the ratio that saves one rank: l Act(C) / ((l - 2) Act(s)).  A cap
    just below it gives r = 0 and D = ceil(s / C); just above it, D = ceil(s / C) - 1."""
    l, C, s = 32, 8 * K, 64 * K  # s / C = 8
    r_lo = (l * C) / ((l - 2) * s)
    below = cost(alpha1=0.0, beta1=(r_lo * 0.999) / 1.0, gamma=0.0, alpha2=1.0, bw=1.0)
    above = cost(alpha1=0.0, beta1=(r_lo * 1.001) / 1.0, gamma=0.0, alpha2=1.0, bw=1.0)
    assert H.offload_ratio(s, C, below) == (0.0, 8)
    r, D = H.offload_ratio(s, C, above)
    assert r > r_lo and D == 7


def test_eq3_matches_brute_force_argmin():
    """Over a fine grid of the admissible r (r = 0, or r between the bounds), the smallest D is
    the one the oracle returns, and the oracle's r is admissible."""
    rng = np.random.default_rng(4)
    for _ in range(200):
        l = int(rng.integers(3, 96))
        C = int(rng.integers(1, 64)) * K
        s = C + int(rng.integers(1, 200 * C))
        c = H.Cost(float(rng.uniform(0, 2e-11)), float(rng.uniform(0, 1e-6)), float(rng.uniform(0, 1e-4)),
                   float(rng.uniform(1e4, 1e6)), float(rng.uniform(0, 1e7)), l,
                   float(rng.uniform(0, 1e11)), float(rng.uniform(0, 1e11)))
        r, D = H.offload_ratio(s, C, c)
        a_s, a_c = c.act(s), c.act(C)
        bw = min(c.bw_d2h, c.bw_h2d)
        lo = min(1.0, l * a_c / ((l - 2) * a_s))
        hi = min(1.0, c.T(s) * bw / a_s)
        grid = [0.0] + ([lo + (hi - lo) * k / 400 for k in range(401)] if hi >= lo else [])
        best = min(math.ceil((2 * a_s + (1 - x) * (l - 2) * a_s) / (l * a_c)) for x in grid)
        assert D == best, (l, C, s, r, D, best)
        assert r == 0.0 or (lo <= r <= hi + 1e-15)
        assert c.T(s) + 1e-12 >= a_s * r / bw if r > 0 else True


def test_best_fit_hand_example_and_any_fit_property():
    """C = 10, lengths 7 5 4 3 2 2 1 (indices 0..6).  By hand: 7 opens A (room 3); 5 opens B (5);
    4 -> B (1); 3 -> A (0); 2 fits nowhere -> C (8); 2 -> C (6); 1 -> B, the fullest that holds it."""
    lengths = [7, 5, 4, 3, 2, 2, 1]
    assert H.best_fit_pack(range(7), lengths, 10) == [[0, 3], [1, 2, 6], [4, 5]]
    rng = np.random.default_rng(8)
    for _ in range(50):
        n = int(rng.integers(1, 60))
        L = [int(x) for x in rng.integers(1, 101, n)]
        bins = H.best_fit_pack(range(n), L, 100)
        assert sorted(i for b in bins for i in b) == list(range(n))
        loads = [sum(L[i] for i in b) for b in bins]
        assert max(loads) <= 100
        assert sum(1 for x in loads if x <= 50) <= 1  # any fit: at most one bin half full or less


def optimal_bins(L, C):
    """Fewest bins of capacity C holding items L (brute force over assignments, tiny inputs)."""
    n = len(L)
    for k in range(1, n + 1):
        for assign in itertools.product(range(k), repeat=n):
            loads = [0] * k
            for i, b in enumerate(assign):
                loads[b] += L[i]
            if max(loads) <= C:
                return k
    return n


def test_best_fit_against_optimal_packing():
    """Best fit decreasing never beats the optimum and stays within 11/9 OPT + 6/9 of it."""
    rng = np.random.default_rng(12)
    for _ in range(40):
        n = int(rng.integers(1, 8))
        L = [int(x) for x in rng.integers(1, 21, n)]
        got = len(H.best_fit_pack(range(n), L, 20))
        opt = optimal_bins(L, 20)
        assert opt <= got <= 11 * opt / 9 + 6 / 9


def plan_invariants(out, rank_time, lengths, C, d, c):
    """Every sequence once; packed micro-batches within C on one rank; a long sequence alone on
    D(s) distinct ranks at T(s) / D; every rank's time is the end of its last unit, and a unit
    starts when the last of its ranks is free (replayed in assignment order)."""
    seen = sorted(i for seqs, _, _, _, _ in out for i in seqs)
    assert seen == list(range(len(lengths)))
    replay = [0.0] * d
    for seqs, ranks, r, start, t in out:
        assert len(set(ranks)) == len(ranks) and all(0 <= g < d for g in ranks)
        if len(seqs) == 1 and lengths[seqs[0]] > C:
            rr, D = H.offload_ratio(lengths[seqs[0]], C, c)
            assert len(ranks) == D and r == rr and t == c.T(lengths[seqs[0]]) / D
        else:
            assert len(ranks) == 1 and r == 0.0 and sum(lengths[i] for i in seqs) <= C
        assert start == max(replay[g] for g in ranks)
        for g in ranks:
            replay[g] = start + t
    assert replay == list(rank_time)


def lognormal_batch(seed, n, C):
    rng = np.random.default_rng(seed)
    return [int(min(16 * C, max(64, x))) for x in rng.lognormal(math.log(2048), 1.6, n)]


@pytest.mark.parametrize("alg", [H.ALG_NAIVE, H.ALG_DP_BALANCE, H.ALG_PP_BALANCE])
def test_plans_keep_their_invariants(alg):
    c = cost(alpha1=2e-11, beta1=5e-8, gamma=1e-5, alpha2=4e5, layers=32, bw=5e10)
    for seed in range(6):
        C = 32 * K
        lengths = lognormal_batch(seed, 300, C)
        out, rt = H.plan(alg, lengths, C, 16, c, delta=1e-4, n_buckets=4)
        plan_invariants(out, rt, lengths, C, 16, c)


def test_naive_deals_by_count_and_balance_evens_equal_work():
    c = cost(alpha1=0.0, beta1=1.0, gamma=0.0)
    # 16 sequences of C/4: best fit makes 4 micro-batches of 4; dealt one per rank
    out, rt = H.naive_hdp([256] * 16, 1024, 4, c)
    assert [len(s) for s, *_ in out] == [4] * 4 and sorted(g for _, (g,), *_ in out) == [0, 1, 2, 3]
    assert rt == [1024.0] * 4
    # DP-Balance on the same batch: the same four equal micro-batches, one per rank
    out, rt = H.balance([256] * 16, 1024, 4, c, 0.0, H.ALG_DP_BALANCE, 4)
    assert rt == [1024.0] * 4
    # a context-parallel unit starts when the last of its ranks is free
    out, rt = H.naive_hdp([512, 4096], 1024, 4, cost(alpha1=0.0, beta1=1.0, gamma=0.0, bw=0.0))
    seqs, ranks, r, start, t = out[0]
    assert seqs == (1,) and len(ranks) == 4 and start == 0.0 and t == 1024.0


def test_balance_shrinks_the_bubble_on_long_tailed_batches():
    """On these seeded long-tailed batches (log-normal lengths, a few context-parallel
    sequences) DP-Balance finishes no later than the naive dealing and idles the ranks less."""
    c = cost(alpha1=2e-11, beta1=5e-8, gamma=1e-5, alpha2=4e5, layers=32, bw=5e10)
    C = 32 * K
    for seed in range(5):
        lengths = lognormal_batch(100 + seed, 400, C)
        _, rt_n = H.naive_hdp(lengths, C, 16, c)
        _, rt_b = H.balance(lengths, C, 16, c, 1e-4, H.ALG_DP_BALANCE, 4)
        bubble = lambda rt: 1 - sum(rt) / (len(rt) * max(rt))
        assert max(rt_b) <= max(rt_n) and bubble(rt_b) < bubble(rt_n), seed


def test_rejects_a_sequence_wider_than_the_ranks():
    with pytest.raises(ValueError):
        H.naive_hdp([10 * 1024], 1024, 4, cost(bw=0.0))
    with pytest.raises(ValueError):
        H.balance([10 * 1024], 1024, 4, cost(bw=0.0), 0.0, H.ALG_DP_BALANCE, 2)


# ---------------------------------------------------------------------------------------------
# Alg. 2 (Sec. 6.4) traced by hand.  T(s) = s (alpha1 = 0, beta1 = 1, gamma = 0) keeps every
# finish time an integer; with no host bandwidth a long sequence of s tokens takes
# D = ceil(s / C) ranks (Eq. 3 at r = 0) and T(s) / D on each.

def linear_cost():
    return cost(alpha1=0.0, beta1=1.0, gamma=0.0, alpha2=1.0, beta2=0.0, bw=0.0)


def test_buckets_cut_by_equal_cost_not_by_count():
    """Step 1 of Alg. 2: the length-sorted batch is cut into runs of about equal total FLOPs, so a
    bucket of longer sequences holds fewer of them.  Lengths (by index) 1 8 2 1 4 1 1, sorted
    8 4 2 1 1 1 1 (indices 1 4 2 0 3 5 6), total cost 18, 2 buckets: the cost before each sequence
    is 0 8 12 14 15 16 17 and a sequence falls into bucket floor(2 * before / 18), which gives
    {8, 4} (cost 12) and {2, 1, 1, 1, 1} (cost 6).  A cut into equal counts would give {8, 4, 2, 1}
    and {1, 1, 1}, whose longer bucket holds more sequences.  With T(s) = s^2 the costs are
    64 16 4 1 1 1 1 (total 88; before: 0 64 80 84 85 86 87) and the first bucket is {8} alone."""
    lengths = [1, 8, 2, 1, 4, 1, 1]
    assert H._buckets(lengths, linear_cost(), 2) == [[1, 4], [2, 0, 3, 5, 6]]
    quad = cost(alpha1=1.0, beta1=0.0, gamma=0.0, alpha2=1.0, bw=0.0)
    assert H._buckets(lengths, quad, 2) == [[1], [4, 2, 0, 3, 5, 6]]
    # three buckets, T(s) = s: floor(3 * before / 18) = floor(before / 6) -> 0 1 2 2 2 2 2
    assert H._buckets(lengths, linear_cost(), 3) == [[1], [4], [2, 0, 3, 5, 6]]


def test_buckets_are_equal_cost_runs_on_random_batches():
    """On seeded random batches: the buckets are consecutive runs of the length-sorted batch; a
    bucket's cost differs from total / n_b by less than the largest single cost; and the bucket
    of the longest sequences holds fewer of them than the bucket of the shortest."""
    rng = np.random.default_rng(21)
    for _ in range(60):
        n = int(rng.integers(8, 120))
        L = [int(x) for x in rng.integers(1, 5000, n)]
        c = cost(alpha1=float(rng.uniform(0, 1e-9)), beta1=float(rng.uniform(1e-8, 1e-6)),
                 gamma=float(rng.uniform(0, 1e-6)), bw=0.0)
        nb = int(rng.integers(2, 6))
        B = H._buckets(L, c, nb)
        flat = [i for b in B for i in b]
        assert flat == sorted(range(n), key=lambda i: (-L[i], i))
        costs = [sum(c.T(L[i]) for i in b) for b in B]
        tot, top = sum(c.T(x) for x in L), max(c.T(x) for x in L)
        for cb in costs:
            assert abs(cb - tot / nb) < top + 1e-12 * tot
        assert len(B[0]) < len(B[-1]), [len(x) for x in B]


def test_dp_balance_traced_by_hand():
    """Lengths 6 5 4 3 3 2 2 1 1 1, C = 6, three ranks, delta = 1.5, two buckets (cost before each
    sequence 0 6 11 15 18 21 23 25 26 27 of 28: B0 = {0, 1, 2}, B1 = {3 .. 9}).  DP-Balance takes
    every unit from the first bucket:
      round 1  nobody lags (all at 0): rank 0 (first to finish) gets {0}            -> 6 0 0
      round 2  max 6, lagging 1, 2:   rank 1 gets {1}                             -> 6 5 0
               lagging 2:             rank 2 gets {2}, B0 empties                 -> 6 5 4
               lagging 2 (6-4 > 1.5): rank 2 gets {3, 4} (first fit in C = 6)     -> 6 5 10
      round 3  max 10, lagging 1, 0:  rank 1 gets {5, 6, 7, 8}                    -> 6 11 10
               lagging 0:             rank 0 gets {9}, B1 empties                 -> 7 11 10"""
    lengths = [6, 5, 4, 3, 3, 2, 2, 1, 1, 1]
    out, rt = H.balance(lengths, 6, 3, linear_cost(), 1.5, H.ALG_DP_BALANCE, 2)
    assert [(s, g, st, t) for s, g, _, st, t in out] == [
        ((0,), (0,), 0.0, 6.0), ((1,), (1,), 0.0, 5.0), ((2,), (2,), 0.0, 4.0),
        ((3, 4), (2,), 4.0, 6.0), ((5, 6, 7, 8), (1,), 5.0, 6.0), ((9,), (0,), 6.0, 1.0)]
    assert rt == [7.0, 11.0, 10.0]


def test_pp_balance_draws_rank_g_from_bucket_g_mod_nb():
    """The same batch under PP-Balance: rank g takes its unit from bucket g mod #buckets, so each
    pipeline stays on one length level while every bucket lasts (Sec. 6.2, Insight 1); once B0
    empties, every rank draws from the one bucket left:
      round 1  nobody lags: rank 0 <- B0: {0}                                    -> 6 0 0
      round 2  lagging 1, 2: rank 1 <- B1: {3, 4}                               -> 6 6 0
               lagging 2:    rank 2 <- B0 (2 mod 2): {1}                         -> 6 6 5
      round 3  max 6, nobody lags by more than 1.5: rank 2 <- B0: {2}, B0 empties -> 6 6 9
      round 4  max 9, lagging 0, 1: rank 0 <- B1 (0 mod 1): {5, 6, 7, 8}         -> 12 6 9
               lagging 1:    rank 1 <- B1: {9}                                   -> 12 7 9"""
    lengths = [6, 5, 4, 3, 3, 2, 2, 1, 1, 1]
    out, rt = H.balance(lengths, 6, 3, linear_cost(), 1.5, H.ALG_PP_BALANCE, 2)
    assert [(s, g, st, t) for s, g, _, st, t in out] == [
        ((0,), (0,), 0.0, 6.0), ((3, 4), (1,), 0.0, 6.0), ((1,), (2,), 0.0, 5.0),
        ((2,), (2,), 5.0, 4.0), ((5, 6, 7, 8), (0,), 6.0, 6.0), ((9,), (1,), 6.0, 1.0)]
    assert rt == [12.0, 7.0, 9.0]


def test_balance_places_a_context_parallel_unit_on_the_first_free_ranks():
    """Lengths 9 3 2 2 1, C = 4, three ranks, delta = 1.5, two buckets (before: 0 9 12 14 16 of 17:
    B0 = {0}, B1 = {1 .. 4}).  Sequence 0 needs ceil(9 / 4) = 3 ranks at T / 3 = 3 each:
      round 1  nobody lags: rank 0 draws {0}, a CP unit on ranks 0 1 2 from 0     -> 3 3 3
      round 2  nobody lags: rank 0 <- {1, 4} (3 + 1 fill C = 4)                   -> 7 3 3
      round 3  max 7, lagging 1, 2: rank 1 <- {2, 3}, the last bucket empties     -> 7 7 3"""
    out, rt = H.balance([9, 3, 2, 2, 1], 4, 3, linear_cost(), 1.5, H.ALG_DP_BALANCE, 2)
    assert [(s, g, st, t) for s, g, _, st, t in out] == [
        ((0,), (0, 1, 2), 0.0, 3.0), ((1, 4), (0,), 3.0, 4.0), ((2, 3), (1,), 3.0, 4.0)]
    assert rt == [7.0, 7.0, 3.0]


def test_pp_balance_keeps_each_pipeline_on_one_length_level():
    """Insight 1 (Sec. 6.2) on seeded batches of short sequences with as many ranks as buckets:
    until the first bucket runs out, every unit rank g receives comes from bucket g, the g-th
    length level, so the units of different ranks never mix levels."""
    c = cost(alpha1=2e-11, beta1=5e-8, gamma=1e-5, alpha2=4e5, layers=32, bw=5e10)
    C, nb = 32 * K, 4
    for seed in range(4):
        lengths = [min(x, C) for x in lognormal_batch(200 + seed, 400, C)]
        B = H._buckets(lengths, c, nb)
        level = {i: b for b, bucket in enumerate(B) for i in bucket}
        out, _ = H.balance(lengths, C, nb, c, 1e-4, H.ALG_PP_BALANCE, nb)
        sizes = [len(b) for b in B]
        taken = [0] * len(B)
        for seqs, (g,), *_ in out:
            if any(taken[b] == sizes[b] for b in range(len(B))):
                break  # a bucket ran out: the rank -> bucket map shifts from here on
            assert {level[i] for i in seqs} == {g}, (seed, seqs, g)
            taken[g] += len(seqs)
