"""Pins of the reference tile planner: the corner rule equals an enumeration of every
(query, key) pair of a tile, and the work lists cover exactly the visible pairs."""
import numpy as np
import pytest

from oracle import attention as A
from oracle import plan as P


def test_corner_rule_matches_pair_enumeration():
    rng = np.random.default_rng(0)
    cases = 0
    for _ in range(300):
        lq, lk = int(rng.integers(0, 40)), int(rng.integers(0, 40))
        diag = int(rng.integers(-45, 45))
        BM, BN = int(rng.choice([1, 3, 4, 8])), int(rng.choice([1, 2, 5, 8]))
        causal = bool(rng.integers(0, 4))
        for qt in range((lq + BM - 1) // BM):
            for kt in range((lk + BN - 1) // BN):
                a = P.tile_class(lq, lk, diag, causal, BM, BN, qt, kt)
                b = P.tile_class_bruteforce(lq, lk, diag, causal, BM, BN, qt, kt)
                assert a == b, (lq, lk, diag, causal, BM, BN, qt, kt)
                cases += 1
    assert cases > 1000


@pytest.mark.parametrize("kind", ["fwd", "bwd"])
def test_work_list_covers_exactly_the_visible_pairs(kind):
    """Summing, over the listed tile pairs, the visible pairs inside each gives A; the pairs in
    SKIP tiles are none."""
    rng = np.random.default_rng(1)
    for _ in range(40):
        lens = [int(x) for x in rng.integers(0, 50, size=int(rng.integers(1, 6)))]
        cu = np.concatenate([[0], np.cumsum(lens)])
        BM, BN = int(rng.choice([4, 8, 16])), int(rng.choice([4, 8, 16]))
        items = P.varlen_plan(cu, cu, True, BM, BN, kind)
        covered = 0
        for it in items:
            if kind == "fwd":
                b, qt, q0, qr, k0, lk, nf, nt, diag = it
                pairs = [(qt, kt) for kt in range(nt)]
            else:
                b, kt, k0, kr, q0, lq, first, nm, nv, diag = it
                pairs = [(qt, kt) for qt in range(first, first + nv)]
            L = lens[b]
            m = A.visible_mask(L, L, 0, True)
            for qt, kt in pairs:
                covered += int(m[qt * BM:(qt + 1) * BM, kt * BN:(kt + 1) * BN].sum())
        assert covered == sum(l * (l + 1) // 2 for l in lens)


@pytest.mark.parametrize("kind", ["fwd", "bwd"])
@pytest.mark.parametrize("causal", [True, False])
def test_order_groups_segments_largest_first_with_cost_descending_inside(kind, causal):
    # segments of equal size (64, 64) keep index order; every segment's tiles are
    # contiguous; inside a segment the tile order is the closed form (forward
    # descending, backward ascending index) and must be non-increasing cost
    lens = [300, 5, 64, 64, 1000, 0, 129]
    cu = np.concatenate([[0], np.cumsum(lens)])
    BM, BN = (64, 32) if kind == "fwd" else (32, 64)
    items = P.varlen_plan(cu, cu, causal, BM, BN, kind)
    segs = [it[0] for it in items]
    runs = [s for i, s in enumerate(segs) if i == 0 or segs[i - 1] != s]
    assert len(runs) == len(set(runs)), "a segment's tiles are not contiguous"
    assert runs == sorted(runs, key=lambda b: (-2 * lens[b], b))
    cost = 7 if kind == "fwd" else 8
    for b in runs:
        mine = [it for it in items if it[0] == b]
        tiles = [it[1] for it in mine]
        assert tiles == (sorted(tiles, reverse=True) if kind == "fwd" else sorted(tiles))
        costs = [it[cost] for it in mine]
        assert costs == sorted(costs, reverse=True)
    tile = BM if kind == "fwd" else BN  # query tiles (forward) or key tiles (backward)
    assert len(items) == sum((l + tile - 1) // tile for l in lens)


def test_chunk_plan_past_diagonal_and_future():
    c = 256
    past = P.chunk_plan(c, c, 10 * c, 3 * c, True, 64, 32, "fwd")
    assert all(it[6] == it[7] == c // 32 for it in past)          # every tile FULL
    fut = P.chunk_plan(c, c, 0, c, True, 64, 32, "fwd")
    assert all(it[7] == 0 for it in fut)                          # nothing visible
    diag = P.chunk_plan(c, c, 5 * c, 5 * c, True, 64, 32, "fwd")
    full, masked = P.tile_counts(diag, "fwd")
    # BM = 2 BN: each 64-row tile has its 64x64 diagonal block split into 2 masked
    # 64x32 tiles, everything left of it full
    assert masked == 2 * (c // 64)
    assert full == sum(2 * qt for qt in range(c // 64))
