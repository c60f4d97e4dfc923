"""Reference tile planner (test infrastructure only; the product path never imports it).

The paper notes that the work of a packed micro-batch is proportional to the
area of its attention mask (Sec. 3.3, Imbalanced FLOPs; Sec. 7, Dist-attn with
packing).  The HIP library turns that into a work list: every segment (or
context-parallel chunk) is cut into query tiles of BM rows and key tiles of BN
keys, and each (query tile, key tile) pair is classed

  SKIP    no existing query row of the tile sees any key of the tile,
  FULL    every existing query row sees all BN key slots (so the tile is full
          width inside the segment and needs no score mask),
  MASKED  anything else (the causal diagonal, or a ragged key tail).

Visibility is "key j visible to query i iff j - i <= diag" (diag = len_k -
len_q for a varlen segment, q_off - k_off for a chunk; always visible when not
causal).  Because visibility only gets harder as j grows and easier as i grows,
the corners decide the class:
  SKIP  iff  kt*BN - q_last > diag,
  FULL  iff  (kt+1)*BN - 1 - q_first <= diag  and  (kt+1)*BN <= len_k.
The tests pin this corner rule against an enumeration of every (i, j) pair.

Forward items are query tiles: (seg, qtile, q_start, q_rows, k_start, k_len,
n_full, n_tiles, diag), the visible key tiles being 0..n_tiles-1 of which the
first n_full are FULL.

Backward items are key tiles: (seg, ktile, k_start, k_rows, q_start, q_len,
qt_first, n_masked, n_vis, diag), the visible query tiles being qt_first ..
qt_first+n_vis-1 of which the first n_masked are MASKED.

Order of the list (largest work first, the tiles of one segment side by side):
segments by len_q + len_k descending, ties by segment index; inside a segment,
forward query tiles by descending index, backward key tiles by ascending index.
Inside a segment that is descending cost (n_tiles, n_vis), which the tests check
against the counts themselves.
"""
from __future__ import annotations

import numpy as np

SKIP, FULL, MASKED = 0, 1, 2
DIAG_CLAMP = 1 << 30


def clamp_diag(diag: int) -> int:
    return max(-DIAG_CLAMP, min(DIAG_CLAMP, int(diag)))


def tile_class(len_q, len_k, diag, causal, BM, BN, qt, kt) -> int:
    """Class of (query tile qt, key tile kt) by the corner rule."""
    q_first = qt * BM
    q_last = min((qt + 1) * BM, len_q) - 1
    k_first = kt * BN
    k_last_slot = (kt + 1) * BN - 1
    if q_last < q_first or k_first >= len_k:
        return SKIP
    if causal and k_first - q_last > diag:
        return SKIP
    in_range = k_last_slot < len_k
    if in_range and (not causal or k_last_slot - q_first <= diag):
        return FULL
    return MASKED


def tile_class_bruteforce(len_q, len_k, diag, causal, BM, BN, qt, kt) -> int:
    """Class of a tile pair from every (i, j) pair of it (small inputs only)."""
    rows = [i for i in range(qt * BM, (qt + 1) * BM) if i < len_q]
    slots = list(range(kt * BN, (kt + 1) * BN))
    vis = [[(j < len_k) and (not causal or j - i <= diag) for j in slots] for i in rows]
    exist = [[(j < len_k) for j in slots] for _ in rows]
    if not any(v and e for rv, re in zip(vis, exist) for v, e in zip(rv, re)):
        return SKIP
    if all(all(rv) for rv in vis):
        return FULL
    return MASKED


def _segments(cu_q, cu_k):
    cu_q = np.asarray(cu_q, np.int64)
    cu_k = np.asarray(cu_k, np.int64)
    for b in range(len(cu_q) - 1):
        yield b, int(cu_q[b]), int(cu_q[b + 1] - cu_q[b]), int(cu_k[b]), int(cu_k[b + 1] - cu_k[b])


def fwd_items_for_segment(b, q0, lq, k0, lk, diag, causal, BM, BN):
    items = []
    nqt = (lq + BM - 1) // BM
    nkt = (lk + BN - 1) // BN
    for qt in range(nqt):
        classes = [tile_class(lq, lk, diag, causal, BM, BN, qt, kt) for kt in range(nkt)]
        vis = [c for c in classes if c != SKIP]
        n_tiles = len(vis)
        n_full = 0
        while n_full < len(classes) and classes[n_full] == FULL:
            n_full += 1
        # the visible tiles must be a prefix: FULL ... FULL MASKED ... MASKED SKIP ... SKIP
        assert classes[:n_tiles] == [FULL] * n_full + [MASKED] * (n_tiles - n_full)
        items.append((b, qt, q0 + qt * BM, min(BM, lq - qt * BM), k0, lk, n_full, n_tiles,
                      clamp_diag(diag)))
    return items


def bwd_items_for_segment(b, q0, lq, k0, lk, diag, causal, BM, BN):
    items = []
    nqt = (lq + BM - 1) // BM
    nkt = (lk + BN - 1) // BN
    for kt in range(nkt):
        classes = [tile_class(lq, lk, diag, causal, BM, BN, qt, kt) for qt in range(nqt)]
        first = next((qt for qt, c in enumerate(classes) if c != SKIP), nqt)
        n_vis = nqt - first
        n_masked = 0
        while first + n_masked < nqt and classes[first + n_masked] == MASKED:
            n_masked += 1
        # the visible tiles must be a suffix: SKIP ... SKIP MASKED ... MASKED FULL ... FULL
        assert classes[first:] == [MASKED] * n_masked + [FULL] * (n_vis - n_masked)
        items.append((b, kt, k0 + kt * BN, min(BN, lk - kt * BN), q0, lq, first, n_masked,
                      n_vis, clamp_diag(diag)))
    return items


def varlen_plan(cu_q, cu_k, causal, BM, BN, kind="fwd"):
    """Ordered work list of a packed buffer (kind 'fwd' = query tiles, 'bwd' = key tiles)."""
    items, size = [], {}
    for b, q0, lq, k0, lk in _segments(cu_q, cu_k):
        diag = lk - lq
        size[b] = lq + lk
        if kind == "fwd":
            items += fwd_items_for_segment(b, q0, lq, k0, lk, diag, causal, BM, BN)
        else:
            items += bwd_items_for_segment(b, q0, lq, k0, lk, diag, causal, BM, BN)
    return _order(items, kind, size)


def packed_plan(cu_q, cu_k, q_pos, k_pos, causal, BM, BN, kind="fwd"):
    """Ordered work list of a packed context-parallel step: segment b is a chunk pair whose
    first query and key sit at global positions q_pos[b], k_pos[b] (diag = q_pos - k_pos)."""
    items, size = [], {}
    for b, q0, lq, k0, lk in _segments(cu_q, cu_k):
        diag = int(q_pos[b]) - int(k_pos[b])
        size[b] = lq + lk
        if kind == "fwd":
            items += fwd_items_for_segment(b, q0, lq, k0, lk, diag, causal, BM, BN)
        else:
            items += bwd_items_for_segment(b, q0, lq, k0, lk, diag, causal, BM, BN)
    return _order(items, kind, size)


def chunk_plan(len_q, len_k, q_off, k_off, causal, BM, BN, kind="fwd"):
    """Ordered work list of one context-parallel chunk pair (a single segment)."""
    diag = int(q_off) - int(k_off)
    if kind == "fwd":
        items = fwd_items_for_segment(0, 0, len_q, 0, len_k, diag, causal, BM, BN)
    else:
        items = bwd_items_for_segment(0, 0, len_q, 0, len_k, diag, causal, BM, BN)
    return _order(items, kind, {0: len_q + len_k})


def _order(items, kind, size):
    """Segments by size descending (ties: index), then forward tiles by descending
    index, backward tiles by ascending index."""
    sign = -1 if kind == "fwd" else 1
    return sorted(items, key=lambda it: (-size[it[0]], it[0], sign * it[1]))


def tile_counts(items, kind="fwd"):
    """(FULL, MASKED) tile-pair totals of a work list."""
    if kind == "fwd":
        full = sum(it[6] for it in items)
        vis = sum(it[7] for it in items)
    else:
        full = sum(it[8] - it[7] for it in items)
        vis = sum(it[8] for it in items)
    return full, vis - full
