"""Float64 CPU oracle for per-device causal attention (test infrastructure only).

This is the plain definition of what the HIP library computes, written for a
reader to check by eye.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import it; the product path never does.

What it follows in the paper (ByteScale, arXiv 2502.21231):
  * Sec. 2.3 (Padding and Packing): packed sequences are processed independently
    under a segmented causal mask -> every segment is attended on its own.
  * Sec. 2.4 (Long Context Training): context parallelism shards Q/K/V along
    the sequence and the ring steps exchange KV slices -> a chunk is attended
    with global positions, returns O and the log-sum-exp, and the partials of
    several KV chunks are combined by their log-sum-exp.
  * Sec. 7 (Implementation, GQA): query heads share KV heads in contiguous
    groups, head h uses KV head h // (Hq / Hkv).
  * Sec. 7 (Dist-attn with packing) and Sec. 2.4 cite FlashAttention as the
    computation; the method's result is exactly softmax attention, so the
    oracle is that definition (FlashAttention only changes the rounding order).

Readings where the paper is silent (no attention formula is printed):
  * softmax attention with an explicit `scale`; LSE is the natural log, fp32
    layout [Hq, T] on the GPU side, float64 here;
  * a row with no visible key has O = 0 and LSE = -inf, and a merge gives such
    a partial weight 0;
  * in varlen mode with len_q != len_k the causal diagonal is aligned
    bottom-right (key j visible to query i iff j <= i + len_k - len_q);
  * in chunk mode key j is visible to query i iff k_off + j <= q_off + i;
  * a packed chunk step (Sec. 7, Dist-attn with packing: the 2N parts of many
    subsequences in one buffer) is a list of segments, each with the global
    positions of its first query and first key, and the chunk rule per segment.

Rows are processed in blocks of query rows only to bound memory: the
arithmetic of every row is exactly the unblocked definition.
"""
from __future__ import annotations

import numpy as np

ROW_BLOCK = 1024


def _as64(x) -> np.ndarray:
    """float64 numpy copy of a numpy array or a CPU torch tensor (bf16 upcast exactly)."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return x.detach().to("cpu", torch.float64).numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.asarray(x, dtype=np.float64)


def visible_mask(len_q: int, len_k: int, diag, causal: bool, rows=None) -> np.ndarray:
    """Boolean [len_q, len_k] (or [r1 - r0, len_k] for rows = (r0, r1)): key j is visible
    to query i iff j - i <= diag.

    `diag` is len_k - len_q for a varlen segment (bottom-right alignment) and
    q_off - k_off for a context-parallel chunk; non-causal sees every key."""
    r0, r1 = (0, len_q) if rows is None else rows
    if not causal:
        return np.ones((r1 - r0, len_k), dtype=bool)
    i = np.arange(r0, r1, dtype=np.int64)[:, None]
    j = np.arange(len_k, dtype=np.int64)[None, :]
    return (j - i) <= int(diag)


def _attend_rows(q, k, v, mask, scale):
    """Softmax attention of query rows q [r, d] over keys k, v [n, d] under mask [r, n].

    Returns O [r, d] and LSE [r]; a row with no visible key gets O = 0, LSE = -inf."""
    s = scale * (q @ k.T)
    s = np.where(mask, s, -np.inf)
    has = mask.any(axis=1)
    m = np.where(has, s.max(axis=1, initial=-np.inf), 0.0)
    e = np.where(mask, np.exp(s - m[:, None]), 0.0)
    l = e.sum(axis=1)
    lse = np.where(has, m + np.log(np.where(has, l, 1.0)), -np.inf)
    p = e / np.where(has, l, 1.0)[:, None]
    o = p @ v
    return o, lse


def _segment_fwd(q, k, v, scale, diag, causal, hq, hkv):
    """O [Lq, Hq, d], LSE [Hq, Lq] of one segment/chunk (q [Lq,Hq,d], k/v [Lk,Hkv,d])."""
    lq, lk = q.shape[0], k.shape[0]
    d = q.shape[2]
    g = hq // hkv
    o = np.zeros((lq, hq, d))
    lse = np.full((hq, lq), -np.inf)
    if lq == 0:
        return o, lse
    for h in range(hq):
        kh, vh = k[:, h // g, :], v[:, h // g, :]
        for r0 in range(0, lq, ROW_BLOCK):
            r1 = min(lq, r0 + ROW_BLOCK)
            mask = visible_mask(lq, lk, diag, causal, (r0, r1))
            if lk == 0:
                continue
            o[r0:r1, h, :], lse[h, r0:r1] = _attend_rows(q[r0:r1, h, :], kh, vh, mask, scale)
    return o, lse


def varlen_fwd(q, k, v, cu_q, cu_k, causal: bool, scale: float):
    """Packed (varlen) attention: q [T, Hq, d], k/v [Tk, Hkv, d], int prefix sums cu_q/cu_k.

    Returns O [T, Hq, d] and LSE [Hq, T] (float64)."""
    q, k, v = _as64(q), _as64(k), _as64(v)
    cu_q, cu_k = np.asarray(cu_q, np.int64), np.asarray(cu_k, np.int64)
    T, hq, d = q.shape
    hkv = k.shape[1]
    o = np.zeros((T, hq, d))
    lse = np.full((hq, T), -np.inf)
    for b in range(len(cu_q) - 1):
        q0, q1, k0, k1 = cu_q[b], cu_q[b + 1], cu_k[b], cu_k[b + 1]
        diag = (k1 - k0) - (q1 - q0)
        ob, lb = _segment_fwd(q[q0:q1], k[k0:k1], v[k0:k1], scale, diag, causal, hq, hkv)
        o[q0:q1], lse[:, q0:q1] = ob, lb
    return o, lse


def chunk_fwd(q, k, v, q_off: int, k_off: int, causal: bool, scale: float):
    """One context-parallel step: the Q shard at global position q_off against the KV shard
    at k_off.  Returns the partial O [Tq, Hq, d] and its LSE [Hq, Tq]."""
    q, k, v = _as64(q), _as64(k), _as64(v)
    hq, hkv = q.shape[1], k.shape[1]
    return _segment_fwd(q, k, v, scale, int(q_off) - int(k_off), causal, hq, hkv)


def packed_chunk_fwd(q, k, v, cu_q, cu_k, q_pos, k_pos, causal: bool, scale: float):
    """One packed context-parallel step: segment b pairs query rows cu_q[b]..cu_q[b+1]-1, whose
    first token sits at global position q_pos[b], with key rows cu_k[b]..cu_k[b+1]-1 starting at
    k_pos[b]; key j is visible to query i iff k_pos[b] + j <= q_pos[b] + i.  Returns the partial
    O [T, Hq, d] and LSE [Hq, T] (rows that see no key: O = 0, LSE = -inf)."""
    q, k, v = _as64(q), _as64(k), _as64(v)
    cu_q, cu_k = np.asarray(cu_q, np.int64), np.asarray(cu_k, np.int64)
    T, hq, d = q.shape
    hkv = k.shape[1]
    o = np.zeros((T, hq, d))
    lse = np.full((hq, T), -np.inf)
    for b in range(len(cu_q) - 1):
        q0, q1, k0, k1 = cu_q[b], cu_q[b + 1], cu_k[b], cu_k[b + 1]
        diag = int(q_pos[b]) - int(k_pos[b])
        ob, lb = _segment_fwd(q[q0:q1], k[k0:k1], v[k0:k1], scale, diag, causal, hq, hkv)
        o[q0:q1], lse[:, q0:q1] = ob, lb
    return o, lse


def lse_merge(o_parts, lse_parts):
    """Combine partials of the same queries over disjoint key sets.

    o_parts [n, T, Hq, d], lse_parts [n, Hq, T]:
      LSE = log sum_c exp(LSE_c),  O = sum_c exp(LSE_c - LSE) O_c.
    A partial with LSE_c = -inf has weight 0; if every partial is -inf, O = 0 and LSE = -inf."""
    o_parts, lse_parts = _as64(o_parts), _as64(lse_parts)
    m = lse_parts.max(axis=0)                                  # [Hq, T]
    finite = np.isfinite(m)
    mm = np.where(finite, m, 0.0)
    w = np.where(np.isfinite(lse_parts), np.exp(lse_parts - mm[None]), 0.0)   # [n, Hq, T]
    tot = w.sum(axis=0)
    lse = np.where(finite, mm + np.log(np.where(finite, tot, 1.0)), -np.inf)
    wn = w / np.where(finite, tot, 1.0)[None]
    o = np.einsum("nht,nthd->thd", wn, o_parts)
    return o, lse


def _segment_bwd(q, k, v, o, lse, do, scale, diag, causal, hq, hkv):
    """Gradients of sum(O * dO) for one segment/chunk, given the (merged) O and LSE.

    P = exp(S - LSE) (0 where masked or LSE = -inf), D = rowsum(dO * O),
    dS = P * (dO V^T - D), dQ = scale dS K, dK = scale dS^T Q, dV = P^T dO;
    dK and dV are summed over the query heads of each KV group."""
    lq, lk = q.shape[0], k.shape[0]
    d = q.shape[2]
    g = hq // hkv
    dq = np.zeros((lq, hq, d))
    dk = np.zeros((lk, hkv, d))
    dv = np.zeros((lk, hkv, d))
    if lq == 0 or lk == 0:
        return dq, dk, dv
    for h in range(hq):
        kv = h // g
        kh, vh = k[:, kv, :], v[:, kv, :]
        for r0 in range(0, lq, ROW_BLOCK):
            r1 = min(lq, r0 + ROW_BLOCK)
            mask = visible_mask(lq, lk, diag, causal, (r0, r1))
            qb, dob, ob, lb = q[r0:r1, h, :], do[r0:r1, h, :], o[r0:r1, h, :], lse[h, r0:r1]
            s = scale * (qb @ kh.T)
            ok = mask & np.isfinite(lb)[:, None]
            p = np.where(ok, np.exp(np.where(ok, s - np.where(np.isfinite(lb), lb, 0.0)[:, None], 0.0)), 0.0)
            D = (dob * ob).sum(axis=1)
            dp = dob @ vh.T
            ds = p * (dp - D[:, None])
            dq[r0:r1, h, :] = scale * (ds @ kh)
            dk[:, kv, :] += scale * (ds.T @ qb)
            dv[:, kv, :] += p.T @ dob
    return dq, dk, dv


def varlen_bwd(q, k, v, o, lse, do, cu_q, cu_k, causal: bool, scale: float):
    """Backward of varlen_fwd: returns dQ [T,Hq,d], dK, dV [Tk,Hkv,d] (float64)."""
    q, k, v, o, lse, do = (_as64(x) for x in (q, k, v, o, lse, do))
    cu_q, cu_k = np.asarray(cu_q, np.int64), np.asarray(cu_k, np.int64)
    hq, hkv = q.shape[1], k.shape[1]
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    for b in range(len(cu_q) - 1):
        q0, q1, k0, k1 = cu_q[b], cu_q[b + 1], cu_k[b], cu_k[b + 1]
        diag = (k1 - k0) - (q1 - q0)
        a, bb, c = _segment_bwd(q[q0:q1], k[k0:k1], v[k0:k1], o[q0:q1], lse[:, q0:q1],
                                do[q0:q1], scale, diag, causal, hq, hkv)
        dq[q0:q1], dk[k0:k1], dv[k0:k1] = a, bb, c
    return dq, dk, dv


def chunk_bwd(q, k, v, o_merged, lse_merged, do, q_off: int, k_off: int, causal: bool,
              scale: float):
    """One context-parallel backward step with the merged O and LSE of all steps.

    Returns this step's dQ contribution [Tq,Hq,d] and the chunk's dK, dV [Tk,Hkv,d]; the dQ
    contributions of all steps sum to the gradient of attention over the union of the chunks."""
    q, k, v, o, lse, do = (_as64(x) for x in (q, k, v, o_merged, lse_merged, do))
    hq, hkv = q.shape[1], k.shape[1]
    return _segment_bwd(q, k, v, o, lse, do, scale, int(q_off) - int(k_off), causal, hq, hkv)


def packed_chunk_bwd(q, k, v, o_merged, lse_merged, do, cu_q, cu_k, q_pos, k_pos, causal: bool,
                     scale: float):
    """Backward of one packed context-parallel step with the merged O and LSE of the query rows:
    this step's dQ contribution [T,Hq,d] and the dK, dV [Tk,Hkv,d] of its key rows."""
    q, k, v, o, lse, do = (_as64(x) for x in (q, k, v, o_merged, lse_merged, do))
    cu_q, cu_k = np.asarray(cu_q, np.int64), np.asarray(cu_k, np.int64)
    hq, hkv = q.shape[1], k.shape[1]
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    for b in range(len(cu_q) - 1):
        q0, q1, k0, k1 = cu_q[b], cu_q[b + 1], cu_k[b], cu_k[b + 1]
        diag = int(q_pos[b]) - int(k_pos[b])
        a, bb, c = _segment_bwd(q[q0:q1], k[k0:k1], v[k0:k1], o[q0:q1], lse[:, q0:q1],
                                do[q0:q1], scale, diag, causal, hq, hkv)
        dq[q0:q1], dk[k0:k1], dv[k0:k1] = a, bb, c
    return dq, dk, dv


def visible_pairs(len_q: int, len_k: int, diag: int, causal: bool) -> int:
    """Exact number of visible (query, key) pairs of one segment/chunk (the work A)."""
    if not causal:
        return len_q * len_k
    total = 0
    for i in range(len_q):
        total += max(0, min(len_k, i + diag + 1))
    return total
