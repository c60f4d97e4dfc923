"""GPU parity where element offsets need more than 32 bits.

2^21 packed tokens with 16 query heads and 8 KV heads at d = 128: Q, O, dO and dQ hold 2^32
bf16 values (8 GiB each), K, V, dK and dV 2^31 (their byte offsets pass 2^32), in about 2,000
ragged segments of 0..2,048 tokens.  Every address the kernels form from a token index and a
head stride must be 64-bit, so the oracle recomputes in full (every row, head and key) the
segments where Q's element offset crosses 2^31 and 3 * 2^30, the first segment and the last
two (Q offsets near 2^32, K byte offsets near 2^32).  The backward of those segments takes the
GPU's row-checked O and LSE as its inputs.  Every other segment is held by finiteness and by
its gradient sums (sum_j dK_j = 0, sum_j dV_j = the group's sum of dO), checked for all
segments and KV heads on the GPU in float64.

The inputs are drawn on the GPU (inputs.normal_device): 52 GB of bf16 would take minutes to
draw on the host.
"""
import math

import numpy as np
import pytest
import torch

from oracle import attention as A
from paper_2502_21231_amd import bs_attn as B
from paper_2502_21231_amd import inputs
from tests.parity_util import check_close, check_lse, f64

pytestmark = pytest.mark.gpu
BF = torch.bfloat16
T, HQ, HKV, D = 1 << 21, 16, 8, 128
G = HQ // HKV
MAXLEN = 2048
SCALE = 1.0 / math.sqrt(D)
SEED = 7


def ragged_lengths(seed):
    """Segment lengths summing to T: uniform in 2..MAXLEN, with about 1% empty and 1% single
    tokens."""
    rng = np.random.default_rng([seed, 77])
    out, tot = [], 0
    while tot < T:
        u = rng.random()
        n = 0 if u < 0.01 else 1 if u < 0.02 else int(rng.integers(2, MAXLEN + 1))
        n = min(n, T - tot)
        out.append(n)
        tot += n
    return out


def test_offsets_beyond_32_bits(gpu):
    lens = ragged_lengths(SEED)
    cu = inputs.cu_seqlens(lens)
    assert int(cu[-1]) == T and max(lens) <= MAXLEN
    dev = torch.device("cuda")
    print(f"large offsets: {len(lens)} segments, T={T}, hq={HQ}, hkv={HKV}, d={D}", flush=True)
    q = inputs.normal_device(SEED, inputs.TID_Q, (T, HQ, D), BF, dev)
    k = inputs.normal_device(SEED, inputs.TID_K, (T, HKV, D), BF, dev)
    v = inputs.normal_device(SEED, inputs.TID_V, (T, HKV, D), BF, dev)
    do = inputs.normal_device(SEED, inputs.TID_DO, (T, HQ, D), BF, dev)
    cug = torch.from_numpy(cu).to(dev)
    out, lse = B.bs_attn_varlen_fwd(q, k, v, cug, cug, MAXLEN, True, SCALE)
    dq, dk, dv = B.bs_attn_varlen_bwd(q, k, v, out, lse, do, cug, cug, MAXLEN, True, SCALE)
    torch.cuda.synchronize()
    for name, t in (("O", out), ("dQ", dq), ("dK", dk), ("dV", dv)):
        assert bool(torch.isfinite(t).all()), f"{name}: non-finite values"
    assert not bool(torch.isnan(lse).any()) and not bool(torch.isposinf(lse).any())

    def seg_of(row):
        return int(np.searchsorted(cu, row, side="right")) - 1  # never an empty segment

    nonempty = [b for b, n in enumerate(lens) if n > 0]
    row_per_elem = HQ * D
    picks = sorted({nonempty[0], nonempty[-2], nonempty[-1],
                    seg_of((1 << 31) // row_per_elem), seg_of((3 << 30) // row_per_elem)})
    for b in picks:
        s, n = int(cu[b]), lens[b]
        qs, ks, vs, dos = (t[s:s + n].cpu() for t in (q, k, v, do))
        cu1 = np.array([0, n], np.int64)
        o_ref, l_ref = A.varlen_fwd(qs, ks, vs, cu1, cu1, True, SCALE)
        o_gpu, l_gpu = out[s:s + n].cpu(), lse[:, s:s + n].cpu()
        tag = f"seg {b} (rows {s}..{s + n - 1})"
        check_close(f"O {tag}", f64(o_gpu), o_ref, 2e-2, True)
        check_lse(f"LSE {tag}", f64(l_gpu), l_ref, 1e-3)
        dq_r, dk_r, dv_r = A.varlen_bwd(qs, ks, vs, o_gpu, l_gpu, dos, cu1, cu1, True, SCALE)
        check_close(f"dQ {tag}", f64(dq[s:s + n]), dq_r, 2e-2, True)
        check_close(f"dK {tag}", f64(dk[s:s + n]), dk_r, 2e-2, True)
        check_close(f"dV {tag}", f64(dv[s:s + n]), dv_r, 2e-2, True)

    # gradient sums of every segment and KV head, in float64 on the GPU, 2^18 rows at a time
    nseg = len(lens)
    seg_id = torch.from_numpy(np.repeat(np.arange(nseg), lens)).to(dev)
    sk = torch.zeros(nseg, HKV, D, dtype=torch.float64, device=dev)
    sv, so = torch.zeros_like(sk), torch.zeros_like(sk)
    step = 1 << 18
    for r0 in range(0, T, step):
        ids = seg_id[r0:r0 + step]
        sk.index_add_(0, ids, dk[r0:r0 + step].double())
        sv.index_add_(0, ids, dv[r0:r0 + step].double())
        so.index_add_(0, ids, do[r0:r0 + step].double().reshape(-1, HKV, G, D).sum(dim=2))
    n_terms = torch.tensor([max(n, 1) * G for n in lens], dtype=torch.float64, device=dev)
    tol = 0.02 * n_terms.sqrt() + 1e-3 * so.abs().amax(dim=(1, 2))
    err_k = sk.abs().amax(dim=(1, 2))
    err_v = (sv - so).abs().amax(dim=(1, 2))
    worst_k, worst_v = int(torch.argmax(err_k - tol)), int(torch.argmax(err_v - tol))
    assert float(err_k[worst_k]) <= float(tol[worst_k]), ("sum dK", worst_k, float(err_k[worst_k]))
    assert float(err_v[worst_v]) <= float(tol[worst_v]), ("sum dV", worst_v, float(err_v[worst_v]))
    del q, k, v, do, out, lse, dq, dk, dv, sk, sv, so, seg_id
    torch.cuda.empty_cache()


def row_oracle(qrow, K, V, dorow, q_pos, k_pos):
    """O, LSE, dQ of one query row [1, 1, d] against one key range [C, 1, d]."""
    o, l = A.chunk_fwd(qrow, K, V, q_pos, k_pos, True, SCALE)
    dq, _, _ = A.chunk_bwd(qrow, K, V, torch.from_numpy(o).to(BF), l, dorow, q_pos, k_pos, True,
                           SCALE)
    return o, l, dq


def chunk_case(q, do, k_off, C, rows, check_keys, merge):
    """Forward and backward of the 2^21 query rows at position 0 against a C-key chunk at
    position k_off, through the C ABI; sampled rows against the oracle row by row.  With
    check_keys, dK and dV of every key are checked element by element (only rows at or after
    k_off see the chunk, so the oracle needs only those rows); otherwise by their sums over the
    chunk.  With merge, a two-way LSE merge of 2^33 elements is checked too."""
    dev = q.device
    kc = inputs.normal_device(SEED, inputs.tid_chunk_k(0), (C, HKV, D), BF, dev)
    vc = inputs.normal_device(SEED, inputs.tid_chunk_v(0), (C, HKV, D), BF, dev)
    out, lse = B.bs_attn_chunk_fwd(q, kc, vc, 0, k_off, True, SCALE)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out).all()) and not bool(torch.isnan(lse).any())
    if k_off > 0:  # rows before the chunk see no key: O = 0, LSE = -inf
        assert not bool(out[:k_off].any()) and bool(torch.isneginf(lse[:, :k_off]).all())

    if merge:
        # two partials that hold the same output with LSEs l and l + 1: O comes back bit for
        # bit (a weighted mean of one bf16 value), the LSE is l + ln(1 + e), -inf stays -inf
        parts = torch.stack([out, out])
        lse_parts = torch.stack([lse, lse + 1.0])
        mo, ml = B.bs_lse_merge(parts, lse_parts)
        torch.cuda.synchronize()
        assert torch.equal(mo, out), "merged O differs from its two identical partials"
        want = lse.double() + math.log1p(math.e)
        assert torch.equal(torch.isneginf(ml), torch.isneginf(lse)), "merged LSE: -inf pattern"
        fin = torch.isfinite(lse)
        lerr = float((ml.double()[fin] - want[fin]).abs().max()) if bool(fin.any()) else 0.0
        assert lerr <= 1e-5, ("merged LSE", lerr)
        del parts, lse_parts, mo, ml
        torch.cuda.empty_cache()

    dq_acc = torch.zeros(T, HQ, D, dtype=torch.float32, device=dev)
    dq_acc, dk, dv = B.bs_attn_chunk_bwd(q, kc, vc, out, lse, do, 0, k_off, True, SCALE,
                                         dq_accum=dq_acc)
    dq = B.bs_dq_finalize(dq_acc, torch.empty_like(q))
    torch.cuda.synchronize()
    del dq_acc
    for name, t in (("dQ", dq), ("dK", dk), ("dV", dv)):
        assert bool(torch.isfinite(t).all()), f"{name}: non-finite values"
    if k_off > 0:
        assert not bool(dq[:k_off].any()), "dQ of rows that see no key"

    rng = np.random.default_rng([SEED, 78, k_off])
    for i in rows:
        for h in sorted({0, HQ - 1, int(rng.integers(0, HQ))}):
            hk = h // G
            o, l, g = row_oracle(q[i:i + 1, h:h + 1].cpu(), kc[:, hk:hk + 1].cpu(),
                                 vc[:, hk:hk + 1].cpu(), do[i:i + 1, h:h + 1].cpu(), i, k_off)
            tag = f"row {i} h{h} (chunk at {k_off})"
            check_close(f"O {tag}", f64(out[i, h]), o[0, 0], 2e-2, True)
            check_lse(f"LSE {tag}", f64(lse[h, i:i + 1]), l[0], 1e-3)
            check_close(f"dQ {tag}", f64(dq[i, h]), g[0, 0], 2e-2, True)

    if check_keys:
        # every key, all heads: the rows from k_off on, with the GPU's row-checked O and LSE
        r0 = k_off
        qb, dob, ob = (t[r0:].cpu() for t in (q, do, out))
        _, gk, gv = A.chunk_bwd(qb, kc.cpu(), vc.cpu(), ob, lse[:, r0:].cpu(), dob, r0, k_off, True,
                                SCALE)
        check_close(f"dK (chunk at {k_off})", f64(dk), gk, 2e-2, True)
        check_close(f"dV (chunk at {k_off})", f64(dv), gv, 2e-2, True)
    else:
        # sum_j dK_j = 0 and sum_j dV_j = the group's sum of dO (this chunk is the only step)
        so = torch.zeros(HKV, D, dtype=torch.float64, device=dev)
        for s0 in range(0, T, 1 << 18):
            so += do[s0:s0 + (1 << 18)].double().reshape(-1, HKV, G, D).sum(dim=(0, 2))
        sk, sv = dk.double().sum(dim=0), dv.double().sum(dim=0)
        tol = 0.02 * math.sqrt(C * G) + 1e-3 * float(so.abs().max())
        assert float(sk.abs().max()) <= tol, ("sum dK", float(sk.abs().max()), tol)
        assert float((sv - so).abs().max()) <= tol, ("sum dV", float((sv - so).abs().max()), tol)
    del kc, vc, out, lse, dq, dk, dv
    torch.cuda.empty_cache()


def test_chunk_merge_finalize_offsets_beyond_32_bits(gpu):
    """The context-parallel path at the same sizes: 2^21 query rows (2^32 elements per
    Q-sized tensor, a float32 dQ accumulator of 16 GiB and its finalize) against a 256-key
    chunk
      * at the end of the sequence: only the last rows (Q offsets near 2^32) see it, the rest
        get O = 0 and LSE = -inf; a two-way LSE merge of 2^33 elements; dK and dV of every key
        element by element;
      * at the start: every row sees it; sampled rows where Q's offset crosses 2^31 and
        3 * 2^30; dK and dV by their sums (each key sums 2^22 bf16 products of P and dS,
        whose rounding alone is of the order of the 2e-2 bound there)."""
    C = 256
    dev = torch.device("cuda")
    q = inputs.normal_device(SEED, inputs.TID_Q, (T, HQ, D), BF, dev)
    do = inputs.normal_device(SEED, inputs.TID_DO, (T, HQ, D), BF, dev)
    row_per_elem = HQ * D
    chunk_case(q, do, T - C, C, [0, T - C - 1, T - C, T - C + 1, T - 2, T - 1], True, True)
    chunk_case(q, do, 0, C, [0, 1, C - 1, C, (1 << 31) // row_per_elem,
                             (3 << 30) // row_per_elem, T - 1], False, False)
    del q, do
    torch.cuda.empty_cache()
