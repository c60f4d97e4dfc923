"""GPU parity of the forward steps that fold each ring step into a running (O, LSE) as it is
computed (Sec. 2.4: the ring overlaps the exchange of key shards with the attention of the
shard at hand).  After every step the running state must equal the oracle's combination of the
per-step partials seen so far; the last step's output, attention over the union of the keys."""
import numpy as np
import pytest
import torch

from oracle import attention as A
from paper_2502_21231_amd import bs_attn as B
from paper_2502_21231_amd import inputs
from tests.parity_util import TOL, check_close, check_lse, f64, make_qkv, scale_for, to_gpu
from tests.test_gpu_packed import g, ring_calls

pytestmark = pytest.mark.gpu

# Key shards of one query shard (300 rows at global position 1000): (position, length).  They
# lie in the past, across the diagonal, wholly in the future (a step that sees no key), and are
# ragged against the 64-key tile; the ring visits them in a scrambled order that starts with the
# future shard, so the first step leaves every row at LSE = -inf.
Q_POS, Q_LEN = 1000, 300
SHARDS = [(0, 257), (257, 643), (900, 130), (1100, 64), (5000, 100)]
ORDER = [4, 2, 0, 3, 1]


def shard_kv(j, hkv, d, dtype):
    n = SHARDS[j][1]
    return (inputs.normal(31, inputs.tid_chunk_k(j), (n, hkv, d), dtype),
            inputs.normal(31, inputs.tid_chunk_v(j), (n, hkv, d), dtype))


@pytest.mark.parametrize("dtype,d", [(torch.float32, 64), (torch.bfloat16, 128)])
def test_chunk_fwd_merge_running_state_matches_oracle(gpu, dtype, d):
    hq, hkv = 4, 2
    tol = TOL[dtype]
    bf16 = dtype == torch.bfloat16
    sc = scale_for(d)
    q = inputs.normal(31, inputs.TID_Q, (Q_LEN, hq, d), dtype)
    qg = q.cuda()
    o_run = torch.empty(Q_LEN, hq, d, dtype=torch.float32, device="cuda")
    lse_run = torch.empty(hq, Q_LEN, dtype=torch.float32, device="cuda")
    out = torch.empty(Q_LEN, hq, d, dtype=dtype, device="cuda")
    parts_o, parts_l = [], []
    for s, j in enumerate(ORDER):
        k, v = shard_kv(j, hkv, d, dtype)
        last = s == len(ORDER) - 1
        before = o_run.clone()
        B.bs_attn_chunk_fwd_merge(qg, k.cuda(), v.cuda(), Q_POS, SHARDS[j][0], o_run, lse_run,
                                  accumulate=s > 0, causal=True, scale=sc,
                                  out=out if last else None)
        po, pl = A.chunk_fwd(q, k, v, Q_POS, SHARDS[j][0], True, sc)
        parts_o.append(po)
        parts_l.append(pl)
        ref_o, ref_l = A.lse_merge(np.stack(parts_o), np.stack(parts_l))
        check_lse(f"LSE after step {s}", f64(lse_run), ref_l, tol["lse"])
        if s == 0:
            assert np.isneginf(ref_l).all()  # the future shard: no row sees a key
        if not last:
            # float32 running output: the step's result is never rounded to the input dtype
            check_close(f"O_run after step {s}", f64(o_run), ref_o, tol["o"])
        else:
            check_close("O final", f64(out), ref_o, tol["o"], bf16)
            assert torch.equal(o_run, before), "a call that writes out must leave o_run as it was"


@pytest.mark.parametrize("dtype,d", [(torch.float32, 128), (torch.bfloat16, 64)])
def test_merge_ignores_o_run_where_running_lse_is_neg_inf(gpu, dtype, d):
    """A running state of LSE = -inf with garbage (NaN) in o_run: accumulating into it gives
    bit for bit what replacing it gives."""
    hq, hkv = 4, 4
    q, k, v, _ = make_qkv(5, 200, 333, hq, hkv, d, dtype, with_do=False)
    qg, kg, vg = to_gpu(q, k, v)
    o_a = torch.full((200, hq, d), float("nan"), dtype=torch.float32, device="cuda")
    l_a = torch.full((hq, 200), float("-inf"), dtype=torch.float32, device="cuda")
    B.bs_attn_chunk_fwd_merge(qg, kg, vg, 400, 300, o_a, l_a, accumulate=True)
    o_b = torch.empty_like(o_a)
    l_b = torch.empty_like(l_a)
    B.bs_attn_chunk_fwd_merge(qg, kg, vg, 400, 300, o_b, l_b, accumulate=False)
    assert torch.equal(o_a, o_b) and torch.equal(l_a, l_b)
    # and both hold the step's own partial (rows 0..; keys at 300.. so every row sees a key)
    o_ref, l_ref = A.chunk_fwd(q, k, v, 400, 300, True, scale_for(d))
    check_close("O", f64(o_b), o_ref, TOL[dtype]["o"])
    check_lse("LSE", f64(l_b), l_ref, TOL[dtype]["lse"])


@pytest.mark.parametrize("dtype,d", [(torch.float32, 64), (torch.bfloat16, 128)])
def test_packed_fwd_merge_zigzag_ring(gpu, dtype, d):
    """Device 1 of N = 3 over subsequences with ragged parts: the 6 packed calls of the ring folded
    one by one, checked after every call against the oracle's merge of the packed partials and at
    the end against varlen attention over the whole subsequences."""
    lens, n_dev, dev, hq, hkv = [390, 768, 66, 12], 3, 1, 4, 2
    tol = TOL[dtype]
    bf16 = dtype == torch.bfloat16
    T = sum(lens)
    q, k, v, _ = make_qkv(23, T, T, hq, hkv, d, dtype, with_do=False)
    sc = scale_for(d)
    rows = inputs.zigzag_rows(lens, n_dev, dev)
    qd = q[rows]
    Tq = len(rows)
    calls = ring_calls(lens, n_dev, dev)
    o_run = torch.empty(Tq, hq, d, dtype=torch.float32, device="cuda")
    lse_run = torch.empty(hq, Tq, dtype=torch.float32, device="cuda")
    out = torch.empty(Tq, hq, d, dtype=dtype, device="cuda")
    parts_o, parts_l = [], []
    for s, (cu_q, cu_k, qp, kp, kr) in enumerate(calls):
        last = s == len(calls) - 1
        B.bs_attn_packed_chunk_fwd_merge(g(qd), g(k[kr]), g(v[kr]), g(cu_q), g(cu_k), g(qp), g(kp),
                                         max(lens), o_run, lse_run, accumulate=s > 0, causal=True,
                                         scale=sc, out=out if last else None)
        po, pl = A.packed_chunk_fwd(qd, k[kr], v[kr], cu_q, cu_k, qp, kp, True, sc)
        parts_o.append(po)
        parts_l.append(pl)
        ref_o, ref_l = A.lse_merge(np.stack(parts_o), np.stack(parts_l))
        check_lse(f"LSE after call {s}", f64(lse_run), ref_l, tol["lse"])
        if not last:
            check_close(f"O_run after call {s}", f64(o_run), ref_o, tol["o"])
    cu = inputs.cu_seqlens(lens)
    o_full, l_full = A.varlen_fwd(q, k, v, cu, cu, True, sc)
    check_close("O final", f64(out), o_full[rows], tol["o"], bf16)
    check_lse("LSE final", f64(lse_run), l_full[:, rows], tol["lse"])


@pytest.mark.parametrize("dtype,d,transport", [(torch.float32, 64, "blit"),
                                               (torch.bfloat16, 128, "blit"),
                                               (torch.bfloat16, 64, "dma")])
def test_chunk_ring_rehearsal_matches_oracle(gpu, dtype, d, transport):
    """The single-GPU ring (shards received on a copy stream into two buffers, fused running
    merge, dK/dV sent out on the copy stream): a 200-row query shard that is the last of five
    shards of 200 tokens (ragged against both tile sizes), its own shard first.  O, LSE, dQ, dK, dV
    against the oracle's whole-sequence attention; a second pass gives the same bits."""
    from paper_2502_21231_amd.ring import ChunkRing
    c, n, hq, hkv = 200, 5, 4, 2
    tol = TOL[dtype]
    bf16 = dtype == torch.bfloat16
    sc = scale_for(d)
    q, k, v, do = make_qkv(41, n * c, n * c, hq, hkv, d, dtype)
    me = n - 1
    qd, dod = q[me * c:], do[me * c:]
    order = [me] + list(range(me - 1, -1, -1))
    ring = ChunkRing(qd.cuda(), dod.cuda(), [k[j * c:(j + 1) * c].cuda() for j in order],
                     [v[j * c:(j + 1) * c].cuda() for j in order], me * c, [j * c for j in order],
                     True, sc, transport=transport)
    results = []
    for _ in range(2):
        o, l = ring.forward()
        dq, dks, dvs = ring.backward()
        torch.cuda.synchronize()
        results.append([o.clone(), l.clone(), dq.clone()] + [t.clone() for t in dks + dvs])
    assert all(torch.equal(a, b) for a, b in zip(*results))
    # the oracle: causal attention of the whole 1000-token sequence, the last shard's rows
    o_ref, l_ref = A.chunk_fwd(q, k, v, 0, 0, True, sc)
    check_close("O", f64(o), o_ref[me * c:], tol["o"], bf16)
    check_lse("LSE", f64(l), l_ref[:, me * c:], tol["lse"])
    o_in = torch.from_numpy(o_ref[me * c:]).to(dtype)
    gq, gk, gv = A.chunk_bwd(qd, k, v, o_in, np.ascontiguousarray(l_ref[:, me * c:]), dod, me * c, 0,
                             True, sc)
    check_close("dQ", f64(dq), gq, tol["grad"], bf16)
    for s, j in enumerate(order):
        check_close(f"dK shard {j}", f64(dks[s]), gk[j * c:(j + 1) * c], tol["grad"], bf16)
        check_close(f"dV shard {j}", f64(dvs[s]), gv[j * c:(j + 1) * c], tol["grad"], bf16)


def test_dma_copy_moves_every_byte(gpu):
    """bs_copy_async: an odd byte count between odd offsets inside larger buffers, nothing
    written outside the destination range."""
    src = torch.randint(0, 256, (3 * 1024 * 1024 + 77,), dtype=torch.uint8, device="cuda")
    dst = torch.zeros(3 * 1024 * 1024 + 301, dtype=torch.uint8, device="cuda")
    n = 3 * 1024 * 1024 - 5
    B.bs_copy_async(dst[13:13 + n], src[7:7 + n])
    torch.cuda.synchronize()
    assert torch.equal(dst[13:13 + n], src[7:7 + n])
    assert not dst[:13].any() and not dst[13 + n:].any()
