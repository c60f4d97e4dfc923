"""GPU parity: the HIP library against the float64 oracle, element by element.

Sizes span several tiles and ragged tails (segments of 1, BM-1, BM, BM+1, ...),
GQA groups, both head dims, causal and not, float32 and bf16.  Every call goes
through the C ABI (ctypes binding)."""
import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import plan as P
from paper_2502_21231_amd import bs_attn as B
from paper_2502_21231_amd import inputs
from tests.parity_util import TOL, check_close, check_lse, f64, make_qkv, scale_for, to_gpu

pytestmark = pytest.mark.gpu

RAGGED = [1, 63, 64, 65, 127, 128, 129, 200, 3, 517]


def run_varlen(lens, hq, hkv, d, dtype, seed=0, causal=True, bwd=True, rel=0.0):
    T = sum(lens)
    cu = torch.from_numpy(inputs.cu_seqlens(lens))
    q, k, v, do = make_qkv(seed, T, T, hq, hkv, d, dtype)
    qg, kg, vg, dog, cug = to_gpu(q, k, v, do, cu)
    scale = scale_for(d)
    maxlen = max(lens) if lens else 0
    out, lse = B.bs_attn_varlen_fwd(qg, kg, vg, cug, cug, maxlen, causal, scale)
    o_ref, lse_ref = A.varlen_fwd(q, k, v, cu.numpy(), cu.numpy(), causal, scale)
    tol = TOL[dtype]
    check_close("O", f64(out), o_ref, tol["o"], dtype == torch.bfloat16, rel)
    check_lse("LSE", f64(lse), lse_ref, tol["lse"])
    if not bwd:
        return
    # both backward passes take the oracle's forward results (O rounded to the input
    # dtype, LSE as float32), so the backward is compared on identical inputs
    o_in = torch.from_numpy(o_ref).to(dtype)
    lse_in = torch.from_numpy(lse_ref).float()
    dq, dk, dv = B.bs_attn_varlen_bwd(qg, kg, vg, o_in.cuda(), lse_in.cuda(), dog, cug, cug, maxlen,
                                      causal, scale)
    dq_r, dk_r, dv_r = A.varlen_bwd(q, k, v, o_in, lse_in, do, cu.numpy(), cu.numpy(), causal, scale)
    check_close("dQ", f64(dq), dq_r, tol["grad"], dtype == torch.bfloat16, rel)
    check_close("dK", f64(dk), dk_r, tol["grad"], dtype == torch.bfloat16, rel)
    check_close("dV", f64(dv), dv_r, tol["grad"], dtype == torch.bfloat16, rel)


def test_tiny_packed_fp32(gpu):
    """Lengths {64,128,320}, 4/4 heads, d=64, float32, seed 0."""
    run_varlen([64, 128, 320], 4, 4, 64, torch.float32)


@pytest.mark.parametrize("d", [64, 128])
def test_ragged_bf16_gqa(gpu, d):
    run_varlen(RAGGED, 4, 2, d, torch.bfloat16, seed=1)


def test_ragged_bf16_mha_d128(gpu):
    run_varlen(RAGGED[::-1], 3, 3, 128, torch.bfloat16, seed=2)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_noncausal(gpu, dtype):
    run_varlen([70, 1, 190], 2, 1, 64, dtype, seed=3, causal=False)


def test_fp32_d128_ragged(gpu):
    run_varlen([1, 65, 130], 2, 2, 128, torch.float32, seed=4)


def test_long_segment_bf16(gpu):
    """One 2000-token segment next to short ones (many full tiles per row)."""
    run_varlen([2000, 5, 300], 8, 1, 128, torch.bfloat16, seed=5)


def test_empty_segments_and_single_tokens(gpu):
    run_varlen([0, 1, 0, 1, 130, 0], 2, 2, 64, torch.bfloat16, seed=6)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_empty_batches(gpu, dtype):
    """No tokens at all: no segments, and three empty ones (forward and backward return empty
    outputs without error)."""
    for lens in ([], [0, 0, 0]):
        run_varlen(lens, 4, 2, 64, dtype, seed=9)


@pytest.mark.parametrize("tq,tk", [(0, 70), (50, 0)])
def test_chunk_without_queries_or_keys(gpu, tq, tk):
    """A chunk with no query rows (dK = dV = 0) or no keys (O = 0, LSE = -inf, dQ unchanged)."""
    hq, hkv, d, dtype = 4, 2, 128, torch.bfloat16
    q, k, v, do = make_qkv(10, tq, tk, hq, hkv, d, dtype)
    qg, kg, vg, dog = to_gpu(q, k, v, do)
    scale = scale_for(d)
    out, lse = B.bs_attn_chunk_fwd(qg, kg, vg, 500, 400, True, scale)
    o_ref, lse_ref = A.chunk_fwd(q, k, v, 500, 400, True, scale)
    check_close("O", f64(out), o_ref, TOL[dtype]["o"], True)
    check_lse("LSE", f64(lse), lse_ref, TOL[dtype]["lse"])
    o_in = torch.from_numpy(o_ref).to(dtype)
    acc = torch.full((tq, hq, d), 0.5, dtype=torch.float32, device="cuda")
    # dK, dV start as 7 so that the kernel has to write the zeros of a key nobody sees
    dk0 = torch.full(k.shape, 7.0, dtype=dtype, device="cuda")
    dv0 = torch.full(v.shape, 7.0, dtype=dtype, device="cuda")
    acc, dk, dv = B.bs_attn_chunk_bwd(qg, kg, vg, o_in.cuda(), torch.from_numpy(lse_ref).float().cuda(),
                                      dog, 500, 400, True, scale, dq_accum=acc, dk=dk0, dv=dv0)
    g = A.chunk_bwd(q, k, v, o_in, lse_ref, do, 500, 400, True, scale)
    check_close("dQacc", f64(acc), g[0] + 0.5, TOL[dtype]["grad"])
    check_close("dK", f64(dk), g[1], TOL[dtype]["grad"], True)
    check_close("dV", f64(dv), g[2], TOL[dtype]["grad"], True)


@pytest.mark.parametrize("hq,hkv", [(16, 16), (16, 4), (24, 8)])
def test_several_heads_per_xcd(gpu, hq, hkv):
    """Head counts that are multiples of 8: each of the 8 XCDs owns hq/8 query heads (hkv/8 KV
    heads in dK/dV, when that divides), interleaved item by item along each segment's run of
    the work list; ragged segments, an empty one and a single token."""
    run_varlen([300, 1, 770, 0, 64, 129], hq, hkv, 128, torch.bfloat16, seed=8)


def test_varlen_q_shorter_than_k_bottom_right(gpu):
    """len_q != len_k: the causal diagonal is aligned bottom-right."""
    lq, lk = [10, 70, 3], [50, 70, 130]
    hq, hkv, d = 2, 1, 64
    for dtype in (torch.float32, torch.bfloat16):
        cq, ck = torch.from_numpy(inputs.cu_seqlens(lq)), torch.from_numpy(inputs.cu_seqlens(lk))
        q, k, v, do = make_qkv(7, sum(lq), sum(lk), hq, hkv, d, dtype)
        qg, kg, vg, dog, cqg, ckg = to_gpu(q, k, v, do, cq, ck)
        out, lse = B.bs_attn_varlen_fwd(qg, kg, vg, cqg, ckg, 130, True, 0.125)
        o_ref, lse_ref = A.varlen_fwd(q, k, v, cq.numpy(), ck.numpy(), True, 0.125)
        check_close("O", f64(out), o_ref, TOL[dtype]["o"], dtype == torch.bfloat16)
        check_lse("LSE", f64(lse), lse_ref, TOL[dtype]["lse"])
        o_in = torch.from_numpy(o_ref).to(dtype)
        lse_in = torch.from_numpy(lse_ref).float()
        dq, dk, dv = B.bs_attn_varlen_bwd(qg, kg, vg, o_in.cuda(), lse_in.cuda(), dog, cqg, ckg, 130,
                                          True, 0.125)
        g = A.varlen_bwd(q, k, v, o_in, lse_in, do, cq.numpy(), ck.numpy(), True, 0.125)
        for name, got, want in zip("QKV", (dq, dk, dv), g):
            check_close("d" + name, f64(got), want, TOL[dtype]["grad"], dtype == torch.bfloat16)


def test_forward_is_bitwise_deterministic(gpu):
    lens = [300, 129, 64]
    T = sum(lens)
    cu = torch.from_numpy(inputs.cu_seqlens(lens)).cuda()
    q, k, v, _ = make_qkv(8, T, T, 4, 4, 128, torch.bfloat16, with_do=False)
    qg, kg, vg = to_gpu(q, k, v)
    o1, l1 = B.bs_attn_varlen_fwd(qg, kg, vg, cu, cu, 300)
    o2, l2 = B.bs_attn_varlen_fwd(qg, kg, vg, cu, cu, 300)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


@pytest.mark.parametrize("hkv", [4, 1])
def test_backward_is_bitwise_deterministic(gpu, hkv):
    # no atomics: dQ is written once per query tile and dK, dV once per key tile (summed over
    # the query heads of a KV group in a fixed order), so two runs agree bit for bit
    lens = [300, 129, 64, 1]
    T = sum(lens)
    cu = torch.from_numpy(inputs.cu_seqlens(lens)).cuda()
    q, k, v, do = make_qkv(11, T, T, 4, hkv, 128, torch.bfloat16)
    qg, kg, vg, dog = to_gpu(q, k, v, do)
    o, lse = B.bs_attn_varlen_fwd(qg, kg, vg, cu, cu, 300)
    g1 = B.bs_attn_varlen_bwd(qg, kg, vg, o, lse, dog, cu, cu, 300)
    g2 = B.bs_attn_varlen_bwd(qg, kg, vg, o, lse, dog, cu, cu, 300)
    for name, a, b in zip(("dQ", "dK", "dV"), g1, g2):
        assert torch.equal(a, b), name


# ------------------------------------------------------------------ chunk mode
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_chunk_offsets_past_diagonal_straddle_future(gpu, dtype):
    Tq, Tk, hq, hkv, d = 300, 257, 4, 2, 64
    q, k, v, do = make_qkv(9, Tq, Tk, hq, hkv, d, dtype)
    qg, kg, vg, dog = to_gpu(q, k, v, do)
    q_off = 1000
    for k_off in (0, 1000, 900, 1100, 1299, 5000, 743):
        out, lse = B.bs_attn_chunk_fwd(qg, kg, vg, q_off, k_off, True, 0.1)
        o_ref, lse_ref = A.chunk_fwd(q, k, v, q_off, k_off, True, 0.1)
        check_close(f"O@{k_off}", f64(out), o_ref, TOL[dtype]["o"], dtype == torch.bfloat16)
        check_lse(f"LSE@{k_off}", f64(lse), lse_ref, TOL[dtype]["lse"])
        acc = torch.zeros(Tq, hq, d, dtype=torch.float32, device="cuda")
        o_in = torch.from_numpy(o_ref).to(dtype)
        B.bs_attn_chunk_bwd(qg, kg, vg, o_in.cuda(), torch.from_numpy(lse_ref).float().cuda(), dog,
                            q_off, k_off, True, 0.1, dq_accum=acc)
        acc2, dk, dv = B.bs_attn_chunk_bwd(qg, kg, vg, o_in.cuda(), torch.from_numpy(lse_ref).float().cuda(),
                                           dog, q_off, k_off, True, 0.1, dq_accum=acc)
        g = A.chunk_bwd(q, k, v, o_in, lse_ref, do, q_off, k_off, True, 0.1)
        check_close(f"dQacc@{k_off}", f64(acc2), 2 * g[0], 2 * TOL[dtype]["grad"] if dtype == torch.bfloat16 else 1e-5)
        check_close(f"dK@{k_off}", f64(dk), g[1], TOL[dtype]["grad"], dtype == torch.bfloat16)
        check_close(f"dV@{k_off}", f64(dv), g[2], TOL[dtype]["grad"], dtype == torch.bfloat16)


def test_cp_ring_share_fwd_merge_bwd(gpu):
    """A Q shard against 4 KV shards (3 past, 1 diagonal): per-step partials merged on the GPU,
    then the per-step backward with the merged O/LSE, against attention over the union."""
    c, n, hq, hkv, d = 192, 4, 4, 4, 128
    dtype = torch.bfloat16
    q_off = 10 * c
    q = inputs.normal(11, inputs.TID_Q, (c, hq, d), dtype)
    do = inputs.normal(11, inputs.TID_DO, (c, hq, d), dtype)
    ks = [inputs.normal(11, inputs.tid_chunk_k(i), (c, hkv, d), dtype) for i in range(n)]
    vs = [inputs.normal(11, inputs.tid_chunk_v(i), (c, hkv, d), dtype) for i in range(n)]
    k_offs = [(7 + i) * c for i in range(n)]
    qg, dog = to_gpu(q, do)
    parts_o, parts_l = [], []
    for i in range(n):
        o, l = B.bs_attn_chunk_fwd(qg, ks[i].cuda(), vs[i].cuda(), q_off, k_offs[i], True, scale_for(d))
        parts_o.append(o)
        parts_l.append(l)
    om, lm = B.bs_lse_merge(torch.stack(parts_o), torch.stack(parts_l))
    K, V = torch.cat(ks), torch.cat(vs)
    o_ref, lse_ref = A.chunk_fwd(q, K, V, q_off, k_offs[0], True, scale_for(d))
    check_close("O merged", f64(om), o_ref, 2e-2, True)
    check_lse("LSE merged", f64(lm), lse_ref, 1e-3)
    acc = torch.zeros(c, hq, d, dtype=torch.float32, device="cuda")
    o_in = torch.from_numpy(o_ref).to(dtype)
    g = A.chunk_bwd(q, K, V, o_in, lse_ref, do, q_off, k_offs[0], True, scale_for(d))
    for i in range(n):
        _, dk, dv = B.bs_attn_chunk_bwd(qg, ks[i].cuda(), vs[i].cuda(), o_in.cuda(),
                                        torch.from_numpy(lse_ref).float().cuda(), dog, q_off,
                                        k_offs[i], True, scale_for(d), dq_accum=acc)
        check_close(f"dK{i}", f64(dk), g[1][i * c:(i + 1) * c], 2e-2, True)
        check_close(f"dV{i}", f64(dv), g[2][i * c:(i + 1) * c], 2e-2, True)
    dq = B.bs_dq_finalize(acc, torch.empty_like(qg))
    check_close("dQ", f64(dq), g[0], 2e-2, True)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_chunk_bwd_accumulates_kv_over_q_parts(gpu, dtype):
    """Symmetric 2-part split: Q parts 0 and 3 (of 4) against KV parts 0 and 3; dK/dV of each KV
    part summed over both Q parts in float32 accumulators, then rounded by bs_dq_finalize."""
    c, hq, hkv, d = 96, 4, 2, 64
    offs = [0, 3 * c]
    Q = [inputs.normal(15, 100 * i, (c, hq, d), dtype) for i in range(2)]
    dO = [inputs.normal(15, 3 + 100 * i, (c, hq, d), dtype) for i in range(2)]
    K = [inputs.normal(15, inputs.tid_chunk_k(j), (c, hkv, d), dtype) for j in range(2)]
    V = [inputs.normal(15, inputs.tid_chunk_v(j), (c, hkv, d), dtype) for j in range(2)]
    # oracle: each Q part over the union of KV parts (merged), gradients per KV part
    ref = []
    for i in range(2):
        parts = [A.chunk_fwd(Q[i], K[j], V[j], offs[i], offs[j], True, 0.125) for j in range(2)]
        ref.append(A.lse_merge(np.stack([p[0] for p in parts]), np.stack([p[1] for p in parts])))
    gk = [np.zeros((c, hkv, d)) for _ in range(2)]
    gv = [np.zeros((c, hkv, d)) for _ in range(2)]
    gq = [np.zeros((c, hq, d)) for _ in range(2)]
    acc = [torch.zeros(c, hq, d, device="cuda") for _ in range(2)]
    dk = [torch.zeros(c, hkv, d, device="cuda") for _ in range(2)]
    dv = [torch.zeros(c, hkv, d, device="cuda") for _ in range(2)]
    for i in range(2):
        o_in = torch.from_numpy(ref[i][0]).to(dtype)
        l_in = torch.from_numpy(ref[i][1]).float()
        for j in range(2):
            a, b_, c_ = A.chunk_bwd(Q[i], K[j], V[j], o_in, l_in, dO[i], offs[i], offs[j], True, 0.125)
            gq[i] += a
            gk[j] += b_
            gv[j] += c_
            B.bs_attn_chunk_bwd(Q[i].cuda(), K[j].cuda(), V[j].cuda(), o_in.cuda(), l_in.cuda(),
                                dO[i].cuda(), offs[i], offs[j], True, 0.125, acc[i], dk[j], dv[j],
                                kv_accumulate=True)
    bf = dtype == torch.bfloat16
    tol = TOL[dtype]["grad"]
    for j in range(2):
        kf = B.bs_dq_finalize(dk[j], torch.empty(c, hkv, d, dtype=dtype, device="cuda"))
        vf = B.bs_dq_finalize(dv[j], torch.empty(c, hkv, d, dtype=dtype, device="cuda"))
        check_close(f"dK{j}", f64(kf), gk[j], tol, bf)
        check_close(f"dV{j}", f64(vf), gv[j], tol, bf)
        check_close(f"dQ{j}", f64(acc[j]), gq[j], tol)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_lse_merge_with_neg_inf_partials(gpu, dtype):
    n, T, hq, d = 5, 37, 3, 64
    rng = np.random.default_rng(12)
    o = torch.from_numpy(rng.standard_normal((n, T, hq, d)).astype(np.float32)).to(dtype)
    l = rng.standard_normal((n, hq, T)).astype(np.float32) * 3
    l[1, :, :5] = -np.inf            # one partial missing on some rows
    l[:, 0, 7] = -np.inf             # a row where every partial is empty
    l[[0, 2, 3, 4], 2, 9] = -np.inf  # a row with exactly one partial
    lt = torch.from_numpy(l)
    om, lm = B.bs_lse_merge(o.cuda(), lt.cuda())
    o_ref, l_ref = A.lse_merge(f64(o), l)
    check_close("O", f64(om), o_ref, TOL[dtype]["o"], dtype == torch.bfloat16)
    check_lse("LSE", f64(lm), l_ref, 1e-5)
    assert np.all(f64(om)[7, 0] == 0)


# ------------------------------------------------------------------ planner
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_plan_export_bit_exact(gpu, dtype):
    rng = np.random.default_rng(13)
    # up to 1024 segments the planner runs as one workgroup, beyond that as three kernels:
    # 1024, 1025 and 1500 segments (many equal sizes: the index breaks the ties) cover both
    cases = [RAGGED, [0, 0, 5], [32768], list(rng.integers(0, 900, size=40)),
             list(rng.integers(0, 300, size=1024)), list(rng.integers(0, 300, size=1025)),
             list(rng.integers(0, 300, size=1500))]
    for lens in cases:
        lens = [int(x) for x in lens]
        cu = torch.from_numpy(inputs.cu_seqlens(lens)).cuda()
        T = sum(lens)
        for op, kind in ((B.BS_OP_VARLEN_FWD, "fwd"), (B.BS_OP_VARLEN_BWD, "bwd")):
            dims = B.bs_dims(T, T, 8, 2, 128, B.BS_BF16 if dtype == torch.bfloat16 else B.BS_F32)
            items, tm, tn = B.bs_attn_plan_export(op, dims, cu, cu, max(lens + [0]))
            want = P.varlen_plan(cu.cpu().numpy(), cu.cpu().numpy(), True, tm, tn, kind)
            got = [tuple(int(x) for x in r[:9 if kind == "fwd" else 10]) for r in items]
            assert got == [tuple(w) for w in want], (lens[:5], kind)


def test_plan_export_chunk_bit_exact(gpu):
    for (Tq, Tk, qo, ko) in [(32768, 32768, 1015808, 786432), (32768, 32768, 1015808, 1015808),
                             (300, 257, 1000, 1100), (100, 64, 0, 229376), (65, 129, 500, 437)]:
        for op, kind in ((B.BS_OP_CHUNK_FWD, "fwd"), (B.BS_OP_CHUNK_BWD, "bwd")):
            dims = B.bs_dims(Tq, Tk, 4, 4, 128, B.BS_BF16)
            items, tm, tn = B.bs_attn_plan_export(op, dims, None, None, 0, qo, ko, True)
            want = P.chunk_plan(Tq, Tk, qo, ko, True, tm, tn, kind)
            got = [tuple(int(x) for x in r[:9 if kind == "fwd" else 10]) for r in items]
            assert got == [tuple(w) for w in want]


def test_invalid_cu_seqlens_sets_device_status(gpu):
    T = 100
    q, k, v, _ = make_qkv(14, T, T, 2, 2, 64, torch.bfloat16, with_do=False)
    qg, kg, vg = to_gpu(q, k, v)
    dims = B.make_dims(qg, kg)
    for bad, code in (([0, 60, 50, 100], 2), ([1, 50, 100, 100], 1), ([0, 50, 90, 99], 3),
                      ([0, 10, 90, 100], 4)):
        cu = torch.tensor(bad, dtype=torch.int32, device="cuda")
        ws = B.alloc_workspace(B.BS_OP_VARLEN_FWD, dims, "cuda", 3, 64)
        out = torch.full_like(qg, 7.0)
        B.bs_attn_varlen_fwd(qg, kg, vg, cu, cu, 64, True, 0.1, out=out, workspace=ws)
        with pytest.raises(B.BsError) as e:
            B.bs_read_device_status(ws)
        assert e.value.status == B.BS_ERR_DEVICE_STATUS and f"code {code}" in str(e.value)
        assert torch.all(out == 7.0)  # compute kernels wrote nothing
