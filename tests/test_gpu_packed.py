"""GPU parity of the packed context-parallel step (Sec. 7, Dist-attn with packing): the
2N-way zig-zag parts of several subsequences in one buffer, two packed calls per ring step.
Every call is compared with the oracle element by element; the merged and summed results
also with varlen attention over the whole subsequences."""
import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import plan as P
from paper_2502_21231_amd import bs_attn as B
from paper_2502_21231_amd import inputs
from tests.parity_util import TOL, check_close, check_lse, f64, make_qkv, scale_for

pytestmark = pytest.mark.gpu


def ring_calls(lens, n_dev, dev):
    """The packed calls of device `dev` over the whole ring: (cu_q, cu_k, q_pos, k_pos, rows of
    the whole-subsequence buffer that form the call's keys)."""
    calls = []
    for kv_dev in range(n_dev):
        kv_rows = inputs.zigzag_rows(lens, n_dev, kv_dev)
        for crossed in (False, True):
            cu_q, cu_k, qp, kp, kr = inputs.zigzag_step(lens, n_dev, dev, kv_dev, crossed)
            calls.append((cu_q, cu_k, qp, kp, kv_rows[kr]))
    return calls


def g(x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x)) if isinstance(x, np.ndarray) else x
    return (t.to(dtype) if dtype is not None else t).cuda()


@pytest.mark.parametrize("dtype,d", [(torch.float32, 64), (torch.bfloat16, 128)])
def test_packed_zigzag_ring_matches_oracle(gpu, dtype, d):
    """Device 0 of N = 2 over subsequences whose parts are ragged (65 rows) and tile-sized:
    every call's partial (O, LSE) and backward (dQ contribution, dK, dV) against the oracle's
    packed step, and the merged O / summed dQ against varlen attention."""
    lens, n_dev, dev, hq, hkv = [260, 512, 128, 4], 2, 0, 4, 2
    tol = TOL[dtype]
    bf16 = dtype == torch.bfloat16
    T = sum(lens)
    q, k, v, do = make_qkv(21, T, T, hq, hkv, d, dtype)
    sc = scale_for(d)
    rows = inputs.zigzag_rows(lens, n_dev, dev)
    qd, dod = q[rows], do[rows]
    calls = ring_calls(lens, n_dev, dev)
    maxlen = max(lens)
    parts_o, parts_l = [], []
    for cu_q, cu_k, qp, kp, kr in calls:
        o, l = B.bs_attn_packed_chunk_fwd(g(qd), g(k[kr]), g(v[kr]), g(cu_q), g(cu_k), g(qp), g(kp),
                                          maxlen, True, sc)
        o_ref, l_ref = A.packed_chunk_fwd(qd, k[kr], v[kr], cu_q, cu_k, qp, kp, True, sc)
        check_close("O part", f64(o), o_ref, tol["o"], bf16)
        check_lse("LSE part", f64(l), l_ref, tol["lse"])
        parts_o.append(o)
        parts_l.append(l)
    om, lm = B.bs_lse_merge(torch.stack(parts_o), torch.stack(parts_l))
    cu = inputs.cu_seqlens(lens)
    o_full, l_full = A.varlen_fwd(q, k, v, cu, cu, True, sc)
    check_close("O merged", f64(om), o_full[rows], tol["o"], bf16)
    check_lse("LSE merged", f64(lm), l_full[:, rows], tol["lse"])

    # backward of every call with the merged results (the oracle's, on both sides)
    o_in = torch.from_numpy(o_full[rows]).to(dtype)
    l_in = torch.from_numpy(np.ascontiguousarray(l_full[:, rows])).float()
    acc = torch.zeros(len(rows), hq, d, dtype=torch.float32, device="cuda")
    dq_ref = np.zeros((len(rows), hq, d))
    for cu_q, cu_k, qp, kp, kr in calls:
        _, dk, dv = B.bs_attn_packed_chunk_bwd(g(qd), g(k[kr]), g(v[kr]), g(o_in), g(l_in), g(dod),
                                               g(cu_q), g(cu_k), g(qp), g(kp), maxlen, True, sc,
                                               dq_accum=acc)
        a, dk_ref, dv_ref = A.packed_chunk_bwd(qd, k[kr], v[kr], o_in, l_in, dod, cu_q, cu_k, qp, kp,
                                               True, sc)
        check_close("dK part", f64(dk), dk_ref, tol["grad"], bf16)
        check_close("dV part", f64(dv), dv_ref, tol["grad"], bf16)
        dq_ref += a
    dq = B.bs_dq_finalize(acc, torch.empty(len(rows), hq, d, dtype=dtype, device="cuda"))
    check_close("dQ", f64(dq), dq_ref, tol["grad"], bf16)
    dq_full = A.varlen_bwd(q, k, v, o_full, l_full, do, cu, cu, True, sc)[0]
    check_close("dQ vs varlen", f64(dq), dq_full[rows], tol["grad"], bf16)


def test_packed_kv_accumulate_over_both_calls(gpu):
    """The straight and crossed calls of one ring step add into the same float32 dK/dV
    accumulators of the step's KV parts (mapped back to their buffer order)."""
    lens, n_dev, dev, hq, hkv, d = [192, 64, 320], 2, 1, 4, 4, 128
    dtype = torch.bfloat16
    T = sum(lens)
    q, k, v, do = make_qkv(22, T, T, hq, hkv, d, dtype)
    sc = scale_for(d)
    rows = inputs.zigzag_rows(lens, n_dev, dev)
    cu = inputs.cu_seqlens(lens)
    o_full, l_full = A.varlen_fwd(q, k, v, cu, cu, True, sc)
    o_in = torch.from_numpy(o_full[rows]).to(dtype)
    l_in = torch.from_numpy(np.ascontiguousarray(l_full[:, rows])).float()
    kv_dev = 0
    kv_rows = inputs.zigzag_rows(lens, n_dev, kv_dev)
    dk_acc = torch.zeros(len(kv_rows), hkv, d, dtype=torch.float32, device="cuda")
    dv_acc = torch.zeros_like(dk_acc)
    dk_ref = np.zeros((len(kv_rows), hkv, d))
    dv_ref = np.zeros_like(dk_ref)
    acc = torch.zeros(len(rows), hq, d, dtype=torch.float32, device="cuda")
    for crossed in (False, True):
        cu_q, cu_k, qp, kp, kr = inputs.zigzag_step(lens, n_dev, dev, kv_dev, crossed)
        kg = g(k[kv_rows[kr]])
        vg = g(v[kv_rows[kr]])
        dk_c = torch.zeros(len(kr), hkv, d, dtype=torch.float32, device="cuda")
        dv_c = torch.zeros_like(dk_c)
        B.bs_attn_packed_chunk_bwd(g(q[rows]), kg, vg, g(o_in), g(l_in), g(do[rows]), g(cu_q), g(cu_k),
                                   g(qp), g(kp), max(lens), True, sc, dq_accum=acc, dk=dk_c, dv=dv_c,
                                   kv_accumulate=True)
        idx = torch.from_numpy(kr).cuda()
        dk_acc.index_add_(0, idx, dk_c)
        dv_acc.index_add_(0, idx, dv_c)
        _, a, b_ = A.packed_chunk_bwd(q[rows], k[kv_rows[kr]], v[kv_rows[kr]], o_in, l_in, do[rows],
                                      cu_q, cu_k, qp, kp, True, sc)
        np.add.at(dk_ref, kr, a)
        np.add.at(dv_ref, kr, b_)
    check_close("dK accumulated", f64(dk_acc), dk_ref, TOL[dtype]["grad"])
    check_close("dV accumulated", f64(dv_acc), dv_ref, TOL[dtype]["grad"])


def test_packed_plan_export_bit_exact(gpu):
    lens, n_dev = [260, 512, 128, 4, 1024], 2
    T = sum(lens)
    for dev in range(n_dev):
        for kv_dev in range(n_dev):
            for crossed in (False, True):
                cu_q, cu_k, qp, kp, _ = inputs.zigzag_step(lens, n_dev, dev, kv_dev, crossed)
                Tq, Tk = int(cu_q[-1]), int(cu_k[-1])
                for op, kind in ((B.BS_OP_PACKED_CHUNK_FWD, "fwd"), (B.BS_OP_PACKED_CHUNK_BWD, "bwd")):
                    dims = B.bs_dims(Tq, Tk, 8, 2, 128, B.BS_BF16)
                    items, tm, tn = B.bs_attn_plan_export(op, dims, g(cu_q), g(cu_k), max(lens),
                                                          q_pos=g(qp), k_pos=g(kp))
                    want = P.packed_plan(cu_q, cu_k, qp, kp, True, tm, tn, kind)
                    got = [tuple(int(x) for x in r[:9 if kind == "fwd" else 10]) for r in items]
                    assert got == [tuple(w) for w in want], (dev, kv_dev, crossed, kind)
