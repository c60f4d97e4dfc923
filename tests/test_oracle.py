"""Pins of the float64 oracle against facts the problem itself fixes (no GPU).

Each test checks the oracle against something other than the oracle: a hand
derivation, a closed form, an invariant the paper states, a library routine
computing a special case, brute force, or finite differences.
"""
import math

import numpy as np
import pytest
import torch

from oracle import attention as A
from paper_2502_21231_amd import inputs


def rnd(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def lens_to_cu(lens):
    return inputs.cu_seqlens(lens)


# ---------------------------------------------------------------- hand example
def test_hand_worked_example():
    """Two keys with scores 0 and ln 3 give weights 1/4 and 3/4 (derived by hand)."""
    q = np.array([[[5.0, 5.0]], [[1.0, 0.0]]])
    k = np.array([[[0.0, 0.0]], [[math.log(3.0), 0.0]]])
    v = np.array([[[4.0, 0.0]], [[0.0, 8.0]]])
    cu = [0, 2]
    o, lse = A.varlen_fwd(q, k, v, cu, cu, True, 1.0)
    assert np.allclose(o[0, 0], [4.0, 0.0], atol=1e-14)      # row 0 sees key 0 only
    assert np.allclose(o[1, 0], [1.0, 6.0], atol=1e-14)      # 1/4*(4,0) + 3/4*(0,8)
    assert lse[0, 0] == pytest.approx(0.0, abs=1e-14)
    assert lse[0, 1] == pytest.approx(math.log(4.0), abs=1e-14)
    do = np.array([[[0.0, 0.0]], [[1.0, 1.0]]])
    dq, dk, dv = A.varlen_bwd(q, k, v, o, lse, do, cu, cu, True, 1.0)
    # D = dO.O = 7; dP = (4, 8); dS = (1/4*(4-7), 3/4*(8-7)) = (-3/4, 3/4)
    assert np.allclose(dq[1, 0], [0.75 * math.log(3.0), 0.0], atol=1e-14)
    assert np.allclose(dq[0, 0], [0.0, 0.0], atol=1e-14)
    assert np.allclose(dk[:, 0], [[-0.75, 0.0], [0.75, 0.0]], atol=1e-14)
    assert np.allclose(dv[:, 0], [[0.25, 0.25], [0.75, 0.75]], atol=1e-14)


# ---------------------------------------------------------------- closed forms
def test_single_token_segment_returns_its_v_row():
    lens = [1, 5, 1, 3]
    cu = lens_to_cu(lens)
    T, hq, hkv, d = sum(lens), 4, 2, 8
    q, k, v = rnd((T, hq, d), 1), rnd((T, hkv, d), 2), rnd((T, hkv, d), 3)
    scale = 0.37
    o, lse = A.varlen_fwd(q, k, v, cu, cu, True, scale)
    for t in (0, 6):
        for h in range(hq):
            assert np.allclose(o[t, h], v[t, h // 2], atol=1e-14)
            assert lse[h, t] == pytest.approx(scale * q[t, h] @ k[t, h // 2], abs=1e-12)


@pytest.mark.parametrize("causal", [True, False])
def test_zero_query_gives_running_mean(causal):
    lens = [7, 3, 12]
    cu = lens_to_cu(lens)
    T, h, d = sum(lens), 2, 5
    q = np.zeros((T, h, d))
    k, v = rnd((T, h, d), 4), rnd((T, h, d), 5)
    o, lse = A.varlen_fwd(q, k, v, cu, cu, causal, 0.5)
    for b, L in enumerate(lens):
        s = cu[b]
        for i in range(L):
            n = i + 1 if causal else L
            assert np.allclose(o[s + i], v[s:s + n].mean(axis=0), atol=1e-13)
            assert np.allclose(lse[:, s + i], math.log(n), atol=1e-13)


def test_value_shift_shifts_output_key_shift_shifts_lse():
    lens = [9, 4]
    cu = lens_to_cu(lens)
    T, h, d = sum(lens), 3, 6
    q, k, v = rnd((T, h, d), 6), rnd((T, h, d), 7), rnd((T, h, d), 8)
    scale = 0.4
    o, lse = A.varlen_fwd(q, k, v, cu, cu, True, scale)
    c = rnd((d,), 9)
    o2, lse2 = A.varlen_fwd(q, k, v + c, cu, cu, True, scale)
    assert np.allclose(o2, o + c, atol=1e-12)
    assert np.allclose(lse2, lse, atol=1e-12)
    o3, lse3 = A.varlen_fwd(q, k + c, v, cu, cu, True, scale)
    assert np.allclose(o3, o, atol=1e-12)
    shift = scale * np.einsum("thd,d->ht", q, c)
    assert np.allclose(lse3, lse + shift, atol=1e-12)


def test_gradient_sums_per_segment():
    """Rows of P sum to 1 and rows of dS sum to 0, so sum_j dK_j = 0 and
    sum_j dV_j = sum over the group's query heads of sum_i dO_i, per segment."""
    lens = [6, 11, 2]
    cu = lens_to_cu(lens)
    T, hq, hkv, d = sum(lens), 4, 2, 5
    q, k, v, do = rnd((T, hq, d), 10), rnd((T, hkv, d), 11), rnd((T, hkv, d), 12), rnd((T, hq, d), 13)
    o, lse = A.varlen_fwd(q, k, v, cu, cu, True, 0.3)
    dq, dk, dv = A.varlen_bwd(q, k, v, o, lse, do, cu, cu, True, 0.3)
    for b in range(len(lens)):
        s, e = cu[b], cu[b + 1]
        assert np.allclose(dk[s:e].sum(axis=0), 0.0, atol=1e-12)
        for g in range(hkv):
            assert np.allclose(dv[s:e, g].sum(axis=0), do[s:e, 2 * g:2 * g + 2].sum(axis=(0, 1)), atol=1e-12)


# ---------------------------------------------------------------- invariants
def test_permuting_segments_permutes_outputs():
    """Packed segments are independent (segmented mask), and the gradient does not depend on
    how sequences are assigned/packed (Eq. 1 = Eq. 2)."""
    lens = [5, 9, 1, 14, 3]
    cu = lens_to_cu(lens)
    T, hq, hkv, d = sum(lens), 2, 1, 4
    q, k, v, do = rnd((T, hq, d), 20), rnd((T, hkv, d), 21), rnd((T, hkv, d), 22), rnd((T, hq, d), 23)
    o, lse = A.varlen_fwd(q, k, v, cu, cu, True, 0.5)
    grads = A.varlen_bwd(q, k, v, o, lse, do, cu, cu, True, 0.5)
    perm = [3, 0, 4, 2, 1]
    idx = np.concatenate([np.arange(cu[p], cu[p + 1]) for p in perm])
    cu2 = lens_to_cu([lens[p] for p in perm])
    o2, lse2 = A.varlen_fwd(q[idx], k[idx], v[idx], cu2, cu2, True, 0.5)
    assert np.allclose(o2, o[idx], atol=1e-13)
    assert np.allclose(lse2, lse[:, idx], atol=1e-13)
    g2 = A.varlen_bwd(q[idx], k[idx], v[idx], o2, lse2, do[idx], cu2, cu2, True, 0.5)
    for a, b in zip(g2, grads):
        assert np.allclose(a, b[idx], atol=1e-13)


def test_gqa_equals_mha_with_replicated_kv():
    lens = [10, 7]
    cu = lens_to_cu(lens)
    T, hq, hkv, d = sum(lens), 6, 2, 4
    G = hq // hkv
    q, k, v, do = rnd((T, hq, d), 30), rnd((T, hkv, d), 31), rnd((T, hkv, d), 32), rnd((T, hq, d), 33)
    o, lse = A.varlen_fwd(q, k, v, cu, cu, True, 0.6)
    kr, vr = np.repeat(k, G, axis=1), np.repeat(v, G, axis=1)
    o2, lse2 = A.varlen_fwd(q, kr, vr, cu, cu, True, 0.6)
    assert np.allclose(o, o2, atol=1e-13) and np.allclose(lse, lse2, atol=1e-13)
    dq, dk, dv = A.varlen_bwd(q, k, v, o, lse, do, cu, cu, True, 0.6)
    dq2, dk2, dv2 = A.varlen_bwd(q, kr, vr, o2, lse2, do, cu, cu, True, 0.6)
    assert np.allclose(dq, dq2, atol=1e-13)
    assert np.allclose(dk, dk2.reshape(T, hkv, G, d).sum(axis=2), atol=1e-13)
    assert np.allclose(dv, dv2.reshape(T, hkv, G, d).sum(axis=2), atol=1e-13)


def test_split_kv_merge_equals_unsplit():
    """Any split of the keys into parts, merged by LSE, equals the unsplit result (ring steps)."""
    Lq, Lk, hq, hkv, d = 13, 29, 4, 4, 5
    q, k, v = rnd((Lq, hq, d), 40), rnd((Lk, hkv, d), 41), rnd((Lk, hkv, d), 42)
    q_off, k_off = 40, 20           # chunk-mode diagonal: key at 20+j visible to 40+i iff j <= i+20
    o, lse = A.chunk_fwd(q, k, v, q_off, k_off, True, 0.4)
    cuts = [0, 4, 17, 18, Lk]
    parts = [A.chunk_fwd(q, k[a:b], v[a:b], q_off, k_off + a, True, 0.4)
             for a, b in zip(cuts[:-1], cuts[1:])]
    om, lm = A.lse_merge(np.stack([p[0] for p in parts]), np.stack([p[1] for p in parts]))
    assert np.allclose(om, o, atol=1e-13) and np.allclose(lm, lse, atol=1e-13)


def test_cp_chunks_fwd_merge_bwd_equal_direct_attention():
    """A Q shard against several KV shards (one diagonal, others in the past), merged, equals
    attention of the Q shard over the union; summed chunk backward gives the union's gradient."""
    c, n, hq, hkv, d = 8, 4, 2, 2, 4
    q_off = 3 * c
    q = rnd((c, hq, d), 50)
    ks = [rnd((c, hkv, d), 51 + i) for i in range(n)]
    vs = [rnd((c, hkv, d), 61 + i) for i in range(n)]
    do = rnd((c, hq, d), 70)
    parts = [A.chunk_fwd(q, ks[i], vs[i], q_off, i * c, True, 0.5) for i in range(n)]
    om, lm = A.lse_merge(np.stack([p[0] for p in parts]), np.stack([p[1] for p in parts]))
    K, V = np.concatenate(ks), np.concatenate(vs)
    o, lse = A.chunk_fwd(q, K, V, q_off, 0, True, 0.5)
    assert np.allclose(om, o, atol=1e-13) and np.allclose(lm, lse, atol=1e-13)
    dq, dK, dV = A.chunk_bwd(q, K, V, o, lse, do, q_off, 0, True, 0.5)
    dq_sum = np.zeros_like(dq)
    for i in range(n):
        a, b_, c_ = A.chunk_bwd(q, ks[i], vs[i], om, lm, do, q_off, i * c, True, 0.5)
        dq_sum += a
        assert np.allclose(b_, dK[i * c:(i + 1) * c], atol=1e-13)
        assert np.allclose(c_, dV[i * c:(i + 1) * c], atol=1e-13)
    assert np.allclose(dq_sum, dq, atol=1e-13)


def test_rows_without_visible_keys_and_all_masked_merge():
    q, k, v = rnd((4, 1, 3), 80), rnd((4, 1, 3), 81), rnd((4, 1, 3), 82)
    o, lse = A.chunk_fwd(q, k, v, 0, 100, True, 1.0)      # keys entirely in the future
    assert np.all(o == 0) and np.all(np.isneginf(lse))
    o, lse = A.chunk_fwd(q, k, v, 0, 2, True, 1.0)        # rows 0,1 see nothing, rows 2,3 do
    assert np.all(o[:2] == 0) and np.all(np.isneginf(lse[:, :2])) and np.all(np.isfinite(lse[:, 2:]))
    om, lm = A.lse_merge(np.zeros((3, 4, 1, 3)), np.full((3, 1, 4), -np.inf))
    assert np.all(om == 0) and np.all(np.isneginf(lm))
    dq, dk, dv = A.chunk_bwd(q, k, v, np.zeros((4, 1, 3)), np.full((1, 4), -np.inf),
                             rnd((4, 1, 3), 83), 0, 100, True, 1.0)
    assert np.all(dq == 0) and np.all(dk == 0) and np.all(dv == 0)


def test_zigzag_split_gives_equal_mask_area():
    """Sec. 7 (Dist-attn with packing): a sequence split into 2N parts, device i holding parts
    i and 2N-1-i, gives every device the same mask area, (2N-1)c^2 + c(c+1) for part size c."""
    for N, c in [(4, 5), (3, 7), (2, 1)]:
        areas = []
        for dev in range(N):
            mine = [dev, 2 * N - 1 - dev]
            area = 0
            for qp in mine:
                for kp in range(2 * N):
                    area += A.visible_pairs(c, c, (qp - kp) * c, True)
            areas.append(area)
        assert all(a == (2 * N - 1) * c * c + c * (c + 1) for a in areas), areas
    # the 141B-shaped zig-zag share at part size 32K: c = 32768, N = 4
    c = 32768
    assert (2 * 4 - 1) * c * c + c * (c + 1) == 8_589_967_360


@pytest.mark.parametrize("n_dev", [2, 3])
def test_packed_zigzag_ring_equals_varlen_attention(n_dev):
    """Sec. 7 (Dist-attn with packing): every device holds parts i and 2N-1-i of several
    subsequences in one buffer; over the ring it attends to every device's KV parts, two packed
    calls per step (straight and crossed part pairs).  Merging a device's partials gives varlen
    attention over the whole subsequences at its rows; the summed packed backward gives the
    varlen gradients (dK/dV summed over every device and step, scattered back to the tokens)."""
    lens = [4 * n_dev, 6 * n_dev, 2 * n_dev * 2]
    hq, hkv, d, sc = 2, 1, 4, 0.7
    T = sum(lens)
    q, k, v, do = (rnd((T, h, d), 300 + i) for i, h in enumerate((hq, hkv, hkv, hq)))
    cu = lens_to_cu(lens)
    o_ref, l_ref = A.varlen_fwd(q, k, v, cu, cu, True, sc)
    dq_ref, dk_ref, dv_ref = A.varlen_bwd(q, k, v, o_ref, l_ref, do, cu, cu, True, sc)
    dk_sum, dv_sum = np.zeros_like(dk_ref), np.zeros_like(dv_ref)
    for dev in range(n_dev):
        rows = inputs.zigzag_rows(lens, n_dev, dev)
        calls = []
        for kv_dev in range(n_dev):
            kv_rows = inputs.zigzag_rows(lens, n_dev, kv_dev)
            for crossed in (False, True):
                cu_q, cu_k, qp, kp, kr = inputs.zigzag_step(lens, n_dev, dev, kv_dev, crossed)
                calls.append((cu_q, cu_k, qp, kp, kv_rows[kr]))
        parts = [A.packed_chunk_fwd(q[rows], k[g], v[g], cq, ck, qp, kp, True, sc)
                 for cq, ck, qp, kp, g in calls]
        om, lm = A.lse_merge(np.stack([p[0] for p in parts]), np.stack([p[1] for p in parts]))
        assert np.allclose(om, o_ref[rows], atol=1e-12)
        assert np.allclose(lm, l_ref[:, rows], atol=1e-12)
        dq = np.zeros((len(rows), hq, d))
        for cq, ck, qp, kp, g in calls:
            a, b_, c_ = A.packed_chunk_bwd(q[rows], k[g], v[g], om, lm, do[rows], cq, ck, qp, kp,
                                           True, sc)
            dq += a
            np.add.at(dk_sum, g, b_)
            np.add.at(dv_sum, g, c_)
        assert np.allclose(dq, dq_ref[rows], atol=1e-12)
    assert np.allclose(dk_sum, dk_ref, atol=1e-12)
    assert np.allclose(dv_sum, dv_ref, atol=1e-12)


def test_visible_pairs_bruteforce():
    for lq, lk, diag in [(5, 5, 0), (3, 7, 4), (7, 3, -4), (6, 6, 10), (6, 6, -10), (9, 4, 2)]:
        brute = int(A.visible_mask(lq, lk, diag, True).sum())
        assert A.visible_pairs(lq, lk, diag, True) == brute


# ---------------------------------------------------------------- library special case
def test_matches_torch_sdpa_float64_per_sequence():
    F = torch.nn.functional
    lens = [1, 17, 40]
    cu = lens_to_cu(lens)
    T, h, d = sum(lens), 3, 8
    q, k, v, do = rnd((T, h, d), 90), rnd((T, h, d), 91), rnd((T, h, d), 92), rnd((T, h, d), 93)
    scale = 1 / math.sqrt(d)
    o, lse = A.varlen_fwd(q, k, v, cu, cu, True, scale)
    dq, dk, dv = A.varlen_bwd(q, k, v, o, lse, do, cu, cu, True, scale)
    for b in range(len(lens)):
        s, e = cu[b], cu[b + 1]
        tq, tk, tv = (torch.tensor(x[s:e].transpose(1, 0, 2), requires_grad=True) for x in (q, k, v))
        out = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True, scale=scale)
        out.backward(torch.tensor(do[s:e].transpose(1, 0, 2)))
        assert np.allclose(out.detach().numpy().transpose(1, 0, 2), o[s:e], atol=1e-12)
        assert np.allclose(tq.grad.numpy().transpose(1, 0, 2), dq[s:e], atol=1e-12)
        assert np.allclose(tk.grad.numpy().transpose(1, 0, 2), dk[s:e], atol=1e-12)
        assert np.allclose(tv.grad.numpy().transpose(1, 0, 2), dv[s:e], atol=1e-12)
        ref_lse = torch.logsumexp(
            (tq @ tk.transpose(1, 2) * scale).masked_fill(
                torch.ones(e - s, e - s, dtype=torch.bool).triu(1), -math.inf), dim=-1)
        assert np.allclose(ref_lse.detach().numpy(), lse[:, s:e], atol=1e-12)


# ---------------------------------------------------------------- finite differences
def test_gradients_match_central_finite_differences():
    lens = [1, 3, 5]
    cu = lens_to_cu(lens)
    T, hq, hkv, d = sum(lens), 4, 2, 4
    q, k, v, do = rnd((T, hq, d), 100), rnd((T, hkv, d), 101), rnd((T, hkv, d), 102), rnd((T, hq, d), 103)
    scale = 0.7

    def loss(q_, k_, v_):
        o_, _ = A.varlen_fwd(q_, k_, v_, cu, cu, True, scale)
        return float((o_ * do).sum())

    o, lse = A.varlen_fwd(q, k, v, cu, cu, True, scale)
    grads = A.varlen_bwd(q, k, v, o, lse, do, cu, cu, True, scale)
    eps = 1e-6
    for which, g in zip(range(3), grads):
        base = [q, k, v]
        num = np.zeros_like(base[which])
        it = np.nditer(base[which], flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            plus = [x.copy() for x in base]
            minus = [x.copy() for x in base]
            plus[which][idx] += eps
            minus[which][idx] -= eps
            num[idx] = (loss(*plus) - loss(*minus)) / (2 * eps)
        assert np.allclose(num, g, rtol=1e-6, atol=1e-7), (which, np.abs(num - g).max())


# ---------------------------------------------------------------- workloads
def test_lognormal_lengths_golden():
    import json
    import os
    with open(os.path.join(os.path.dirname(__file__), "golden", "lognormal_lengths_seed0.json")) as f:
        gold = json.load(f)
    assert inputs.lognormal_packed_lengths(0) == gold["lengths"]
    assert sum(gold["lengths"]) == 32768


def test_workload_areas():
    """Exact visible-pair counts of the packed workloads (closed form vs the oracle's count)."""
    want = {0: 71_253_208, 1: 40_069_418, 2: 225_933_286, 3: 438_388_129, 4: 157_515_915}
    for seed, a in want.items():
        lens = inputs.lognormal_packed_lengths(seed)
        assert sum(l * (l + 1) // 2 for l in lens) == a
    lens = inputs.mixed_long_short_lengths(0)
    assert sum(lens) == 131072 and max(lens) == 60642
    assert sum(l * (l + 1) // 2 for l in lens) == 1_937_101_526
    # tiny packed config {64, 128, 320}
    assert sum(A.visible_pairs(l, l, 0, True) for l in (64, 128, 320)) == 61_696
