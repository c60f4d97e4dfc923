"""Seeded random sweep of the GPU parity checks: shapes that the fixed cases do not name.

Each case draws, from its own seed, a packed batch (segment lengths mixing tile edges 0, 1,
BM-1, BM, BM+1 with random lengths), a head layout (MHA and GQA groups up to 8), a head dim,
a dtype and causal or not, and compares forward and backward with the float64 oracle at the
tolerances of the fixed cases, except that float32 results may also differ by 1e-5 of the
reference: the stated float32 bound is the tiny float32 configuration's, whose sums run over a
few hundred terms, while a GQA dV here sums up to 8 heads x 420 queries in one float32
accumulator (about sqrt(n) units of 2^-24 relative error; 1e-5 is 168 such units).  Chunk
cases draw q/k lengths and global offsets around, across and away from the diagonal.  Sizes
keep the oracle at a few seconds per case."""
import numpy as np
import pytest
import torch

from oracle import attention as A
from paper_2502_21231_amd import bs_attn as B
from tests.parity_util import TOL, check_close, check_lse, f64, make_qkv, to_gpu
from tests.test_gpu_parity import run_varlen

pytestmark = pytest.mark.gpu

HEADS = [(1, 1), (2, 1), (4, 2), (3, 3), (6, 2), (8, 1), (4, 4)]
REL_F32 = 1e-5  # relative part of the float32 bound for these shapes
EDGES = [0, 1, 63, 64, 65, 127, 128, 129]


def draw_case(seed):
    rng = np.random.default_rng(10_000 + seed)
    n = int(rng.integers(1, 6))
    lens = [int(rng.choice(EDGES)) if rng.random() < 0.4 else int(rng.integers(2, 420)) for _ in range(n)]
    if sum(lens) == 0:
        lens.append(37)
    hq, hkv = HEADS[int(rng.integers(len(HEADS)))]
    d = int(rng.choice([64, 128]))
    dtype = torch.float32 if rng.random() < 0.25 else torch.bfloat16
    causal = bool(rng.random() < 0.75)
    return lens, hq, hkv, d, dtype, causal


@pytest.mark.parametrize("case", range(14))
def test_random_varlen(gpu, case):
    lens, hq, hkv, d, dtype, causal = draw_case(case)
    print(f"case {case}: lens={lens} hq={hq} hkv={hkv} d={d} {dtype} causal={causal}", flush=True)
    run_varlen(lens, hq, hkv, d, dtype, seed=200 + case, causal=causal,
               rel=REL_F32 if dtype == torch.float32 else 0.0)


@pytest.mark.parametrize("case", range(8))
def test_random_chunk(gpu, case):
    rng = np.random.default_rng(20_000 + case)
    tq, tk = int(rng.integers(1, 330)), int(rng.integers(1, 330))
    hq, hkv = HEADS[int(rng.integers(len(HEADS)))]
    d = int(rng.choice([64, 128]))
    dtype = torch.float32 if rng.random() < 0.25 else torch.bfloat16
    causal = bool(rng.random() < 0.8)
    q_off = int(rng.integers(0, 4000))
    # keys entirely past, straddling the diagonal, or partly in the future
    k_off = int(np.clip(q_off + rng.integers(-tk - 200, tq + 50), 0, None))
    scale = float(rng.uniform(0.05, 0.2))
    print(f"case {case}: tq={tq} tk={tk} hq={hq} hkv={hkv} d={d} {dtype} causal={causal} "
          f"q_off={q_off} k_off={k_off}", flush=True)
    q, k, v, do = make_qkv(300 + case, tq, tk, hq, hkv, d, dtype)
    qg, kg, vg, dog = to_gpu(q, k, v, do)
    tol = TOL[dtype]
    bf = dtype == torch.bfloat16
    rel = 0.0 if bf else REL_F32
    out, lse = B.bs_attn_chunk_fwd(qg, kg, vg, q_off, k_off, causal, scale)
    o_ref, lse_ref = A.chunk_fwd(q, k, v, q_off, k_off, causal, scale)
    check_close("O", f64(out), o_ref, tol["o"], bf, rel)
    check_lse("LSE", f64(lse), lse_ref, tol["lse"])
    o_in = torch.from_numpy(o_ref).to(dtype)
    lse_in = torch.from_numpy(lse_ref).float()
    acc = torch.zeros(tq, hq, d, dtype=torch.float32, device="cuda")
    acc, dk, dv = B.bs_attn_chunk_bwd(qg, kg, vg, o_in.cuda(), lse_in.cuda(), dog, q_off, k_off, causal,
                                      scale, dq_accum=acc)
    g = A.chunk_bwd(q, k, v, o_in, lse_ref, do, q_off, k_off, causal, scale)
    check_close("dQacc", f64(acc), g[0], tol["grad"] if bf else 1e-5, rel=rel)
    check_close("dK", f64(dk), g[1], tol["grad"], bf, rel)
    check_close("dV", f64(dv), g[2], tol["grad"], bf, rel)
