"""The allocation-free varlen forward (plan scratch in a device array owned by the library)
against bs_attn_varlen_fwd with a caller workspace: two calls in a row, the second smaller,
each compared bit for bit (same kernels, same plan) and against the oracle's bound."""
import numpy as np
import pytest
import torch

from oracle import attention as A
from paper_2502_21231_amd import bs_attn as B
from paper_2502_21231_amd import inputs
from tests.parity_util import TOL, check_close, check_lse, f64, make_qkv, scale_for, to_gpu

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_noalloc_forward_matches_workspace_forward(gpu, dtype):
    cases = [([300, 1, 0, 517, 129, 64], 8, 2, 128), ([70, 33], 4, 4, 64)]  # second call smaller
    for seed, (lens, hq, hkv, d) in enumerate(cases):
        print(f"noalloc case seed={seed} lens={lens} hq={hq} hkv={hkv} d={d} {dtype}", flush=True)
        T = sum(lens)
        cu = torch.from_numpy(inputs.cu_seqlens(lens))
        q, k, v, _ = make_qkv(seed, T, T, hq, hkv, d, dtype, with_do=False)
        qg, kg, vg, cug = to_gpu(q, k, v, cu)
        scale = scale_for(d)
        # preallocated outputs, filled with garbage so that every entry must be written
        out_n = torch.full_like(qg, 7.0)
        lse_n = torch.full((hq, T), 7.0, dtype=torch.float32, device=gpu)
        B.bs_attn_varlen_fwd_noalloc(qg, kg, vg, cug, cug, max(lens), True, scale, out=out_n,
                                     lse=lse_n)
        out_w, lse_w = B.bs_attn_varlen_fwd(qg, kg, vg, cug, cug, max(lens), True, scale)
        torch.cuda.synchronize()
        assert torch.equal(out_n.view(torch.int16 if dtype == torch.bfloat16 else torch.int32),
                           out_w.view(torch.int16 if dtype == torch.bfloat16 else torch.int32))
        assert torch.equal(lse_n.view(torch.int32), lse_w.view(torch.int32))
        o_ref, lse_ref = A.varlen_fwd(q, k, v, cu.numpy(), cu.numpy(), True, scale)
        tol = TOL[dtype]
        check_close("O", f64(out_n), o_ref, tol["o"], bf16_out=dtype == torch.bfloat16)
        check_lse("LSE", f64(lse_n), lse_ref, tol["lse"])


def test_noalloc_forward_rejects_a_plan_beyond_its_scratch(gpu):
    T = (B.BS_NOALLOC_SCRATCH_BYTES // 48) * 128 + 128  # more work items than the scratch holds
    q = torch.empty((T, 1, 64), dtype=torch.bfloat16, device=gpu)
    k = torch.empty((T, 1, 64), dtype=torch.bfloat16, device=gpu)
    cu = torch.tensor([0, T], dtype=torch.int32, device=gpu)
    with pytest.raises(B.BsError) as e:
        B.bs_attn_varlen_fwd_noalloc(q, k, k, cu, cu, T, True, 0.125)
    assert e.value.status == B.BS_ERR_WORKSPACE
