"""GPU parity of the fused softmax cross-entropy (Sec. 7, Fused SoftmaxCrossEntropy) against the
float64 oracle, element by element, on seeded logits.

Tolerances, from the fp32 arithmetic: each of the 256 lanes of a row sums at most ceil(V/256)
positive terms below 2^8 (relative error <= n * 2^-24 ~ 3e-5 at V = 128256), the exponent
arguments are rounded once (<= |x| * 2^-24 with |x| < 64) and v_exp_f32 is within an ulp; lse and
loss are therefore held to 5e-5 absolute.  A gradient entry g (p - [j = y]) with p <= 1 is held to
|g| * 1e-4, plus half a bf16 ulp of the reference for a bf16 gradient (the rounding of the stored
value)."""
import numpy as np
import pytest
import torch

from oracle.xent import softmax_xent
from paper_2502_21231_amd import bs_attn as B
from paper_2502_21231_amd import inputs
from tests.parity_util import check_close, f64

pytestmark = pytest.mark.gpu
LSE_TOL = 5e-5


def check_row_results(name, loss, lse, dz, z_cpu, y_cpu, g, ignore_index, bf16):
    l_ref, s_ref, d_ref = softmax_xent(z_cpu, y_cpu, ignore_index, g, with_grad=dz is not None)
    check_close(f"{name} loss", f64(loss), l_ref, LSE_TOL)
    check_close(f"{name} lse", f64(lse), s_ref, LSE_TOL)
    if dz is not None:
        check_close(f"{name} dlogits", f64(dz), d_ref, abs(g) * 1e-4, bf16)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("rows,vocab", [(37, 1), (37, 7), (64, 1000), (33, 32003), (9, 128256),
                                       (21, 16392), (12, 65536), (7, 131072), (5, 131080),
                                       (6, 152064)])
def test_xent_matches_oracle(gpu, dtype, rows, vocab):
    """bf16: the register-resident form for vocab multiples of 8 in (16384, 131072] with 4, 8 and
    16 chunks per lane (16392, 65536, 128256, 131072), the streamed form beyond it (131080,
    152064) and below it (1000); float32 always streams.  Element path for vocab 7, 32003 and 1.
    Labels at both ends of the vocabulary, ignored rows, token-level scale 1/rows."""
    z, y = inputs.xent_inputs(7, rows, vocab, dtype=dtype, ignore_every=8)
    y[0] = 0
    y[-1] = vocab - 1
    y[rows // 2] = -100
    g = 1.0 / rows
    loss, lse, dz = B.bs_softmax_xent(z.cuda(), y.cuda(), -100, g)
    check_row_results("xent", loss, lse, dz, z, y.numpy(), g, -100, dtype == torch.bfloat16)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_xent_in_place_loss_only_and_determinism(gpu, dtype):
    z, y = inputs.xent_inputs(11, 48, 4096, dtype=dtype)
    zg, yg = z.cuda(), y.cuda()
    l1, s1, d1 = B.bs_softmax_xent(zg, yg, grad_scale=0.5)
    l2, s2, d2 = B.bs_softmax_xent(zg, yg, grad_scale=0.5)
    assert torch.equal(l1, l2) and torch.equal(s1, s2) and torch.equal(d1, d2)
    l3, s3, none = B.bs_softmax_xent(zg, yg, grad_scale=0.5, with_grad=False)
    assert none is None and torch.equal(l1, l3) and torch.equal(s1, s3)
    zi = zg.clone()
    l4, s4, d4 = B.bs_softmax_xent(zi, yg, grad_scale=0.5, dlogits=zi)  # gradient over the logits
    assert d4.data_ptr() == zi.data_ptr()
    assert torch.equal(l1, l4) and torch.equal(s1, s4) and torch.equal(d1, zi)


def test_xent_extreme_rows(gpu):
    """Rows with -inf entries (a masked part of the vocabulary), a row that is -inf up to its last
    entry, large offsets (|z| ~ 1e4, where exp overflows without the max shift), a row whose label
    logit dominates (loss ~ 0), an out-of-range label (NaN loss, no one-hot term) and a custom
    ignore index."""
    V = 2048
    z = torch.randn(6, V, generator=torch.Generator().manual_seed(3), dtype=torch.float32) * 2
    z[0, 100:1900] = -float("inf")
    z[1, :-1] = -float("inf")
    z[2] += 10000.0
    z[3] -= 10000.0
    z[4, 5] = 80.0
    y = torch.tensor([50, V - 1, 3, 7, 5, V + 3], dtype=torch.int64)
    loss, lse, dz = B.bs_softmax_xent(z.cuda(), y.cuda(), ignore_index=-7, grad_scale=0.125)
    z64 = z.double().numpy()
    l_ref, s_ref, d_ref = softmax_xent(z64[:5], y[:5].numpy(), -7, 0.125)
    for rows, tol in (([0, 1, 4], LSE_TOL), ([2, 3], 4e-3)):
        # rows 2, 3: at |z| ~ 1e4 an fp32 ulp is ~1e-3, in lse and in the exponent arguments
        check_close(f"loss {rows}", f64(loss[rows]), l_ref[rows], tol)
        check_close(f"lse {rows}", f64(lse[rows]), s_ref[rows], tol)
        check_close(f"dlogits {rows}", f64(dz[rows]), d_ref[rows], 0.125 * max(tol, 1e-4) * 2)
    assert torch.isnan(loss[5])
    # row 5: the label is out of range, so the gradient is g * softmax with no one-hot term (the
    # oracle's gradient for label 0 with the one-hot term added back)
    _, _, d5 = softmax_xent(z64[5:6], np.array([0]), -7, 0.125)
    d5[0, 0] += 0.125
    check_close("dlogits row 5", f64(dz[5]), d5[0], 0.125 * 1e-4)
    z_ign = z.clone()
    y_ign = y.clone()
    y_ign[1] = -7
    loss_i, _, dz_i = B.bs_softmax_xent(z_ign.cuda(), y_ign.cuda(), ignore_index=-7)
    assert loss_i[1].item() == 0.0 and not dz_i[1].any()
