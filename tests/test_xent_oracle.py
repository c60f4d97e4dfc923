"""Pins of the softmax cross-entropy oracle against what the mathematics fixes: closed forms,
torch's float64 cross_entropy and its autograd gradient (a library routine computing the same
function another way), central finite differences, and invariants."""
import numpy as np
import pytest
import torch

from oracle.xent import softmax_xent


def test_uniform_logits_closed_form():
    """Equal logits: loss = log V exactly, gradient g (1/V - onehot)."""
    T, V, g = 5, 1000, 0.25
    z = np.full((T, V), 3.5)
    y = np.array([0, 999, 17, 500, 3])
    loss, lse, dz = softmax_xent(z, y, grad_scale=g)
    assert np.allclose(loss, np.log(V), rtol=0, atol=1e-12)
    assert np.allclose(lse, 3.5 + np.log(V), rtol=0, atol=1e-12)
    want = np.full((T, V), g / V)
    want[np.arange(T), y] -= g
    assert np.allclose(dz, want, rtol=0, atol=1e-15)


def test_matches_torch_float64_cross_entropy_and_autograd():
    rng = np.random.default_rng(3)
    T, V, g = 33, 517, 1.0 / 29
    z = rng.normal(0, 3, (T, V))
    y = rng.integers(0, V, T)
    y[[4, 20]] = -100
    loss, lse, dz = softmax_xent(z, y, ignore_index=-100, grad_scale=g)
    zt = torch.tensor(z, dtype=torch.float64, requires_grad=True)
    yt = torch.tensor(y)
    ref = torch.nn.functional.cross_entropy(zt, yt, ignore_index=-100, reduction="none")
    assert np.allclose(loss, ref.detach().numpy(), rtol=0, atol=1e-12)
    (ref.sum() * g).backward()
    assert np.allclose(dz, zt.grad.numpy(), rtol=0, atol=1e-14)
    assert np.allclose(lse, torch.logsumexp(zt.detach(), dim=1).numpy(), rtol=0, atol=1e-12)


def test_gradient_is_the_derivative_of_the_loss():
    """Central differences of loss_i in z_ij on a tiny vocabulary."""
    rng = np.random.default_rng(5)
    T, V, h = 3, 7, 1e-6
    z = rng.normal(0, 2, (T, V))
    y = np.array([1, 6, 0])
    _, _, dz = softmax_xent(z, y)
    for i in range(T):
        for j in range(V):
            zp, zm = z.copy(), z.copy()
            zp[i, j] += h
            zm[i, j] -= h
            fd = (softmax_xent(zp, y, with_grad=False)[0][i] - softmax_xent(zm, y, with_grad=False)[0][i]) / (2 * h)
            assert abs(fd - dz[i, j]) < 1e-8, (i, j, fd, dz[i, j])


def test_invariants_shift_large_values_and_ignored_rows():
    rng = np.random.default_rng(9)
    T, V = 6, 300
    z = rng.normal(0, 1, (T, V))
    y = rng.integers(0, V, T)
    y[2] = -1
    loss, lse, dz = softmax_xent(z, y, ignore_index=-1, grad_scale=2.0)
    # adding a constant per row changes lse by it and nothing else, even at magnitudes where a
    # plain exp would overflow
    c = np.array([1000.0, -1000.0, 50.0, 0.0, 700.0, -3.0])[:, None]
    loss2, lse2, dz2 = softmax_xent(z + c, y, ignore_index=-1, grad_scale=2.0)
    assert np.allclose(loss2, loss, atol=1e-9) and np.allclose(lse2, lse + c[:, 0], atol=1e-9)
    assert np.allclose(dz2, dz, atol=1e-12)
    # gradient rows of valid tokens sum to zero and lie in [-g, g]; the ignored row is all zero
    valid = y != -1
    assert np.allclose(dz[valid].sum(axis=1), 0.0, atol=1e-12)
    assert np.all(np.abs(dz) <= 2.0 + 1e-12)
    assert loss[2] == 0.0 and not dz[2].any()
    assert np.isclose(lse[2], np.log(np.exp(z[2]).sum()))
    # a one-entry vocabulary: loss 0, gradient 0
    l1, s1, d1 = softmax_xent(np.array([[4.0], [-2.0]]), np.array([0, 0]))
    assert np.all(l1 == 0) and np.allclose(s1, [4.0, -2.0]) and not d1.any()


def test_rejects_out_of_range_labels():
    with pytest.raises(ValueError):
        softmax_xent(np.zeros((2, 5)), np.array([0, 5]))
    with pytest.raises(ValueError):
        softmax_xent(np.zeros((2, 5)), np.array([-2, 1]), ignore_index=-100)
