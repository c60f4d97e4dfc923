"""Softmax cross-entropy over a large vocabulary, fused with its gradient: the oracle.

TEST INFRASTRUCTURE.  Only tests/, the smoke check and the benchmark's CPU-baseline leg may
import this module; the library never does.  Plain float64 NumPy, written from the definition,
sharing no code with the HIP path.

Sec. 7 (Implementation, Fused SoftmaxCrossEntropy): the next-token loss over a vocabulary of
about 128K entries is taken from bf16 logits while the arithmetic runs in higher precision, and
the operations around it are fused into one kernel.  What that kernel computes, per token i with
logits z_i (V entries) and label y_i:
    lse_i  = log sum_j exp(z_ij)
    loss_i = lse_i - z_i,y_i
    dz_ij  = g * (exp(z_ij - lse_i) - [j == y_i])
where g is the upstream gradient of every token's loss: g = 1/N for the token-level loss that
divides the summed loss by the batch's token count (Sec. 5.1, Loss and Model Update).  A token
whose label is ignore_index (padding) contributes loss 0 and gradient 0; its lse is still the
row's log-sum-exp.
"""
from __future__ import annotations

import numpy as np


def _as64(x) -> np.ndarray:
    if hasattr(x, "detach"):  # a torch tensor
        x = x.detach().to("cpu")
        import torch
        x = x.to(torch.float64).numpy()
    return np.asarray(x, dtype=np.float64)


def softmax_xent(logits, labels, ignore_index: int = -100, grad_scale: float = 1.0,
                 with_grad: bool = True):
    """logits [T, V], labels int [T].  Returns (loss [T], lse [T], dz [T, V] or None) in float64.
    A label outside [0, V) that is not ignore_index raises ValueError."""
    z = _as64(logits)
    if z.ndim != 2:
        raise ValueError("logits must be [T, V]")
    T, V = z.shape
    y = np.asarray(labels, dtype=np.int64).reshape(-1)
    if y.shape[0] != T:
        raise ValueError("one label per row")
    valid = y != ignore_index
    if np.any((y[valid] < 0) | (y[valid] >= V)):
        raise ValueError("label out of range")
    rows = np.nonzero(valid)[0]
    if T == 0:
        return np.zeros(0), np.zeros(0), (np.zeros((0, V)) if with_grad else None)
    m = z.max(axis=1, keepdims=True)                       # shift by the row max: exp never overflows
    e = np.exp(z - m)
    lse = m[:, 0] + np.log(e.sum(axis=1))
    loss = np.zeros(T)
    loss[rows] = lse[rows] - z[rows, y[rows]]
    if not with_grad:
        return loss, lse, None
    dz = np.exp(z - lse[:, None])
    dz[rows, y[rows]] -= 1.0
    dz[~valid] = 0.0
    return loss, lse, dz * grad_scale
