"""Helpers of the GPU parity tests: seeded inputs, tolerances, comparisons."""
from __future__ import annotations

import math

import numpy as np
import torch

from paper_2502_21231_amd import inputs

# Tolerances: float32 problems max |err| <= 1e-5 everywhere; bf16 problems
# <= 2e-2 on O, dQ, dK, dV and <= 1e-3 on the finite LSE entries.
TOL = {
    torch.float32: dict(o=1e-5, lse=1e-5, grad=1e-5),
    torch.bfloat16: dict(o=2e-2, lse=1e-3, grad=2e-2),
}


def make_qkv(seed, T, Tk, hq, hkv, d, dtype, with_do=True):
    q = inputs.normal(seed, inputs.TID_Q, (T, hq, d), dtype)
    k = inputs.normal(seed, inputs.TID_K, (Tk, hkv, d), dtype)
    v = inputs.normal(seed, inputs.TID_V, (Tk, hkv, d), dtype)
    do = inputs.normal(seed, inputs.TID_DO, (T, hq, d), dtype) if with_do else None
    return q, k, v, do


def to_gpu(*ts):
    return [t.cuda() if t is not None else None for t in ts]


def f64(t) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def max_err(got, want) -> float:
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    if got.size == 0:
        return 0.0
    return float(np.max(np.abs(got - want)))


def half_ulp_bf16(x) -> np.ndarray:
    """Half the spacing of bfloat16 numbers at |x| (8 significand bits): the error that
    storing a value in bf16 alone can add."""
    ax = np.abs(np.asarray(x, np.float64))
    e = np.floor(np.log2(np.maximum(ax, 2.0 ** -126)))
    return 0.5 * np.exp2(e - 7)


def check_close(name, got, want, tol, bf16_out=False, rel=0.0):
    """max |got - want| <= tol; for a bf16 result the bound is tol plus half a bf16 ulp of the
    reference (the rounding of the stored value, which no bf16 output can avoid: at |x| >= 8 it
    alone exceeds 2e-2).  `rel` adds rel * |reference| (the randomized float32 cases beyond the
    stated float32 configuration, whose sums run over thousands of terms)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (name, got.shape, want.shape)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    if got.size == 0:
        return 0.0
    diff = np.abs(got - want)
    bound = tol + (half_ulp_bf16(want) if bf16_out else 0.0) + rel * np.abs(want)
    excess = diff - bound
    worst = int(np.argmax(excess))
    assert excess.flat[worst] <= 0, (
        f"{name}: |err| {diff.flat[worst]:.3e} > bound {np.broadcast_to(bound, diff.shape).flat[worst]:.3e} "
        f"at ref {want.flat[worst]:.4g} (max |err| {diff.max():.3e})")
    return float(diff.max())


def check_lse(name, got, want, tol):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape
    ninf_w = np.isneginf(want)
    ninf_g = np.isneginf(got)
    assert np.array_equal(ninf_w, ninf_g), f"{name}: -inf pattern differs ({ninf_w.sum()} vs {ninf_g.sum()})"
    assert not np.any(np.isnan(got)) and not np.any(np.isposinf(got)), f"{name}: NaN/+inf"
    fin = ~ninf_w
    err = max_err(got[fin], want[fin]) if fin.any() else 0.0
    assert err <= tol, f"{name}: max |err| {err:.3e} > {tol:.1e}"
    return err


def scale_for(d):
    return 1.0 / math.sqrt(d)
