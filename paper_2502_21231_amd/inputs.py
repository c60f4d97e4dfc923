"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

This module only draws numbers: sequence-length mixes shaped after the paper's
long-tailed datasets (Sec. 3.1, Observation 1, and the skew it reports) and
i.i.d. N(0,1) tensors.  It holds none of the attention arithmetic, and it
imports neither the HIP binding nor the oracle.

Tensors are drawn as float32 from ``numpy.random.default_rng([seed, tensor_id,
chunk])`` over fixed 4 Mi-element chunks (so the values never depend on the
thread count) and, for bf16, rounded to nearest-even by ``torch``'s float32 ->
bfloat16 conversion.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

_CHUNK = 1 << 22

# tensor ids used by every caller, so that the oracle side and the GPU side draw
# exactly the same values for the same (seed, role)
TID_Q, TID_K, TID_V, TID_DO = 0, 1, 2, 3


def tid_chunk_k(c: int) -> int:
    """Tensor id of the c-th KV chunk's K (context-parallel workloads)."""
    return 10 + c


def tid_chunk_v(c: int) -> int:
    """Tensor id of the c-th KV chunk's V (context-parallel workloads)."""
    return 20 + c


def normal(seed: int, tensor_id: int, shape, dtype: torch.dtype = torch.bfloat16) -> torch.Tensor:
    """CPU tensor of i.i.d. N(0,1) values of `shape`, drawn as float32 and cast to `dtype`."""
    n = int(np.prod(shape)) if len(shape) else 1
    out = np.empty(n, dtype=np.float32)
    nchunks = max(1, (n + _CHUNK - 1) // _CHUNK)

    def fill(i: int) -> None:
        lo, hi = i * _CHUNK, min(n, (i + 1) * _CHUNK)
        if hi > lo:
            np.random.default_rng([seed, tensor_id, i]).standard_normal(
                hi - lo, dtype=np.float32, out=out[lo:hi])

    if nchunks == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(min(8, nchunks)) as ex:
            list(ex.map(fill, range(nchunks)))
    t = torch.from_numpy(out).reshape(tuple(shape))
    return t if dtype == torch.float32 else t.to(dtype)


def cu_seqlens(lengths) -> np.ndarray:
    """int32 prefix sums [0, l0, l0+l1, ...] of a list of segment lengths."""
    cu = np.zeros(len(lengths) + 1, dtype=np.int64)
    cu[1:] = np.cumsum(np.asarray(lengths, dtype=np.int64))
    return cu.astype(np.int32)


# log-normal sigma such that 80% of the draws are <= 4x the median:
# sigma = ln 4 / Phi^-1(0.8) (median 1K, "nearly 80% of the samples are 4K or shorter")
LOGNORMAL_SIGMA = math.log(4.0) / 0.8416212335729143


def lognormal_packed_lengths(seed: int, total: int = 32768, median: int = 1024,
                             sigma: float = LOGNORMAL_SIGMA, lo: int = 128,
                             hi: int = 32768) -> list[int]:
    """Long-tailed packed buffer: log-normal lengths clipped to [lo, hi], appended
    until `total` tokens are reached; the last segment is truncated to fit."""
    rng = np.random.default_rng(seed)
    out: list[int] = []
    filled = 0
    while filled < total:
        l = int(round(rng.lognormal(math.log(median), sigma)))
        l = min(max(l, lo), hi)
        l = min(l, total - filled)
        out.append(l)
        filled += l
    return out


def mixed_long_short_lengths(seed: int, total: int = 131072) -> list[int]:
    """1-2 long segments in [32K, 64K] that hold about half of the tokens, the
    rest filled with U[256, 4K] short segments (last one truncated), shuffled."""
    rng = np.random.default_rng(seed)
    longs = [int(rng.integers(32768, 65536, endpoint=True))]
    if longs[0] <= 49152:
        longs.append(int(rng.integers(32768, 81920 - longs[0], endpoint=True)))
    segs = list(longs)
    filled = sum(longs)
    while filled < total:
        l = int(rng.integers(256, 4096, endpoint=True))
        l = min(l, total - filled)
        segs.append(l)
        filled += l
    perm = rng.permutation(len(segs))
    return [segs[i] for i in perm]
