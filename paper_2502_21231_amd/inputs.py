"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

This module only draws numbers and lays out indices: sequence-length mixes
shaped after the paper's long-tailed datasets (Sec. 3.1, Observation 1, and the
skew it reports), i.i.d. N(0,1) tensors, the token bookkeeping of the zig-zag
packing layout (Sec. 7), and logits with labels for the cross-entropy.  It holds
none of the attention or cross-entropy arithmetic, and it imports neither the HIP
binding nor the oracle.

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


def normal_device(seed: int, tensor_id: int, shape, dtype: torch.dtype = torch.bfloat16,
                  device="cuda") -> torch.Tensor:
    """Tensor of i.i.d. N(0,1) values of `shape` drawn on `device` by torch's seeded Philox
    generator, 2^28 float32 values per draw (draw i seeded from (seed, tensor_id, i)), then cast
    to `dtype`.  For tensors too large to draw on the host; the values differ from normal()'s."""
    n = int(np.prod(shape)) if len(shape) else 1
    out = torch.empty(n, dtype=dtype, device=device)
    g = torch.Generator(device=device)
    step = 1 << 28
    for i, lo in enumerate(range(0, n, step)):
        g.manual_seed(seed * 1000003 + tensor_id * 7919 + i)
        hi = min(n, lo + step)
        out[lo:hi] = torch.randn(hi - lo, generator=g, device=device).to(dtype)
    return out.view(tuple(shape))


TID_LOGITS, TID_LABELS = 40, 41


def xent_inputs(seed: int, rows: int, vocab: int, std: float = 3.0, dtype=torch.bfloat16,
                ignore_every: int = 1024, ignore_index: int = -100, device=None):
    """Logits [rows, vocab] ~ N(0, std^2) in `dtype` and int64 labels uniform in [0, vocab),
    about one row in `ignore_every` labelled ignore_index (the last token of a packed sequence
    has no next token).  With `device` (a GPU) the values are drawn there by torch's seeded
    Philox generator, chunk by chunk of rows, which keeps a 256K x 128K matrix off the host;
    without it they come from the CPU generator of normal().  Either way the same (seed,
    shape, device type) gives the same values."""
    if device is None:
        z = normal(seed, TID_LOGITS, (rows, vocab), torch.float32) * std
        rng = np.random.default_rng([seed, TID_LABELS])
        y = rng.integers(0, vocab, rows)
        y[rng.random(rows) < 1.0 / ignore_every] = ignore_index
        return z.to(dtype), torch.from_numpy(y)
    g = torch.Generator(device=device)
    z = torch.empty(rows, vocab, dtype=dtype, device=device)
    step = max(1, (1 << 28) // max(vocab, 1))  # rows per draw: 256 Mi float32 of scratch at most
    for r0 in range(0, rows, step):
        g.manual_seed(seed * 1000003 + TID_LOGITS * 7919 + r0)
        r1 = min(rows, r0 + step)
        z[r0:r1] = (torch.randn(r1 - r0, vocab, generator=g, device=device) * std).to(dtype)
    g.manual_seed(seed * 1000003 + TID_LABELS * 7919)
    y = torch.randint(0, vocab, (rows,), generator=g, device=device, dtype=torch.int64)
    drop = torch.rand(rows, generator=g, device=device) < 1.0 / ignore_every
    y[drop] = ignore_index
    return z, y


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


# ---------------------------------------------------------------- zig-zag packing layout
# Index bookkeeping only (which tokens a device holds, and the segment tables of one
# packed call); no attention arithmetic.

def zigzag_parts(lengths, n_dev: int, dev: int):
    """Parts that device `dev` holds under the symmetric 2N-way split (Sec. 7, Dist-attn
    with packing): each subsequence (its length a multiple of 2 * n_dev) is cut into 2 * n_dev
    equal parts and the device holds parts dev and 2 * n_dev - 1 - dev.  Returns, in the
    device's buffer order (per subsequence: the low part, then the high part), tuples
    (subsequence, part, global position of the part's first token, part length)."""
    out = []
    for s, L in enumerate(lengths):
        c = L // (2 * n_dev)
        assert c * 2 * n_dev == L, "subsequence length must be a multiple of 2 * n_dev"
        for part in (dev, 2 * n_dev - 1 - dev):
            out.append((s, part, part * c, c))
    return out


def zigzag_step(lengths, n_dev: int, q_dev: int, kv_dev: int, crossed: bool):
    """Segment table of one packed call in which device q_dev attends to the KV parts that
    device kv_dev holds: the "straight" call pairs each subsequence's low query part with
    the low key part and high with high, the "crossed" call low with high and high with low.

    Returns (cu_q, cu_k, q_pos, k_pos, kv_rows): int32 prefix sums over the query buffer of
    q_dev and over the call's key buffer, int64 global positions of each segment's first
    query and key, and kv_rows, the rows of kv_dev's buffer (in zigzag_parts order) that make
    up the call's key buffer, in order (the crossed call swaps each subsequence's two parts)."""
    qp = zigzag_parts(lengths, n_dev, q_dev)
    kp = zigzag_parts(lengths, n_dev, kv_dev)
    kstart = np.concatenate([[0], np.cumsum([p[3] for p in kp])]).astype(np.int64)
    qlen, klen, qpos, kpos, rows = [], [], [], [], []
    for i in range(0, len(qp), 2):  # the two parts of one subsequence
        pairs = [(i, i), (i + 1, i + 1)] if not crossed else [(i, i + 1), (i + 1, i)]
        for a, b in pairs:
            qlen.append(qp[a][3])
            klen.append(kp[b][3])
            qpos.append(qp[a][2])
            kpos.append(kp[b][2])
            rows.append(np.arange(kstart[b], kstart[b] + kp[b][3]))
    cu_q = np.concatenate([[0], np.cumsum(qlen)]).astype(np.int32)
    cu_k = np.concatenate([[0], np.cumsum(klen)]).astype(np.int32)
    return (cu_q, cu_k, np.asarray(qpos, np.int64), np.asarray(kpos, np.int64),
            np.concatenate(rows) if rows else np.zeros(0, np.int64))


def zigzag_rows(lengths, n_dev: int, dev: int):
    """Row of each token of device `dev`'s buffer in the packed buffer of whole subsequences
    (subsequences concatenated in order)."""
    starts = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    return np.concatenate([starts[s] + pos + np.arange(c)
                           for s, _, pos, c in zigzag_parts(lengths, n_dev, dev)])
