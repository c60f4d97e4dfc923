"""Benchmark of the per-device HDP attention hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

A step is one causal attention forward + backward of the workload through the
C ABI: device planning, forward, the dQ kernel (which also forms D =
rowsum(dO * O)) and the dK/dV kernel (and for the context-parallel workloads the
per-step chunk calls with their dQ finalize, plus the LSE merge, or the running
merge of the ring rehearsal).  Two workloads measure the
other rows of the build: hdp_batch7b (the HDP planners, checked by running every
planned micro-batch) and xent_llama3_256k (the fused softmax cross-entropy, its
own HBM metric).  Inputs are resident in HBM before timing starts; K steps are
timed with HIP events on the library's stream, bracketed by device
synchronisation.  Prints ONE JSON line.

FLOPs are causal-adjusted: forward 4*d*Hq*A, backward 10*d*Hq*A, where A is
the exact number of visible (query, key) pairs.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

BF16_PEAK_TFLOPS = 256 * 2.4e9 * 4096 / 1e12   # 2516.6: MI355X dense bf16 MFMA (AMD's 2.5 PF)
REPO = os.path.dirname(os.path.abspath(__file__))
# sources whose text fixes each timed kernel (a counter record applies only to them)
KERNEL_SOURCES = {"fwd": ["fwd_bf16.hip", "attn.hpp", "common.hpp"],
                  "bwd_dq": ["dq_bf16.hip", "bwd_common.hpp", "attn.hpp", "common.hpp"],
                  "bwd_dkdv": ["dkdv_bf16.hip", "bwd_common.hpp", "attn.hpp", "common.hpp"],
                  "xent": ["xent.hip", "common.hpp"]}


def kernel_source_hash(kernel):
    """sha256 of the kernel's source files with comments and blank lines removed, so that a
    counter record outlives edits of the comments alone."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(REPO, "paper_2502_21231_amd", "csrc", f), encoding="utf-8") as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        code = "\n".join(line.rstrip() for line in text.splitlines() if line.strip())
        h.update(code.encode("utf-8"))
    return h.hexdigest()


def recorded_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` on `workload` from the counter record in a
    profiles/*.md summary (a fenced json block with a "traffic_record" key), or None
    when there is no record or the kernel's sources changed since it was taken."""
    import glob
    want = kernel_source_hash(kernel)
    for path in sorted(glob.glob(os.path.join(REPO, "profiles", "*.md"))):
        text = open(path).read()
        for block in text.split("```json")[1:]:
            try:
                rec = json.loads(block.split("```")[0])
            except ValueError:
                continue
            for r in rec.get("traffic_record", []):
                if r.get("workload") == workload and r.get("kernel") == kernel and r.get("source_sha256") == want:
                    return r["read_bytes"] + r["write_bytes"]
    return None
HBM_PEAK_GBS = 8000.0

WORKLOADS = {
    "packed7b": "7B-shaped packed varlen causal attention fwd+bwd: 32 q heads, 32 kv heads, "
                "head_dim 128, one 32768-token buffer of log-normal lengths (median 1K, "
                "clipped to [128, 32K]), seed 0",
    "gqa70b": "70B-shaped GQA packed varlen causal attention fwd+bwd: 64 q heads, 8 kv heads, "
              "head_dim 128, 131072 tokens, 1-2 long segments (32K-64K) + U[256,4K] shorts",
    "cp7b": "context-parallel share on the 7B shape: a 32768-token Q chunk at offset 1015808 vs 8 "
            "KV chunks of 32768 (7 past, 1 diagonal), fwd x8 + LSE merge + bwd x8",
    "cp7b_ring": "the cp7b share run as one device of an 8-step ring on one GPU: its own (diagonal) "
                 "KV shard first, then the 7 before it, each next shard received by a device copy "
                 "on a second HIP stream into a double buffer while the current step computes; "
                 "every forward step folded into a running float32 (O, LSE) in the kernel epilogue "
                 "(no partials, no merge pass); the backward receives the shards the same way and "
                 "sends each shard's dK, dV out on the copy stream",
    "hdp_batch7b": "HDP planning checked on the GPU: a 524288-token global batch of log-normal "
                   "lengths (median 1K, clipped to [128, 128K]) planned for 16 ranks of 8K tokens "
                   "by the native Alg. 1 / Alg. 2 planners with T(s) fitted from this library's "
                   "measured attention; a step runs the attention fwd+bwd (7B shape: 32/32 heads, "
                   "head_dim 128) of every micro-batch of the DP-Balance plan (a context-parallel "
                   "sequence once, whole)",
    "xent_llama3_256k": "fused softmax cross-entropy fwd+bwd (loss, lse and the bf16 gradient of "
                        "bf16 logits) over 262144 tokens x a 128256-entry vocabulary (LLaMA3), "
                        "logits N(0, 3^2), labels uniform, ~1/1024 ignored; the gradient is "
                        "scaled by 1/(valid tokens) and written to its own buffer",
    "zigzag141b": "141B-shaped zig-zag CP share: 48 q heads, 8 kv heads, Q halves of 32768 at 0 "
                  "and 229376 against the matching KV halves, fwd + merge + bwd",
    "zigzag_packed7b": "7B-shaped packed CP share (dist-attn with packing): device 0 of a 4-way "
                       "zig-zag split of 4 subsequences (131072, 65536, 32768, 32768 tokens), its "
                       "2 parts of each (65536 query tokens) against every device's KV parts over "
                       "the ring: 8 packed calls fwd + 8-way merge + 8 packed calls bwd; 32 q "
                       "heads, 32 kv heads, head_dim 128",
}
ZIGZAG_PACKED = dict(lens=[131072, 65536, 32768, 32768], n_dev=4, dev=0, hq=32, hkv=32, d=128)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def visible_pairs_chunk(lq, lk, diag):
    tot = 0
    for i in range(lq):
        tot += max(0, min(lk, i + diag + 1))
    return tot


def setup_varlen(name, seed, dev):
    import torch
    from paper_2502_21231_amd import inputs
    if name == "packed7b":
        lens, hq, hkv = inputs.lognormal_packed_lengths(seed), 32, 32
    else:
        lens, hq, hkv = inputs.mixed_long_short_lengths(seed), 64, 8
    d, T = 128, sum(lens)
    cu = torch.from_numpy(inputs.cu_seqlens(lens))
    q = inputs.normal(seed, inputs.TID_Q, (T, hq, d))
    k = inputs.normal(seed, inputs.TID_K, (T, hkv, d))
    v = inputs.normal(seed, inputs.TID_V, (T, hkv, d))
    do = inputs.normal(seed, inputs.TID_DO, (T, hq, d))
    A = sum(l * (l + 1) // 2 for l in lens)
    return dict(lens=lens, hq=hq, hkv=hkv, d=d, T=T, A=A, cu_cpu=cu, q_cpu=q, k_cpu=k, v_cpu=v,
                do_cpu=do, cu=cu.to(dev), q=q.to(dev), k=k.to(dev), v=v.to(dev), do=do.to(dev))


def run_varlen_bench(args, dev):
    import torch
    from paper_2502_21231_amd import bs_attn as B
    W = setup_varlen(args.workload, args.seed, dev)
    hq, hkv, d, T, A = W["hq"], W["hkv"], W["d"], W["T"], W["A"]
    maxlen = max(W["lens"])
    scale = 1.0 / math.sqrt(d)
    dims = B.make_dims(W["q"], W["k"])
    nseq = len(W["lens"])
    ws_f = B.alloc_workspace(B.BS_OP_VARLEN_FWD, dims, dev, nseq, maxlen)
    ws_b = B.alloc_workspace(B.BS_OP_VARLEN_BWD, dims, dev, nseq, maxlen)
    out = torch.empty_like(W["q"])
    lse = torch.empty(hq, T, dtype=torch.float32, device=dev)
    dq, dk, dv = torch.empty_like(W["q"]), torch.empty_like(W["k"]), torch.empty_like(W["v"])

    def step():
        B.bs_attn_varlen_fwd(W["q"], W["k"], W["v"], W["cu"], W["cu"], maxlen, True, scale, out, lse, ws_f)
        B.bs_attn_varlen_bwd(W["q"], W["k"], W["v"], out, lse, W["do"], W["cu"], W["cu"], maxlen, True,
                             scale, dq, dk, dv, ws_b)

    flops_fwd = 4 * d * hq * A
    flops_bwd = 10 * d * hq * A
    res = time_steps(step, args, dev, flops_fwd, flops_bwd)
    B.bs_read_device_status(ws_b)
    res["config"] = {"workload": WORKLOADS[args.workload], "tokens": T, "heads_q": hq, "heads_kv": hkv,
                     "head_dim": d, "segments": nseq, "seed": args.seed, "visible_pairs": A,
                     "longest_segment": maxlen}
    res["flops_per_step"] = flops_fwd + flops_bwd
    # causal counted as half of each segment's s^2: A - T/2 pairs
    res["value_half_s2"] = res["value"] * (A - T / 2) / A
    if args.cpu_baseline:
        res["cpu_baseline"] = cpu_baseline_varlen(W, scale)
    return res


def time_steps(step, args, dev, flops_fwd, flops_bwd):
    import torch
    from paper_2502_21231_amd import bs_attn as B
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)
    s = torch.cuda.current_stream(dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    B.bs_set_profiling(True)
    torch.cuda.synchronize(dev)
    ev[0].record(s)
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
        ev[i + 1].record(s)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - t0
    total_ms = ev[0].elapsed_time(ev[-1])
    per_step = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps))
    median_ms = per_step[len(per_step) // 2] if len(per_step) % 2 else \
        0.5 * (per_step[len(per_step) // 2 - 1] + per_step[len(per_step) // 2])
    kern = {}
    names = {B.BS_KERNEL_PLAN: "plan", B.BS_KERNEL_FWD: "fwd", B.BS_KERNEL_PREPROCESS: "bwd_preprocess",
             B.BS_KERNEL_BWD_DQ: "bwd_dq", B.BS_KERNEL_BWD_DKDV: "bwd_dkdv",
             B.BS_KERNEL_FINALIZE: "dq_finalize", B.BS_KERNEL_MERGE: "lse_merge"}
    for kind, nm in names.items():
        ms, n = B.bs_profile_read(kind)
        if n:
            kern[nm] = {"ms_per_step": ms / args.steps, "launches_per_step": n / args.steps,
                        "avg_ms_per_launch": ms / n}
    B.bs_set_profiling(False)
    ms_step = total_ms / args.steps
    flops = flops_fwd + flops_bwd
    value = flops / (ms_step * 1e-3) / 1e12
    fwd_ms = kern.get("fwd", {}).get("ms_per_step", float("nan"))
    bwd_ms = sum(kern.get(k, {}).get("ms_per_step", 0.0) for k in ("bwd_dq", "bwd_dkdv")) or float("nan")
    # MFMA work each attention kernel must do, per visible pair and query head:
    # forward S and PV (4d); dQ kernel S, dP, dQ (6d); dK/dV kernel S, dP, dV, dK (8d)
    per_pair = {"fwd": 4, "bwd_dq": 6, "bwd_dkdv": 8}
    dom = max((k for k in per_pair if k in kern), key=lambda k: kern[k]["ms_per_step"])
    dom_flops = flops_fwd / 4 * per_pair[dom]
    dom_launches = kern[dom]["launches_per_step"]
    achieved = dom_flops / dom_launches / (kern[dom]["avg_ms_per_launch"] * 1e-3) / 1e12
    return {
        "value": value, "ms_per_step": ms_step, "ms_per_step_median": median_ms, "wall_s": wall,
        "pct_of_bf16_peak": 100.0 * value / BF16_PEAK_TFLOPS,
        "fwd_tflops": flops_fwd / (fwd_ms * 1e-3) / 1e12 if fwd_ms == fwd_ms else None,
        "bwd_tflops": flops_bwd / (bwd_ms * 1e-3) / 1e12 if bwd_ms == bwd_ms else None,
        "kernels": kern,
        "roofline": {"kernel": f"bs_attn {dom} (bf16 MFMA)", "bound": "mfma", "achieved": achieved,
                     "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": achieved / BF16_PEAK_TFLOPS,
                     # HBM bytes (read + write) per launch, from the FETCH_SIZE / WRITE_SIZE
                     # record in profiles/ (null when the kernel changed since)
                     "traffic": recorded_traffic(args.workload, dom)},
    }


# The CPU oracle runs on a bounded sample of each workload (about 10-30 s of float64 work on
# the benchmark host's 16 cores), so that a default benchmark run stays within minutes; the
# full-problem time is extrapolated from it and labelled as such.  The oracle computes every
# (row, key) score of a segment or chunk and masks it, so its time is proportional to
# rows x keys x query heads (not to the visible pairs): that is the extrapolation factor.
CPU_BASELINE_HEADS = 6  # packed7b: query heads 0..5 of 32 over every segment (about 14 s)
CPU_BASELINE_CHUNK_ROWS = {"cp7b": 2048, "zigzag141b": 1024}  # Q rows per part, KV group 0
CPU_BASELINE_GQA_AREA = 8e8  # gqa70b: rows x keys x query heads of KV group 0's sample


def blas_cores():
    try:
        import threadpoolctl
        return int(max(i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()
                       if i.get("user_api") == "blas"))
    except Exception:
        return len(os.sched_getaffinity(0))


def cpu_baseline_varlen(W, scale):
    """The float64 oracle (fwd + bwd) on a sample of the same workload: the first query heads
    over every segment when a KV group is a single head (MHA); otherwise KV group 0 (all its
    query heads) over every segment but the longest."""
    import numpy as np
    from oracle import attention as A
    hq, hkv, d = W["hq"], W["hkv"], W["d"]
    g = hq // hkv
    lens = W["lens"]
    if g == 1:
        H, segs = min(CPU_BASELINE_HEADS, hq), list(range(len(lens)))
    else:  # the segments in order, skipping the longest, within the sample's budget of work
        longest = int(np.argmax(lens))
        H, segs, area = g, [], 0
        for b in range(len(lens)):
            if b != longest and area + g * lens[b] ** 2 <= CPU_BASELINE_GQA_AREA:
                segs.append(b)
                area += g * lens[b] ** 2
    Hk = (H - 1) // g + 1  # the KV heads those query heads read
    cu_all = W["cu_cpu"].numpy()
    rows = np.concatenate([np.arange(cu_all[b], cu_all[b + 1]) for b in segs])
    sl = np.array([lens[b] for b in segs], dtype=np.int64)
    cu = np.concatenate([[0], np.cumsum(sl)]).astype(np.int32)
    q = W["q_cpu"][rows, :H]
    k = W["k_cpu"][rows, :Hk]
    v = W["v_cpu"][rows, :Hk]
    do = W["do_cpu"][rows, :H]
    t0 = time.perf_counter()
    o, l = A.varlen_fwd(q, k, v, cu, cu, True, scale)
    A.varlen_bwd(q, k, v, o, l, do, cu, cu, True, scale)
    dt = time.perf_counter() - t0
    a_s = int(sum(x * (x + 1) // 2 for x in sl))
    flops = 14 * d * H * a_s
    area_s = float(sum(x * x for x in sl)) * H
    area_full = float(sum(x * x for x in lens)) * hq
    what = (f"query heads 0..{H - 1} of {hq} (KV heads 0..{Hk - 1}) over "
            + (f"all {len(lens)} segments" if len(segs) == len(lens)
               else f"{len(segs)} of {len(lens)} segments (in order, the longest left out)"))
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": blas_cores(), "kind": "oracle",
            "sample": f"{what}, fwd+bwd in float64 NumPy: {flops:.3e} FLOP in {dt:.1f} s",
            "seconds": dt, "extrapolated_full_seconds": dt * area_full / area_s,
            "extrapolation": "extrapolated: sample time x (rows x keys x query heads of the full "
                             "problem) / (the same of the sample)"}


def cpu_baseline_chunk(name, Qs, dOs, Ks, Vs, q_offs, kv_offs, pairs, hq, hkv, c, scale):
    """The float64 oracle on KV group 0 (its query heads) and the first rows of every Q part of a
    context-parallel share: per-step chunk forward, LSE merge, per-step chunk backward.  Qs, dOs:
    the sampled rows [R, G, d] of each Q part; Ks, Vs: KV head 0 [c, 1, d] of each KV part."""
    import numpy as np
    from oracle import attention as A
    d = Qs[0].shape[2]
    g = hq // hkv
    R = Qs[0].shape[0]
    per_q = {i: [j for (a, j) in pairs if a == i] for i in range(len(q_offs))}
    t0 = time.perf_counter()
    for i, js in per_q.items():
        outs = [A.chunk_fwd(Qs[i], Ks[j], Vs[j], q_offs[i], kv_offs[j], True, scale) for j in js]
        o, l = A.lse_merge(np.stack([x[0] for x in outs]), np.stack([x[1] for x in outs]))
        for j in js:
            A.chunk_bwd(Qs[i], Ks[j], Vs[j], o, l, dOs[i], q_offs[i], kv_offs[j], True, scale)
    dt = time.perf_counter() - t0
    a_s = sum(visible_pairs_chunk_closed(R, c, q_offs[i] - kv_offs[j]) for i, j in pairs)
    flops = 14 * d * g * a_s
    scale_up = (c / R) * (hq / g)  # every row of a part costs the same: rows x keys x heads
    return {"value": flops / dt / 1e12 if dt > 0 else None, "unit": "TFLOP/s", "cores": blas_cores(),
            "kind": "oracle",
            "sample": f"KV group 0 (query heads 0..{g - 1} of {hq}), the first {R} of {c} rows of "
                      f"each of {len(q_offs)} Q part(s) against all {len(kv_offs)} KV part(s) "
                      f"({len(pairs)} steps), fwd + merge + bwd in float64 NumPy: {flops:.3e} FLOP "
                      f"({a_s} visible pairs per head) in {dt:.1f} s",
            "seconds": dt, "extrapolated_full_seconds": dt * scale_up,
            "extrapolation": f"extrapolated: sample time x {c}/{R} rows x {hq}/{g} query heads"}


def chunk_workload(name):
    """(hq, hkv, chunk tokens, Q part offsets, KV part offsets, (q, kv) pairs) of a CP share."""
    c = 32768
    if name == "cp7b":
        # one 32K Q chunk at 1015808 (the last of a 2048K sequence's 31st..32nd positions) against
        # 8 KV chunks, the 7 before it and its own (diagonal)
        q_offs = [1015808]
        kv_offs = [(24 + i) * c for i in range(8)]
        return 32, 32, c, q_offs, kv_offs, [(0, j) for j in range(8)]
    # device 0 of a 4-way symmetric split of a 256K sequence into 8 parts: parts 0 and 7
    q_offs = [0, 7 * c]
    kv_offs = [0, 7 * c]
    return 48, 8, c, q_offs, kv_offs, [(i, j) for i in range(2) for j in range(2)]


def run_chunk_bench(args, dev):
    import torch
    from paper_2502_21231_amd import bs_attn as B
    from paper_2502_21231_amd import inputs
    hq, hkv, c, q_offs, kv_offs, pairs = chunk_workload(args.workload)
    d, seed = 128, args.seed
    scale = 1.0 / math.sqrt(d)
    g = hq // hkv
    R = CPU_BASELINE_CHUNK_ROWS[args.workload]
    sample = {"Q": [], "dO": [], "K": [], "V": []}  # the CPU oracle's rows: KV group 0

    def load(tid, shape, key, rows, heads):
        t = inputs.normal(seed, tid, shape)
        if args.cpu_baseline:
            sample[key].append(t[:rows, :heads].clone())
        return t.to(dev)

    Q = [load(inputs.TID_Q + 100 * i, (c, hq, d), "Q", R, g) for i in range(len(q_offs))]
    dO = [load(inputs.TID_DO + 100 * i, (c, hq, d), "dO", R, g) for i in range(len(q_offs))]
    K = [load(inputs.tid_chunk_k(j), (c, hkv, d), "K", c, 1) for j in range(len(kv_offs))]
    V = [load(inputs.tid_chunk_v(j), (c, hkv, d), "V", c, 1) for j in range(len(kv_offs))]
    dims = B.make_dims(Q[0], K[0])
    ws_f = B.alloc_workspace(B.BS_OP_CHUNK_FWD, dims, dev)
    ws_b = B.alloc_workspace(B.BS_OP_CHUNK_BWD, dims, dev)
    per_q = {i: [j for (a, j) in pairs if a == i] for i in range(len(q_offs))}
    per_kv = {j: [i for (i, b) in pairs if b == j] for j in range(len(kv_offs))}
    parts_o = {i: torch.empty(len(per_q[i]), c, hq, d, dtype=torch.bfloat16, device=dev) for i in per_q}
    parts_l = {i: torch.empty(len(per_q[i]), hq, c, dtype=torch.float32, device=dev) for i in per_q}
    O = [torch.empty(c, hq, d, dtype=torch.bfloat16, device=dev) for _ in q_offs]
    L = [torch.empty(hq, c, dtype=torch.float32, device=dev) for _ in q_offs]
    dq_acc = [torch.empty(c, hq, d, dtype=torch.float32, device=dev) for _ in q_offs]
    dQ = [torch.empty(c, hq, d, dtype=torch.bfloat16, device=dev) for _ in q_offs]
    multi = any(len(v) > 1 for v in per_kv.values())   # a KV part seen by several Q parts
    kv_dtype = torch.float32 if multi else torch.bfloat16
    dK = [torch.empty(c, hkv, d, dtype=kv_dtype, device=dev) for _ in kv_offs]
    dV = [torch.empty(c, hkv, d, dtype=kv_dtype, device=dev) for _ in kv_offs]
    dKb = [torch.empty(c, hkv, d, dtype=torch.bfloat16, device=dev) for _ in kv_offs] if multi else dK
    dVb = [torch.empty(c, hkv, d, dtype=torch.bfloat16, device=dev) for _ in kv_offs] if multi else dV

    def step():
        for i in per_q:
            for s, j in enumerate(per_q[i]):
                B.bs_attn_chunk_fwd(Q[i], K[j], V[j], q_offs[i], kv_offs[j], True, scale,
                                    parts_o[i][s], parts_l[i][s], ws_f)
            B.bs_lse_merge(parts_o[i], parts_l[i], O[i], L[i])
        for t in dq_acc:
            t.zero_()
        if multi:
            for t in dK + dV:
                t.zero_()
        for i, j in pairs:
            B.bs_attn_chunk_bwd(Q[i], K[j], V[j], O[i], L[i], dO[i], q_offs[i], kv_offs[j], True,
                                scale, dq_acc[i], dK[j], dV[j], multi, ws_b)
        for i in range(len(q_offs)):
            B.bs_dq_finalize(dq_acc[i], dQ[i])
        if multi:
            for j in range(len(kv_offs)):
                B.bs_dq_finalize(dK[j], dKb[j])
                B.bs_dq_finalize(dV[j], dVb[j])

    A = sum(visible_pairs_chunk_closed(c, c, q_offs[i] - kv_offs[j]) for i, j in pairs)
    flops_fwd = 4 * d * hq * A
    flops_bwd = 10 * d * hq * A
    res = time_steps(step, args, dev, flops_fwd, flops_bwd)
    res["config"] = {"workload": WORKLOADS[args.workload], "chunk_tokens": c, "heads_q": hq,
                     "heads_kv": hkv, "head_dim": d, "q_offsets": q_offs, "kv_offsets": kv_offs,
                     "pairs": pairs, "seed": seed, "visible_pairs": A}
    res["flops_per_step"] = flops_fwd + flops_bwd
    # causal counted as half of c^2 for each diagonal chunk pair (c(c+1)/2 exact)
    n_diag = sum(1 for i, j in pairs if q_offs[i] == kv_offs[j])
    res["value_half_s2"] = res["value"] * (A - n_diag * c / 2) / A
    merge = res["kernels"].get("lse_merge")
    if merge:
        # algorithmic bytes of one merge of n partials: read n O and LSE rows, write one of each
        n = len(per_q[0])
        nbytes = n * c * hq * d * 2 + n * hq * c * 4 + c * hq * d * 2 + hq * c * 4
        res["lse_merge_gbs"] = nbytes / (merge["avg_ms_per_launch"] * 1e-3) / 1e9
        res["lse_merge_bytes"] = nbytes
    if args.cpu_baseline:
        res["cpu_baseline"] = cpu_baseline_chunk(args.workload, sample["Q"], sample["dO"], sample["K"],
                                                 sample["V"], q_offs, kv_offs, pairs, hq, hkv, c, scale)
    return res


def run_cp_ring_bench(args, dev):
    """cp7b through the single-GPU ring rehearsal (paper_2502_21231_amd.ring.ChunkRing): same
    shards, seeds and FLOPs as cp7b; the timed step also carries every shard transfer."""
    import torch
    from paper_2502_21231_amd import inputs
    from paper_2502_21231_amd.ring import ChunkRing
    hq, hkv, c, q_offs, kv_offs, pairs = chunk_workload("cp7b")
    d, seed = 128, args.seed
    scale = 1.0 / math.sqrt(d)
    q = inputs.normal(seed, inputs.TID_Q, (c, hq, d)).to(dev)
    do = inputs.normal(seed, inputs.TID_DO, (c, hq, d)).to(dev)
    order = sorted(range(len(kv_offs)), key=lambda j: -kv_offs[j])  # own shard, then those behind
    K = [inputs.normal(seed, inputs.tid_chunk_k(j), (c, hkv, d)).to(dev) for j in order]
    V = [inputs.normal(seed, inputs.tid_chunk_v(j), (c, hkv, d)).to(dev) for j in order]
    ring = ChunkRing(q, do, K, V, q_offs[0], [kv_offs[j] for j in order], True, scale,
                     time_copies=True)

    def step():
        ring.forward()
        ring.backward()

    A = sum(visible_pairs_chunk_closed(c, c, q_offs[0] - kv_offs[j]) for j in order)
    flops_fwd = 4 * d * hq * A
    flops_bwd = 10 * d * hq * A
    res = time_steps(step, args, dev, flops_fwd, flops_bwd)
    copy_ms, copy_bytes = ring.copy_stats()  # every copy of the warmup and timed steps
    n_steps = args.warmup + args.steps
    res["config"] = {"workload": WORKLOADS[args.workload], "chunk_tokens": c, "heads_q": hq,
                     "heads_kv": hkv, "head_dim": d, "q_offsets": q_offs,
                     "kv_offsets_in_ring_order": [kv_offs[j] for j in order], "seed": seed,
                     "visible_pairs": A}
    res["flops_per_step"] = flops_fwd + flops_bwd
    res["value_half_s2"] = res["value"] * (A - c / 2) / A
    # transfers per step: 7 shards received in each pass, 8 shards' dK, dV sent
    res["ring_copies"] = {"ms_per_step": copy_ms / n_steps, "bytes_per_step": copy_bytes / n_steps,
                          "gbs": copy_bytes / (copy_ms * 1e-3) / 1e9 if copy_ms > 0 else None}
    return res


def run_zigzag_packed_bench(args, dev):
    """The packed context-parallel share of one device over a whole ring: each ring step is two
    packed calls (straight and crossed part pairs).  The key buffers of both layouts are staged
    before timing (laying them out is the ring transport's job); every call writes its own dK, dV."""
    import numpy as np
    import torch
    from paper_2502_21231_amd import bs_attn as B
    from paper_2502_21231_amd import inputs
    cfg = ZIGZAG_PACKED
    lens, n_dev, me, hq, hkv, d = (cfg[k] for k in ("lens", "n_dev", "dev", "hq", "hkv", "d"))
    seed = args.seed
    scale = 1.0 / math.sqrt(d)
    T = sum(lens)
    rows = torch.from_numpy(inputs.zigzag_rows(lens, n_dev, me))
    q = inputs.normal(seed, inputs.TID_Q, (T, hq, d))[rows].to(dev)
    do = inputs.normal(seed, inputs.TID_DO, (T, hq, d))[rows].to(dev)
    k_all = inputs.normal(seed, inputs.TID_K, (T, hkv, d))
    v_all = inputs.normal(seed, inputs.TID_V, (T, hkv, d))
    calls, A = [], 0
    for kv_dev in range(n_dev):
        kv_rows = inputs.zigzag_rows(lens, n_dev, kv_dev)
        for crossed in (False, True):
            cu_q, cu_k, qp, kp, kr = inputs.zigzag_step(lens, n_dev, me, kv_dev, crossed)
            g = torch.from_numpy(kv_rows[kr])
            calls.append(dict(k=k_all[g].to(dev), v=v_all[g].to(dev),
                              cu_q=torch.from_numpy(cu_q).to(dev), cu_k=torch.from_numpy(cu_k).to(dev),
                              qp=torch.from_numpy(qp).to(dev), kp=torch.from_numpy(kp).to(dev)))
            for b in range(len(qp)):
                A += visible_pairs_chunk_closed(int(cu_q[b + 1] - cu_q[b]), int(cu_k[b + 1] - cu_k[b]),
                                                int(qp[b] - kp[b]))
    del k_all, v_all
    maxlen = max(lens)
    n = len(calls)
    Tq = q.shape[0]
    dims = B.make_dims(q, calls[0]["k"])
    ws_f = B.alloc_workspace(B.BS_OP_PACKED_CHUNK_FWD, dims, dev, len(lens) * 2, maxlen)
    ws_b = B.alloc_workspace(B.BS_OP_PACKED_CHUNK_BWD, dims, dev, len(lens) * 2, maxlen)
    parts_o = torch.empty(n, Tq, hq, d, dtype=torch.bfloat16, device=dev)
    parts_l = torch.empty(n, hq, Tq, dtype=torch.float32, device=dev)
    O = torch.empty(Tq, hq, d, dtype=torch.bfloat16, device=dev)
    L = torch.empty(hq, Tq, dtype=torch.float32, device=dev)
    dq_acc = torch.empty(Tq, hq, d, dtype=torch.float32, device=dev)
    dQ = torch.empty_like(q)
    dK = [torch.empty_like(c["k"]) for c in calls]
    dV = [torch.empty_like(c["v"]) for c in calls]

    def step():
        for i, c in enumerate(calls):
            B.bs_attn_packed_chunk_fwd(q, c["k"], c["v"], c["cu_q"], c["cu_k"], c["qp"], c["kp"], maxlen,
                                       True, scale, parts_o[i], parts_l[i], ws_f)
        B.bs_lse_merge(parts_o, parts_l, O, L)
        dq_acc.zero_()
        for i, c in enumerate(calls):
            B.bs_attn_packed_chunk_bwd(q, c["k"], c["v"], O, L, do, c["cu_q"], c["cu_k"], c["qp"], c["kp"],
                                       maxlen, True, scale, dq_acc, dK[i], dV[i], False, ws_b)
        B.bs_dq_finalize(dq_acc, dQ)

    flops_fwd = 4 * d * hq * A
    flops_bwd = 10 * d * hq * A
    res = time_steps(step, args, dev, flops_fwd, flops_bwd)
    res["config"] = {"workload": WORKLOADS[args.workload], "subsequences": lens, "devices": n_dev,
                     "device": me, "query_tokens": Tq, "packed_calls_per_pass": n, "heads_q": hq,
                     "heads_kv": hkv, "head_dim": d, "seed": seed, "visible_pairs": A}
    res["flops_per_step"] = flops_fwd + flops_bwd
    res["value_half_s2"] = res["value"] * (A - Tq / 2) / A
    merge = res["kernels"].get("lse_merge")
    if merge:
        nbytes = n * Tq * hq * d * 2 + n * hq * Tq * 4 + Tq * hq * d * 2 + hq * Tq * 4
        res["lse_merge_gbs"] = nbytes / (merge["avg_ms_per_launch"] * 1e-3) / 1e9
        res["lse_merge_bytes"] = nbytes
    return res


XENT = dict(rows=262144, vocab=128256, cpu_rows=16384)
HDP = dict(total=524288, capacity=8192, ranks=16, max_len=131072, hq=32, hkv=32, d=128,
           fit_lengths=[1024, 2048, 4096, 8192, 16384, 32768, 65536], layers=32,
           act_bytes_per_token=34 * 4096, delta=1e-4, buckets=4)


def _varlen_call(q, k, v, do, cu, maxlen, ws_f, ws_b, out, lse, dq, dk, dv, scale):
    from paper_2502_21231_amd import bs_attn as B
    B.bs_attn_varlen_fwd(q, k, v, cu, cu, maxlen, True, scale, out, lse, ws_f)
    B.bs_attn_varlen_bwd(q, k, v, out, lse, do, cu, cu, maxlen, True, scale, dq, dk, dv, ws_b)


def _event_ms(fn, dev, reps=5, warmup=2):
    import torch
    for _ in range(warmup):
        fn()
    s = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(s)
    for _ in range(reps):
        fn()
    e1.record(s)
    torch.cuda.synchronize(dev)
    return e0.elapsed_time(e1) / reps


def _host_link_gbs(dev):
    """B_d2h and B_h2d (Sec. 4 profiles them): 1 GiB copies between pinned host memory and HBM."""
    import torch
    n = 1 << 30
    h = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    g = torch.empty(n, dtype=torch.uint8, device=dev)
    h2d = _event_ms(lambda: g.copy_(h, non_blocking=True), dev, reps=3, warmup=1)
    d2h = _event_ms(lambda: h.copy_(g, non_blocking=True), dev, reps=3, warmup=1)
    return n / (d2h * 1e-3), n / (h2d * 1e-3)


def _replay(mbs, unit_ms, d):
    """Finish time of every rank when the plan's units take unit_ms[k] (a unit's ranks start it
    together when the last of them is free)."""
    fin = [0.0] * d
    for k, (_, ranks, _, _, _) in enumerate(mbs):
        start = max(fin[g] for g in ranks)
        for g in ranks:
            fin[g] = start + unit_ms[k]
    return fin


def run_hdp_bench(args, dev):
    """Plans a long-tailed global batch with the native planners, using a cost model fitted from
    this library's own attention times, then runs every micro-batch on the GPU: the modelled
    per-rank finish times of the naive and balanced plans are set against the measured ones."""
    import numpy as np
    import torch
    from paper_2502_21231_amd import bs_attn as B
    from paper_2502_21231_amd import hdp as N
    from paper_2502_21231_amd import inputs
    cfg = HDP
    hq, hkv, d = cfg["hq"], cfg["hkv"], cfg["d"]
    C, R = cfg["capacity"], cfg["ranks"]
    scale = 1.0 / math.sqrt(d)
    lens = inputs.lognormal_packed_lengths(args.seed, cfg["total"], hi=cfg["max_len"])
    T = sum(lens)
    q = inputs.normal(args.seed, inputs.TID_Q, (T, hq, d)).to(dev)
    k = inputs.normal(args.seed, inputs.TID_K, (T, hkv, d)).to(dev)
    v = inputs.normal(args.seed, inputs.TID_V, (T, hkv, d)).to(dev)
    do = inputs.normal(args.seed, inputs.TID_DO, (T, hq, d)).to(dev)
    starts = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)

    # 1. T(s) of this library: attention fwd+bwd of one sequence, least squares over lengths
    fit_ms = []
    for L in cfg["fit_lengths"]:
        sl = slice(0, L)
        qs, ks, vs, dos = (t[sl].contiguous() for t in (q, k, v, do))
        cu = torch.tensor([0, L], dtype=torch.int32, device=dev)
        dims = B.make_dims(qs, ks)
        wf = B.alloc_workspace(B.BS_OP_VARLEN_FWD, dims, dev, 1, L)
        wb = B.alloc_workspace(B.BS_OP_VARLEN_BWD, dims, dev, 1, L)
        bufs = (torch.empty_like(qs), torch.empty(hq, L, device=dev), torch.empty_like(qs),
                torch.empty_like(ks), torch.empty_like(vs))
        fit_ms.append(_event_ms(lambda: _varlen_call(qs, ks, vs, dos, cu, L, wf, wb, *bufs, scale), dev))
    # non-negative least squares on relative errors (each length weighs alike)
    from scipy.optimize import nnls
    Ls = np.array(cfg["fit_lengths"], dtype=np.float64)
    y = np.array(fit_ms) * 1e-3
    A = np.stack([Ls * Ls, Ls, np.ones_like(Ls)], axis=1) / y[:, None]
    coef, _ = nnls(A, np.ones_like(y))
    a1, b1, g0 = (float(x) for x in coef)
    bw_d2h, bw_h2d = _host_link_gbs(dev)
    cost = N.make_cost(a1, b1, g0, float(cfg["act_bytes_per_token"]), 0.0, cfg["layers"], bw_d2h, bw_h2d)

    # 2. the plans (native planners; the oracle planners timed on the same batch for reference)
    plans, plan_ms = {}, {}
    for name, alg in (("naive", N.NAIVE), ("dp_balance", N.DP_BALANCE), ("pp_balance", N.PP_BALANCE)):
        t0 = time.perf_counter()
        plans[name] = N.plan(alg, lens, C, R, cost, cfg["delta"], cfg["buckets"])
        plan_ms[name] = (time.perf_counter() - t0) * 1e3

    # 3. every unit's measured time: a packed micro-batch runs as one varlen call; a
    # context-parallel sequence runs once, whole, and each of its D ranks is charged 1/D of it
    # (the zig-zag split gives every rank of the group the same mask area)
    unit_cache = {}

    def unit(seqs):
        key = tuple(sorted(seqs))
        if key in unit_cache:
            return unit_cache[key]
        rows = np.concatenate([np.arange(starts[i], starts[i + 1]) for i in key])
        ri = torch.from_numpy(rows).to(dev)
        qs, ks, vs, dos = (t.index_select(0, ri) for t in (q, k, v, do))
        seg = [lens[i] for i in key]
        cu = torch.from_numpy(inputs.cu_seqlens(seg)).to(dev)
        dims = B.make_dims(qs, ks)
        ml = max(seg)
        wf = B.alloc_workspace(B.BS_OP_VARLEN_FWD, dims, dev, len(seg), ml)
        wb = B.alloc_workspace(B.BS_OP_VARLEN_BWD, dims, dev, len(seg), ml)
        bufs = (torch.empty_like(qs), torch.empty(hq, qs.shape[0], device=dev), torch.empty_like(qs),
                torch.empty_like(ks), torch.empty_like(vs))
        fn = (lambda: _varlen_call(qs, ks, vs, dos, cu, ml, wf, wb, *bufs, scale))
        unit_cache[key] = (fn, seg)
        return unit_cache[key]

    hdp_report = {"cost_fit": {"alpha1_s_per_token2": a1, "beta1_s_per_token": b1, "gamma_s": g0,
                               "lengths": cfg["fit_lengths"], "measured_ms": fit_ms,
                               "model_ms": [float((a1 * L * L + b1 * L + g0) * 1e3) for L in cfg["fit_lengths"]]},
                  "bw_d2h_gbs": bw_d2h / 1e9, "bw_h2d_gbs": bw_h2d / 1e9,
                  "act_bytes_per_token_per_layer": cfg["act_bytes_per_token"], "layers": cfg["layers"],
                  "sequences": len(lens), "longest": max(lens),
                  "long_sequences": sum(1 for L in lens if L > C), "plans": {}}
    for name, (mbs, rank_time) in plans.items():
        unit_ms = []
        for seqs, ranks, r, start, t in mbs:
            fn, seg = unit(seqs)
            unit_ms.append(_event_ms(fn, dev, reps=3, warmup=1) / len(ranks))
        fin = _replay(mbs, unit_ms, R)
        bub = lambda f: 1.0 - sum(f) / (len(f) * max(f))
        hdp_report["plans"][name] = {
            "micro_batches": len(mbs), "plan_ms_native": plan_ms[name],
            "model_makespan_ms": max(rank_time) * 1e3, "model_bubble": bub(rank_time),
            "measured_makespan_ms": max(fin), "measured_bubble": bub(fin),
            "measured_rank_ms": fin, "model_rank_ms": [x * 1e3 for x in rank_time],
            "offloaded": [[list(s), r] for s, _, r, _, _ in mbs if r > 0]}
    from oracle import hdp as H
    oc = H.Cost(a1, b1, g0, float(cfg["act_bytes_per_token"]), 0.0, cfg["layers"], bw_d2h, bw_h2d)
    t0 = time.perf_counter()
    H.plan(H.ALG_DP_BALANCE, lens, C, R, oc, cfg["delta"], cfg["buckets"])
    hdp_report["plan_ms_oracle_dp_balance"] = (time.perf_counter() - t0) * 1e3
    # the native planners at cluster scale: 32M tokens (about 30K sequences) on 1024 ranks of 32K
    big = inputs.lognormal_packed_lengths(args.seed, 1 << 25, hi=1 << 20)
    scale_ms = {}
    for name, alg in (("naive", N.NAIVE), ("dp_balance", N.DP_BALANCE), ("pp_balance", N.PP_BALANCE)):
        t0 = time.perf_counter()
        N.plan(alg, big, 32768, 1024, cost, cfg["delta"], 16)
        scale_ms[name] = (time.perf_counter() - t0) * 1e3
    hdp_report["native_plan_ms_32m_tokens_1024_ranks"] = {"sequences": len(big), **scale_ms}

    # 4. the timed step: every micro-batch of the DP-Balance plan, a CP sequence once
    mbs = plans["dp_balance"][0]
    fns = [unit(seqs)[0] for seqs, *_ in mbs]

    def step():
        for fn in fns:
            fn()

    A_pairs = sum(L * (L + 1) // 2 for L in lens)
    res = time_steps(step, args, dev, 4 * d * hq * A_pairs, 10 * d * hq * A_pairs)
    res["config"] = {"workload": WORKLOADS[args.workload], "tokens": T, "heads_q": hq, "heads_kv": hkv,
                     "head_dim": d, "capacity": C, "ranks": R, "seed": args.seed,
                     "visible_pairs": A_pairs}
    res["flops_per_step"] = 14 * d * hq * A_pairs
    res["hdp"] = hdp_report
    return res


def run_xent_bench(args, dev):
    """The fused cross-entropy: whole-call HIP events on the library's stream, the kernel's own
    events from the profiling hooks; HBM bytes counted algorithmically (logits read once, gradient
    written once, labels, loss, lse)."""
    import torch
    from paper_2502_21231_amd import bs_attn as B
    from paper_2502_21231_amd import inputs
    T, V = XENT["rows"], XENT["vocab"]
    z, y = inputs.xent_inputs(args.seed, T, V, device=dev)
    n_valid = int((y != -100).sum())
    g = 1.0 / n_valid
    loss = torch.empty(T, dtype=torch.float32, device=dev)
    lse = torch.empty(T, dtype=torch.float32, device=dev)
    dz = torch.empty_like(z)

    def step():
        B.bs_softmax_xent(z, y, -100, g, loss, lse, dz)

    for _ in range(args.warmup):
        step()
    s = torch.cuda.current_stream(dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize(dev)
    B.bs_set_profiling(True)
    ev[0].record(s)
    for i in range(args.steps):
        step()
        ev[i + 1].record(s)
    torch.cuda.synchronize(dev)
    k_ms, k_n = B.bs_profile_read(B.BS_KERNEL_XENT)
    B.bs_set_profiling(False)
    total_ms = ev[0].elapsed_time(ev[-1])
    per = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps))
    ms = total_ms / args.steps
    nbytes = 2 * T * V * z.element_size() + T * 8 + 2 * T * 4
    kern_ms = k_ms / k_n
    res = {
        "metric": "fused softmax cross-entropy fwd+bwd, algorithmic HBM GB/s, 1 GPU",
        "value": nbytes / (ms * 1e-3) / 1e9, "unit": "GB/s", "ms_per_step": ms,
        "ms_per_step_median": per[len(per) // 2], "dtype": "bf16",
        "config": {"workload": WORKLOADS[args.workload], "rows": T, "vocab": V, "valid_rows": n_valid,
                   "seed": args.seed, "bytes_per_step": nbytes},
        "kernels": {"xent": {"ms_per_step": k_ms / args.steps, "launches_per_step": k_n / args.steps,
                             "avg_ms_per_launch": kern_ms}},
        "roofline": {"kernel": "bs_softmax_xent (bf16, fused gradient)", "bound": "hbm",
                     "achieved": nbytes / (kern_ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": nbytes / (kern_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                     "traffic": recorded_traffic(args.workload, "xent")},
    }
    if args.cpu_baseline:
        res["cpu_baseline"] = cpu_baseline_xent(z, y, g)
    return res


def cpu_baseline_xent(z, y, g):
    """The float64 oracle on the first rows of the same logits (a bounded sample), as GB/s of the
    same algorithmic bytes per row."""
    from oracle.xent import softmax_xent
    R, blk = XENT["cpu_rows"], 2048  # blocks of rows bound the oracle's float64 temporaries
    dt = 0.0
    for r0 in range(0, R, blk):
        zc, yc = z[r0:r0 + blk].cpu(), y[r0:r0 + blk].cpu().numpy()
        t0 = time.perf_counter()
        softmax_xent(zc, yc, -100, g)
        dt += time.perf_counter() - t0
    V = z.shape[1]
    nbytes = 2 * R * V * z.element_size() + R * 8 + 2 * R * 4
    return {"value": nbytes / dt / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"rows 0..{R - 1} of {z.shape[0]} (all {V} vocabulary entries), float64 NumPy "
                      f"(element-wise, one thread), in blocks of {blk} rows: {dt:.1f} s", "seconds": dt}


def visible_pairs_chunk_closed(lq, lk, diag):
    """Exact visible (query, key) pairs of a chunk pair: key j visible to query i iff j - i <= diag."""
    tot = 0
    # rows i with i + diag + 1 in (0, lk): a triangle; rows beyond see every key
    lo = max(0, -diag)                  # first row that sees key 0
    hi = min(lq, lk - diag - 1)         # rows below hi see fewer than lk keys
    if hi > lo:
        n = hi - lo
        first = lo + diag + 1
        tot += n * first + n * (n - 1) // 2
    full_from = max(lo, hi, 0)
    if lq > full_from:
        tot += (lq - full_from) * lk
    return tot


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="packed7b")
    ap.add_argument("--no-cpu-baseline", dest="cpu_baseline", action="store_false")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run 3 plain 1 GiB device-to-device copies (the reference kernel "
                         "that scales the HBM byte counters of a profiler run) and exit")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": 1 << 30, "copy_calibration_bytes_written": 1 << 30,
                          "launches": 3}))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU's share of the work; --gpus {args.gpus} is not supported "
              f"(this build has no multi-GPU path: use --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    if args.workload in ("packed7b", "gqa70b"):
        res = run_varlen_bench(args, dev)
    elif args.workload == "zigzag_packed7b":
        res = run_zigzag_packed_bench(args, dev)
    elif args.workload == "cp7b_ring":
        res = run_cp_ring_bench(args, dev)
    elif args.workload == "hdp_batch7b":
        res = run_hdp_bench(args, dev)
    elif args.workload == "xent_llama3_256k":
        res = run_xent_bench(args, dev)
        line = {"metric": res["metric"], "value": round(res["value"], 3), "unit": res["unit"], "n_gpus": 1,
                "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(res["ms_per_step"], 4),
                "ms_per_step_median": round(res["ms_per_step_median"], 4), "higher_is_better": True,
                "scaling": "weak", "vs_baseline": None, "dtype": res["dtype"], "data": "synthetic",
                "config": res["config"], "kernels": res["kernels"], "roofline": res["roofline"],
                "cpu_baseline": res.get("cpu_baseline")}
        print(json.dumps(line), flush=True)
        return
    else:
        res = run_chunk_bench(args, dev)
    line = {
        "metric": "attention fwd+bwd TFLOP/s (causal-adjusted) and % of bf16 MFMA peak, 1 GPU",
        "value": round(res["value"], 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(res["ms_per_step"], 4),
        "ms_per_step_median": round(res["ms_per_step_median"], 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": res["config"],
        "pct_of_bf16_peak": round(res["pct_of_bf16_peak"], 2),
        # the same FLOPs counted the common way for causal attention (half of the dense S^2 per
        # segment): 0.5 * 14 d Hq sum(s^2) instead of 14 d Hq A with A = sum s(s+1)/2
        "value_half_s2_convention": res.get("value_half_s2"),
        "fwd_tflops": res["fwd_tflops"], "bwd_tflops": res["bwd_tflops"],
        "kernels": res["kernels"], "flops_per_step": res["flops_per_step"],
        "roofline": res["roofline"],
        "lse_merge_gbs": res.get("lse_merge_gbs"),
        "lse_merge_bytes": res.get("lse_merge_bytes"),
        "ring_copies": res.get("ring_copies"),
        "hdp": res.get("hdp"),
        "cpu_baseline": res.get("cpu_baseline"),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
