"""One device's share of a context-parallel ring, rehearsed on one GPU (Sec. 2.4, Long Context
Training: KV shards travel around a ring of devices and each step's attention overlaps the
transfer of the next shard).

The device holds a query shard and is handed, in turn, every KV shard of the ring: its own
first, then those of the devices behind it.  Here the other devices' shards sit in this GPU's
memory and a transfer is a device-to-device copy, on a second HIP stream, into one of two
receive buffers, so that step s computes while shard s+1 arrives.  A copy runs as a copy kernel
(transport="blit", the default) or on the DMA engines (transport="dma", bs_copy_async); on
MI355X the DMA form slowed the overlapped attention kernels more than the copy kernel did.
Each forward step folds its result into a running float32 (O, LSE) in the attention kernel's epilogue
(bs_attn_chunk_fwd_merge), and the last step writes O in the input dtype: no per-step partials
and no merge pass.  The backward walks the ring again; shards arrive the same way, and each
shard's dK, dV leave on the copy stream for the shard's owner (here a buffer per shard).  A pass
ends on the compute stream only once everything it sent has left.

Orchestration only: every step of the arithmetic runs in the library's kernels.
"""
from __future__ import annotations

import torch

from . import bs_attn as B


class ChunkRing:
    """k_shards[s], v_shards[s]: the KV shard the ring delivers at step s (s = 0: the device's
    own), at global position k_pos[s]; q, dout: the device's query shard at q_pos.  All shards
    have one shape.  Buffers, workspaces, the copy stream and its events are made once."""

    def __init__(self, q, dout, k_shards, v_shards, q_pos: int, k_pos, causal: bool = True,
                 scale: float | None = None, time_copies: bool = False, transport: str = "blit"):
        n = len(k_shards)
        if n < 1 or len(v_shards) != n or len(k_pos) != n:
            raise ValueError("need as many K shards, V shards and positions, at least one")
        if any(t.shape != k_shards[0].shape for t in list(k_shards) + list(v_shards)):
            raise ValueError("ring shards must all have one shape")
        dev = q.device
        self.n, self.q, self.do = n, q, dout
        self.ks, self.vs = list(k_shards), list(v_shards)
        self.q_pos, self.k_pos = int(q_pos), [int(p) for p in k_pos]
        self.causal, self.scale = causal, scale
        dims = B.make_dims(q, k_shards[0])
        self.ws_f = B.alloc_workspace(B.BS_OP_CHUNK_FWD, dims, dev)
        self.ws_b = B.alloc_workspace(B.BS_OP_CHUNK_BWD, dims, dev)
        self.recv_k = [torch.empty_like(k_shards[0]) for _ in range(2)]
        self.recv_v = [torch.empty_like(v_shards[0]) for _ in range(2)]
        self.send_k = [torch.empty_like(k_shards[0]) for _ in range(2)]
        self.send_v = [torch.empty_like(v_shards[0]) for _ in range(2)]
        self.o_run = torch.empty(q.shape, dtype=torch.float32, device=dev)
        self.lse = torch.empty(q.shape[1], q.shape[0], dtype=torch.float32, device=dev)
        self.out = torch.empty_like(q)
        self.dq_acc = torch.empty(q.shape, dtype=torch.float32, device=dev)
        self.dq = torch.empty_like(q)
        self.dk = [torch.empty_like(k) for k in k_shards]
        self.dv = [torch.empty_like(v) for v in v_shards]
        self.copy = torch.cuda.Stream(dev)  # default priority, like the compute stream
        ev = lambda: [torch.cuda.Event() for _ in range(n)]
        self.ev_start = torch.cuda.Event()
        self.ev_recv, self.ev_done, self.ev_sent = ev(), ev(), ev()
        if transport not in ("dma", "blit"):
            raise ValueError("transport is 'dma' (bs_copy_async, DMA engines) or 'blit' (a copy kernel)")
        self.dma = transport == "dma"
        self.time_copies = time_copies
        self.copy_log: list[tuple[torch.cuda.Event, torch.cuda.Event, int]] = []

    def _on_copy(self, after, pairs, done):
        """On the copy stream, once event `after` (if any) has completed: dst.copy_(src) for each
        pair, then record `done`."""
        with torch.cuda.stream(self.copy):
            if after is not None:
                self.copy.wait_event(after)
            if self.time_copies:
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(self.copy)
            for dst, src in pairs:
                if self.dma:
                    B.bs_copy_async(dst, src)
                else:
                    dst.copy_(src, non_blocking=True)
            if self.time_copies:
                e1.record(self.copy)
                self.copy_log.append((e0, e1, sum(2 * s.numel() * s.element_size() for _, s in pairs)))
            done.record(self.copy)

    def _receive(self, s, after):
        """Shard s into receive buffer s % 2, after the compute step that last read it."""
        b = s % 2
        self._on_copy(after, [(self.recv_k[b], self.ks[s]), (self.recv_v[b], self.vs[s])],
                      self.ev_recv[s])

    def _start(self, comp):
        # the receive and send buffers are free once the compute stream reaches this point
        self.ev_start.record(comp)
        self.copy.wait_event(self.ev_start)

    def _shard(self, comp, s):
        if s == 0:
            return self.ks[0], self.vs[0]
        comp.wait_event(self.ev_recv[s])
        return self.recv_k[s % 2], self.recv_v[s % 2]

    def forward(self):
        """Returns (O in q's dtype, LSE float32 [hq, T]) over every shard of the ring."""
        comp = torch.cuda.current_stream(self.q.device)
        self._start(comp)
        n = self.n
        if n > 1:
            self._receive(1, None)
        for s in range(n):
            if 1 <= s < n - 1:
                self._receive(s + 1, self.ev_done[s - 1])
            k, v = self._shard(comp, s)
            B.bs_attn_chunk_fwd_merge(self.q, k, v, self.q_pos, self.k_pos[s], self.o_run, self.lse,
                                      accumulate=s > 0, causal=self.causal, scale=self.scale,
                                      out=self.out if s == n - 1 else None, workspace=self.ws_f)
            self.ev_done[s].record(comp)
        return self.out, self.lse

    def backward(self):
        """Needs forward() first.  Returns (dQ, [dK per shard], [dV per shard]) in q's dtype."""
        comp = torch.cuda.current_stream(self.q.device)
        self._start(comp)
        n = self.n
        self.dq_acc.zero_()
        if n > 1:
            self._receive(1, None)
        for s in range(n):
            if 1 <= s < n - 1:
                self._receive(s + 1, self.ev_done[s - 1])
            k, v = self._shard(comp, s)
            b = s % 2
            if s >= 2:
                comp.wait_event(self.ev_sent[s - 2])  # send buffer b has left
            B.bs_attn_chunk_bwd(self.q, k, v, self.out, self.lse, self.do, self.q_pos, self.k_pos[s],
                                causal=self.causal, scale=self.scale, dq_accum=self.dq_acc,
                                dk=self.send_k[b], dv=self.send_v[b], kv_accumulate=False,
                                workspace=self.ws_b)
            self.ev_done[s].record(comp)
            self._on_copy(self.ev_done[s], [(self.dk[s], self.send_k[b]), (self.dv[s], self.send_v[b])],
                          self.ev_sent[s])
        B.bs_dq_finalize(self.dq_acc, self.dq)
        comp.wait_event(self.ev_sent[n - 1])
        return self.dq, self.dk, self.dv

    def copy_stats(self):
        """(milliseconds, bytes read + written) summed over the copies logged since the last
        call; synchronises the copy stream."""
        self.copy.synchronize()
        ms = sum(e0.elapsed_time(e1) for e0, e1, _ in self.copy_log)
        nbytes = sum(b for _, _, b in self.copy_log)
        self.copy_log = []
        return ms, nbytes
