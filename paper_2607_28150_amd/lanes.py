"""Parallel on-demand transfer (Section 4.2) and speculative transfer (Section
4.3) on one GPU: stream plumbing only.

After Algorithm 1 splits a step's KV index (sg_split, remote entries first), two
lanes fill the decode pool at once:
  - the local lane (sg_fetch) gathers the local entries from the decode side's
    KV store into pool rows [n_remote, n_remote + n_local) of each index row;
  - the remote lane (sg_fetch_keep, or sg_fetch without reuse) fetches the
    remote entries from the prefill side's copy into pool rows [0, n_remote),
    and with reuse keeps them in the store and marks them local.
Each lane runs on its own stream; the caller's stream waits for both, so the
attention that follows on it sees the whole pool.

SpecPusher sends the blocks that the proactive transfer left behind, a quota at
a time in importance order, on a side stream, without holding up any decode
step: a push moves rows only (sg_spec_push without a mask), and once its
completion event has fired, the next step boundary enqueues the marking
(sg_spec_commit) on the caller's stream, ordered after the rows.  Every copy
runs in the library's kernels; this module only orders them.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import smartgen as sg


@dataclass
class StepBuffers:
    """Per-step outputs of the split, sized for `rows` index rows of `total` entries."""
    order: torch.Tensor
    local: torch.Tensor
    remote: torch.Tensor
    n_local: torch.Tensor
    n_remote: torch.Tensor
    n_kept: torch.Tensor
    zeros: torch.Tensor

    @staticmethod
    def alloc(rows: int, total: int, device="cuda") -> "StepBuffers":
        i32 = dict(dtype=torch.int32, device=device)
        return StepBuffers(torch.empty(max(total, 1), **i32), torch.empty(max(total, 1), **i32),
                           torch.empty(max(total, 1), **i32), torch.empty(rows, **i32), torch.empty(rows, **i32),
                           torch.empty(rows, **i32), torch.zeros(rows, **i32))


class TwoLane:
    """Streams and events of the two lanes; create once, reuse every step."""

    def __init__(self, device=None):
        self.local_stream = torch.cuda.Stream(device=device)
        self.remote_stream = torch.cuda.Stream(device=device)

    def gather(self, *, row_off, kv_index, mask, mask_off, mask_len, store_k, store_v, store_base, src_k, src_v,
               src_base, page_table, page_size, k_pool, v_pool, buf: StepBuffers, reuse=True, stream=None):
        """Split the step's index and fill the pool; returns buf.n_kept (rows per index row).

        store_base / src_base: int64 [rows], the row of token 0 of each index row in the
        store and in the prefill side's copy; mask_off / mask_len address each row's
        mask entries (the same token positions as the store)."""
        main = stream if stream is not None else torch.cuda.current_stream()
        total = kv_index.numel()
        sg.sg_split(row_off, kv_index, mask, mask_off, mask_len, 1, buf.local, buf.remote, buf.n_local,
                    buf.n_remote, out_index=buf.order, n_kept=buf.n_kept, stream=main)
        split_done = torch.cuda.Event()
        split_done.record(main)
        self.local_stream.wait_event(split_done)
        self.remote_stream.wait_event(split_done)
        sg.sg_fetch(row_off, total, buf.local, buf.n_local, store_base, store_k, store_v, page_table, page_size,
                    buf.n_remote, k_pool, v_pool, stream=self.local_stream)
        if reuse:
            sg.sg_fetch_keep(row_off, total, buf.remote, buf.n_remote, src_base, src_k, src_v, page_table, page_size,
                             buf.zeros, k_pool, v_pool, store_base, store_k, store_v, mask, mask_off, mask_len,
                             stream=self.remote_stream)
        else:
            sg.sg_fetch(row_off, total, buf.remote, buf.n_remote, src_base, src_k, src_v, page_table, page_size,
                        buf.zeros, k_pool, v_pool, stream=self.remote_stream)
        done_l, done_r = torch.cuda.Event(), torch.cuda.Event()
        done_l.record(self.local_stream)
        done_r.record(self.remote_stream)
        main.wait_event(done_l)
        main.wait_event(done_r)
        return buf.n_kept


class SpecPusher:
    """Speculative transfer of one request's remaining blocks (Section 4.3).

    ``imp`` is the request's L * M block importances (eq. 1).  At most one
    push is in flight; each step calls ``commit_if_landed`` before its split
    and ``launch_if_idle`` after its lanes.  Neither waits: a push that has
    not landed is committed at a later step."""

    def __init__(self, src_k, src_v, imp, s0, N, M, store_k, store_v, mask, quota, L=None, device=None):
        self.src_k, self.src_v = src_k, src_v
        self.store_k, self.store_v, self.mask = store_k, store_v, mask
        self.s0, self.N, self.M = int(s0), int(N), int(M)
        self.L = store_k.shape[0] if L is None else L
        self.Hkv, self.T = store_k.shape[1], store_k.shape[2]
        self.LM = self.L * self.M
        self.rem = imp.reshape(-1)[: self.LM].clone()
        self.quota = int(quota)
        self.left = self.LM
        self.pushes = 0
        dev = imp.device
        self.ids = torch.empty(max(1, self.quota), dtype=torch.int32, device=dev)
        self.cu_row = torch.tensor([0, self.LM], dtype=torch.int32, device=dev)
        self.cu_q = {q: torch.tensor([0, q], dtype=torch.int32, device=dev)
                     for q in {self.quota, self.LM % self.quota or self.quota}}
        self.stream = torch.cuda.Stream(device=device)
        self.inflight = None        # (block count, completion event)

    def commit_if_landed(self, stream):
        """Marks the in-flight push's blocks on `stream` if its rows have landed."""
        if self.inflight is None or not self.inflight[1].query():
            return False
        q, done = self.inflight
        stream.wait_event(done)
        sg.sg_spec_commit(self.ids[:q], self.L, self.Hkv, self.T, self.s0, self.N, self.M, self.mask, self.rem,
                          stream=stream)
        self.inflight = None
        return True

    def launch_if_idle(self, stream):
        """Chooses the next quota of blocks on `stream` and pushes their rows on
        the side stream, if no push is in flight and blocks are left."""
        if self.inflight is not None or self.left == 0:
            return False
        q = min(self.quota, self.left)
        sg.sg_topk(self.rem.view(1, 1, self.LM), self.cu_row, self.LM, self.LM, self.cu_q[q], q,
                   self.ids[:q].view(1, 1, q), stream=stream)
        chosen = torch.cuda.Event()
        chosen.record(stream)
        self.stream.wait_event(chosen)
        sg.sg_spec_push(self.src_k, self.src_v, self.ids[:q], self.s0, self.N, self.M, self.store_k, self.store_v,
                        None, None, L=self.L, stream=self.stream)
        done = torch.cuda.Event()
        done.record(self.stream)
        self.inflight = (q, done)
        self.left -= q
        self.pushes += 1
        return True

    def drain(self, stream):
        """Waits on `stream` for the in-flight push and commits it."""
        if self.inflight is not None:
            self.inflight[1].synchronize()
            self.commit_if_landed(stream)
