"""Parallel on-demand transfer on one GPU (Section 4.2): stream plumbing only.

After Algorithm 1 splits a step's KV index (sg_split, remote entries first), two
lanes fill the decode pool at once:
  - the local lane (sg_fetch) gathers the local entries from the decode side's
    KV store into pool rows [n_remote, n_remote + n_local) of each index row;
  - the remote lane (sg_fetch_keep, or sg_fetch without reuse) fetches the
    remote entries from the prefill side's copy into pool rows [0, n_remote),
    and with reuse keeps them in the store and marks them local.
Each lane runs on its own stream; the caller's stream waits for both, so the
attention that follows on it sees the whole pool.  Every copy runs in the
library's kernels; this module only orders them.
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
