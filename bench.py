"""Benchmark of the selective KV-transfer hot path on one MI355X.

Headline workload (``--workload batched64``, the default): 64 requests with
prompt lengths uniform in [2048, 32768] (1.21 M tokens in all), Llama-3-8B
attention shape (32 layers, 32 q heads / 8 KV heads, d = 128, bf16), one K/V
source read by every layer, 64-query score window, 10% of each request's
tokens selected per (layer, KV head), 2% more fetched on demand per decode
step, 16-row pages.

One step is one pass of the whole path over that batch:

  prefill side   sg_score -> sg_topk -> sg_pack  (transfer buffer in HBM)
  receive        sg_fetch: the transfer buffer's rows into the decode side's
                 paged pool (logical rows 0 .. k-1 of every unit)
  D decode steps sg_split (Algorithm 1 on [extras ++ selected], per-head mask)
                 -> sg_fetch of the remote entries from the pinned-host copy
                    of the prompt K/V (the prefill node) into logical rows
                    k .. k+e-1
                 -> sg_decode_attn, one launch per layer in model order
                    (a HIP graph of L launches)

Inputs are generated on the GPU before timing.  Prints one JSON line:
  value               select+pack rate: bytes of the KV cache (K and V of every
                      layer and head, 146 GB here) turned into a transfer
                      buffer per second of score + top-k + pack time
  decode_tokens_per_s the other half of the metric: requests x decode steps per
                      second of attention time (per-layer launches, model order)
  roofline            sg_decode_attn, the HBM-bound kernel of the decode steps
  cpu_baseline        the oracle on a bounded sample, in the same run
  ops                 every op's median time (>= 20 repetitions after >= 3
                      warm-ups, HIP events on the launch stream), rates and
                      fractions of peak; ops.workloads holds the 8B 8K, 8B 32K
                      and 70B 16K workloads (including pinned-host staging)
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
import statistics
import sys
import time

_ROOT = os.path.dirname(os.path.abspath(__file__))
if _ROOT not in sys.path:
    sys.path.insert(0, _ROOT)

HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
FP32_MFMA_PEAK_TFLOPS = 157.3
# the counter summary that gives the decode kernel's measured HBM traffic at
# the headline workload, and the sources whose hash it records (a changed
# kernel makes the figure stale)
TRAFFIC_SUMMARY = os.path.join(_ROOT, "profiles", "decode_attn.batched64.hbm_traffic.md")
TRACE_SUMMARY = os.path.join(_ROOT, "profiles", "all_kernels.batched64.kernel_trace.md")
TRAFFIC_SOURCES = ("paper_2607_28150_amd/csrc/decode_attn.hip", "paper_2607_28150_amd/csrc/sg_internal.h")
REPS, WARM = 20, 3
# workgroup budget of a request pair's pack beside the next pair's score: it
# finishes within that score and disturbs it less than the full-rate grid
# (64-request workload, the select region: 47.6 ms at 1,024, 47.8 at 2,048,
# 48.6 without a budget, 54.5 at 512)
PAIR_PACK_WORKGROUPS = 1024


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=5)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--workload", default="batched64")
    p.add_argument("--decode-steps", type=int, default=16, help="decode steps per step")
    p.add_argument("--seed", type=int, default=None, help="override the workload's seed")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-ops", action="store_true", help="time the steps only (profiling runs)")
    p.add_argument("--no-workloads", action="store_true", help="skip the other workloads' ops")
    p.add_argument("--only", choices=["decode_side", "workload"], default=None,
                   help="run one section on its own and print its JSON line (profiling one workload)")
    p.add_argument("--cpu-seconds", type=float, default=8.0, help="repeat each oracle sample to at least this long")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="only run a plain device copy of MIB MiB three times (counter calibration) and exit")
    return p.parse_args()


# --------------------------------------------------------------------------- timing

def _ev():
    import torch
    return torch.cuda.Event(enable_timing=True)


def median_ms(fn, reps=REPS, warm=WARM):
    """Median over `reps` calls of fn(i) after `warm` untimed calls; each call is
    bracketed by its own pair of HIP events on the current stream."""
    import torch
    for i in range(warm):
        fn(i)
    torch.cuda.synchronize()
    evs = [(_ev(), _ev()) for _ in range(reps)]
    for i, (a, b) in enumerate(evs):
        a.record()
        fn(i)
        b.record()
    torch.cuda.synchronize()
    return statistics.median(a.elapsed_time(b) for a, b in evs)


def gbs(nbytes, ms):
    return nbytes / (ms * 1e-3) / 1e9


def r4(x):
    return round(float(x), 4)


# --------------------------------------------------------------------------- the path of one workload

class Path:
    """Every buffer of the hot path of one workload, resident before timing,
    and the library calls of one step.

    Units are ordered u = (l * B + b) * Hkv + h, so a layer's units are the
    [B][Hkv] block that one per-layer sg_decode_attn call takes, and the whole
    table is the [L * B][Hkv] block of the batched-layer call.  Every unit owns
    ceil((k_b + e_b) / P) pages of the pool, placed at seeded random pool pages.
    """

    def __init__(self, sg, cfg, decode_steps, device="cuda", staged=None):
        import torch
        from datagen import inputs, rng

        self.sg, self.cfg, self.D = sg, cfg, decode_steps
        L, Hq, Hkv, d, W, P = cfg.L, cfg.Hq, cfg.Hkv, cfg.d, cfg.W, cfg.page_size
        dev = device
        self.staged = cfg.stage_host if staged is None else staged
        pre = inputs.make_prefill(cfg, device=dev)
        self.pre = pre
        lens, T, B = pre["seqlens"], pre["T"], cfg.B
        self.lens, self.T, self.B, self.N_max = lens, T, B, max(lens)
        bud = inputs.make_budget(cfg, lens)
        self.kb, self.cu_k, self.K_total = bud["k"], bud["cu_k"], bud["K_total"]
        self.eb = [inputs.extras_count(n, cfg.extra_bp) for n in lens]
        self.E_total = sum(self.eb)
        i32 = dict(dtype=torch.int32, device=dev)
        self.cus = torch.tensor(pre["cu_seqlens"], **i32)
        self.cuk = torch.tensor(self.cu_k, **i32)
        self.esize = pre["k"].element_size()
        self.scores = torch.empty((L, Hkv, T), device=dev)
        self.idx = torch.empty((L, Hkv, self.K_total), **i32)
        self.ws_score = torch.empty(sg.score_workspace_size(B, L, Hq, Hkv, d, W, self.N_max), dtype=torch.uint8,
                                    device=dev)
        S = L * Hkv * self.K_total
        self.S = S
        nbytes = sg.pack_bytes(pre["k"].dtype, L, Hkv, d, self.K_total)
        self.tbuf = (torch.empty(nbytes, dtype=torch.uint8, pin_memory=True) if self.staged
                     else torch.empty(nbytes, dtype=torch.uint8, device=dev))
        rb = d * self.esize
        self.tk = self.tbuf[: S * rb].view(pre["k"].dtype).view(S, d)
        self.tv = self.tbuf[S * rb: 2 * S * rb].view(pre["k"].dtype).view(S, d)

        # ---- decode-side pool and page tables
        units = L * B * Hkv
        self.units = units
        rows_b = [k + e for k, e in zip(self.kb, self.eb)]
        pages_b = [-(-r // P) for r in rows_b]
        self.max_pages = max(pages_b)
        lbh = lambda v: torch.tensor(v, dtype=torch.int64, device=dev)[None, :, None].expand(L, B, Hkv).reshape(-1)  # noqa: E731
        pages_u = lbh(pages_b)
        total_pages = int(pages_u.sum())
        place = torch.argsort(rng.raw64(rng.stream_key(cfg.seed, 99, 1), total_pages, dev), stable=True)
        first = torch.cumsum(pages_u, 0) - pages_u
        j = torch.arange(self.max_pages, device=dev)[None, :]
        ok = j < pages_u[:, None]
        flat = (first[:, None] + j).clamp(max=total_pages - 1)
        self.page_table = torch.where(ok, place[flat] * P, torch.full_like(flat, -1)).to(torch.int32)
        self.page_table = self.page_table.view(L * B, Hkv, self.max_pages).contiguous()
        pool_rows = total_pages * P
        self.pool_bytes = 2 * pool_rows * rb
        # enough pool replicas that a decode step's reads do not hit in the 256 MB last-level cache
        self.reps = max(1, math.ceil(600e6 / self.pool_bytes))
        self.pools = [(torch.empty((pool_rows, d), dtype=pre["k"].dtype, device=dev),
                       torch.empty((pool_rows, d), dtype=pre["k"].dtype, device=dev)) for _ in range(self.reps)]
        self.pages_read_per_layer = int(pages_u[: B * Hkv].sum())
        self.rows_per_layer = Hkv * sum(rows_b)

        # receive: unit u's k_b rows from transfer-buffer slot (l * Hkv + h) * K_total + cu_k[b]
        l_u = torch.arange(L, device=dev)[:, None, None].expand(L, B, Hkv).reshape(-1)
        b_u = torch.arange(B, device=dev)[None, :, None].expand(L, B, Hkv).reshape(-1)
        h_u = torch.arange(Hkv, device=dev)[None, None, :].expand(L, B, Hkv).reshape(-1)
        k_u = lbh(self.kb)
        e_u = lbh(self.eb)
        cuk_t = torch.tensor(self.cu_k[:-1], dtype=torch.int64, device=dev)
        cus_t = torch.tensor(pre["cu_seqlens"][:-1], dtype=torch.int64, device=dev)
        self.recv_off = torch.cat([torch.zeros(1, dtype=torch.int64, device=dev), torch.cumsum(k_u, 0)]).to(torch.int32)
        self.recv_src = (l_u * Hkv + h_u) * self.K_total + cuk_t[b_u]
        self.zeros = torch.zeros(units, **i32)

        # decode steps: index row of unit u = [e_b extras ++ k_b selected], mask per (l, h, token)
        rows_u = k_u + e_u
        self.row_off = torch.cat([torch.zeros(1, dtype=torch.int64, device=dev), torch.cumsum(rows_u, 0)])
        self.total = int(self.row_off[-1])
        self.row_off = self.row_off.to(torch.int32)
        self.mask = torch.full((L, Hkv, T), 2, dtype=torch.int8, device=dev)
        self.mask_off = (l_u * Hkv + h_u) * T + cus_t[b_u]
        self.mask_len = lbh(lens).to(torch.int32)
        lk = torch.zeros_like(l_u) if cfg.kv_shared_layers else l_u
        self.src_base = (lk * Hkv + h_u) * T + cus_t[b_u]
        self.dst_start = k_u.to(torch.int32)
        self.host_k = pre["k"].cpu().pin_memory() if self.E_total else None
        self.host_v = pre["v"].cpu().pin_memory() if self.E_total else None
        self.local = torch.empty(max(1, self.total), **i32)
        self.remote = torch.empty(max(1, self.total), **i32)
        self.n_local = torch.empty(units, **i32)
        self.n_remote = torch.empty(units, **i32)
        self.n_kept = torch.empty(units, **i32)
        # position of every index entry in cat([extras of all layers, selection of all layers])
        u_of = torch.repeat_interleave(torch.arange(units, device=dev), rows_u)
        jj = torch.arange(self.total, device=dev) - self.row_off[:-1].to(torch.int64)[u_of]
        lu, bu, hu = l_u[u_of], b_u[u_of], h_u[u_of]
        eu = e_u[u_of]
        cue_t = torch.tensor(inputs.cu_from_lengths(self.eb)[:-1], dtype=torch.int64, device=dev)
        ext_pos = (lu * Hkv + hu) * self.E_total + cue_t[bu] + jj
        sel_pos = L * Hkv * self.E_total + (lu * Hkv + hu) * self.K_total + cuk_t[bu] + (jj - eu)
        self._entry_src = torch.where(jj < eu, ext_pos, sel_pos)
        del u_of, jj, lu, bu, hu, eu, ext_pos, sel_pos
        self.qdec = [inputs.decode_queries(cfg, s, device=dev, mu=pre["mu"]).permute(1, 0, 2, 3).contiguous()
                     for s in range(decode_steps)]                    # [L][B][Hq][d]
        self.out = torch.empty((L, B, Hq, d), device=dev)
        self.ws_layer = torch.zeros(max(16, sg.decode_workspace_size(B, Hq, Hkv, d, self.max_pages, P)),
                                    dtype=torch.uint8, device=dev)
        self.ws_all = torch.zeros(max(16, sg.decode_workspace_size(L * B, Hq, Hkv, d, self.max_pages, P)),
                                  dtype=torch.uint8, device=dev)
        self.kv_index = []
        self.graphs = []
        # the select region in request groups: pairs of consecutive requests,
        # the longest pairs first, each pair's top-k and pack on a second
        # stream beside the next pair's score.  Used only when every pair's
        # score call keeps full-length key chunks (enough workgroups), so the
        # outputs are bit-identical to one call over the whole batch.
        full_chunks = lambda b0, b1: (b1 - b0) * L * Hkv * -(-max(lens[b0:b1]) // 2048) >= 1024  # noqa: E731
        pairs = [(b, min(B, b + 2)) for b in range(0, B, 2)]
        self.select_groups = []
        if B >= 4 and all(full_chunks(a, b) for a, b in pairs):
            pairs.sort(key=lambda ab: -sum(lens[ab[0]:ab[1]]))
            self.select_groups = [dict(a=a, b=b, nmax=max(lens[a:b]), maxk=max(self.kb[a:b])) for a, b in pairs]
        self.sel_stream = torch.cuda.Stream(device=dev)

    # ---- the calls of a step
    def score(self, lse_in=None):
        c = self.cfg
        self.sg.sg_score(self.pre["q_win"], self.pre["k"], self.cus, self.T, self.N_max, c.Hkv, self.scores,
                         ws=self.ws_score, lse_in=lse_in)

    def topk(self):
        self.sg.sg_topk(self.scores, self.cus, self.T, self.N_max, self.cuk, self.K_total, self.idx)

    def pack(self):
        self.sg.sg_pack(self.pre["k"], self.pre["v"], self.idx, self.cus, self.T, self.cuk, self.K_total,
                        max(self.kb), self.tbuf, L=self.cfg.L, Hkv=self.cfg.Hkv)

    def select(self):
        """score -> top-k -> pack over the batch; in request groups when
        `select_groups` is set (see the constructor)."""
        import torch
        if not self.select_groups:
            self.score()
            self.topk()
            self.pack()
            return
        c = self.cfg
        main = torch.cuda.current_stream()
        side = self.sel_stream
        side.wait_stream(main)
        for g in self.select_groups:
            a, b = g["a"], g["b"]
            self.sg.sg_score(self.pre["q_win"][a:b], self.pre["k"], self.cus[a:b + 1], self.T, g["nmax"], c.Hkv,
                             self.scores, ws=self.ws_score)
            done = torch.cuda.Event()
            done.record(main)
            side.wait_event(done)
            with torch.cuda.stream(side):
                self.sg.sg_topk(self.scores, self.cus[a:b + 1], self.T, g["nmax"], self.cuk[a:b + 1], self.K_total,
                                self.idx)
                self.sg.sg_pack(self.pre["k"], self.pre["v"], self.idx, self.cus[a:b + 1], self.T,
                                self.cuk[a:b + 1], self.K_total, g["maxk"], self.tbuf, L=c.L, Hkv=c.Hkv,
                                max_workgroups=PAIR_PACK_WORKGROUPS)
        main.wait_stream(side)

    def receive(self, rep=0):
        kp, vp = self.pools[rep]
        self.sg.sg_fetch(self.recv_off, self.S, None, None, self.recv_src, self.tk, self.tv,
                         self.page_table.view(self.units, -1), self.cfg.page_size, self.zeros, kp, vp)

    def split(self, s):
        self.sg.sg_split(self.row_off, self.kv_index[s], self.mask.view(-1), self.mask_off, self.mask_len, 0,
                         self.local, self.remote, self.n_local, self.n_remote, n_kept=self.n_kept)

    def fetch(self, s):
        if not self.E_total:
            return
        kp, vp = self.pools[s % self.reps]
        self.sg.sg_fetch(self.row_off, self.total, self.remote, self.n_remote, self.src_base, self.host_k,
                         self.host_v, self.page_table.view(self.units, -1), self.cfg.page_size, self.dst_start,
                         kp, vp)

    def attn_layers(self, s):
        c = self.cfg
        B, Hkv = self.B, c.Hkv
        kp, vp = self.pools[s % self.reps]
        q = self.qdec[s]
        nk = self.n_kept.view(c.L * B, Hkv)
        for l in range(c.L):
            self.sg.sg_decode_attn(q[l], kp, vp, self.page_table[l * B:(l + 1) * B], nk[l * B:(l + 1) * B],
                                   c.page_size, self.out[l], ws=self.ws_layer)

    def attn_batched(self, s):
        c = self.cfg
        kp, vp = self.pools[s % self.reps]
        self.sg.sg_decode_attn(self.qdec[s].view(c.L * self.B, c.Hq, c.d), kp, vp, self.page_table,
                               self.n_kept.view(c.L * self.B, c.Hkv), c.page_size,
                               self.out.view(c.L * self.B, c.Hq, c.d), ws=self.ws_all)

    def attn_graph(self, s):
        self.graphs[s].replay()

    # ---- set-up that needs the selection
    def prepare(self, capture=True, selection=None, verify=True):
        """Runs the select region once (or takes `selection`, an index table
        [L][Hkv][K_total], in place of score and top-k), then builds what the
        decode side holds after the transfer (the per-head mask from the
        selection, every pool replica with the received rows) and each decode
        step's KV index (extras drawn from the complement of the selection).
        Captures one graph per decode step of the per-layer attention launches
        and (`verify`) checks every replay bit for bit against eager launches;
        profiling runs skip the check so that every traced launch is a timed
        one."""
        import torch
        from datagen import inputs
        c = self.cfg
        L, Hkv, B, dev = c.L, c.Hkv, self.B, self.idx.device
        if selection is None:
            self.score()
            self.topk()
        else:
            self.idx.copy_(selection)
        self.pack()
        for r in range(self.reps):
            self.receive(r)
        ks = torch.tensor(self.kb, dtype=torch.int64, device=dev)
        col_off = torch.tensor(self.pre["cu_seqlens"][:-1], dtype=torch.int64, device=dev)
        col_off = torch.repeat_interleave(col_off, ks)
        self.mask.view(L * Hkv, self.T).scatter_(1, self.idx.view(L * Hkv, -1).to(torch.int64) + col_off[None, :], 1)
        for s in range(self.D):
            if self.E_total:
                ex = torch.stack([inputs.extras_layer(c, s, self.lens, self.idx[l], self.cu_k, l)[0]
                                  for l in range(L)])                    # [L][Hkv][E_total]
                src = torch.cat([ex.reshape(-1), self.idx.reshape(-1)])
            else:
                src = self.idx.reshape(-1)
            self.kv_index.append(src[self._entry_src].contiguous())
        del self._entry_src
        torch.cuda.synchronize()
        if not capture:
            return
        if not verify:
            # one eager decode step before capture (the library's first-call set-up)
            self.split(0)
            self.fetch(0)
            self.attn_layers(0)
            torch.cuda.synchronize()
        for s in range(self.D):
            if not verify:
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g):
                    self.attn_layers(s)
                self.graphs.append(g)
                continue
            self.split(s)
            self.fetch(s)
            self.attn_layers(s)
            torch.cuda.synchronize()
            ref = self.out.clone()
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                self.attn_layers(s)
            torch.cuda.current_stream().wait_stream(side)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                self.attn_layers(s)
            for _ in range(3):
                self.out.fill_(float("nan"))
                g.replay()
                torch.cuda.synchronize()
                assert torch.equal(self.out, ref), "graph replay differs from the eager launches"
                self.attn_layers(s)
                torch.cuda.synchronize()
            self.graphs.append(g)

    # ---- algorithmic work
    def score_flops(self):
        c = self.cfg
        W = c.W
        return sum(2.0 * c.d * c.G * (W * n - W * (W - 1) / 2) for n in self.lens) * c.L * c.Hkv

    def kv_cache_bytes(self):
        c = self.cfg
        return 2 * c.L * c.Hkv * self.T * c.d * self.esize

    def pack_bytes(self):
        return 2 * self.S * self.cfg.d * self.esize * 2 + self.S * 4 * 2      # rows read + written, ids read + written

    def receive_bytes(self):
        return 2 * self.S * self.cfg.d * self.esize * 2                         # rows read + written

    def fetch_bytes(self):
        return self.cfg.L * self.cfg.Hkv * self.E_total * 2 * self.cfg.d * self.esize

    def decode_layer_bytes(self):
        c = self.cfg
        return (self.rows_per_layer * 2 * c.d * self.esize + self.B * c.Hq * c.d * (self.esize + 4)
                + self.pages_read_per_layer * 4 + self.B * c.Hkv * 4)

    def free(self):
        import torch
        for k in list(self.__dict__):
            setattr(self, k, None)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()


# --------------------------------------------------------------------------- ops of a path

def path_ops(p: Path, lse=False):
    """Median time of every op of the path, with rates and fractions of peak."""
    import torch
    c = p.cfg
    peak_mfma = BF16_MFMA_PEAK_TFLOPS if c.dtype == "bf16" else FP32_MFMA_PEAK_TFLOPS
    fl = p.score_flops()
    ops = {}
    t = median_ms(lambda i: p.score())
    ops["score"] = {"ms": r4(t), "tflops": round(fl / (t * 1e-3) / 1e12, 1),
                    "frac_mfma_peak": r4(fl / (t * 1e-3) / 1e12 / peak_mfma), "gflop_algorithmic": round(fl / 1e9, 1),
                    "note": "self-contained: row statistics pass + column-sum pass (the contraction runs twice)"}
    if lse:
        lse_win = window_lse(p.pre["q_win"], p.pre["k"], p.lens, c.Hkv, c.W, c.d, c.kv_shared_layers)
        t = median_ms(lambda i: p.score(lse_in=lse_win))
        ops["score_lse_in"] = {"ms": r4(t), "tflops": round(fl / (t * 1e-3) / 1e12, 1),
                               "frac_mfma_peak": r4(fl / (t * 1e-3) / 1e12 / peak_mfma),
                               "note": "one pass: window-row log-sum-exp supplied by the prefill attention"}
        del lse_win
        p.score()
    t = median_ms(lambda i: p.topk())
    ops["topk"] = {"ms": r4(t), "rows": c.L * c.Hkv * p.B, "k_total": p.K_total}
    t = median_ms(lambda i: p.pack())
    pb = p.pack_bytes()
    if p.staged:
        ops["stage_host"] = {"ms": r4(t), "host_link_mb": round((pb / 2) / 1e6, 1),
                             "host_link_gbs": round(gbs(pb / 2, t), 1),
                             "note": "sg_pack with a pinned-host destination: rows + ids read from HBM, written "
                                     "over the host link"}
    else:
        ops["pack"] = {"ms": r4(t), "gbs": round(gbs(pb, t), 1), "frac_hbm_peak": r4(gbs(pb, t) / HBM_PEAK_GBS),
                       "mb_algorithmic": round(pb / 1e6, 1)}
    kvb = p.kv_cache_bytes()
    t = median_ms(lambda i: (p.score(), p.topk(), p.pack()))
    ops["select_one_call"] = {"ms": r4(t), "gbs_kv_cache": round(gbs(kvb, t), 1),
                              "note": "score, top-k and pack over the whole batch, one call each on one stream"}
    if p.select_groups:
        t = median_ms(lambda i: p.select())
        ops["select_request_pairs"] = {"ms": r4(t), "gbs_kv_cache": round(gbs(kvb, t), 1), "groups": len(p.select_groups),
                                       "note": "the timed form: pairs of requests, each pair's top-k and pack on a "
                                               "second stream beside the next pair's score"}
    t = median_ms(lambda i: p.receive(i % p.reps))
    rb = p.receive_bytes()
    ops["receive"] = {"ms": r4(t), "mb_algorithmic": round(rb / 1e6, 1)}
    if p.staged:
        ops["receive"].update({"host_link_gbs": round(gbs(rb / 2, t), 1),
                               "note": "sg_fetch from the pinned-host transfer buffer into the pool pages"})
    else:
        ops["receive"].update({"gbs": round(gbs(rb, t), 1), "frac_hbm_peak": r4(gbs(rb, t) / HBM_PEAK_GBS)})
    t = median_ms(lambda i: p.split(i % p.D))
    ops["split"] = {"ms": r4(t), "entries": p.total}
    if p.E_total:
        p.split(0)
        t = median_ms(lambda i: p.fetch(0))
        fb = p.fetch_bytes()
        ops["fetch"] = {"ms": r4(t), "host_link_mb": round(fb / 1e6, 1), "host_link_gbs": round(gbs(fb, t), 1),
                        "rows": c.L * c.Hkv * p.E_total}
    p.split(0)
    p.fetch(0)
    lb = p.decode_layer_bytes()
    t = median_ms(lambda i: p.attn_graph(0)) if p.graphs else median_ms(lambda i: p.attn_layers(0))
    ops["decode_attn_per_layer"] = {
        "ms_per_step": r4(t), "launches_per_step": c.L, "mb_per_launch": round(lb / 1e6, 1),
        "gbs": round(gbs(lb * c.L, t), 1), "frac_hbm_peak": r4(gbs(lb * c.L, t) / HBM_PEAK_GBS),
        "tokens_per_s": round(p.B / (t * 1e-3), 1),
        "note": "one sg_decode_attn per layer in model order, replayed from a HIP graph (bit-identical to eager)"}
    t = median_ms(lambda i: p.attn_batched(0))
    ops["decode_attn_batched_layers"] = {
        "ms_per_step": r4(t), "gbs": round(gbs(lb * c.L, t), 1), "frac_hbm_peak": r4(gbs(lb * c.L, t) / HBM_PEAK_GBS),
        "tokens_per_s": round(p.B / (t * 1e-3), 1),
        "note": "all layers in one launch as L x B sequences: a kernel-bandwidth ceiling, not a model order"}
    return ops


def select_per_layer_kv(sg, cfg):
    """The select region of `cfg` with a K/V source per layer instead of one
    shared by the layers (the headline workload shares one to keep its decode
    side in memory): no layer finds another layer's keys in the last-level
    cache.  Both forms, one call and request pairs; outputs compared."""
    import torch
    from datagen import inputs
    c = cfg.with_(kv_shared_layers=False)
    pre = inputs.make_prefill(c, device="cuda")
    lens, T, B, L, Hkv, d = pre["seqlens"], pre["T"], c.B, c.L, c.Hkv, c.d
    bud = inputs.make_budget(c, lens)
    kb, K_total = bud["k"], bud["K_total"]
    i32 = dict(dtype=torch.int32, device="cuda")
    cus, cuk = torch.tensor(pre["cu_seqlens"], **i32), torch.tensor(bud["cu_k"], **i32)
    scores = torch.empty((L, Hkv, T), device="cuda")
    idx = torch.empty((L, Hkv, K_total), **i32)
    ws = torch.empty(sg.score_workspace_size(B, L, c.Hq, Hkv, d, c.W, max(lens)), dtype=torch.uint8, device="cuda")
    tbuf = torch.empty(sg.pack_bytes(pre["k"].dtype, L, Hkv, d, K_total), dtype=torch.uint8, device="cuda")
    side = torch.cuda.Stream()

    def one_call():
        sg.sg_score(pre["q_win"], pre["k"], cus, T, max(lens), Hkv, scores, ws=ws)
        sg.sg_topk(scores, cus, T, max(lens), cuk, K_total, idx)
        sg.sg_pack(pre["k"], pre["v"], idx, cus, T, cuk, K_total, max(kb), tbuf, L=L, Hkv=Hkv)

    pairs = sorted([(b, min(B, b + 2)) for b in range(0, B, 2)], key=lambda ab: -sum(lens[ab[0]:ab[1]]))

    def pairs_call():
        main = torch.cuda.current_stream()
        side.wait_stream(main)
        for a, b in pairs:
            sg.sg_score(pre["q_win"][a:b], pre["k"], cus[a:b + 1], T, max(lens[a:b]), Hkv, scores, ws=ws)
            done = torch.cuda.Event()
            done.record(main)
            side.wait_event(done)
            with torch.cuda.stream(side):
                sg.sg_topk(scores, cus[a:b + 1], T, max(lens[a:b]), cuk[a:b + 1], K_total, idx)
                sg.sg_pack(pre["k"], pre["v"], idx, cus[a:b + 1], T, cuk[a:b + 1], K_total, max(kb[a:b]), tbuf,
                           L=L, Hkv=Hkv)
        main.wait_stream(side)

    kvb = 2 * L * Hkv * T * d * pre["k"].element_size()
    one_call()
    torch.cuda.synchronize()
    ref = (scores.clone(), idx.clone())
    t1 = median_ms(lambda i: one_call(), reps=5, warm=1)
    pairs_call()
    torch.cuda.synchronize()
    same = bool(torch.equal(scores, ref[0]) and torch.equal(idx, ref[1]))
    t2 = median_ms(lambda i: pairs_call(), reps=5, warm=1)
    res = {"one_call_ms": r4(t1), "one_call_gbs": round(gbs(kvb, t1), 1), "request_pairs_ms": r4(t2),
           "request_pairs_gbs": round(gbs(kvb, t2), 1), "pairs_identical_to_one_call": same,
           "note": "K/V source per layer (159 GB): no cross-layer cache reuse; 5 repetitions each"}
    del pre, scores, idx, ws, tbuf, ref
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def window_lse(q_win, k, lens, Hkv, W, d, shared):
    """[B][L][Hq][W] natural-log LSE of the scaled causal logits of every
    request's window rows (row w sits at position N - W + w), in fp32 with
    torch: what a prefill attention kernel leaves behind."""
    import torch
    B, L, Hq, _, _ = q_win.shape
    G = Hq // Hkv
    out = torch.empty((B, L, Hq, W), dtype=torch.float32, device=q_win.device)
    off = 0
    for b, N in enumerate(lens):
        pos = torch.arange(N - W, N, device=q_win.device)[:, None]
        late = torch.arange(N, device=q_win.device)[None, :] > pos
        for l in range(L):
            lk = 0 if shared else l
            for h in range(Hkv):
                q = q_win[b, l, h * G:(h + 1) * G].float().reshape(G * W, d)
                kt = k[lk, h, off:off + N].float().t().contiguous()
                z = ((q @ kt) * (d ** -0.5)).view(G, W, N).masked_fill(late, float("-inf"))
                out[b, l, h * G:(h + 1) * G] = torch.logsumexp(z, dim=-1)
        off += N
    return out


# --------------------------------------------------------------------------- host link and device copy

def host_link(nbytes=1 << 30):
    """Pinned-host <-> device hipMemcpyAsync rates (the host link's measured peak)."""
    import torch
    h = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    g = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    t_h2d = median_ms(lambda i: g.copy_(h, non_blocking=True), reps=10, warm=2)
    t_d2h = median_ms(lambda i: h.copy_(g, non_blocking=True), reps=10, warm=2)
    del h, g
    return {"h2d_gbs": round(gbs(nbytes, t_h2d), 1), "d2h_gbs": round(gbs(nbytes, t_d2h), 1),
            "mb": round(nbytes / 1e6, 1), "note": "hipMemcpyAsync between pinned host memory and HBM, median of 10"}


def device_copy(nbytes):
    """A plain device-to-device copy (bytes read + written) over rotating
    buffers: the on-box ceiling for the gathers."""
    import torch
    src = [torch.ones(nbytes, dtype=torch.uint8, device="cuda") for _ in range(3)]
    dst = [torch.empty(nbytes, dtype=torch.uint8, device="cuda") for _ in range(3)]
    t = median_ms(lambda i: dst[i % 3].copy_(src[(i + 1) % 3]))
    del src, dst
    return {"gbs": round(gbs(2 * nbytes, t), 1), "ms": r4(t), "mb": round(nbytes / 1e6, 1)}


# --------------------------------------------------------------------------- main

def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the path runs on one GPU only; --gpus must be 1",
                          "n_gpus_requested": args.gpus}), flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    if args.copy_calibration:
        n = args.copy_calibration << 20
        a = torch.ones(n, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 3}), flush=True)
        return

    from datagen.configs import get
    from paper_2607_28150_amd import smartgen as sg

    if not os.path.exists(sg.LIB_PATH):
        from paper_2607_28150_amd import build as hip_build
        hip_build.build()
    sg.load()
    assert torch.cuda.is_available(), "bench needs a GPU"
    if args.only == "decode_side":
        print(json.dumps({"section": "decode_side", "n_gpus": 1, "decode_side": decode_side(sg)}), flush=True)
        return
    cfg = get(args.workload)
    if args.seed is not None:
        cfg = cfg.with_(seed=args.seed)
    if args.only == "workload":
        print(json.dumps({"section": "workload", "workload": cfg.name, "ops": workload_ops(sg, cfg.name)}),
              flush=True)
        return
    D = args.decode_steps
    L, Hkv = cfg.L, cfg.Hkv

    # ------------------------------------------------------------- inputs (resident in HBM)
    t0 = time.time()
    p = Path(sg, cfg, D)
    print(f"[bench] {cfg.name}: inputs made in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
    p.prepare(verify=not args.no_ops)         # profiling runs (--no-ops) trace the timed launches only
    setup_s = time.time() - t0
    print(f"[bench] {cfg.name}: set-up done in {setup_s:.1f} s", file=sys.stderr, flush=True)

    NE = 3 + 3 * D

    def step(e):
        rec = (lambda i: e[i].record()) if e is not None else (lambda i: None)
        rec(0)
        p.select()
        rec(1)
        p.receive()
        rec(2)
        for s in range(D):
            p.split(s)
            rec(3 + 3 * s)
            p.fetch(s)
            rec(4 + 3 * s)
            p.attn_graph(s)
            rec(5 + 3 * s)

    for _ in range(args.warmup):
        step(None)
    torch.cuda.synchronize()
    evs = [[_ev() for _ in range(NE)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    print(f"[bench] {cfg.name}: {args.steps} steps in {wall:.2f} s", file=sys.stderr, flush=True)

    def seg(i, j):
        return float(np.median([e[i].elapsed_time(e[j]) for e in evs]))

    def seg_dec(part):
        # decode step s: split from the previous mark to 3 + 3s, fetch to 4 + 3s, attention to 5 + 3s
        def one(e, s):
            return e[2 + 3 * s + part].elapsed_time(e[3 + 3 * s + part])
        return float(np.median([np.mean([one(e, s) for s in range(D)]) for e in evs]))

    t_select, t_recv = seg(0, 1), seg(1, 2)
    t_split, t_fetch, t_attn = seg_dec(0), seg_dec(1), seg_dec(2)
    ms_per_step = wall * 1e3 / args.steps
    value = gbs(p.kv_cache_bytes(), t_select)
    lb = p.decode_layer_bytes()
    dec_gbs = gbs(lb, t_attn / L)
    tokens_per_s = p.B / (t_attn * 1e-3)
    step_tok_s = p.B / ((t_split + t_fetch + t_attn) * 1e-3)

    line = {
        "metric": "select+pack GB/s and sparse decode-attn tokens/s; % of MI355X HBM/MFMA peak",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name, "requests": p.B, "layers": L, "q_heads": cfg.Hq, "kv_heads": Hkv,
                   "head_dim": cfg.d, "prompt_tokens": p.T, "prompt_min": min(p.lens), "prompt_max": max(p.lens),
                   "score_window": cfg.W, "budget_bp": cfg.budget_bp, "extra_bp": cfg.extra_bp,
                   "selected_rows": p.K_total, "extra_rows": p.E_total, "decode_steps": D,
                   "page_size": cfg.page_size, "kv_source_shared_by_layers": cfg.kv_shared_layers,
                   "seed": cfg.seed},
        "select_ms": r4(t_select),
        "value_note": "bytes of the KV cache of every layer and head turned into a transfer buffer per second of "
                      "score + top-k + pack time (medians over the timed steps); the select region runs in pairs "
                      "of requests, each pair's top-k and pack (under a budget of 1,024 workgroups) beside the next "
                      "pair's score (outputs bit-identical "
                      "to one call over the batch); the layers share one K/V source, whose keys the last-level "
                      "cache serves to later layers: ops.select_per_layer_kv times a source per layer" if p.select_groups else
                      "bytes of the KV cache of every layer and head turned into a transfer buffer per second of "
                      "score + top-k + pack time (medians over the timed steps)",
        "decode_tokens_per_s": round(tokens_per_s, 1),
        "decode_tokens_per_s_note": "requests per second of decode attention, one launch per layer in model order "
                                    "(HIP graph); without the on-demand fetch",
        "decode_step_tokens_per_s": round(step_tok_s, 1),
        "decode_step_tokens_per_s_note": "requests per second of whole decode steps: Algorithm 1 + on-demand "
                                         "fetch over the host link + attention",
        "step_ms": {"select": r4(t_select), "receive": r4(t_recv),
                    "split_per_decode_step": r4(t_split), "fetch_per_decode_step": r4(t_fetch),
                    "attention_per_decode_step": r4(t_attn)},
        "roofline": {"kernel": "sg_decode_attn", "bound": "hbm", "achieved": round(dec_gbs, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": r4(dec_gbs / HBM_PEAK_GBS),
                     "traffic": measured_traffic(), "bytes_per_launch": lb,
                     "avg_launch_ms": round(t_attn / L, 5),
                     "basis": f"HIP events around each decode step's graph of {L} per-layer launches in the timed "
                              "steps (median), divided by the launches; includes the gaps between launches"},
        "roofline_kernel_trace": None,
        "setup_s": round(setup_s, 1),
    }
    kt = _summary_figure(TRACE_SUMMARY, "kernel_trace_avg_us")
    if kt:
        line["roofline_kernel_trace"] = {
            "avg_launch_us": kt, "achieved": round(lb / (kt * 1e-6) / 1e9, 1),
            "frac": r4(lb / (kt * 1e-6) / 1e9 / HBM_PEAK_GBS),
            "basis": "rocprofv3 kernel-trace average of the same launches (committed summary), gaps excluded"}
    if not args.no_ops:
        ops = path_ops(p)
        ops["host_link"] = host_link()
        ops["measured_copy"] = device_copy(lb // 2)
        cp = ops["measured_copy"]["gbs"]
        for k in ("pack", "receive", "decode_attn_per_layer", "decode_attn_batched_layers"):
            if k in ops and "gbs" in ops[k]:
                ops[k]["frac_measured_copy"] = r4(ops[k]["gbs"] / cp)
        if "fetch" in ops:
            ops["fetch"]["frac_host_link_peak"] = r4(ops["fetch"]["host_link_gbs"] / ops["host_link"]["h2d_gbs"])
        line["roofline"]["frac_measured_copy"] = r4(dec_gbs / cp)
        line["ops"] = ops
    cpu_in = None
    if not args.no_cpu_baseline:
        cpu_in = cpu_inputs(p)
    p.free()
    del p
    if not args.no_ops and cfg.kv_shared_layers and cfg.B >= 4:
        print("[bench] select with a K/V source per layer", file=sys.stderr, flush=True)
        torch.cuda.empty_cache()
        line["ops"]["select_per_layer_kv"] = select_per_layer_kv(sg, cfg)
    if not args.no_ops and not args.no_workloads:
        wl = {}
        for name in ("llama8b_8k", "llama8b_32k", "llama70b_16k"):
            print(f"[bench] workload {name}", file=sys.stderr, flush=True)
            wl[name] = workload_ops(sg, name)
        print("[bench] decode side (8B 32K)", file=sys.stderr, flush=True)
        wl["llama8b_32k"]["decode_side"] = decode_side(sg)
        for name in ("llama70b_16k", "llama8b_32k"):
            o = wl[name]
            for k in ("stage_host", "fetch"):
                if k in o and "host_link_gbs" in o[k]:
                    o[k]["frac_host_link_peak"] = r4(o[k]["host_link_gbs"] / line["ops"]["host_link"][
                        "d2h_gbs" if k == "stage_host" else "h2d_gbs"])
        line["ops"]["workloads"] = wl

    # ------------------------------------------------------------- oracle on the host cores
    if cpu_in is not None:
        print("[bench] oracle baseline", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(cfg, cpu_in, args.cpu_seconds)
        line["gpu_over_cpu"] = round(value / line["cpu_baseline"]["value"], 1)
        line["decode_gpu_over_cpu"] = round(tokens_per_s / line["cpu_baseline"]["decode"]["tokens_per_s"], 1)
    print(json.dumps(line), flush=True)


# --------------------------------------------------------------------------- other workloads

def workload_ops(sg, name, decode_steps=2):
    """Ops of one of the other workloads through the same path (the 70B slice
    stages its transfer buffer in pinned host memory and the decode side
    receives it from there); the 8B 8K workload also times block mode and the
    selector variants."""
    import torch
    from datagen.configs import get
    cfg = get(name)
    p = Path(sg, cfg, decode_steps)
    p.prepare()
    ops = path_ops(p, lse=True)
    ops["config"] = {"layers": cfg.L, "q_heads": cfg.Hq, "kv_heads": cfg.Hkv, "prompt": p.lens[0], "k": p.K_total,
                     "extras": p.E_total, "staged_in_host_memory": p.staged, "pool_replicas": p.reps}
    if name == "llama8b_8k":
        esize = p.esize
        ops["block_mode"] = block_mode(sg, p.scores, p.cus, p.T, p.lens[0], cfg.L, cfg.Hkv, cfg.d, p.pre, esize)
        ops["selectors"] = selectors(sg, cfg, p.pre, p.cus, p.cuk, p.T, p.lens[0], p.K_total, p.idx)
    p.free()
    torch.cuda.empty_cache()
    return ops


def block_mode(sg, scores, cus, T, N, L, Hkv, d, pre, esize, M=1024, ratio=1 / 6.5):
    """Times eq. 1 (block importance), the top-K_r over the L * M blocks and the
    push of the chosen blocks (device destination, two alternating buffers).
    The default T_p / T_t of 1 / 6.5 is the transfer-to-prefill time ratio
    that Section 1 reports for a 48K-token prompt."""
    import torch
    dev = scores.device
    Kr = sg.block_budget(M, L, ratio, 1.0)
    imp = torch.empty((1, L, M), device=dev)
    ids = torch.empty((1, 1, Kr), dtype=torch.int32, device=dev)
    cu_row, cu_kr = (torch.tensor([0, L * M], dtype=torch.int32, device=dev),
                     torch.tensor([0, Kr], dtype=torch.int32, device=dev))
    nbytes = sg.pack_blocks_bytes(pre["k"].dtype, Hkv, d, N, M, Kr)
    dsts = [torch.empty(nbytes, dtype=torch.uint8, device=dev) for _ in range(3)]
    t_imp = median_ms(lambda i: sg.sg_block_importance(scores, cus, T, M, imp))
    t_top = median_ms(lambda i: sg.sg_topk(imp.view(1, 1, L * M), cu_row, L * M, L * M, cu_kr, Kr, ids))
    t_pack = median_ms(lambda i: sg.sg_pack_blocks(pre["k"], pre["v"], ids.view(-1), 0, N, M, dsts[i % 3]))
    Nb = -(-N // M)
    rows = Kr * Hkv * Nb
    pack_bytes = 2 * 2 * rows * d * esize + 2 * Kr * 4                # rows read + written, ids read + written
    imp_bytes = L * Hkv * N * 4 + L * M * 4
    return {"M": M, "transfer_over_prefill": round(1 / ratio, 2), "K_r": Kr, "blocks": L * M,
            "importance_ms": r4(t_imp), "importance_gbs": round(gbs(imp_bytes, t_imp), 1),
            "topk_ms": r4(t_top),
            "pack_ms": r4(t_pack), "pack_gbs": round(gbs(pack_bytes, t_pack), 1),
            "pack_frac_hbm_peak": r4(gbs(pack_bytes, t_pack) / HBM_PEAK_GBS),
            "pack_mb_algorithmic": round(pack_bytes / 1e6, 2)}


def decode_side(sg, nsteps=12, long_steps=256, ratio_bp=1000, M=1024):
    """Decode side of the 8B-shaped 32K-token workload (5% of the rows sent at
    prefill, 2% more fetched on demand per step, all 32 layers per step):
    Algorithm 1 and the two lanes of Section 4.2 (serial on one stream, or on
    two streams; with and without reuse of fetched rows), and speculative
    transfer (Section 4.3: the quota of remaining blocks pushed on a side stream
    while the decode steps go on; a step's split waits only for pushes that
    have already completed).  The prefill side's copy of K / V is pinned host
    memory, so the remote lane and the speculative push cross the host link;
    the decode side's store is in HBM."""
    import numpy as np
    import torch
    from datagen import inputs
    from datagen.configs import get
    from paper_2607_28150_amd.lanes import SpecPusher, StepBuffers, TwoLane

    cfg = get("llama8b_32k")
    dev = "cuda"
    L, Hq, Hkv, d, W, P = cfg.L, cfg.Hq, cfg.Hkv, cfg.d, cfg.W, cfg.page_size
    pre = inputs.make_prefill(cfg, device=dev)
    lens, T = pre["seqlens"], pre["T"]
    N = lens[0]
    bud = inputs.make_budget(cfg, lens)
    kb = bud["k"][0]
    e = inputs.extras_count(N, cfg.extra_bp)
    sel = inputs.random_selection(cfg, lens, bud["k"], device=dev)               # [L][Hkv][kb]
    src_k = pre["k"].cpu().pin_memory()
    src_v = pre["v"].cpu().pin_memory()
    store_k = torch.zeros_like(pre["k"])
    store_v = torch.zeros_like(pre["v"])
    mask = torch.empty((L, Hkv, T), dtype=torch.int8, device=dev)
    rows = L * Hkv
    base = torch.arange(rows, device=dev, dtype=torch.int64) * T
    mlen = torch.full((rows,), N, dtype=torch.int32, device=dev)
    sel_off = (torch.arange(rows + 1, device=dev) * kb).to(torch.int32)

    def reset():
        mask.fill_(2)
        sg.sg_fetch_keep(sel_off, rows * kb, sel.view(-1), None, base, src_k, src_v, None, 1, None, None, None,
                         base, store_k, store_v, mask.view(-1), base, mlen)

    # each step's KV index per (layer, head): that step's extras, then the selected rows
    per = kb + e
    nidx = max(nsteps, long_steps)
    idx = torch.empty((nidx, rows, per), dtype=torch.int32, device=dev)
    for s in range(nidx):
        ex, _ = inputs.extras_layers(cfg, s, lens, sel, bud["cu_k"], range(L))
        idx[s, :, :e] = ex.view(rows, e)
        idx[s, :, e:] = sel.view(rows, kb)
    row_off = (torch.arange(rows + 1, device=dev) * per).to(torch.int32)
    max_pages = -(-per // P)
    page_table = ((torch.arange(rows, device=dev)[:, None] * max_pages + torch.arange(max_pages, device=dev))
                  * P).to(torch.int32).contiguous()
    pool_rows = rows * max_pages * P
    kp = torch.empty((pool_rows, d), dtype=pre["k"].dtype, device=dev)
    vp = torch.empty_like(kp)
    qdec = torch.stack([inputs.decode_queries(cfg, s, device=dev, mu=pre["mu"])[0] for s in range(nsteps)])
    out = torch.empty((L, Hq, d), device=dev)
    ws = torch.empty(max(16, sg.decode_workspace_size(L, Hq, Hkv, d, max_pages, P)), dtype=torch.uint8, device=dev)
    buf = StepBuffers.alloc(rows, rows * per)
    lanes = TwoLane()
    zeros = buf.zeros
    # speculative transfer: block importances from the window score (eq. 1)
    scores = torch.empty((L, Hkv, T), device=dev)
    cus = torch.tensor(pre["cu_seqlens"], dtype=torch.int32, device=dev)
    ws_score = torch.empty(sg.score_workspace_size(1, L, Hq, Hkv, d, W, N), dtype=torch.uint8, device=dev)
    sg.sg_score(pre["q_win"], pre["k"], cus, T, N, Hkv, scores, ws=ws_score)
    imp = torch.empty((1, L, M), device=dev)
    sg.sg_block_importance(scores, cus, T, M, imp)
    LM = L * M
    quota = sg.spec_quota(LM, ratio_bp)
    main = torch.cuda.current_stream()
    ev = _ev
    counts = torch.empty((nidx, 2, rows), dtype=torch.int32, device=dev)

    def run(mode, quota_blocks=quota, steps=nsteps, serving=False):
        # serving: the host waits for every step before it launches the next,
        # as a serving loop does (it needs the step's token), so the pusher's
        # completion checks see the device's progress
        reset()
        pusher = SpecPusher(src_k, src_v, imp.view(-1), 0, N, M, store_k, store_v, mask, quota_blocks) \
            if mode.startswith("speculative") else None
        torch.cuda.synchronize()
        t = []
        t_host = time.perf_counter()
        for s in range(steps):
            a, b = ev(), ev()
            a.record(main)
            if pusher is not None:
                pusher.commit_if_landed(main)
            if mode == "serial":
                sg.sg_split(row_off, idx[s].view(-1), mask.view(-1), base, mlen, 1, buf.local, buf.remote,
                            buf.n_local, buf.n_remote, out_index=buf.order, n_kept=buf.n_kept)
                sg.sg_fetch(row_off, rows * per, buf.local, buf.n_local, base, store_k, store_v, page_table, P,
                            buf.n_remote, kp, vp)
                sg.sg_fetch_keep(row_off, rows * per, buf.remote, buf.n_remote, base, src_k, src_v, page_table, P,
                                 zeros, kp, vp, base, store_k, store_v, mask.view(-1), base, mlen)
            else:
                lanes.gather(row_off=row_off, kv_index=idx[s].view(-1), mask=mask.view(-1), mask_off=base,
                             mask_len=mlen, store_k=store_k, store_v=store_v, store_base=base, src_k=src_k,
                             src_v=src_v, src_base=base, page_table=page_table, page_size=P, k_pool=kp, v_pool=vp,
                             buf=buf, reuse=mode != "two_lane_no_reuse")
            if pusher is not None:
                pusher.launch_if_idle(main)
            sg.sg_decode_attn(qdec[s % nsteps], kp, vp, page_table.view(L, Hkv, max_pages), buf.n_kept, P, out,
                              ws=ws)
            b.record(main)
            counts[s, 0].copy_(buf.n_remote)
            counts[s, 1].copy_(buf.n_kept)
            t.append((a, b))
            if serving:
                b.synchronize()
        torch.cuda.synchronize()
        c = counts[:steps].double().sum(dim=2).cpu().numpy()
        ratio = c[:, 0] / c[:, 1]
        ms_steps = [a.elapsed_time(b) for a, b in t]
        res = {"steps": steps, "ms_per_step": round(float(np.median(ms_steps[1:])), 3),
               "ms_first": round(ms_steps[0], 3), "ms_total": round(float(np.sum(ms_steps)), 2)}
        if steps <= 16:
            res.update({"ms_steps": [round(x, 3) for x in ms_steps],
                        "on_demand_ratio": [r4(x) for x in ratio], "remote_rows_per_step": [int(x) for x in c[:, 0]]})
        else:
            marks = sorted({0, 1, 5, 10, 20, 50, 100, steps // 2, steps - 1} & set(range(steps)))
            res.update({"ms_at_step": {str(i): round(ms_steps[i], 3) for i in marks},
                        "on_demand_ratio_at_step": {str(i): r4(ratio[i]) for i in marks},
                        "on_demand_ratio_mean": r4(ratio.mean())})
        if pusher is not None:
            res.update({"pushes_done": pusher.pushes, "blocks_left": pusher.left})
        if serving:
            res["ms_total_host_clock"] = round((time.perf_counter() - t_host) * 1e3, 2)
        return res

    res = {"workload": cfg.name, "steps": nsteps, "rows_per_unit": per, "selected": kb, "extras": e}
    for mode in ("serial", "two_lane", "two_lane_no_reuse", "speculative"):
        res[mode] = run(mode)
    res["speculative"]["ratio_bp"] = ratio_bp
    res["speculative"]["blocks_per_push"] = quota
    res["speculative"]["pushes_to_complete"] = -(-LM // quota)
    # the workload's whole decode: two lanes with reuse, without and with
    # speculative transfer, cumulative time over every step
    res["over_all_steps"] = {"two_lane": run("two_lane", steps=long_steps, serving=True),
                             "speculative": run("speculative", steps=long_steps, serving=True),
                             "note": "the host waits for each step before launching the next (a serving loop)"}
    a, b2 = res["over_all_steps"]["two_lane"]["ms_total"], res["over_all_steps"]["speculative"]["ms_total"]
    res["over_all_steps"]["speculative_speedup"] = round(a / b2, 3)
    # lane rates and interference, each on its own
    reset()
    torch.cuda.synchronize()
    sg.sg_split(row_off, idx[1].view(-1), mask.view(-1), base, mlen, 1, buf.local, buf.remote, buf.n_local,
                buf.n_remote, out_index=buf.order, n_kept=buf.n_kept)
    torch.cuda.synchronize()
    n_loc = int(buf.n_local.sum().item())
    n_rem = int(buf.n_remote.sum().item())
    rowb = 2 * d * pre["k"].element_size()
    t_loc = median_ms(lambda i: sg.sg_fetch(row_off, rows * per, buf.local, buf.n_local, base, store_k, store_v,
                                            page_table, P, buf.n_remote, kp, vp))
    t_rem = median_ms(lambda i: sg.sg_fetch(row_off, rows * per, buf.remote, buf.n_remote, base, src_k, src_v,
                                            page_table, P, zeros, kp, vp))
    t_dec = median_ms(lambda i: sg.sg_decode_attn(qdec[1], kp, vp, page_table.view(L, Hkv, max_pages), buf.n_kept, P,
                                                  out, ws=ws))
    # decode attention alone and beside a speculative push on another stream
    rem = imp.view(-1).clone()
    ids = torch.empty(quota, dtype=torch.int32, device=dev)
    cu_row = torch.tensor([0, LM], dtype=torch.int32, device=dev)
    cu_q = torch.tensor([0, quota], dtype=torch.int32, device=dev)
    sg.sg_topk(rem.view(1, 1, LM), cu_row, LM, LM, cu_q, quota, ids.view(1, 1, quota))
    spec_stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    f0, f1, s0, s1 = ev(), ev(), ev(), ev()
    s0.record(spec_stream)
    sg.sg_spec_push(src_k, src_v, ids, 0, N, M, store_k, store_v, mask, None, stream=spec_stream)
    s1.record(spec_stream)
    f0.record(main)
    for r in range(10):
        sg.sg_decode_attn(qdec[r % nsteps], kp, vp, page_table.view(L, Hkv, max_pages), buf.n_kept, P, out, ws=ws)
    f1.record(main)
    torch.cuda.synchronize()
    t_dec_busy = f0.elapsed_time(f1) / 10
    t_push = s0.elapsed_time(s1)
    Nb = -(-N // M)
    push_bytes = quota * Hkv * Nb * rowb
    res["lanes"] = {"local_rows": n_loc, "local_ms": r4(t_loc), "local_gbs": round(gbs(n_loc * rowb * 2, t_loc), 1),
                    "remote_rows": n_rem, "remote_ms": r4(t_rem),
                    "remote_host_link_gbs": round(gbs(n_rem * rowb, t_rem), 1), "decode_ms": r4(t_dec)}
    res["spec_push"] = {"blocks": quota, "mb": round(push_bytes / 1e6, 1), "ms": round(t_push, 3),
                        "host_link_gbs": round(gbs(push_bytes, t_push), 1),
                        "decode_ms_alone": r4(t_dec), "decode_ms_beside_push": r4(t_dec_busy),
                        "decode_slowdown": round(t_dec_busy / t_dec, 3)}
    del pre, src_k, src_v, store_k, store_v
    torch.cuda.synchronize()
    return res


def selectors(sg, cfg, pre, cus, cuk, T, N, K_total, idx_score, nsteps=8, alpha=5.0, cap_bp=2000):
    """Selector variants on the request of the 8B 8K workload: the alpha-rule
    and top-20% selection-frequency scores (Section 4.1 importance under either
    Section 5.1 selector) and decode-time dynamic selection (Section 2.3; alpha
    5, at most 20% of the tokens), each timed on its own; then the on-demand
    ratio (Section 3: entries the decode step selects that were not sent at
    prefill) seen by that decode-time selector over `nsteps` steps, for five
    proactive choices of the same budget: top-k of the window score, top-k of
    either selector's counts, the first tokens, and a random set."""
    import numpy as np
    import torch
    from datagen import inputs

    dev = "cuda"
    L, Hq, Hkv, d, W = cfg.L, cfg.Hq, cfg.Hkv, cfg.d, cfg.W
    esize = pre["k"].element_size()
    units = L * Hkv
    counts = torch.empty((L, Hkv, T), device=dev)
    ws = torch.empty(sg.score_workspace_size(1, L, Hq, Hkv, d, W, N), dtype=torch.uint8, device=dev)
    t_count = median_ms(lambda i: sg.sg_score_count(pre["q_win"], pre["k"], cus, T, N, Hkv, counts, alpha, ws))
    idx_count = torch.empty_like(idx_score)
    sg.sg_topk(counts, cus, T, N, cuk, K_total, idx_count)
    # the other Section 5.1 selector: each window row picks its top 20%
    ts_counts = torch.empty((L, Hkv, T), device=dev)
    ws_ts = torch.empty(sg.score_topshare_workspace_size(1, L, Hq, Hkv, d, W, N), dtype=torch.uint8, device=dev)
    t_ts = median_ms(lambda i: sg.sg_score_topshare(pre["q_win"], pre["k"], cus, T, N, Hkv, ts_counts, cap_bp, ws_ts))
    idx_ts = torch.empty_like(idx_score)
    sg.sg_topk(ts_counts, cus, T, N, cuk, K_total, idx_ts)
    # logit passes: one per digit (6 bits, 5 above 256 rows) until 18 bits, the
    # gather, the count; rows with large bins (ties) take the remaining digits
    db = 6 if cfg.G * W <= 256 else 5
    ts_gather_after = -(-18 // db)
    ts_passes = {"when_every_row_gathers": ts_gather_after + 2, "at_most": -(-32 // db) + 2}
    cap = N * cap_bp // 10000
    cu_cap = torch.tensor([0, cap], dtype=torch.int32, device=dev)
    ws_sel = torch.empty(sg.decode_select_workspace_size(1, L, Hq, N), dtype=torch.uint8, device=dev)
    idx_dec = torch.empty((L, Hkv, cap), dtype=torch.int32, device=dev)
    n_sel = torch.empty((1, L, Hkv), dtype=torch.int32, device=dev)
    qs = [inputs.decode_queries(cfg, s, device=dev, mu=pre["mu"]) for s in range(nsteps)]     # [1][L][Hq][d]
    t_sel = median_ms(lambda i: sg.sg_decode_select(qs[0], pre["k"], cus, T, N, Hkv, cu_cap, cap, idx_dec, n_sel,
                                                    alpha, ws_sel))
    # InfiniGen's partial ratio 0.3: 40 of the 128 channels (here the first 40;
    # the paper's selector picks them with skewing matrices from the weights),
    # kept as a contiguous partial-key cache, with the full head's scale
    dp = 40
    k_part = pre["k"][..., :dp].contiguous()
    qp = [x[..., :dp].contiguous() for x in qs]
    t_sel_p = median_ms(lambda i: sg.sg_decode_select(qp[0], k_part, cus, T, N, Hkv, cu_cap, cap, idx_dec, n_sel,
                                                      alpha, ws_sel, scale=d ** -0.5))
    kp_bytes = units * N * dp * esize
    score_flops = 2.0 * d * cfg.G * (W * N - W * (W - 1) / 2) * units
    k_bytes = units * N * d * esize
    # on-demand ratio by proactive choice
    seq = torch.arange(K_total, device=dev, dtype=torch.int32).expand(L, Hkv, K_total).contiguous()
    rnd = inputs.random_selection(cfg, [N], [K_total], device=dev, tag_extra=7)
    row_off = (torch.arange(units + 1, device=dev) * cap).to(torch.int32)
    mask_off = torch.arange(units, device=dev, dtype=torch.int64) * N
    mask_len = torch.full((units,), N, dtype=torch.int32, device=dev)
    loc = torch.empty(units * cap, dtype=torch.int32, device=dev)
    rem = torch.empty_like(loc)
    nl = torch.empty(units, dtype=torch.int32, device=dev)
    nr = torch.empty_like(nl)
    nk = torch.empty_like(nl)
    ratios = {}
    sel_frac = []
    for name, sel, partial in (("score", idx_score, False), ("count", idx_count, False),
                               ("topshare_count", idx_ts, False),
                               ("sequential", seq, False), ("random", rnd, False),
                               ("score_partial_selector", idx_score, True)):
        mask = torch.full((units, N), 2, dtype=torch.int8, device=dev)
        mask.scatter_(1, sel.view(units, K_total).long(), 1)
        rs = []
        for s in range(nsteps):
            if partial:
                sg.sg_decode_select(qp[s], k_part, cus, T, N, Hkv, cu_cap, cap, idx_dec, n_sel, alpha, ws_sel,
                                    scale=d ** -0.5)
            else:
                sg.sg_decode_select(qs[s], pre["k"], cus, T, N, Hkv, cu_cap, cap, idx_dec, n_sel, alpha, ws_sel)
            sg.sg_split(row_off, idx_dec.view(-1), mask.view(-1), mask_off, mask_len, 0, loc, rem, nl, nr, n_kept=nk)
            rs.append(nr.sum().item() / max(1, nk.sum().item()))
            if name == "score":
                sel_frac.append(n_sel.float().mean().item() / N)
        ratios[name] = r4(np.mean(rs))
    return {"alpha": alpha, "count_score": {"ms": r4(t_count), "tflops": round(score_flops / (t_count * 1e-3) / 1e12, 1),
                                            "frac_mfma_peak": r4(score_flops / (t_count * 1e-3) / 1e12
                                                                 / BF16_MFMA_PEAK_TFLOPS)},
            "topshare_score": {"ratio_bp": cap_bp, "ms": r4(t_ts), "logit_passes": ts_passes,
                               "tflops_one_contraction": round(score_flops / (t_ts * 1e-3) / 1e12, 1),
                               "note": "each pass recomputes the logits; a unit with no row left to resolve "
                                       "returns at the start of the remaining radix passes"},
            "decode_select": {"ms": r4(t_sel), "cap": cap, "k_read_gbs": round(gbs(k_bytes, t_sel), 1),
                              "frac_hbm_peak": r4(gbs(k_bytes, t_sel) / HBM_PEAK_GBS),
                              "selected_fraction": r4(np.mean(sel_frac))},
            "decode_select_partial_40_of_128": {"ms": r4(t_sel_p), "k_read_gbs": round(gbs(kp_bytes, t_sel_p), 1),
                                                "frac_hbm_peak": r4(gbs(kp_bytes, t_sel_p) / HBM_PEAK_GBS)},
            "on_demand_ratio_by_proactive_choice": ratios, "budget_k": K_total, "steps": nsteps}


# --------------------------------------------------------------------------- counters

def sources_sha256(paths) -> str:
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(_ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _summary_figure(path, key):
    """A figure of a committed profile summary, or None when the summary is
    missing or the decode kernel's sources changed since it was taken."""
    import re
    try:
        with open(path) as f:
            text = f.read()
    except OSError:
        return None
    h = re.search(r"^kernel_sources_sha256:\s*([0-9a-f]{64})\s*$", text, re.M)
    t = re.search(r"^" + key + r":\s*([0-9.]+)\s*$", text, re.M)
    if not h or not t or h.group(1) != sources_sha256(TRAFFIC_SOURCES):
        return None
    return float(t.group(1))


def measured_traffic():
    """HBM bytes per decode launch from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, each scaled by a plain copy's reading)."""
    v = _summary_figure(TRAFFIC_SUMMARY, "traffic_bytes_per_launch")
    return None if v is None else int(v)


# --------------------------------------------------------------------------- oracle baseline

def cpu_inputs(p: Path):
    """Host copies of the oracle's samples, taken from the seeded inputs (never
    from a GPU result):
      select half - request 0, every layer and KV head;
      decode half - layer 0 of decode step 0 for every request and KV head,
                    attending over a seeded random selection of k_b rows plus
                    the e_b extras drawn from its complement (the workload's
                    sizes), gathered into a contiguous float32 pool."""
    import numpy as np
    import torch
    from datagen import inputs
    c = p.cfg
    n0 = p.lens[0]
    q0 = p.pre["q_win"][:1].float().cpu().numpy()
    lk = 1 if c.kv_shared_layers else c.L
    k0 = p.pre["k"][:lk, :, :n0].float().cpu().numpy()
    u16 = lambda t: t.cpu().contiguous().view(torch.int16).numpy().view(np.uint16)  # noqa: E731
    kraw0 = u16(p.pre["k"][:lk, :, :n0])
    vraw0 = u16(p.pre["v"][:lk, :, :n0])
    sel = inputs.random_selection(c.with_(L=1), p.lens, p.kb, device=p.idx.device, tag_extra=11)[0]   # [Hkv][K]
    ex, cu_e = inputs.extras_layer(c, 0, p.lens, sel, p.cu_k, 0)
    kf = p.pre["k"][0].float()                  # [Hkv][T][d] (layer 0's source)
    vf = p.pre["v"][0].float()
    rows_k, rows_v, n_rows = [], [], np.zeros((p.B, c.Hkv), np.int32)
    for b in range(p.B):
        for h in range(c.Hkv):
            ids = torch.cat([ex[h, cu_e[b]:cu_e[b + 1]], sel[h, p.cu_k[b]:p.cu_k[b + 1]]]).long() + p.pre["cu_seqlens"][b]
            rows_k.append(kf[h, ids])
            rows_v.append(vf[h, ids])
            n_rows[b, h] = ids.numel()
    P = c.page_size
    per = -(-int(n_rows.max()) // P) * P
    kp = np.zeros((p.B * c.Hkv * per, c.d), np.float32)
    vp = np.zeros_like(kp)
    for u, (rk, rv) in enumerate(zip(rows_k, rows_v)):
        kp[u * per:u * per + rk.shape[0]] = rk.cpu().numpy()
        vp[u * per:u * per + rv.shape[0]] = rv.cpu().numpy()
    npg = per // P
    pt = ((np.arange(p.B * c.Hkv)[:, None] * per + np.arange(npg)[None, :] * P).astype(np.int32)
          .reshape(p.B, c.Hkv, npg))
    qd = p.qdec[0][0].float().cpu().numpy()     # layer 0: [B][Hq][d]
    return {"q0": q0, "k0": k0, "kraw0": kraw0, "vraw0": vraw0, "n0": n0, "k_b0": p.kb[0],
            "dec": (qd, kp, vp, pt, n_rows, P), "dec_rows": int(n_rows.sum()), "esize": p.esize}


def cpu_baseline(cfg, s, min_seconds):
    """The oracle timed on the host cores on the bounded samples of cpu_inputs,
    each repeated until at least `min_seconds` have passed; reported in the
    metric's units (select+pack GB/s of KV cache, decode tokens/s)."""
    import numpy as np

    import oracle
    if not os.path.exists(oracle.LIB_PATH):
        from oracle import build as ob
        ob.build()
    threads = oracle.threads()
    cu = [0, s["n0"]]
    ck = [0, s["k_b0"]]
    units = cfg.L * cfg.Hkv

    def select_once():
        sc = oracle.score(s["q0"], s["k0"], cu, cfg.Hkv)
        ix = oracle.topk(sc.astype(np.float32), cu, ck)
        oracle.pack(s["kraw0"], s["vraw0"], ix, cu, ck, kv_layer_rows=0 if cfg.kv_shared_layers else None)

    def decode_once():
        oracle.decode_attn(*s["dec"])

    def timed(fn, seconds=min_seconds):
        reps = 0
        t0 = time.perf_counter()
        while True:
            fn()
            reps += 1
            if time.perf_counter() - t0 >= seconds:
                break
        return (time.perf_counter() - t0) / reps, reps

    dt, reps = timed(select_once)
    kv_bytes = 2 * units * s["n0"] * cfg.d * s["esize"]
    ddt, dreps = timed(decode_once)
    # one thread, on a slice of the same samples: the select half for layer 0's
    # KV heads, the decode half as above
    q1, k1, kr1, vr1 = s["q0"][:, :1], s["k0"][:1], s["kraw0"][:1], s["vraw0"][:1]

    def select_one_layer():
        sc = oracle.score(q1, k1, cu, cfg.Hkv)
        ix = oracle.topk(sc.astype(np.float32), cu, ck)
        oracle.pack(kr1, vr1, ix, cu, ck)

    oracle.set_threads(1)
    try:
        dt1, reps1 = timed(select_one_layer, min_seconds / 4)
        ddt1, dreps1 = timed(decode_once, min_seconds / 4)
    finally:
        oracle.set_threads(threads)
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    cpu = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    dec_bytes = s["dec_rows"] * 2 * cfg.d * s["esize"]
    B = s["dec"][4].shape[0]
    return {"value": round(kv_bytes / dt / 1e9, 4), "unit": "GB/s", "cores": min(threads, units), "kind": "oracle",
            "seconds_per_pass": round(dt, 3), "passes": reps,
            "sample": f"score+topk+pack of request 0 ({s['n0']} tokens), all {cfg.L} layers x {cfg.Hkv} KV heads "
                      f"({units} units); fp64 C oracle, OpenMP over units, repeated {reps}x",
            "decode": {"tokens_per_s": round(B / (ddt * cfg.L), 2), "gbs": round(dec_bytes / ddt / 1e9, 4),
                       "seconds_per_pass": round(ddt, 3), "passes": dreps,
                       "sample": f"decode attention of layer 0, decode step 0, all {B} requests x {cfg.Hkv} KV heads "
                                 f"({s['dec_rows']} rows: seeded selection + extras at the workload's sizes); "
                                 f"tokens/s = requests / (seconds per layer x {cfg.L} layers)"},
            "single_thread": {"value": round(2 * cfg.Hkv * s["n0"] * cfg.d * s["esize"] / dt1 / 1e9, 4),
                              "unit": "GB/s", "seconds_per_pass": round(dt1, 3), "passes": reps1,
                              "decode_tokens_per_s": round(B / (ddt1 * cfg.L), 2),
                              "decode_seconds_per_pass": round(ddt1, 3), "decode_passes": dreps1,
                              "sample": f"select half: layer 0's {cfg.Hkv} KV heads of request 0; decode half: "
                                        "the decode sample above; one OpenMP thread"},
            "cpu_model": cpu, "host": platform.node()}


if __name__ == "__main__":
    main()
