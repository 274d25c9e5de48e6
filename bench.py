"""Benchmark of the selective KV-transfer hot path on one MI355X.

One step = one pass of the whole path over one request of the Llama-3-8B-shaped
workload (32 layers, 32 q heads / 8 KV heads, d = 128, bf16, 8192-token prompt,
64-query score window, 10% budget, 128 decode steps):

  prefill side   sg_score -> sg_topk -> sg_pack (transfer buffer in HBM)
  decode side    128 x [ sg_split (Algorithm 1 on the step's KV index)
                         -> sg_decode_attn over the selected rows of all 32
                            layers, batched as 32 sequences ]

Inputs are generated on the GPU before timing.  The decode reads rotate over
several replicas of the transfer buffer so the working set exceeds the 256 MB
last-level cache (a real decode step streams the model weights between layers).

Prints one JSON line.  ``value`` is select+pack throughput: bytes of the KV
cache (K and V of every layer and head) turned into a transfer buffer per
second of score + top-k + pack time.  The decode rate is reported as
``decode_tokens_per_s``; the roofline object covers the dominant kernel
(sparse decode attention).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
import sys
import time

_ROOT = os.path.dirname(os.path.abspath(__file__))
if _ROOT not in sys.path:
    sys.path.insert(0, _ROOT)

HBM_PEAK_GBS = 8000.0
# the counter summary that gives the decode kernel's measured HBM traffic, and
# the sources whose hash it records (a changed kernel makes the figure stale)
TRAFFIC_SUMMARY = os.path.join(_ROOT, "profiles", "all_kernels.llama8b_8k.hbm_traffic.md")
TRAFFIC_SOURCES = ("paper_2607_28150_amd/csrc/decode_attn.hip", "paper_2607_28150_amd/csrc/sg_internal.h")
BF16_MFMA_PEAK_TFLOPS = 2500.0
FP32_MFMA_PEAK_TFLOPS = 157.3


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=5)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--workload", default="llama8b_8k")
    p.add_argument("--decode-steps", type=int, default=None, help="decode steps per step (default: workload's)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-decode-side", action="store_true", help="skip the 32K-token decode-side section")
    p.add_argument("--only", choices=["decode_side"], default=None,
                   help="run one section on its own and print its JSON line (profiling one workload)")
    p.add_argument("--cpu-layers", type=int, default=0, help="layers the oracle is timed on (0 = all)")
    p.add_argument("--cpu-seconds", type=float, default=10.0, help="repeat the oracle sample to at least this long")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="only run a plain device copy of MIB MiB three times (counter calibration) and exit")
    return p.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
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

    from datagen import inputs
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
    dev = "cuda"
    cfg = get(args.workload)
    assert cfg.B == 1 and cfg.extra_bp == 0, "the bench step covers single-request workloads without extras"
    nsteps_dec = cfg.steps if args.decode_steps is None else args.decode_steps
    L, Hq, Hkv, d, W, G = cfg.L, cfg.Hq, cfg.Hkv, cfg.d, cfg.W, cfg.G

    # ------------------------------------------------------------- inputs (resident in HBM)
    t0 = time.time()
    pre = inputs.make_prefill(cfg, device=dev)
    lens, T = pre["seqlens"], pre["T"]
    N = lens[0]
    bud = inputs.make_budget(cfg, lens)
    K_total = bud["K_total"]
    cus = torch.tensor(pre["cu_seqlens"], dtype=torch.int32, device=dev)
    cuk = torch.tensor(bud["cu_k"], dtype=torch.int32, device=dev)
    qdec = torch.stack([inputs.decode_queries(cfg, s, device=dev, mu=pre["mu"])[0] for s in range(nsteps_dec)])
    qdec = qdec.contiguous()                                           # [steps][L][Hq][d]
    esize = 2 if cfg.dtype == "bf16" else 4
    S = L * Hkv * K_total
    nbytes = sg.pack_bytes(pre["k"].dtype, L, Hkv, d, K_total)
    reps = max(2, math.ceil(640e6 / nbytes))
    bufs = [torch.empty(nbytes, dtype=torch.uint8, device=dev) for _ in range(reps)]
    scores = torch.empty((L, Hkv, T), device=dev)
    idx = torch.empty((L, Hkv, K_total), dtype=torch.int32, device=dev)
    ws_score = torch.empty(sg.score_workspace_size(1, L, Hq, Hkv, d, W, N), dtype=torch.uint8, device=dev)
    P = cfg.page_size
    npg = (K_total + P - 1) // P
    units = L * Hkv
    # decode: sequence = layer; unit (l, h) rows are slots (l*Hkv + h)*K_total + i of the K / V regions
    page_table = (torch.arange(units, device=dev)[:, None] * K_total
                  + torch.arange(npg, device=dev)[None, :] * P).to(torch.int32).view(L, Hkv, npg).contiguous()
    n_rows = torch.full((L, Hkv), K_total, dtype=torch.int32, device=dev)
    ws_dec = torch.zeros(max(sg.decode_workspace_size(L, Hq, Hkv, d, npg, P), 16), dtype=torch.uint8, device=dev)
    out = torch.empty((L, Hq, d), device=dev)
    pools = []
    for b in bufs:
        kp = b[: S * d * esize].view(pre["k"].dtype).view(S, d)
        vp = b[S * d * esize: 2 * S * d * esize].view(pre["k"].dtype).view(S, d)
        pools.append((kp, vp))
    # Algorithm 1 inputs: every selected row is local (mask 1) in this workload
    split_rows = units
    row_off = (torch.arange(split_rows + 1, device=dev) * K_total).to(torch.int32)
    mask = torch.ones((units, N), dtype=torch.int8, device=dev)
    mask_off = (torch.arange(units, device=dev, dtype=torch.int64) * N)
    mask_len = torch.full((units,), N, dtype=torch.int32, device=dev)
    sp_local = torch.empty(S, dtype=torch.int32, device=dev)
    sp_remote = torch.empty(S, dtype=torch.int32, device=dev)
    sp_order = torch.empty(S, dtype=torch.int32, device=dev)
    sp_nl = torch.empty(split_rows, dtype=torch.int32, device=dev)
    sp_nr = torch.empty(split_rows, dtype=torch.int32, device=dev)
    # row log-sum-exp of the window queries, as a prefill attention kernel
    # leaves it behind (here: plain fp32 torch on the GPU, before timing); it
    # feeds the one-pass score measured beside the self-contained one
    lse_win = window_lse(pre["q_win"], pre["k"], N, Hkv, W, d)
    torch.cuda.synchronize()
    setup_s = time.time() - t0

    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    decode = sg.DecodeCall(qdec[0], pools[0][0], pools[0][1], page_table, n_rows, P, out, ws=ws_dec)
    ev_pool = [[ev() for _ in range(6)] for _ in range(args.steps)]

    # one step: score, top-k, pack; Algorithm 1 on the step's KV index (the
    # selected set, all local in this workload, so once per request); then the
    # decode steps, each one attention launch over all layers.  The decode
    # launches run back to back between two events (an event between every
    # launch would add its own marker to each measured interval).
    # (events mark only the ends of the select region, the split and the
    # decode launches; each op's own time is measured apart, below)
    def step(r, e):
        if e is None:
            e = [None] * 6
        rec = lambda i: e[i].record() if e[i] is not None else None  # noqa: E731
        rec(0)
        sg.sg_score(pre["q_win"], pre["k"], cus, T, N, Hkv, scores, ws=ws_score)
        sg.sg_topk(scores, cus, T, N, cuk, K_total, idx)
        sg.sg_pack(pre["k"], pre["v"], idx, cus, T, cuk, K_total, K_total, bufs[r % reps])
        rec(3)
        sg.sg_split(row_off, idx.view(-1), mask.view(-1), mask_off, mask_len, 1, sp_local, sp_remote, sp_nl,
                    sp_nr, out_index=sp_order)
        rec(4)
        for s in range(nsteps_dec):
            kp, vp = pools[(r + s) % reps]
            decode(qdec[s], kp, vp, out)
        rec(5)

    # every replica holds a packed buffer before timing
    for r in range(reps):
        step(r, None)
    for w in range(args.warmup):
        step(w, None)
    torch.cuda.synchronize()

    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        step(k, ev_pool[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start

    # each op of the select region on its own (back-to-back launches), and the
    # one-pass score (row normalisers supplied)
    nrep = 10

    def per_launch(fn):
        fn()
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record()
        for i in range(nrep):
            fn(i)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / nrep

    t_score = per_launch(lambda i=0: sg.sg_score(pre["q_win"], pre["k"], cus, T, N, Hkv, scores, ws=ws_score))
    t_topk = per_launch(lambda i=0: sg.sg_topk(scores, cus, T, N, cuk, K_total, idx))
    t_pack = per_launch(lambda i=0: sg.sg_pack(pre["k"], pre["v"], idx, cus, T, cuk, K_total, K_total,
                                               bufs[i % reps]))
    t_score_lse = per_launch(lambda i=0: sg.sg_score(pre["q_win"], pre["k"], cus, T, N, Hkv, scores, ws=ws_score,
                                                     lse_in=lse_win))

    # the on-box reference: a plain device-to-device copy of the decode step's
    # byte count, over rotating buffers so that the last-level cache cannot serve it
    copy_bytes = 2 * S * d * esize
    copy_src = [torch.empty(copy_bytes, dtype=torch.uint8, device=dev).fill_(1) for _ in range(6)]
    copy_dst = [torch.empty(copy_bytes, dtype=torch.uint8, device=dev) for _ in range(6)]
    t_copy = min(per_launch(lambda i=0: copy_dst[i % 6].copy_(copy_src[(i + 3) % 6])) for _ in range(3))
    copy_gbs = 2 * copy_bytes / (t_copy * 1e-3) / 1e9             # bytes read + written
    del copy_src, copy_dst

    # the decode step as a model runs it: one launch per layer, in a HIP graph
    dec_layers = per_layer_mode(sg, qdec[0], pools[0][0], pools[0][1], page_table, n_rows, P)

    # block-granular proactive selection (eq. 1, eq. 2; M = 1024 blocks per
    # layer, transfer time 6.5x the prefill time), timed on its own
    blk = block_mode(sg, scores, cus, T, N, L, Hkv, d, pre, esize)

    # selector variants: alpha-rule counts, decode-time selection, on-demand ratio
    sel_ops = selectors(sg, cfg, pre, cus, cuk, T, N, K_total, idx)

    # the decode side of the 32K-token workload: two lanes, reuse, speculative transfer
    dside = None if args.no_decode_side else decode_side(sg)

    # ------------------------------------------------------------- per-op times (HIP events on the launch stream)
    def ms(a, b):
        return a.elapsed_time(b)
    t_select = np.mean([ms(e[0], e[3]) for e in ev_pool])        # score + top-k + pack, back to back
    t_split = np.mean([ms(e[3], e[4]) for e in ev_pool])
    t_dec = np.mean([ms(e[4], e[5]) for e in ev_pool]) / nsteps_dec
    ms_per_step = wall * 1e3 / args.steps

    kv_bytes = 2 * L * Hkv * T * d * esize                       # the whole KV cache
    sel_ms = t_select
    value = kv_bytes / (sel_ms * 1e-3) / 1e9
    score_flops = 2.0 * d * G * (W * N - W * (W - 1) / 2) * units
    pack_bytes_alg = 2 * S * d * esize * 2 + S * 4 * 2          # rows read + written, index read + written
    dec_bytes = (2 * S * d * esize + L * Hq * d * esize + L * Hq * d * 4 + page_table.numel() * 4
                 + n_rows.numel() * 4)
    dec_gbs = dec_bytes / (t_dec * 1e-3) / 1e9
    tokens_per_s = 1.0 / (t_dec * 1e-3)                          # one token of one request per decode step
    peak_mfma = BF16_MFMA_PEAK_TFLOPS if cfg.dtype == "bf16" else FP32_MFMA_PEAK_TFLOPS
    ops = {
        "score": {"ms": round(t_score, 4), "tflops": round(score_flops / (t_score * 1e-3) / 1e12, 2),
                  "frac_mfma_peak": round(score_flops / (t_score * 1e-3) / 1e12 / peak_mfma, 4),
                  "gflop_algorithmic": round(score_flops / 1e9, 2)},
        "score_lse_in": {"ms": round(t_score_lse, 4),
                         "tflops": round(score_flops / (t_score_lse * 1e-3) / 1e12, 2),
                         "frac_mfma_peak": round(score_flops / (t_score_lse * 1e-3) / 1e12 / peak_mfma, 4),
                         "note": "one pass: row normalisers supplied by the prefill attention"},
        "block_mode": blk,
        "decode_side": dside,
        "selectors": sel_ops,
        "topk": {"ms": round(t_topk, 4),
                 "gbs": round((scores.numel() * 4 + idx.numel() * 4) / (t_topk * 1e-3) / 1e9, 1)},
        "pack": {"ms": round(t_pack, 4), "gbs": round(pack_bytes_alg / (t_pack * 1e-3) / 1e9, 1),
                 "frac_hbm_peak": round(pack_bytes_alg / (t_pack * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                 "frac_measured_copy": round(pack_bytes_alg / (t_pack * 1e-3) / 1e9 / copy_gbs, 4),
                 "mb_algorithmic": round(pack_bytes_alg / 1e6, 2)},
        "split": {"ms": round(t_split, 4)},
        "decode_attn": {"ms": round(t_dec, 4), "gbs": round(dec_gbs, 1),
                        "frac_hbm_peak": round(dec_gbs / HBM_PEAK_GBS, 4),
                        "frac_measured_copy": round(dec_gbs / copy_gbs, 4),
                        "mb_algorithmic": round(dec_bytes / 1e6, 2)},
        "decode_attn_per_layer": dec_layers,
        "measured_copy": {"gbs": round(copy_gbs, 1), "ms": round(t_copy, 4), "mb": round(copy_bytes / 1e6, 2),
                          "note": "device-to-device copy (bytes read + written) over six rotating buffer pairs; "
                                  "the fractions named frac_measured_copy are against it"},
    }
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
        "config": {"workload": cfg.name, "layers": L, "q_heads": Hq, "kv_heads": Hkv, "head_dim": d,
                   "prompt": N, "score_window": W, "budget_bp": cfg.budget_bp, "k": K_total,
                   "decode_steps": nsteps_dec, "page_size": P, "transfer_replicas": reps},
        "select_ms": round(t_select, 4),
        "value_lse_in": round(kv_bytes / ((t_select - t_score + t_score_lse) * 1e-3) / 1e9, 2),
        "decode_tokens_per_s": round(tokens_per_s, 1),
        "roofline": {"kernel": "sg_decode_attn", "bound": "hbm", "achieved": round(dec_gbs, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(dec_gbs / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(), "bytes_per_launch": dec_bytes,
                     "avg_launch_ms": round(t_dec, 5), "frac_measured_copy": round(dec_gbs / copy_gbs, 4)},
        "ops": ops,
        "setup_s": round(setup_s, 2),
    }

    # ------------------------------------------------------------- oracle on the host cores
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg, pre, bud, args.cpu_layers or cfg.L, args.cpu_seconds)
        if line["cpu_baseline"].get("value"):
            line["gpu_over_cpu"] = round(value / line["cpu_baseline"]["value"], 1)
    print(json.dumps(line), flush=True)


def block_mode(sg, scores, cus, T, N, L, Hkv, d, pre, esize, M=1024, ratio=1 / 6.5, nrep=10):
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
    dsts = [torch.empty(nbytes, dtype=torch.uint8, device=dev) for _ in range(2)]

    def run(i, ev=None):
        if ev:
            ev[0].record()
        sg.sg_block_importance(scores, cus, T, M, imp)
        if ev:
            ev[1].record()
        sg.sg_topk(imp.view(1, 1, L * M), cu_row, L * M, L * M, cu_kr, Kr, ids)
        if ev:
            ev[2].record()
        sg.sg_pack_blocks(pre["k"], pre["v"], ids.view(-1), 0, N, M, dsts[i % 2])
        if ev:
            ev[3].record()
    run(0)
    run(1)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(nrep)]
    for i in range(nrep):
        run(i, evs[i])
    torch.cuda.synchronize()
    t = [sum(e[j].elapsed_time(e[j + 1]) for e in evs) / nrep for j in range(3)]
    Nb = -(-N // M)
    rows = Kr * Hkv * Nb
    pack_bytes = 2 * 2 * rows * d * esize + 2 * Kr * 4                # rows read + written, ids read + written
    imp_bytes = L * Hkv * N * 4 + L * M * 4
    return {"M": M, "transfer_over_prefill": round(1 / ratio, 2), "K_r": Kr, "blocks": L * M,
            "importance_ms": round(t[0], 4), "importance_gbs": round(imp_bytes / (t[0] * 1e-3) / 1e9, 1),
            "topk_ms": round(t[1], 4),
            "pack_ms": round(t[2], 4), "pack_gbs": round(pack_bytes / (t[2] * 1e-3) / 1e9, 1),
            "pack_frac_hbm_peak": round(pack_bytes / (t[2] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "pack_mb_algorithmic": round(pack_bytes / 1e6, 2)}


def decode_side(sg, nsteps=12, ratio_bp=1000, M=1024):
    """Decode side of the 8B-shaped 32K-token workload (5% of the rows sent at
    prefill, 2% more fetched on demand per step, all 32 layers per step):
    Algorithm 1 and the two lanes of Section 4.2 (serial on one stream, or on
    two streams; with and without reuse of fetched rows), and speculative
    transfer (Section 4.3: the quota of remaining blocks pushed while the
    attention runs; the next step's split waits for it).  The prefill side's
    copy of K / V is pinned host memory, so the remote lane and the speculative
    push cross the host link; the decode side's store is in HBM."""
    import numpy as np
    import torch
    from datagen import inputs
    from datagen.configs import get
    from paper_2607_28150_amd.lanes import StepBuffers, TwoLane

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
    idx = torch.empty((nsteps, rows, per), dtype=torch.int32, device=dev)
    for s in range(nsteps):
        for l in range(L):
            ex = inputs.extras_for_step(cfg, s, lens, sel[l], bud["cu_k"], l)
            for h in range(Hkv):
                idx[s, l * Hkv + h, :e] = ex[h].to(torch.int32)
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
    rem = torch.empty(LM, device=dev)
    ids = torch.empty(quota, dtype=torch.int32, device=dev)
    cu_row = torch.tensor([0, LM], dtype=torch.int32, device=dev)
    spec_stream = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    counts = torch.empty((nsteps, 2, rows), dtype=torch.int32, device=dev)
    # top-k offsets of every push size, made before any stream uses them
    cu_q = {q: torch.tensor([0, q], dtype=torch.int32, device=dev) for q in {quota, LM % quota or quota}}

    def run(mode):
        reset()
        rem.copy_(imp.view(-1))
        left = LM
        torch.cuda.synchronize()
        t = []
        for s in range(nsteps):
            a, b = ev(), ev()
            a.record(main)
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
            if mode == "speculative" and left > 0:
                # the prefill side pushes the next blocks while the attention runs
                q = min(quota, left)
                go = torch.cuda.Event()
                go.record(main)
                spec_stream.wait_event(go)
                sg.sg_topk(rem.view(1, 1, LM), cu_row, LM, LM, cu_q[q], q, ids[:q].view(1, 1, q), stream=spec_stream)
                sg.sg_spec_push(src_k, src_v, ids[:q], 0, N, M, store_k, store_v, mask, rem, stream=spec_stream)
                left -= q
            sg.sg_decode_attn(qdec[s], kp, vp, page_table.view(L, Hkv, max_pages), buf.n_kept, P, out, ws=ws)
            if mode == "speculative":
                done = torch.cuda.Event()
                done.record(spec_stream)
                main.wait_event(done)
            b.record(main)
            counts[s, 0].copy_(buf.n_remote)
            counts[s, 1].copy_(buf.n_kept)
            t.append((a, b))
        torch.cuda.synchronize()
        c = counts.double().sum(dim=2).cpu().numpy()
        ratio = [round(float(x), 4) for x in c[:, 0] / c[:, 1]]
        ms_steps = [a.elapsed_time(b) for a, b in t]
        return {"ms_per_step": round(float(np.mean(ms_steps[1:])), 3), "ms_first": round(ms_steps[0], 3),
                "ms_steps": [round(x, 3) for x in ms_steps],
                "on_demand_ratio": ratio, "remote_rows_per_step": [int(x) for x in c[:, 0]]}

    res = {"workload": cfg.name, "steps": nsteps, "rows_per_unit": per, "selected": kb, "extras": e}
    for mode in ("serial", "two_lane", "two_lane_no_reuse", "speculative"):
        res[mode] = run(mode)
    res["speculative"]["ratio_bp"] = ratio_bp
    res["speculative"]["blocks_per_push"] = quota
    res["speculative"]["pushes_to_complete"] = -(-LM // quota)
    # lane rates and interference, each on its own
    reset()
    torch.cuda.synchronize()
    sg.sg_split(row_off, idx[1].view(-1), mask.view(-1), base, mlen, 1, buf.local, buf.remote, buf.n_local,
                buf.n_remote, out_index=buf.order, n_kept=buf.n_kept)
    torch.cuda.synchronize()
    n_loc = int(buf.n_local.sum().item())
    n_rem = int(buf.n_remote.sum().item())
    rowb = 2 * d * pre["k"].element_size()
    e0, e1, e2, e3 = ev(), ev(), ev(), ev()
    e0.record()
    sg.sg_fetch(row_off, rows * per, buf.local, buf.n_local, base, store_k, store_v, page_table, P, buf.n_remote,
                kp, vp)
    e1.record()
    sg.sg_fetch(row_off, rows * per, buf.remote, buf.n_remote, base, src_k, src_v, page_table, P, zeros, kp, vp)
    e2.record()
    sg.sg_decode_attn(qdec[1], kp, vp, page_table.view(L, Hkv, max_pages), buf.n_kept, P, out, ws=ws)
    e3.record()
    torch.cuda.synchronize()
    t_loc, t_rem, t_dec = e0.elapsed_time(e1), e1.elapsed_time(e2), e2.elapsed_time(e3)
    # decode attention alone and beside a speculative push on another stream
    rem.copy_(imp.view(-1))
    sg.sg_topk(rem.view(1, 1, LM), cu_row, LM, LM, cu_q[quota], quota, ids.view(1, 1, quota))
    torch.cuda.synchronize()
    f0, f1 = ev(), ev()
    s0, s1 = ev(), ev()
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
    g0, g1 = ev(), ev()
    g0.record()
    for r in range(10):
        sg.sg_decode_attn(qdec[r % nsteps], kp, vp, page_table.view(L, Hkv, max_pages), buf.n_kept, P, out, ws=ws)
    g1.record()
    torch.cuda.synchronize()
    t_dec_alone = g0.elapsed_time(g1) / 10
    Nb = -(-N // M)
    push_bytes = quota * Hkv * Nb * rowb
    res["lanes"] = {"local_rows": n_loc, "local_ms": round(t_loc, 4),
                    "local_gbs": round(n_loc * rowb * 2 / (t_loc * 1e-3) / 1e9, 1),
                    "remote_rows": n_rem, "remote_ms": round(t_rem, 4),
                    "remote_host_link_gbs": round(n_rem * rowb / (t_rem * 1e-3) / 1e9, 1),
                    "decode_ms": round(t_dec, 4)}
    res["spec_push"] = {"blocks": quota, "mb": round(push_bytes / 1e6, 1), "ms": round(t_push, 3),
                        "host_link_gbs": round(push_bytes / (t_push * 1e-3) / 1e9, 1),
                        "decode_ms_alone": round(t_dec_alone, 4), "decode_ms_beside_push": round(t_dec_busy, 4),
                        "decode_slowdown": round(t_dec_busy / t_dec_alone, 3)}
    del pre, src_k, src_v, store_k, store_v
    torch.cuda.synchronize()
    return res


def selectors(sg, cfg, pre, cus, cuk, T, N, K_total, idx_score, nsteps=8, alpha=5.0, cap_bp=2000, nrep=10):
    """Selector variants on the request of the main step: the alpha-rule
    selection-frequency score (Section 4.1 importance under the Section 5.1
    selector) and decode-time dynamic selection (Section 2.3; alpha 5, at most
    20% of the tokens), each timed on its own; then the on-demand ratio
    (Section 3: entries the decode step selects that were not sent at prefill)
    seen by that decode-time selector over `nsteps` steps, for four proactive
    choices of the same budget: top-k of the window score, top-k of the
    alpha-rule counts, the first tokens, and a random set."""
    import numpy as np
    import torch
    from datagen import inputs

    dev = "cuda"
    L, Hq, Hkv, d, W = cfg.L, cfg.Hq, cfg.Hkv, cfg.d, cfg.W
    esize = pre["k"].element_size()
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    units = L * Hkv

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record()
        for _ in range(nrep):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / nrep

    counts = torch.empty((L, Hkv, T), device=dev)
    ws = torch.empty(sg.score_workspace_size(1, L, Hq, Hkv, d, W, N), dtype=torch.uint8, device=dev)
    t_count = timed(lambda: sg.sg_score_count(pre["q_win"], pre["k"], cus, T, N, Hkv, counts, alpha, ws))
    idx_count = torch.empty_like(idx_score)
    sg.sg_topk(counts, cus, T, N, cuk, K_total, idx_count)
    cap = N * cap_bp // 10000
    cu_cap = torch.tensor([0, cap], dtype=torch.int32, device=dev)
    ws_sel = torch.empty(sg.decode_select_workspace_size(1, L, Hq, N), dtype=torch.uint8, device=dev)
    idx_dec = torch.empty((L, Hkv, cap), dtype=torch.int32, device=dev)
    n_sel = torch.empty((1, L, Hkv), dtype=torch.int32, device=dev)
    qs = [inputs.decode_queries(cfg, s, device=dev, mu=pre["mu"]) for s in range(nsteps)]     # [1][L][Hq][d]
    t_sel = timed(lambda: sg.sg_decode_select(qs[0], pre["k"], cus, T, N, Hkv, cu_cap, cap, idx_dec, n_sel, alpha,
                                              ws_sel))
    # InfiniGen's partial ratio 0.3: 40 of the 128 channels (here the first 40;
    # the paper's selector picks them with skewing matrices from the weights),
    # kept as a contiguous partial-key cache, with the full head's scale
    dp = 40
    k_part = pre["k"][..., :dp].contiguous()
    qp = [x[..., :dp].contiguous() for x in qs]
    t_sel_p = timed(lambda: sg.sg_decode_select(qp[0], k_part, cus, T, N, Hkv, cu_cap, cap, idx_dec, n_sel, alpha,
                                                ws_sel, scale=d ** -0.5))
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
                               ("sequential", seq, False), ("random", rnd, False), ("score_partial_selector", idx_score, True)):
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
        ratios[name] = round(float(np.mean(rs)), 4)
    return {"alpha": alpha, "count_score": {"ms": round(t_count, 4),
                                            "tflops": round(score_flops / (t_count * 1e-3) / 1e12, 2),
                                            "frac_mfma_peak": round(score_flops / (t_count * 1e-3) / 1e12
                                                                    / BF16_MFMA_PEAK_TFLOPS, 4)},
            "decode_select": {"ms": round(t_sel, 4), "cap": cap,
                              "k_read_gbs": round(k_bytes / (t_sel * 1e-3) / 1e9, 1),
                              "frac_hbm_peak": round(k_bytes / (t_sel * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                              "selected_fraction": round(float(np.mean(sel_frac)), 4)},
            "decode_select_partial_40_of_128": {"ms": round(t_sel_p, 4),
                                                "k_read_gbs": round(kp_bytes / (t_sel_p * 1e-3) / 1e9, 1),
                                                "frac_hbm_peak": round(kp_bytes / (t_sel_p * 1e-3) / 1e9
                                                                       / HBM_PEAK_GBS, 4)},
            "on_demand_ratio_by_proactive_choice": ratios, "budget_k": K_total, "steps": nsteps}


def window_lse(q_win, k, N, Hkv, W, d):
    """[1][L][Hq][W] natural-log LSE of the scaled causal logits of the window
    rows (row w sits at position N - W + w), in fp32 with torch."""
    import torch
    _, L, Hq, _, _ = q_win.shape
    G = Hq // Hkv
    out = torch.empty((1, L, Hq, W), dtype=torch.float32, device=q_win.device)
    pos = torch.arange(N - W, N, device=q_win.device)[:, None]
    late = torch.arange(N, device=q_win.device)[None, :] > pos          # [W][N] keys past the row
    for l in range(L):
        for h in range(Hkv):
            q = q_win[0, l, h * G:(h + 1) * G].float().reshape(G * W, d)
            kt = k[l, h].float().t().contiguous()                       # [d][N]
            z = (q @ kt) * (d ** -0.5)
            z = z.view(G, W, N).masked_fill(late, float("-inf"))
            out[0, l, h * G:(h + 1) * G] = torch.logsumexp(z, dim=-1)
    return out


def sources_sha256(paths) -> str:
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(_ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per decode launch from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, each scaled by a plain copy's reading), or None
    when the summary is missing or the kernel sources changed since."""
    import re
    try:
        with open(TRAFFIC_SUMMARY) as f:
            text = f.read()
    except OSError:
        return None
    h = re.search(r"^kernel_sources_sha256:\s*([0-9a-f]{64})\s*$", text, re.M)
    t = re.search(r"^traffic_bytes_per_launch:\s*([0-9]+)\s*$", text, re.M)
    if not h or not t or h.group(1) != sources_sha256(TRAFFIC_SOURCES):
        return None
    return int(t.group(1))


def per_layer_mode(sg, q, k_pool, v_pool, page_table, n_rows, P, nrep=20):
    """One decode step as a model runs it: one sg_decode_attn launch per layer
    (B = 1, the layer's KV heads), the layers in order, captured once in a HIP
    graph and replayed.  Every replay is checked bit for bit against the same
    launches made eagerly (with eager work between the replays) before it is
    timed."""
    import torch
    L, Hkv, npg = page_table.shape
    Hq, d = q.shape[1], q.shape[2]
    dev = q.device
    ws = torch.zeros(max(sg.decode_workspace_size(1, Hq, Hkv, d, npg, P), 16), dtype=torch.uint8, device=dev)
    out = torch.empty((L, Hq, d), device=dev)

    def layers():
        for l in range(L):
            sg.sg_decode_attn(q[l:l + 1], k_pool, v_pool, page_table[l:l + 1], n_rows[l:l + 1], P, out[l:l + 1],
                              ws=ws)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(nrep):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / nrep

    layers()
    torch.cuda.synchronize()
    ref = out.clone()
    t_eager = timed(layers)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        layers()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        layers()
    for _ in range(3):
        out.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), "graph replay differs from the eager launches"
        layers()
        torch.cuda.synchronize()
    t_graph = timed(graph.replay)
    graph.replay()
    torch.cuda.synchronize()
    assert torch.equal(out, ref), "graph replay differs from the eager launches"
    return {"launches": f"{L} sg_decode_attn calls per step, one per layer ({Hkv} KV heads, {Hq} q heads each)",
            "graph_ms": round(t_graph, 4), "eager_ms": round(t_eager, 4),
            "tokens_per_s_graph": round(1.0 / (t_graph * 1e-3), 1),
            "note": "graph replays checked bit for bit against eager launches"}


def cpu_baseline(cfg, pre, bud, layers, min_seconds):
    """The oracle's select+pack (score, top-k, pack) timed on a bounded sample:
    the first ``layers`` layers of the same request, all KV heads, repeated
    until at least ``min_seconds`` have passed."""
    import numpy as np

    import oracle
    if not os.path.exists(oracle.LIB_PATH):
        from oracle import build as ob
        ob.build()
    layers = max(1, min(layers, cfg.L))
    q = pre["q_win"][:, :layers].float().cpu().numpy()
    k = pre["k"][:layers].float().cpu().numpy()
    kraw = pre["k"][:layers].cpu().contiguous().view(__import__("torch").int16).numpy().view(np.uint16)
    vraw = pre["v"][:layers].cpu().contiguous().view(__import__("torch").int16).numpy().view(np.uint16)
    units = layers * cfg.Hkv
    threads = oracle.threads()
    reps = 0
    t0 = time.perf_counter()
    while True:
        s = oracle.score(q, k, pre["cu_seqlens"], cfg.Hkv)
        idx = oracle.topk(s.astype(np.float32), pre["cu_seqlens"], bud["cu_k"])
        oracle.pack(kraw, vraw, idx, pre["cu_seqlens"], bud["cu_k"])
        reps += 1
        if time.perf_counter() - t0 >= min_seconds:
            break
    dt = (time.perf_counter() - t0) / reps
    esize = 2 if cfg.dtype == "bf16" else 4
    kv_bytes = 2 * units * pre["T"] * cfg.d * esize
    # one thread on the first layer alone
    oracle.set_threads(1)
    try:
        t1 = time.perf_counter()
        s1 = oracle.score(q[:, :1], k[:1], pre["cu_seqlens"], cfg.Hkv)
        i1 = oracle.topk(s1.astype(np.float32), pre["cu_seqlens"], bud["cu_k"])
        oracle.pack(kraw[:1], vraw[:1], i1, pre["cu_seqlens"], bud["cu_k"])
        dt1 = time.perf_counter() - t1
    finally:
        oracle.set_threads(threads)
    kv1 = 2 * cfg.Hkv * pre["T"] * cfg.d * esize
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    cpu = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": round(kv_bytes / dt / 1e9, 4), "unit": "GB/s", "cores": min(threads, units),
            "kind": "oracle", "seconds_per_pass": round(dt, 3), "passes": reps,
            "sample": f"score+topk+pack of layers 0..{layers - 1} ({units} of {cfg.L * cfg.Hkv} units), "
                      f"same request, fp64 C oracle with OpenMP over units, repeated {reps}x",
            "cpu_model": cpu, "host": platform.node(),
            "single_thread": {"value": round(kv1 / dt1 / 1e9, 4), "unit": "GB/s", "seconds": round(dt1, 3),
                              "sample": f"score+topk+pack of layer 0 ({cfg.Hkv} units), one thread"}}


if __name__ == "__main__":
    main()
