"""Seeded synthetic inputs for the selective-transfer hot path.

Value model (the workload text fixes K, V ~ N(0, 1); the query model is a
reading of it):

* every unit (request b, layer l, KV head h) has a query mean mu ~ N(0, I_d);
  every window query and every decode query of the unit's q-head group is
  mu + eps with eps ~ N(0, I_d);
* heavy hitters: for each planted token j the component of k_j along
  u = mu / |mu| is set to +4, i.e. k_j <- k_j + (4 - k_j . u) u;
* sinks: tokens 0..sinks-1 get the same boost;
* heavy-hitter positions are drawn without replacement from [sinks, N - W)
  (never inside the score window);
* bf16 workloads round the float64 values to bfloat16 (round to nearest even);
* on-demand extras of a decode step are drawn uniformly without replacement
  from the complement of the selected set, per unit, ascending.

Every tensor is produced on ``device`` with torch; the same call on the CPU
gives the same integer streams.  This module computes nothing of the method
itself (no attention, no selection, no packing).
"""
from __future__ import annotations

import torch

from . import rng
from .configs import Config, budget_k, extras_count, heavy_count

TAG_LEN, TAG_MU, TAG_Q, TAG_K, TAG_V, TAG_HH, TAG_QDEC, TAG_EXTRA, TAG_SEL, TAG_SCORE = range(1, 11)


def storage_dtype(cfg: Config) -> torch.dtype:
    return torch.float32 if cfg.dtype == "f32" else torch.bfloat16


def seqlens(cfg: Config) -> list[int]:
    if cfg.seqlens:
        if len(cfg.seqlens) == cfg.B:
            return [int(n) for n in cfg.seqlens]
        return [int(cfg.seqlens[0])] * cfg.B
    u = rng.uniform(rng.stream_key(cfg.seed, TAG_LEN), cfg.B)
    span = cfg.varlen_hi - cfg.varlen_lo + 1
    return [cfg.varlen_lo + int(x) for x in torch.floor(u * span).tolist()]


def cu_from_lengths(lengths) -> list[int]:
    out = [0]
    for n in lengths:
        out.append(out[-1] + int(n))
    return out


def kv_layers(cfg: Config) -> int:
    """Layers held by the K/V source (1 when every layer shares one source)."""
    return 1 if cfg.kv_shared_layers else cfg.L


def query_means(cfg: Config, device="cpu") -> torch.Tensor:
    """mu for every (request, source layer, KV head): float64 [B][Lkv][Hkv][d]."""
    Lkv = kv_layers(cfg)
    n = cfg.B * Lkv * cfg.Hkv * cfg.d
    return rng.normal(rng.stream_key(cfg.seed, TAG_MU), n, device).view(cfg.B, Lkv, cfg.Hkv, cfg.d)


def _mu_for_layer(cfg: Config, mu: torch.Tensor, l: int) -> torch.Tensor:
    return mu[:, 0 if cfg.kv_shared_layers else l]


def make_prefill(cfg: Config, device="cpu", want_v: bool = True) -> dict:
    """Prompt-side inputs: window queries, K, V and the varlen offsets.

    Shapes: q_win [B][L][Hq][W][d]; k, v [Lkv][Hkv][T][d] with T = sum N_b and
    Lkv = 1 when the layers share one source, else L.  ``heavy`` maps
    (b, l_src, h) to the boosted token ids (sinks first).
    """
    lens = seqlens(cfg)
    cu = cu_from_lengths(lens)
    T = cu[-1]
    G, d, W = cfg.G, cfg.d, cfg.W
    Lkv = kv_layers(cfg)
    sd = storage_dtype(cfg)
    mu = query_means(cfg, device)
    unit = mu / torch.linalg.vector_norm(mu, dim=-1, keepdim=True)
    k = torch.empty((Lkv, cfg.Hkv, T, d), dtype=sd, device=device)
    v = torch.empty((Lkv, cfg.Hkv, T, d), dtype=sd, device=device) if want_v else None
    heavy = {}
    for l in range(Lkv):
        for h in range(cfg.Hkv):
            kk = rng.normal(rng.stream_key(cfg.seed, TAG_K, l, h), T * d, device).view(T, d)
            for b in range(cfg.B):
                n = lens[b]
                u = unit[b, l, h]
                lo, hi = cfg.sinks, n - W
                nh = min(heavy_count(cfg, n), max(0, hi - lo))
                pos = rng.choice_without_replacement(rng.stream_key(cfg.seed, TAG_HH, b, l, h), lo, hi, nh, device)
                pos = torch.cat([torch.arange(min(cfg.sinks, n), dtype=torch.int64, device=device), pos])
                heavy[(b, l, h)] = pos
                rows = kk[cu[b] + pos]
                rows = rows + (4.0 - rows @ u)[:, None] * u[None, :]
                kk[cu[b] + pos] = rows
            k[l, h] = kk.to(sd)
            del kk
            if want_v:
                v[l, h] = rng.normal(rng.stream_key(cfg.seed, TAG_V, l, h), T * d, device).view(T, d).to(sd)
    q = torch.empty((cfg.B, cfg.L, cfg.Hq, W, d), dtype=sd, device=device)
    per_b = cfg.L * cfg.Hq * W * d
    qkey = rng.stream_key(cfg.seed, TAG_Q)
    for b in range(cfg.B):
        eps = rng.normal(qkey, per_b, device, start=b * per_b).view(cfg.L, cfg.Hq, W, d)
        for l in range(cfg.L):
            m = _mu_for_layer(cfg, mu, l)[b].repeat_interleave(G, dim=0)  # [Hq][d]
            q[b, l] = (m[:, None, :] + eps[l]).to(sd)
        del eps
    return dict(q_win=q, k=k, v=v, seqlens=lens, cu_seqlens=cu, T=T, heavy=heavy, mu=mu)


def make_budget(cfg: Config, lens) -> dict:
    ks = [budget_k(n, cfg.budget_bp) for n in lens]
    return dict(k=ks, cu_k=cu_from_lengths(ks), K_total=sum(ks))


def decode_queries(cfg: Config, step: int, device="cpu", mu: torch.Tensor | None = None) -> torch.Tensor:
    """Decode query of every (request, layer, q head) at one step: [B][L][Hq][d]."""
    if mu is None:
        mu = query_means(cfg, device)
    G, d = cfg.G, cfg.d
    n = cfg.B * cfg.L * cfg.Hq * d
    eps = rng.normal(rng.stream_key(cfg.seed, TAG_QDEC, step), n, device).view(cfg.B, cfg.L, cfg.Hq, d)
    if cfg.kv_shared_layers:
        m = mu[:, :1].expand(cfg.B, cfg.L, cfg.Hkv, d)
    else:
        m = mu
    m = m.repeat_interleave(G, dim=2)
    return (m + eps).to(storage_dtype(cfg))


def random_selection(cfg: Config, lens, ks, device="cpu", tag_extra: int = 0) -> torch.Tensor:
    """A method-independent selected set: per unit, k_b distinct ascending ids.

    Returns idx [L][Hkv][K_total] int32 in the layout of a top-k result.
    """
    cu_k = cu_from_lengths(ks)
    out = torch.empty((cfg.L, cfg.Hkv, cu_k[-1]), dtype=torch.int32, device=device)
    for l in range(cfg.L):
        for h in range(cfg.Hkv):
            for b, (n, kb) in enumerate(zip(lens, ks)):
                key = rng.stream_key(cfg.seed, TAG_SEL, tag_extra, b, l, h)
                out[l, h, cu_k[b]:cu_k[b + 1]] = rng.choice_without_replacement(key, 0, n, kb, device).to(torch.int32)
    return out


def synthetic_scores(cfg: Config, lens, device="cpu", levels: int = 0, tag_extra: int = 0) -> torch.Tensor:
    """Method-independent score arrays [L][Hkv][T] f32 for selection tests.

    ``levels`` > 0 quantises the scores to that many distinct values, which
    creates heavy ties.
    """
    T = sum(lens)
    n = cfg.L * cfg.Hkv * T
    u = rng.uniform(rng.stream_key(cfg.seed, TAG_SCORE, tag_extra), n, device)
    if levels > 0:
        u = torch.floor(u * levels) / levels
    return u.to(torch.float32).view(cfg.L, cfg.Hkv, T)


def extras_for_step(cfg: Config, step: int, lens, sel_layer: torch.Tensor, cu_k, layer: int) -> list:
    """On-demand extras of one layer at one decode step.

    ``sel_layer`` is that layer's selected set [Hkv][K_total].  Returns a list
    over (h, b), h-major, of ascending int64 token-id tensors of
    floor(N_b * extra_bp / 10000) ids each, none of them selected.
    """
    device = sel_layer.device
    out = []
    big = torch.iinfo(torch.int64).max
    for h in range(cfg.Hkv):
        for b, n in enumerate(lens):
            e = extras_count(n, cfg.extra_bp)
            r = rng.raw64(rng.stream_key(cfg.seed, TAG_EXTRA, step, b, layer, h), n, device)
            r = r & big  # non-negative, so the sentinel below sorts last
            r[sel_layer[h, cu_k[b]:cu_k[b + 1]].to(torch.int64)] = big
            pick = torch.argsort(r, stable=True)[:e]
            out.append(torch.sort(pick).values)
    return out


def extras_layer(cfg: Config, step: int, lens, sel_layer: torch.Tensor, cu_k, layer: int):
    """The same draws as ``extras_for_step`` for one layer, for every (KV head,
    request) at once (one sort per layer instead of one per unit).

    Returns (ids, cu_e): ids int32 [Hkv][E_total] with request b's ascending
    ids at columns cu_e[b] .. cu_e[b + 1] of every head row, E_total = sum of
    floor(N_b * extra_bp / 10000).
    """
    ids, cu_e = extras_layers(cfg, step, lens, sel_layer[None], cu_k, [layer])
    return ids[0], cu_e


def extras_layers(cfg: Config, step: int, lens, sel: torch.Tensor, cu_k, layers):
    """``extras_layer`` for several layers at once: sel [len(layers)][Hkv][K_total]
    holds each listed layer's selection; returns ids int32
    [len(layers)][Hkv][E_total] and cu_e."""
    device = sel.device
    B, H, nl = len(lens), cfg.Hkv, len(layers)
    R = nl * H                                                    # rows (layer, head)
    cu = cu_from_lengths(lens)
    T = cu[-1]
    ecount = [extras_count(n, cfg.extra_bp) for n in lens]
    cu_e = cu_from_lengths(ecount)
    big = torch.iinfo(torch.int64).max
    lens_t = torch.tensor(lens, dtype=torch.int64, device=device)
    cu_t = torch.tensor(cu[:-1], dtype=torch.int64, device=device)
    keys = torch.tensor([[rng._s64(rng.stream_key(cfg.seed, TAG_EXTRA, step, b, layer, h)) for b in range(B)]
                         for layer in layers for h in range(H)], dtype=torch.int64, device=device)   # [R][B]
    seg_b = torch.repeat_interleave(torch.arange(B, device=device), lens_t)             # token -> request
    local = torch.arange(T, dtype=torch.int64, device=device) - cu_t[seg_b]
    # element i of stream `key` is mix64(i * gamma + key), as in rng.raw64
    r = rng.mix64(local[None, :] * rng._s64(rng._GAMMA) + keys[:, seg_b]) & big          # [R][T]
    ks = torch.tensor([cu_k[b + 1] - cu_k[b] for b in range(B)], dtype=torch.int64, device=device)
    sel_tok = sel.reshape(R, -1).to(torch.int64) + cu_t[torch.repeat_interleave(torch.arange(B, device=device), ks)]
    r.scatter_(1, sel_tok, big)
    flat = r.reshape(-1)
    seg = (torch.arange(R, device=device)[:, None] * B + seg_b[None, :]).reshape(-1)
    o1 = torch.argsort(flat, stable=True)                     # by key, ties by position
    o2 = torch.argsort(seg[o1], stable=True)                  # grouped by (row, request), key order kept
    order = o1[o2]                                            # segment (row i, request b) starts at i * T + cu[b]
    es = torch.tensor(ecount, dtype=torch.int64, device=device)
    e_seg = torch.repeat_interleave(torch.arange(B, device=device), es)                 # pick -> request
    j = torch.arange(int(cu_e[-1]), dtype=torch.int64, device=device) - torch.tensor(cu_e[:-1], dtype=torch.int64,
                                                                                      device=device)[e_seg]
    start = torch.arange(R, device=device)[:, None] * T + cu_t[e_seg][None, :]             # [R][E_total]
    picks = order[start + j[None, :]]
    picks = torch.sort(picks.reshape(-1)).values.view(R, -1)  # segments are disjoint increasing ranges
    return (picks - start).to(torch.int32).view(nl, H, -1), cu_e
