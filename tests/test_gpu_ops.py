"""GPU parity of every C-ABI entry point against the CPU oracle, on seeded
inputs that span several tiles and a ragged tail, plus the edge cases
(empty rows, k = N, ties, NaN / -0, varlen, invalid entries)."""
import numpy as np
import pytest
import torch

import oracle
from datagen import inputs, rng
from datagen.configs import Config
from tests.gpu_util import assert_scores_close, cu, f32, raw, say

pytestmark = pytest.mark.gpu


def _cfg(**kw):
    base = dict(name="t", L=2, Hq=8, Hkv=2, d=128, dtype="bf16", W=16, budget_bp=1000, extra_bp=0, steps=1,
                seqlens=(700,), B=1, heavy_bp=100, sinks=4, seed=11)
    base.update(kw)
    return Config(**base)


# ----------------------------------------------------------------------------- pack

@pytest.mark.parametrize("dtype,d,lens,ks", [
    ("bf16", 128, (700,), (70,)),
    ("bf16", 64, (300, 5, 1000), (31, 5, 1)),
    ("f32", 64, (2048,), (204,)),
    ("f32", 128, (129, 64), (129, 0)),
])
def test_pack_bit_exact(gpu_lib, dtype, d, lens, ks):
    cfg = _cfg(dtype=dtype, d=d, seqlens=lens, B=len(lens), W=4)
    say("pack", dtype, d, lens, ks)
    pre = inputs.make_prefill(cfg, device="cuda")
    cuk = inputs.cu_from_lengths(ks)
    idx = inputs.random_selection(cfg, list(lens), list(ks), device="cuda")
    nbytes = gpu_lib.pack_bytes(pre["k"].dtype, cfg.L, cfg.Hkv, d, cuk[-1])
    dst = torch.full((nbytes,), 0xAB, dtype=torch.uint8, device="cuda")
    gpu_lib.sg_pack(pre["k"], pre["v"], idx, cu(pre["cu_seqlens"]), pre["T"], cu(cuk), cuk[-1], max(ks), dst)
    torch.cuda.synchronize()
    ref = oracle.pack(raw(pre["k"]), raw(pre["v"]), raw(idx), pre["cu_seqlens"], cuk)
    assert np.array_equal(dst.cpu().numpy(), ref)


@pytest.mark.parametrize("max_k", [0, 1])
def test_pack_small_launch_bound_covers_every_row(gpu_lib, max_k):
    """max_k does not shape the launch: a bound of 0 or 1 still packs every k_b."""
    cfg = _cfg(dtype="bf16", d=128, seqlens=(900, 300), B=2, W=4)
    say("pack launch bound", max_k)
    pre = inputs.make_prefill(cfg, device="cuda")
    ks = (300, 40)
    cuk = inputs.cu_from_lengths(ks)
    idx = inputs.random_selection(cfg, [900, 300], list(ks), device="cuda")
    nbytes = gpu_lib.pack_bytes(pre["k"].dtype, cfg.L, cfg.Hkv, 128, cuk[-1])
    dst = torch.full((nbytes,), 0xAB, dtype=torch.uint8, device="cuda")
    gpu_lib.sg_pack(pre["k"], pre["v"], idx, cu(pre["cu_seqlens"]), pre["T"], cu(cuk), cuk[-1], max_k, dst)
    torch.cuda.synchronize()
    ref = oracle.pack(raw(pre["k"]), raw(pre["v"]), raw(idx), pre["cu_seqlens"], cuk)
    assert np.array_equal(dst.cpu().numpy(), ref)


@pytest.mark.parametrize("d,dtype,groups,budget", [(128, torch.bfloat16, 1, 0), (64, torch.bfloat16, 1, 0),
                                                   (128, torch.float32, 1, 0), (128, torch.bfloat16, 3, 0),
                                                   (128, torch.bfloat16, 1, 8), (64, torch.bfloat16, 3, 7)])
def test_pack_many_requests_chunks_across_boundaries(gpu_lib, d, dtype, groups, budget):
    """Chunks that span request boundaries, requests without selected rows, a
    request without tokens (its rows are zero) and invalid indices, over two
    layers; with groups > 1 the requests are packed in calls over consecutive
    groups of them into one buffer (offsets into the whole batch); a budget
    of workgroups makes each take many chunks a grid stride apart."""
    lens = [50, 0, 7, 300, 33, 1, 0, 64, 129, 5, 2, 40, 31, 90, 17]
    ks = [9, 4, 7, 61, 0, 1, 0, 32, 33, 0, 2, 40, 1, 45, 3]
    say("pack across request boundaries", d, dtype, groups, budget)
    g = torch.Generator().manual_seed(77)
    L, Hkv, T = 2, 3, sum(lens)
    k = torch.randn((L, Hkv, T, d), generator=g).to(dtype).cuda()
    v = torch.randn((L, Hkv, T, d), generator=g).to(dtype).cuda()
    cuk = inputs.cu_from_lengths(ks)
    idx = torch.empty((L, Hkv, cuk[-1]), dtype=torch.int32)
    for l in range(L):
        for h in range(Hkv):
            for b, (n, kb) in enumerate(zip(lens, ks)):
                if kb == 0:
                    continue
                sel = torch.randperm(max(n, 1), generator=g)[:kb].sort().values if n >= kb else \
                    torch.randint(-3, 5, (kb,), generator=g)
                idx[l, h, cuk[b]:cuk[b + 1]] = sel.to(torch.int32)
    idx[0, 1, 5] = -1                 # invalid entries inside a valid request
    idx[1, 2, cuk[3] + 7] = lens[3]
    idx = idx.cuda()
    cus = inputs.cu_from_lengths(lens)
    nbytes = gpu_lib.pack_bytes(dtype, L, Hkv, d, cuk[-1])
    dst = torch.full((nbytes,), 0xAB, dtype=torch.uint8, device="cuda")
    cus_d, cuk_d = cu(cus), cu(cuk)
    cuts = [len(lens) * g // groups for g in range(groups + 1)]
    for a, b in zip(cuts[:-1], cuts[1:]):
        gpu_lib.sg_pack(k, v, idx, cus_d[a:b + 1], T, cuk_d[a:b + 1], cuk[-1], max(ks[a:b]), dst, L=L, Hkv=Hkv,
                        max_workgroups=budget)
    torch.cuda.synchronize()
    ref = oracle.pack(raw(k), raw(v), raw(idx), cus, cuk)
    assert np.array_equal(dst.cpu().numpy(), ref)


def test_pack_bad_offsets_leave_slots_unwritten(gpu_lib):
    """Offsets past K_total make a request's segment empty: its slots keep
    their bytes, the valid request is packed as usual."""
    say("pack bad offsets")
    g = torch.Generator().manual_seed(5)
    L, Hkv, d, T = 1, 2, 128, 90
    k = torch.randn((L, Hkv, T, d), generator=g).to(torch.bfloat16).cuda()
    v = torch.randn((L, Hkv, T, d), generator=g).to(torch.bfloat16).cuda()
    K_total = 40
    idx = torch.randint(0, 30, (L, Hkv, K_total), generator=g, dtype=torch.int32).cuda()
    cus = [0, 30, 60, 90]
    cuk_bad = [0, 20, 100, 40]          # requests 1 and 2 end or start past K_total
    nbytes = gpu_lib.pack_bytes(torch.bfloat16, L, Hkv, d, K_total)
    dst = torch.full((nbytes,), 0xAB, dtype=torch.uint8, device="cuda")
    gpu_lib.sg_pack(k, v, idx, cu(cus), T, cu(cuk_bad), K_total, 20, dst)
    torch.cuda.synchronize()
    # request 0 alone with the same slots, from the oracle
    ref = oracle.pack(raw(k), raw(v), raw(idx), [0, 30, 30, 30], [0, 20, 20, 40])
    got = dst.cpu().numpy()
    S, rowb = L * Hkv * K_total, d * 2
    for h in range(Hkv):
        for region, width in ((0, rowb), (S * rowb, rowb), (2 * S * rowb, 4)):
            lo = region + h * K_total * width
            assert np.array_equal(got[lo:lo + 20 * width], ref[lo:lo + 20 * width])
            assert (got[lo + 20 * width:lo + K_total * width] == 0xAB).all()


def test_pack_to_pinned_host_and_full_selection(gpu_lib):
    cfg = _cfg(seqlens=(333,), L=1, W=4)
    say("pack pinned host full selection")
    pre = inputs.make_prefill(cfg, device="cuda")
    N = 333
    idx = torch.arange(N, dtype=torch.int32, device="cuda").expand(1, cfg.Hkv, N).contiguous()
    nbytes = gpu_lib.pack_bytes(torch.bfloat16, 1, cfg.Hkv, 128, N)
    dst = torch.zeros((nbytes,), dtype=torch.uint8, pin_memory=True)
    gpu_lib.sg_pack(pre["k"], pre["v"], idx, cu([0, N]), N, cu([0, N]), N, N, dst)
    torch.cuda.synchronize()
    S = cfg.Hkv * N * 256
    assert dst[:S].numpy().tobytes() == raw(pre["k"]).tobytes()          # full transfer = the cache itself
    assert dst[S:2 * S].numpy().tobytes() == raw(pre["v"]).tobytes()


def test_pack_invalid_index_zero_row(gpu_lib):
    say("pack invalid index")
    k = torch.ones((1, 1, 8, 64), dtype=torch.float32, device="cuda")
    idx = torch.tensor([[[8, -1, 3]]], dtype=torch.int32, device="cuda")
    nbytes = gpu_lib.pack_bytes(torch.float32, 1, 1, 64, 3)
    dst = torch.full((nbytes,), 0x7F, dtype=torch.uint8, device="cuda")
    gpu_lib.sg_pack(k, k, idx, cu([0, 8]), 8, cu([0, 3]), 3, 3, dst)
    torch.cuda.synchronize()
    ref = oracle.pack(k.cpu().numpy(), k.cpu().numpy(), idx.cpu().numpy(), [0, 8], [0, 3])
    assert np.array_equal(dst.cpu().numpy(), ref)


# ----------------------------------------------------------------------------- topk

def _topk_case(lens, ks, levels, seed, specials=False, L=2, Hkv=3):
    cfg = _cfg(L=L, Hkv=Hkv, Hq=Hkv, seqlens=tuple(lens), B=len(lens), seed=seed)
    s = inputs.synthetic_scores(cfg, lens, levels=levels)
    if specials:
        g = np.random.default_rng(seed)
        flat = s.view(-1)
        n = flat.numel()
        flat[torch.from_numpy(g.integers(0, n, n // 50))] = float("nan")
        flat[torch.from_numpy(g.integers(0, n, n // 50))] = -0.0
        flat[torch.from_numpy(g.integers(0, n, n // 50))] = 0.0
        flat[torch.from_numpy(g.integers(0, n, n // 100))] = float("inf")
        flat[torch.from_numpy(g.integers(0, n, n // 100))] = -float("inf")
    return cfg, s


@pytest.mark.parametrize("lens,ks,levels,specials", [
    ((8192,), (819,), 0, False),
    ((8192,), (819,), 7, False),               # heavy ties
    ((2048, 17, 1000), (204, 17, 999), 0, True),
    ((32768,), (1638,), 40, True),
    ((65536,), (6553,), 1000, False),
    ((5000, 1, 64), (1, 1, 32), 0, False),
])
def test_topk_bit_exact(gpu_lib, lens, ks, levels, specials):
    cfg, s = _topk_case(lens, ks, levels, seed=sum(lens) + levels, specials=specials)
    cus, cuk = inputs.cu_from_lengths(lens), inputs.cu_from_lengths(ks)
    say("topk", lens, ks, levels, specials)
    sd = s.cuda()
    idx = torch.full((cfg.L, cfg.Hkv, cuk[-1]), -7, dtype=torch.int32, device="cuda")
    gpu_lib.sg_topk(sd, cu(cus), cus[-1], max(lens), cu(cuk), cuk[-1], idx)
    torch.cuda.synchronize()
    ref = oracle.topk(s.numpy(), cus, cuk)
    np.testing.assert_array_equal(idx.cpu().numpy(), ref)


@pytest.mark.parametrize("lens,ks,levels,specials", [
    ((12000, 32768), (1200, 3276), 0, True),
    ((9000, 20000), (900, 19999), 25, False),     # heavy ties, k close to N
])
def test_topk_many_rows_bit_exact(gpu_lib, lens, ks, levels, specials):
    """512 rows of 8K-32K keys: the calls with at least two rows per CU take
    the 512-thread workgroups (64 keys per thread)."""
    cfg, s = _topk_case(lens, ks, levels, seed=sum(lens) + levels, specials=specials, L=32, Hkv=8)
    cus, cuk = inputs.cu_from_lengths(lens), inputs.cu_from_lengths(ks)
    say("topk many rows", lens, ks, levels, specials)
    sd = s.cuda()
    idx = torch.full((cfg.L, cfg.Hkv, cuk[-1]), -7, dtype=torch.int32, device="cuda")
    gpu_lib.sg_topk(sd, cu(cus), cus[-1], max(lens), cu(cuk), cuk[-1], idx)
    torch.cuda.synchronize()
    ref = oracle.topk(s.numpy(), cus, cuk)
    np.testing.assert_array_equal(idx.cpu().numpy(), ref)


def test_topk_all_equal_is_address_prefix(gpu_lib):
    say("topk all equal")
    s = torch.full((1, 2, 4000), 0.5, dtype=torch.float32, device="cuda")
    idx = torch.empty((1, 2, 400), dtype=torch.int32, device="cuda")
    gpu_lib.sg_topk(s, cu([0, 4000]), 4000, 4000, cu([0, 400]), 400, idx)
    torch.cuda.synchronize()
    assert (idx.cpu() == torch.arange(400, dtype=torch.int32)).all()


def test_topk_bad_metadata_marks_segment(gpu_lib):
    say("topk k > N")
    s = torch.rand((1, 1, 10), device="cuda")
    idx = torch.zeros((1, 1, 12), dtype=torch.int32, device="cuda")
    gpu_lib.sg_topk(s, cu([0, 10]), 10, 10, cu([0, 12]), 12, idx)
    torch.cuda.synchronize()
    assert (idx.cpu() == -1).all()


# ----------------------------------------------------------------------------- split

@pytest.mark.parametrize("reorder", [0, 1])
@pytest.mark.parametrize("rows,maxn,N", [(37, 300, 1000), (5, 2000, 4096), (3, 0, 10)])
def test_split_bit_exact(gpu_lib, reorder, rows, maxn, N):
    g = np.random.default_rng(rows * 7 + maxn + reorder)
    n = g.integers(0, maxn + 1, rows)
    n[0] = maxn
    row_off = np.cumsum([0] + list(n)).astype(np.int32)
    mask = g.integers(0, 3, rows * N).astype(np.int8)
    mask[g.random(rows * N) < 0.01] = 5
    mask_off = (np.arange(rows) * N).astype(np.int64)
    mask_len = np.full(rows, N, np.int32)
    ix = (np.concatenate([g.integers(-3, N + 3, k) for k in n]) if n.sum() else np.zeros(0)).astype(np.int32)
    total = int(row_off[-1])
    say("split", rows, maxn, N, reorder)
    T = max(total, 1)
    loc = torch.full((T,), -9, dtype=torch.int32, device="cuda")
    rem = torch.full((T,), -9, dtype=torch.int32, device="cuda")
    out = torch.full((T,), -9, dtype=torch.int32, device="cuda")
    nl = torch.zeros(rows, dtype=torch.int32, device="cuda")
    nr = torch.zeros(rows, dtype=torch.int32, device="cuda")
    gpu_lib.sg_split(cu(row_off), cu(ix) if total else torch.zeros(1, dtype=torch.int32, device="cuda")[:0],
                     cu(mask, dtype=torch.int8), cu(mask_off, dtype=torch.int64), cu(mask_len), reorder,
                     loc, rem, nl, nr, out_index=out if reorder else None)
    torch.cuda.synchronize()
    r_out, r_loc, r_rem, r_nl, r_nr = oracle.split(row_off, ix, mask, mask_off, mask_len, reorder)
    np.testing.assert_array_equal(nl.cpu().numpy(), r_nl)
    np.testing.assert_array_equal(nr.cpu().numpy(), r_nr)
    np.testing.assert_array_equal(loc.cpu().numpy()[:total], r_loc)
    np.testing.assert_array_equal(rem.cpu().numpy()[:total], r_rem)
    if reorder:
        np.testing.assert_array_equal(out.cpu().numpy()[:total], r_out)


# ----------------------------------------------------------------------------- fetch

@pytest.mark.parametrize("host_src", [True, False])
@pytest.mark.parametrize("dtype,d,P", [("bf16", 128, 16), ("f32", 64, 1), ("bf16", 64, 4)])
def test_fetch_bit_exact(gpu_lib, host_src, dtype, d, P):
    g = np.random.default_rng(d + P + host_src)
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    src_rows = 5000
    ks = torch.randn((src_rows, d), generator=torch.Generator().manual_seed(1)).to(td)
    vs = torch.randn((src_rows, d), generator=torch.Generator().manual_seed(2)).to(td)
    if host_src:
        ks, vs = ks.pin_memory(), vs.pin_memory()
    else:
        ks, vs = ks.cuda(), vs.cuda()
    rows = 9
    n = g.integers(0, 300, rows)
    row_off = np.cumsum([0] + list(n)).astype(np.int32)
    index = g.integers(-2, 1002, max(int(row_off[-1]), 1))[: row_off[-1]].astype(np.int32)
    n_valid = (n - g.integers(0, 3, rows)).astype(np.int32)
    src_base = (np.arange(rows) * 500).astype(np.int64)
    max_pages = 330 // P + 2
    pool_rows = rows * max_pages * P
    pages = (g.permutation(rows * max_pages).reshape(rows, max_pages) * P).astype(np.int32)
    dst_start = g.integers(0, 20, rows).astype(np.int32)
    say("fetch", host_src, dtype, d, P)
    kp = torch.zeros((pool_rows, d), dtype=td, device="cuda")
    vp = torch.zeros((pool_rows, d), dtype=td, device="cuda")
    gpu_lib.sg_fetch(cu(row_off), int(row_off[-1]), cu(index), cu(n_valid), cu(src_base, dtype=torch.int64),
                     ks, vs, cu(pages), P, cu(dst_start), kp, vp)
    torch.cuda.synchronize()
    rk = np.zeros((pool_rows, d), raw(ks).dtype)
    rv = np.zeros((pool_rows, d), raw(vs).dtype)
    oracle.fetch(row_off, index, n_valid, src_base, raw(ks), raw(vs), pages, P, dst_start, rk, rv)
    assert np.array_equal(raw(kp), rk) and np.array_equal(raw(vp), rv)


# ----------------------------------------------------------------------------- decode attention

def _paged_set(g, B, Hkv, d, nmax, P, td, empty_some=True):
    n = g.integers(0, nmax + 1, (B, Hkv)).astype(np.int32)
    n[0, 0] = nmax
    if empty_some and B * Hkv > 2:
        n[-1, -1] = 0
        n[-1, 0] = 1
    max_pages = (nmax + P - 1) // P
    pool_rows = B * Hkv * max_pages * P + 3 * P
    pages = (g.permutation(B * Hkv * max_pages + 3).astype(np.int64)[: B * Hkv * max_pages]
             .reshape(B, Hkv, max_pages) * P).astype(np.int32)
    kp = torch.randn((pool_rows, d), generator=torch.Generator().manual_seed(int(g.integers(1 << 30)))).to(td)
    vp = torch.randn((pool_rows, d), generator=torch.Generator().manual_seed(int(g.integers(1 << 30)))).to(td)
    return n, pages, kp, vp


@pytest.mark.parametrize("dtype,d,G,nmax,P,B", [
    ("bf16", 128, 4, 819, 16, 3),
    ("bf16", 128, 8, 1700, 16, 2),
    ("bf16", 128, 1, 300, 1, 2),
    ("bf16", 64, 16, 520, 4, 1),
    ("f32", 64, 1, 204, 16, 2),
    ("f32", 128, 2, 1000, 1, 2),
    ("bf16", 128, 4, 256, 16, 4),              # exactly one split
    ("bf16", 128, 4, 819, 16, 128),            # >= 256 units: one split, several tiles per wavefront
    ("bf16", 128, 8, 1700, 16, 128),
    # every lane layout of the end-of-kernel reduction (lanes per row 4, 8, 16)
    ("bf16", 64, 2, 700, 16, 3),
    ("bf16", 64, 4, 333, 8, 2),
    ("bf16", 128, 2, 900, 16, 130),
    ("f32", 128, 8, 500, 16, 2),
    ("f32", 64, 4, 611, 2, 3),
    ("f32", 128, 4, 410, 16, 140),
    # more units than CUs, one row per lane group and two head groups
    ("f32", 64, 1, 204, 16, 129),
    ("bf16", 64, 16, 300, 4, 130),
    # one to four units per CU with at least 512 rows: equal parts over the
    # shader engines (units not a multiple of 8, engine bins of up to 125 units)
    ("bf16", 128, 4, 1500, 16, 150),
    ("f32", 128, 8, 700, 16, 257),
    ("bf16", 64, 1, 1200, 1, 500),
    # four or more units per CU: one workgroup per unit (unit counts not a
    # multiple of 8)
    ("bf16", 128, 4, 300, 16, 520),
    ("f32", 64, 2, 150, 16, 1101),
])
def test_decode_parity(gpu_lib, dtype, d, G, nmax, P, B):
    g = np.random.default_rng(nmax + G + d + P)
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    Hkv = 2
    Hq = G * Hkv
    n, pages, kp, vp = _paged_set(g, B, Hkv, d, nmax, P, td)
    q = (torch.randn((B, Hq, d), generator=torch.Generator().manual_seed(3)) * 2).to(td)
    say("decode", dtype, d, G, nmax, P, B)
    out = torch.full((B, Hq, d), float("nan"), device="cuda")
    wsz = gpu_lib.decode_workspace_size(B, Hq, Hkv, d, pages.shape[-1], P)
    ws = torch.empty((max(wsz, 4),), dtype=torch.uint8, device="cuda")
    gpu_lib.sg_decode_attn(q.cuda(), kp.cuda(), vp.cuda(), cu(pages), cu(n), P, out, ws=ws)
    torch.cuda.synchronize()
    ref = oracle.decode_attn(f32(q), f32(kp), f32(vp), pages, n, P)
    o = out.cpu().numpy()
    assert np.isfinite(o).all()
    tol = 2e-2 if dtype == "bf16" else 1e-4
    np.testing.assert_allclose(o, ref, atol=tol, rtol=0)


def test_decode_equal_parts_tiny_units(gpu_lib):
    """Equal-parts launches where most units hold 0 to 3 rows: parts of such
    units are empty or one row long, and both still meet in the merge."""
    say("decode equal parts, tiny units")
    g = np.random.default_rng(4242)
    B, Hkv, G, d, P = 140, 2, 4, 128, 16
    Hq = G * Hkv
    n, pages, kp, vp = _paged_set(g, B, Hkv, d, 640, P, torch.bfloat16)
    n[:] = g.integers(0, 4, n.shape)
    n[0, 0], n[77, 1], n[-1, 0] = 640, 513, 3
    q = (torch.randn((B, Hq, d), generator=torch.Generator().manual_seed(9)) * 2).to(torch.bfloat16)
    out = torch.full((B, Hq, d), float("nan"), device="cuda")
    ws = torch.empty((gpu_lib.decode_workspace_size(B, Hq, Hkv, d, pages.shape[-1], P),), dtype=torch.uint8,
                     device="cuda")
    gpu_lib.sg_decode_attn(q.cuda(), kp.cuda(), vp.cuda(), cu(pages), cu(n), P, out, ws=ws)
    torch.cuda.synchronize()
    ref = oracle.decode_attn(f32(q), f32(kp), f32(vp), pages, n, P)
    o = out.cpu().numpy()
    assert np.isfinite(o).all()
    np.testing.assert_allclose(o, ref, atol=1e-4, rtol=0)
    assert (o[n.reshape(-1).repeat(G).reshape(B, Hq) == 0] == 0).all()


def test_decode_split_workspace_reused(gpu_lib):
    """Few units split their rows over several workgroups and a merge combines
    them through the workspace; one workspace serves call after call."""
    say("decode split workspace reuse")
    g = np.random.default_rng(77)
    B, Hkv, G, d, nmax, P = 2, 2, 4, 128, 1500, 16
    Hq = G * Hkv
    n, pages, kp, vp = _paged_set(g, B, Hkv, d, nmax, P, torch.bfloat16, empty_some=False)
    wsz = gpu_lib.decode_workspace_size(B, Hq, Hkv, d, pages.shape[-1], P)
    assert wsz > 0                         # this shape splits
    ws = torch.empty((wsz,), dtype=torch.uint8, device="cuda")
    kd, vd, pd, nd = kp.cuda(), vp.cuda(), cu(pages), cu(n)
    for call in range(3):
        q = (torch.randn((B, Hq, d), generator=torch.Generator().manual_seed(100 + call)) * 2).to(torch.bfloat16)
        out = torch.full((B, Hq, d), float("nan"), device="cuda")
        gpu_lib.sg_decode_attn(q.cuda(), kd, vd, pd, nd, P, out, ws=ws)
        torch.cuda.synchronize()
        ref = oracle.decode_attn(f32(q), f32(kp), f32(vp), pages, n, P)
        np.testing.assert_allclose(out.cpu().numpy(), ref, atol=2e-2, rtol=0)


def test_decode_invalid_pages_are_skipped(gpu_lib):
    say("decode invalid pages")
    d, P = 128, 16
    kp = torch.randn((64, d)).to(torch.bfloat16)
    vp = torch.randn((64, d)).to(torch.bfloat16)
    pages = np.array([[[0, 10_000, 32, -16]]], np.int32)      # two pages point outside the pool
    n = np.array([[64]], np.int32)
    q = torch.randn((1, 4, d)).to(torch.bfloat16)
    out = torch.empty((1, 4, d), device="cuda")
    ws = torch.empty(max(16, gpu_lib.decode_workspace_size(1, 4, 1, d, 4, P)), dtype=torch.uint8, device="cuda")
    gpu_lib.sg_decode_attn(q.cuda(), kp.cuda(), vp.cuda(), cu(pages), cu(n), P, out, ws=ws)
    torch.cuda.synchronize()
    ref = oracle.decode_attn(f32(q), f32(kp), f32(vp), pages, n, P)
    np.testing.assert_allclose(out.cpu().numpy(), ref, atol=2e-2, rtol=0)


# ----------------------------------------------------------------------------- score

@pytest.mark.parametrize("dtype,d,Hq,Hkv,W,lens", [
    ("f32", 64, 8, 8, 32, (2048,)),               # the tiny workload's shape
    ("bf16", 128, 8, 2, 64, (1500, 700)),          # G=4, R=256, varlen, ragged last tile
    ("bf16", 128, 16, 2, 64, (1100,)),             # G=8, R=512
    ("bf16", 64, 4, 4, 20, (97, 513, 64)),         # R=20 (one partial wavefront), W = N edge
    ("f32", 128, 2, 1, 16, (600,)),
])
def test_score_parity(gpu_lib, dtype, d, Hq, Hkv, W, lens):
    cfg = _cfg(dtype=dtype, d=d, Hq=Hq, Hkv=Hkv, W=W, seqlens=lens, B=len(lens), L=2, seed=len(lens) + d)
    say("score", dtype, d, Hq, Hkv, W, lens)
    pre = inputs.make_prefill(cfg, device="cuda", want_v=False)
    T = pre["T"]
    scores = torch.full((cfg.L, Hkv, T), float("nan"), device="cuda")
    wsz = gpu_lib.score_workspace_size(cfg.B, cfg.L, Hq, Hkv, d, W, max(lens))
    ws = torch.empty((wsz,), dtype=torch.uint8, device="cuda")
    gpu_lib.sg_score(pre["q_win"], pre["k"], cu(pre["cu_seqlens"]), T, max(lens), Hkv, scores, ws=ws)
    torch.cuda.synchronize()
    ref = oracle.score(f32(pre["q_win"]), f32(pre["k"]), pre["cu_seqlens"], Hkv)
    got = scores.cpu().numpy()
    assert_scores_close(got, ref)
    # each unit's scores add up to G * W
    G = Hq // Hkv
    c = pre["cu_seqlens"]
    for b in range(cfg.B):
        tot = got[:, :, c[b]:c[b + 1]].astype(np.float64).sum(-1)
        np.testing.assert_allclose(tot, G * W, rtol=1e-4)


def test_score_with_caller_lse(gpu_lib):
    """The one-pass path: LSE supplied (here computed by torch in float64 on the CPU)."""
    cfg = _cfg(W=32, seqlens=(900,), L=1, Hq=8, Hkv=2)
    say("score lse_in")
    pre = inputs.make_prefill(cfg, device="cuda", want_v=False)
    N, W, d, G = 900, 32, 128, 4
    q = pre["q_win"].double().cpu()[0, 0]                      # [Hq][W][d]
    k = pre["k"].double().cpu()[0]                             # [Hkv][N][d]
    kk = k.repeat_interleave(G, dim=0)
    z = q @ kk.transpose(1, 2) / d ** 0.5                       # [Hq][W][N]
    pos = torch.arange(N - W, N)[:, None]
    z = z.masked_fill(torch.arange(N)[None, :] > pos, float("-inf"))
    lse = torch.logsumexp(z, dim=-1).float().reshape(1, 1, 8, W).cuda()
    scores = torch.empty((1, 2, N), device="cuda")
    gpu_lib.sg_score(pre["q_win"], pre["k"], cu([0, N]), N, N, 2, scores, lse_in=lse)
    torch.cuda.synchronize()
    ref = oracle.score(f32(pre["q_win"]), f32(pre["k"]), [0, N], 2)
    assert_scores_close(scores.cpu().numpy(), ref)


def test_score_deterministic(gpu_lib):
    cfg = _cfg(W=64, seqlens=(3000,), L=1, Hq=32, Hkv=8)
    say("score determinism")
    pre = inputs.make_prefill(cfg, device="cuda", want_v=False)
    wsz = gpu_lib.score_workspace_size(1, 1, 32, 8, 128, 64, 3000)
    ws = torch.empty((wsz,), dtype=torch.uint8, device="cuda")
    outs = []
    for _ in range(2):
        s = torch.empty((1, 8, 3000), device="cuda")
        gpu_lib.sg_score(pre["q_win"], pre["k"], cu([0, 3000]), 3000, 3000, 8, s, ws=ws)
        outs.append(s)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])
