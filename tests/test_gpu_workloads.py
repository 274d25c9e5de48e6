"""The five workloads at their full sizes, in the launch configurations the
bench uses, checked against the CPU oracle: in full where the oracle finishes
in seconds, otherwise on sampled layers, units or steps.

The GPU and the oracle each run the whole chain on their own: every later
oracle step takes the oracle's own earlier results (its top-k, its packed
bytes, its pools), never a GPU output; only inputs from the seeded generators
(and host-built tables such as page tables and masks) feed both sides."""
import numpy as np
import pytest
import torch

import oracle
from datagen import configs, inputs
from tests.gpu_util import assert_scores_close, assert_topk_sets_agree, cu, f32, raw, say

pytestmark = pytest.mark.gpu


def bf16_bits_to_f32(a: np.ndarray) -> np.ndarray:
    """Exact widening of raw bfloat16 bits (uint16) to float32."""
    return (a.astype(np.uint32) << 16).view(np.float32)


def rows_as_f32(a: np.ndarray, dtype: torch.dtype) -> np.ndarray:
    return bf16_bits_to_f32(a) if dtype == torch.bfloat16 else a.view(np.float32)


def _seeded(cfg, seed):
    """The workload as configured, or re-drawn from another seed (the robustness reruns)."""
    return cfg if seed is None else cfg.with_(seed=seed)


def _score_units(gpu_lib, cfg, pre, units):
    """GPU scores of the whole workload, compared with the oracle on `units` = [(l, h)]."""
    T, lens = pre["T"], pre["seqlens"]
    ws = torch.empty(gpu_lib.score_workspace_size(cfg.B, cfg.L, cfg.Hq, cfg.Hkv, cfg.d, cfg.W, max(lens)),
                     dtype=torch.uint8, device="cuda")
    scores = torch.full((cfg.L, cfg.Hkv, T), float("nan"), device="cuda")
    gpu_lib.sg_score(pre["q_win"], pre["k"], cu(pre["cu_seqlens"]), T, max(lens), cfg.Hkv, scores, ws=ws)
    torch.cuda.synchronize()
    G = cfg.G
    for (l, h) in units:
        say("score unit", l, h)
        q = f32(pre["q_win"][:, l:l + 1, h * G:(h + 1) * G])
        lk = 0 if cfg.kv_shared_layers else l
        k = f32(pre["k"][lk:lk + 1, h:h + 1])
        ref = oracle.score(q, k, pre["cu_seqlens"], 1)
        assert_scores_close(scores[l, h].cpu().numpy()[None, None], ref)
    return scores


def _topk_exact(gpu_lib, cfg, pre, bud, levels=0, layers=None):
    """Top-k of a method-independent full-size score array on the GPU; the
    oracle's top-k of the same array on every layer (or on `layers`) must be
    bit-identical.  Returns (GPU idx of every layer, oracle idx of the layers)."""
    lens, T = pre["seqlens"], pre["T"]
    s = inputs.synthetic_scores(cfg, lens, device="cuda", levels=levels)
    idx = torch.empty((cfg.L, cfg.Hkv, bud["K_total"]), dtype=torch.int32, device="cuda")
    gpu_lib.sg_topk(s, cu(pre["cu_seqlens"]), T, max(lens), cu(bud["cu_k"]), bud["K_total"], idx)
    torch.cuda.synchronize()
    ls = list(range(cfg.L)) if layers is None else list(layers)
    ref_idx = oracle.topk(s[ls].cpu().numpy(), pre["cu_seqlens"], bud["cu_k"])
    np.testing.assert_array_equal(idx[ls].cpu().numpy(), ref_idx)
    return idx, ref_idx


def _pack_exact(gpu_lib, cfg, pre, bud, idx_dev, ref_idx, pinned=False, layers=None):
    """GPU pack of every layer; the oracle packs its own index table for every
    layer (or for `layers`) and the K, V and index blocks must match bit for
    bit.  Returns (GPU buffer, oracle K rows, oracle V rows) where the oracle
    rows of the checked layers are stacked [len(layers) * Hkv * K_total][d]."""
    nbytes = gpu_lib.pack_bytes(pre["k"].dtype, cfg.L, cfg.Hkv, cfg.d, bud["K_total"])
    if pinned:
        dst = torch.empty((nbytes,), dtype=torch.uint8, pin_memory=True)
    else:
        dst = torch.empty((nbytes,), dtype=torch.uint8, device="cuda")
    gpu_lib.sg_pack(pre["k"], pre["v"], idx_dev, cu(pre["cu_seqlens"]), pre["T"], cu(bud["cu_k"]), bud["K_total"],
                    max(bud["k"]), dst, L=cfg.L, Hkv=cfg.Hkv)
    torch.cuda.synchronize()

    def got(lo, hi):
        return dst[lo:hi].numpy() if pinned else dst[lo:hi].cpu().numpy()

    kraw, vraw = raw(pre["k"]), raw(pre["v"])
    ls = list(range(cfg.L)) if layers is None else list(layers)
    es = pre["k"].element_size()
    row_b = cfg.d * es
    per_layer = cfg.Hkv * bud["K_total"]
    S = cfg.L * per_layer
    kb = per_layer * row_b
    kref, vref = [], []
    if layers is None:
        ref = oracle.pack(kraw, vraw, ref_idx, pre["cu_seqlens"], bud["cu_k"],
                          kv_layer_rows=0 if cfg.kv_shared_layers else None)
        assert np.array_equal(got(0, nbytes), ref)
        kref.append(ref[:S * row_b])
        vref.append(ref[S * row_b:2 * S * row_b])
    else:
        for i, l in enumerate(ls):
            lk = 0 if cfg.kv_shared_layers else l
            ref = oracle.pack(kraw[lk:lk + 1], vraw[lk:lk + 1], ref_idx[i:i + 1], pre["cu_seqlens"], bud["cu_k"])
            ko = l * kb
            vo = S * row_b + ko
            io = 2 * S * row_b + l * per_layer * 4
            assert np.array_equal(got(ko, ko + kb), ref[:kb]), f"K block of layer {l}"
            assert np.array_equal(got(vo, vo + kb), ref[kb:2 * kb]), f"V block of layer {l}"
            assert np.array_equal(got(io, io + per_layer * 4), ref[2 * kb:]), f"index block of layer {l}"
            kref.append(ref[:kb])
            vref.append(ref[kb:2 * kb])
    nd = np.uint16 if es == 2 else np.float32
    kr = np.concatenate(kref).view(nd).reshape(-1, cfg.d)
    vr = np.concatenate(vref).view(nd).reshape(-1, cfg.d)
    return dst, kr, vr


def _pools(dst, cfg, K_total, dtype):
    """K and V row views [S][d] of a transfer buffer (device)."""
    S = cfg.L * cfg.Hkv * K_total
    es = 2 if dtype == torch.bfloat16 else 4
    kp = dst[: S * cfg.d * es].view(dtype).view(S, cfg.d)
    vp = dst[S * cfg.d * es: 2 * S * cfg.d * es].view(dtype).view(S, cfg.d)
    return kp, vp


def _contiguous_table(n_seq, Hkv, K, P, device="cuda"):
    """Page table of sequences whose rows sit back to back, K per (seq, head)."""
    npg = (K + P - 1) // P
    t = (torch.arange(n_seq * Hkv, device=device)[:, None] * K
         + torch.arange(npg, device=device)[None, :] * P).to(torch.int32)
    return t.view(n_seq, Hkv, npg).contiguous()


def _decode_check(gpu_lib, q, kp, vp, pt, nr, P, ref_k, ref_v, ref_pt, seqs=None, atol=2e-2):
    """GPU decode of every sequence over (kp, vp, pt); the oracle attends over
    its own pools (ref_k, ref_v: float32 [rows][d], addressed by ref_pt whose
    rows are the sequences `seqs`, all when None)."""
    B, Hq, d = q.shape
    out = torch.full((B, Hq, d), float("nan"), device="cuda")
    wsz = gpu_lib.decode_workspace_size(B, Hq, pt.shape[1], d, pt.shape[2], P)
    ws = torch.zeros((max(wsz, 16),), dtype=torch.uint8, device="cuda")
    gpu_lib.sg_decode_attn(q, kp, vp, pt, nr, P, out, ws=ws)
    torch.cuda.synchronize()
    seqs = list(range(B)) if seqs is None else list(seqs)
    ref = oracle.decode_attn(f32(q)[seqs], ref_k, ref_v, ref_pt, nr.cpu().numpy()[seqs], P)
    o = out.cpu().numpy()[seqs]
    assert np.isfinite(o).all()
    np.testing.assert_allclose(o, ref, atol=atol, rtol=0)


# ----------------------------------------------------------------------------- tiny (whole pipeline, in full)

@pytest.mark.parametrize("seed", [None, 101])
def test_tiny_whole_pipeline(gpu_lib, seed):
    cfg = _seeded(configs.get("tiny"), seed)
    say("workload tiny", "seed", cfg.seed)
    pre = inputs.make_prefill(cfg, device="cuda")
    lens, T = pre["seqlens"], pre["T"]
    bud = inputs.make_budget(cfg, lens)
    K = bud["K_total"]
    scores = _score_units(gpu_lib, cfg, pre, [(0, h) for h in range(cfg.Hkv)])
    ref_scores = oracle.score(f32(pre["q_win"]), f32(pre["k"]), pre["cu_seqlens"], cfg.Hkv)
    # top-k of the oracle's scores (rounded to float32 as the kernels store them): bit-exact
    s32 = ref_scores.astype(np.float32)
    idx = torch.empty((1, cfg.Hkv, K), dtype=torch.int32, device="cuda")
    gpu_lib.sg_topk(torch.from_numpy(s32).cuda(), cu(pre["cu_seqlens"]), T, T, cu(bud["cu_k"]), K, idx)
    torch.cuda.synchronize()
    ref_idx = oracle.topk(s32, pre["cu_seqlens"], bud["cu_k"])
    np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)
    # end to end: GPU scores -> GPU top-k vs oracle scores -> oracle top-k, differing on near-ties only
    idx_e2e = torch.empty_like(idx)
    gpu_lib.sg_topk(scores, cu(pre["cu_seqlens"]), T, T, cu(bud["cu_k"]), K, idx_e2e)
    torch.cuda.synchronize()
    for h in range(cfg.Hkv):
        assert_topk_sets_agree(idx_e2e[0, h].cpu().numpy(), ref_idx[0, h], ref_scores[0, h], K)
    # the planted heavy hitters rank at the top
    for h in range(cfg.Hkv):
        hh = set(pre["heavy"][(0, 0, h)].tolist())
        assert len(hh & set(ref_idx[0, h].tolist())) >= 0.9 * len(hh)
    dst, kr, vr = _pack_exact(gpu_lib, cfg, pre, bud, idx, ref_idx)
    kp, vp = _pools(dst, cfg, K, torch.float32)
    pt = _contiguous_table(1, cfg.Hkv, K, cfg.page_size)
    nr = torch.full((1, cfg.Hkv), K, dtype=torch.int32, device="cuda")
    q = inputs.decode_queries(cfg, 0, device="cuda", mu=pre["mu"])[0].contiguous()
    _decode_check(gpu_lib, q, kp, vp, pt, nr, cfg.page_size, kr, vr, pt.cpu().numpy(), atol=1e-4)


# ----------------------------------------------------------------------------- Llama-3-8B shape, 8K prompt

@pytest.mark.parametrize("seed", [None, 102])
def test_llama8b_8k(gpu_lib, seed):
    cfg = _seeded(configs.get("llama8b_8k"), seed)
    say("workload llama8b_8k", "seed", cfg.seed)
    pre = inputs.make_prefill(cfg, device="cuda")
    bud = inputs.make_budget(cfg, pre["seqlens"])
    K = bud["K_total"]
    _score_units(gpu_lib, cfg, pre, [(0, 0), (17, 5), (31, 7)])
    idx, ref_idx = _topk_exact(gpu_lib, cfg, pre, bud, levels=0)
    dst, kr, vr = _pack_exact(gpu_lib, cfg, pre, bud, idx, ref_idx)
    # decode in the bench's launch configuration: the 32 layers as 32 sequences, 16-row pages
    kp, vp = _pools(dst, cfg, K, torch.bfloat16)
    pt = _contiguous_table(cfg.L, cfg.Hkv, K, cfg.page_size)
    nr = torch.full((cfg.L, cfg.Hkv), K, dtype=torch.int32, device="cuda")
    kf, vf = bf16_bits_to_f32(kr), bf16_bits_to_f32(vr)
    for step in (0, cfg.steps - 1):
        say("llama8b_8k decode step", step)
        q = inputs.decode_queries(cfg, step, device="cuda", mu=pre["mu"])[0].contiguous()
        _decode_check(gpu_lib, q, kp, vp, pt, nr, cfg.page_size, kf, vf, pt.cpu().numpy())


# ----------------------------------------------------------------------------- paged decode with on-demand fetch

def _paged_decode_layer(gpu_lib, cfg, pre, bud, layer, step, sel_ref, kr_l, vr_l, kp_t, vp_t, host_k, host_v, seed):
    """One decode step of one layer (units (h, b), h-major):

    * Algorithm 1 on each unit's index = [on-demand extras ++ selected set],
      with the mask 1 on the selected set, 2 elsewhere inside the prompt;
    * receive: the unit's selected rows copied from the transfer buffer to
      logical rows e .. e+k-1 of its paged row;
    * remote lane: the remote entries fetched from the pinned host K/V into
      logical rows 0 .. e-1;
    * decode over the e + k rows.

    The GPU reads its own transfer buffer (kp_t, vp_t); the oracle reads its
    own packed rows of this layer (kr_l, vr_l: [Hkv * K_total][d] raw) and its
    own selection sel_ref [Hkv][K_total]."""
    lens = pre["seqlens"]
    P, d = cfg.page_size, cfg.d
    cu_s, cu_k, K = pre["cu_seqlens"], bud["cu_k"], bud["K_total"]
    units = [(h, b) for h in range(cfg.Hkv) for b in range(cfg.B)]
    nu = len(units)
    ex = inputs.extras_for_step(cfg, step, lens, torch.from_numpy(sel_ref).cuda(), cu_k, layer)
    e_cnt = [len(x) for x in ex]
    k_cnt = [bud["k"][b] for (h, b) in units]
    rows_u = [e + k for e, k in zip(e_cnt, k_cnt)]
    max_pages = max((r + P - 1) // P for r in rows_u)
    total_pages = sum((r + P - 1) // P for r in rows_u)
    perm = np.random.default_rng(seed).permutation(total_pages + 7)[:total_pages]
    pt = np.zeros((nu, max_pages), np.int32)
    o = 0
    for i, r in enumerate(rows_u):
        n = (r + P - 1) // P
        pt[i, :n] = perm[o:o + n] * P
        o += n
    pool_rows = (total_pages + 7) * P
    dt = pre["k"].dtype
    kpool = torch.zeros((pool_rows, d), dtype=dt, device="cuda")
    vpool = torch.zeros_like(kpool)
    pt_d = cu(pt)
    e_d = cu(np.array(e_cnt, np.int32))
    # receive the selected rows
    row_off_k = np.cumsum([0] + k_cnt).astype(np.int32)
    slot_gpu = np.array([(layer * cfg.Hkv + h) * K + cu_k[b] for (h, b) in units], np.int64)
    slot_ref = np.array([h * K + cu_k[b] for (h, b) in units], np.int64)
    gpu_lib.sg_fetch(cu(row_off_k), int(row_off_k[-1]), None, None, cu(slot_gpu, dtype=torch.int64), kp_t, vp_t,
                     pt_d, P, e_d, kpool, vpool)
    # Algorithm 1 on the step's index
    ex_h = [x.cpu().numpy() for x in ex]
    kv_rows = [np.concatenate([ex_h[i], sel_ref[h, cu_k[b]:cu_k[b + 1]]]) for i, (h, b) in enumerate(units)]
    row_off = np.cumsum([0] + [len(r) for r in kv_rows]).astype(np.int32)
    kv_index = np.concatenate(kv_rows).astype(np.int32)
    nmax = max(lens)
    mask = np.full((nu, nmax), 2, np.int8)
    for i, (h, b) in enumerate(units):
        mask[i, sel_ref[h, cu_k[b]:cu_k[b + 1]]] = 1
        mask[i, lens[b]:] = 0
    mask_off = (np.arange(nu) * nmax).astype(np.int64)
    mask_len = np.array([lens[b] for (h, b) in units], np.int32)
    tot = int(row_off[-1])
    loc = torch.empty(tot, dtype=torch.int32, device="cuda")
    rem = torch.empty(tot, dtype=torch.int32, device="cuda")
    order = torch.empty(tot, dtype=torch.int32, device="cuda")
    nl = torch.empty(nu, dtype=torch.int32, device="cuda")
    nrm = torch.empty(nu, dtype=torch.int32, device="cuda")
    row_off_d = cu(row_off)
    gpu_lib.sg_split(row_off_d, cu(kv_index), cu(mask.ravel(), dtype=torch.int8), cu(mask_off, dtype=torch.int64),
                     cu(mask_len), 1, loc, rem, nl, nrm, out_index=order)
    # remote lane from the pinned host copy of the prompt's K / V
    lk = 0 if cfg.kv_shared_layers else layer
    src_base = np.array([(lk * cfg.Hkv + h) * pre["T"] + cu_s[b] for (h, b) in units], np.int64)
    gpu_lib.sg_fetch(row_off_d, tot, rem, nrm, cu(src_base, dtype=torch.int64), host_k, host_v, pt_d, P,
                     cu(np.zeros(nu, np.int32)), kpool, vpool)
    torch.cuda.synchronize()
    # the oracle walks the same steps on its own data
    r_out, r_loc, r_rem, r_nl, r_nr = oracle.split(row_off, kv_index, mask.ravel(), mask_off, mask_len, 1)
    np.testing.assert_array_equal(order.cpu().numpy(), r_out)
    np.testing.assert_array_equal(loc.cpu().numpy(), r_loc)
    np.testing.assert_array_equal(rem.cpu().numpy(), r_rem)
    np.testing.assert_array_equal(nl.cpu().numpy(), r_nl)
    np.testing.assert_array_equal(nrm.cpu().numpy(), r_nr)
    assert list(r_nr) == e_cnt and list(r_nl) == k_cnt
    nd = np.uint16 if dt == torch.bfloat16 else np.float32
    okp = np.zeros((pool_rows, d), nd)
    ovp = np.zeros_like(okp)
    oracle.fetch(row_off_k, None, None, slot_ref, kr_l, vr_l, pt, P, np.array(e_cnt, np.int32), okp, ovp)
    oracle.fetch(row_off, r_rem, r_nr, src_base, raw(host_k).reshape(-1, d), raw(host_v).reshape(-1, d),
                 pt, P, np.zeros(nu, np.int32), okp, ovp)
    assert np.array_equal(raw(kpool), okp) and np.array_equal(raw(vpool), ovp)
    # decode: sequence b, KV head h
    q = inputs.decode_queries(cfg, step, device="cuda", mu=pre["mu"])[:, layer].contiguous()   # [B][Hq][d]
    ptd = np.zeros((cfg.B, cfg.Hkv, max_pages), np.int32)
    nrd = np.zeros((cfg.B, cfg.Hkv), np.int32)
    for i, (h, b) in enumerate(units):
        ptd[b, h] = pt[i]
        nrd[b, h] = rows_u[i]
    _decode_check(gpu_lib, q, kpool, vpool, cu(ptd), cu(nrd), P, rows_as_f32(okp, dt), rows_as_f32(ovp, dt), ptd)


def _layer_rows(kr, vr, i, cfg, K):
    n = cfg.Hkv * K
    return kr[i * n:(i + 1) * n], vr[i * n:(i + 1) * n]


@pytest.mark.parametrize("seed", [None, 103])
def test_llama8b_32k_long_context(gpu_lib, seed):
    cfg = _seeded(configs.get("llama8b_32k"), seed)
    say("workload llama8b_32k", "seed", cfg.seed)
    pre = inputs.make_prefill(cfg, device="cuda")
    bud = inputs.make_budget(cfg, pre["seqlens"])
    K = bud["K_total"]
    _score_units(gpu_lib, cfg, pre, [(3, 2)])
    layers = (0, 31)
    idx, ref_idx = _topk_exact(gpu_lib, cfg, pre, bud, levels=50, layers=layers)
    dst, kr, vr = _pack_exact(gpu_lib, cfg, pre, bud, idx, ref_idx, layers=layers)
    kp, vp = _pools(dst, cfg, K, torch.bfloat16)
    host_k = pre["k"].cpu().pin_memory()
    host_v = pre["v"].cpu().pin_memory()
    for i, (layer, step) in enumerate(zip(layers, (0, cfg.steps - 1))):
        say("llama8b_32k decode layer", layer, "step", step)
        kl, vl = _layer_rows(kr, vr, i, cfg, K)
        _paged_decode_layer(gpu_lib, cfg, pre, bud, layer, step, ref_idx[i], kl, vl, kp, vp, host_k, host_v,
                            3 + layer)


# ----------------------------------------------------------------------------- 70B-shaped slice, pinned-host staging

@pytest.mark.parametrize("seed", [None, 104])
def test_llama70b_16k_staging(gpu_lib, seed):
    cfg = _seeded(configs.get("llama70b_16k"), seed)
    say("workload llama70b_16k", "seed", cfg.seed)
    pre = inputs.make_prefill(cfg, device="cuda")
    bud = inputs.make_budget(cfg, pre["seqlens"])
    K = bud["K_total"]
    _score_units(gpu_lib, cfg, pre, [(0, 0), (79, 7)])
    layers = (0, 40, 79)
    idx, ref_idx = _topk_exact(gpu_lib, cfg, pre, bud, layers=layers)
    staged, kr, vr = _pack_exact(gpu_lib, cfg, pre, bud, idx, ref_idx, pinned=True, layers=layers)
    # the decode side copies the staged buffer into its HBM and attends over it
    dst = staged.to("cuda")
    kp, vp = _pools(dst, cfg, K, torch.bfloat16)
    pt = _contiguous_table(cfg.L, cfg.Hkv, K, cfg.page_size)
    nr = torch.full((cfg.L, cfg.Hkv), K, dtype=torch.int32, device="cuda")
    q = inputs.decode_queries(cfg, 0, device="cuda", mu=pre["mu"])[0].contiguous()
    ref_pt = _contiguous_table(len(layers), cfg.Hkv, K, cfg.page_size, device="cpu").numpy()
    _decode_check(gpu_lib, q, kp, vp, pt, nr, cfg.page_size, bf16_bits_to_f32(kr), bf16_bits_to_f32(vr), ref_pt,
                  seqs=layers)


# ----------------------------------------------------------------------------- 64 varlen requests, paged

@pytest.mark.parametrize("seed", [None, 105])
def test_batched64_paged(gpu_lib, seed):
    cfg = _seeded(configs.get("batched64"), seed)
    say("workload batched64", "seed", cfg.seed)
    pre = inputs.make_prefill(cfg, device="cuda")
    lens = pre["seqlens"]
    assert min(lens) >= 2048 and max(lens) <= 32768
    bud = inputs.make_budget(cfg, lens)
    K = bud["K_total"]
    # scores of every layer (all read one K source); the oracle on sampled (layer, head, request)
    T = pre["T"]
    ws = torch.empty(gpu_lib.score_workspace_size(cfg.B, cfg.L, cfg.Hq, cfg.Hkv, cfg.d, cfg.W, max(lens)),
                     dtype=torch.uint8, device="cuda")
    scores = torch.full((cfg.L, cfg.Hkv, T), float("nan"), device="cuda")
    gpu_lib.sg_score(pre["q_win"], pre["k"], cu(pre["cu_seqlens"]), T, max(lens), cfg.Hkv, scores, ws=ws)
    torch.cuda.synchronize()
    c = pre["cu_seqlens"]
    for (l, h, b) in ((0, 0, 0), (31, 7, 63), (12, 3, int(np.argmax(lens)))):
        say("batched64 score", l, h, b)
        q = f32(pre["q_win"][b:b + 1, l:l + 1, h * cfg.G:(h + 1) * cfg.G])
        k = f32(pre["k"][0:1, h:h + 1, c[b]:c[b + 1]])
        ref = oracle.score(q, k, [0, lens[b]], 1)
        assert_scores_close(scores[l, h, c[b]:c[b + 1]].cpu().numpy()[None, None], ref)
    del scores, ws
    layers = (0, 5, 31)
    idx, ref_idx = _topk_exact(gpu_lib, cfg, pre, bud, levels=1000, layers=layers)
    dst, kr, vr = _pack_exact(gpu_lib, cfg, pre, bud, idx, ref_idx, layers=layers)
    kp, vp = _pools(dst, cfg, K, torch.bfloat16)
    host_k = pre["k"].cpu().pin_memory()
    host_v = pre["v"].cpu().pin_memory()
    say("batched64 decode layer 5 step 0")
    kl, vl = _layer_rows(kr, vr, 1, cfg, K)
    _paged_decode_layer(gpu_lib, cfg, pre, bud, 5, 0, ref_idx[1], kl, vl, kp, vp, host_k, host_v, 11)
