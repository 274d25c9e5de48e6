"""Pins of the CPU oracle against facts that do not come from the oracle itself:
hand-worked examples (tests/golden), closed forms, invariants, special cases
that reduce to a library routine, and brute force on tiny inputs."""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _rand(shape, seed, scale=1.0):
    g = np.random.default_rng(seed)
    return (g.standard_normal(shape) * scale).astype(np.float32)


# ----------------------------------------------------------------------------- score

def test_score_worked_examples():
    for case in _golden("score_worked.json")["cases"]:
        G, W, d = case["G"], case["W"], case["d"]
        q = np.array(case["q"], dtype=np.float32)[None, None]          # [B=1][L=1][Hq=G][W][d]
        k = np.array(case["k"], dtype=np.float32)[None, None]          # [L][Hkv=1][T][d]
        N = k.shape[2]
        s = oracle.score(q, k, [0, N], Hkv=1)
        # inputs pass through float32 (ln 2, ln 3 round at ~3e-8 relative)
        np.testing.assert_allclose(s[0, 0], case["expect"], rtol=1e-7, atol=0, err_msg=case["name"])


def test_score_rows_sum_to_GW():
    # every window row is a probability distribution, so a unit's scores add up to G*W
    B, L, Hq, Hkv, W, d = 2, 2, 6, 2, 5, 16
    lens = [37, 21]
    cu = [0, 37, 58]
    q = _rand((B, L, Hq, W, d), 1)
    k = _rand((L, Hkv, cu[-1], d), 2)
    s = oracle.score(q, k, cu, Hkv)
    G = Hq // Hkv
    for l in range(L):
        for h in range(Hkv):
            for b in range(B):
                tot = s[l, h, cu[b]:cu[b + 1]].sum()
                assert abs(tot - G * W) <= 1e-9 * G * W
            assert (s[l, h] >= 0).all()


def test_score_equal_keys_closed_form():
    # all keys equal: row at position p spreads 1/(p+1) over keys 0..p
    B, L, Hq, Hkv, W, d, N = 1, 1, 4, 2, 7, 8, 19
    q = _rand((B, L, Hq, W, d), 3)
    row = _rand((d,), 4)
    k = np.broadcast_to(row, (L, Hkv, N, d)).copy()
    s = oracle.score(q, k, [0, N], Hkv)
    G = Hq // Hkv
    pos = np.arange(N - W, N)
    expect = np.array([G * sum(1.0 / (p + 1) for p in pos if p >= j) for j in range(N)])
    for h in range(Hkv):
        np.testing.assert_allclose(s[0, h], expect, rtol=1e-12)


def test_score_causal_and_window_match_torch_softmax():
    # special case reducing to a library routine: the window rows are the last W rows
    # of the full causal attention-probability matrix (torch.softmax in fp64)
    B, L, Hq, Hkv, d = 2, 2, 8, 2, 32
    W = 6
    lens = [29, 40]
    cu = [0, 29, 69]
    G = Hq // Hkv
    q = _rand((B, L, Hq, W, d), 5)
    k = _rand((L, Hkv, cu[-1], d), 6)
    s = oracle.score(q, k, cu, Hkv)
    for b in range(B):
        N = lens[b]
        for l in range(L):
            # full query matrix: random rows for non-window positions, the window rows at the end
            qfull = torch.from_numpy(_rand((Hq, N, d), 100 + b * 10 + l)).double()
            qfull[:, N - W:] = torch.from_numpy(q[b, l]).double()
            kk = torch.from_numpy(k[l, :, cu[b]:cu[b + 1]]).double()
            kk = kk.repeat_interleave(G, dim=0)                      # q head g reads KV head g // G
            logits = qfull @ kk.transpose(1, 2) / math.sqrt(d)
            causal = torch.ones(N, N, dtype=torch.bool).tril()
            p = torch.softmax(logits.masked_fill(~causal, float("-inf")), dim=-1)
            colsum = p[:, N - W:].sum(dim=1)                         # [Hq][N]
            expect = colsum.view(Hkv, G, N).sum(dim=1).numpy()
            np.testing.assert_allclose(s[l, :, cu[b]:cu[b + 1]], expect, rtol=1e-10, atol=1e-14)


def test_score_window_equals_prompt_reduces_to_full_causal():
    B, L, Hq, Hkv, d, N = 1, 1, 2, 1, 8, 12
    q = _rand((B, L, Hq, N, d), 7)
    k = _rand((L, Hkv, N, d), 8)
    s = oracle.score(q, k, [0, N], Hkv)
    qq = torch.from_numpy(q[0, 0]).double()
    kk = torch.from_numpy(k[0, 0]).double()
    causal = torch.ones(N, N, dtype=torch.bool).tril()
    p = torch.softmax((qq @ kk.T / math.sqrt(d)).masked_fill(~causal, float("-inf")), dim=-1)
    np.testing.assert_allclose(s[0, 0], p.sum(dim=(0, 1)).numpy(), rtol=1e-10)


def test_score_aligned_heavy_key_takes_almost_all_mass():
    B, L, Hq, Hkv, W, d, N = 1, 1, 4, 1, 8, 16, 64
    q = np.zeros((B, L, Hq, W, d), dtype=np.float32)
    q[..., 0] = 10.0
    k = _rand((L, Hkv, N, d), 9, 0.01)
    k[0, 0, 20, 0] = 10.0                  # before the window: every row sees it
    s = oracle.score(q, k, [0, N], Hkv)
    assert s[0, 0, 20] > 4 * 8 * (1 - 1e-6)
    assert s[0, 0, 20] <= 4 * 8


def test_score_last_key_only_seen_by_last_row():
    B, L, Hq, Hkv, W, d, N = 1, 1, 1, 1, 4, 8, 30
    q = _rand((B, L, Hq, W, d), 10)
    k = _rand((L, Hkv, N, d), 11)
    s = oracle.score(q, k, [0, N], Hkv)
    z = k[0, 0].astype(np.float64) @ q[0, 0, 0, W - 1].astype(np.float64) / math.sqrt(d)
    p_last = np.exp(z[-1] - z.max()) / np.exp(z - z.max()).sum()
    np.testing.assert_allclose(s[0, 0, -1], p_last, rtol=1e-12)


def test_score_shared_layer_source():
    # a layer stride of 0 rows means every layer reads the same K
    B, L, Hq, Hkv, W, d, N = 1, 3, 2, 1, 3, 8, 10
    q = _rand((B, L, Hq, W, d), 12)
    k1 = _rand((1, Hkv, N, d), 13)
    s_shared = oracle.score(q, k1, [0, N], Hkv, k_layer_rows=0)
    k3 = np.repeat(k1, L, axis=0)
    s_full = oracle.score(q, k3, [0, N], Hkv)
    np.testing.assert_array_equal(s_shared, s_full)


def test_score_rejects_window_longer_than_prompt():
    q = _rand((1, 1, 1, 5, 4), 1)
    k = _rand((1, 1, 4, 4), 2)
    with pytest.raises(ValueError):
        oracle.score(q, k, [0, 4], 1)


# ----------------------------------------------------------------------------- topk

def _brute_topk(s, k):
    s = np.asarray(s, dtype=np.float32)
    key = np.where(np.isnan(s), -np.inf, s).astype(np.float64)
    nan = np.isnan(s)
    # lexsort: last key is primary -> (nan last, -score, index)
    order = np.lexsort((np.arange(len(s)), -key, nan))
    return np.sort(order[:k])


def test_topk_worked_example():
    g = _golden("topk_worked.json")
    s = np.array([float(x) for x in g["scores"]], dtype=np.float32)
    N = len(s)
    for kk, expect in g["expect"].items():
        kk = int(kk)
        out = oracle.topk(s[None, None], [0, N], [0, kk])
        np.testing.assert_array_equal(out[0, 0], expect)


@pytest.mark.parametrize("levels", [0, 3, 50])
def test_topk_brute_force(levels):
    g = np.random.default_rng(levels)
    lens = [1, 15, 16, 17, 200]
    cu = np.cumsum([0] + lens)
    L, Hkv = 2, 3
    s = g.random((L, Hkv, cu[-1])).astype(np.float32)
    if levels:
        s = (np.floor(s * levels) / levels).astype(np.float32)
    ks = [1, 7, 16, 1, 50]
    ck = np.cumsum([0] + ks)
    out = oracle.topk(s, cu, ck)
    for l in range(L):
        for h in range(Hkv):
            for b in range(len(lens)):
                row = s[l, h, cu[b]:cu[b + 1]]
                got = out[l, h, ck[b]:ck[b + 1]]
                np.testing.assert_array_equal(got, _brute_topk(row, ks[b]))
                # invariants: k distinct ascending, selected >= unselected, ties go low
                assert len(set(got.tolist())) == ks[b] and (np.diff(got) > 0).all()
                mask = np.zeros(len(row), bool)
                mask[got] = True
                if (~mask).any():
                    assert row[mask].min() >= row[~mask].max()
                    thr = row[mask].min()
                    tied_sel = np.nonzero(mask & (row == thr))[0]
                    tied_unsel = np.nonzero(~mask & (row == thr))[0]
                    if len(tied_unsel):
                        assert tied_sel.max() < tied_unsel.min()


def test_topk_all_equal_is_address_prefix():
    # equal scores select the first k tokens in address order (the paper's partial-transfer baseline)
    N, k = 100, 13
    s = np.full((1, 1, N), 0.25, dtype=np.float32)
    out = oracle.topk(s, [0, N], [0, k])
    np.testing.assert_array_equal(out[0, 0], np.arange(k))


def test_topk_full_budget_selects_everything():
    N = 33
    s = np.random.default_rng(0).random((1, 2, N)).astype(np.float32)
    out = oracle.topk(s, [0, N], [0, N])
    np.testing.assert_array_equal(out[0, 0], np.arange(N))
    np.testing.assert_array_equal(out[0, 1], np.arange(N))


def test_topk_rejects_k_above_n():
    s = np.zeros((1, 1, 4), dtype=np.float32)
    with pytest.raises(ValueError):
        oracle.topk(s, [0, 4], [0, 5])


# ----------------------------------------------------------------------------- pack

def test_pack_worked_example():
    g = _golden("pack_worked.json")
    k = np.array(g["k"], dtype=np.float32)[None, None]
    v = np.array(g["v"], dtype=np.float32)[None, None]
    idx = np.array(g["idx"], dtype=np.int32)[None, None]
    buf = oracle.pack(k, v, idx, [0, 4], [0, 2])
    S, d = 2, 2
    kr = buf[:S * d * 4].view(np.float32).reshape(S, d)
    vr = buf[S * d * 4:2 * S * d * 4].view(np.float32).reshape(S, d)
    ir = buf[2 * S * d * 4:].view(np.int32)
    np.testing.assert_array_equal(kr, g["expect_k_rows"])
    np.testing.assert_array_equal(vr, g["expect_v_rows"])
    np.testing.assert_array_equal(ir, g["expect_idx"])


@pytest.mark.parametrize("dtype", [np.float32, np.uint16])
def test_pack_slots_are_source_rows(dtype):
    g = np.random.default_rng(1)
    L, Hkv, d = 3, 2, 8
    lens = [10, 3, 25]
    cu = np.cumsum([0] + lens)
    ks = [4, 3, 1]
    ck = np.cumsum([0] + ks)
    T = cu[-1]
    if dtype == np.uint16:
        k = g.integers(0, 65535, (L, Hkv, T, d), dtype=np.uint16)
        v = g.integers(0, 65535, (L, Hkv, T, d), dtype=np.uint16)
    else:
        k = g.standard_normal((L, Hkv, T, d)).astype(np.float32)
        v = g.standard_normal((L, Hkv, T, d)).astype(np.float32)
    idx = np.zeros((L, Hkv, ck[-1]), dtype=np.int32)
    for l in range(L):
        for h in range(Hkv):
            for b in range(3):
                idx[l, h, ck[b]:ck[b + 1]] = np.sort(g.choice(lens[b], ks[b], replace=False))
    buf = oracle.pack(k, v, idx, cu, ck)
    S = L * Hkv * ck[-1]
    rb = d * k.dtype.itemsize
    kr = buf[:S * rb].view(k.dtype).reshape(L, Hkv, ck[-1], d)
    vr = buf[S * rb:2 * S * rb].view(k.dtype).reshape(L, Hkv, ck[-1], d)
    ir = buf[2 * S * rb:].view(np.int32).reshape(L, Hkv, ck[-1])
    for l in range(L):
        for h in range(Hkv):
            for b in range(3):
                for i in range(ks[b]):
                    s = ck[b] + i
                    t = idx[l, h, s]
                    assert kr[l, h, s].tobytes() == k[l, h, cu[b] + t].tobytes()
                    assert vr[l, h, s].tobytes() == v[l, h, cu[b] + t].tobytes()
    np.testing.assert_array_equal(ir, idx)


def test_pack_full_selection_is_concatenation():
    # k = N with idx = 0..N-1 reproduces the source: the full-transfer baseline
    g = np.random.default_rng(2)
    L, Hkv, N, d = 2, 2, 9, 4
    k = g.standard_normal((L, Hkv, N, d)).astype(np.float32)
    v = g.standard_normal((L, Hkv, N, d)).astype(np.float32)
    idx = np.broadcast_to(np.arange(N, dtype=np.int32), (L, Hkv, N)).copy()
    buf = oracle.pack(k, v, idx, [0, N], [0, N])
    S = L * Hkv * N
    assert buf[:S * d * 4].tobytes() == k.tobytes()
    assert buf[S * d * 4:2 * S * d * 4].tobytes() == v.tobytes()


def test_pack_invalid_index_gives_zero_row():
    k = np.ones((1, 1, 4, 2), dtype=np.float32)
    idx = np.array([[[4, -1, 2]]], dtype=np.int32)
    buf = oracle.pack(k, k, idx, [0, 4], [0, 3])
    kr = buf[:3 * 8].view(np.float32).reshape(3, 2)
    np.testing.assert_array_equal(kr, [[0, 0], [0, 0], [1, 1]])


# ----------------------------------------------------------------------------- split (Algorithm 1)

def _split_inputs(rows):
    masks = [np.array(r["mask"], np.int8) for r in rows]
    idxs = [np.array(r["kv_index"], np.int32) for r in rows]
    row_off = np.cumsum([0] + [len(i) for i in idxs]).astype(np.int32)
    mask_off = np.cumsum([0] + [len(m) for m in masks])[:-1].astype(np.int64)
    mask_len = np.array([len(m) for m in masks], np.int32)
    return row_off, np.concatenate(idxs), np.concatenate(masks), mask_off, mask_len


@pytest.mark.parametrize("reorder", [0, 1])
def test_split_worked_example(reorder):
    rows = _golden("split_worked.json")["rows"]
    row_off, ix, m, mo, ml = _split_inputs(rows)
    out, loc, rem, nl, nr = oracle.split(row_off, ix, m, mo, ml, reorder)
    for r, row in enumerate(rows):
        o = row_off[r]
        assert nl[r] == len(row["local"]) and nr[r] == len(row["remote"])
        np.testing.assert_array_equal(loc[o:o + nl[r]], row["local"])
        np.testing.assert_array_equal(rem[o:o + nr[r]], row["remote"])
        if reorder:
            np.testing.assert_array_equal(out[o:row_off[r + 1]], row["reordered"])


def test_split_brute_force_and_invariants():
    g = np.random.default_rng(3)
    rows, N = 40, 64
    n = g.integers(0, 30, rows)
    row_off = np.cumsum([0] + list(n)).astype(np.int32)
    mask = g.integers(0, 3, rows * N).astype(np.int8)
    mask[g.random(rows * N) < 0.02] = 7                  # invalid codes count as pads
    mo = (np.arange(rows) * N).astype(np.int64)
    ml = np.full(rows, N, np.int32)
    ix = np.concatenate([g.integers(-2, N + 2, k) for k in n]).astype(np.int32)
    out, loc, rem, nl, nr = oracle.split(row_off, ix, mask, mo, ml, 1)
    for r in range(rows):
        seg = ix[row_off[r]:row_off[r + 1]]
        valid = (seg >= 0) & (seg < N)
        m = np.where(valid, mask[r * N + np.clip(seg, 0, N - 1)], 0)
        m = np.where((m == 1) | (m == 2), m, 0)
        o = row_off[r]
        np.testing.assert_array_equal(loc[o:o + nl[r]], seg[m == 1])
        np.testing.assert_array_equal(rem[o:o + nr[r]], seg[m == 2])
        order = np.argsort(-m, kind="stable")
        np.testing.assert_array_equal(out[o:row_off[r + 1]], seg[order])
        assert nl[r] + nr[r] + (m == 0).sum() == len(seg)
        assert (loc[o + nl[r]:row_off[r + 1]] == -1).all()


def test_split_all_local_and_all_remote():
    N = 10
    ix = np.arange(N, dtype=np.int32)
    for code, want_local in ((1, True), (2, False)):
        mask = np.full(N, code, np.int8)
        _, loc, rem, nl, nr = oracle.split([0, N], ix, mask, [0], [N], 0)
        if want_local:
            assert nl[0] == N and nr[0] == 0
        else:
            assert nl[0] == 0 and nr[0] == N


# ----------------------------------------------------------------------------- fetch

def test_fetch_paged_destination_brute_force():
    g = np.random.default_rng(4)
    d, P, rows = 4, 4, 5
    src_rows = 100
    ks = g.standard_normal((src_rows, d)).astype(np.float32)
    vs = g.standard_normal((src_rows, d)).astype(np.float32)
    n = g.integers(0, 9, rows)
    row_off = np.cumsum([0] + list(n)).astype(np.int32)
    index = g.integers(0, 20, row_off[-1]).astype(np.int32)
    n_valid = np.minimum(n, g.integers(0, 9, rows)).astype(np.int32)
    src_base = (np.arange(rows) * 20).astype(np.int64)
    max_pages = 5
    pool_rows = 128
    pages = g.permutation(pool_rows // P)[:rows * max_pages].reshape(rows, max_pages) * P
    dst_start = g.integers(0, 6, rows).astype(np.int32)
    kp = np.zeros((pool_rows, d), np.float32)
    vp = np.zeros((pool_rows, d), np.float32)
    oracle.fetch(row_off, index, n_valid, src_base, ks, vs, pages, P, dst_start, kp, vp)
    ek = np.zeros_like(kp)
    ev = np.zeros_like(vp)
    for r in range(rows):
        for i in range(n_valid[r]):
            t = index[row_off[r] + i]
            lr = dst_start[r] + i
            dst = pages[r, lr // P] + lr % P
            ek[dst] = ks[src_base[r] + t]
            ev[dst] = vs[src_base[r] + t]
    np.testing.assert_array_equal(kp, ek)
    np.testing.assert_array_equal(vp, ev)


def test_fetch_identity_index_and_bounds():
    d = 2
    ks = np.arange(20, dtype=np.float32).reshape(10, d)
    kp = np.zeros((4, d), np.float32)
    vp = np.zeros((4, d), np.float32)
    # 6 entries starting at logical row 0 of a 1-page (4-row) destination: entries 4,5 fall off the table
    oracle.fetch([0, 6], None, None, [3], ks, ks, [[0]], 4, [0], kp, vp)
    np.testing.assert_array_equal(kp, ks[3:7])


# ----------------------------------------------------------------------------- decode attention

def test_decode_worked_example():
    g = _golden("decode_worked.json")
    q = np.array(g["q"], np.float32)[None]                      # [B=1][Hq=2][d]
    pt = np.array(g["page_table"], np.int32)[None, None]       # [B][Hkv=1][pages]
    o = oracle.decode_attn(q, np.array(g["pool_k"], np.float32), np.array(g["pool_v"], np.float32),
                           pt, np.array([[g["n_rows"]]], np.int32), 1, scale=g["scale"])
    np.testing.assert_allclose(o[0], g["expect"], rtol=1e-7, atol=1e-12)


def _dense_case(seed, B=2, Hq=8, Hkv=2, d=16, N=37, P=4):
    g = np.random.default_rng(seed)
    q = g.standard_normal((B, Hq, d)).astype(np.float32)
    kd = g.standard_normal((B, Hkv, N, d)).astype(np.float32)
    vd = g.standard_normal((B, Hkv, N, d)).astype(np.float32)
    npg = (N + P - 1) // P
    # scatter the dense rows into a pool through shuffled pages
    pages = g.permutation(B * Hkv * npg).reshape(B, Hkv, npg)
    kp = np.zeros((B * Hkv * npg * P, d), np.float32)
    vp = np.zeros_like(kp)
    for b in range(B):
        for h in range(Hkv):
            for i in range(N):
                r = pages[b, h, i // P] * P + i % P
                kp[r] = kd[b, h, i]
                vp[r] = vd[b, h, i]
    return q, kd, vd, kp, vp, (pages * P).astype(np.int32), np.full((B, Hkv), N, np.int32)


def test_decode_full_selection_equals_dense_sdpa():
    q, kd, vd, kp, vp, pt, nr = _dense_case(5)
    o = oracle.decode_attn(q, kp, vp, pt, nr, 4)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).double()[:, :, None], torch.from_numpy(kd).double(),
        torch.from_numpy(vd).double(), enable_gqa=True)[:, :, 0]
    np.testing.assert_allclose(o, ref.numpy(), rtol=1e-12, atol=1e-12)


def test_decode_page_order_does_not_matter():
    q, kd, vd, kp, vp, pt, nr = _dense_case(6, N=32)           # whole pages only
    o1 = oracle.decode_attn(q, kp, vp, pt, nr, 4)
    g = np.random.default_rng(0)
    pt2 = pt.copy()
    for b in range(pt.shape[0]):
        for h in range(pt.shape[1]):
            pt2[b, h] = pt[b, h][g.permutation(pt.shape[2])]
    o2 = oracle.decode_attn(q, kp, vp, pt2, nr, 4)
    np.testing.assert_allclose(o1, o2, rtol=1e-12, atol=1e-12)


def test_decode_single_row_returns_its_value_and_equal_keys_average():
    g = np.random.default_rng(7)
    d = 8
    kp = g.standard_normal((10, d)).astype(np.float32)
    vp = g.standard_normal((10, d)).astype(np.float32)
    q = g.standard_normal((1, 1, d)).astype(np.float32)
    o = oracle.decode_attn(q, kp, vp, np.array([[[6]]], np.int32), np.array([[1]], np.int32), 1)
    np.testing.assert_allclose(o[0, 0], vp[6], rtol=0, atol=0)
    kp[:] = kp[0]
    o = oracle.decode_attn(q, kp, vp, np.array([[[2, 5, 7]]], np.int32), np.array([[3]], np.int32), 1)
    np.testing.assert_allclose(o[0, 0], vp[[2, 5, 7]].astype(np.float64).mean(0), rtol=1e-12, atol=1e-14)


def test_decode_empty_set_is_zero():
    q = np.ones((1, 2, 4), np.float32)
    o = oracle.decode_attn(q, np.ones((4, 4), np.float32), np.ones((4, 4), np.float32),
                           np.zeros((1, 1, 1), np.int32), np.zeros((1, 1), np.int32), 4)
    assert (o == 0).all()


# ----------------------------------------------------------------------------- block mode (eq. 1, eq. 2)

def _fl(x):
    return float(x)                      # "inf" and "-inf" parse to the infinities


def test_block_importance_worked_examples():
    for case in _golden("block_worked.json")["importance"]:
        L, Hkv, N, M = case["L"], case["Hkv"], case["N"], case["M"]
        sc = np.arange(L * Hkv * N, dtype=np.float32).reshape(L, Hkv, N)
        got = oracle.block_importance(sc, [0, N], M)[0]
        want = np.array([[_fl(x) for x in row] for row in case["expect"]])
        np.testing.assert_array_equal(got, want, err_msg=case["name"])


def test_block_importance_is_reshape_mean_when_blocks_divide():
    L, Hkv, M, Nb = 4, 3, 8, 5
    N = M * Nb
    sc = _rand((L, Hkv, N), 11)
    got = oracle.block_importance(sc, [0, N], M)[0]
    want = sc.astype(np.float64).reshape(L, Hkv, M, Nb).mean(axis=(1, 3))
    assert np.isinf(got[:2]).all() and (got[:2] > 0).all()
    np.testing.assert_allclose(got[2:], want[2:], rtol=1e-12)


def test_block_importance_size_weighted_sum_is_total_varlen():
    L, Hkv, M = 3, 2, 7
    lens = [23, 5, 7]                                  # blocks of 4, 1 and 1 tokens; 23 leaves a short last block
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    sc = _rand((L, Hkv, int(cu[-1])), 12)
    imp = oracle.block_importance(sc, cu, M)
    for b, N in enumerate(lens):
        Nb = -(-N // M)
        sizes = np.array([max(0, min(N, (m + 1) * Nb) - m * Nb) for m in range(M)])
        for l in range(2, L):
            tot = sc[l, :, cu[b]:cu[b + 1]].astype(np.float64).sum()
            finite = sizes > 0
            assert (imp[b, l, ~finite] == -np.inf).all()
            np.testing.assert_allclose((imp[b, l, finite] * sizes[finite] * Hkv).sum(), tot, rtol=1e-9, atol=1e-9)


def test_block_budget_worked_and_first_form_of_eq2():
    for case in _golden("block_worked.json")["budget"]:
        assert oracle.block_budget(case["M"], case["L"], case["Tp"], case["Tt"]) == case["expect"], case
    # eq. 2 written as L*M*((L-1)/L * Tp/Tt) gives the same count before the clip
    for M, L, r in [(1024, 32, 0.154), (512, 80, 0.07), (1024, 40, 0.9)]:
        first = L * M * ((L - 1) / L * r)
        k = oracle.block_budget(M, L, r, 1.0)
        assert k == min(L * M, max(2 * M, math.floor(first + 1e-9))) or k == min(L * M, max(2 * M, math.floor(first)))


def test_block_selection_keeps_first_two_layers_and_ranks_the_rest():
    L, Hkv, M, N = 6, 2, 16, 100
    sc = _rand((L, Hkv, N), 13) ** 2
    imp = oracle.block_importance(sc, [0, N], M)            # [1][L][M]
    Kr = oracle.block_budget(M, L, 0.3, 1.0)                 # floor(16 * 5 * 0.3) = 24 -> clipped to 32
    assert Kr == 2 * M
    row = imp.reshape(1, 1, L * M).astype(np.float32)
    for kr in (Kr, 2 * M + 5, L * M - 3):
        sel = oracle.topk(row, [0, L * M], [0, kr])[0, 0]
        assert set(range(2 * M)) <= set(sel.tolist())      # layers 0 and 1 always go
        rest = np.array(sorted(range(2 * M, L * M), key=lambda c: (-row[0, 0, c], c)))
        np.testing.assert_array_equal(np.sort(sel), np.sort(np.concatenate([np.arange(2 * M), rest[:kr - 2 * M]])))


def test_pack_blocks_worked_example():
    c = _golden("block_worked.json")["pack"]
    k = np.array(c["k"], dtype=np.float32)
    v = np.array(c["v"], dtype=np.float32)
    buf = oracle.pack_blocks(k, v, c["ids"], 0, c["N"], c["M"])
    S = len(c["expect_k"])
    d = c["d"]
    kr = buf[:S * d * 4].view(np.float32).reshape(S, d)
    vr = buf[S * d * 4:2 * S * d * 4].view(np.float32).reshape(S, d)
    ids = buf[2 * S * d * 4:].view(np.int32)
    np.testing.assert_array_equal(kr, np.array(c["expect_k"], dtype=np.float32))
    np.testing.assert_array_equal(vr, np.array(c["expect_v"], dtype=np.float32))
    np.testing.assert_array_equal(ids, c["ids"])


@pytest.mark.parametrize("dtype", [np.float32, np.uint16])
def test_pack_blocks_slots_are_source_rows(dtype):
    L, Hkv, d, M = 3, 2, 8, 5
    lens = [13, 9]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    g = np.random.default_rng(14)
    k = g.integers(0, 60000, (L, Hkv, T, d)).astype(dtype)
    v = g.integers(0, 60000, (L, Hkv, T, d)).astype(dtype)
    b, N = 0, lens[0]
    Nb = -(-N // M)
    ids = np.array([1, 7, 14, 3], dtype=np.int32)
    buf = oracle.pack_blocks(k, v, ids, cu[b], N, M)
    S = len(ids) * Hkv * Nb
    es = np.dtype(dtype).itemsize
    kr = buf[:S * d * es].view(dtype).reshape(len(ids), Hkv, Nb, d)
    vr = buf[S * d * es:2 * S * d * es].view(dtype).reshape(len(ids), Hkv, Nb, d)
    for s, c in enumerate(ids):
        l, m = divmod(int(c), M)
        for h in range(Hkv):
            for r in range(Nb):
                t = m * Nb + r
                want_k = k[l, h, cu[b] + t] if t < N else np.zeros(d, dtype)
                want_v = v[l, h, cu[b] + t] if t < N else np.zeros(d, dtype)
                np.testing.assert_array_equal(kr[s, h, r], want_k)
                np.testing.assert_array_equal(vr[s, h, r], want_v)


# ----------------------------------------------------------------------------- speculative transfer, reuse

def test_spec_push_worked_example():
    c = _golden("spec_keep_worked.json")["spec_push"]
    k = np.array(c["k_src"], dtype=np.float32)
    v = -k
    kd, vd = np.zeros_like(k), np.zeros_like(v)
    mask = np.array(c["mask_in"], dtype=np.int8)
    rem = np.array(c["rem_in"], dtype=np.float32)
    oracle.spec_push(k, v, c["ids"], c["s0"], c["N"], c["M"], kd, vd, mask, rem)
    np.testing.assert_array_equal(kd, np.array(c["expect_k"], dtype=np.float32))
    np.testing.assert_array_equal(vd, -np.array(c["expect_k"], dtype=np.float32))
    np.testing.assert_array_equal(mask, np.array(c["expect_mask"], dtype=np.int8))
    np.testing.assert_array_equal(rem, np.array([float(x) for x in c["expect_rem"]], dtype=np.float32))


@pytest.mark.parametrize("shared", [False, True])
def test_spec_push_of_every_block_delivers_the_request(shared):
    L, Hkv, d, M = 3, 2, 4, 5
    lens = [11, 7]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    g = np.random.default_rng(31)
    k = g.standard_normal((1 if shared else L, Hkv, T, d)).astype(np.float32)
    v = g.standard_normal(k.shape).astype(np.float32)
    kd = np.full((L, Hkv, T, d), 7.0, np.float32)
    vd = kd.copy()
    mask = np.full((L, Hkv, T), 2, np.int8)
    b, s0, N = 1, int(cu[1]), lens[1]
    oracle.spec_push(k, v, g.permutation(L * M), s0, N, M, kd, vd, mask, L=L, src_layer_rows=0 if shared else None)
    for l in range(L):
        src = 0 if shared else l
        np.testing.assert_array_equal(kd[l, :, s0:s0 + N], k[src, :, s0:s0 + N])
        np.testing.assert_array_equal(vd[l, :, s0:s0 + N], v[src, :, s0:s0 + N])
    assert (kd[:, :, :s0] == 7).all() and (mask[:, :, :s0] == 2).all()     # the other request is untouched
    assert (mask[:, :, s0:s0 + N] == 1).all()


def test_spec_quota_matches_the_papers_step_counts():
    # 10% delivers every block within 10 transfers, 20% within 5, 5% within 20
    for L in (32, 40, 80):
        LM = L * 1024
        for bp, steps in ((1000, 10), (2000, 5), (500, 20)):
            assert -(-LM // oracle.spec_quota(LM, bp)) == steps
    for LM in range(1, 3001):
        for bp, steps in ((1000, 10), (2000, 5), (500, 20)):
            r = oracle.spec_quota(LM, bp)
            assert 1 <= r <= LM and -(-LM // r) <= steps


def test_spec_steps_follow_the_importance_order():
    """Proactive top-K_r, then speculative transfers of the quota each: step s
    delivers exactly the blocks ranked [K_r + (s-1) r, K_r + s r) by (importance
    descending, id ascending), and the last step completes the request."""
    L, Hkv, d, M, N = 5, 2, 4, 8, 37                   # Nb = 5; block 7 of each layer holds 2 tokens
    g = np.random.default_rng(32)
    sc = (g.standard_normal((L, Hkv, N)) ** 2).astype(np.float32)
    sc[3, :, 10:15] = sc[4, :, 0:5]                    # equal blocks (ties go to the lower id)
    imp = oracle.block_importance(sc, [0, N], M)[0].reshape(-1)
    LM = L * M
    order = np.array(sorted(range(LM), key=lambda c: (-imp[c], c)))
    k = g.standard_normal((L, Hkv, N, d)).astype(np.float32)
    v = g.standard_normal(k.shape).astype(np.float32)
    kd, vd = np.zeros_like(k), np.zeros_like(v)
    mask = np.full((L, Hkv, N), 2, np.int8)
    rem = imp.astype(np.float32)
    Kr = oracle.block_budget(M, L, 0.3, 1.0)
    r = oracle.spec_quota(LM, 1000)
    done, step, quota = 0, 0, Kr
    while done < LM:
        q = min(quota, LM - done)
        sel = oracle.topk(rem.reshape(1, 1, LM), [0, LM], [0, q])[0, 0]
        np.testing.assert_array_equal(np.sort(sel), np.sort(order[done:done + q]))
        oracle.spec_push(k, v, sel, 0, N, M, kd, vd, mask, rem)
        done += q
        step += 1
        quota = r
        pushed = np.zeros(LM, bool)
        pushed[order[:done]] = True
        assert np.isnan(rem[pushed]).all() and not np.isnan(rem[~pushed]).any()
        Nb = -(-N // M)
        for c in range(LM):
            l, m = divmod(c, M)
            toks = slice(m * Nb, min(N, (m + 1) * Nb))
            assert (mask[l, :, toks] == (1 if pushed[c] else 2)).all()
    assert step == 1 + -(-(LM - Kr) // r)
    np.testing.assert_array_equal(kd, k)
    np.testing.assert_array_equal(vd, v)


def test_fetch_keep_worked_example():
    c = _golden("spec_keep_worked.json")["fetch_keep"]
    ks = np.array(c["k_src"], dtype=np.float32)
    vs = -ks
    kp, vp = np.zeros((c["pool_rows"], 2), np.float32), np.zeros((c["pool_rows"], 2), np.float32)
    kk, vk = np.zeros((c["keep_rows"], 2), np.float32), np.zeros((c["keep_rows"], 2), np.float32)
    mask = np.array(c["mask_in"], dtype=np.int8)
    n = len(c["index"])
    oracle.fetch_keep([0, n], c["index"], None, [c["src_row_base"]], ks, vs, np.array([c["page_table"]]),
                      c["page_size"], [c["dst_start"]], kp, vp, [c["keep_row_base"]], kk, vk, mask,
                      [c["mask_off"]], [c["mask_len"]])
    np.testing.assert_array_equal(kp, np.array(c["expect_pool_k"], np.float32))
    np.testing.assert_array_equal(vp, -np.array(c["expect_pool_k"], np.float32))
    np.testing.assert_array_equal(kk, np.array(c["expect_keep_k"], np.float32))
    np.testing.assert_array_equal(vk, -np.array(c["expect_keep_k"], np.float32))
    np.testing.assert_array_equal(mask, np.array(c["expect_mask"], np.int8))


def test_fetch_keep_brute_force_and_reuse():
    """Every fetched entry lands in the pool like a plain fetch and in the store
    at its own token row, its mask entry turns local; a split of the same
    index afterwards finds no remote entry (Algorithm 1), so a later step loads
    them on the local lane."""
    g = np.random.default_rng(33)
    rows, N, d, P = 6, 50, 4, 4
    src = g.standard_normal((rows * N, d)).astype(np.float32)
    vsrc = g.standard_normal((rows * N, d)).astype(np.float32)
    mask = np.where(g.random(rows * N) < 0.6, 2, 1).astype(np.int8)
    lens = g.integers(0, 12, rows)
    row_off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    index = np.concatenate([np.sort(g.choice(N, size=n, replace=False)) for n in lens]).astype(np.int32)
    base = np.arange(rows, dtype=np.int64) * N
    mo, ml = base.copy(), np.full(rows, N, np.int32)
    _, loc, rem_idx, nl, nr = oracle.split(row_off, index, mask, mo, ml, 0)
    # fetch the remote partition only: pool pages in reverse order, store = [rows][N]
    max_pages = 4
    pt = (np.arange(rows * max_pages)[::-1].reshape(rows, max_pages) * P).astype(np.int32)
    kp = np.zeros((rows * max_pages * P, d), np.float32)
    vp = np.zeros_like(kp)
    kk = np.zeros((rows * N, d), np.float32)
    vk = np.zeros_like(kk)
    mask0 = mask.copy()
    oracle.fetch_keep(row_off, rem_idx, nr, base, src, vsrc, pt, P, np.zeros(rows, np.int32), kp, vp,
                      base, kk, vk, mask, mo, ml)
    want_mask = mask0.copy()
    for r in range(rows):
        for i in range(nr[r]):
            t = rem_idx[row_off[r] + i]
            prow = pt[r, i // P] + i % P
            np.testing.assert_array_equal(kp[prow], src[base[r] + t])
            np.testing.assert_array_equal(vp[prow], vsrc[base[r] + t])
            np.testing.assert_array_equal(kk[base[r] + t], src[base[r] + t])
            np.testing.assert_array_equal(vk[base[r] + t], vsrc[base[r] + t])
            want_mask[base[r] + t] = 1
    np.testing.assert_array_equal(mask, want_mask)
    kept = np.zeros(rows * N, bool)
    for r in range(rows):
        kept[base[r] + rem_idx[row_off[r]:row_off[r] + nr[r]]] = True
    assert (kk[~kept] == 0).all()
    _, loc2, _, nl2, nr2 = oracle.split(row_off, index, mask, mo, ml, 0)
    assert (nr2 == 0).all()
    np.testing.assert_array_equal(nl2, lens)
    np.testing.assert_array_equal(loc2, index)


# ----------------------------------------------------------------------------- selector variants

def test_score_count_worked_examples():
    for c in _golden("selector_worked.json")["count"]:
        k = np.array(c["k"], np.float32).reshape(1, 1, -1, 1)
        q = np.array(c["q"], np.float32).reshape(1, 1, 1, c["W"], 1)
        got = oracle.score_count(q, k, [0, len(c["k"])], 1, c["alpha"])
        np.testing.assert_array_equal(got[0, 0], c["expect"], err_msg=c["name"])


def _brute_counts(q, k, N, W, G, alpha):
    d = k.shape[-1]
    out = np.zeros(N, np.int64)
    for g in range(G):
        for w in range(W):
            p = N - W + w
            z = (k[:p + 1].astype(np.float64) @ q[g, w].astype(np.float64)) / math.sqrt(d)
            out[:p + 1] += z >= z.max() - alpha
    return out


@pytest.mark.parametrize("alpha", [0.5, 2.0, 5.0])
def test_score_count_brute_force(alpha):
    G, W, d, N = 3, 5, 8, 40
    q = _rand((1, 1, G, W, d), 21)
    k = _rand((1, 1, N, d), 22)
    got = oracle.score_count(q, k, [0, N], 1, alpha)[0, 0]
    np.testing.assert_array_equal(got, _brute_counts(q[0, 0], k[0, 0], N, W, G, alpha))
    assert got.sum() >= G * W                                  # every row picks at least its maximum


def test_score_count_limits():
    G, W, d, N = 2, 6, 4, 30
    q = _rand((1, 1, G, W, d), 23)
    k = _rand((1, 1, N, d), 24)
    # alpha beyond every logit gap: each row picks all it sees, G * #{w : N - W + w >= j}
    seen = np.array([G * sum(1 for w in range(W) if N - W + w >= j) for j in range(N)])
    np.testing.assert_array_equal(oracle.score_count(q, k, [0, N], 1, 1e9)[0, 0], seen)
    # equal keys tie at the maximum: the same closed form at any alpha
    keq = np.repeat(k[:, :, :1], N, axis=2)
    np.testing.assert_array_equal(oracle.score_count(q, keq, [0, N], 1, 0.0)[0, 0], seen)
    # alpha = 0 with distinct logits: each row picks its argmax only
    want = np.zeros(N, np.int64)
    for g in range(G):
        for w in range(W):
            p = N - W + w
            want[np.argmax(k[0, 0, :p + 1].astype(np.float64) @ q[0, 0, g, w].astype(np.float64))] += 1
    np.testing.assert_array_equal(oracle.score_count(q, k, [0, N], 1, 0.0)[0, 0], want)
    # the near-threshold count is exact ties when eps = 0
    _, near = oracle.score_count(q, keq, [0, N], 1, 0.0, eps=0.0)
    np.testing.assert_array_equal(near[0, 0], seen)


def test_score_topshare_worked_examples():
    for c in _golden("selector_worked.json")["topshare"]:
        k = np.array(c["k"], np.float32).reshape(1, 1, -1, 1)
        q = np.array(c["q"], np.float32).reshape(1, 1, 1, c["W"], 1)
        got = oracle.score_topshare(q, k, [0, len(c["k"])], 1, c["ratio_bp"])
        np.testing.assert_array_equal(got[0, 0], c["expect"], err_msg=c["name"])


def _brute_topshare(q, k, N, W, G, ratio_bp):
    d = k.shape[-1]
    out = np.zeros(N, np.int64)
    picked = 0
    for g in range(G):
        for w in range(W):
            n = N - W + w + 1
            z = (k[:n].astype(np.float64) @ q[g, w].astype(np.float64)) / math.sqrt(d)
            kk = min(n, max(1, n * ratio_bp // 10000))
            order = np.argsort(-z, kind="stable")
            thr = z[order[kk - 1]]
            out[:n] += z >= thr
            picked += kk
    return out, picked


@pytest.mark.parametrize("ratio_bp", [100, 2000, 5000])
def test_score_topshare_brute_force(ratio_bp):
    G, W, d, N = 3, 5, 8, 60
    q = _rand((1, 1, G, W, d), 31)
    k = _rand((1, 1, N, d), 32)
    got = oracle.score_topshare(q, k, [0, N], 1, ratio_bp)[0, 0]
    want, picked = _brute_topshare(q[0, 0], k[0, 0], N, W, G, ratio_bp)
    np.testing.assert_array_equal(got, want)
    assert got.sum() == picked                       # distinct logits: each row picks exactly its k


def test_score_topshare_limits():
    G, W, d, N = 2, 6, 4, 30
    q = _rand((1, 1, G, W, d), 33)
    k = _rand((1, 1, N, d), 34)
    seen = np.array([G * sum(1 for w in range(W) if N - W + w >= j) for j in range(N)])
    # the whole share: every row picks all it sees
    np.testing.assert_array_equal(oracle.score_topshare(q, k, [0, N], 1, 10000)[0, 0], seen)
    # equal keys all tie with the threshold: the same closed form at any share
    keq = np.repeat(k[:, :, :1], N, axis=2)
    np.testing.assert_array_equal(oracle.score_topshare(q, keq, [0, N], 1, 500)[0, 0], seen)
    # a share below one key: each row picks its argmax, as the alpha rule at alpha = 0
    np.testing.assert_array_equal(oracle.score_topshare(q, k, [0, N], 1, 100)[0, 0],
                                  oracle.score_count(q, k, [0, N], 1, 0.0)[0, 0])
    # two requests and a shared-layer source address like the single-request calls
    k2 = _rand((1, 1, 2 * N, d), 35)
    q2 = _rand((2, 3, G, W, d), 36)
    both = oracle.score_topshare(q2, k2, [0, N, 2 * N], 1, 3000)
    for b in range(2):
        for l in range(3):
            one = oracle.score_topshare(q2[b:b + 1, l:l + 1], k2[:, :, b * N:(b + 1) * N], [0, N], 1, 3000)
            np.testing.assert_array_equal(both[l, 0, b * N:(b + 1) * N], one[0, 0])


def test_decode_select_worked_examples():
    for c in _golden("selector_worked.json")["select"]:
        k = np.array(c["k"], np.float32).reshape(1, 1, -1, 1)
        q = np.array(c["q"], np.float32).reshape(1, 1, 2, 1)
        N = len(c["k"])
        idx, n, _ = oracle.decode_select(q, k, [0, N], 1, [0, c["cap"]], c["alpha"])
        assert n[0, 0, 0] == c["n"], c["name"]
        np.testing.assert_array_equal(idx[0, 0, :c["n"]], c["expect"], err_msg=c["name"])
        assert (idx[0, 0, c["n"]:] == -1).all()


@pytest.mark.parametrize("alpha,cap_frac", [(5.0, 0.2), (1.0, 1.0), (3.0, 0.05), (0.0, 0.2)])
def test_decode_select_brute_force(alpha, cap_frac):
    B, L, Hq, Hkv, d = 2, 2, 4, 2, 16
    lens = [50, 23]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    q = _rand((B, L, Hq, d), 25, scale=2.0)
    k = _rand((L, Hkv, T, d), 26)
    caps = [max(1, int(n * cap_frac)) for n in lens]
    cc = np.concatenate([[0], np.cumsum(caps)])
    idx, n_sel, r = oracle.decode_select(q, k, cu, Hkv, cc, alpha)
    G = Hq // Hkv
    for b in range(B):
        for l in range(L):
            for h in range(Hkv):
                kb = k[l, h, cu[b]:cu[b + 1]].astype(np.float64)
                z = np.stack([kb @ q[b, l, g].astype(np.float64) / math.sqrt(d) for g in range(h * G, (h + 1) * G)])
                rr = (z - z.max(axis=1, keepdims=True)).max(axis=0)
                np.testing.assert_allclose(r[l, h, cu[b]:cu[b + 1]], rr, rtol=0, atol=1e-12)
                cand = [j for j in range(lens[b]) if rr[j] >= -alpha]
                cand = sorted(cand, key=lambda j: (-rr[j], j))[:caps[b]]
                seg = idx[l, h, cc[b]:cc[b + 1]]
                assert n_sel[b, l, h] == len(cand)
                np.testing.assert_array_equal(seg[:len(cand)], sorted(cand))
                assert (seg[len(cand):] == -1).all()
                # each head's maximum passes the rule (r = 0), so at least one entry is picked
                assert n_sel[b, l, h] >= 1


def test_decode_select_partial_channels_is_a_scaled_subset():
    """Selection on a subset of channels with the full head's scale equals the
    selection of a query zeroed outside the subset (scale 1/sqrt(d_full))."""
    B, L, Hq, Hkv, d, ds = 1, 1, 4, 1, 16, 6
    N = 40
    q = _rand((B, L, Hq, d), 27, scale=3.0)
    k = _rand((L, Hkv, N, d), 28)
    qz = q.copy()
    qz[..., ds:] = 0.0
    full = oracle.decode_select(qz, k, [0, N], Hkv, [0, 9], 2.0)
    part = oracle.decode_select(q[..., :ds].copy(), k[..., :ds].copy(), [0, N], Hkv, [0, 9], 2.0, scale=d ** -0.5)
    np.testing.assert_array_equal(part[0], full[0])
    np.testing.assert_array_equal(part[1], full[1])
    np.testing.assert_allclose(part[2], full[2], rtol=0, atol=1e-12)
