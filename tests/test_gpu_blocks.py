"""GPU parity of block-granular proactive selection (Section 4.1: eq. 1 block
importance, eq. 2 block budget, the global top-K_r over the blocks, and the
block push) against the CPU oracle, through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
from datagen import inputs
from datagen.configs import get
from tests.gpu_util import assert_scores_close, assert_topk_sets_agree, cu, raw, say

pytestmark = pytest.mark.gpu


def _importance_close(gpu, ref, rtol):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    inf = np.isinf(ref)
    np.testing.assert_array_equal(gpu[inf], ref[inf])                 # +inf (layers 0, 1) and -inf (empty)
    assert_scores_close(gpu[~inf], ref[~inf], rtol=rtol)


@pytest.mark.parametrize("lens,M", [
    ((8192,), 1024),              # the paper's M: blocks of 8 tokens
    ((1000, 3, 5000), 7),         # blocks of 143 (short last), 1 (4 empty) and 715 (short last) tokens
    ((300,), 1024),               # M > N: one token per block, 724 empty blocks
    ((0, 64), 16),                # an empty request
])
def test_block_importance_parity(gpu_lib, lens, M):
    L, Hkv = 4, 8
    say("block importance", lens, M)
    g = np.random.default_rng(sum(lens) + M)
    cus = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cus[-1])
    sc = (g.standard_normal((L, Hkv, max(T, 1))) ** 2).astype(np.float32)[:, :, :T]
    sc = np.ascontiguousarray(sc)
    imp = torch.full((len(lens), L, M), float("nan"), device="cuda")
    gpu_lib.sg_block_importance(torch.from_numpy(sc).cuda(), cu(cus), T, M, imp)
    torch.cuda.synchronize()
    ref = oracle.block_importance(sc, cus, M)
    _importance_close(imp.cpu().numpy(), ref, rtol=1e-5)


@pytest.mark.parametrize("L,M,ratio,levels", [
    (32, 1024, 1 / 6.5, 0),       # llama8b shape, the paper's transfer / prefill ratio
    (80, 1024, 1 / 6.5, 0),       # 70B shape: a row of 81920 blocks
    (6, 64, 0.5, 5),              # heavy ties
    (3, 100, 10.0, 0),            # clipped to every block
])
def test_block_topk_bit_exact(gpu_lib, L, M, ratio, levels):
    say("block top-k", L, M, ratio, levels)
    g = np.random.default_rng(L * M + levels)
    B = 2
    rows = g.standard_normal((B, L, M)).astype(np.float32)
    if levels:
        rows = np.floor(rows * levels).astype(np.float32)
    rows[:, :2] = np.inf                                          # eq. 1: layers 0 and 1
    rows[1, -1, -3:] = -np.inf                                    # empty blocks
    Kr = gpu_lib.block_budget(M, L, ratio, 1.0)
    assert Kr == oracle.block_budget(M, L, ratio, 1.0)
    cus = np.arange(B + 1, dtype=np.int32) * (L * M)
    cuk = np.arange(B + 1, dtype=np.int32) * Kr
    flat = rows.reshape(1, 1, B * L * M)
    ids = torch.empty((1, 1, B * Kr), dtype=torch.int32, device="cuda")
    gpu_lib.sg_topk(torch.from_numpy(flat).cuda(), cu(cus), B * L * M, L * M, cu(cuk), B * Kr, ids)
    torch.cuda.synchronize()
    ref = oracle.topk(flat, cus, cuk)
    np.testing.assert_array_equal(ids.cpu().numpy(), ref)
    for b in range(B):
        assert set(range(2 * M)) <= set(ref[0, 0, b * Kr:(b + 1) * Kr].tolist())


@pytest.mark.parametrize("dtype,d,lens,M,shared", [
    ("bf16", 128, (8192,), 1024, False),
    ("bf16", 64, (1000, 37), 7, False),        # short last blocks, second request
    ("f32", 64, (300,), 1024, False),          # one-token blocks and empty ones
    ("f32", 128, (513, 90), 64, True),         # one K/V source shared by every layer
])
def test_pack_blocks_bit_exact(gpu_lib, dtype, d, lens, M, shared):
    L, Hkv = 3, 2
    say("pack blocks", dtype, d, lens, M, shared)
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    g = np.random.default_rng(d + M + len(lens))
    cus = np.concatenate([[0], np.cumsum(lens)])
    T = int(cus[-1])
    Lkv = 1 if shared else L
    k = torch.from_numpy(g.standard_normal((Lkv, Hkv, T, d)).astype(np.float32)).to(td)
    v = torch.from_numpy(g.standard_normal((Lkv, Hkv, T, d)).astype(np.float32)).to(td)
    kd, vd = k.cuda(), v.cuda()
    for b, N in enumerate(lens):
        ids = np.sort(g.choice(L * M, size=min(L * M, 37), replace=False)).astype(np.int32)
        ids[-1] = L * M + 5                                        # invalid: zero rows
        nbytes = gpu_lib.pack_blocks_bytes(td, Hkv, d, N, M, len(ids))
        dst = torch.full((nbytes,), 0xAB, dtype=torch.uint8, device="cuda")
        gpu_lib.sg_pack_blocks(kd, vd, cu(ids), int(cus[b]), N, M, dst, L=L, kv_layer_rows=0 if shared else None)
        torch.cuda.synchronize()
        ref = oracle.pack_blocks(raw(k), raw(v), ids, int(cus[b]), N, M, L=L, kv_layer_rows=0 if shared else None)
        np.testing.assert_array_equal(dst.cpu().numpy(), ref)


def test_block_mode_llama8b_8k(gpu_lib):
    """The whole block path at the bench's size: score -> eq. 1 -> eq. 2 -> top-K_r -> block push."""
    cfg = get("llama8b_8k")
    M, ratio = 1024, 1 / 6.5
    say("block mode llama8b_8k")
    pre = inputs.make_prefill(cfg, device="cuda")
    N, T, L, Hkv, d = pre["seqlens"][0], pre["T"], cfg.L, cfg.Hkv, cfg.d
    cus = cu(pre["cu_seqlens"])
    ws = torch.empty(gpu_lib.score_workspace_size(1, L, cfg.Hq, Hkv, d, cfg.W, N), dtype=torch.uint8, device="cuda")
    scores = torch.empty((L, Hkv, T), device="cuda")
    gpu_lib.sg_score(pre["q_win"], pre["k"], cus, T, N, Hkv, scores, ws=ws)
    imp = torch.empty((1, L, M), device="cuda")
    gpu_lib.sg_block_importance(scores, cus, T, M, imp)
    Kr = gpu_lib.block_budget(M, L, ratio, 1.0)
    ids = torch.empty((1, 1, Kr), dtype=torch.int32, device="cuda")
    gpu_lib.sg_topk(imp.view(1, 1, L * M), cu([0, L * M]), L * M, L * M, cu([0, Kr]), Kr, ids)
    torch.cuda.synchronize()

    ref_scores = oracle.score(pre["q_win"].float().cpu().numpy(), pre["k"].float().cpu().numpy(),
                              pre["cu_seqlens"], Hkv)
    ref_imp = oracle.block_importance(ref_scores.astype(np.float32), pre["cu_seqlens"], M)
    assert Kr == oracle.block_budget(M, L, ratio, 1.0) == 4883
    # importance: from the GPU scores vs from the oracle's (within the score tolerance)
    _importance_close(imp.cpu().numpy(), ref_imp, rtol=1e-3)
    # selection from the same importances is bit-exact; end to end only near-ties may differ
    imp32 = ref_imp.astype(np.float32).reshape(1, 1, L * M)
    ref_ids = oracle.topk(imp32, [0, L * M], [0, Kr])
    same = torch.empty((1, 1, Kr), dtype=torch.int32, device="cuda")
    gpu_lib.sg_topk(torch.from_numpy(imp32).cuda(), cu([0, L * M]), L * M, L * M, cu([0, Kr]), Kr, same)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(same.cpu().numpy(), ref_ids)
    finite = np.where(np.isinf(imp32[0, 0]), 1e30, imp32[0, 0]).astype(np.float64)
    assert_topk_sets_agree(ids.cpu().numpy()[0, 0], ref_ids[0, 0], finite, Kr)
    assert set(range(2 * M)) <= set(ids.cpu().numpy()[0, 0].tolist())
    # the push of the chosen blocks (the oracle's ids on both sides): bit-exact
    nbytes = gpu_lib.pack_blocks_bytes(pre["k"].dtype, Hkv, d, N, M, Kr)
    dst = torch.empty((nbytes,), dtype=torch.uint8, device="cuda")
    gpu_lib.sg_pack_blocks(pre["k"], pre["v"], cu(ref_ids[0, 0]), 0, N, M, dst)
    torch.cuda.synchronize()
    ref_buf = oracle.pack_blocks(raw(pre["k"]), raw(pre["v"]), ref_ids[0, 0], 0, N, M)
    np.testing.assert_array_equal(dst.cpu().numpy(), ref_buf)
