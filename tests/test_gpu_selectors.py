"""GPU parity of the selector variants against the CPU oracle, through the C ABI:
selection-frequency counts under the alpha rule and under the top-share rule
(Section 4.1 importance with either Section 5.1 selector) and decode-time
dynamic selection capped at a maximum ratio (Section 2.3, Section 5.1).

Where fp32 and fp64 would decide a threshold differently, the inputs are
integer-valued with d = 64 (scale 1/8) and alpha = 5.0625: every logit and
margin is then exact on both sides and no logit can sit on the threshold, so
the results must be identical.  With real-valued inputs the decisions within a
rounding band of the threshold may go either way; all others must agree."""
import numpy as np
import pytest
import torch

import oracle
from datagen import configs, inputs
from tests.gpu_util import cu, say

pytestmark = pytest.mark.gpu

ALPHA_EXACT = 5.0625          # alpha * sqrt(64) = 40.5: integer logits never tie the threshold


def _ints(shape, lo, hi, seed, dtype):
    x = np.random.default_rng(seed).integers(lo, hi + 1, shape).astype(np.float32)
    return torch.from_numpy(x).to(torch.bfloat16 if dtype == "bf16" else torch.float32)


def _count(gpu_lib, q, k, lens, Hkv, alpha):
    B, L, Hq, W, d = q.shape
    cus = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cus[-1])
    ws = torch.empty(gpu_lib.score_workspace_size(B, L, Hq, Hkv, d, W, max(lens)), dtype=torch.uint8, device="cuda")
    out = torch.full((L, Hkv, T), -1.0, device="cuda")
    gpu_lib.sg_score_count(q.cuda(), k.cuda(), cu(cus), T, max(lens), Hkv, out, alpha, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy(), cus


@pytest.mark.parametrize("dtype,G,W,lens", [
    ("f32", 4, 16, (2500, 700)),          # two chunks, a second request
    ("bf16", 4, 64, (5000,)),
    ("bf16", 8, 64, (64, 3000)),          # N = W
    ("bf16", 1, 32, (4100,)),
])
def test_score_count_exact(gpu_lib, dtype, G, W, lens):
    say("score count exact", dtype, G, W, lens)
    L, Hkv, d = 2, 2, 64
    T = sum(lens)
    q = _ints((len(lens), L, Hkv * G, W, d), -3, 3, G + W, dtype)
    k = _ints((L, Hkv, T, d), -3, 3, G * W + 1, dtype)
    got, cus = _count(gpu_lib, q, k, lens, Hkv, ALPHA_EXACT)
    ref = oracle.score_count(q.float().numpy(), k.float().numpy(), cus, Hkv, ALPHA_EXACT)
    np.testing.assert_array_equal(got, ref.astype(np.float32))
    assert got.min() >= 0 and got.max() <= G * W


@pytest.mark.parametrize("G,W,lens", [(4, 64, (3000, 5000)), (8, 64, (2048,))])
def test_score_count_band(gpu_lib, G, W, lens):
    say("score count band", G, W, lens)
    L, Hkv, d = 2, 2, 128
    T = sum(lens)
    g = np.random.default_rng(G * 100 + W)
    q = torch.from_numpy(g.standard_normal((len(lens), L, Hkv * G, W, d), dtype=np.float32) * 1.5).to(torch.bfloat16)
    k = torch.from_numpy(g.standard_normal((L, Hkv, T, d), dtype=np.float32)).to(torch.bfloat16)
    got, cus = _count(gpu_lib, q, k, lens, Hkv, 5.0)
    ref, near = oracle.score_count(q.float().numpy(), k.float().numpy(), cus, Hkv, 5.0, eps=1e-3)
    diff = np.abs(got.astype(np.int64) - ref)
    assert (diff <= near).all(), f"{int((diff > near).sum())} counts differ beyond the rounding band"
    assert (got > 0).sum() > 0.05 * got.size             # the rule picks something


def test_score_count_llama8b_8k_sampled(gpu_lib):
    cfg = configs.get("llama8b_8k")
    say("score count llama8b_8k")
    pre = inputs.make_prefill(cfg, device="cuda")
    N, T, L, Hkv, d = pre["seqlens"][0], pre["T"], cfg.L, cfg.Hkv, cfg.d
    ws = torch.empty(gpu_lib.score_workspace_size(1, L, cfg.Hq, Hkv, d, cfg.W, N), dtype=torch.uint8, device="cuda")
    out = torch.empty((L, Hkv, T), device="cuda")
    gpu_lib.sg_score_count(pre["q_win"], pre["k"], cu(pre["cu_seqlens"]), T, N, Hkv, out, 5.0, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    for l, h in ((0, 0), (31, 7)):
        q = pre["q_win"][:, l:l + 1, h * cfg.G:(h + 1) * cfg.G].float().cpu().numpy()
        k = pre["k"][l:l + 1, h:h + 1].float().cpu().numpy()
        ref, near = oracle.score_count(q, k, pre["cu_seqlens"], 1, 5.0, eps=1e-3)
        diff = np.abs(got[l, h].astype(np.int64) - ref[0, 0])
        assert (diff <= near[0, 0]).all()
        heavy = pre["heavy"][(0, l, h)].cpu().numpy()
        assert got[l, h, heavy].mean() > 2 * got[l, h].mean()     # the planted heavy hitters are picked often


def _select(gpu_lib, q, k, lens, Hkv, caps, alpha, scale=None):
    B, L, Hq, d = q.shape
    cus = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    cc = np.concatenate([[0], np.cumsum(caps)]).astype(np.int32)
    T, Kc = int(cus[-1]), int(cc[-1])
    ws = torch.empty(gpu_lib.decode_select_workspace_size(B, L, Hq, max(lens)), dtype=torch.uint8, device="cuda")
    idx = torch.full((L, Hkv, Kc), -7, dtype=torch.int32, device="cuda")
    n_sel = torch.full((B, L, Hkv), -7, dtype=torch.int32, device="cuda")
    gpu_lib.sg_decode_select(q.cuda(), k.cuda(), cu(cus), T, max(lens), Hkv, cu(cc), Kc, idx, n_sel, alpha, ws,
                             scale=scale)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), n_sel.cpu().numpy(), cus, cc


@pytest.mark.parametrize("dtype,G,d,lens,cap_bp,alpha", [
    ("bf16", 4, 64, (3000, 1234), 2000, ALPHA_EXACT),     # the 20% cap
    ("f32", 2, 64, (5000,), 50, ALPHA_EXACT),             # the cap binds hard
    ("bf16", 8, 64, (700, 64, 2100), 10000, ALPHA_EXACT),
    ("bf16", 1, 64, (2049,), 2000, 0.0),                   # alpha 0: each head's maxima only
    ("bf16", 4, 40, (3000, 900), 2000, ALPHA_EXACT),      # a partial set of 40 channels
    ("f32", 8, 48, (1500,), 2000, ALPHA_EXACT),
    ("bf16", 2, 32, (2500,), 500, ALPHA_EXACT),
])
def test_decode_select_exact(gpu_lib, dtype, G, d, lens, cap_bp, alpha):
    say("decode select exact", dtype, G, d, lens, cap_bp, alpha)
    L, Hkv = 2, 2
    T = sum(lens)
    q = _ints((len(lens), L, Hkv * G, d), -2, 2, G + T, dtype)
    k = _ints((L, Hkv, T, d), -2, 2, G * T + 3, dtype)
    caps = [max(1, n * cap_bp // 10000) for n in lens]
    # scale 1/8 keeps every logit exact at every width (that of a 64-wide head)
    idx, n_sel, cus, cc = _select(gpu_lib, q, k, lens, Hkv, caps, alpha, scale=0.125)
    r_idx, r_n, _ = oracle.decode_select(q.float().numpy(), k.float().numpy(), cus, Hkv, cc, alpha, scale=0.125)
    np.testing.assert_array_equal(n_sel, r_n)
    np.testing.assert_array_equal(idx, r_idx)


def _check_band(idx, n_sel, r_idx, r_n, r, cus, cc, alpha, eps=1e-3):
    B = len(cus) - 1
    L, Hkv = idx.shape[0], idx.shape[1]
    for b in range(B):
        cap = cc[b + 1] - cc[b]
        for l in range(L):
            for h in range(Hkv):
                rr = r[l, h, cus[b]:cus[b + 1]]
                cnt_lo, cnt_hi = int((rr >= -alpha + eps).sum()), int((rr >= -alpha - eps).sum())
                n = int(n_sel[b, l, h])
                assert min(cnt_lo, cap) <= n <= min(cnt_hi, cap)
                sel = idx[l, h, cc[b]:cc[b] + n]
                assert (np.diff(sel) > 0).all() and (idx[l, h, cc[b] + n:cc[b + 1]] == -1).all()
                order = np.sort(rr)[::-1]
                edge = max(-alpha, order[n - 1]) if n > 0 else np.inf
                inside = np.zeros(len(rr), bool)
                inside[sel] = True
                assert inside[rr > edge + eps].all(), "a clearly selected entry is missing"
                assert not inside[rr < edge - eps].any(), "a clearly rejected entry is selected"


@pytest.mark.parametrize("G,d,lens", [(4, 128, (4000, 900)), (8, 128, (2500,)), (4, 40, (3000, 1000))])
def test_decode_select_band(gpu_lib, G, d, lens):
    say("decode select band", G, d, lens)
    L, Hkv, alpha = 2, 2, 5.0
    T = sum(lens)
    scale = 128 ** -0.5                   # the full head's scale, also for a partial set of channels
    g = np.random.default_rng(G + T + d)
    q = torch.from_numpy(g.standard_normal((len(lens), L, Hkv * G, d), dtype=np.float32) * 2).to(torch.bfloat16)
    k = torch.from_numpy(g.standard_normal((L, Hkv, T, d), dtype=np.float32)).to(torch.bfloat16)
    caps = [n // 5 for n in lens]
    idx, n_sel, cus, cc = _select(gpu_lib, q, k, lens, Hkv, caps, alpha, scale=scale)
    r_idx, r_n, r = oracle.decode_select(q.float().numpy(), k.float().numpy(), cus, Hkv, cc, alpha, scale=scale)
    _check_band(idx, n_sel, r_idx, r_n, r, cus, cc, alpha)


def test_decode_select_llama8b_32k_step(gpu_lib):
    """One decode step of the 8B / 32K-token workload, all 32 layers; the oracle
    checks two layers."""
    cfg = configs.get("llama8b_32k")
    say("decode select llama8b_32k")
    pre = inputs.make_prefill(cfg, device="cuda", want_v=False)
    N, T, L, Hkv = pre["seqlens"][0], pre["T"], cfg.L, cfg.Hkv
    q = inputs.decode_queries(cfg, 0, device="cuda", mu=pre["mu"])          # [1][L][Hq][d]
    cap = N * 2000 // 10000
    idx, n_sel, cus, cc = _select(gpu_lib, q, pre["k"], [N], Hkv, [cap], 5.0)
    for l in (0, 31):
        r_idx, r_n, r = oracle.decode_select(q[:, l:l + 1].float().cpu().numpy(), pre["k"][l:l + 1].float().cpu().numpy(),
                                             cus, Hkv, cc, 5.0)
        _check_band(idx[l:l + 1], n_sel[:, l:l + 1], r_idx, r_n, r, cus, cc, 5.0)
    assert (n_sel >= 1).all() and (n_sel <= cap).all()


# ----------------------------------------------------------------- top-share counts

def _topshare(gpu_lib, q, k, lens, Hkv, ratio_bp, ws=None):
    B, L, Hq, W, d = q.shape
    cus = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cus[-1])
    if ws is None:       # garbage contents: the call must not depend on them
        ws = torch.full((gpu_lib.score_topshare_workspace_size(B, L, Hq, Hkv, d, W, max(lens)),), 0xA5,
                        dtype=torch.uint8, device="cuda")
    out = torch.full((L, Hkv, T), -1.0, device="cuda")
    gpu_lib.sg_score_topshare(q.cuda(), k.cuda(), cu(cus), T, max(lens), Hkv, out, ratio_bp, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy(), cus


@pytest.mark.parametrize("dtype,G,W,d,lens,bp,span", [
    ("f32", 4, 16, 64, (2500, 700), 2000, 3),        # two chunks, a second request, many ties
    ("bf16", 4, 64, 64, (5000,), 2000, 3),           # 256 rows: 6-bit digits
    ("bf16", 4, 64, 128, (3000, 1111), 2000, 40),    # d = 128, few ties
    ("bf16", 8, 64, 64, (64, 3000), 2000, 3),        # 512 rows (5-bit digits); N = W
    ("bf16", 8, 64, 64, (2345,), 700, 40),
    ("bf16", 1, 32, 64, (4100,), 1, 3),              # k = 1: each row's maxima
    ("bf16", 2, 64, 64, (3000, 1500), 10000, 3),     # k = n: every visible key
    ("f32", 8, 16, 64, (1300,), 5000, 40),           # 128 rows
    ("bf16", 4, 20, 64, (2222, 999), 333, 3),        # 80 rows: padded wavefront rows
    ("f32", 2, 8, 128, (777, 130), 2000, 3),         # a single wavefront, short prompts
    ("f32", 8, 64, 128, (700,), 2000, 40),           # fp32 at 512 rows (8 wavefronts, 5-bit digits)
    ("f32", 8, 64, 64, (1100, 64), 1500, 3),
])
def test_score_topshare_exact(gpu_lib, dtype, G, W, d, lens, bp, span):
    """Integer inputs: every logit is exact in fp32 and fp64, so the thresholds,
    their ties and every count must match the oracle."""
    say("score topshare exact", dtype, G, W, d, lens, bp, span)
    L, Hkv = 2, 2
    T = sum(lens)
    q = _ints((len(lens), L, Hkv * G, W, d), -span, span, G + W + d, dtype)
    k = _ints((L, Hkv, T, d), -span, span, G * W + d + 1, dtype)
    got, cus = _topshare(gpu_lib, q, k, lens, Hkv, bp)
    ref = oracle.score_topshare(q.float().numpy(), k.float().numpy(), cus, Hkv, bp)
    np.testing.assert_array_equal(got, ref.astype(np.float32))
    assert got.min() >= 0 and got.max() <= G * W


def test_score_topshare_mixed_rows(gpu_lib):
    """One unit whose rows take both ways to their threshold: keys in {-1, 0, 1};
    window rows w < 32 with queries in [-40, 40] see a few keys per logit value
    (their last bins are gathered and ranked), rows w >= 32 with queries in
    {-1, 0, 1} see dozens of keys tied at every value (their bins stay too large
    to gather and the radix passes go on).  Integer logits: exact."""
    G, W, d, L, Hkv, lens = 4, 64, 64, 2, 2, (3000, 2100)
    say("score topshare mixed rows", lens)
    T = sum(lens)
    q = _ints((len(lens), L, Hkv * G, W, d), -40, 40, 81, "bf16")
    q[..., 32:, :] = _ints((len(lens), L, Hkv * G, W - 32, d), -1, 1, 82, "bf16")
    k = _ints((L, Hkv, T, d), -1, 1, 83, "bf16")
    for bp in (2000, 500):
        got, cus = _topshare(gpu_lib, q, k, lens, Hkv, bp)
        ref = oracle.score_topshare(q.float().numpy(), k.float().numpy(), cus, Hkv, bp)
        np.testing.assert_array_equal(got, ref.astype(np.float32))


def test_score_topshare_shared_layer_source(gpu_lib):
    """One K source read by every layer (k_layer_rows = 0, as the batched
    workload stores it), three requests; integer inputs: exact."""
    G, W, d, L, Hkv, lens = 2, 32, 64, 3, 2, (900, 2300, 32)
    say("score topshare shared layer source", lens)
    T = sum(lens)
    q = _ints((len(lens), L, Hkv * G, W, d), -40, 40, 91, "bf16")
    k = _ints((1, Hkv, T, d), -40, 40, 92, "bf16")
    cus = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    ws = torch.empty(gpu_lib.score_topshare_workspace_size(len(lens), L, Hkv * G, Hkv, d, W, max(lens)),
                     dtype=torch.uint8, device="cuda")
    out = torch.full((L, Hkv, T), -1.0, device="cuda")
    gpu_lib.sg_score_topshare(q.cuda(), k.cuda(), cu(cus), T, max(lens), Hkv, out, 2000, ws, k_layer_rows=0)
    torch.cuda.synchronize()
    ref = oracle.score_topshare(q.float().numpy(), k.float().numpy(), cus, Hkv, 2000, k_layer_rows=0)
    np.testing.assert_array_equal(out.cpu().numpy(), ref.astype(np.float32))


def test_score_topshare_all_keys_closed_form(gpu_lib):
    """ratio 100%: each row picks every key it sees, so key j's count is G times
    the number of window rows at or after it, whatever the values."""
    G, W, d, lens = 4, 64, 128, (2100, 64, 700)
    L, Hkv = 1, 2
    T = sum(lens)
    say("score topshare closed form", lens)
    g = np.random.default_rng(9)
    q = torch.from_numpy(g.standard_normal((len(lens), L, Hkv * G, W, d), dtype=np.float32)).to(torch.bfloat16)
    k = torch.from_numpy(g.standard_normal((L, Hkv, T, d), dtype=np.float32)).to(torch.bfloat16)
    got, cus = _topshare(gpu_lib, q, k, lens, Hkv, 10000)
    for b, N in enumerate(lens):
        j = np.arange(N)
        want = G * np.minimum(W, N - j)        # rows w with N - W + w >= j
        for l in range(L):
            for h in range(Hkv):
                np.testing.assert_array_equal(got[l, h, cus[b]:cus[b + 1]], want.astype(np.float32))


def test_score_topshare_short_request_and_reuse(gpu_lib):
    """A request shorter than the window gets zero counts; the others match the
    oracle; a second, smaller call on the same workspace matches too."""
    G, W, d, L, Hkv = 4, 64, 64, 2, 2
    lens = (40, 3000)
    say("score topshare short request", lens)
    T = sum(lens)
    q = _ints((2, L, Hkv * G, W, d), -3, 3, 71, "bf16")
    k = _ints((L, Hkv, T, d), -3, 3, 72, "bf16")
    ws = torch.full((gpu_lib.score_topshare_workspace_size(2, L, Hkv * G, Hkv, d, W, max(lens)),), 0x5A,
                    dtype=torch.uint8, device="cuda")
    got, cus = _topshare(gpu_lib, q, k, lens, Hkv, 2000, ws=ws)
    assert (got[:, :, :40] == 0).all()
    ref = oracle.score_topshare(q[1:].float().numpy(), k[:, :, 40:].float().numpy(), [0, 3000], Hkv, 2000)
    np.testing.assert_array_equal(got[:, :, 40:], ref.astype(np.float32))
    lens2 = (1500,)
    q2 = _ints((1, L, Hkv * G, W, d), -3, 3, 73, "bf16")
    k2 = _ints((L, Hkv, 1500, d), -3, 3, 74, "bf16")
    got2, cus2 = _topshare(gpu_lib, q2, k2, lens2, Hkv, 2000, ws=ws)
    ref2 = oracle.score_topshare(q2.float().numpy(), k2.float().numpy(), cus2, Hkv, 2000)
    np.testing.assert_array_equal(got2, ref2.astype(np.float32))


@pytest.mark.parametrize("G,W,lens,bp", [(4, 64, (3000, 5000), 2000), (8, 64, (2048,), 500)])
def test_score_topshare_band(gpu_lib, G, W, lens, bp):
    """Real-valued inputs: the fp32 threshold is within rounding of the exact
    one, so only decisions within that band of it may differ."""
    say("score topshare band", G, W, lens, bp)
    L, Hkv, d = 2, 2, 128
    T = sum(lens)
    g = np.random.default_rng(G * 100 + W + bp)
    q = torch.from_numpy(g.standard_normal((len(lens), L, Hkv * G, W, d), dtype=np.float32) * 1.5).to(torch.bfloat16)
    k = torch.from_numpy(g.standard_normal((L, Hkv, T, d), dtype=np.float32)).to(torch.bfloat16)
    got, cus = _topshare(gpu_lib, q, k, lens, Hkv, bp)
    ref, near = oracle.score_topshare(q.float().numpy(), k.float().numpy(), cus, Hkv, bp, eps=1e-3)
    diff = np.abs(got.astype(np.int64) - ref)
    assert (diff <= near).all(), f"{int((diff > near).sum())} counts differ beyond the rounding band"
    # every row picks at least its k keys
    for b, N in enumerate(lens):
        ks = [max(1, min(n, n * bp // 10000)) for n in range(N - W + 1, N + 1)]
        for l in range(L):
            for h in range(Hkv):
                assert got[l, h, cus[b]:cus[b + 1]].sum() >= G * sum(ks)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_score_topshare_one_row_units(gpu_lib, dtype):
    """One row per unit (G = W = 1), real values: each unit's counts are that
    row's picks, at least its k and, with no tie at the threshold, exactly k.
    A threshold taken from logits other than those the count pass compares
    would leave the threshold key itself out (k - 1 picks)."""
    L, Hkv, d, lens, bp = 8, 4, 128, (6000, 2500, 1), 2000
    say("score topshare one-row units", dtype, lens)
    T = sum(lens)
    g = np.random.default_rng(31)
    mk = (lambda a: torch.from_numpy(a).to(torch.bfloat16)) if dtype == "bf16" else torch.from_numpy
    q = mk(g.standard_normal((len(lens), L, Hkv, 1, d), dtype=np.float32))
    k = mk(g.standard_normal((L, Hkv, T, d), dtype=np.float32))
    got, cus = _topshare(gpu_lib, q, k, lens, Hkv, bp)
    ref, near = oracle.score_topshare(q.float().numpy(), k.float().numpy(), cus, Hkv, bp, eps=1e-4)
    assert set(np.unique(got)) <= {0.0, 1.0}
    assert (np.abs(got.astype(np.int64) - ref) <= near).all()
    for b, N in enumerate(lens):
        kb = max(1, N * bp // 10000)
        picks = got[:, :, cus[b]:cus[b + 1]].sum(axis=2)
        assert (picks >= kb).all()
        exact = ref[:, :, cus[b]:cus[b + 1]].sum(axis=2) == kb      # no tie at the oracle's threshold
        assert (picks[exact] <= kb + near[:, :, cus[b]:cus[b + 1]].sum(axis=2)[exact]).all()


def test_score_topshare_llama8b_8k_sampled(gpu_lib):
    """The 8B / 8K-token workload, all 32 layers at the 20% share; the oracle
    checks two units."""
    cfg = configs.get("llama8b_8k")
    say("score topshare llama8b_8k")
    pre = inputs.make_prefill(cfg, device="cuda")
    N, T, L, Hkv, d = pre["seqlens"][0], pre["T"], cfg.L, cfg.Hkv, cfg.d
    ws = torch.empty(gpu_lib.score_topshare_workspace_size(1, L, cfg.Hq, Hkv, d, cfg.W, N), dtype=torch.uint8,
                     device="cuda")
    out = torch.empty((L, Hkv, T), device="cuda")
    gpu_lib.sg_score_topshare(pre["q_win"], pre["k"], cu(pre["cu_seqlens"]), T, N, Hkv, out, 2000, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    for l, h in ((0, 0), (31, 7)):
        q = pre["q_win"][:, l:l + 1, h * cfg.G:(h + 1) * cfg.G].float().cpu().numpy()
        k = pre["k"][l:l + 1, h:h + 1].float().cpu().numpy()
        ref, near = oracle.score_topshare(q, k, pre["cu_seqlens"], 1, 2000, eps=1e-3)
        diff = np.abs(got[l, h].astype(np.int64) - ref[0, 0])
        assert (diff <= near[0, 0]).all()
        heavy = pre["heavy"][(0, l, h)].cpu().numpy()
        assert got[l, h, heavy].mean() > 2 * got[l, h].mean()     # the planted heavy hitters are picked often
