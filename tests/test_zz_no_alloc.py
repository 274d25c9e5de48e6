"""sg_decode_attn_noalloc (the entry point for callers that cannot allocate)
against sg_decode_attn with a caller workspace, through the C ABI: the same
kernels, so outputs must be bit-identical; both within the decode tolerance of
the oracle.  Calls in a row, each smaller than the one before, share the
static scratch."""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import cu, say

pytestmark = pytest.mark.gpu


def _case(B, Hq, Hkv, d, rows, P, seed):
    g = np.random.default_rng(seed)
    npg = max(-(-max(rows) // P), 1)
    units = B * Hkv
    pool_rows = (units * npg + 5) * P
    perm = g.permutation(units * npg + 5)[: units * npg]
    pt = (perm.reshape(B, Hkv, npg) * P).astype(np.int32)
    nr = np.array(rows, np.int32).reshape(B, Hkv)
    k = torch.from_numpy(g.standard_normal((pool_rows, d), dtype=np.float32)).to(torch.bfloat16)
    v = torch.from_numpy(g.standard_normal((pool_rows, d), dtype=np.float32)).to(torch.bfloat16)
    q = torch.from_numpy(2 * g.standard_normal((B, Hq, d), dtype=np.float32)).to(torch.bfloat16)
    return q, k, v, pt, nr, P


@pytest.mark.parametrize("order", ["large_then_small"])
def test_noalloc_matches_workspace_entry_point(gpu_lib, order):
    # the first call cuts 320 units into equal parts over the shader engines;
    # the second splits every unit's rows over several workgroups (16 units on
    # a 256-CU chip); the third is smaller still.  Each one's states go through
    # the scratch array the previous call left behind
    cases = [(40, 32, 8, 128, [400 + (97 * i) % 1200 for i in range(320)], 16, 3),
             (2, 32, 8, 128, [3000 + 37 * i for i in range(16)], 16, 1),
             (1, 32, 8, 128, [700 + 5 * i for i in range(8)], 16, 2)]
    assert gpu_lib.decode_noalloc_scratch_bytes() == 16 << 20
    for (B, Hq, Hkv, d, rows, P, seed) in cases:
        say("noalloc decode", B, Hq, Hkv, d, max(rows))
        q, k, v, pt, nr, P = _case(B, Hq, Hkv, d, rows, P, seed)
        qd, kd, vd, ptd, nrd = q.cuda(), k.cuda(), v.cuda(), cu(pt), cu(nr)
        ws_bytes = gpu_lib.decode_workspace_size(B, Hq, Hkv, d, pt.shape[2], P)
        assert 0 < ws_bytes <= (16 << 20)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
        ref_out = torch.full((B, Hq, d), float("nan"), device="cuda")
        out = torch.full((B, Hq, d), float("nan"), device="cuda")
        gpu_lib.sg_decode_attn(qd, kd, vd, ptd, nrd, P, ref_out, ws=ws)
        gpu_lib.sg_decode_attn_noalloc(qd, kd, vd, ptd, nrd, P, out)
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out)
        o = oracle.decode_attn(q.float().numpy(), k.float().numpy(), v.float().numpy(), pt, nr, P)
        got = out.cpu().numpy()
        assert np.isfinite(got).all()
        np.testing.assert_allclose(got, o, atol=2e-2, rtol=0)
        assert np.abs(got - o).max() <= 1e-4


def test_noalloc_rejects_states_beyond_scratch(gpu_lib):
    # 16 units of up to 2^20 rows through a per-row index table: 512 splits of
    # 2048 rows each, 16 x 512 x 4 heads x 130 floats = 17.0 MB of split
    # states > 16 MiB; rejected on the host, nothing is launched
    B, Hq, Hkv, d, P, npg = 2, 32, 8, 128, 1, 1 << 20
    say("noalloc decode rejection")
    q = torch.zeros((B, Hq, d), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((16, d), dtype=torch.bfloat16, device="cuda")
    pt = torch.zeros((B, Hkv, npg), dtype=torch.int32, device="cuda")
    nr = torch.zeros((B, Hkv), dtype=torch.int32, device="cuda")
    out = torch.zeros((B, Hq, d), device="cuda")
    with pytest.raises(gpu_lib.SmartgenError) as e:
        gpu_lib.sg_decode_attn_noalloc(q, k, k, pt, nr, P, out)
    assert e.value.status == gpu_lib.SG_EWORKSPACE
