"""The C ABI: the library loads, exports every function include/smartgen.h
declares, and rejects bad scalar arguments on the host (no GPU needed: the
checks run before anything is enqueued)."""
import ctypes
import os
import re

import pytest

from paper_2607_28150_amd import smartgen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(sg_[a-z0-9_]+)\s*\(", text))
    return names


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(smartgen.LIB_PATH):
        from paper_2607_28150_amd import build
        build.build()
    return smartgen.load()


def test_exports_every_declared_symbol(lib):
    declared = _declared()
    assert {"sg_score", "sg_topk", "sg_pack", "sg_split", "sg_fetch", "sg_decode_attn"} <= declared
    for name in declared:
        assert hasattr(lib, name), f"{name} declared but not exported"
    assert set(smartgen.EXPORTS) == declared


def test_version_and_status_strings(lib):
    assert smartgen.version() == 100
    assert lib.sg_status_str(0) == b"ok"
    assert lib.sg_status_str(-3).startswith(b"workspace")


def test_sizes(lib):
    # [K | V | idx] of 2 layers x 8 heads x 819 rows of 128 bf16
    S = 2 * 8 * 819
    assert smartgen.pack_bytes(__import__("torch").bfloat16, 2, 8, 128, 819) == 2 * S * 256 + 4 * S
    # 8 units are few: the keys split into 128-key chunks so that the launch
    # fills the chip; (reference, sum) per row and chunk
    assert smartgen.score_workspace_size(1, 1, 8, 8, 64, 32, 2048) == 8 * 16 * 32 * 8
    # 256 units (32 layers x 8 heads) at 8192 keys: 2048-key chunks
    assert smartgen.score_workspace_size(1, 32, 32, 8, 128, 64, 8192) == 256 * 4 * 256 * 8
    assert smartgen.decode_workspace_size(1, 32, 8, 128, 1, 16) == 0          # one split: no workspace
    # workspace bound: 2400 units x up to 8 splits of 128 rows x 4 heads x 130 floats
    assert smartgen.decode_workspace_size(300, 32, 8, 128, 64, 16) == 2400 * 8 * 4 * 130 * 4
    assert smartgen.decode_workspace_size(2, 32, 8, 128, 64, 16) == 2 * 8 * 8 * 4 * 130 * 4   # <= 8 splits of 128 rows


P = ctypes.c_void_p(16)   # never dereferenced: every call below fails validation first


def _err(lib):
    return lib.sg_last_error().decode()


def test_score_rejections(lib):
    rc = lib.sg_score(None, 1, 1, 1, 8, 8, 96, 32, P, 100, 100, P, P, 0, None, P, P, 1 << 20)
    assert rc == smartgen.SG_EUNSUPPORTED and "head dimension" in _err(lib)
    rc = lib.sg_score(None, 1, 1, 1, 6, 4, 64, 32, P, 100, 100, P, P, 0, None, P, P, 1 << 20)
    assert rc == smartgen.SG_EINVAL
    rc = lib.sg_score(None, 1, 1, 1, 64, 8, 128, 65, P, 100, 100, P, P, 0, None, P, P, 1 << 20)
    assert rc == smartgen.SG_EUNSUPPORTED and "G*W" in _err(lib)
    rc = lib.sg_score(None, 1, 1, 1, 8, 8, 64, 32, P, 4096, 4096, P, P, 0, None, P, P, 16)
    assert rc == smartgen.SG_EWORKSPACE
    rc = lib.sg_score(None, 7, 1, 1, 8, 8, 64, 32, P, 100, 100, P, P, 0, None, P, P, 1 << 20)
    assert rc == smartgen.SG_EINVAL and "dtype" in _err(lib)


def test_topk_rejections(lib):
    rc = lib.sg_topk(None, 1, 1, 1, P, 100000, 90000, P, 100, P, P)      # rows above 80 x 1024
    assert rc == smartgen.SG_EUNSUPPORTED
    rc = lib.sg_topk(None, 0, 1, 1, P, 100, 100, P, 10, P, P)
    assert rc == smartgen.SG_EINVAL
    assert lib.sg_topk(None, 1, 1, 1, P, 100, 100, P, 0, P, P) == smartgen.SG_OK   # nothing to select


def test_pack_rejections(lib):
    rc = lib.sg_pack(None, 1, 1, 1, 1, 128, P, 100, P, 10, 10, P, P, 100, P, P, 100, 0)
    assert rc == smartgen.SG_EWORKSPACE
    rc = lib.sg_pack(None, 1, 1, 1, 1, 80, P, 100, P, 10, 10, P, P, 100, P, P, 1 << 20, 0)
    assert rc == smartgen.SG_EUNSUPPORTED
    rc = lib.sg_pack(None, 1, 1, 1, 1, 128, P, 100, P, 10, 10, ctypes.c_void_p(18), P, 100, P, P, 1 << 20, 0)
    assert rc == smartgen.SG_EINVAL and "aligned" in _err(lib)
    rc = lib.sg_pack(None, 1, 1, 1, 1, 128, P, 100, P, 10, 10, P, P, 100, P, P, 1 << 20, -1)
    assert rc == smartgen.SG_EINVAL and "budget" in _err(lib)


def test_split_fetch_decode_rejections(lib):
    assert lib.sg_split(None, -1, P, 0, P, P, 0, P, P, 0, None, P, P, P, P, None) == smartgen.SG_EINVAL
    assert lib.sg_split(None, 2, P, 5, P, P, 10, P, P, 1, None, P, P, P, P, None) == smartgen.SG_EINVAL
    assert lib.sg_fetch(None, 1, 128, 1, P, 5, P, None, P, 10, P, P, P, 0, 1, P, P, P, 10) == smartgen.SG_EINVAL
    rc = lib.sg_decode_attn(None, 1, 1, 6, 4, 128, 0.1, P, P, P, 10, P, P, 16, 4, P, None, 0)
    assert rc == smartgen.SG_EINVAL
    rc = lib.sg_decode_attn(None, 1, 1, 8, 8, 128, -1.0, P, P, P, 10, P, P, 16, 4, P, None, 0)
    assert rc == smartgen.SG_EINVAL
    rc = lib.sg_decode_attn(None, 1, 2, 32, 8, 128, 0.1, P, P, P, 10, P, P, 16, 64, P, None, 0)
    assert rc == smartgen.SG_EWORKSPACE
    rc = lib.sg_decode_attn(None, 1, 1, 24, 8, 128, 0.1, P, P, P, 10, P, P, 16, 4, P, None, 0)
    assert rc == smartgen.SG_EUNSUPPORTED       # group size 3


def test_block_mode_host_checks(lib):
    # eq. 2 on the host: the worked values of the paper's setting and the clip
    assert smartgen.block_budget(1024, 32, 1.0, 6.5) == 4883
    assert smartgen.block_budget(1024, 32, 1.0, 100.0) == 2048
    assert smartgen.block_budget(1024, 32, 1.0, 0.5) == 32768
    assert smartgen.block_budget(1024, 32, 1.0, 0.0) == 32768
    assert lib.sg_block_budget(0, 32, 1.0, 1.0) == -1
    assert lib.sg_block_budget(1024, 32, -1.0, 1.0) == -1
    # [K | V | ids] of 5 blocks of ceil(8192 / 1024) = 8 tokens in 8 heads, bf16 d = 128
    assert smartgen.pack_blocks_bytes(__import__("torch").bfloat16, 8, 128, 8192, 1024, 5) == 2 * 5 * 8 * 8 * 256 + 20
    assert lib.sg_block_importance(None, 0, 1, 1, P, 10, 4, P, P) == smartgen.SG_EINVAL
    assert lib.sg_block_importance(None, 1, 1, 1, P, 10, 0, P, P) == smartgen.SG_EINVAL
    rc = lib.sg_pack_blocks(None, 1, 2, 8, 128, 100, 90, 20, 4, P, P, 800, 3, P, P, 1 << 20)   # s0 + N > T
    assert rc == smartgen.SG_EINVAL
    rc = lib.sg_pack_blocks(None, 1, 2, 8, 128, 100, 0, 20, 4, P, P, 800, 3, P, P, 16)          # too small
    assert rc == smartgen.SG_EWORKSPACE
    rc = lib.sg_pack_blocks(None, 1, 2, 8, 80, 100, 0, 20, 4, P, P, 800, 3, P, P, 1 << 20)      # d = 80
    assert rc == smartgen.SG_EUNSUPPORTED
    assert lib.sg_pack_blocks(None, 1, 2, 8, 128, 100, 0, 20, 4, P, P, 800, 0, P, P, 0) == smartgen.SG_OK


def test_spec_and_keep_host_checks(lib):
    # the paper's speculative ratios: 10% delivers 32 x 1024 blocks in 10 transfers, 20% in 5, 5% in 20
    assert smartgen.spec_quota(32768, 1000) == 3277
    assert smartgen.spec_quota(32768, 2000) == 6554
    assert smartgen.spec_quota(32768, 500) == 1639
    assert smartgen.spec_quota(5, 1) == 1 and smartgen.spec_quota(0, 1000) == 0
    assert smartgen.spec_quota(10, 20000) == 10
    assert lib.sg_spec_quota(-1, 1000) == -1 and lib.sg_spec_quota(10, 0) == -1
    rc = lib.sg_spec_push(None, 1, 2, 8, 128, 100, 90, 20, 4, P, P, 800, P, P, 800, 3, P, P, None)   # s0 + N > T
    assert rc == smartgen.SG_EINVAL
    rc = lib.sg_spec_push(None, 1, 2, 8, 96, 100, 0, 20, 4, P, P, 800, P, P, 800, 3, P, P, None)     # d = 96
    assert rc == smartgen.SG_EUNSUPPORTED
    rc = lib.sg_spec_push(None, 1, 2, 8, 128, 100, 0, 20, 4, P, P, -1, P, P, 800, 3, P, P, None)     # stride
    assert rc == smartgen.SG_EINVAL
    assert lib.sg_spec_push(None, 1, 2, 8, 128, 100, 0, 20, 4, P, P, 800, P, P, 800, 0, P, P, None) == smartgen.SG_OK
    # fetch with reuse: the index is required, and a mask needs its offsets
    rc = lib.sg_fetch_keep(None, 1, 128, 1, P, 5, None, None, P, 10, P, P, None, 1, 1, None, None, None, 0,
                           P, P, P, 10, None, 0, None, None)
    assert rc == smartgen.SG_EINVAL and "null" in _err(lib)
    rc = lib.sg_fetch_keep(None, 1, 128, 1, P, 5, P, None, P, 10, P, P, None, 1, 1, None, None, None, 0,
                           P, P, P, 10, P, 10, None, None)
    assert rc == smartgen.SG_EINVAL and "mask" in _err(lib)
    rc = lib.sg_fetch_keep(None, 1, 128, 1, P, 5, P, None, P, 10, P, P, P, 1, 1, None, P, P, 10,
                           P, P, P, 10, None, 0, None, None)
    assert rc == smartgen.SG_EINVAL and "dst_start" in _err(lib)


def test_selector_host_checks(lib):
    rc = lib.sg_score_count(None, 1, 1, 1, 8, 8, 64, 32, P, 100, 100, P, P, 0, -1.0, P, P, 1 << 20)
    assert rc == smartgen.SG_EINVAL and "alpha" in _err(lib)
    rc = lib.sg_score_count(None, 1, 1, 1, 8, 8, 64, 32, P, 4096, 4096, P, P, 0, 5.0, P, P, 16)
    assert rc == smartgen.SG_EWORKSPACE
    assert smartgen.decode_select_workspace_size(1, 32, 32, 8192) == 32 * 32 * (8192 + 16) * 4   # logits, chunk maxima
    rc = lib.sg_decode_select(None, 1, 1, 1, 24, 8, 128, P, P, 100, 100, P, 0, 0.0, 5.0, P, 10, P, P, P, 1 << 30)
    assert rc == smartgen.SG_EUNSUPPORTED and "group" in _err(lib)          # G = 3
    rc = lib.sg_decode_select(None, 1, 1, 1, 32, 8, 128, P, P, 40000, 40000, P, 0, 0.0, 5.0, P, 10, P, P, P, 1 << 30)
    assert rc == smartgen.SG_EUNSUPPORTED                                   # rows above 32 x 1024
    rc = lib.sg_decode_select(None, 1, 1, 1, 32, 8, 128, P, P, 100, 100, P, 0, 0.0, float("nan"), P, 10, P, P, P, 1 << 30)
    assert rc == smartgen.SG_EINVAL
    rc = lib.sg_decode_select(None, 1, 1, 1, 32, 8, 56, P, P, 100, 100, P, 0, 0.0, 5.0, P, 10, P, P, P, 1 << 30)
    assert rc == smartgen.SG_EUNSUPPORTED and "width" in _err(lib)         # 56 channels
    rc = lib.sg_decode_select(None, 1, 1, 1, 32, 8, 128, P, P, 100, 100, P, 0, -1.0, 5.0, P, 10, P, P, P, 1 << 30)
    assert rc == smartgen.SG_EINVAL and "scale" in _err(lib)
    rc = lib.sg_decode_select(None, 1, 1, 1, 32, 8, 128, P, P, 100, 100, P, 0, 0.0, 5.0, P, 10, P, P, P, 64)
    assert rc == smartgen.SG_EWORKSPACE


def test_topshare_host_checks(lib):
    # rows x (prefix, rank, gathered count, 64 bins, 32 gathered values) + units x (8 pass flags, gather flag)
    rows, units = 1 * 32 * 8 * 4 * 64, 1 * 32 * 8
    assert smartgen.score_topshare_workspace_size(1, 32, 32, 8, 128, 64, 8192) == (rows * 99 + units * 9) * 4
    assert smartgen.score_topshare_workspace_size(0, 32, 32, 8, 128, 64, 8192) == 0
    for bp in (0, 10001, -5):
        rc = lib.sg_score_topshare(None, 1, 1, 1, 8, 8, 64, 32, P, 100, 100, P, P, 0, bp, P, P, 1 << 20)
        assert rc == smartgen.SG_EINVAL and "ratio_bp" in _err(lib)
    rc = lib.sg_score_topshare(None, 1, 1, 1, 8, 8, 96, 32, P, 100, 100, P, P, 0, 2000, P, P, 1 << 20)
    assert rc == smartgen.SG_EUNSUPPORTED and "head dimension" in _err(lib)
    rc = lib.sg_score_topshare(None, 1, 1, 1, 64, 8, 128, 65, P, 100, 100, P, P, 0, 2000, P, P, 1 << 20)
    assert rc == smartgen.SG_EUNSUPPORTED and "G*W" in _err(lib)
    rc = lib.sg_score_topshare(None, 1, 1, 1, 8, 8, 64, 32, P, 4096, 4096, P, P, 0, 2000, P, P, 16)
    assert rc == smartgen.SG_EWORKSPACE
    rc = lib.sg_score_topshare(None, 1, 1, 1, 8, 8, 64, 32, P, 0, 0, P, P, 0, 2000, P, P, 0)
    assert rc == smartgen.SG_OK                                             # nothing to do
