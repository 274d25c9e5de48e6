"""Python face of the plain CPU oracle (``sg_oracle.c``).

TEST INFRASTRUCTURE ONLY.  The tests, ``__graft_entry__.smoke()`` and the
bench's ``cpu_baseline`` leg may import this package; the product library and
its binding never do.  Every function takes and returns NumPy arrays on the
host; floating-point inputs are widened to float32 (exact for bf16 values) and
floating-point results come back in float64.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# SG_ORACLE_LIB points at another build of the same source (the sanitizer run)
LIB_PATH = os.environ.get("SG_ORACLE_LIB") or os.path.join(_HERE, "libsg_oracle.so")
_lib = None

_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_i8p = ctypes.POINTER(ctypes.c_int8)
_vp = ctypes.c_void_p
_i = ctypes.c_int
_l = ctypes.c_int64


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from .build import build
        build()
    lib = ctypes.CDLL(LIB_PATH)
    lib.sgo_score.argtypes = [_i, _i, _i, _i, _i, _i, _i32p, _l, _f32p, _f32p, _l, _f64p]
    lib.sgo_topk.argtypes = [_i, _i, _i, _i32p, _l, _i32p, _l, _f32p, _i32p]
    lib.sgo_pack.argtypes = [_i, _i, _i, _i, _i, _i32p, _l, _i32p, _l, _vp, _vp, _l, _i32p, _vp]
    lib.sgo_split.argtypes = [_i, _i32p, _i32p, _i8p, _i64p, _i32p, _i, _i32p, _i32p, _i32p, _i32p, _i32p]
    lib.sgo_fetch.argtypes = [_i, _i, _i, _i32p, _i32p, _i32p, _i64p, _l, _vp, _vp, _i32p, _i, _i, _i32p,
                              _vp, _vp, _l]
    lib.sgo_decode_attn.argtypes = [_i, _i, _i, _i, ctypes.c_double, _f32p, _f32p, _f32p, _l, _i32p, _i32p,
                                    _i, _i, _f64p]
    lib.sgo_block_importance.argtypes = [_i, _i, _i, _i32p, _l, _i, _f32p, _f64p]
    lib.sgo_pack_blocks.argtypes = [_i, _i, _i, _i, _l, _l, _l, _i, _vp, _vp, _l, _i, _i32p, _vp]
    lib.sgo_spec_push.argtypes = [_i, _i, _i, _i, _l, _l, _l, _i, _vp, _vp, _l, _vp, _vp, _l, _i, _i32p, _i8p,
                                  _f32p]
    lib.sgo_fetch_keep.argtypes = [_i, _i, _i, _i32p, _i32p, _i32p, _i64p, _l, _vp, _vp, _i32p, _i, _i, _i32p,
                                   _vp, _vp, _l, _i64p, _vp, _vp, _l, _i8p, _l, _i64p, _i32p]
    lib.sgo_score_count.argtypes = [_i, _i, _i, _i, _i, _i, _i32p, _l, _f32p, _f32p, _l, ctypes.c_double,
                                    ctypes.c_double, _i32p, _i32p]
    lib.sgo_score_topshare.argtypes = [_i, _i, _i, _i, _i, _i, _i32p, _l, _f32p, _f32p, _l, _i, ctypes.c_double,
                                       _i32p, _i32p]
    lib.sgo_decode_select.argtypes = [_i, _i, _i, _i, _i, _f32p, _i32p, _l, _f32p, _l, _i32p, _l, ctypes.c_double,
                                      ctypes.c_double, _i32p, _i32p, _f64p]
    for f in ("sgo_score", "sgo_topk", "sgo_pack", "sgo_split", "sgo_fetch", "sgo_decode_attn", "sgo_threads",
              "sgo_block_importance", "sgo_pack_blocks", "sgo_spec_push", "sgo_fetch_keep", "sgo_score_count",
              "sgo_decode_select", "sgo_score_topshare"):
        getattr(lib, f).restype = ctypes.c_int
    lib.sgo_set_threads.argtypes = [_i]
    lib.sgo_set_threads.restype = None
    _lib = lib
    return lib


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _p(a, ptype):
    return a.ctypes.data_as(ptype)


def _check(rc, name):
    if rc != 0:
        raise ValueError(f"oracle {name} rejected its arguments (status {rc})")


def threads() -> int:
    return _load().sgo_threads()


def set_threads(n: int) -> None:
    _load().sgo_set_threads(int(n))


def score(q_win, k, cu_seqlens, Hkv, k_layer_rows=None):
    """Scores [L][Hkv][T] float64.  q_win [B][L][Hq][W][d]; k [Lkv][Hkv][T][d]."""
    q = _c(q_win, np.float32)
    kk = _c(k, np.float32)
    B, L, Hq, W, d = q.shape
    T = kk.shape[2]
    if k_layer_rows is None:
        k_layer_rows = 0 if kk.shape[0] == 1 and L > 1 else Hkv * T
    cu = _c(cu_seqlens, np.int32)
    out = np.zeros((L, Hkv, T), dtype=np.float64)
    rc = _load().sgo_score(B, L, Hq, Hkv, d, W, _p(cu, _i32p), T, _p(q, _f32p), _p(kk, _f32p),
                           int(k_layer_rows), _p(out, _f64p))
    _check(rc, "score")
    return out


def topk(scores, cu_seqlens, cu_k):
    """idx [L][Hkv][K_total] int32 from float32 scores [L][Hkv][T]."""
    s = _c(scores, np.float32)
    L, Hkv, T = s.shape
    cu = _c(cu_seqlens, np.int32)
    ck = _c(cu_k, np.int32)
    B = len(cu) - 1
    K_total = int(ck[-1])
    out = np.empty((L, Hkv, K_total), dtype=np.int32)
    rc = _load().sgo_topk(B, L, Hkv, _p(cu, _i32p), T, _p(ck, _i32p), K_total, _p(s, _f32p), _p(out, _i32p))
    _check(rc, "topk")
    return out


def pack(k, v, idx, cu_seqlens, cu_k, kv_layer_rows=None):
    """Transfer buffer bytes [K rows | V rows | int32 idx] as a uint8 array."""
    assert k.dtype == v.dtype and k.shape == v.shape
    kk = np.ascontiguousarray(k)
    vv = np.ascontiguousarray(v)
    ix = _c(idx, np.int32)
    L, Hkv, K_total = ix.shape
    Lkv, _, T, d = kk.shape
    esize = kk.dtype.itemsize
    if kv_layer_rows is None:
        kv_layer_rows = 0 if Lkv == 1 and L > 1 else Hkv * T
    cu = _c(cu_seqlens, np.int32)
    ck = _c(cu_k, np.int32)
    B = len(cu) - 1
    S = L * Hkv * K_total
    out = np.zeros(2 * S * d * esize + 4 * S, dtype=np.uint8)
    rc = _load().sgo_pack(B, L, Hkv, d, esize, _p(cu, _i32p), T, _p(ck, _i32p), K_total,
                          kk.ctypes.data, vv.ctypes.data, int(kv_layer_rows), _p(ix, _i32p), out.ctypes.data)
    _check(rc, "pack")
    return out


def split(row_off, kv_index, mask, mask_off, mask_len, reorder):
    """Algorithm 1.  Returns (out_index or None, local, remote, n_local, n_remote)."""
    ro = _c(row_off, np.int32)
    ix = _c(kv_index, np.int32)
    m = _c(mask, np.int8)
    mo = _c(mask_off, np.int64)
    ml = _c(mask_len, np.int32)
    rows = len(ro) - 1
    n = max(int(ro[-1]), 1)
    out = np.full(n, -1, dtype=np.int32)
    loc = np.full(n, -1, dtype=np.int32)
    rem = np.full(n, -1, dtype=np.int32)
    nl = np.zeros(max(rows, 1), dtype=np.int32)
    nr = np.zeros(max(rows, 1), dtype=np.int32)
    rc = _load().sgo_split(rows, _p(ro, _i32p), _p(ix, _i32p), _p(m, _i8p), _p(mo, _i64p), _p(ml, _i32p),
                           int(bool(reorder)), _p(out, _i32p), _p(loc, _i32p), _p(rem, _i32p),
                           _p(nl, _i32p), _p(nr, _i32p))
    _check(rc, "split")
    t = int(ro[-1])
    return (out[:t] if reorder else None), loc[:t], rem[:t], nl[:rows], nr[:rows]


def fetch(row_off, index, n_valid, src_row_base, k_src, v_src, page_table, page_size, dst_start,
          k_pool, v_pool):
    """Copies rows into k_pool / v_pool (modified in place, 2-D [pool_rows][d])."""
    ro = _c(row_off, np.int32)
    rows = len(ro) - 1
    ix = None if index is None else _c(index, np.int32)
    nv = None if n_valid is None else _c(n_valid, np.int32)
    sb = _c(src_row_base, np.int64)
    ks = np.ascontiguousarray(k_src)
    vs = np.ascontiguousarray(v_src)
    pt = _c(page_table, np.int32)
    ds = _c(dst_start, np.int32)
    assert k_pool.flags.c_contiguous and v_pool.flags.c_contiguous
    d = ks.shape[-1]
    esize = ks.dtype.itemsize
    max_pages = pt.shape[-1]
    src_rows = ks.size // d
    pool_rows = k_pool.size // d
    rc = _load().sgo_fetch(rows, esize, d, _p(ro, _i32p), None if ix is None else _p(ix, _i32p),
                           None if nv is None else _p(nv, _i32p), _p(sb, _i64p), src_rows,
                           ks.ctypes.data, vs.ctypes.data, _p(pt, _i32p), int(page_size), int(max_pages),
                           _p(ds, _i32p), k_pool.ctypes.data, v_pool.ctypes.data, pool_rows)
    _check(rc, "fetch")


def decode_attn(q, k_pool, v_pool, page_table, n_rows, page_size, scale=None):
    """o [B][Hq][d] float64.  q [B][Hq][d]; pools [pool_rows][d]; page_table [B][Hkv][max_pages]."""
    qq = _c(q, np.float32)
    kp = _c(k_pool, np.float32)
    vp = _c(v_pool, np.float32)
    pt = _c(page_table, np.int32)
    nr = _c(n_rows, np.int32)
    B, Hq, d = qq.shape
    _, Hkv, max_pages = pt.shape
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros((B, Hq, d), dtype=np.float64)
    rc = _load().sgo_decode_attn(B, Hq, Hkv, d, float(scale), _p(qq, _f32p), _p(kp, _f32p), _p(vp, _f32p),
                                 kp.shape[0], _p(pt, _i32p), _p(nr, _i32p), int(page_size), int(max_pages),
                                 _p(out, _f64p))
    _check(rc, "decode_attn")
    return out


def block_importance(scores, cu_seqlens, M):
    """Eq. 1 block importance [B][L][M] float64 from float32 scores [L][Hkv][T]."""
    sc = _c(scores, np.float32)
    L, Hkv, T = sc.shape
    cu = _c(cu_seqlens, np.int32)
    B = len(cu) - 1
    out = np.zeros((B, L, M), dtype=np.float64)
    rc = _load().sgo_block_importance(B, L, Hkv, _p(cu, _i32p), T, int(M), _p(sc, _f32p), _p(out, _f64p))
    _check(rc, "block_importance")
    return out


def block_budget(M, L, Tp, Tt):
    """Eq. 2: K_r = M (L - 1) Tp / Tt blocks (an upper bound, so floored), clipped to [2M, L M]."""
    if M < 1 or L < 1 or not (Tp >= 0) or not (Tt >= 0):
        raise ValueError("block_budget needs M, L >= 1 and non-negative times")
    k = L * M if Tt == 0 else int(np.floor(M * (L - 1) * (Tp / Tt)))
    return min(L * M, max(2 * M, k))


def pack_blocks(k, v, ids, s0, N, M, L=None, kv_layer_rows=None):
    """Block transfer buffer [K rows | V rows | int32 ids] (uint8) of one request.
    k, v: [Lkv][Hkv][T][d]; L layers (default Lkv); kv_layer_rows: layer stride in rows
    (default Hkv * T; 0 for one source shared by every layer)."""
    assert k.dtype == v.dtype and k.shape == v.shape
    kk = np.ascontiguousarray(k)
    vv = np.ascontiguousarray(v)
    ix = _c(ids, np.int32)
    _, Hkv, T, d = kk.shape
    return _pack_blocks(kk, vv, ix, s0, N, M, kv_layer_rows, Hkv, T, d, L=L)


def _pack_blocks(kk, vv, ix, s0, N, M, kv_layer_rows, Hkv, T, d, L=None):
    esize = kk.dtype.itemsize
    if L is None:
        L = kk.shape[0]
    if kv_layer_rows is None:
        kv_layer_rows = Hkv * T
    Nb = (N + M - 1) // M
    S = len(ix) * Hkv * Nb
    out = np.zeros(2 * S * d * esize + 4 * len(ix), dtype=np.uint8)
    rc = _load().sgo_pack_blocks(L, Hkv, d, esize, T, int(s0), int(N), int(M), kk.ctypes.data, vv.ctypes.data,
                                 int(kv_layer_rows), len(ix), _p(ix, _i32p), out.ctypes.data)
    _check(rc, "pack_blocks")
    return out


def spec_quota(blocks, ratio_bp):
    """Section 4.3: a speculative transfer sends a fixed fraction (the
    speculative ratio, in basis points) of all KV blocks, rounded up so that
    1 / ratio transfers deliver everything; at least one block."""
    if blocks < 0 or ratio_bp < 1:
        raise ValueError("spec_quota needs blocks >= 0 and a positive ratio")
    return min(blocks, max(1, -(-blocks * ratio_bp // 10000)))


def spec_push(k_src, v_src, ids, s0, N, M, k_dst, v_dst, mask, rem=None, L=None, src_layer_rows=None,
              dst_layer_rows=None):
    """Section 4.3: copies the blocks `ids` of one request from the prefill
    side's K/V [Lkv][Hkv][T][d] into the decode side's store [Ld][Hkv][T][d] at
    the same rows, sets their mask [L][Hkv][T] (int8) entries to 1 and their
    entries of rem [L*M] (float32) to NaN.  k_dst, v_dst, mask, rem change in place."""
    assert k_src.dtype == v_src.dtype == k_dst.dtype == v_dst.dtype
    for a in (k_src, v_src, k_dst, v_dst, mask):
        assert a.flags.c_contiguous
    assert mask.dtype == np.int8 and (rem is None or (rem.dtype == np.float32 and rem.flags.c_contiguous))
    _, Hkv, T, d = k_src.shape
    if L is None:
        L = k_src.shape[0]
    ix = _c(ids, np.int32)
    rc = _load().sgo_spec_push(int(L), Hkv, d, k_src.dtype.itemsize, T, int(s0), int(N), int(M),
                               k_src.ctypes.data, v_src.ctypes.data,
                               Hkv * T if src_layer_rows is None else int(src_layer_rows),
                               k_dst.ctypes.data, v_dst.ctypes.data,
                               Hkv * T if dst_layer_rows is None else int(dst_layer_rows),
                               len(ix), _p(ix, _i32p), _p(mask, _i8p), None if rem is None else _p(rem, _f32p))
    _check(rc, "spec_push")


def fetch_keep(row_off, index, n_valid, src_row_base, k_src, v_src, page_table, page_size, dst_start,
               k_pool, v_pool, keep_row_base, k_keep, v_keep, mask, mask_off, mask_len):
    """The fetch of `fetch` (pool written when page_table is not None) that also
    keeps every copied row at keep row keep_row_base[r] + index and turns its
    mask entry to 1.  Pools, keep arrays (2-D [rows][d]) and mask change in place."""
    ro = _c(row_off, np.int32)
    rows = len(ro) - 1
    ix = _c(index, np.int32)
    nv = None if n_valid is None else _c(n_valid, np.int32)
    sb = _c(src_row_base, np.int64)
    kb = _c(keep_row_base, np.int64)
    ks = np.ascontiguousarray(k_src)
    vs = np.ascontiguousarray(v_src)
    d = ks.shape[-1]
    for a in (k_keep, v_keep) + ((k_pool, v_pool) if page_table is not None else ()):
        assert a.flags.c_contiguous and a.dtype == ks.dtype
    pt = None if page_table is None else _c(page_table, np.int32)
    ds = _c(dst_start, np.int32)
    max_pages = 1 if pt is None else pt.shape[-1]
    mo = None if mask is None else _c(mask_off, np.int64)
    ml = None if mask is None else _c(mask_len, np.int32)
    if mask is not None:
        assert mask.dtype == np.int8 and mask.flags.c_contiguous
    rc = _load().sgo_fetch_keep(rows, ks.dtype.itemsize, d, _p(ro, _i32p), _p(ix, _i32p),
                                None if nv is None else _p(nv, _i32p), _p(sb, _i64p), ks.size // d,
                                ks.ctypes.data, vs.ctypes.data, None if pt is None else _p(pt, _i32p),
                                int(page_size), int(max_pages), _p(ds, _i32p),
                                None if pt is None else k_pool.ctypes.data, None if pt is None else v_pool.ctypes.data,
                                0 if pt is None else k_pool.size // d,
                                _p(kb, _i64p), k_keep.ctypes.data, v_keep.ctypes.data, k_keep.size // d,
                                None if mask is None else _p(mask, _i8p), 0 if mask is None else mask.size,
                                None if mask is None else _p(mo, _i64p), None if mask is None else _p(ml, _i32p))
    _check(rc, "fetch_keep")


def score_count(q_win, k, cu_seqlens, Hkv, alpha, k_layer_rows=None, eps=None):
    """Selection counts [L][Hkv][T] int32 under the alpha rule (and, with eps, the
    per-key number of decisions within eps of the threshold: (counts, near))."""
    q = _c(q_win, np.float32)
    kk = _c(k, np.float32)
    B, L, Hq, W, d = q.shape
    T = kk.shape[2]
    if k_layer_rows is None:
        k_layer_rows = 0 if kk.shape[0] == 1 and L > 1 else Hkv * T
    cu = _c(cu_seqlens, np.int32)
    out = np.zeros((L, Hkv, T), dtype=np.int32)
    near = np.zeros((L, Hkv, T), dtype=np.int32) if eps is not None else None
    rc = _load().sgo_score_count(B, L, Hq, Hkv, d, W, _p(cu, _i32p), T, _p(q, _f32p), _p(kk, _f32p),
                                 int(k_layer_rows), float(alpha), float(eps or 0.0), _p(out, _i32p),
                                 None if near is None else _p(near, _i32p))
    _check(rc, "score_count")
    return out if eps is None else (out, near)


def score_topshare(q_win, k, cu_seqlens, Hkv, ratio_bp, k_layer_rows=None, eps=None):
    """Selection counts [L][Hkv][T] int32 when every window row picks its top
    ratio_bp / 10000 of the keys it sees (ties with the row's threshold all
    picked); with eps also the per-key number of decisions within eps of a
    row's threshold: (counts, near)."""
    q = _c(q_win, np.float32)
    kk = _c(k, np.float32)
    B, L, Hq, W, d = q.shape
    T = kk.shape[2]
    if k_layer_rows is None:
        k_layer_rows = 0 if kk.shape[0] == 1 and L > 1 else Hkv * T
    cu = _c(cu_seqlens, np.int32)
    out = np.zeros((L, Hkv, T), dtype=np.int32)
    near = np.zeros((L, Hkv, T), dtype=np.int32) if eps is not None else None
    rc = _load().sgo_score_topshare(B, L, Hq, Hkv, d, W, _p(cu, _i32p), T, _p(q, _f32p), _p(kk, _f32p),
                                    int(k_layer_rows), int(ratio_bp), float(eps or 0.0), _p(out, _i32p),
                                    None if near is None else _p(near, _i32p))
    _check(rc, "score_topshare")
    return out if eps is None else (out, near)


def decode_select(q, k, cu_seqlens, Hkv, cu_cap, alpha, k_layer_rows=None, scale=None):
    """Decode-time selection: (idx [L][Hkv][K_cap] int32, n_sel [B][L][Hkv] int32,
    r [L][Hkv][T] float64).  q [B][L][Hq][d]; k [Lkv][Hkv][T][d]; scale defaults
    to 1/sqrt(d) (pass the full head's for partial channels)."""
    qq = _c(q, np.float32)
    kk = _c(k, np.float32)
    B, L, Hq, d = qq.shape
    T = kk.shape[2]
    if k_layer_rows is None:
        k_layer_rows = 0 if kk.shape[0] == 1 and L > 1 else Hkv * T
    cu = _c(cu_seqlens, np.int32)
    cc = _c(cu_cap, np.int32)
    K_cap = int(cc[-1])
    idx = np.full((L, Hkv, max(K_cap, 1)), -7, dtype=np.int32)
    n_sel = np.zeros((B, L, Hkv), dtype=np.int32)
    r = np.full((L, Hkv, max(T, 1)), np.nan)
    rc = _load().sgo_decode_select(B, L, Hq, Hkv, d, _p(qq, _f32p), _p(cu, _i32p), T, _p(kk, _f32p),
                                   int(k_layer_rows), _p(cc, _i32p), K_cap, float(alpha),
                                   float(d ** -0.5 if scale is None else scale), _p(idx, _i32p),
                                   _p(n_sel, _i32p), _p(r, _f64p))
    _check(rc, "decode_select")
    return idx[:, :, :K_cap], n_sel, r[:, :, :T]
