"""ctypes binding of libsmartgen.so (the C ABI declared in include/smartgen.h).

Argument marshalling only: every function takes torch tensors (device memory or
pinned host memory), checks dtypes/shapes that the C call cannot see, passes
raw pointers and the current HIP stream, and raises ``SmartgenError`` on a
non-zero status.  All computation runs in the library's HIP kernels.  There is
no fallback: if the library is missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# SG_LIB_PATH points at another build of the same sources (the sanitizer run)
LIB_PATH = os.environ.get("SG_LIB_PATH") or os.path.join(_HERE, "libsmartgen.so")

SG_F32, SG_BF16 = 0, 1
SG_OK, SG_EINVAL, SG_EUNSUPPORTED, SG_EWORKSPACE, SG_EHIP, SG_EINTERNAL = 0, -1, -2, -3, -4, -5

EXPORTS = [
    "sg_version", "sg_status_str", "sg_last_error",
    "sg_score_workspace_size", "sg_score",
    "sg_topk",
    "sg_pack_bytes", "sg_pack",
    "sg_split",
    "sg_fetch",
    "sg_decode_attn_workspace_size", "sg_decode_attn", "sg_decode_attn_noalloc_scratch_bytes",
    "sg_decode_attn_noalloc",
    "sg_block_importance", "sg_block_budget", "sg_pack_blocks_bytes", "sg_pack_blocks",
    "sg_fetch_keep", "sg_spec_quota", "sg_spec_push", "sg_spec_commit", "sg_score_count",
    "sg_decode_select_workspace_size", "sg_decode_select",
    "sg_score_topshare_workspace_size", "sg_score_topshare",
]


class SmartgenError(RuntimeError):
    def __init__(self, fn: str, status: int, detail: str):
        super().__init__(f"{fn} failed with status {status}: {detail}")
        self.status = status


_lib = None
_vp, _i, _l, _sz, _f = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float


def load() -> ctypes.CDLL:
    """Load libsmartgen.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_28150_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    lib.sg_version.restype = _i
    lib.sg_status_str.argtypes = [_i]
    lib.sg_status_str.restype = ctypes.c_char_p
    lib.sg_last_error.restype = ctypes.c_char_p
    lib.sg_score_workspace_size.argtypes = [_i] * 7
    lib.sg_score_workspace_size.restype = _sz
    lib.sg_score.argtypes = [_vp, _i, _i, _i, _i, _i, _i, _i, _vp, _l, _i, _vp, _vp, _l, _vp, _vp, _vp, _sz]
    lib.sg_topk.argtypes = [_vp, _i, _i, _i, _vp, _l, _i, _vp, _l, _vp, _vp]
    lib.sg_pack_bytes.argtypes = [_i, _i, _i, _i, _l]
    lib.sg_pack_bytes.restype = _sz
    lib.sg_pack.argtypes = [_vp, _i, _i, _i, _i, _i, _vp, _l, _vp, _l, _i, _vp, _vp, _l, _vp, _vp, _sz, _i]
    lib.sg_split.argtypes = [_vp, _i, _vp, _l, _vp, _vp, _l, _vp, _vp, _i, _vp, _vp, _vp, _vp, _vp, _vp]
    lib.sg_fetch.argtypes = [_vp, _i, _i, _i, _vp, _l, _vp, _vp, _vp, _l, _vp, _vp, _vp, _i, _i, _vp, _vp, _vp, _l]
    lib.sg_decode_attn_workspace_size.argtypes = [_i] * 6
    lib.sg_decode_attn_workspace_size.restype = _sz
    lib.sg_decode_attn.argtypes = [_vp, _i, _i, _i, _i, _i, _f, _vp, _vp, _vp, _l, _vp, _vp, _i, _i, _vp, _vp, _sz]
    lib.sg_decode_attn_noalloc.argtypes = [_vp, _i, _i, _i, _i, _i, _f, _vp, _vp, _vp, _l, _vp, _vp, _i, _i, _vp]
    lib.sg_decode_attn_noalloc_scratch_bytes.restype = _sz
    lib.sg_block_importance.argtypes = [_vp, _i, _i, _i, _vp, _l, _i, _vp, _vp]
    lib.sg_block_budget.argtypes = [_i, _i, ctypes.c_double, ctypes.c_double]
    lib.sg_block_budget.restype = _l
    lib.sg_pack_blocks_bytes.argtypes = [_i, _i, _i, _l, _i, _i]
    lib.sg_pack_blocks_bytes.restype = _sz
    lib.sg_pack_blocks.argtypes = [_vp, _i, _i, _i, _i, _l, _l, _l, _i, _vp, _vp, _l, _i, _vp, _vp, _sz]
    lib.sg_fetch_keep.argtypes = [_vp, _i, _i, _i, _vp, _l, _vp, _vp, _vp, _l, _vp, _vp, _vp, _i, _i, _vp, _vp, _vp,
                                  _l, _vp, _vp, _vp, _l, _vp, _l, _vp, _vp]
    lib.sg_score_count.argtypes = [_vp, _i, _i, _i, _i, _i, _i, _i, _vp, _l, _i, _vp, _vp, _l, _f, _vp, _vp, _sz]
    lib.sg_score_topshare_workspace_size.argtypes = [_i] * 7
    lib.sg_score_topshare_workspace_size.restype = _sz
    lib.sg_score_topshare.argtypes = [_vp, _i, _i, _i, _i, _i, _i, _i, _vp, _l, _i, _vp, _vp, _l, _i, _vp, _vp, _sz]
    lib.sg_decode_select_workspace_size.argtypes = [_i, _i, _i, _i]
    lib.sg_decode_select_workspace_size.restype = _sz
    lib.sg_decode_select.argtypes = [_vp, _i, _i, _i, _i, _i, _i, _vp, _vp, _l, _i, _vp, _l, _f, _f, _vp, _l, _vp,
                                     _vp, _vp, _sz]
    lib.sg_spec_quota.argtypes = [_l, _i]
    lib.sg_spec_quota.restype = _l
    lib.sg_spec_push.argtypes = [_vp, _i, _i, _i, _i, _l, _l, _l, _i, _vp, _vp, _l, _vp, _vp, _l, _i, _vp, _vp, _vp]
    lib.sg_spec_commit.argtypes = [_vp, _i, _i, _l, _l, _l, _i, _i, _vp, _vp, _vp]
    for f in ("sg_score", "sg_topk", "sg_pack", "sg_split", "sg_fetch", "sg_decode_attn", "sg_decode_attn_noalloc",
              "sg_block_importance",
              "sg_pack_blocks", "sg_fetch_keep", "sg_spec_push", "sg_spec_commit", "sg_score_count",
              "sg_decode_select", "sg_score_topshare"):
        getattr(lib, f).restype = _i
    _lib = lib
    return lib


def version() -> int:
    return load().sg_version()


def _check(fn: str, rc: int) -> None:
    if rc != SG_OK:
        raise SmartgenError(fn, rc, load().sg_last_error().decode())


_hip = None


def _hip_runtime():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipHostGetDevicePointer.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_void_p, ctypes.c_uint]
        _hip.hipHostGetDevicePointer.restype = ctypes.c_int
    return _hip


def _ptr(t):
    """Device-usable address of a tensor: device memory as is, pinned host memory
    through hipHostGetDevicePointer (pageable host memory is refused)."""
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    if t.is_cuda or t.numel() == 0:
        return ctypes.c_void_p(t.data_ptr())
    if not t.is_pinned():
        raise ValueError("host tensors passed to the library must be pinned (pin_memory=True)")
    dptr = ctypes.c_void_p()
    rc = _hip_runtime().hipHostGetDevicePointer(ctypes.byref(dptr), ctypes.c_void_p(t.data_ptr()), 0)
    if rc != 0 or not dptr.value:
        raise RuntimeError(f"hipHostGetDevicePointer failed ({rc}) for a pinned tensor")
    return dptr


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return SG_F32
    if t.dtype == torch.bfloat16:
        return SG_BF16
    raise TypeError(f"unsupported element type {t.dtype}")


def _need(cond: bool, msg: str) -> None:
    if not cond:
        raise ValueError(msg)


# ------------------------------------------------------------------------ score

def score_workspace_size(B, L, Hq, Hkv, d, W, max_seqlen) -> int:
    return int(load().sg_score_workspace_size(B, L, Hq, Hkv, d, W, max_seqlen))


def sg_score(q_win, k, cu_seqlens, T, max_seqlen, Hkv, scores, ws=None, lse_in=None, k_layer_rows=None,
             stream=None):
    """scores[L][Hkv][T] (float32, written) from q_win [B][L][Hq][W][d] and k rows."""
    B, L, Hq, W, d = q_win.shape
    _need(k.dtype == q_win.dtype, "q_win and k must share a dtype")
    _need(scores.dtype == torch.float32 and scores.numel() >= L * Hkv * T, "scores must be float32 [L][Hkv][T]")
    _need(cu_seqlens.dtype == torch.int32 and cu_seqlens.numel() == B + 1, "cu_seqlens must be int32 [B+1]")
    if k_layer_rows is None:
        k_layer_rows = 0 if (k.dim() == 4 and k.shape[0] == 1 and L > 1) else Hkv * T
    _need(k.numel() >= ((L - 1) * k_layer_rows + Hkv * T) * d, "k is smaller than its layout needs")
    _need(lse_in is None or (lse_in.dtype == torch.float32 and lse_in.numel() >= B * L * Hq * W),
          "lse_in must be float32 [B][L][Hq][W]")
    rc = load().sg_score(_stream(stream), _dtype_code(q_win), B, L, Hq, Hkv, d, W, _ptr(cu_seqlens), int(T),
                         int(max_seqlen), _ptr(q_win), _ptr(k), int(k_layer_rows), _ptr(lse_in), _ptr(scores),
                         _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size())
    _check("sg_score", rc)
    return scores


def sg_score_count(q_win, k, cu_seqlens, T, max_seqlen, Hkv, counts, alpha, ws, k_layer_rows=None, stream=None):
    """counts[L][Hkv][T] (float32 integers, written): how many (q head, window row)
    pairs pick each key under the rule logit >= row max - alpha."""
    B, L, Hq, W, d = q_win.shape
    _need(k.dtype == q_win.dtype, "q_win and k must share a dtype")
    _need(counts.dtype == torch.float32 and counts.numel() >= L * Hkv * T, "counts must be float32 [L][Hkv][T]")
    _need(cu_seqlens.dtype == torch.int32 and cu_seqlens.numel() == B + 1, "cu_seqlens must be int32 [B+1]")
    if k_layer_rows is None:
        k_layer_rows = 0 if (k.dim() == 4 and k.shape[0] == 1 and L > 1) else Hkv * T
    _need(k.numel() >= ((L - 1) * k_layer_rows + Hkv * T) * d, "k is smaller than its layout needs")
    rc = load().sg_score_count(_stream(stream), _dtype_code(q_win), B, L, Hq, Hkv, d, W, _ptr(cu_seqlens), int(T),
                               int(max_seqlen), _ptr(q_win), _ptr(k), int(k_layer_rows), float(alpha), _ptr(counts),
                               _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size())
    _check("sg_score_count", rc)
    return counts


def score_topshare_workspace_size(B, L, Hq, Hkv, d, W, max_seqlen) -> int:
    return int(load().sg_score_topshare_workspace_size(B, L, Hq, Hkv, d, W, max_seqlen))


def sg_score_topshare(q_win, k, cu_seqlens, T, max_seqlen, Hkv, counts, ratio_bp, ws, k_layer_rows=None,
                      stream=None):
    """counts[L][Hkv][T] (float32 integers, written): how many (q head, window row)
    pairs pick each key when every row picks its top ratio_bp / 10000 of the
    keys it sees (ties with the row's threshold included)."""
    B, L, Hq, W, d = q_win.shape
    _need(k.dtype == q_win.dtype, "q_win and k must share a dtype")
    _need(counts.dtype == torch.float32 and counts.numel() >= L * Hkv * T, "counts must be float32 [L][Hkv][T]")
    _need(cu_seqlens.dtype == torch.int32 and cu_seqlens.numel() == B + 1, "cu_seqlens must be int32 [B+1]")
    if k_layer_rows is None:
        k_layer_rows = 0 if (k.dim() == 4 and k.shape[0] == 1 and L > 1) else Hkv * T
    _need(k.numel() >= ((L - 1) * k_layer_rows + Hkv * T) * d, "k is smaller than its layout needs")
    rc = load().sg_score_topshare(_stream(stream), _dtype_code(q_win), B, L, Hq, Hkv, d, W, _ptr(cu_seqlens),
                                  int(T), int(max_seqlen), _ptr(q_win), _ptr(k), int(k_layer_rows), int(ratio_bp),
                                  _ptr(counts), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size())
    _check("sg_score_topshare", rc)
    return counts


def decode_select_workspace_size(B, L, Hq, max_seqlen) -> int:
    return int(load().sg_decode_select_workspace_size(B, L, Hq, max_seqlen))


def sg_decode_select(q, k, cu_seqlens, T, max_seqlen, Hkv, cu_cap, K_cap, idx, n_sel, alpha, ws,
                     k_layer_rows=None, scale=None, stream=None):
    """Decode-time selection: idx [L][Hkv][K_cap] (ids ascending, then -1) and
    n_sel [B][L][Hkv] from the step's queries q [B][L][Hq][d] and the keys (whole
    heads or a partial set of channels; scale defaults to 1/sqrt(d))."""
    B, L, Hq, d = q.shape
    _need(k.dtype == q.dtype, "q and k must share a dtype")
    _need(cu_seqlens.dtype == torch.int32 and cu_seqlens.numel() == B + 1, "cu_seqlens must be int32 [B+1]")
    _need(cu_cap.dtype == torch.int32 and cu_cap.numel() == B + 1, "cu_cap must be int32 [B+1]")
    _need(idx.dtype == torch.int32 and idx.numel() >= L * Hkv * K_cap, "idx must be int32 [L][Hkv][K_cap]")
    _need(n_sel.dtype == torch.int32 and n_sel.numel() >= B * L * Hkv, "n_sel must be int32 [B][L][Hkv]")
    if k_layer_rows is None:
        k_layer_rows = 0 if (k.dim() == 4 and k.shape[0] == 1 and L > 1) else Hkv * T
    _need(k.numel() >= ((L - 1) * k_layer_rows + Hkv * T) * d, "k is smaller than its layout needs")
    rc = load().sg_decode_select(_stream(stream), _dtype_code(q), B, L, Hq, Hkv, d, _ptr(q), _ptr(cu_seqlens), int(T),
                                 int(max_seqlen), _ptr(k), int(k_layer_rows), float(scale or 0.0), float(alpha),
                                 _ptr(cu_cap),
                                 int(K_cap), _ptr(idx), _ptr(n_sel), _ptr(ws),
                                 0 if ws is None else ws.numel() * ws.element_size())
    _check("sg_decode_select", rc)
    return idx


# ------------------------------------------------------------------------ topk

def sg_topk(scores, cu_seqlens, T, max_seqlen, cu_k, K_total, idx, B=None, stream=None):
    L, Hkv = scores.shape[0], scores.shape[1]
    B = cu_seqlens.numel() - 1 if B is None else B
    _need(scores.dtype == torch.float32 and scores.numel() >= L * Hkv * T, "scores must be float32 [L][Hkv][T]")
    _need(cu_seqlens.numel() >= B + 1 and cu_k.numel() >= B + 1, "cu_seqlens and cu_k need B+1 entries")
    _need(idx.dtype == torch.int32 and idx.numel() >= L * Hkv * K_total, "idx must be int32 [L][Hkv][K_total]")
    rc = load().sg_topk(_stream(stream), B, L, Hkv, _ptr(cu_seqlens), int(T), int(max_seqlen), _ptr(cu_k),
                        int(K_total), _ptr(scores), _ptr(idx))
    _check("sg_topk", rc)
    return idx


# ------------------------------------------------------------------------ pack

def pack_bytes(dtype: torch.dtype, L, Hkv, d, K_total) -> int:
    code = SG_F32 if dtype == torch.float32 else SG_BF16
    return int(load().sg_pack_bytes(code, L, Hkv, d, int(K_total)))


def sg_pack(k, v, idx, cu_seqlens, T, cu_k, K_total, max_k, dst, L=None, Hkv=None, kv_layer_rows=None,
            stream=None, max_workgroups=0):
    """Writes [K rows | V rows | idx] of every unit into ``dst`` (uint8, device or pinned host).
    max_workgroups > 0 caps the launch's workgroups (a pack beside other kernels)."""
    _need(k.dtype == v.dtype, "k and v must share a dtype")
    L = idx.shape[0] if L is None else L
    Hkv = idx.shape[1] if Hkv is None else Hkv
    d = k.shape[-1]
    B = cu_seqlens.numel() - 1
    if kv_layer_rows is None:
        kv_layer_rows = 0 if (k.dim() == 4 and k.shape[0] == 1 and L > 1) else Hkv * T
    rows_needed = ((L - 1) * kv_layer_rows + Hkv * T) * d
    _need(k.numel() >= rows_needed and v.numel() >= rows_needed, "k / v smaller than their layout needs")
    _need(idx.dtype == torch.int32 and idx.numel() >= L * Hkv * K_total, "idx must be int32 [L][Hkv][K_total]")
    _need(cu_k.numel() == B + 1, "cu_k must have B+1 entries")
    rc = load().sg_pack(_stream(stream), _dtype_code(k), B, L, Hkv, d, _ptr(cu_seqlens), int(T), _ptr(cu_k),
                        int(K_total), int(max_k), _ptr(k), _ptr(v), int(kv_layer_rows), _ptr(idx), _ptr(dst),
                        dst.numel() * dst.element_size(), int(max_workgroups))
    _check("sg_pack", rc)
    return dst


# ------------------------------------------------------------------------ split

def sg_split(row_off, kv_index, mask, mask_off, mask_len, reorder, local, remote, n_local, n_remote,
             out_index=None, n_kept=None, stream=None):
    rows = row_off.numel() - 1
    total = kv_index.numel()
    _need(mask.dtype == torch.int8, "mask must be int8")
    for t in (mask_off, mask_len, n_local, n_remote) + ((n_kept,) if n_kept is not None else ()):
        _need(t.numel() >= rows, "per-row arrays need one entry per row")
    for t in (local, remote) + ((out_index,) if out_index is not None else ()):
        _need(t.numel() >= total, "outputs need one entry per index")
    rc = load().sg_split(_stream(stream), rows, _ptr(row_off), int(total), _ptr(kv_index), _ptr(mask),
                         mask.numel(), _ptr(mask_off), _ptr(mask_len), int(bool(reorder)), _ptr(out_index),
                         _ptr(local), _ptr(remote), _ptr(n_local), _ptr(n_remote), _ptr(n_kept))
    _check("sg_split", rc)


# ------------------------------------------------------------------------ fetch

def sg_fetch(row_off, total, index, n_valid, src_row_base, k_src, v_src, page_table, page_size, dst_start,
             k_pool, v_pool, stream=None):
    rows = row_off.numel() - 1
    d = k_src.shape[-1]
    _need(k_pool.dtype == k_src.dtype and v_pool.dtype == v_src.dtype, "pool and source dtypes differ")
    max_pages = page_table.shape[-1]
    src_rows = k_src.numel() // d
    pool_rows = k_pool.numel() // d
    _need(v_src.numel() >= src_rows * d and v_pool.numel() >= pool_rows * d, "v arrays smaller than k arrays")
    _need(page_table.numel() >= rows * max_pages, "page_table must be [rows][max_pages]")
    _need(src_row_base.dtype == torch.int64 and src_row_base.numel() >= rows, "src_row_base must be int64 [rows]")
    _need(dst_start.numel() >= rows and (n_valid is None or n_valid.numel() >= rows), "per-row arrays too short")
    _need(index is None or index.numel() >= total, "index shorter than total")
    rc = load().sg_fetch(_stream(stream), _dtype_code(k_src), d, rows, _ptr(row_off), int(total), _ptr(index),
                         _ptr(n_valid), _ptr(src_row_base), src_rows, _ptr(k_src), _ptr(v_src), _ptr(page_table),
                         int(page_size), int(max_pages), _ptr(dst_start), _ptr(k_pool), _ptr(v_pool), pool_rows)
    _check("sg_fetch", rc)


def sg_fetch_keep(row_off, total, index, n_valid, src_row_base, k_src, v_src, page_table, page_size, dst_start,
                  k_pool, v_pool, keep_row_base, k_keep, v_keep, mask=None, mask_off=None, mask_len=None,
                  stream=None):
    """sg_fetch that also keeps each fetched row at keep row keep_row_base[r] + index
    of k_keep / v_keep and turns its mask entry local; page_table=None skips the pool."""
    rows = row_off.numel() - 1
    d = k_src.shape[-1]
    _need(k_keep.dtype == k_src.dtype and v_keep.dtype == v_src.dtype, "store and source dtypes differ")
    src_rows = k_src.numel() // d
    keep_rows = k_keep.numel() // d
    _need(v_src.numel() >= src_rows * d and v_keep.numel() >= keep_rows * d, "v arrays smaller than k arrays")
    _need(keep_row_base.dtype == torch.int64 and keep_row_base.numel() >= rows, "keep_row_base must be int64 [rows]")
    _need(src_row_base.dtype == torch.int64 and src_row_base.numel() >= rows, "src_row_base must be int64 [rows]")
    _need(index is not None and index.numel() >= total, "index shorter than total")
    _need(n_valid is None or n_valid.numel() >= rows, "n_valid too short")
    max_pages, pool_rows = 1, 0
    if page_table is not None:
        _need(k_pool.dtype == k_src.dtype and v_pool.dtype == v_src.dtype, "pool and source dtypes differ")
        max_pages = page_table.shape[-1]
        pool_rows = k_pool.numel() // d
        _need(v_pool.numel() >= pool_rows * d, "v_pool smaller than k_pool")
        _need(page_table.numel() >= rows * max_pages, "page_table must be [rows][max_pages]")
        _need(dst_start.numel() >= rows, "dst_start too short")
    if mask is not None:
        _need(mask.dtype == torch.int8, "mask must be int8")
        _need(mask_off.dtype == torch.int64 and mask_off.numel() >= rows and mask_len.numel() >= rows,
              "mask_off (int64) and mask_len need one entry per row")
    rc = load().sg_fetch_keep(_stream(stream), _dtype_code(k_src), d, rows, _ptr(row_off), int(total), _ptr(index),
                              _ptr(n_valid), _ptr(src_row_base), src_rows, _ptr(k_src), _ptr(v_src),
                              _ptr(page_table), int(page_size), int(max_pages),
                              _ptr(dst_start) if page_table is not None else None,
                              _ptr(k_pool) if page_table is not None else None,
                              _ptr(v_pool) if page_table is not None else None, pool_rows,
                              _ptr(keep_row_base), _ptr(k_keep), _ptr(v_keep), keep_rows,
                              _ptr(mask), 0 if mask is None else mask.numel(),
                              _ptr(mask_off) if mask is not None else None,
                              _ptr(mask_len) if mask is not None else None)
    _check("sg_fetch_keep", rc)


# ------------------------------------------------------------------------ decode attention

def decode_workspace_size(B, Hq, Hkv, d, max_pages, page_size) -> int:
    return int(load().sg_decode_attn_workspace_size(B, Hq, Hkv, d, max_pages, page_size))


def sg_decode_attn(q, k_pool, v_pool, page_table, n_rows, page_size, out, ws=None, scale=None, stream=None):
    """out[B][Hq][d] (float32) = attention of q [B][Hq][d] over the paged partial set."""
    B, Hq, d = q.shape
    Hkv, max_pages = page_table.shape[1], page_table.shape[2]
    _need(k_pool.dtype == q.dtype and v_pool.dtype == q.dtype, "q and pools must share a dtype")
    _need(out.dtype == torch.float32 and out.numel() >= B * Hq * d, "out must be float32 [B][Hq][d]")
    if scale is None:
        scale = d ** -0.5
    pool_rows = k_pool.numel() // d
    _need(v_pool.numel() >= pool_rows * d, "v_pool smaller than k_pool")
    _need(page_table.shape[0] == B and n_rows.numel() >= B * Hkv, "page_table [B][Hkv][max_pages], n_rows [B][Hkv]")
    _need(Hq % Hkv == 0, "Hq must be a multiple of Hkv")
    rc = load().sg_decode_attn(_stream(stream), _dtype_code(q), B, Hq, Hkv, d, float(scale), _ptr(q), _ptr(k_pool),
                               _ptr(v_pool), pool_rows, _ptr(page_table), _ptr(n_rows), int(page_size),
                               int(max_pages), _ptr(out), _ptr(ws),
                               0 if ws is None else ws.numel() * ws.element_size())
    _check("sg_decode_attn", rc)
    return out


def decode_noalloc_scratch_bytes() -> int:
    return int(load().sg_decode_attn_noalloc_scratch_bytes())


def sg_decode_attn_noalloc(q, k_pool, v_pool, page_table, n_rows, page_size, out, scale=None, stream=None):
    """sg_decode_attn without a workspace: the split states live in the
    library's static per-GPU scratch array (calls on one GPU must not overlap)."""
    B, Hq, d = q.shape
    Hkv, max_pages = page_table.shape[1], page_table.shape[2]
    _need(k_pool.dtype == q.dtype and v_pool.dtype == q.dtype, "q and pools must share a dtype")
    _need(out.dtype == torch.float32 and out.numel() >= B * Hq * d, "out must be float32 [B][Hq][d]")
    if scale is None:
        scale = d ** -0.5
    pool_rows = k_pool.numel() // d
    _need(v_pool.numel() >= pool_rows * d, "v_pool smaller than k_pool")
    _need(page_table.shape[0] == B and n_rows.numel() >= B * Hkv, "page_table [B][Hkv][max_pages], n_rows [B][Hkv]")
    _need(Hq % Hkv == 0, "Hq must be a multiple of Hkv")
    rc = load().sg_decode_attn_noalloc(_stream(stream), _dtype_code(q), B, Hq, Hkv, d, float(scale), _ptr(q),
                                       _ptr(k_pool), _ptr(v_pool), pool_rows, _ptr(page_table), _ptr(n_rows),
                                       int(page_size), int(max_pages), _ptr(out))
    _check("sg_decode_attn_noalloc", rc)
    return out


class DecodeCall:
    """A prepared sg_decode_attn call for a fixed geometry: per call only the
    query, the pools and the output change.  Cuts host overhead in decode loops
    (the same marshalling as sg_decode_attn, done once)."""

    def __init__(self, q, k_pool, v_pool, page_table, n_rows, page_size, out, ws=None, scale=None, stream=None):
        sg_decode_attn(q, k_pool, v_pool, page_table, n_rows, page_size, out, ws=ws, scale=scale, stream=stream)
        B, Hq, d = q.shape
        self._lib = load()
        self._keep = (page_table, n_rows, ws)
        self._dt = _dtype_code(q)
        self._shape = (B, Hq, page_table.shape[1], d)
        self._scale = float(d ** -0.5 if scale is None else scale)
        self._pt, self._nr = _ptr(page_table), _ptr(n_rows)
        self._geom = (int(page_size), int(page_table.shape[2]))
        self._ws = _ptr(ws)
        self._wsb = 0 if ws is None else ws.numel() * ws.element_size()
        # a stream given here is kept; otherwise each call launches on torch's
        # current stream at the time of the call (graph capture, stream contexts)
        self._stream = None if stream is None else _stream(stream)
        self._pool_rows = k_pool.numel() // d
        self._numel = (q.numel(), k_pool.numel(), out.numel())

    def __call__(self, q, k_pool, v_pool, out):
        _need(q.numel() == self._numel[0] and k_pool.numel() == self._numel[1] and out.numel() == self._numel[2]
              and v_pool.numel() == self._numel[1], "prepared decode call used with other shapes")
        B, Hq, Hkv, d = self._shape
        st = self._stream if self._stream is not None else _stream(None)
        rc = self._lib.sg_decode_attn(st, self._dt, B, Hq, Hkv, d, self._scale, q.data_ptr(),
                                      k_pool.data_ptr(), v_pool.data_ptr(), self._pool_rows, self._pt, self._nr,
                                      self._geom[0], self._geom[1], out.data_ptr(), self._ws, self._wsb)
        _check("sg_decode_attn", rc)



# ----------------------------------------------------------------------------- block mode (Section 4.1)

def sg_block_importance(scores, cu_seqlens, T, M, imp, stream=None):
    """imp[B][L][M] (float32, written): eq. 1 block importance from scores [L][Hkv][T]."""
    L, Hkv = scores.shape[0], scores.shape[1]
    B = cu_seqlens.numel() - 1
    _need(scores.dtype == torch.float32 and scores.numel() >= L * Hkv * T, "scores must be float32 [L][Hkv][T]")
    _need(imp.dtype == torch.float32 and imp.numel() >= B * L * M, "imp must be float32 [B][L][M]")
    _need(cu_seqlens.dtype == torch.int32, "cu_seqlens must be int32 [B+1]")
    rc = load().sg_block_importance(_stream(stream), B, L, Hkv, _ptr(cu_seqlens), int(T), int(M), _ptr(scores),
                                    _ptr(imp))
    _check("sg_block_importance", rc)
    return imp


def block_budget(M, L, Tp, Tt) -> int:
    """Eq. 2 block budget K_r (host only)."""
    k = load().sg_block_budget(int(M), int(L), float(Tp), float(Tt))
    if k < 0:
        raise SmartgenError("sg_block_budget", SG_EINVAL, "need M, L >= 1 and non-negative times")
    return int(k)


def pack_blocks_bytes(dtype, Hkv, d, N, M, nblk) -> int:
    return int(load().sg_pack_blocks_bytes(SG_BF16 if dtype == torch.bfloat16 else SG_F32, Hkv, d, int(N), int(M),
                                           int(nblk)))


def sg_pack_blocks(k, v, ids, s0, N, M, dst, L=None, kv_layer_rows=None, stream=None):
    """Block transfer buffer of one request (tokens [s0, s0 + N) of k / v [Lkv][Hkv][T][d])."""
    _need(k.dtype == v.dtype and k.shape == v.shape, "k and v must match")
    _need(ids.dtype == torch.int32, "ids must be int32")
    Lkv, Hkv, T, d = k.shape
    if L is None:
        L = Lkv
    if kv_layer_rows is None:
        kv_layer_rows = 0 if (Lkv == 1 and L > 1) else Hkv * T
    rc = load().sg_pack_blocks(_stream(stream), _dtype_code(k), int(L), Hkv, d, int(T), int(s0), int(N), int(M),
                               _ptr(k), _ptr(v), int(kv_layer_rows), ids.numel(), _ptr(ids), _ptr(dst),
                               dst.numel() * dst.element_size())
    _check("sg_pack_blocks", rc)
    return dst


# ----------------------------------------------------------------------------- speculative transfer (Section 4.3)

def spec_quota(blocks, ratio_bp) -> int:
    """Blocks per speculative transfer (host only): ceil(blocks * ratio_bp / 10000)."""
    r = load().sg_spec_quota(int(blocks), int(ratio_bp))
    if r < 0:
        raise SmartgenError("sg_spec_quota", SG_EINVAL, "need blocks >= 0 and ratio_bp >= 1")
    return int(r)


def sg_spec_push(k_src, v_src, ids, s0, N, M, k_dst, v_dst, mask, rem=None, L=None, src_layer_rows=None,
                 dst_layer_rows=None, stream=None):
    """Delivers the blocks `ids` of one request from k_src / v_src [Lkv][Hkv][T][d]
    (device or pinned host) into the store k_dst / v_dst [L][Hkv][T][d] at the same
    rows, turns their mask [L][Hkv][T] entries local and their rem [L*M] entries NaN
    (mask=None: the rows only; sg_spec_commit marks them later)."""
    _need(k_src.dtype == v_src.dtype == k_dst.dtype == v_dst.dtype, "k/v source and store dtypes differ")
    _need(ids.dtype == torch.int32, "ids must be int32")
    Lkv, Hkv, T, d = k_src.shape
    Ld = k_dst.shape[0]
    if L is None:
        L = Ld
    _need(tuple(k_dst.shape[1:]) == (Hkv, T, d) and v_dst.shape == k_dst.shape, "store must be [L][Hkv][T][d]")
    _need(mask is None or (mask.dtype == torch.int8 and mask.numel() >= L * Hkv * T), "mask must be int8 [L][Hkv][T]")
    _need(rem is None or (rem.dtype == torch.float32), "rem must be float32 [L*M]")
    if src_layer_rows is None:
        src_layer_rows = 0 if (Lkv == 1 and L > 1) else Hkv * T
    if dst_layer_rows is None:
        dst_layer_rows = 0 if (Ld == 1 and L > 1) else Hkv * T
    rc = load().sg_spec_push(_stream(stream), _dtype_code(k_src), int(L), Hkv, d, int(T), int(s0), int(N), int(M),
                             _ptr(k_src), _ptr(v_src), int(src_layer_rows), _ptr(k_dst), _ptr(v_dst),
                             int(dst_layer_rows), ids.numel(), _ptr(ids), _ptr(mask), _ptr(rem))
    _check("sg_spec_push", rc)


def sg_spec_commit(ids, L, Hkv, T, s0, N, M, mask, rem=None, stream=None):
    """Marks the delivered blocks `ids` of one request: mask [L][Hkv][T] entries
    local, rem [L*M] entries NaN (the marking half of sg_spec_push)."""
    _need(ids.dtype == torch.int32 and mask.dtype == torch.int8, "ids must be int32 and mask int8")
    _need(mask.numel() >= L * Hkv * T, "mask must be int8 [L][Hkv][T]")
    _need(rem is None or (rem.dtype == torch.float32 and rem.numel() >= L * M), "rem must be float32 [L*M]")
    rc = load().sg_spec_commit(_stream(stream), int(L), int(Hkv), int(T), int(s0), int(N), int(M), ids.numel(),
                               _ptr(ids), _ptr(mask), _ptr(rem))
    _check("sg_spec_commit", rc)
