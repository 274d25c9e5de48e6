"""Helpers for the GPU parity tests: tensor movement and comparison rules."""
from __future__ import annotations

import sys

import numpy as np
import torch


def say(*a):
    """Name the case before each GPU step (flushed, so a fault still shows it)."""
    print("[gpu-case]", *a, file=sys.stderr, flush=True)


def cu(x, device="cuda", dtype=torch.int32):
    return torch.as_tensor(np.asarray(x), dtype=dtype).to(device)


def f32(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def raw(t: torch.Tensor) -> np.ndarray:
    """Host copy keeping the exact bits (bf16 as uint16)."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def assert_scores_close(gpu: np.ndarray, ref: np.ndarray, rtol=1e-3, floor=1e-30):
    """|g - o| <= rtol * |o| + floor, element by element (scores are sums of positive terms)."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    bad = ~(np.abs(gpu - ref) <= rtol * np.abs(ref) + floor)     # NaN counts as a mismatch
    if bad.any():
        i = np.argwhere(bad)[:5]
        raise AssertionError(f"{int(bad.sum())} scores out of tolerance; first {i.tolist()}: "
                             f"gpu {gpu[bad][:5]} oracle {ref[bad][:5]}")


def assert_topk_sets_agree(idx_gpu, idx_ref, ref_scores, k, rtol=1e-3):
    """Selections from GPU scores vs oracle scores may differ only on entries whose
    oracle score is within rtol of the oracle's k-th largest score."""
    a, b = set(np.asarray(idx_gpu).tolist()), set(np.asarray(idx_ref).tolist())
    if a == b:
        return
    kth = np.sort(ref_scores)[::-1][k - 1]
    for j in a ^ b:
        assert abs(ref_scores[j] - kth) <= rtol * abs(kth), f"token {j} differs but is not a near-tie"
