"""The five synthetic workloads, shaped like the paper's evaluation.

The paper measures on LongBench prompts (average 3K-10K tokens, batches up to
60K tokens) with Llama-3.1-8B, Qwen3-14B, Gemma-3-12B and Phi-4 (Section 5.1).
None of those datasets or weights is used here; these seeded configurations
stand in for them with the models' attention shapes and the prompt-length range.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace


@dataclass(frozen=True)
class Config:
    name: str
    L: int                 # attention layers
    Hq: int                # query heads
    Hkv: int               # KV heads (GQA groups of Hq // Hkv consecutive q heads)
    d: int                 # head dimension
    dtype: str             # "f32" or "bf16": storage type of q, K and V
    W: int                 # score window: the last W prompt positions
    budget_bp: int         # selection budget in basis points of the prompt (1000 = 10%)
    extra_bp: int          # on-demand extras per decode step, basis points (0 = none)
    steps: int             # decode steps
    seqlens: tuple = ()    # fixed per-request prompt lengths; empty = drawn (varlen)
    B: int = 1             # requests
    heavy_fixed: int = 0   # planted heavy hitters per unit when fixed (tiny config)
    heavy_bp: int = 0      # planted heavy hitters in basis points of the prompt
    sinks: int = 0         # leading tokens boosted like heavy hitters
    page_size: int = 16    # decode-side page size in rows
    kv_shared_layers: bool = False  # one K/V source shared by every layer
    stage_host: bool = False        # transfer buffer staged in pinned host memory
    seed: int = 1
    varlen_lo: int = 2048
    varlen_hi: int = 32768
    notes: str = ""

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def esize(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def with_(self, **kw) -> "Config":
        return replace(self, **kw)


CONFIGS = {
    "tiny": Config(
        name="tiny", L=1, Hq=8, Hkv=8, d=64, dtype="f32", W=32, budget_bp=1000,
        extra_bp=0, steps=1, seqlens=(2048,), heavy_fixed=32, sinks=0, seed=1,
        notes="1 layer, 8q=8kv heads, d=64, fp32, 2048-token prompt, 32 planted heavy hitters"),
    "llama8b_8k": Config(
        name="llama8b_8k", L=32, Hq=32, Hkv=8, d=128, dtype="bf16", W=64, budget_bp=1000,
        extra_bp=0, steps=128, seqlens=(8192,), heavy_bp=100, sinks=4, seed=2,
        notes="Llama-3-8B-shaped, 8K prompt, 10% budget, 128 decode steps"),
    "llama8b_32k": Config(
        name="llama8b_32k", L=32, Hq=32, Hkv=8, d=128, dtype="bf16", W=64, budget_bp=500,
        extra_bp=200, steps=256, seqlens=(32768,), heavy_bp=100, sinks=4, seed=3,
        notes="8B-shaped long context, 32K prompt, 5% budget, 2% on-demand per step"),
    "llama70b_16k": Config(
        name="llama70b_16k", L=80, Hq=64, Hkv=8, d=128, dtype="bf16", W=64, budget_bp=1000,
        extra_bp=0, steps=128, seqlens=(16384,), heavy_bp=100, sinks=4, stage_host=True, seed=4,
        notes="70B-shaped single-GPU slice, 16K prompt, pinned-host staging"),
    "batched64": Config(
        name="batched64", L=32, Hq=32, Hkv=8, d=128, dtype="bf16", W=64, budget_bp=1000,
        extra_bp=200, steps=512, seqlens=(), B=64, heavy_bp=100, sinks=4, page_size=16,
        kv_shared_layers=True, seed=5,
        notes="64 requests, prompts uniform in [2048, 32768], 16-token pages"),
}

# the order in which the workloads are listed (tiny first, the bench workload second)
ORDER = ["tiny", "llama8b_8k", "llama8b_32k", "llama70b_16k", "batched64"]


def get(name: str) -> Config:
    return CONFIGS[name]


def budget_k(n: int, budget_bp: int) -> int:
    """Selected rows for a prompt of ``n`` tokens: floor(n * bp / 10000), at least 1."""
    return max(1, min(n, (n * budget_bp) // 10000))


def extras_count(n: int, extra_bp: int) -> int:
    return (n * extra_bp) // 10000


def heavy_count(cfg: Config, n: int) -> int:
    if cfg.heavy_fixed:
        return cfg.heavy_fixed
    return (n * cfg.heavy_bp) // 10000
