"""The five synthetic verify-step workloads.

Shapes follow the Llama-2 family with Medusa heads (SpecMemo, Sec. 3.1 memory
model symbols: b batch, k KV heads, d head dim, l heads = tree levels, w vocab,
N tree nodes).  Every field is a plain number so that the workload can be
rebuilt bit-for-bit from (name, seed).
"""

from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class Config:
    name: str
    dtype: str                  # "fp32" or "bf16": storage and operand type
    B: int                      # sequences in the batch
    n_q: int                    # query heads
    n_kv: int                   # KV heads (GQA when n_kv < n_q)
    head_dim: int
    hidden: int
    vocab: int
    n_heads: int                # Medusa heads == tree levels (l)
    topk: Tuple[int, ...]       # top-k per head (tree arity per level)
    tree: str                   # "T16", "T64" or "random"
    tree_sizes: Tuple[int, ...] = ()    # random trees: sizes drawn uniformly from this set
    kv_len: Tuple[int, int] = (0, 0)    # committed length range, inclusive
    kv_len_dist: str = "fixed"          # "fixed", "uniform" or "loguniform"
    pool: str = "exact"                 # "exact", "cap1.1" or "fixed1.1"
    p_accept: Optional[float] = 0.6     # None: per-sequence p ~ U[p_range]
    p_range: Tuple[float, float] = (0.6, 0.6)
    w_std: float = 0.02                 # head-weight std
    seed: int = 0
    layers: int = 1                     # decoder layers of the model the shapes come from
    params: int = 0                     # its parameter count (memory model only; 0: not a real model)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "fp32" else 2

    @property
    def kmax(self) -> int:
        return max(self.topk)

    @property
    def group(self) -> int:
        return self.n_q // self.n_kv


TINY_FP32 = Config(
    name="tiny_fp32", dtype="fp32", B=1, n_q=4, n_kv=4, head_dim=64, hidden=256,
    vocab=1000, n_heads=3, topk=(4, 2, 2), tree="T16", kv_len=(128, 128),
    kv_len_dist="fixed", pool="exact", p_accept=0.6, w_std=1.0, seed=0)

LLAMA2_7B = Config(
    name="llama2_7b_b1", dtype="bf16", B=1, n_q=32, n_kv=32, head_dim=128, hidden=4096,
    vocab=32000, n_heads=4, topk=(10, 10, 10, 10), tree="T64", kv_len=(1024, 1024),
    kv_len_dist="fixed", pool="exact", p_accept=0.6, seed=1, layers=32, params=6_738_415_616)

LLAMA2_13B = Config(
    name="llama2_13b_b4", dtype="bf16", B=4, n_q=40, n_kv=40, head_dim=128, hidden=5120,
    vocab=32000, n_heads=4, topk=(10, 10, 10, 10), tree="T64", kv_len=(512, 2048),
    kv_len_dist="uniform", pool="exact", p_accept=0.6, seed=2, layers=40, params=13_015_864_320)

LLAMA2_70B = Config(
    name="llama2_70b_b10", dtype="bf16", B=10, n_q=64, n_kv=8, head_dim=128, hidden=8192,
    vocab=32000, n_heads=4, topk=(10, 10, 10, 10), tree="T64", kv_len=(512, 4096),
    kv_len_dist="uniform", pool="cap1.1", p_accept=0.6, seed=3, layers=80, params=68_976_648_192)

STRESS = Config(
    name="stress_b32", dtype="bf16", B=32, n_q=64, n_kv=8, head_dim=128, hidden=8192,
    vocab=32000, n_heads=4, topk=(10, 10, 10, 10), tree="random",
    tree_sizes=(8, 16, 32, 64, 128), kv_len=(256, 16384), kv_len_dist="loguniform",
    pool="fixed1.1", p_accept=None, p_range=(0.3, 0.8), seed=4, layers=80,
    params=68_976_648_192)

ALL = (TINY_FP32, LLAMA2_7B, LLAMA2_13B, LLAMA2_70B, STRESS)
BY_NAME = {c.name: c for c in ALL}


def get(name: str) -> Config:
    return BY_NAME[name]
