"""Workload records for the refine + verify path.

Each record fixes the shapes, dtypes and value distributions of one synthetic
workload.  The refiner shapes follow the paper's setting: a Qwen3-8B target
(hidden width 4096, vocabulary 151936) with a block-16 diffusion drafter and a
low-rank refiner of rank r = 256 (section 4.1, equations fuse..correct;
section 5.1).  The attention-layer fields (heads, KV heads, head_dim, FFN width,
context length) describe the surrounding decoder layers; the refiner itself does
not read them (Proposition 1: the context reaches the refiner only through the
drafter hidden states), so they are carried here for completeness only.

This module holds no arithmetic of the method.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class Workload:
    index: int                 # stable id, part of every random-stream key
    name: str
    dtype: str                 # "f32" or "bf16": storage type of weights and h
    H: int                     # drafter / target hidden width
    r: int                     # refiner rank (section 4.1 fixes r = 256)
    V: int                     # vocabulary size
    B: int                     # block length (refined positions; anchor extra)
    batch: int
    K: int                     # Jacobi passes (section 4.2; K about 6)
    temp: str                  # "greedy", "sample" or "mixed" (row b: b % 2)
    w_sigma: float = 0.02      # std of every weight entry
    h_sigma: float = 1.0       # std of drafter hidden states
    seed_mode: str = "base"    # "base": Y0 from the base logits; "given": supplied ids
    p_match: Optional[float] = None          # T=0 rows: P(target == draft)
    p_match_range: Optional[Tuple[float, float]] = None   # per-sequence U(lo, hi)
    target_logit_sigma: float = 2.0          # T=1 rows: target logits iid N(0, s^2)
    # decoder-layer fields, recorded but not consumed by the refiner
    n_heads: int = 32
    n_kv_heads: int = 8
    head_dim: int = 128
    ffn: int = 12288
    ctx_len: Optional[int] = None
    ctx_len_range: Optional[Tuple[int, int]] = None

    @property
    def M(self) -> int:
        return self.batch * self.B

    def row_is_sample(self, b: int) -> bool:
        if self.temp == "greedy":
            return False
        if self.temp == "sample":
            return True
        return b % 2 == 1


TINY_F32 = Workload(
    index=0, name="tiny-f32-H256-V1024-B8-b1", dtype="f32", H=256, r=256, V=1024,
    B=8, batch=1, K=8, temp="greedy", seed_mode="given", p_match=0.7,
    n_heads=4, n_kv_heads=4, head_dim=64, ffn=1024, ctx_len=64)

QWEN_B1 = Workload(
    index=1, name="qwen3-8b-bf16-B16-b1-greedy", dtype="bf16", H=4096, r=256,
    V=151936, B=16, batch=1, K=6, temp="greedy", p_match=0.8, ctx_len=2048)

QWEN_B8_T1 = Workload(
    index=2, name="qwen3-8b-bf16-B16-b8-sample", dtype="bf16", H=4096, r=256,
    V=151936, B=16, batch=8, K=6, temp="sample", h_sigma=1.5625, ctx_len=4096)

QWEN_B32 = Workload(
    index=3, name="qwen3-8b-bf16-B16-b32-greedy", dtype="bf16", H=4096, r=256,
    V=151936, B=16, batch=32, K=6, temp="greedy", p_match=0.8, ctx_len=8192)

QWEN_B64_MIXED = Workload(
    index=4, name="qwen3-8b-bf16-B32-b64-mixed", dtype="bf16", H=4096, r=256,
    V=151936, B=32, batch=64, K=6, temp="mixed", p_match_range=(0.5, 0.95),
    ctx_len_range=(512, 16384))

WORKLOADS = (TINY_F32, QWEN_B1, QWEN_B8_T1, QWEN_B32, QWEN_B64_MIXED)
BY_NAME = {w.name: w for w in WORKLOADS}


def scaled(w: Workload, **changes) -> Workload:
    """A copy of ``w`` with some fields replaced (e.g. a smaller V or batch).

    The copy keeps ``w.index`` unless ``index`` is given, so that streams of a
    reduced workload are still keyed by the record they came from; pass a fresh
    index when the reduced case must not share draws with the full one.
    """
    from dataclasses import replace
    return replace(w, **changes)
