"""Seeded synthetic inputs for the refine + verify path.

Every tensor is drawn from its own counter-keyed stream,
``PCG64(SeedSequence(0, spawn_key=(workload.index, stream_id[, block])))``, so a
tensor never depends on which other tensors were generated or in which order.
Large tensors are cut into fixed row blocks, each with its own stream, and the
blocks are drawn on a thread pool; the values do not depend on the number of
threads.

bf16 tensors are drawn by inverse-transform sampling: a uniform 16-bit word
``i`` indexes the table ``bf16(sigma * Phi^-1((i + 0.5) / 65536))``.  That is an
exact sample of a normal law quantised to 65536 equiprobable levels (tails cut
at about 4.3 sigma), stored directly as bf16 bit patterns, and it is two orders
of magnitude faster than drawing normals and rounding them on the host.

The module only produces inputs: it contains none of the method's arithmetic.
Random numbers the method consumes (``u_draft``, ``r_accept``, ``u_res``) are
drawn here and handed to both sides as inputs.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from functools import lru_cache
from typing import Dict, Optional

import numpy as np

from .configs import Workload

MASTER_SEED = 0
STREAMS = {
    "W_lm": 1, "W_h": 2, "W_g": 3, "W_e": 4, "W_in": 5, "L": 6, "W_1": 7,
    "W_2": 8, "W_r": 9, "h": 10, "anchor": 11, "seed_ids": 12, "u_draft": 13,
    "r_accept": 14, "u_res": 15, "coins": 16, "alts": 17, "target_logits": 18,
    "p_match": 19, "ctx_len": 20,
    # the context layer
    "layer.g_attn": 21, "layer.Wq": 22, "layer.Wk": 23, "layer.Wv": 24, "layer.g_q": 25,
    "layer.g_k": 26, "layer.Wo": 27, "layer.g_mlp": 28, "layer.Wg": 29, "layer.Wu": 30,
    "layer.Wd": 31, "layer.x": 32, "layer.k": 33, "layer.v": 34, "layer.ctx": 35,
}
_BLOCK = 1 << 22          # elements per independently keyed block
_THREADS = max(1, min(16, os.cpu_count() or 1))


def _rng(w: Workload, stream: str, *extra: int) -> np.random.Generator:
    key = (w.index, STREAMS[stream]) + tuple(extra)
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(MASTER_SEED, spawn_key=key)))


# --- bf16 storage helpers (bit-level; used only to build and view inputs) ----

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round to nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@lru_cache(maxsize=16)
def _quantile_table(sigma: float) -> np.ndarray:
    from scipy.special import ndtri
    q = sigma * ndtri((np.arange(65536, dtype=np.float64) + 0.5) / 65536.0)
    return f32_to_bf16_bits(q.astype(np.float32))


def _blocks(n: int):
    return [(i, min(n, i + _BLOCK)) for i in range(0, n, _BLOCK)]


def normal_bf16(w: Workload, stream: str, shape, sigma: float) -> np.ndarray:
    """bf16 bit patterns of N(0, sigma^2) (quantised inverse-transform sample)."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    tab = _quantile_table(float(sigma))

    def work(args):
        bi, (lo, hi) = args
        g = _rng(w, stream, bi)
        idx = g.integers(0, 65536, hi - lo, dtype=np.uint16)
        np.take(tab, idx, out=out[lo:hi])

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(work, enumerate(_blocks(n))))
    return out.reshape(shape)


def normal_f32(w: Workload, stream: str, shape, sigma: float) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)

    def work(args):
        bi, (lo, hi) = args
        g = _rng(w, stream, bi)
        out[lo:hi] = g.standard_normal(hi - lo, dtype=np.float32) * np.float32(sigma)

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(work, enumerate(_blocks(n))))
    return out.reshape(shape)


def _tensor(w: Workload, stream: str, shape, sigma: float) -> np.ndarray:
    if w.dtype == "bf16":
        return normal_bf16(w, stream, shape, sigma)
    return normal_f32(w, stream, shape, sigma)


def as_f32(w: Workload, x: np.ndarray) -> np.ndarray:
    """View a stored tensor (bf16 bits or float32) as float32 values."""
    return bf16_bits_to_f32(x) if x.dtype == np.uint16 else x


# --- problem instances -------------------------------------------------------

WEIGHT_SHAPES = {
    # layout: row-major, one row per output unit; W_e and W_r keep one row per
    # vocabulary token (the paper writes W_e as r x V, here it is stored as its
    # transpose so that a token's embedding is one contiguous row).
    "W_lm": lambda w: (w.V, w.H),
    "W_h": lambda w: (w.r, w.H),
    "W_g": lambda w: (w.r, w.H),
    "W_e": lambda w: (w.V, w.r),
    "W_in": lambda w: (w.r, 3 * w.r),
    "L": lambda w: (w.r, w.B, w.B),
    "W_1": lambda w: (2 * w.r, w.r),
    "W_2": lambda w: (w.r, 2 * w.r),
    "W_r": lambda w: (w.V, w.r),
}


def make_weights(w: Workload, names=None, upper_fill: Optional[float] = 0.0) -> Dict[str, np.ndarray]:
    """All refiner weights plus the target LM head.

    ``L`` is drawn in full and then only its strictly lower triangle (entry
    [d][k][i] with i < k) is kept; the rest is set to ``upper_fill`` (0 by
    default).  Both implementations must ignore that part, so tests may fill it
    with a large value to prove it is never read.
    """
    names = names or list(WEIGHT_SHAPES)
    out = {}
    for n in names:
        out[n] = _tensor(w, n, WEIGHT_SHAPES[n](w), w.w_sigma)
    if "L" in out and upper_fill is not None:
        keep = np.tril(np.ones((w.B, w.B), dtype=bool), k=-1)
        L = out["L"]
        if L.dtype == np.uint16:
            fill = f32_to_bf16_bits(np.array([upper_fill], dtype=np.float32))[0]
        else:
            fill = np.float32(upper_fill)
        L[:, ~keep] = fill
    return out


@dataclass
class Inputs:
    h: np.ndarray                      # [batch][B][H] bf16 bits or float32
    anchor: np.ndarray                 # [batch] int32, x_0
    seed_ids: Optional[np.ndarray]     # [batch][B] int32, or None
    temp: np.ndarray                   # [batch] uint8: 0 greedy, 1 sample
    u_draft: np.ndarray                # [batch][B] float32 in [0, 1)
    r_accept: np.ndarray               # [batch][B] float32 in [0, 1)
    u_res: np.ndarray                  # [batch] float32 in [0, 1)
    coins: np.ndarray                  # [batch][B] bool: target copies the draft
    alts: np.ndarray                   # [batch][B+1] int32: otherwise this token
    p_match: np.ndarray                # [batch] float32
    target_logits: Optional[np.ndarray]  # [batch][B+1][V] float32 (sample rows), or None
    ctx_len: np.ndarray                # [batch] int32 (recorded only)

    def target_ids(self, draft: np.ndarray) -> np.ndarray:
        """Greedy-row targets built around a given draft block.

        Position k copies the draft token with probability ``p_match`` and is
        an independent uniform token otherwise; position B+1 is always the
        independent token.  Coins and alternatives are drawn up front, so the
        targets are a fixed function of the draft they are built around.
        """
        draft = np.asarray(draft, dtype=np.int32)
        bsz, B = draft.shape
        t = self.alts.copy()
        t[:, :B] = np.where(self.coins, draft, self.alts[:, :B])
        return t.astype(np.int32)


def make_inputs(w: Workload, batch: Optional[int] = None) -> Inputs:
    bsz = w.batch if batch is None else batch
    B, V = w.B, w.V
    h = _tensor(w, "h", (bsz, B, w.H), w.h_sigma)
    anchor = _rng(w, "anchor").integers(0, V, bsz, dtype=np.int64).astype(np.int32)
    seed_ids = None
    if w.seed_mode == "given":
        seed_ids = _rng(w, "seed_ids").integers(0, V, (bsz, B), dtype=np.int64).astype(np.int32)
    temp = np.array([1 if w.row_is_sample(b) else 0 for b in range(bsz)], dtype=np.uint8)
    u_draft = _rng(w, "u_draft").random((bsz, B), dtype=np.float32)
    r_accept = _rng(w, "r_accept").random((bsz, B), dtype=np.float32)
    u_res = _rng(w, "u_res").random(bsz, dtype=np.float32)
    if w.p_match_range is not None:
        lo, hi = w.p_match_range
        p = _rng(w, "p_match").uniform(lo, hi, bsz).astype(np.float32)
    else:
        p = np.full(bsz, w.p_match if w.p_match is not None else 0.0, dtype=np.float32)
    coins = _rng(w, "coins").random((bsz, B)) < p[:, None]
    alts = _rng(w, "alts").integers(0, V, (bsz, B + 1), dtype=np.int64).astype(np.int32)
    target_logits = None
    if temp.any():
        target_logits = np.zeros((bsz, B + 1, V), dtype=np.float32)
        for b in np.nonzero(temp)[0]:
            target_logits[b] = normal_f32_row(w, b, (B + 1, V), w.target_logit_sigma)
    if w.ctx_len_range is not None:
        lo, hi = w.ctx_len_range
        ctx = _rng(w, "ctx_len").integers(lo, hi + 1, bsz, dtype=np.int64).astype(np.int32)
    else:
        ctx = np.full(bsz, w.ctx_len or 0, dtype=np.int32)
    return Inputs(h=h, anchor=anchor, seed_ids=seed_ids, temp=temp, u_draft=u_draft,
                  r_accept=r_accept, u_res=u_res, coins=coins, alts=alts, p_match=p,
                  target_logits=target_logits, ctx_len=ctx)


def normal_f32_row(w: Workload, b: int, shape, sigma: float) -> np.ndarray:
    """float32 N(0, sigma^2) for sequence ``b``'s target logits (own stream per row)."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)

    def work(args):
        bi, (lo, hi) = args
        g = _rng(w, "target_logits", b, bi)
        out[lo:hi] = g.standard_normal(hi - lo, dtype=np.float32) * np.float32(sigma)

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(work, enumerate(_blocks(n))))
    return out.reshape(shape)


# --- the context layer (the configuration's decoder-layer fields) --------------

LAYER_SHAPES = {
    "g_attn": lambda w: (w.H,),
    "Wq": lambda w: (w.n_heads * w.head_dim, w.H),
    "Wk": lambda w: (w.n_kv_heads * w.head_dim, w.H),
    "Wv": lambda w: (w.n_kv_heads * w.head_dim, w.H),
    "g_q": lambda w: (w.head_dim,),
    "g_k": lambda w: (w.head_dim,),
    "Wo": lambda w: (w.H, w.n_heads * w.head_dim),
    "g_mlp": lambda w: (w.H,),
    "Wg": lambda w: (w.ffn, w.H),
    "Wu": lambda w: (w.ffn, w.H),
    "Wd": lambda w: (w.H, w.ffn),
}


def make_layer_weights(w: Workload) -> Dict[str, np.ndarray]:
    """bf16 bit patterns: projections N(0, w_sigma^2); norm weights 1 + N(0, 0.1^2)."""
    out = {}
    for n, shape_fn in LAYER_SHAPES.items():
        if n.startswith("g_"):
            f = 1.0 + normal_f32(w, "layer." + n, shape_fn(w), 0.1)
            out[n] = f32_to_bf16_bits(f)
        else:
            out[n] = normal_bf16(w, "layer." + n, shape_fn(w), w.w_sigma)
    return out


@dataclass
class LayerInputs:
    x: np.ndarray          # [batch][B][H] bf16 bits: block hidden states, N(0, h_sigma^2)
    k_cache: np.ndarray    # [batch][C_max][n_kv][hd] bf16 bits, N(0, 1) (post-norm keys)
    v_cache: np.ndarray    # [batch][C_max][n_kv][hd] bf16 bits, N(0, 1)
    ctx_len: np.ndarray    # [batch] int32: ctx_len, or U{lo..hi} per sequence


def make_layer_inputs(w: Workload, batch: Optional[int] = None,
                      c_max: Optional[int] = None) -> LayerInputs:
    batch = w.batch if batch is None else batch
    if w.ctx_len_range is not None:
        lo, hi = w.ctx_len_range
        ctx = _rng(w, "layer.ctx").integers(lo, hi + 1, batch).astype(np.int32)
    else:
        ctx = np.full(batch, w.ctx_len or 0, dtype=np.int32)
    cm = int(ctx.max()) if c_max is None else c_max
    cm = max(cm, 1)
    kv = (batch, cm, w.n_kv_heads, w.head_dim)
    return LayerInputs(x=normal_bf16(w, "layer.x", (batch, w.B, w.H), w.h_sigma),
                       k_cache=normal_bf16(w, "layer.k", kv, 1.0),
                       v_cache=normal_bf16(w, "layer.v", kv, 1.0), ctx_len=ctx)
