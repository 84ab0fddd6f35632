"""fp64 CPU oracle of the context layer: one Qwen3-8B-shaped decoder layer over
the positions of a drafted block, attending to the sequence's context KV.

TEST INFRASTRUCTURE.  Only the test suite and the CPU-baseline leg of the
benchmark import this module; the device path never imports, calls or links
it, and it shares no code with the device path.

The paper's refiner does not read the context (Proposition 1: the context
reaches it only through the drafter's hidden states h); in the paper's
pipeline such layers are the drafter's and the target's (sections 3.1 and
5.1).  This layer produces the h that the base readout s_k = W_lm h_k
(section 4.1) consumes.  Its structure is the configuration's Qwen3-8B layer
(heads, KV heads, head_dim, FFN width, context length); the paper gives no
formula for it, so each step below is the standard definition, stated here:

* RMSNorm      y = x / sqrt(mean(x^2) + eps) * g                    (eps 1e-6)
* projections  q = u Wq^T, k = u Wk^T, v = u Wv^T                    (no biases)
* QK-norm      RMSNorm over head_dim of every q and k head, weights g_q, g_k
* RoPE         rotate-half pairs (j, j + hd/2), angle pos * theta^(-2j/hd),
               theta = 1e6, applied after the QK-norm; position of block
               position i of sequence b is ctx_len[b] + i
* attention    GQA: query head h reads KV head h // (n_heads / n_kv); scores
               q.k / sqrt(hd); the keys are the context cache (post-norm,
               post-RoPE, as a cache holds them) and the block's own keys,
               block key j visible to block query i iff j <= i (causal) or
               always (bidirectional); softmax over the visible keys
* output       x1 = x + attn Wo^T
* FFN          h = x1 + (silu(u2 Wg^T) * (u2 Wu^T)) Wd^T,  u2 = RMSNorm(x1) g_mlp

Rounding points (the device stores these tensors in bf16 between kernels and
feeds them to bf16 matrix products): u, the normed and rotated q and k, v,
the normalised attention output, u2 and the SwiGLU activation are rounded to
bf16 here too.  Everything else is fp64; the device's fp32 accumulation and
its softmax numerators, which enter the P.V product as two bf16 parts (about
16 significant bits), are covered by the parity tolerance.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .xpress_ref import round_bf16, silu, to_f64

F64 = np.float64


@dataclass
class LayerParams:
    n_heads: int
    n_kv: int
    head_dim: int
    eps: float
    theta: float
    g_attn: np.ndarray   # [H]
    Wq: np.ndarray       # [n_heads*hd][H]
    Wk: np.ndarray       # [n_kv*hd][H]
    Wv: np.ndarray       # [n_kv*hd][H]
    g_q: np.ndarray      # [hd]
    g_k: np.ndarray      # [hd]
    Wo: np.ndarray       # [H][n_heads*hd]
    g_mlp: np.ndarray    # [H]
    Wg: np.ndarray       # [ffn][H]
    Wu: np.ndarray       # [ffn][H]
    Wd: np.ndarray       # [H][ffn]

    NAMES = ("g_attn", "Wq", "Wk", "Wv", "g_q", "g_k", "Wo", "g_mlp", "Wg", "Wu", "Wd")

    @staticmethod
    def from_arrays(w: dict, n_heads, n_kv, head_dim, eps=1e-6, theta=1e6) -> "LayerParams":
        """Stored weights (bf16 bit patterns as uint16, or float) widened to fp64."""
        return LayerParams(n_heads, n_kv, head_dim, eps, theta,
                           **{n: to_f64(w[n]) for n in LayerParams.NAMES})


def rmsnorm(x, g, eps):
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = np.asarray(x, dtype=F64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def rope(x, pos, theta):
    """Rotate-half RoPE of x [n][hd] or [n][heads][hd] at integer positions
    pos [n]: the pair (j, j + hd/2) turns by pos * theta^(-2j/hd)."""
    x = np.asarray(x, dtype=F64)
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=F64) / hd)
    ang = np.asarray(pos, dtype=F64)[:, None] * inv[None, :]          # [n][half]
    if x.ndim == 3:
        ang = ang[:, None, :]                                            # every head alike
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def attention(q, k_ctx, v_ctx, k_blk, v_blk, n_kv, causal=True):
    """Block attention of one sequence.

    q [B][n_heads][hd]; k_ctx, v_ctx [C][n_kv][hd] (the context cache);
    k_blk, v_blk [B][n_kv][hd] (the block's own keys and values).  Query i of
    head h sees every context key and block keys j <= i (causal) or all block
    keys; scores are q.k / sqrt(hd).  Returns [B][n_heads][hd].
    """
    B, nh, hd = q.shape
    C = k_ctx.shape[0]
    grp = nh // n_kv
    out = np.zeros((B, nh, hd), dtype=F64)
    for h in range(nh):
        kv = h // grp
        K = np.concatenate([k_ctx[:, kv, :], k_blk[:, kv, :]], axis=0)   # [C + B][hd]
        Vv = np.concatenate([v_ctx[:, kv, :], v_blk[:, kv, :]], axis=0)
        for i in range(B):
            n = C + (i + 1 if causal else B)
            sc = K[:n] @ q[i, h] / np.sqrt(hd)
            w = np.exp(sc - sc.max())
            out[i, h] = (w / w.sum()) @ Vv[:n]
    return out


def layer_forward(P: LayerParams, x, k_cache, v_cache, ctx_len, causal=True):
    """The context layer over a batch of blocks.

    x [batch][B][H] (block hidden states); k_cache, v_cache
    [batch][C_max][n_kv][hd] (entries past ctx_len[b] are never read);
    ctx_len [batch].  Returns h [batch][B][H] in fp64 (before any output
    rounding).
    """
    x = to_f64(x)
    batch, B, H = x.shape
    nh, nkv, hd = P.n_heads, P.n_kv, P.head_dim
    kc, vc = to_f64(k_cache), to_f64(v_cache)
    h = np.zeros_like(x)
    for b in range(batch):
        C = int(ctx_len[b])
        u = round_bf16(rmsnorm(x[b], P.g_attn, P.eps))
        q = (u @ P.Wq.T).reshape(B, nh, hd)
        k = (u @ P.Wk.T).reshape(B, nkv, hd)
        v = round_bf16((u @ P.Wv.T).reshape(B, nkv, hd))
        pos = C + np.arange(B)
        q = round_bf16(rope(rmsnorm(q, P.g_q, P.eps), pos, P.theta))
        k = round_bf16(rope(rmsnorm(k, P.g_k, P.eps), pos, P.theta))
        a = round_bf16(attention(q, kc[b, :C], vc[b, :C], k, v, nkv, causal).reshape(B, nh * hd))
        x1 = x[b] + a @ P.Wo.T
        u2 = round_bf16(rmsnorm(x1, P.g_mlp, P.eps))
        act = round_bf16(silu(u2 @ P.Wg.T) * (u2 @ P.Wu.T))
        h[b] = x1 + act @ P.Wd.T
    return h
