"""How far an fp32 evaluation of the context layer's own steps lies from the
fp64 oracle: the floor below which no fp32 implementation with the same bf16
rounding points can be held, and from which the layer parity bar is set.

Run by hand (CPU, about a minute):  python tests/layer_fp32_floor.py

It evaluates oracle/layer_ref.py's steps once in fp64 (and checks that this
re-evaluation equals layer_forward exactly) and once with every array and
product in fp32 (numpy's own summation order), rounding to bf16 at the same
points, on the Qwen3-8B layer at the batch-64 shape (32 positions per block,
contexts drawn from 512..16384 keys), the sequences the GPU test checks.
Measured: max |h_fp32 - h_fp64| = 0.0196 at max |h| = 12.29 (1.6e-3 of it),
mean 1.2e-3.
"""
import os
import sys

import numpy as np

sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), ".."))

import oracle as O                      # noqa: E402
import oracle.layer_ref as LR           # noqa: E402
import synth                            # noqa: E402
from synth.configs import QWEN_B1       # noqa: E402


def forward(P, x, kc_all, vc_all, ctx_len, dt, seqs, causal=True):
    """layer_forward's steps with arrays of type dt (bf16 rounding points
    unchanged; RoPE angles in fp64, rounded to dt)."""
    rb, f64 = O.xpress_ref.round_bf16, O.xpress_ref.to_f64
    c = lambda a: np.asarray(a, dtype=dt)
    W = {n: c(getattr(P, n)) for n in P.NAMES}
    nh, nkv, hd = P.n_heads, P.n_kv, P.head_dim
    out = []
    for b in seqs:
        xb = c(f64(x[b]))
        B, C = xb.shape[0], int(ctx_len[b])

        def rms(v, g):
            v = c(v)
            return c(v / np.sqrt(np.mean(v * v, axis=-1, keepdims=True) + dt(P.eps)) * g)

        def rope(v, pos):
            half = hd // 2
            ang = np.asarray(pos, dtype=np.float64)[:, None] * P.theta ** (-2.0 * np.arange(half) / hd)
            cs, sn = c(np.cos(ang))[:, None, :], c(np.sin(ang))[:, None, :]
            a_, b_ = v[..., :half], v[..., half:]
            return np.concatenate([a_ * cs - b_ * sn, b_ * cs + a_ * sn], axis=-1)

        u = c(rb(rms(xb, W["g_attn"])))
        q = (u @ W["Wq"].T).reshape(B, nh, hd)
        k = (u @ W["Wk"].T).reshape(B, nkv, hd)
        v = c(rb((u @ W["Wv"].T).reshape(B, nkv, hd)))
        pos = C + np.arange(B)
        q = c(rb(rope(rms(q, W["g_q"]), pos)))
        k = c(rb(rope(rms(k, W["g_k"]), pos)))
        kc, vc = c(f64(kc_all[b, :C])), c(f64(vc_all[b, :C]))
        att = np.zeros((B, nh, hd), dtype=dt)
        for h in range(nh):
            kv = h // (nh // nkv)
            K = np.concatenate([kc[:, kv], k[:, kv]], 0)
            V = np.concatenate([vc[:, kv], v[:, kv]], 0)
            for i in range(B):
                n = C + (i + 1 if causal else B)
                sc = K[:n] @ q[i, h] / dt(np.sqrt(hd))
                w = np.exp(sc - sc.max())
                att[i, h] = (w / w.sum()) @ V[:n]
        a = c(rb(att.reshape(B, nh * hd)))
        x1 = xb + a @ W["Wo"].T
        u2 = c(rb(rms(x1, W["g_mlp"])))
        act = c(rb(O.xpress_ref.silu(u2 @ W["Wg"].T) * (u2 @ W["Wu"].T)))
        out.append(x1 + act @ W["Wd"].T)
    return np.stack(out)


def main():
    w = synth.scaled(QWEN_B1, index=905 + 64, B=32, batch=64, ctx_len=None,
                     ctx_len_range=(512, 16384))
    weights = synth.make_layer_weights(w)
    inp = synth.make_layer_inputs(w)
    order = np.argsort(inp.ctx_len)
    seqs = sorted({int(order[0]), int(order[-1]), 5, 40})
    P = LR.LayerParams.from_arrays(weights, w.n_heads, w.n_kv_heads, w.head_dim)
    ref = LR.layer_forward(P, inp.x[seqs], inp.k_cache[seqs], inp.v_cache[seqs],
                           inp.ctx_len[seqs])
    h64 = forward(P, inp.x, inp.k_cache, inp.v_cache, inp.ctx_len, np.float64, seqs)
    assert np.array_equal(h64, ref), "the re-evaluation must equal layer_forward"
    h32 = forward(P, inp.x, inp.k_cache, inp.v_cache, inp.ctx_len, np.float32, seqs)
    d = np.abs(h32.astype(np.float64) - ref)
    print(f"sequences {seqs} ctx {inp.ctx_len[seqs].tolist()}: max|h| {np.abs(ref).max():.4g} "
          f"fp32 vs fp64 max {d.max():.4g} mean {d.mean():.3g} "
          f"(max / max|h| = {d.max() / np.abs(ref).max():.3g})")


if __name__ == "__main__":
    main()
