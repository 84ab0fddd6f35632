"""Pins of the context-layer oracle (oracle/layer_ref.py) against closed forms,
invariances and special cases, so that a dropped term, a wrong sign, a wrong
head mapping or a wrong mask in it fails here.  CPU only."""
import numpy as np
import pytest

import oracle as O

L = O.layer_ref


def _params(H=64, nh=4, nkv=2, hd=8, ffn=96, seed=0, scale=0.3):
    g = np.random.default_rng(seed)
    w = dict(g_attn=1.0 + 0.1 * g.normal(size=H), Wq=scale * g.normal(size=(nh * hd, H)),
             Wk=scale * g.normal(size=(nkv * hd, H)), Wv=scale * g.normal(size=(nkv * hd, H)),
             g_q=1.0 + 0.1 * g.normal(size=hd), g_k=1.0 + 0.1 * g.normal(size=hd),
             Wo=scale * g.normal(size=(H, nh * hd)), g_mlp=1.0 + 0.1 * g.normal(size=H),
             Wg=scale * g.normal(size=(ffn, H)), Wu=scale * g.normal(size=(ffn, H)),
             Wd=scale * g.normal(size=(H, ffn)))
    return L.LayerParams.from_arrays(w, nh, nkv, hd, eps=1e-6, theta=1e4), w


def _inputs(P, batch=2, B=5, Cmax=9, seed=1):
    g = np.random.default_rng(seed)
    H = P.Wq.shape[1]
    x = g.normal(size=(batch, B, H))
    kc = g.normal(size=(batch, Cmax, P.n_kv, P.head_dim))
    vc = g.normal(size=(batch, Cmax, P.n_kv, P.head_dim))
    return x, kc, vc


# ------------------------------------------------------------- RMSNorm --------

def test_rmsnorm_closed_forms():
    # [3, 4]: mean square 12.5
    y = L.rmsnorm(np.array([3.0, 4.0]), np.array([1.0, 2.0]), 0.0)
    assert np.allclose(y, [3 / np.sqrt(12.5), 8 / np.sqrt(12.5)], rtol=1e-15)
    # a constant vector c becomes g * sign(c) (eps = 0); eps enters as c / sqrt(c^2 + eps)
    g = np.array([0.5, -1.5, 2.0])
    assert np.allclose(L.rmsnorm(np.full(3, -7.0), g, 0.0), -g, rtol=1e-15)
    assert np.allclose(L.rmsnorm(np.full(3, 1e-3), g, 1e-6), g * 1e-3 / np.sqrt(2e-6), rtol=1e-12)


# ------------------------------------------------------------- RoPE -----------

def test_rope_rotation_of_one_pair():
    # hd = 2: one pair turning by pos * theta^0 = pos radians; none at position 0,
    # two turns by 1 radian are one by 2, and one turn is the plane rotation
    x = np.array([[3.0, -2.0]])
    assert np.array_equal(L.rope(x, np.array([0]), 1e6), x)
    r1 = L.rope(L.rope(x, np.array([1]), 1e6), np.array([1]), 1e6)
    assert np.allclose(r1, L.rope(x, np.array([2]), 1e6), rtol=1e-14)
    r = L.rope(x, np.array([1]), 1e6)[0]
    c, s = np.cos(1.0), np.sin(1.0)
    assert np.allclose(r, [3 * c + 2 * s, -2 * c + 3 * s], rtol=1e-14)   # (a, b) -> (a c - b s, b c + a s)


def test_rope_frequency_schedule_by_hand():
    # theta = 1e4, head_dim 8: pair j = (j, j + 4) turns by pos * 1e4^(-2j/8)
    # = pos * 10^-j radians, i.e. 3, 0.3, 0.03 and 0.003 at position 3
    for j, ang in enumerate([3.0, 0.3, 0.03, 0.003]):
        x = np.zeros((2, 8))
        x[0, j] = 1.0                      # first member of pair j
        x[1, j + 4] = 1.0                  # second member
        y = L.rope(x, np.array([3, 3]), 1e4)
        e0 = np.zeros(8)
        e0[j], e0[j + 4] = np.cos(ang), np.sin(ang)
        e1 = np.zeros(8)
        e1[j], e1[j + 4] = -np.sin(ang), np.cos(ang)
        assert np.allclose(y[0], e0, rtol=0, atol=1e-15), j
        assert np.allclose(y[1], e1, rtol=0, atol=1e-15), j


def test_swiglu_applies_silu_to_the_gate_by_hand():
    """One FFN unit with gate 2 and up -1, attention switched off (Wo = 0):
    silu(2) * -1 = -1.76159..., which rounds to the bf16 value -1.7578125, so
    h = x1 + (-1.7578125, 0) with x1 = x = (1, 1).  SiLU on up instead,
    silu(-1) * 2 = -0.53788... (bf16 -0.5390625), would give 0.4609375."""
    w = dict(g_attn=np.ones(2), Wq=np.eye(2), Wk=np.eye(2), Wv=np.eye(2), g_q=np.ones(2),
             g_k=np.ones(2), Wo=np.zeros((2, 2)), g_mlp=np.ones(2), Wg=np.array([[2.0, 0.0]]),
             Wu=np.array([[0.0, -1.0]]), Wd=np.array([[1.0], [0.0]]))
    P = L.LayerParams.from_arrays(w, 1, 1, 2, eps=0.0, theta=1e4)
    x = np.ones((1, 1, 2))
    h = L.layer_forward(P, x, np.zeros((1, 1, 1, 2)), np.zeros((1, 1, 1, 2)), np.array([0]))
    assert h[0, 0, 0] == 1.0 - 1.7578125
    assert h[0, 0, 1] == 1.0


def test_rope_preserves_pair_norms_and_depends_on_relative_position():
    g = np.random.default_rng(3)
    hd = 16
    q, k = g.normal(size=(1, 3, hd)), g.normal(size=(1, 3, hd))
    for pos in (0, 7, 12345):
        r = L.rope(q, np.array([pos]), 1e6)
        a, b = r[..., :hd // 2], r[..., hd // 2:]
        qa, qb = q[..., :hd // 2], q[..., hd // 2:]
        assert np.allclose(a * a + b * b, qa * qa + qb * qb, rtol=1e-12)
    d1 = np.sum(L.rope(q, np.array([40]), 1e6) * L.rope(k, np.array([33]), 1e6), axis=-1)
    d2 = np.sum(L.rope(q, np.array([1007]), 1e6) * L.rope(k, np.array([1000]), 1e6), axis=-1)
    assert np.allclose(d1, d2, rtol=1e-9)


# ------------------------------------------------------------- attention ------

def test_attention_two_keys_in_ratio_three_to_one():
    """Scores differing by ln 3 after the 1/sqrt(hd) scale weight v in 3:1."""
    hd = 4
    q = np.zeros((1, 1, hd))
    q[0, 0, 0] = 1.0
    kc = np.zeros((1, 1, hd))
    kc[0, 0, 0] = np.log(3.0) * np.sqrt(hd)      # score ln 3
    kb = np.zeros((1, 1, hd))                    # the block key: score 0
    vc = np.full((1, 1, hd), 4.0)
    vb = np.full((1, 1, hd), -8.0)
    out = L.attention(q, kc, vc, kb, vb, n_kv=1)
    assert np.allclose(out, 0.75 * 4.0 + 0.25 * -8.0, rtol=1e-14)


def test_attention_equal_keys_average_the_visible_values():
    g = np.random.default_rng(4)
    B, C, hd = 4, 3, 8
    q = g.normal(size=(B, 2, hd))
    key = g.normal(size=hd)
    kc = np.broadcast_to(key, (C, 1, hd)).copy()
    kb = np.broadcast_to(key, (B, 1, hd)).copy()
    vc, vb = g.normal(size=(C, 1, hd)), g.normal(size=(B, 1, hd))
    out = L.attention(q, kc, vc, kb, vb, n_kv=1, causal=True)
    for i in range(B):
        want = np.concatenate([vc[:, 0], vb[:i + 1, 0]]).mean(axis=0)
        assert np.allclose(out[i, 0], want, rtol=1e-12) and np.allclose(out[i, 1], want, rtol=1e-12)
    bi = L.attention(q, kc, vc, kb, vb, n_kv=1, causal=False)
    assert np.allclose(bi[0, 0], np.concatenate([vc[:, 0], vb[:, 0]]).mean(axis=0), rtol=1e-12)


def test_attention_causal_mask_and_bidirectional_last_query():
    g = np.random.default_rng(5)
    B, C, nh, nkv, hd = 6, 4, 4, 2, 8
    q = g.normal(size=(B, nh, hd))
    kc, vc = g.normal(size=(C, nkv, hd)), g.normal(size=(C, nkv, hd))
    kb, vb = g.normal(size=(B, nkv, hd)), g.normal(size=(B, nkv, hd))
    out = L.attention(q, kc, vc, kb, vb, nkv, causal=True)
    for i in range(B):                      # block keys and values after i are never read
        kb2, vb2 = kb.copy(), vb.copy()
        kb2[i + 1:] = g.normal(size=kb2[i + 1:].shape) * 50
        vb2[i + 1:] = np.nan
        assert np.array_equal(L.attention(q, kc, vc, kb2, vb2, nkv, causal=True)[i], out[i])
    bi = L.attention(q, kc, vc, kb, vb, nkv, causal=False)
    assert np.array_equal(bi[B - 1], out[B - 1])       # the last query sees the whole block
    assert not np.allclose(bi[0], out[0])


def test_attention_gqa_equals_mha_on_repeated_kv_heads():
    g = np.random.default_rng(6)
    B, C, nh, nkv, hd = 3, 5, 6, 2, 8
    q = g.normal(size=(B, nh, hd))
    kc, vc = g.normal(size=(C, nkv, hd)), g.normal(size=(C, nkv, hd))
    kb, vb = g.normal(size=(B, nkv, hd)), g.normal(size=(B, nkv, hd))
    rep = lambda t: np.repeat(t, nh // nkv, axis=1)      # head h reads KV head h // 3
    assert np.allclose(L.attention(q, kc, vc, kb, vb, nkv),
                       L.attention(q, rep(kc), rep(vc), rep(kb), rep(vb), nh), rtol=1e-13)


# ------------------------------------------------------------- the layer ------

def test_layer_without_output_projections_is_the_identity():
    P, _ = _params()
    P.Wo[:] = 0.0
    P.Wd[:] = 0.0
    x, kc, vc = _inputs(P)
    assert np.array_equal(L.layer_forward(P, x, kc, vc, [9, 3]), x)


def test_layer_reads_no_cache_entry_past_the_context_length():
    P, _ = _params()
    x, kc, vc = _inputs(P)
    ctx = [4, 9]
    h = L.layer_forward(P, x, kc, vc, ctx)
    kc2, vc2 = kc.copy(), vc.copy()
    kc2[0, 4:] = np.nan
    vc2[0, 4:] = np.nan
    assert np.array_equal(L.layer_forward(P, x, kc2, vc2, ctx), h)


def test_layer_is_causal_over_the_block():
    P, _ = _params()
    x, kc, vc = _inputs(P, batch=1, B=6)
    h = L.layer_forward(P, x, kc, vc, [7])
    for i in range(5):
        x2 = x.copy()
        x2[0, i + 1:] += 3.0
        h2 = L.layer_forward(P, x2, kc, vc, [7])
        assert np.array_equal(h2[0, :i + 1], h[0, :i + 1])
        assert not np.allclose(h2[0, i + 1:], h[0, i + 1:])


def test_layer_block_of_one_without_context_ignores_the_query_path():
    """One query and one visible key: softmax weight 1 whatever q is, so Wq and g_q
    cannot matter; with context they do."""
    P, w = _params()
    x, kc, vc = _inputs(P, batch=1, B=1)
    h = L.layer_forward(P, x, kc, vc, [0])
    P.Wq[:] = np.random.default_rng(9).normal(size=P.Wq.shape)
    P.g_q[:] = -3.0
    assert np.array_equal(L.layer_forward(P, x, kc, vc, [0]), h)
    P2, _ = _params()
    assert not np.allclose(L.layer_forward(P, x, kc, vc, [5]), L.layer_forward(P2, x, kc, vc, [5]))


def test_layer_qk_norm_makes_q_and_k_projections_scale_free():
    P, _ = _params()
    x, kc, vc = _inputs(P)
    h = L.layer_forward(P, x, kc, vc, [9, 2])
    P.Wq *= 8.0
    P.Wk *= 0.125
    assert np.allclose(L.layer_forward(P, x, kc, vc, [9, 2]), h, atol=1e-9)
