"""Seeded random configurations of the context layer, device vs the fp64
oracle (needs an MI355X).

Each case draws its shape from a generator seeded by the case number: hidden
width, query heads and query-group size (every built group: 1, 2, 4, 8),
FFN width, block length 1..32, batch sizes on both sides of the projections'
streaming limit (64 positions) so that the streamed, the tiled and the
split-K projection paths all occur, ragged context lengths from 0 to a few
hundred keys past the 64- and 128-key chunk boundaries, causal or full block
attention, and a layer created for a larger batch, block and context than
the call uses.  The fixed cases in test_gpu_layer.py cover each path on
purpose; these cover combinations of them, to the same bar.
"""
import numpy as np
import pytest

from test_gpu_layer import _case, _check, _run

N_CASES = 48


def _say(*a):
    print(*a, flush=True)


def draw_case(i):
    """The configuration of case i (a pure function of i)."""
    g = np.random.default_rng(0xBEEF + 104729 * i)
    H = int(g.choice([256, 512, 768, 1024]))
    grp = int(g.choice([1, 2, 4, 8]))
    nkv = int(g.choice([1, 2]))
    nh = grp * nkv
    if nh % 2:                      # n_heads * 128 must be a multiple of 256
        nkv, nh = 2, 2 * grp
    ffn = int(g.choice([256, 512, 768, 1280]))
    B = int(g.choice([1, 3, 8, 16, 17, 32]))
    batch = int(g.choice([1, 2, 3, 5, 9, 17]))
    ctx = [int(c) for c in g.choice([0, 1, 63, 64, 65, 127, 128, 129, 200, 257, 511, 700], batch)]
    causal = bool(g.random() < 0.7)
    grow = bool(g.random() < 0.3)
    return dict(H=H, nh=nh, nkv=nkv, ffn=ffn, B=B, batch=batch, ctx=ctx, causal=causal,
                max_batch=batch + (3 if grow else 0), max_B=min(32, B + (8 if grow else 0)),
                max_ctx=max(ctx) + (300 if grow else 0))


def test_layer_draws_cover_every_path():
    """Host-side check of the drawn table: every group size, both sides of
    the streaming limit, block lengths 1 and 32, empty contexts, both
    attention masks, larger layers than calls; all within the built set."""
    cases = [draw_case(i) for i in range(N_CASES)]
    assert {c["nh"] // c["nkv"] for c in cases} == {1, 2, 4, 8}
    assert any(c["batch"] * c["B"] > 64 for c in cases)
    assert any(c["batch"] * c["B"] <= 16 for c in cases)
    assert any(c["B"] == 1 for c in cases) and any(c["B"] == 32 for c in cases)
    assert any(0 in c["ctx"] for c in cases)
    assert {c["causal"] for c in cases} == {True, False}
    assert any(c["max_batch"] > c["batch"] for c in cases)
    for c in cases:
        assert c["H"] % 256 == 0 and (c["nh"] * 128) % 256 == 0 and c["ffn"] % 256 == 0
        assert c["nh"] // c["nkv"] in (1, 2, 4, 8) and c["nh"] % c["nkv"] == 0
        assert 1 <= c["B"] <= c["max_B"] <= 32 and c["batch"] <= c["max_batch"]


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(N_CASES))
def test_layer_random_case(i):
    c = draw_case(i)
    _say(f"case {i}: " + " ".join(f"{k}={v}" for k, v in c.items()))
    w, weights, inp = _case(c["H"], c["nh"], c["nkv"], c["ffn"], c["B"], c["batch"], c["ctx"],
                            index=1300 + i, c_max=c["max_ctx"])
    h32, hb, layer, _ = _run(w, weights, inp, c["causal"], max_ctx=c["max_ctx"],
                             max_batch=c["max_batch"], max_B=c["max_B"])
    _check(w, weights, inp, h32, hb, c["causal"])
    layer.close()
