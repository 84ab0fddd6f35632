"""The context layer on the device vs the fp64 oracle, through the C ABI
(needs an MI355X).

Small shapes span several k-split chunks of every projection, several
attention chunks (64-key ones for small calls, 128-key ones for large) with
ragged context lengths (0, chunk boundaries),
every built query-group size, blocks of 1, 8, 16 and 32 positions, and the
projection paths (streaming up to 64 positions, the tiled GEMM with 128 x 128
tiles, split over k where those are fewer than the CUs, and 256 x 256 ones
where a launch has 512 of them or more);
the full-size case runs the
Qwen3-8B layer at batch 1 with a 2048-key context.

Tolerance: h is compared in fp32 against the oracle's fp64 h with the bf16
rounding points of the device (u, q, k, v, the attention output, u2 and the
SwiGLU activation); what remains is fp32 accumulation order, the softmax
numerators of P.V (two bf16 parts each) and the rare bf16 rounding that the
fp32 and fp64 values of an intermediate take to different neighbours.  That
remainder is not the device's own: the oracle's steps evaluated in fp32 with
the same rounding points (tests/layer_fp32_floor.py) lie up to 0.0196 from
the fp64 result at the batch-64 shape, 1.6e-3 of its largest |h| (12.3).  The
bar is therefore one bf16 unit at the output's scale, 2^-8 max|h|, and never
below the 2e-2 absolute of bf16 logits: 2e-2 on the small shapes, 0.048 at
|h| = 12.3, 2.4 times the fp32 floor.
"""
import numpy as np
import pytest

import oracle as O
import synth
from synth.configs import QWEN_B1

pytestmark = pytest.mark.gpu

ATOL = 2e-2


def _say(*a):
    print(*a, flush=True)


def _case(H, nh, nkv, ffn, B, batch, ctx, index, c_max=None):
    w = synth.scaled(QWEN_B1, index=index, H=H, B=B, batch=batch, n_heads=nh, n_kv_heads=nkv,
                     ffn=ffn, ctx_len=None, ctx_len_range=None)
    weights = synth.make_layer_weights(w)
    inp = synth.make_layer_inputs(w, c_max=c_max if c_max is not None else max(max(ctx), 1))
    inp.ctx_len = np.asarray(ctx, dtype=np.int32)
    return w, weights, inp


def _run(w, weights, inp, causal=True, max_ctx=None, layer=None, max_batch=None, max_B=None):
    import torch
    from paper_2608_02438_amd.xpress import LAYER_WEIGHT_NAMES, Layer, device_tensor
    dw = {n: device_tensor(weights[n]) for n in LAYER_WEIGHT_NAMES}
    if layer is None:
        layer = Layer(dw, w.H, w.n_heads, w.n_kv_heads, w.ffn, max_batch=max_batch or w.batch,
                      max_B=max_B or w.B, max_ctx=max_ctx or inp.k_cache.shape[1])
    dev = [device_tensor(a) for a in (inp.x, inp.k_cache, inp.v_cache, inp.ctx_len)]
    h32, hb = layer.forward(*dev, causal=causal)
    torch.cuda.synchronize()
    hb_bits = hb.cpu().view(torch.int16).numpy().view(np.uint16)
    return h32.cpu().numpy(), hb_bits, layer, dw


def _check(w, weights, inp, h32, hb_bits, causal=True, seqs=None):
    """h of the chosen sequences (default all) against the oracle run on just
    those sequences (each sequence's layer output depends only on its own
    inputs and context)."""
    P = O.layer_ref.LayerParams.from_arrays(weights, w.n_heads, w.n_kv_heads, w.head_dim)
    sl = slice(None) if seqs is None else list(seqs)
    ref = O.layer_ref.layer_forward(P, inp.x[sl], inp.k_cache[sl], inp.v_cache[sl],
                                    inp.ctx_len[sl], causal)
    err = np.abs(h32[sl] - ref)
    bar = max(ATOL, 2.0 ** -8 * float(np.abs(ref).max()))
    _say(f"  max|h|={np.abs(ref).max():.3g} max|dh|={err.max():.3g} mean|dh|={err.mean():.3g} "
         f"bar={bar:.3g}")
    assert np.all(np.isfinite(h32))
    assert err.max() <= bar
    # the bf16 output is the rounding of the fp32 one
    assert np.array_equal(hb_bits, synth.f32_to_bf16_bits(h32))


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("H,nh,nkv,ffn,B,batch,ctx", [
    (256, 4, 2, 512, 8, 3, [600, 3, 256]),          # group 2, three KV chunks, ragged
    (512, 8, 2, 768, 16, 2, [0, 257]),              # group 4 (the Qwen3 ratio), no context
    (256, 8, 1, 256, 32, 1, [300]),                 # group 8, two position blocks
    (256, 2, 2, 256, 1, 2, [1, 511]),               # group 1, blocks of one position
])
def test_layer_matches_oracle(H, nh, nkv, ffn, B, batch, ctx, causal):
    _say(f"case: layer H={H} heads={nh}/{nkv} ffn={ffn} B={B} batch={batch} ctx={ctx} "
         f"causal={causal}")
    w, weights, inp = _case(H, nh, nkv, ffn, B, batch, ctx, index=700 + H + B)
    h32, hb, layer, _ = _run(w, weights, inp, causal)
    _check(w, weights, inp, h32, hb, causal)
    layer.close()


def test_layer_large_call_takes_128_key_chunks():
    """8 sequences x 8 KV heads x up to 33 chunks of 128 keys: at least 512
    workgroups, so the forward takes the 128-key attention chunks (smaller
    calls take 64-key ones); ragged contexts from 0 to 4095 keys."""
    ctx = [4000, 3000, 2500, 1, 0, 257, 4095, 100]
    _say(f"case: layer 128-key chunks H=256 heads 8/8 B=16 batch=8 ctx={ctx}")
    w, weights, inp = _case(256, 8, 8, 256, 16, 8, ctx, index=811, c_max=4096)
    h32, hb, layer, _ = _run(w, weights, inp)
    _check(w, weights, inp, h32, hb)
    layer.close()


def test_layer_projections_as_gemm_with_128_tiles():
    """192 positions: the projections run as the tiled GEMM with 128 x 128
    tiles in three position tiles, the last one ragged (the streaming kernel
    takes up to 64 positions)."""
    ctx = [5, 700, 33, 0, 256, 1000, 64, 129, 300, 2, 511, 90]
    _say(f"case: layer GEMM path H=512 heads 8/2 ffn=512 B=16 batch=12 ctx={ctx}")
    w, weights, inp = _case(512, 8, 2, 512, 16, 12, ctx, index=833)
    h32, hb, layer, _ = _run(w, weights, inp)
    _check(w, weights, inp, h32, hb)
    layer.close()


def test_layer_projections_split_over_k():
    """96 positions at H = 1024, ffn = 2048: the tiled GEMM's 128 x 128 tiles
    are fewer than the CUs, so the q/k/v (12 tiles, K = 1024), output (8
    tiles, K = 1024) and down (8 tiles, K = 2048) projections cut k into 2, 2
    and 4 parts whose slabs the next kernel adds; the gate/up projection
    forms the SwiGLU product in its epilogue."""
    ctx = [0, 129, 1000, 64, 7, 513]
    _say(f"case: layer split-K H=1024 heads 8/2 ffn=2048 B=16 batch=6 ctx={ctx}")
    w, weights, inp = _case(1024, 8, 2, 2048, 16, 6, ctx, index=845)
    h32, hb, layer, _ = _run(w, weights, inp)
    _check(w, weights, inp, h32, hb)
    layer.close()


def test_layer_gate_up_as_gemm_with_256_tiles():
    """1024 positions and ffn = 16384: the gate/up launch (32768 stacked rows)
    has 128 x 4 tiles of 256 x 256 and takes them; the other projections
    stay on 128 x 128 tiles."""
    ctx = [(37 * i) % 300 for i in range(32)]
    _say(f"case: layer 256-tile GEMM H=256 heads 2/2 ffn=16384 B=32 batch=32 ctx={ctx}")
    w, weights, inp = _case(256, 2, 2, 16384, 32, 32, ctx, index=857)
    h32, hb, layer, _ = _run(w, weights, inp)
    _check(w, weights, inp, h32, hb)
    layer.close()


def test_layer_largest_hidden_size():
    """H = 8192, the largest built: 32 values per thread in the RMSNorm row,
    K = 8192 in the q/k/v, gate and up projections."""
    _say("case: layer H=8192 heads 4/2 ffn=256 B=8 batch=1 ctx=[50]")
    w, weights, inp = _case(8192, 4, 2, 256, 8, 1, [50], index=871)
    h32, hb, layer, _ = _run(w, weights, inp)
    _check(w, weights, inp, h32, hb)
    layer.close()


def test_layer_run_to_run_and_cache_past_context_unread():
    import torch
    from paper_2608_02438_amd.xpress import device_tensor
    _say("case: layer determinism, H=512 heads 8/2 B=16 batch=2 ctx=[100, 700]")
    w, weights, inp = _case(512, 8, 2, 512, 16, 2, [100, 700], index=777)
    h1, b1, layer, _ = _run(w, weights, inp)
    h2, b2, _, _ = _run(w, weights, inp, layer=layer)
    assert np.array_equal(h1, h2) and np.array_equal(b1, b2)
    inp.k_cache[0, 100:] = 0x7FC0                  # NaN bit patterns past sequence 0's context
    inp.v_cache[0, 100:] = 0x7FC0
    h3, _, _, _ = _run(w, weights, inp, layer=layer)
    assert np.array_equal(h3, h1)
    layer.close()


def test_layer_rejects_bad_calls():
    import torch
    from paper_2608_02438_amd.xpress import XpError
    w, weights, inp = _case(256, 4, 2, 256, 8, 1, [10], index=790)
    _, _, layer, _ = _run(w, weights, inp, max_ctx=10)
    from paper_2608_02438_amd.xpress import device_tensor
    x, k, v, c = (device_tensor(a) for a in (inp.x, inp.k_cache, inp.v_cache, inp.ctx_len))
    big = torch.zeros((1, 64, 2, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(XpError):
        layer.forward(x, big, big, c)              # C_max beyond the layer's max_ctx
    x2 = torch.zeros((2, 8, 256), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(XpError):
        layer.forward(x2, k, v, c)                 # batch beyond max_batch
    layer.close()


def test_layer_qwen3_shape_batch1_ctx2048():
    _say("case: layer Qwen3-8B shape H=4096 heads 32/8 ffn=12288 B=16 batch=1 ctx=2048")
    w, weights, inp = _case(4096, 32, 8, 12288, 16, 1, [2048], index=901)
    h32, hb, layer, _ = _run(w, weights, inp)
    _check(w, weights, inp, h32, hb)
    layer.close()


@pytest.mark.parametrize("max_batch,max_B,batch,B", [(2, 32, 1, 16), (2, 32, 2, 8),
                                                     (8, 16, 1, 16), (8, 16, 3, 16)])
def test_layer_called_below_its_created_maxima(max_batch, max_B, batch, B):
    """A layer serves any call up to the sizes it was created for, whichever
    projection path that call takes: created for 64 or 128 positions and
    called with one block of 16 (the stream kernel, gate and up through the
    fp32 gate/up buffer), two blocks of 8, or 48 positions (the k-split
    kernel)."""
    ctx = [(97 * i + 40) % 500 for i in range(batch)]
    _say(f"case: layer created max_batch={max_batch} max_B={max_B}, called batch={batch} B={B} "
         f"ctx={ctx}")
    w, weights, inp = _case(512, 8, 2, 768, B, batch, ctx, index=950 + 10 * max_B + batch)
    h32, hb, layer, _ = _run(w, weights, inp, max_batch=max_batch, max_B=max_B, max_ctx=512)
    _check(w, weights, inp, h32, hb)
    layer.close()


# The Qwen3-8B layer at the shapes of the three larger workloads (batch 8 with
# 4096 context keys, batch 32 with 8192, batch 64 of 32 positions with ragged
# contexts U{512..16384}); the device runs the whole batch, and the oracle
# checks a few sequences of it (the longest and the shortest context among them).
@pytest.mark.parametrize("batch,B,ctx_len,ctx_range,seqs", [
    (8, 16, 4096, None, [0, 7]),
    (32, 16, 8192, None, [0, 13, 31]),
    (64, 32, None, (512, 16384), None),
])
def test_layer_qwen3_shape_at_workload_sizes(batch, B, ctx_len, ctx_range, seqs):
    w = synth.scaled(QWEN_B1, index=905 + batch, B=B, batch=batch, ctx_len=ctx_len,
                     ctx_len_range=ctx_range)
    weights = synth.make_layer_weights(w)
    inp = synth.make_layer_inputs(w)
    if seqs is None:
        order = np.argsort(inp.ctx_len)
        seqs = sorted({int(order[0]), int(order[-1]), 5, 40})
    _say(f"case: layer Qwen3-8B shape batch={batch} B={B} ctx max {int(inp.ctx_len.max())} "
         f"min {int(inp.ctx_len.min())}; oracle checks sequences {seqs} "
         f"(ctx {[int(inp.ctx_len[q]) for q in seqs]})")
    h32, hb, layer, _ = _run(w, weights, inp)
    _check(w, weights, inp, h32, hb, seqs=seqs)
    layer.close()
