"""The allocation-free context-layer forward (xp_layer_forward_noalloc) on the
device, through the C ABI: its output must match the handle-based
xp_layer_forward on the same inputs (bit for bit where both take the same
attention chunking; to the bf16 tolerance 2e-2 where the static scratch makes
it read the context in longer chunks), on consecutive calls whose second one
is smaller, and the oracle within the same tolerance."""
import numpy as np
import pytest

import oracle as O
import synth
from synth.configs import QWEN_B1

pytestmark = pytest.mark.gpu

ATOL = 2e-2


def _say(*a):
    print(*a, flush=True)


def _case(H, nh, nkv, ffn, B, batch, ctx, index):
    w = synth.scaled(QWEN_B1, index=index, H=H, B=B, batch=batch, n_heads=nh, n_kv_heads=nkv,
                     ffn=ffn, ctx_len=None, ctx_len_range=None)
    weights = synth.make_layer_weights(w)
    inp = synth.make_layer_inputs(w, c_max=max(max(ctx), 1))
    inp.ctx_len = np.asarray(ctx, dtype=np.int32)
    return w, weights, inp


def _both(w, weights, inp):
    """(handle forward, allocation-free forward) outputs as numpy arrays."""
    import torch
    from paper_2608_02438_amd.xpress import (LAYER_WEIGHT_NAMES, Layer, device_tensor,
                                             layer_forward_noalloc, layer_weights_struct)
    dw = {n: device_tensor(weights[n]) for n in LAYER_WEIGHT_NAMES}
    x, kc, vc, cl = (device_tensor(a) for a in (inp.x, inp.k_cache, inp.v_cache, inp.ctx_len))
    layer = Layer(dw, w.H, w.n_heads, w.n_kv_heads, w.ffn, max_batch=w.batch, max_B=w.B,
                  max_ctx=inp.k_cache.shape[1])
    r32, rb = layer.forward(x, kc, vc, cl)
    torch.cuda.synchronize()
    layer.close()
    s = layer_weights_struct(dw, w.H, w.n_heads, w.n_kv_heads, w.ffn)
    n32 = torch.full_like(r32, float("nan"))
    nb = torch.zeros_like(rb)
    layer_forward_noalloc(s, x, kc, vc, cl, n32, nb)
    torch.cuda.synchronize()
    bits = lambda t: t.cpu().view(torch.int16).numpy().view(np.uint16)
    return r32.cpu().numpy(), bits(rb), n32.cpu().numpy(), bits(nb)


def _oracle(w, weights, inp):
    P = O.layer_ref.LayerParams.from_arrays(weights, w.n_heads, w.n_kv_heads, w.head_dim)
    return O.layer_ref.layer_forward(P, inp.x, inp.k_cache, inp.v_cache, inp.ctx_len)


def test_noalloc_forward_matches_the_handle_forward_on_consecutive_calls():
    cases = [
        # (H, heads, kv, ffn, B, batch, ctx, exact): the first call, a smaller
        # second one, then one whose default attention partials (8448 of
        # 8.3 KB) exceed the scratch, so it reads the context in longer chunks
        (512, 8, 2, 768, 16, 3, [600, 3, 256], True),
        (256, 4, 2, 256, 8, 1, [50], True),
        (512, 64, 8, 512, 16, 4, [4096, 4000, 1, 2500], False),
    ]
    for i, (H, nh, nkv, ffn, B, batch, ctx, exact) in enumerate(cases):
        _say(f"case {i}: noalloc layer H={H} heads={nh}/{nkv} ffn={ffn} B={B} batch={batch} "
             f"ctx={ctx}")
        w, weights, inp = _case(H, nh, nkv, ffn, B, batch, ctx, index=990 + i)
        r32, rb, n32, nb = _both(w, weights, inp)
        assert np.all(np.isfinite(n32))
        d = float(np.abs(n32 - r32).max())
        ref = _oracle(w, weights, inp)
        e = float(np.abs(n32 - ref).max())
        _say(f"  max|noalloc - forward|={d:.3g} max|noalloc - oracle|={e:.3g}")
        if exact:
            assert np.array_equal(n32, r32) and np.array_equal(nb, rb)
        assert d <= ATOL and e <= ATOL
        assert np.array_equal(nb, synth.f32_to_bf16_bits(n32))
