"""The device path against hand-computed values (needs an MI355X).

The tiny refiner of tests/golden/refiner_tiny.json (H = r = 1, V = 2, B = 2,
worked out by hand) embedded in the smallest built shape: H = r = 256 and
V = 16, every weight zero except the fixture's entries in channel 0 and
tokens 0 and 1.  Tokens 2..15 then have s = delta = 0 and never win, the
other 255 channels carry zeros, and every value on the path is an exact
binary fraction in bf16 and in fp32, so the device must reproduce the hand
values bit for bit: the seed from s, the logits and ids of each pass, the
pass count at the fixed point, and the verification that follows.  No oracle
is involved.
"""
import json
import os

import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
H, R, V, B = 256, 256, 16, 2


def _embedded(dtype):
    with open(os.path.join(GOLDEN, "refiner_tiny.json")) as f:
        g = json.load(f)
    t = g["weights"]
    w = {
        "W_lm": np.zeros((V, H), np.float32), "W_h": np.zeros((R, H), np.float32),
        "W_g": np.zeros((R, H), np.float32), "W_e": np.zeros((V, R), np.float32),
        "W_in": np.zeros((R, 3 * R), np.float32), "L": np.zeros((R, B, B), np.float32),
        "W_1": np.zeros((2 * R, R), np.float32), "W_2": np.zeros((R, 2 * R), np.float32),
        "W_r": np.zeros((V, R), np.float32),
    }
    w["W_lm"][0, 0], w["W_lm"][1, 0] = t["W_lm"][0][0], t["W_lm"][1][0]
    w["W_h"][0, 0], w["W_g"][0, 0] = t["W_h"][0][0], t["W_g"][0][0]
    w["W_e"][0, 0], w["W_e"][1, 0] = t["W_e"][0][0], t["W_e"][1][0]
    w["W_in"][0, 0], w["W_in"][0, R], w["W_in"][0, 2 * R] = t["W_in"][0]
    w["L"][0, 1, 0] = t["L"][0][1][0]                 # the only entry below the diagonal
    w["W_r"][0, 0], w["W_r"][1, 0] = t["W_r"][0][0], t["W_r"][1][0]
    h = np.zeros((1, B, H), np.float32)
    h[0, :, 0] = [row[0] for row in g["h"]]
    if dtype == "bf16":
        w = {n: synth.f32_to_bf16_bits(a) for n, a in w.items()}
        h = synth.f32_to_bf16_bits(h)
    return g, w, h


def _padded(rows):
    out = np.zeros((len(rows), V), np.float32)
    out[:, :2] = np.asarray(rows, np.float32)
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_device_reproduces_the_hand_computed_refiner(dtype):
    import torch
    from paper_2608_02438_amd.xpress import device_tensor, refiner_from_arrays
    print(f"case: hand-computed refiner embedded at H=r=256 V=16 B=2, {dtype}", flush=True)
    g, w, h = _embedded(dtype)
    ref = refiner_from_arrays(w, H, R, V, B, 1)
    hid = device_tensor(h)
    anchor = torch.tensor([g["anchor"]], dtype=torch.int32, device="cuda")
    # K = 0: the seed from the base logits, and l = s
    out0 = ref.refine_block(hid, anchor, K=0, write_logits=True)
    torch.cuda.synchronize()
    assert out0.ids.cpu().numpy()[0].tolist() == g["Y0"]
    assert np.array_equal(out0.logits.cpu().numpy()[0], _padded(g["s"]))
    # K = 1, 2, 3: the logits and ids of each pass, then the fixed point
    for K in (1, 2, 3):
        out = ref.refine_block(hid, anchor, K=K, write_logits=True, want_traj=True)
        torch.cuda.synchronize()
        ps = g["passes"][min(K, 2) - 1]
        assert np.array_equal(out.logits.cpu().numpy()[0], _padded(ps["l"])), K
        assert out.ids.cpu().numpy()[0].tolist() == ps["Y"], K
        traj = out.traj.cpu().numpy()[:, 0]
        assert traj[0].tolist() == g["Y0"] and traj[1].tolist() == g["passes"][0]["Y"]
        assert int(out.iters.cpu()[0]) == (g["iters"] if K >= g["iters"] else K)
    e = ref.refine_block(hid, anchor, K=3, early_exit=True)
    torch.cuda.synchronize()
    assert e.ids.cpu().numpy()[0].tolist() == g["ids"] and int(e.iters.cpu()[0]) == g["iters"]
    # greedy verification of the refined block [0, 0] (section 3.1): targets
    # [0, 1, 5] agree on the first draft only (n = 1, next = t_2 = 1); targets
    # [0, 0, 5] accept both and the bonus token 5 follows
    for tgt, want in (([0, 1, 5], (1, 1)), ([0, 0, 5], (2, 5))):
        n, nxt = ref.verify_block(e.ids, torch.tensor([tgt], dtype=torch.int32, device="cuda"))
        torch.cuda.synchronize()
        assert (int(n.cpu()[0]), int(nxt.cpu()[0])) == want, tgt
    assert ref.device_errors() == 0
