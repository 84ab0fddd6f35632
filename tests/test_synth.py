"""Sanity of the seeded input generator (no arithmetic of the method here)."""
import numpy as np
import torch

import synth
from synth import gen
from synth.configs import TINY_F32, QWEN_B1, QWEN_B64_MIXED, scaled


def test_bf16_bit_helpers_match_torch():
    x = np.random.default_rng(0).normal(0, 3, 5000).astype(np.float32)
    x[:4] = [0.0, -0.0, 1.00390625, 1.01171875]      # two exact ties
    bits = gen.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bits, ref)
    assert np.array_equal(gen.bf16_bits_to_f32(bits), torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_streams_are_deterministic_and_order_free():
    w = scaled(QWEN_B1, V=3000, H=512)
    a = synth.make_weights(w, ["W_r", "W_e"])
    b = synth.make_weights(w, ["W_e", "W_r"])
    assert np.array_equal(a["W_r"], b["W_r"]) and np.array_equal(a["W_e"], b["W_e"])
    assert not np.array_equal(a["W_r"], a["W_e"])


def test_bf16_normal_moments():
    w = scaled(QWEN_B1, V=20000)
    x = gen.bf16_bits_to_f32(synth.make_weights(w, ["W_r"])["W_r"]).astype(np.float64)
    assert abs(x.mean()) < 2e-4 and abs(x.std() - 0.02) < 2e-4


def test_smaller_batch_is_a_prefix_of_the_full_batch():
    w = scaled(QWEN_B64_MIXED, V=2000, H=256)
    full = synth.make_inputs(w)
    part = synth.make_inputs(w, batch=5)
    assert np.array_equal(full.h[:5], part.h)
    assert np.array_equal(full.anchor[:5], part.anchor)
    assert np.array_equal(full.temp[:5], part.temp)


def test_lower_triangle_only_and_upper_fill():
    w = scaled(TINY_F32, B=6)
    L = synth.make_weights(w, ["L"], upper_fill=7.0)["L"]
    keep = np.tril(np.ones((6, 6), bool), -1)
    assert np.all(L[:, ~keep] == 7.0) and np.all(L[:, keep] != 7.0)


def test_greedy_target_acceptance_has_geometric_mean():
    """E[n] = p (1 - p^B) / (1 - p) when each position matches w.p. p."""
    p, B, N = 0.8, 16, 20000
    w = scaled(QWEN_B1, batch=N, V=1000, H=256, index=77)
    inp = synth.make_inputs(w)
    draft = np.zeros((N, B), np.int32)
    inp.alts[inp.alts == 0] = 1            # alternatives never equal the draft here
    t = inp.target_ids(draft)
    n = np.argmin(np.concatenate([t[:, :B] == draft, np.zeros((N, 1), bool)], 1), axis=1)
    expect = p * (1 - p ** B) / (1 - p)
    assert abs(n.mean() - expect) < 0.05
