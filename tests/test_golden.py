"""The oracle against the hand-computed fixtures in tests/golden/ (CPU).

Each fixture was worked out by hand from the definition it cites (the work is
written next to the values), so these pins do not depend on the oracle or on
any library routine it calls.
"""
import json
import os

import numpy as np
import pytest

import oracle as O

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_mix_block_of_three():
    g = _load("mix_b3.json")
    L = np.asarray(g["L"], dtype=np.float64)          # [d][k][i], 99 above the diagonal
    A = np.asarray(g["A"], dtype=np.float64)          # [k][d]
    C = O.mix(L, A)
    assert np.array_equal(C, np.asarray(g["C"], dtype=np.float64))


def test_greedy_tie_rule_and_inverse_cdf_boundaries():
    g = _load("select_rules.json")
    for c in g["greedy"]:
        y, margin = O.select_greedy(np.asarray(c["l"]))
        assert y == c["y"] and margin == c["margin"], c
    for c in g["inverse_cdf"]:
        y, _ = O.inverse_cdf(np.asarray(c["w"], dtype=np.float64), c["u"])
        assert y == c["y"], c


def test_speculative_verification_cases():
    g = _load("verify_v4.json")
    for c in g["cases"]:
        q_logits = np.log(np.asarray(c["q"], dtype=np.float64))
        p_logits = np.log(np.asarray(c["p"], dtype=np.float64))
        v = O.verify_sample(q_logits, c["ids"], p_logits, np.asarray(c["r"]), c["u_res"], g["T"])
        assert (v.n, v.next) == (c["n"], c["next"]), c["name"]


def test_acceptance_probability_is_one_minus_tv():
    """P(accept y ~ q) = sum_y q(y) min(1, p(y) / q(y)): the oracle's accept
    test flips exactly at r = p(y) / q(y) for every y, and the accepted mass
    it implies equals the hand value sum_v min(p, q) = 1 - TV."""
    g = _load("verify_v4.json")["accept_rate"]
    q = np.asarray(g["q"], dtype=np.float64)
    p = np.asarray(g["p"], dtype=np.float64)
    ql, pl = np.log(q)[None, :], np.log(np.vstack([p, p]))
    mass = 0.0
    for y in range(q.shape[0]):
        ratio = p[y] / q[y]
        if ratio < 1.0:
            below = O.verify_sample(ql, [y], pl, np.array([ratio * (1 - 1e-9)]), 0.5)
            above = O.verify_sample(ql, [y], pl, np.array([ratio * (1 + 1e-9)]), 0.5)
            assert below.n == 1 and above.n == 0
        else:
            assert O.verify_sample(ql, [y], pl, np.array([1.0 - 1e-12]), 0.5).n == 1
        mass += q[y] * min(1.0, ratio)
    assert mass == pytest.approx(g["sum_min"], abs=1e-12)
    assert 1.0 - 0.5 * np.abs(p - q).sum() == pytest.approx(g["sum_min"], abs=1e-12)
    assert 0.5 * np.abs(p - q).sum() == pytest.approx(g["tv"], abs=1e-12)


def test_bf16_round_to_nearest_even():
    g = _load("bf16_rne.json")
    x = np.asarray([c["x"] for c in g["cases"]], dtype=np.float32)
    want = np.asarray([c["bf16"] for c in g["cases"]], dtype=np.float64)
    got = np.asarray(O.round_bf16(x), dtype=np.float64)
    assert np.array_equal(got, want), list(zip(x.tolist(), got.tolist(), want.tolist()))


def test_tiny_refiner_by_hand():
    """Fuse (block order [h | g | token], g the mean, x_{k-1} the previous
    guess), Mix, Read, Correct and the Jacobi loop at H = r = 1, V = 2, B = 2."""
    g = _load("refiner_tiny.json")
    w = {k: np.asarray(v, dtype=np.float64) for k, v in g["weights"].items()}
    P = O.Params.from_arrays(w, round_z=False)
    h = np.asarray(g["h"], dtype=np.float64)
    s = O.base_logits(w["W_lm"], h)
    assert np.array_equal(s, np.asarray(g["s"]))
    st = O.fuse_static(P, h)
    for ps in g["passes"]:
        x_prev = np.concatenate([[g["anchor"]], np.asarray(ps["Y_prev"])[:-1]])
        A = O.fuse(P, st, x_prev)
        C = O.mix(P.L, A)
        assert np.array_equal(A, np.asarray(ps["A"])) and np.array_equal(C, np.asarray(ps["C"]))
        delta, _ = O.refiner(P, st, x_prev)
        assert np.array_equal(delta, np.asarray(ps["delta"]))
        Y, _, l = O.pass_from(P, s, h, g["anchor"], ps["Y_prev"], False, None)
        assert np.array_equal(l, np.asarray(ps["l"])) and list(Y) == ps["Y"]
    r = O.refine_block(P, s, h, g["anchor"], K=3)
    assert list(r.traj[0]) == g["Y0"]
    assert list(r.ids) == g["ids"] and r.iters == g["iters"]
    assert list(O.sequential_decode(P, s, h, g["anchor"])) == g["sequential"]
