"""Pins of the oracle's truncated (top-k / top-p) sampling against special
cases, hand-computed kept sets, brute force over subsets, Theorem 1 and exact
enumeration of speculative verification against the truncated target.  CPU
only."""
import itertools

import numpy as np
import pytest
import scipy.special

import oracle as O
from test_oracle_pins import _exact_sd_law, stress_params


def _kept(l, T=1.0, k=0, p=1.0):
    return set(np.nonzero(O.filtered_weights(np.asarray(l, dtype=float), T, k, p))[0].tolist())


def _brute_filter(probs, k, p):
    """The truncated distribution by definition, on a tiny vocabulary: top-k
    keeps v iff fewer than k tokens are strictly more probable; top-p keeps,
    among the top-k set, the subset of fewest tokens whose mass reaches p of
    the set's mass (the heaviest one if several), found by enumerating every
    subset.  Returns the renormalised distribution."""
    V = len(probs)
    keep = [v for v in range(V) if k <= 0 or sum(probs[u] > probs[v] for u in range(V)) < k]
    if p < 1.0:
        Z = sum(probs[v] for v in keep)
        best = None
        for n in range(1, len(keep) + 1):
            subsets = [c for c in itertools.combinations(keep, n)
                       if sum(probs[v] for v in c) >= p * Z]
            if subsets:
                best = max(subsets, key=lambda c: sum(probs[v] for v in c))
                break
        keep = list(best)
    out = np.zeros(V)
    out[keep] = np.asarray(probs)[keep]
    return out / out.sum()


def test_no_truncation_is_plain_sampling():
    g = np.random.default_rng(0)
    for _ in range(50):
        l = g.normal(0, 2, 40)
        T = float(g.uniform(0.3, 2.0))
        for k, p in [(0, 1.0), (40, 1.0), (100, 1.0), (0, 1.5)]:
            assert np.array_equal(O.filtered_weights(l, T, k, p), O.softmax_weights(l, T))
            u = float(g.random())
            assert O.select_sample(l, u, T, k, p)[0] == O.select_sample(l, u, T)[0]


def test_top1_is_greedy():
    g = np.random.default_rng(1)
    for _ in range(200):
        l = g.normal(0, 2, 30)
        assert O.select_sample(l, float(g.random()), float(g.uniform(0.2, 3)), 1)[0] == \
            int(np.argmax(l))
        assert O.select_sample(l, float(g.random()), 1.0, 0, 1e-9)[0] == int(np.argmax(l))


def test_top_k_kept_sets_by_hand():
    assert _kept([1, 3, 3, 2], k=2) == {1, 2}
    assert _kept([1, 3, 3, 2], k=3) == {1, 2, 3}
    assert _kept([3, 2, 2, 1], k=2) == {0, 1, 2}          # ties with the k-th value stay
    assert _kept([0.5, -1, 4, 2, 2.5], k=1) == {2}


def test_top_p_kept_sets_by_hand():
    probs = np.array([0.1, 0.4, 0.2, 0.3])
    assert _kept(np.log(probs), p=0.65) == {1, 3}          # 0.4 + 0.3 reaches 0.65
    assert _kept(np.log(probs), p=0.35) == {1}
    assert _kept([0, 0, 0, 0], p=0.5) == {0, 1}            # ties: lower index first
    assert _kept([0, 0, 0, 0], p=0.25) == {0}              # mass 1/4 reaches 1/4
    assert _kept([0, 0, 0, 0], p=0.2500001) == {0, 1}


def test_top_k_is_applied_before_top_p():
    # top-k 2 leaves (0.625, 0.375): top-p 0.6 keeps only token 0; top-p
    # first (0.5, 0.3 reach 0.6) would keep tokens 0 and 1
    assert _kept(np.log([0.5, 0.3, 0.2]), k=2, p=0.6) == {0}


def test_truncation_matches_brute_force_over_subsets():
    g = np.random.default_rng(2)
    for _ in range(300):
        V = int(g.integers(2, 7))
        l = g.normal(0, 1.5, V)
        T = float(g.uniform(0.5, 2.0))
        k = int(g.integers(0, V + 1))
        p = float(g.choice([1.0, g.uniform(0.05, 0.999)]))
        want = _brute_filter(scipy.special.softmax(l / T), k, p)
        got = O.softmax(l, T, k, p)
        assert np.allclose(got, want, rtol=1e-12, atol=1e-15), (l, T, k, p)


@pytest.mark.parametrize("k,p", [(3, 1.0), (0, 0.7), (3, 0.8)])
def test_thm1_holds_for_the_truncated_sampler(k, p):
    """The truncated inverse-CDF choice is still a function of the prefix, so
    Jacobi pins one more position per pass, reaches the sequential decode in
    B passes and that block is the only fixed point."""
    from test_oracle_pins import _all_stress
    for seed, (P, h) in _all_stress(12):
        g = np.random.default_rng(seed)
        s = O.base_logits(P.W_lm, h)
        u = g.random(4)
        ystar = O.sequential_decode(P, s, h, anchor=2, sample=True, u=u, top_k=k, top_p=p)
        res = O.refine_block(P, s, h, 2, seed=g.integers(0, 5, 4), sample=True, u=u, K=4,
                             early_exit=False, top_k=k, top_p=p)
        traj = res.traj_padded(4)
        for j in range(5):
            assert np.array_equal(traj[j][:j], ystar[:j])
        assert np.array_equal(traj[4], ystar)
        if seed < 3:
            fixed = [Y for Y in itertools.product(range(5), repeat=4)
                     if np.array_equal(O.pass_from(P, s, h, 2, np.array(Y), True, u, 1.0, k, p)[0],
                                       Y)]
            assert fixed == [tuple(ystar)]


@pytest.mark.parametrize("T,k,p", [(1.0, 3, 1.0), (1.0, 0, 0.75), (0.7, 3, 0.8)])
def test_truncated_speculative_verify_is_lossless_by_exact_enumeration(T, k, p):
    """Drafting and verifying with the same truncation emits tokens that
    follow the truncated target distribution exactly (computed here by brute
    force over subsets, not by the oracle)."""
    V, B = 4, 2
    P, h = stress_params(220, H=5, r=3, V=V, B=B, we_sigma=2.0)
    s = O.base_logits(P.W_lm, h)
    g = np.random.default_rng(13)
    table = {}
    for n in range(B + 2):
        for pre in itertools.product(range(V), repeat=n):
            table[pre] = g.normal(0, 1.5, V).astype(np.float32).astype(np.float64)
    target = lambda l: _brute_filter(scipy.special.softmax(l / T), k, p)
    m = B + 1
    law = _exact_sd_law(P, h, s, 1, table, B, V, m, T=T, top_k=k, top_p=p, target=target)
    assert abs(sum(law.values()) - 1.0) < 1e-12
    for x in itertools.product(range(V), repeat=m):
        want = 1.0
        for t in range(m):
            want *= target(table[x[:t]])[x[t]]
        assert abs(law.get(x, 0.0) - want) < 1e-12


def _icdf(probs, u):
    """Smallest v whose cumulative probability exceeds u (scipy's discrete ppf)."""
    import scipy.stats
    return int(scipy.stats.rv_discrete(values=(np.arange(len(probs)), probs)).ppf(u))


def test_sampled_seed_is_the_truncated_inverse_cdf_of_the_base_logits():
    """With K = 0 a sampled block is its seed: each position's inverse-CDF
    sample of the truncated softmax(s / T) at its own uniform."""
    P, h = stress_params(230, H=6, r=4, V=9, B=5)
    s = O.base_logits(P.W_lm, h)
    g = np.random.default_rng(14)
    for k, p, T in [(2, 1.0, 1.0), (0, 0.5, 0.8), (4, 0.7, 1.3)]:
        for _ in range(20):
            u = g.random(5)
            res = O.refine_block(P, s, h, 0, sample=True, u=u, K=0, T=T, top_k=k, top_p=p)
            want = [_icdf(_brute_filter(scipy.special.softmax(s[j] / T), k, p), u[j])
                    for j in range(5)]
            assert res.ids.tolist() == want


def test_bonus_token_samples_the_truncated_last_target_row():
    """Drafts the target always accepts (r = 0, q = p): the next token is the
    inverse-CDF sample of the truncated p_{B+1}.  With p_{B+1} = (0.1, 0.2,
    0.3, 0.4) and top-k 2 the kept tokens are 2 and 3 with mass 3/7 and 4/7,
    so u = 0.05 gives token 2 (plain sampling would give 0) and u = 0.5 gives
    token 3."""
    rows = np.log(np.array([[0.4, 0.3, 0.2, 0.1], [0.3, 0.4, 0.2, 0.1],
                            [0.1, 0.2, 0.3, 0.4]]))
    for u_res, want in [(0.05, 2), (0.5, 3), (0.42, 2), (0.43, 3)]:
        v = O.verify_sample(rows[:2], [0, 1], rows, [0.0, 0.0], u_res, 1.0, 2)
        assert (v.n, v.next) == (2, want)
