"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these tests compares the oracle with itself: each checks it against a
library routine, a closed form, a structural property the paper proves
(Proposition 1, Theorem 1, the Toeplitz remark, the Fuse-Mix fold), or brute
force / exact enumeration on tiny inputs.  They use "stress" weights (large
token embeddings, tiny V and r) so that Jacobi trajectories really take several
passes.
"""
import itertools

import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

import oracle as O


def stress_params(seed, H=6, r=4, V=5, B=4, we_sigma=3.0, round_z=False, upper_fill=0.0):
    g = np.random.default_rng(seed)
    L = g.normal(0, 0.7, (r, B, B))
    keep = np.tril(np.ones((B, B), bool), -1)
    L[:, ~keep] = upper_fill
    w = dict(
        W_lm=g.normal(0, 1.0, (V, H)),
        W_h=g.normal(0, 1 / np.sqrt(H), (r, H)),
        W_g=g.normal(0, 1 / np.sqrt(H), (r, H)),
        W_e=g.normal(0, we_sigma, (V, r)),
        W_in=g.normal(0, 1 / np.sqrt(3 * r), (r, 3 * r)),
        L=L,
        W_1=g.normal(0, 1 / np.sqrt(r), (2 * r, r)),
        W_2=g.normal(0, 1 / np.sqrt(2 * r), (r, 2 * r)),
        W_r=g.normal(0, 1.5, (V, r)),
    )
    h = g.normal(0, 1.0, (B, H))
    return O.Params.from_arrays(w, round_z=round_z), h


# ---------------------------------------------------------------- rounding ----

def test_round_bf16_matches_torch_rne():
    g = np.random.default_rng(1)
    x = np.concatenate([
        g.normal(0, 1, 20000), g.normal(0, 1e-3, 2000), g.normal(0, 1e30, 200),
        # exact halfway cases between bf16 neighbours (ties to even) and edges
        1.0 + np.arange(0, 64) * 2.0 ** -8, -(1.0 + np.arange(0, 64) * 2.0 ** -8),
        [0.0, -0.0, 2.0 ** -126, 2.0 ** -130, 2.0 ** -133, 3 * 2.0 ** -134, 3.3e38, -3.3e38],
    ]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.round_bf16(x.astype(np.float64))
    assert np.array_equal(got, ref)
    assert np.array_equal(np.signbit(got), np.signbit(ref))


def test_round_bf16_overflow_to_inf():
    got = O.round_bf16(np.array([3.4e38, -3.4e38, 1e300]))
    assert np.all(np.isinf(got)) and got[1] < 0


def test_silu_matches_scipy_expit():
    x = np.linspace(-60, 60, 4001)
    assert np.allclose(O.silu(x), x * scipy.special.expit(x), rtol=1e-14, atol=1e-300)


def test_widen_bf16_bits_exact():
    bits = np.array([0x3F80, 0xBF80, 0x0001, 0x7F7F, 0x0000, 0x8000], dtype=np.uint16)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(O.to_f64(bits), ref)


# --------------------------------------------------------- base readout A1 ----

def test_zero_readout_reduces_to_library_argmax():
    """With W_r = 0 the correction vanishes and the block is argmax(W_lm h)."""
    P, h = stress_params(3, H=16, r=4, V=50, B=5)
    P.W_r[:] = 0.0
    s = O.base_logits(P.W_lm, h)
    assert np.allclose(s, h @ P.W_lm.T, rtol=1e-13, atol=1e-13)
    res = O.refine_block(P, s, h, anchor=2, K=3)
    assert np.array_equal(res.ids, np.argmax(h @ P.W_lm.T, axis=1))
    assert res.iters == 1


@pytest.mark.parametrize("V,chunk", [(20011, 8192), (50, 7)])
def test_base_logits_across_chunk_seams_is_the_exact_integer_product(V, chunk):
    """Small-integer weights (exact in bf16) and states make every product and
    partial sum an integer below 2^53, so the chunked fp64 readout must equal
    the int64 matrix product exactly in every row, on both sides of each chunk
    seam (8192 and 16384 at V = 20011; every 7 rows at V = 50)."""
    g = np.random.default_rng(11)
    H = 24
    Wi = g.integers(-8, 9, size=(V, H))
    hi = g.integers(-8, 9, size=(3, H))
    W_bits = (Wi.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    s = O.base_logits(W_bits, hi.astype(np.float32), chunk=chunk)
    assert s.shape == (3, V)
    assert np.array_equal(s, (hi @ Wi.T).astype(np.float64))


def test_argmax_ties_go_to_lowest_index():
    l = np.array([0.5, 2.0, -1.0, 2.0, 2.0])
    assert O.select_greedy(l)[0] == 1
    assert O.select_greedy(np.array([-0.0, 0.0, -1.0]))[0] == 0
    assert O.select_greedy(np.array([-1.0, 0.0, -0.0]))[0] == 1


def test_selection_is_taken_on_the_exact_logits():
    """Algorithm 1's argmax and the refined distribution are defined on the
    logits themselves: a gap of 1e-9 at 1.0 (below fp32 resolution, 6e-8)
    still decides.  Greedy: index 1.  Sampling at u = 0.5 - 1e-10: the first
    weight e^-1e-9 = 1 - 1e-9 is below u * Z = 1 - 7e-10, so the CDF crosses
    at index 1 (with the logits rounded to fp32 it would stay at index 0)."""
    l = np.array([1.0, 1.0 + 1e-9])
    assert O.select_greedy(l)[0] == 1
    assert O.select_sample(l, 0.5 - 1e-10)[0] == 1


# ------------------------------------------------------------- Fuse stages ----

def _with_win(P, block):
    r = P.r
    W = np.zeros((r, 3 * r))
    W[:, block * r:(block + 1) * r] = np.eye(r)
    P.W_in = W
    return P


def test_fuse_blocks_follow_equation_order():
    """W_in = [I|0|0], [0|I|0], [0|0|I] select W_h h_k, W_g g and W_e[x_{k-1}]."""
    P, h = stress_params(5, H=8, r=4, V=7, B=4)
    x_prev = np.array([6, 1, 3, 0])
    st = O.fuse_static(P, h)
    A = O.fuse(_with_win(P, 0), st, x_prev)
    assert np.allclose(A, h @ P.W_h.T)
    A = O.fuse(_with_win(P, 1), st, x_prev)
    assert np.allclose(A, np.tile(P.W_g @ h.mean(0), (4, 1)))
    A = O.fuse(_with_win(P, 2), st, x_prev)
    assert np.array_equal(A, P.W_e[x_prev])


def test_global_summary_of_equal_states_is_the_state():
    hj = np.random.default_rng(0).normal(size=9)
    assert np.allclose(O.global_summary(np.tile(hj, (7, 1))), hj, rtol=1e-15)


def test_token_feeding_position_k_is_the_previous_guess():
    """Position 1 reads the anchor, position k reads y_{k-1} (never y_k)."""
    P, h = stress_params(6, H=8, r=4, V=7, B=4)
    _with_win(P, 2)
    P.L[:] = 0.0
    P.W_1[:] = 0.0
    st = O.fuse_static(P, h)
    anchor, Y = 5, np.array([1, 2, 3, 4])
    delta, Z = O.refiner(P, st, np.concatenate([[anchor], Y[:-1]]))
    assert np.array_equal(Z, P.W_e[[5, 1, 2, 3]])


# ---------------------------------------------------------------- Mix ---------

@pytest.mark.parametrize("r,B", [(5, 7), (3, 1), (2, 32)])
def test_toeplitz_mix_is_causal_depthwise_conv1d(r, B):
    """The oracle's Toeplitz mixer makes Mix np.convolve with kernel
    [1, kappa_d[1], ..., kappa_d[B-1]] (Toeplitz remark), whatever kappa_d[0] is."""
    g = np.random.default_rng(7 + B)
    kappa = g.normal(size=(r, B))
    L = O.toeplitz_mixer(kappa)
    assert L.shape == (r, B, B)
    assert (L[:, np.triu(np.ones((B, B), bool))] == 0).all()          # strictly lower
    A = g.normal(size=(B, r))
    C = O.mix(L, A)
    for d in range(r):
        ker = kappa[d].copy()
        ker[0] = 1.0
        assert np.allclose(C[:, d], np.convolve(A[:, d], ker)[:B], rtol=1e-13, atol=1e-13)
    # one hand-checked entry: position 3 of channel 0 at B = 7
    if B == 7:
        want = A[3, 0] + kappa[0, 1] * A[2, 0] + kappa[0, 2] * A[1, 0] + kappa[0, 3] * A[0, 0]
        assert abs(C[3, 0] - want) < 1e-12


def test_mix_never_reads_diagonal_or_upper_triangle():
    P0, h = stress_params(8, upper_fill=0.0)
    P1, _ = stress_params(8, upper_fill=1e30)
    A = np.random.default_rng(1).normal(size=(4, P0.r))
    assert np.array_equal(O.mix(P0.L, A), O.mix(P1.L, A))


def test_fuse_mix_fold_identity():
    """The folded operator of section 4.1 equals Fuse followed by Mix."""
    P, h = stress_params(9, H=8, r=4, V=7, B=5)
    st = O.fuse_static(P, h)
    x_prev = np.array([3, 0, 6, 2, 2])
    At = np.concatenate([st.hh, np.tile(st.gg, (5, 1)), P.W_e[x_prev]], axis=1)
    unfolded = O.mix(P.L, O.fuse(P, st, x_prev))
    folded = O.fuse_mix_folded(P.W_in, P.L, At)
    assert np.allclose(unfolded, folded, rtol=1e-12, atol=1e-12)


def test_trans_special_case_is_elementwise_silu():
    """W_1 = I (stacked twice), W_2 = [I 0]: z = c + silu(c) elementwise."""
    r = 6
    P, _ = stress_params(10, r=r)
    P.W_1 = np.vstack([np.eye(r), np.zeros((r, r))])
    P.W_2 = np.hstack([np.eye(r), np.zeros((r, r))])
    C = np.random.default_rng(2).normal(0, 4, (3, r))
    assert np.allclose(O.trans(P, C), C + C * scipy.special.expit(C), rtol=1e-14)


def test_linear_path_is_plain_matmul():
    """L = 0 and W_2 = 0: delta_k = W_r W_in at_k."""
    P, h = stress_params(11, H=8, r=4, V=9, B=4)
    P.L[:] = 0.0
    P.W_2[:] = 0.0
    st = O.fuse_static(P, h)
    x_prev = np.array([8, 1, 1, 4])
    At = np.concatenate([h @ P.W_h.T, np.tile(P.W_g @ h.mean(0), (4, 1)), P.W_e[x_prev]], axis=1)
    delta, _ = O.refiner(P, st, x_prev)
    assert np.allclose(delta, At @ (P.W_r @ P.W_in).T, rtol=1e-12, atol=1e-12)


# -------------------------------------------------------- Proposition 1 -------

@pytest.mark.parametrize("seed", range(4))
def test_prop1_later_guesses_never_change_earlier_logits(seed):
    P, h = stress_params(20 + seed, H=6, r=4, V=6, B=5)
    s = O.base_logits(P.W_lm, h)
    st = O.fuse_static(P, h)
    g = np.random.default_rng(seed)
    Y = g.integers(0, 6, 5)
    base, _ = O.refiner(P, st, np.concatenate([[1], Y[:-1]]))
    for k in range(5):
        Y2 = Y.copy()
        Y2[k:] = g.integers(0, 6, 5 - k)      # change every guess at positions >= k
        d2, _ = O.refiner(P, st, np.concatenate([[1], Y2[:-1]]))
        # positions 0..k see x_0..x_{k} which are unchanged up to index k
        assert np.array_equal(d2[:k + 1], base[:k + 1])


def test_prop1_hidden_states_enter_only_through_own_state_and_summary():
    P, h = stress_params(30, H=6, r=4, V=6, B=5)
    x_prev = np.array([2, 3, 1, 0, 5])
    base, _ = O.refiner(P, O.fuse_static(P, h), x_prev)
    k, i, j = 1, 3, 4
    dlt = np.random.default_rng(0).normal(size=6)
    h2 = h.copy()
    h2[i] += dlt
    h2[j] -= dlt                                # g unchanged, h_k unchanged
    d2, _ = O.refiner(P, O.fuse_static(P, h2), x_prev)
    assert np.allclose(d2[k], base[k], rtol=1e-12, atol=1e-12)
    h3 = h.copy()
    h3[j] += dlt                                # g moves: position k must notice
    d3, _ = O.refiner(P, O.fuse_static(P, h3), x_prev)
    assert np.max(np.abs(d3[k] - base[k])) > 1e-6


# ------------------------------------------------------------ Theorem 1 -------

def _all_stress(n):
    for seed in range(n):
        yield seed, stress_params(100 + seed, H=6, r=4, V=5, B=4)


@pytest.mark.parametrize("sample,T", [(False, 1.0), (True, 1.0), (True, 0.5)])
def test_thm1_jacobi_pins_one_position_per_pass_and_reaches_sequential(sample, T):
    long_traj = 0
    for seed, (P, h) in _all_stress(40):
        g = np.random.default_rng(seed)
        s = O.base_logits(P.W_lm, h)
        u = g.random(4)
        ystar = O.sequential_decode(P, s, h, anchor=3, sample=sample, u=u, T=T)
        seed_ids = g.integers(0, 5, 4)
        res = O.refine_block(P, s, h, 3, seed=seed_ids, sample=sample, u=u, K=4,
                             early_exit=False, T=T)
        traj = res.traj_padded(4)
        for j in range(5):
            assert np.array_equal(traj[j][:j], ystar[:j])      # y_k^(j) = y*_k, k <= j
        assert np.array_equal(traj[4], ystar)                  # Y^(B) = Y*
        long_traj += res.iters >= 3
    assert long_traj >= 5, "stress weights should produce multi-pass trajectories"


@pytest.mark.parametrize("sample", [False, True])
def test_thm1_sequential_decode_is_the_unique_fixed_point(sample):
    for seed, (P, h) in _all_stress(6):
        s = O.base_logits(P.W_lm, h)
        u = np.random.default_rng(seed).random(4)
        ystar = O.sequential_decode(P, s, h, anchor=0, sample=sample, u=u)
        fixed = []
        for Y in itertools.product(range(5), repeat=4):
            Yn, _, _ = O.pass_from(P, s, h, 0, np.array(Y), sample, u)
            if np.array_equal(Yn, Y):
                fixed.append(Y)
        assert fixed == [tuple(ystar)]


def test_running_past_the_fixed_point_is_a_no_op():
    for seed, (P, h) in _all_stress(10):
        s = O.base_logits(P.W_lm, h)
        a = O.refine_block(P, s, h, 1, K=9, early_exit=True)
        b = O.refine_block(P, s, h, 1, K=9, early_exit=False)
        assert np.array_equal(a.ids, b.ids) and a.iters == b.iters
        assert np.array_equal(a.logits, b.logits)


def test_block_of_one_is_single_position_decoding():
    """B = 1: Mix is empty, g = h_1, and the block converges from any seed."""
    P, h = stress_params(40, H=6, r=4, V=7, B=1)
    s = O.base_logits(P.W_lm, h)
    outs = {tuple(O.refine_block(P, s, h, 4, seed=[y0], K=3).ids) for y0 in range(7)}
    assert len(outs) == 1
    st = O.fuse_static(P, h)
    assert np.allclose(st.gg, P.W_g @ h[0])
    res = O.refine_block(P, s, h, 4, seed=[0], K=3)
    assert res.iters <= 2


# --------------------------------------------------------- selection rules ----

def test_inverse_cdf_matches_scipy_discrete_ppf():
    g = np.random.default_rng(3)
    for _ in range(20):
        w = g.random(9) ** 3
        w[g.integers(0, 9)] = 0.0
        p = w / w.sum()
        dist = scipy.stats.rv_discrete(values=(np.arange(9), p))
        for u in g.random(200):
            assert O.inverse_cdf(w, u)[0] == int(dist.ppf(u))


def test_inverse_cdf_frequencies_follow_the_weights():
    w = np.array([0.1, 0.0, 2.0, 0.7, 1.2])
    us = (np.arange(200000) + 0.5) / 200000
    toks = np.array([O.inverse_cdf(w, u)[0] for u in us[::10]])
    freq = np.bincount(toks, minlength=5) / toks.size
    assert np.allclose(freq, w / w.sum(), atol=2e-4)


def test_select_sample_is_softmax_sampling():
    g = np.random.default_rng(4)
    l = g.normal(0, 2, 6)
    p = scipy.special.softmax(l.astype(np.float32).astype(np.float64))
    us = (np.arange(50000) + 0.5) / 50000
    toks = np.array([O.select_sample(l, u)[0] for u in us])
    assert np.allclose(np.bincount(toks, minlength=6) / toks.size, p, atol=1e-4)


@pytest.mark.parametrize("T", [0.3, 0.7, 2.5])
def test_select_sample_at_temperature_is_tempered_softmax_sampling(T):
    g = np.random.default_rng(12)
    l = g.normal(0, 2, 6)
    p = scipy.special.softmax(l.astype(np.float32).astype(np.float64) / T)
    us = (np.arange(50000) + 0.5) / 50000
    toks = np.array([O.select_sample(l, u, T)[0] for u in us])
    assert np.allclose(np.bincount(toks, minlength=6) / toks.size, p, atol=1e-4)


def test_low_temperature_sampling_is_the_argmax():
    """T -> 0: all mass on the largest logit (gaps >= 0.08 against T = 1e-3)."""
    g = np.random.default_rng(13)
    for _ in range(50):
        l = g.permutation(11) * 0.1 + g.uniform(-0.01, 0.01, 11)
        for u in (0.001, 0.3, 0.999):
            assert O.select_sample(l, u, 1e-3)[0] == int(np.argmax(l))


def test_high_temperature_sampling_is_uniform():
    """T -> infinity: every token has mass 1/V, so u picks floor(u V)."""
    l = np.random.default_rng(14).normal(0, 1, 7)
    for u in (np.arange(70) + 0.5) / 70:
        assert O.select_sample(l, u, 1e9)[0] == int(np.floor(u * 7))


# ------------------------------------------------------------ verification ----

def test_verify_greedy_is_brute_force_longest_prefix():
    g = np.random.default_rng(5)
    for _ in range(500):
        B = int(g.integers(1, 9))
        y = g.integers(0, 3, B)
        t = g.integers(0, 3, B + 1)
        n, nxt = O.verify_greedy(y, t)
        best = max(m for m in range(B + 1) if all(y[i] == t[i] for i in range(m)))
        assert n == best and nxt == t[best]


def _cells(probs):
    """Intervals of [0, 1) an inverse-CDF sampler maps to each token."""
    c = np.concatenate([[0.0], np.cumsum(probs)])
    c[-1] = 1.0
    return [(c[v], c[v + 1]) for v in range(len(probs)) if c[v + 1] > c[v]]


def _exact_sd_law(P, h, s, anchor, table, B, V, m, T=1.0, top_k=0, top_p=1.0, target=None):
    """Law of the first m emitted tokens of one SD round + target continuation.

    Enumerates every cell of (u_draft, r_accept, u_res) exactly and evaluates
    the oracle at the cell's midpoint.  ``table[prefix]`` are target logits;
    ``target(logits)`` is the target distribution (default softmax(l / T)).
    """
    law = {}
    if target is None:
        target = lambda l: scipy.special.softmax(l / T)
    p_of = lambda pre: target(table[tuple(pre)])

    def cont(prefix, prob):
        if len(prefix) >= m:
            key = tuple(prefix[:m])
            law[key] = law.get(key, 0.0) + prob
            return
        p = p_of(prefix)
        for x in range(V):
            if p[x] > 0:
                cont(prefix + [x], prob * p[x])

    def draft_cells(k, u_pre, prob):
        if k == B:
            yield np.array(u_pre), prob
            return
        u_try = np.array(u_pre + [0.5] + [0.5] * (B - k - 1))
        res = O.refine_block(P, s, h, anchor, sample=True, u=u_try, K=B, T=T, top_k=top_k,
                             top_p=top_p)
        q = O.softmax(res.logits[k], T, top_k, top_p)
        for lo, hi in _cells(q):
            yield from draft_cells(k + 1, u_pre + [(lo + hi) / 2], prob * (hi - lo))

    for u, pu in draft_cells(0, [], 1.0):
        res = O.refine_block(P, s, h, anchor, sample=True, u=u, K=B, T=T, top_k=top_k,
                             top_p=top_p)
        y = [int(t) for t in res.ids]
        plog = np.stack([table[tuple(y[:k])] for k in range(B + 1)])

        def branch(k, r_pre, prob):
            # enumerate accept/reject cells position by position
            if k == B:
                pb = p_of(y)
                for lo, hi in _cells(pb):
                    v = O.verify_sample(res.logits, y, plog, r_pre + [0.5] * (B - k), (lo + hi) / 2, T,
                                        top_k, top_p)
                    cont(y[:v.n] + [v.next], prob * (hi - lo))
                return
            q = O.softmax(res.logits[k], T, top_k, top_p)
            p = p_of(y[:k])
            a = min(1.0, p[y[k]] / q[y[k]])
            branch(k + 1, r_pre + [a / 2], prob * a)                  # accept cell
            if a < 1.0:
                rr = r_pre + [(1.0 + a) / 2] + [0.5] * (B - k - 1)     # reject cell
                resid = np.maximum(p - q, 0.0)
                resid = resid / resid.sum()
                for lo, hi in _cells(resid):
                    v = O.verify_sample(res.logits, y, plog, rr, (lo + hi) / 2, T, top_k, top_p)
                    assert v.n == k
                    cont(y[:k] + [v.next], prob * (1 - a) * (hi - lo))

        branch(0, [], pu)
    return law


@pytest.mark.parametrize("seed", range(3))
def test_speculative_verify_is_lossless_by_exact_enumeration(seed):
    V, B = 3, 2
    P, h = stress_params(200 + seed, H=5, r=3, V=V, B=B, we_sigma=2.0)
    s = O.base_logits(P.W_lm, h)
    g = np.random.default_rng(seed)
    table = {}
    for n in range(B + 2):
        for pre in itertools.product(range(V), repeat=n):
            table[pre] = g.normal(0, 1.5, V).astype(np.float32).astype(np.float64)
    m = B + 1
    law = _exact_sd_law(P, h, s, 1, table, B, V, m)
    assert abs(sum(law.values()) - 1.0) < 1e-12
    for x in itertools.product(range(V), repeat=m):
        target = 1.0
        for t in range(m):
            target *= scipy.special.softmax(table[x[:t]])[x[t]]
        assert abs(law.get(x, 0.0) - target) < 1e-12


@pytest.mark.parametrize("T", [0.6, 1.8])
def test_speculative_verify_at_temperature_is_lossless_by_exact_enumeration(T):
    """At temperature T the emitted tokens follow softmax(target / T) exactly."""
    V, B = 3, 2
    P, h = stress_params(210, H=5, r=3, V=V, B=B, we_sigma=2.0)
    s = O.base_logits(P.W_lm, h)
    g = np.random.default_rng(11)
    table = {}
    for n in range(B + 2):
        for pre in itertools.product(range(V), repeat=n):
            table[pre] = g.normal(0, 1.5, V).astype(np.float32).astype(np.float64)
    m = B + 1
    law = _exact_sd_law(P, h, s, 1, table, B, V, m, T=T)
    assert abs(sum(law.values()) - 1.0) < 1e-12
    for x in itertools.product(range(V), repeat=m):
        target = 1.0
        for t in range(m):
            target *= scipy.special.softmax(table[x[:t]] / T)[x[t]]
        assert abs(law.get(x, 0.0) - target) < 1e-12


def test_first_position_acceptance_is_one_minus_tv():
    """P(accept y_1) = sum_x min(p, q) = 1 - TV(p, q)  (section 4.3)."""
    V, B = 4, 1
    P, h = stress_params(300, H=5, r=3, V=V, B=B, we_sigma=2.0)
    s = O.base_logits(P.W_lm, h)
    pl = np.random.default_rng(9).normal(0, 1.5, (B + 1, V)).astype(np.float32).astype(np.float64)
    p = scipy.special.softmax(pl[0])
    tot = 0.0
    for lo, hi in _cells(O.softmax(O.refine_block(P, s, h, 0, sample=True, u=[0.5], K=1).logits[0])):
        res = O.refine_block(P, s, h, 0, sample=True, u=[(lo + hi) / 2], K=1)
        q = O.softmax(res.logits[0])
        y = int(res.ids[0])
        a = min(1.0, p[y] / q[y])
        # the oracle must accept just below the threshold and reject just above it
        assert O.verify_sample(res.logits, [y], pl, [a * 0.999], 0.5).n == 1
        if a < 1:
            assert O.verify_sample(res.logits, [y], pl, [a * 1.001 + 1e-12], 0.5).n == 0
        tot += (hi - lo) * a
    q = O.softmax(O.refine_block(P, s, h, 0, sample=True, u=[0.5], K=1).logits[0])
    assert abs(tot - (1 - 0.5 * np.abs(p - q).sum())) < 1e-12


def test_inverse_cdf_boundary_is_strict():
    """y = min{v : C_v > u Z}: a uniform landing exactly on C_v selects v + 1."""
    w = np.array([1.0, 1.0, 2.0])
    assert O.inverse_cdf(w, 0.25)[0] == 1
    assert O.inverse_cdf(w, 0.5)[0] == 2
    assert O.inverse_cdf(w, 0.0)[0] == 0
    assert O.inverse_cdf(np.array([0.0, 3.0, 0.0]), 0.0)[0] == 1


def test_sampling_is_shift_invariant_at_large_logits():
    """softmax is taken relative to the maximum: huge logits must not overflow."""
    l = np.array([1000.0, 999.0, 998.5, -1000.0])
    p = scipy.special.softmax(l)
    dist = scipy.stats.rv_discrete(values=(np.arange(4), p))
    for u in np.random.default_rng(0).random(300):
        assert O.select_sample(l, u)[0] == int(dist.ppf(u))
    assert np.allclose(O.softmax(l), p, rtol=1e-12)


def test_sampled_seed_is_inverse_cdf_of_base_softmax():
    """At temperature 1, Y^(0)_k samples softmax(s_k) with the position's uniform."""
    P, h = stress_params(50, H=8, r=4, V=9, B=6)
    s = O.base_logits(P.W_lm, h)
    g = np.random.default_rng(1)
    for _ in range(30):
        u = g.random(6)
        res = O.refine_block(P, s, h, 2, sample=True, u=u, K=0)
        for k in range(6):
            p = scipy.special.softmax(s[k].astype(np.float32).astype(np.float64))
            dist = scipy.stats.rv_discrete(values=(np.arange(9), p))
            assert res.ids[k] == int(dist.ppf(u[k]))
        assert res.iters == 0 and res.logits is s
