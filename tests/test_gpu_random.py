"""Seeded random configurations, device path vs the fp64 oracle (needs an MI355X).

Each case draws its own shape and options from a generator seeded by the case
number: element type, hidden width, a vocabulary from the smallest built (16)
to 33001 with a ragged tail, block length 1..32, batch sizes that
select the per-sequence LM-head stream, the LM-head GEMM and the many-position
Read, greedy / sampled / mixed rows, per-sequence temperatures, top-k and
top-p, seeded or base-logit initial iterates, pass budgets 0..9, weights at the
workloads' scale or at the stress scale (trajectories of several passes), and a
refiner built for a larger batch than the call uses.  The fixed cases in the
other modules cover each path on purpose; these cover combinations of them.

Per case: every decision of every pass is the oracle's or a near-tie within
the device error bound (checked inside ``check_refine``), the final logits lie
within that bound, verification agrees, and an early-exit run returns the same
ids and pass counts.  At most two decisions per case, and 3% over all, may be
near-tie decisions that differ from the oracle's.
"""
import numpy as np
import pytest

from _parity import Tally, custom_problem, make_refiner, run_device, upload

STRESS = dict(W_e=1.0, W_r=0.3, L=0.3, W_in=0.08, W_1=0.08, W_2=0.06)
N_CASES = 128
_TOTAL = Tally()


def _say(*a):
    print(*a, flush=True)


def draw_case(i):
    """The configuration of case i (a pure function of i)."""
    g = np.random.default_rng(0xC0FFEE + 7919 * i)
    dtype = "bf16" if g.random() < 0.7 else "f32"
    H = int(g.choice([256, 512, 768, 1024, 1280, 2048]))
    V = int(g.choice([16, 17, 64, 255, 1000, 2047, 3001, 4099, 5000, 12007, 33001]))
    B = int(g.choice([1, 2, 5, 8, 13, 16, 24, 31, 32]))
    # batch sizes on both sides of the LM-head GEMM threshold and of the
    # many-position Read groups
    batch = int(g.choice([1, 2, 3, 4, 6, 9, 17, 24]))
    temp = str(g.choice(["greedy", "sample", "mixed"]))
    K = int(g.integers(0, 10))
    seed_given = bool(g.random() < 0.3)
    stress = bool(g.random() < 0.7)
    tau = top_k = top_p = None
    if temp != "greedy":
        if g.random() < 0.6:
            tau = [float(np.float32(t)) for t in g.uniform(0.3, 3.0, batch)]
        if g.random() < 0.4:
            top_k = [int(k) for k in g.choice([0, 1, 2, 5, 40, V - 1, V, V + 3], batch)]
        if g.random() < 0.4:
            top_p = [float(np.float32(p)) for p in g.choice([1.0, 0.95, 0.8, 0.5, 0.1], batch)]
    extra = int(g.choice([0, 0, 1, 7]))
    return dict(dtype=dtype, H=H, V=V, B=B, batch=batch, K=K, temp=temp, seed_given=seed_given,
                stress=stress, tau=tau, top_k=top_k, top_p=top_p, max_batch=batch + extra)


def test_draws_cover_every_path():
    """The drawn cases reach every element type, selection mode and batch
    path, and stay within the built sizes (host-side check of the table)."""
    cases = [draw_case(i) for i in range(N_CASES)]
    assert {c["dtype"] for c in cases} == {"f32", "bf16"}
    assert {c["temp"] for c in cases} == {"greedy", "sample", "mixed"}
    assert any(c["batch"] * c["B"] > 256 and c["dtype"] == "bf16" for c in cases)
    assert any(c["batch"] * c["B"] <= 16 for c in cases)
    assert any(c["batch"] == 1 for c in cases)
    assert any(c["seed_given"] for c in cases) and any(c["K"] == 0 for c in cases)
    assert any(c["top_k"] is not None or c["top_p"] is not None for c in cases)
    for c in cases:
        assert c["H"] % 256 == 0 and 16 <= c["V"] and 1 <= c["B"] <= 32
        assert c["max_batch"] * c["B"] <= 65536


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(N_CASES))
def test_random_case(i):
    c = draw_case(i)
    _say(f"case {i}: " + " ".join(f"{k}={v}" for k, v in c.items() if v is not None))
    prob = custom_problem(c["dtype"], H=c["H"], V=c["V"], B=c["B"], batch=c["batch"], K=c["K"],
                          sigmas=STRESS if c["stress"] else None, temp=c["temp"],
                          seed=1000 + i, seed_given=c["seed_given"], tau=c["tau"],
                          top_k=c["top_k"], top_p=c["top_p"])
    if not prob.inp.temp.any():
        # a "mixed" draw whose rows all came out greedy: the options of
        # sampled rows need sampled rows (the library rejects them otherwise)
        prob.tau = prob.top_k = prob.top_p = None
    ref = make_refiner(prob, max_batch=c["max_batch"])
    dev = upload(prob)
    from test_gpu_parity import _full_check
    run, tally = _full_check(prob, ref, dev, min_exact=0.0)
    assert tally.decisions - tally.exact <= 2, f"{tally.decisions - tally.exact} near-tie decisions"
    ee = run_device(ref, prob, dev, early_exit=True, write_logits=False)
    assert np.array_equal(ee.ids, run.ids) and np.array_equal(ee.iters, run.iters)
    assert ref.device_errors() == 0
    _TOTAL.add(tally)


@pytest.mark.gpu
def test_random_cases_exact_overall():
    if _TOTAL.seqs == 0:
        pytest.skip("no random case ran in this process")
    _say(f"overall: decisions={_TOTAL.decisions} exact={_TOTAL.exact} seqs={_TOTAL.seqs}")
    assert _TOTAL.exact >= 0.97 * _TOTAL.decisions
