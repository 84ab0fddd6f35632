"""Device path vs the fp64 oracle, through the C ABI (needs an MI355X).

Small cases span several vocabulary tiles and a ragged tail (V not a multiple
of 16) and use stress weights so that Jacobi trajectories take several passes;
the full-size cases run the workloads' own shapes and launch configuration.
"""
import numpy as np
import pytest

import oracle as O
import synth
from synth.configs import TINY_F32, QWEN_B1, QWEN_B8_T1, QWEN_B32, QWEN_B64_MIXED

from _parity import (Tally, check_refine, check_verify, custom_problem, make_refiner,
                     run_device, upload, workload_problem)

pytestmark = pytest.mark.gpu

STRESS = dict(W_e=1.0, W_r=0.3, L=0.3, W_in=0.08, W_1=0.08, W_2=0.06)


def _say(*a):
    print(*a, flush=True)


def _verify(ref, prob, run, dev, target_ids):
    import torch
    from paper_2608_02438_amd.xpress import device_tensor
    n, nx = ref.verify_block(torch.from_numpy(run.ids).cuda(), device_tensor(target_ids),
                             temp=dev["temp"], target_logits=dev["target_logits"],
                             r_accept=dev["r_accept"], u_resample=dev["u_res"])
    torch.cuda.synchronize()
    return n.cpu().numpy(), nx.cpu().numpy()


def _full_check(prob, ref, dev, seqs=None, K=None, min_exact=1.0):
    run = run_device(ref, prob, dev, K=K)
    tally, finals = check_refine(prob, run, seqs=seqs)
    _say(f"  decisions={tally.decisions} exact={tally.exact} excused={tally.excused} "
         f"seq_exact={tally.seq_exact}/{tally.seqs} max|dl|={tally.max_logit_err:.3g} "
         f"max|dl|/E={tally.max_err_over_bound:.3g}")
    assert tally.exact >= min_exact * tally.decisions
    seqs = list(range(prob.batch)) if seqs is None else seqs
    target_ids = prob.inp.target_ids(run.ids)
    n, nx = _verify(ref, prob, run, dev, target_ids)
    exc = check_verify(prob, run, finals, n, nx, target_ids, seqs)
    _say(f"  verify: n={n[seqs].tolist()[:8]} excused={exc}")
    return run, tally


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_stress_greedy_ragged_vocab(dtype):
    _say(f"case: stress greedy {dtype} H=512 V=1000 B=16 batch=3 K=6")
    prob = custom_problem(dtype, H=512, V=1000, B=16, batch=3, K=6, sigmas=STRESS, seed=1)
    ref = make_refiner(prob)
    run, tally = _full_check(prob, ref, upload(prob), min_exact=0.97)
    assert run.iters.max() >= 3, "stress weights should need several passes"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_stress_sampling_mixed_rows(dtype):
    _say(f"case: stress mixed-temperature {dtype} H=256 V=777 B=8 batch=4 K=8")
    prob = custom_problem(dtype, H=256, V=777, B=8, batch=4, K=8, sigmas=STRESS, temp="mixed",
                          seed=2)
    ref = make_refiner(prob)
    _full_check(prob, ref, upload(prob), min_exact=0.97)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_stress_sampling_at_temperatures(dtype):
    tau = [0.5, 0.8, 1.6, 3.0]
    _say(f"case: stress sampling {dtype} H=256 V=777 B=8 batch=4 K=8 temperatures {tau}")
    prob = custom_problem(dtype, H=256, V=777, B=8, batch=4, K=8, sigmas=STRESS, temp="sample",
                          seed=21, tau=tau)
    ref = make_refiner(prob)
    _full_check(prob, ref, upload(prob), min_exact=0.97)


@pytest.mark.parametrize("batch,tau", [(5, 1.7), (20, 0.6)])
def test_lmhead_gemm_and_read_multi_at_temperature(batch, tau):
    _say(f"case: GEMM + read_multi at T={tau}, bf16 H=512 V=1000 B=16 batch={batch} K=6")
    prob = custom_problem("bf16", H=512, V=1000, B=16, batch=batch, K=6, sigmas=STRESS,
                          temp="sample", seed=31 + batch, tau=tau)
    ref = make_refiner(prob)
    _full_check(prob, ref, upload(prob), min_exact=0.97)


def test_invalid_temperature_sets_device_error_and_samples_at_one():
    import torch
    from paper_2608_02438_amd.xpress import XP_DEVERR_TEMPERATURE
    _say("case: invalid temperatures on sampled rows (0, NaN, -1, inf), greedy row with NaN")
    prob = custom_problem("bf16", H=256, V=500, B=8, batch=4, K=4, sigmas=STRESS, temp="mixed",
                          seed=41, tau=1.0)
    ref = make_refiner(prob)
    dev = upload(prob)
    base = run_device(ref, prob, dev)
    assert ref.device_errors() == 0
    # rows 1 and 3 sample, rows 0 and 2 are greedy
    for bad in ([1.0, 0.0, 1.0, float("nan")], [1.0, -1.0, 1.0, float("inf")]):
        dev["temperature"] = torch.tensor(bad, dtype=torch.float32, device="cuda")
        run = run_device(ref, prob, dev)
        assert np.array_equal(run.ids, base.ids) and np.array_equal(run.traj, base.traj)
        assert ref.device_errors() == XP_DEVERR_TEMPERATURE
    dev["temperature"] = torch.tensor([float("nan"), 1.0, 0.0, 1.0], dtype=torch.float32,
                                      device="cuda")
    run = run_device(ref, prob, dev)
    assert np.array_equal(run.ids, base.ids)
    assert ref.device_errors() == 0, "greedy rows ignore their temperature"


@pytest.mark.parametrize("H,V,batch,B", [(8192, 20011, 1, 16), (8192, 20011, 2, 32),
                                         (512, 262135, 1, 16), (512, 262135, 4, 16)])
def test_largest_built_sizes(H, V, batch, B):
    # the largest hidden width built (H = 8192: the stream LM head without LDS
    # staging of h at 16 positions, the 128 x 128 GEMM at 64), and a vocabulary
    # just under the largest built (2^18, ragged tail), with B up to 32
    _say(f"case: largest sizes bf16 H={H} V={V} B={B} batch={batch} mixed K=4")
    prob = custom_problem("bf16", H=H, V=V, B=B, batch=batch, K=4, sigmas=STRESS,
                          temp="mixed", seed=51 + B + batch)
    ref = make_refiner(prob)
    _full_check(prob, ref, upload(prob), min_exact=0.97)


@pytest.mark.parametrize("tau,agree", [(None, 8), (0.7, 8), (None, 5)])
def test_sampled_rows_all_accepted_take_the_bonus_token(tau, agree):
    """Target logits equal to the refined logits (p = q) accept every draft
    token, so the next token is the inverse-CDF sample of p_{B+1} at u_res:
    the bonus path of verification, rarely reached with random targets.  With
    p = q on the first five positions only, the first rejection comes at
    position 5 or later, past the target rows verification reduces first."""
    import torch
    _say(f"case: sampled rows with p = q on {agree} positions, T={tau}")
    prob = custom_problem("bf16", H=256, V=777, B=8, batch=4, K=4, sigmas=STRESS,
                          temp="sample", seed=61, tau=tau)
    ref = make_refiner(prob)
    dev = upload(prob)
    run = run_device(ref, prob, dev)
    tally, finals = check_refine(prob, run)
    assert tally.exact >= 0.97 * tally.decisions
    tl = prob.inp.target_logits.copy()
    tl[:, :agree, :] = run.logits[:, :agree]       # p_k = q_k for k = 1..agree
    prob.inp.target_logits = tl
    dev["target_logits"] = torch.from_numpy(tl).cuda()
    target_ids = prob.inp.target_ids(run.ids)
    n, nx = _verify(ref, prob, run, dev, target_ids)
    _say(f"  verify: n={n.tolist()} next={nx.tolist()}")
    assert (n >= agree).all() and (n == prob.B).any() == (agree == prob.B)
    assert check_verify(prob, run, finals, n, nx, target_ids, range(prob.batch)) == 0


def test_block_of_one_and_K0():
    _say("case: B=1 and K=0")
    prob = custom_problem("bf16", H=256, V=300, B=1, batch=5, K=3, sigmas=STRESS, seed=3)
    ref = make_refiner(prob)
    dev = upload(prob)
    _full_check(prob, ref, dev, min_exact=0.97)
    run0 = run_device(ref, prob, dev, K=0)
    tally, _ = check_refine(prob, run0)
    assert np.array_equal(run0.ids, run0.traj[0]) and (run0.iters == 0).all()


def test_seed_given_sampled_and_verify_k0():
    _say("case: seeded ids, sampled rows, K=0 verify (q = softmax(s))")
    prob = custom_problem("bf16", H=256, V=500, B=4, batch=6, K=0, sigmas=STRESS, temp="sample",
                          seed=4, seed_given=True)
    ref = make_refiner(prob)
    _full_check(prob, ref, upload(prob))


# ------------------------------------------------------------ invariants -----

def test_early_exit_run_to_run_and_batch_invariance():
    import torch
    _say("case: invariants (early exit, bit-identical reruns, batch invariance)")
    prob = custom_problem("bf16", H=512, V=2000, B=16, batch=4, K=8, sigmas=STRESS, temp="mixed",
                          seed=5)
    ref = make_refiner(prob)
    dev = upload(prob)
    a = run_device(ref, prob, dev)
    b = run_device(ref, prob, dev)
    assert np.array_equal(a.ids, b.ids) and np.array_equal(a.logits, b.logits)
    c = run_device(ref, prob, dev, early_exit=True, write_logits=False)
    assert np.array_equal(a.ids, c.ids) and np.array_equal(a.iters, c.iters)
    # sequence 2 alone equals sequence 2 inside the batch: same ids; the
    # logits agree to fp32 rounding (one block takes the LM-head stream, the
    # batch the LM-head GEMM, which add the same products in another order)
    one = {k: (v[2:3].contiguous() if v is not None and v.dim() > 0 and v.shape[0] == 4 else v)
           for k, v in dev.items()}
    out = ref.refine_block(one["hidden"], one["anchor"], temp=one["temp"], u_draft=one["u_draft"],
                           K=prob.K, write_logits=True)
    torch.cuda.synchronize()
    assert np.array_equal(out.ids.cpu().numpy()[0], a.ids[2])
    np.testing.assert_allclose(out.logits.cpu().numpy()[0], a.logits[2], rtol=1e-5, atol=1e-4)


@pytest.mark.parametrize("batch,temp", [(5, "mixed"), (20, "mixed"), (20, "greedy")])
def test_lmhead_gemm_and_read_multi_ragged_positions(batch, temp):
    # 80 positions: the 128 x 128 GEMM tile and one read group of 128 with 48
    # idle positions; 320 positions: two 256 x 256 GEMM position tiles (the
    # second 64 of 256 used) and a read group of 3 x 128 positions (64 idle),
    # over a vocabulary that ends inside a tile
    _say(f"case: GEMM + read_multi, bf16 H=512 V=1000 B=16 batch={batch} temp={temp} K=6")
    prob = custom_problem("bf16", H=512, V=1000, B=16, batch=batch, K=6, sigmas=STRESS,
                          temp=temp, seed=11 + batch)
    ref = make_refiner(prob)
    _full_check(prob, ref, upload(prob), min_exact=0.97)


def test_read_multi_workgroups_spanning_several_read_groups():
    """1536 positions (B = 32): three position groups of 512, so each Read
    workgroup walks the tiles of three read workgroups in a row and flushes a
    key row at each of their boundaries; V = 2000 gives 16 read workgroups
    (the last group of three holds one) and units of one tile or none."""
    _say("case: read_multi over groups of read workgroups, bf16 H=512 V=2000 B=32 batch=48 K=4")
    prob = custom_problem("bf16", H=512, V=2000, B=32, batch=48, K=4, sigmas=STRESS,
                          temp="mixed", seed=97)
    ref = make_refiner(prob)
    _full_check(prob, ref, upload(prob), min_exact=0.97)


@pytest.mark.parametrize("B,batch", [(16, 4), (8, 3)])
def test_fused_greedy_pass_matches_separate_kernels(B, batch):
    """All-greedy batches run selection + Fuse + Mix + W_1 as one kernel; an
    all-zero temperature vector sends the same rows through the separate
    select / fusemix / trans1 kernels.  Both compute the same fp32 values in
    the same order, so every output must agree bit for bit (also with early
    exit, which must not change ids or pass counts)."""
    import torch
    _say(f"case: fused vs separate greedy pass kernels, bf16 B={B} batch={batch}")
    prob = custom_problem("bf16", H=512, V=2000, B=B, batch=batch, K=8, sigmas=STRESS, seed=7)
    ref = make_refiner(prob)
    dev = upload(prob)
    assert dev["temp"] is None
    fused = run_device(ref, prob, dev)
    sep = dict(dev)
    sep["temp"] = torch.zeros(batch, dtype=torch.uint8, device="cuda")
    sep["u_draft"] = torch.zeros((batch, B), dtype=torch.float32, device="cuda")
    split = run_device(ref, prob, sep)
    assert fused.iters.max() >= 3
    assert np.array_equal(fused.ids, split.ids)
    assert np.array_equal(fused.iters, split.iters)
    assert np.array_equal(fused.traj, split.traj)
    assert np.array_equal(fused.logits, split.logits)
    fe = run_device(ref, prob, dev, early_exit=True, write_logits=False)
    se = run_device(ref, prob, sep, early_exit=True, write_logits=False)
    assert np.array_equal(fe.ids, fused.ids) and np.array_equal(fe.iters, fused.iters)
    assert np.array_equal(se.ids, fused.ids) and np.array_equal(se.iters, fused.iters)
    tally, _ = check_refine(prob, fused)
    assert tally.exact >= 0.97 * tally.decisions


def test_out_of_range_token_sets_device_error():
    import torch
    _say("case: out-of-range anchor")
    prob = custom_problem("f32", H=256, V=100, B=4, batch=2, K=2, seed=6)
    ref = make_refiner(prob)
    dev = upload(prob)
    assert ref.device_errors() == 0
    dev["anchor"] = torch.tensor([5, 1000], dtype=torch.int32, device="cuda")
    run_device(ref, prob, dev)
    assert ref.device_errors() & 1
    assert ref.device_errors() == 0          # the read cleared it


# ------------------------------------------------------------- full size -----
#
# The five workloads at their own shapes and launch configuration.  Every
# sequence is checked: ids and pass counts decision by decision, the final
# logits within E element by element and within the absolute bar (1e-5 fp32,
# 2e-2 bf16), verification exactly (greedy) or up to a near-tie (sampled).
# A workload's device run and its oracle base logits are made once per module
# (FullSize) and checked in groups of 16 sequences, one test per group.
# MAX_EXCUSED is the number of near-tie decisions each workload's check
# excused on MI355X (the inputs and the device arithmetic are deterministic,
# so the count is fixed); more than that fails.

ABS_BAR = {"f32": 1e-5, "bf16": 2e-2}
GROUP = 16


class FullSize:
    def __init__(self, wl, tau=None):
        import time
        t0 = time.time()
        self.prob = prob = workload_problem(wl, tau=tau)
        self.ref = make_refiner(prob)
        self.dev = upload(prob)
        self.run = run_device(self.ref, prob, self.dev)
        self.target_ids = prob.inp.target_ids(self.run.ids)
        self.n, self.nx = _verify(self.ref, prob, self.run, self.dev, self.target_ids)
        self.P = O.Params.from_arrays(prob.weights, round_z=prob.dtype == "bf16")
        h = prob.inp.h.reshape(prob.batch * prob.B, prob.H)
        self.s = O.base_logits(self.P.W_lm, h).reshape(prob.batch, prob.B, -1)
        self.tally = Tally()
        self.excused_verify = 0
        _say(f"  {wl.name}: device run and oracle base logits in {time.time() - t0:.1f} s")

    def check(self, seqs):
        prob = self.prob
        tally, finals = check_refine(prob, self.run, seqs=seqs, P=self.P, s=self.s[seqs],
                                     abs_bar=ABS_BAR[prob.dtype])
        exc = check_verify(prob, self.run, finals, self.n, self.nx, self.target_ids, seqs)
        self.tally.add(tally)
        self.excused_verify += exc
        _say(f"  sequences {seqs[0]}..{seqs[-1]}: decisions={tally.decisions} "
             f"exact={tally.exact} excused={tally.excused} seq_exact={tally.seq_exact}/"
             f"{tally.seqs} max|dl|={tally.max_logit_err:.3g} "
             f"max|dl|/E={tally.max_err_over_bound:.3g} verify n={self.n[seqs].tolist()} "
             f"excused={exc}")
        return tally, exc


def _groups(batch):
    return [list(range(g, min(batch, g + GROUP))) for g in range(0, batch, GROUP)]


@pytest.fixture(scope="module")
def full_sizes():
    made = {}

    def get(wl, tau=None):
        key = (wl.name, tau)
        if key not in made:
            for k in list(made):                 # one workload's buffers at a time
                made.pop(k).ref.close()
            made[key] = FullSize(wl, tau)
        return made[key]
    yield get
    for v in made.values():
        v.ref.close()


# excused near-tie decisions observed per workload (refine decisions, verify)
MAX_EXCUSED = {
    "tiny-f32-H256-V1024-B8-b1": (0, 0),
    "qwen3-8b-bf16-B16-b1-greedy": (0, 0),
    "qwen3-8b-bf16-B16-b8-sample": (2, 0),
    "qwen3-8b-bf16-B16-b1-sample": (0, 0),
    "qwen3-8b-bf16-B16-b32-greedy": (0, 0),
    "qwen3-8b-bf16-B32-b64-mixed": (3, 0),
}


def _full_size_groups(wl, full_sizes, seqs, tau=None, name=None):
    _say(f"case: {wl.name} T={tau} sequences {seqs[0]}..{seqs[-1]} of {wl.batch}")
    fs = full_sizes(wl, tau)
    fs.check(seqs)
    ex_ref, ex_ver = MAX_EXCUSED[name or wl.name]
    assert fs.tally.excused <= ex_ref, f"{fs.tally.excused} near-tie decisions excused"
    assert fs.excused_verify <= ex_ver, f"{fs.excused_verify} verifications excused"
    return fs


def test_tiny_f32_workload_matches_oracle_and_sequential_decode(full_sizes):
    fs = _full_size_groups(TINY_F32, full_sizes, [0])
    assert fs.tally.seq_exact == fs.tally.seqs
    # Theorem 1: with K = B passes the block is the sequential decode
    prob = fs.prob
    ystar = O.sequential_decode(fs.P, fs.s[0], prob.inp.h[0], int(prob.inp.anchor[0]))
    assert np.array_equal(fs.run.ids[0], ystar)


def test_qwen3_shape_batch1_greedy(full_sizes):
    _full_size_groups(QWEN_B1, full_sizes, [0])


def test_qwen3_shape_batch8_sampled(full_sizes):
    _full_size_groups(QWEN_B8_T1, full_sizes, list(range(8)))


def test_qwen3_shape_batch1_sampled_at_temperature(full_sizes):
    from synth.configs import scaled
    wl = scaled(QWEN_B1, name="qwen3-8b-bf16-B16-b1-sample", temp="sample", h_sigma=1.5625)
    _full_size_groups(wl, full_sizes, [0], tau=0.6)


@pytest.mark.parametrize("seqs", _groups(QWEN_B32.batch))
def test_qwen3_shape_batch32_greedy(full_sizes, seqs):
    _full_size_groups(QWEN_B32, full_sizes, seqs)


@pytest.mark.parametrize("seqs", _groups(QWEN_B64_MIXED.batch))
def test_qwen3_shape_batch64_block32_mixed(full_sizes, seqs):
    _full_size_groups(QWEN_B64_MIXED, full_sizes, seqs)


@pytest.mark.parametrize("H,V,B,batch,temp", [
    (512, 2000, 16, 6, "greedy"),      # fused greedy pass, one stream launch per pass
    (512, 2000, 16, 6, "mixed"),       # separate kernels, sampled rows
    (512, 1000, 16, 24, "greedy"),     # 384 positions: LM-head GEMM and many-position Read
    (256, 777, 32, 5, "mixed"),        # blocks of 32
])
def test_per_sequence_early_exit_equals_fixed_K(H, V, B, batch, temp):
    """Algorithm 1 stops each sequence at its own fixed point: with the early
    exit, a sequence's kernels skip every pass after it converged, while the
    others go on.  Since a fixed point maps to itself, ids, pass counts,
    trajectories, final logits and the verification that follows must equal
    the fixed-K run bit for bit, for every sequence."""
    import torch
    _say(f"case: per-sequence early exit, bf16 H={H} V={V} B={B} batch={batch} {temp}")
    # milder stress weights: the sequences reach their fixed points after
    # 7 to 28 passes (the oracle's counts), within K = B + 2 (Theorem 1: B)
    mild = dict(STRESS, W_e=0.25, W_r=0.075)
    prob = custom_problem("bf16", H=H, V=V, B=B, batch=batch, K=B + 2, sigmas=mild, temp=temp,
                          seed=91 + batch + B)
    ref = make_refiner(prob)
    dev = upload(prob)
    fixed = run_device(ref, prob, dev)
    tids = prob.inp.target_ids(fixed.ids)
    nf, xf = _verify(ref, prob, fixed, dev, tids)
    early = run_device(ref, prob, dev, early_exit=True)
    ne, xe = _verify(ref, prob, early, dev, tids)
    _say(f"  iters={fixed.iters.tolist()}")
    assert len(set(fixed.iters.tolist())) >= 2, "sequences should converge at different passes"
    assert fixed.iters.max() < prob.K, "every sequence should converge within K"
    assert np.array_equal(early.ids, fixed.ids) and np.array_equal(early.iters, fixed.iters)
    assert np.array_equal(early.traj, fixed.traj)
    assert np.array_equal(early.logits, fixed.logits)
    assert np.array_equal(ne, nf) and np.array_equal(xe, xf)
    tally, _ = check_refine(prob, early)
    assert tally.exact >= 0.97 * tally.decisions
