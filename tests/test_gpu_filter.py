"""Truncated (top-k / top-p) sampling on the device vs the fp64 oracle, through
the C ABI (needs an MI355X): refinement decision by decision, the final
logits within the bound, verification exactly or up to a near-tie, on the
stream kernels (one block), the GEMM / many-position Read (more), seeded
K = 0, the all-accepted bonus path, bad parameters, and the batch-8 Qwen3-8B
shape at top-k 50 and top-p 0.9."""
import numpy as np
import pytest

import oracle as O
from synth.configs import QWEN_B8_T1

from _parity import (check_refine, check_verify, custom_problem, make_refiner, run_device,
                     upload, workload_problem)

pytestmark = pytest.mark.gpu

STRESS = dict(W_e=1.0, W_r=0.3, L=0.3, W_in=0.08, W_1=0.08, W_2=0.06)
# per-sequence (top_k, top_p): none, top-k only, top-p only, both, top-1, a
# tiny top-p (one token), k >= V (none), and both on a greedy row (ignored)
KS = [0, 5, 0, 50, 1, 0, 5000, 7]
PS = [1.0, 1.0, 0.8, 0.9, 1.0, 1e-6, 1.0, 0.5]


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


def _check(prob, ref, dev, max_excused=0, K=None):
    run = run_device(ref, prob, dev, K=K)
    tally, finals = check_refine(prob, run)
    _say(f"  decisions={tally.decisions} exact={tally.exact} excused={tally.excused} "
         f"seq_exact={tally.seq_exact}/{tally.seqs} max|dl|={tally.max_logit_err:.3g}")
    target_ids = prob.inp.target_ids(run.ids)
    n, nx = _verify(ref, prob, run, dev, target_ids)
    exc = check_verify(prob, run, finals, n, nx, target_ids, range(prob.batch))
    _say(f"  verify: n={n.tolist()} next={nx.tolist()} excused={exc}")
    assert tally.excused + exc <= max_excused
    return run


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_truncated_sampling_stream_path(dtype):
    _say(f"case: truncated sampling {dtype} H=256 V=777 B=8 batch=8 K=8, (k, p) = "
         f"{list(zip(KS, PS))}, row 7 greedy")
    prob = custom_problem(dtype, H=256, V=777, B=8, batch=8, K=8, sigmas=STRESS, temp="sample",
                          seed=71, tau=[1.0, 0.7, 1.3, 1.0, 1.0, 1.0, 2.0, 1.0], top_k=KS,
                          top_p=PS)
    prob.inp.temp[7] = 0                       # a greedy row with truncation given: ignored
    ref = make_refiner(prob)
    run = _check(prob, ref, upload(prob))
    assert run.iters.max() >= 3


@pytest.mark.parametrize("batch", [5, 20])
def test_truncated_sampling_gemm_and_read_multi(batch):
    # 80 and 320 positions: the LM-head GEMM and the many-position Read
    ks = [(3 * b) % 60 for b in range(batch)]
    ps = [1.0 if b % 3 == 0 else 0.5 + (0.04 * b) % 0.5 for b in range(batch)]
    _say(f"case: truncated sampling bf16 H=512 V=1000 B=16 batch={batch} K=6 mixed rows")
    prob = custom_problem("bf16", H=512, V=1000, B=16, batch=batch, K=6, sigmas=STRESS,
                          temp="mixed", seed=73 + batch, top_k=ks, top_p=ps)
    ref = make_refiner(prob)
    _check(prob, ref, upload(prob))


def test_truncated_seeded_k0_and_logits():
    """Caller seed ids with K = 0: the seed is the block, and verification
    uses q = the truncated softmax of the base logits."""
    _say("case: truncated sampling with seeds, K=0")
    prob = custom_problem("bf16", H=256, V=500, B=4, batch=6, K=0, sigmas=STRESS, temp="sample",
                          seed=75, seed_given=True, top_k=[3, 0, 10, 1, 0, 40],
                          top_p=[1.0, 0.6, 0.9, 1.0, 0.2, 0.95])
    ref = make_refiner(prob)
    _check(prob, ref, upload(prob))


def test_truncated_bonus_token_when_all_accepted():
    """Target logits equal to the refined logits accept every draft token;
    the next token samples the truncated p_{B+1}."""
    import torch
    _say("case: truncated sampling, all accepted (p = q), bonus token")
    prob = custom_problem("bf16", H=256, V=777, B=8, batch=4, K=4, sigmas=STRESS, temp="sample",
                          seed=77, top_k=[5, 0, 20, 2], top_p=[1.0, 0.7, 0.9, 1.0])
    ref = make_refiner(prob)
    dev = upload(prob)
    run = run_device(ref, prob, dev)
    tally, finals = check_refine(prob, run)
    assert tally.excused == 0
    tl = prob.inp.target_logits.copy()
    tl[:, :prob.B, :] = run.logits
    prob.inp.target_logits = tl
    dev["target_logits"] = torch.from_numpy(tl).cuda()
    target_ids = prob.inp.target_ids(run.ids)
    n, nx = _verify(ref, prob, run, dev, target_ids)
    _say(f"  verify: n={n.tolist()} next={nx.tolist()}")
    assert (n == prob.B).all()
    assert check_verify(prob, run, finals, n, nx, target_ids, range(prob.batch)) == 0


def test_bad_truncation_parameters_set_the_device_error_and_mean_none():
    import torch
    from paper_2608_02438_amd.xpress import XP_DEVERR_FILTER
    _say("case: top_k < 0, top_p <= 0 / NaN on sampled rows")
    prob = custom_problem("bf16", H=256, V=500, B=8, batch=4, K=4, sigmas=STRESS, temp="sample",
                          seed=79)
    ref = make_refiner(prob)
    dev = upload(prob)
    base = run_device(ref, prob, dev)
    assert ref.device_errors() == 0
    dev["top_k"] = torch.tensor([-1, 0, 0, 0], dtype=torch.int32, device="cuda")
    dev["top_p"] = torch.tensor([1.0, 0.0, float("nan"), -0.5], dtype=torch.float32,
                                device="cuda")
    run = run_device(ref, prob, dev)
    assert np.array_equal(run.ids, base.ids) and np.array_equal(run.traj, base.traj)
    assert np.array_equal(run.logits, base.logits)
    assert ref.device_errors() == XP_DEVERR_FILTER


def test_truncated_early_exit_and_reruns_are_identical():
    _say("case: truncated sampling, early exit = fixed K, bit-identical reruns")
    prob = custom_problem("bf16", H=512, V=2000, B=16, batch=4, K=8, sigmas=STRESS,
                          temp="mixed", seed=81, top_k=[0, 30, 0, 100], top_p=[0.9, 1.0, 0.9, 0.8])
    ref = make_refiner(prob)
    dev = upload(prob)
    a = run_device(ref, prob, dev)
    b = run_device(ref, prob, dev)
    assert np.array_equal(a.ids, b.ids) and np.array_equal(a.logits, b.logits)
    c = run_device(ref, prob, dev, early_exit=True, write_logits=False)
    assert np.array_equal(a.ids, c.ids) and np.array_equal(a.iters, c.iters)
    tally, _ = check_refine(prob, a)
    assert tally.excused == 0


def test_qwen3_shape_batch8_top_k50_top_p09():
    _say("case: Qwen3-8B shape, batch 8, B=16, T=1, top-k 50, top-p 0.9, K=6")
    prob = workload_problem(QWEN_B8_T1, top_k=50, top_p=0.9)
    ref = make_refiner(prob)
    _check(prob, ref, upload(prob))
