"""The Toeplitz form of Mix (remark after Proposition 1) on the device, through
the C ABI (needs an MI355X): the mixer written from kernel taps equals the
oracle's, bit for bit, and a handle created from it refines and verifies as
the fp64 oracle does with the same mixer."""
import numpy as np
import pytest

import oracle as O
from synth import gen

from _parity import check_refine, check_verify, custom_problem, run_device, upload

pytestmark = pytest.mark.gpu

STRESS = dict(W_e=1.0, W_r=0.3, L=0.3, W_in=0.08, W_1=0.08, W_2=0.06)


def _say(*a):
    print(*a, flush=True)


def _taps(dtype, r, B, sigma, seed):
    f = np.random.default_rng(seed).normal(0.0, sigma, size=(r, B)).astype(np.float32)
    return gen.f32_to_bf16_bits(f) if dtype == "bf16" else f


def _host(t):
    import torch
    t = t.cpu()
    return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("r,B", [(256, 16), (256, 32), (256, 1), (3, 7)])
def test_toeplitz_mixer_matches_oracle_bit_for_bit(dtype, r, B):
    import torch
    from paper_2608_02438_amd.xpress import device_tensor, toeplitz_mixer
    _say(f"case: toeplitz mixer {dtype} r={r} B={B}")
    kappa = _taps(dtype, r, B, 1.0, seed=r * 100 + B)
    out = toeplitz_mixer(device_tensor(kappa))
    torch.cuda.synchronize()
    assert np.array_equal(_host(out), O.toeplitz_mixer(kappa))     # copies and zeros


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_refine_and_verify_with_a_toeplitz_mixer(dtype):
    import torch
    from paper_2608_02438_amd.xpress import WEIGHT_NAMES, Refiner, device_tensor, toeplitz_mixer
    _say(f"case: toeplitz refine {dtype} H=256 V=777 B=8 batch=4 K=8 mixed rows")
    prob = custom_problem(dtype, H=256, V=777, B=8, batch=4, K=8, sigmas=STRESS, temp="mixed",
                          seed=11)
    kappa = _taps(dtype, 256, prob.B, STRESS["L"], seed=5)
    prob.weights["L"] = O.toeplitz_mixer(kappa)                    # what the oracle reads
    dw = {n: device_tensor(prob.weights[n]) for n in WEIGHT_NAMES if n != "L"}
    dw["L"] = toeplitz_mixer(device_tensor(kappa))                  # what the device reads
    torch.cuda.synchronize()
    ref = Refiner(dw, prob.H, prob.r, prob.V, prob.B, prob.batch)
    dev = upload(prob)
    run = run_device(ref, prob, dev)
    tally, finals = check_refine(prob, run)
    _say(f"  decisions={tally.decisions} exact={tally.exact} excused={tally.excused} "
         f"iters={run.iters.tolist()}")
    assert tally.exact >= 0.97 * tally.decisions
    assert run.iters.max() >= 2, "stress weights should need more than one pass"
    target_ids = prob.inp.target_ids(run.ids)
    n, nx = ref.verify_block(torch.from_numpy(run.ids).cuda(), device_tensor(target_ids),
                             temp=dev["temp"], target_logits=dev["target_logits"],
                             r_accept=dev["r_accept"], u_resample=dev["u_res"])
    torch.cuda.synchronize()
    exc = check_verify(prob, run, finals, n.cpu().numpy(), nx.cpu().numpy(), target_ids,
                       list(range(prob.batch)))
    _say(f"  verify: n={n.cpu().numpy().tolist()} excused={exc}")
    ref.close()
