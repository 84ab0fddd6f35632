#!/usr/bin/env python3
"""Throughput of the xPress refine + verify hot path on one MI355X.

One step = one xp_refine_block (base readout through the target LM head,
seed selection, K Jacobi passes of the refiner) plus one xp_verify_block over
a batch of synthetic draft blocks whose inputs are already resident in HBM.
The default workload is the largest one that fits one GPU: the Qwen3-8B shape
at batch 64 with blocks of 32 positions, rows alternating greedy and
temperature-1 sampling (H = 4096, V = 151936, r = 256, K = 6).  The same run
also measures the batch-1 (block 16, greedy) and batch-32 (block 16, greedy)
workloads briefly, for the LM-head kernel targets: the stream kernel against
the HBM peak at batch 1, the GEMM against the bf16 matrix peak at batch 32.

Prints one JSON line.  `value` is refined draft blocks per second; `roofline`
rates the dominant kernel, the LM-head launch (the stream kernel for one
16-position block, the GEMM for more), by its algorithmic bytes (HBM-bound
workloads) or flops (MFMA-bound ones, above the ridge) over its own duration,
measured with HIP events recorded by the library on the stream the kernel runs
on, against the published peak and against the peak measured on this GPU by
the library's probes (an HBM read stream, an MFMA loop); `cpu_baseline` times
the fp64 oracle on blocks of the workload for about 10 s (all threads), and
`cpu_baseline_1thread` on one block with one thread.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu] [--no-peaks]
    python bench.py --copy-probe BYTES      (a plain device copy, for counter scaling)
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "refined draft blocks/sec (refine+LM-head+verify), Qwen3-8B shape; % HBM/MFMA peak"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFS = 2517.0          # dense bf16 matrix peak of the MI355X
CSRC = os.path.join(ROOT, "paper_2608_02438_amd", "csrc")
# committed counter summaries of the LM-head kernel, per workload: (file, kernel sources)
GEMM_SRC = ("xp_gemm.hip", "xp_gemm_pipe.h")
TRAFFIC = {
    "qwen3-8b-bf16-B16-b1-greedy": ("k_lmhead_qwen3-8b-bf16-B16-b1_traffic.md", ("xp_lmhead.hip",)),
    "qwen3-8b-bf16-B16-b32-greedy": ("k_lmhead_gemm_qwen3-8b-bf16-B16-b32_traffic.md", GEMM_SRC),
    "qwen3-8b-bf16-B32-b64-mixed": ("k_lmhead_gemm_qwen3-8b-bf16-B32-b64_traffic.md", GEMM_SRC),
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash(srcs) -> str:
    """First 16 hex digits of the sha256 of the kernel's source files, concatenated."""
    h = hashlib.sha256()
    for src in srcs:
        h.update(open(os.path.join(CSRC, src), "rb").read())
    return h.hexdigest()[:16]


def committed_traffic(workload: str):
    """HBM bytes per LM-head launch from the committed counter summary of this
    workload, if it was taken on the current kernel source; otherwise None."""
    if workload not in TRAFFIC:
        return None
    fn, src = TRAFFIC[workload]
    path = os.path.join(ROOT, "profiles", fn)
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    m = re.search(r"source_sha256_16:\s*([0-9a-f]{16})", txt)
    t = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", txt)
    if not m or not t or m.group(1) != kernel_source_hash(src):
        return None
    return float(t.group(1))


def copy_probe(nbytes: int):
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": src.numel() * 4, "dispatches": 3}), flush=True)


def cpu_baseline(wl, weights, inp, min_seconds=10.0, threads=None):
    """The oracle, as it stands, on blocks of the workload (refine + verify of
    batch rows 0, 1, ... in turn) until at least `min_seconds` have passed;
    `threads` limits the BLAS pool (None: as configured)."""
    import contextlib

    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits

    import oracle as O
    limit = threadpool_limits(limits=threads) if threads else contextlib.nullcontext()
    with limit:
        used = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
        P = O.Params.from_arrays(weights)          # the fp64 widening, before the window
        t0 = time.perf_counter()
        n = 0
        while True:
            b = n % wl.batch
            sl = slice(b, b + 1)
            res = O.refine_batch(P, inp.h[sl], inp.anchor[sl], inp.temp[sl], inp.u_draft[sl], wl.K,
                                 seed_ids=None if inp.seed_ids is None else inp.seed_ids[sl],
                                 early_exit=False)
            r0 = res.refined[0]
            if inp.temp[b]:
                O.verify_sample(r0.logits, r0.ids, inp.target_logits[b].astype(np.float64),
                                inp.r_accept[b], float(inp.u_res[b]))
            else:
                O.verify_greedy(r0.ids, inp.target_ids(r0.ids[None, :])[0])
            n += 1
            dt = time.perf_counter() - t0
            if dt >= min_seconds:
                break
    return {"value": n / dt, "unit": "blocks/s", "cores": int(used), "kind": "oracle",
            "sample": f"{n} block(s) of {wl.name} (batch rows in turn): fp64 base readout, "
                      f"{wl.K} Jacobi passes and verification, {dt:.1f} s (the refiner "
                      f"weights widened to fp64 beforehand; the LM head is widened chunk by "
                      f"chunk inside the readout, as the oracle does)",
            "cpu_model": _cpu_model()}


def _cpu_model():
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def measured_peaks(lib_probe_read, lib_probe_mfma):
    """What this GPU delivers on the two resources: HBM read bandwidth (a 2 GiB
    stream, best of three launch shapes) and the bf16 MFMA rate on random
    operands (8 independent 32x32x16 chains per wave, 2048 workgroups)."""
    import numpy as np
    import torch

    def timed(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / reps

    nbytes = 2 << 30
    buf = torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), dtype=torch.int32, device="cuda")
    out = torch.zeros(1, dtype=torch.int32, device="cuda")
    gbs = max(nbytes / timed(lambda: lib_probe_read(buf, out, wgs)) / 1e9
              for wgs in (1024, 2048, 4096))
    del buf
    rng = np.random.default_rng(0)
    x = rng.standard_normal((8, 64, 2, 8)).astype(np.float32)
    bits = ((x.view(np.uint32).astype(np.uint64) + 0x7FFF + ((x.view(np.uint32) >> 16) & 1))
            >> 16).astype(np.uint16)
    ops = torch.from_numpy(bits.view(np.int16)).cuda()
    wgs, iters = 2048, 2000
    mout = torch.empty(wgs * 4 * 64 * 16, dtype=torch.float32, device="cuda")
    t = timed(lambda: lib_probe_mfma(ops, wgs, iters, mout))
    tfs = wgs * 4 * iters * 8 * 32768 / t / 1e12
    return {"hbm_read_GBs": gbs, "mfma_bf16_TFs": tfs,
            "how": "xp_probe_hbm_read over 2 GiB (best of 1024/2048/4096 workgroups, each "
                   "streaming a contiguous range); xp_probe_mfma_bf16, 2048 workgroups x 4 "
                   "waves (2 per SIMD) x 8 chains x 2000 v_mfma_f32_32x32x16_bf16 on random "
                   "bf16 operands"}


def read_per_pass(wl, breakdown):
    """A7 (Read + Correct + the select partials) per launch, from the stage
    events of the breakdown steps: algorithmic bytes W_r once, s once, z once;
    flops 2 M r V."""
    ms, n = breakdown["read"]
    if n == 0:
        return None
    us = ms * 1e3 / n
    es = 2 if wl.dtype == "bf16" else 4
    M = wl.batch * wl.B
    nbytes = wl.V * wl.r * es + M * wl.V * 4 + M * wl.r * es
    flops = 2.0 * M * wl.r * wl.V
    gbs = nbytes / (us * 1e-6) / 1e9
    return {"launch_us": us, "launches": n, "algorithmic_bytes": nbytes, "GB_s": gbs,
            "frac_hbm_peak": gbs / HBM_PEAK_GBS, "TFLOP_s": flops / (us * 1e-6) / 1e12}


class Setup:
    """A workload's inputs resident in HBM, its handle, and one step (refine +
    verify over the batch)."""

    def __init__(self, wl):
        import torch

        import synth
        from paper_2608_02438_amd.xpress import device_tensor, refiner_from_arrays
        self.wl = wl
        log(f"[bench] workload {wl.name}: generating inputs")
        self.weights = synth.make_weights(wl)
        self.inp = inp = synth.make_inputs(wl)
        log("[bench] uploading and creating the handle")
        self.ref = refiner_from_arrays(self.weights, wl.H, wl.r, wl.V, wl.B, wl.batch)
        self.hid = device_tensor(inp.h)
        self.anchor = device_tensor(inp.anchor)
        self.seed = device_tensor(inp.seed_ids) if inp.seed_ids is not None else None
        sample_rows = bool(inp.temp.any())
        self.temp = device_tensor(inp.temp) if sample_rows else None
        self.u_draft = device_tensor(inp.u_draft) if sample_rows else None
        self.tl = device_tensor(inp.target_logits) if sample_rows else None
        self.r_acc = device_tensor(inp.r_accept)
        self.u_res = device_tensor(inp.u_res)
        self.out = self.ref.refine_block(self.hid, self.anchor, seed_ids=self.seed, temp=self.temp,
                                         u_draft=self.u_draft, K=wl.K)
        torch.cuda.synchronize()
        # greedy targets are built around the refined block (fixed by the inputs)
        self.tids = device_tensor(inp.target_ids(self.out.ids.cpu().numpy()))
        self.vout = self.ref.verify_block(self.out.ids, self.tids, temp=self.temp,
                                          target_logits=self.tl, r_accept=self.r_acc,
                                          u_resample=self.u_res)

    def step(self, K=None, early_exit=False):
        self.ref.refine_block(self.hid, self.anchor, seed_ids=self.seed, temp=self.temp,
                              u_draft=self.u_draft, K=self.wl.K if K is None else K,
                              early_exit=early_exit, out=self.out)
        self.ref.verify_block(self.out.ids, self.tids, temp=self.temp, target_logits=self.tl,
                              r_accept=self.r_acc, u_resample=self.u_res, out=self.vout)

    def close(self):
        self.ref.close()


def lm_roofline(wl, lm_us):
    """Roofline of one LM-head launch of duration lm_us: algorithmic bytes
    W_lm once, h once, s written once; algorithmic flops 2 M V H.  The launch
    is HBM-bound below the ridge (peak flops / peak bytes, about 315 flop/B)
    and MFMA-bound above it."""
    M = wl.batch * wl.B
    es = 2 if wl.dtype == "bf16" else 4
    lm_bytes = wl.V * wl.H * es + M * wl.H * es + M * wl.V * 4
    lm_flops = 2.0 * M * wl.V * wl.H
    mfma_bound = wl.dtype == "bf16" and lm_flops / lm_bytes > MFMA_BF16_PEAK_TFS * 1e3 / HBM_PEAK_GBS
    if mfma_bound:
        achieved = lm_flops / (lm_us * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK_TFS,
                "unit": "TFLOP/s", "frac": achieved / MFMA_BF16_PEAK_TFS,
                "kernel": "k_lmhead_gemm (base readout s = W_lm h, GEMM + selection)",
                "algorithmic_flops_per_launch": lm_flops}
    else:
        achieved = lm_bytes / (lm_us * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS,
                "kernel": "k_lmhead_sk (base readout s = W_lm h, stream + selection)"
                          if M <= 16 else
                          "k_lmhead_gemm (base readout s = W_lm h, GEMM + selection)"}
    roof.update({"traffic": committed_traffic(wl.name), "algorithmic_bytes_per_launch": lm_bytes,
                 "launch_us": lm_us})
    return roof


def timed_steps(st, steps):
    """Time exactly `steps` steps between two synchronizations; the LM-head
    launch carries an event pair recorded by the library on its stream.
    Returns (elapsed s, LM-head us per launch, per-round ms per step)."""
    import torch
    st.ref.timing_enable(("lmhead",), capacity=max(steps, 1))
    torch.cuda.synchronize()
    # up to 5 rounds of equal length inside the timed steps, each bracketed by
    # events on the stream the steps run on (the mean of the rounds and the
    # fastest are reported beside the wall-clock figure)
    nr = min(5, steps)
    bounds = [steps * i // nr for i in range(nr + 1)]
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(nr + 1)]
    t0 = time.perf_counter()
    for i in range(steps):
        if i in bounds:
            evs[bounds.index(i)].record()
        st.step()
    evs[nr].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    rounds = [evs[j].elapsed_time(evs[j + 1]) / (bounds[j + 1] - bounds[j]) for j in range(nr)]
    tm = st.ref.timing_read()
    st.ref.timing_enable((), 1)
    lm_ms, lm_n = tm["lmhead"]
    return t1 - t0, lm_ms * 1e3 / max(lm_n, 1), rounds


def secondary(wl, steps, warmup):
    """A short measurement of another workload in the same run: blocks/s and
    its LM-head launch against its own roofline."""
    st = Setup(wl)
    for _ in range(warmup):
        st.step()
    elapsed, lm_us, rounds = timed_steps(st, steps)
    st.close()
    roof = lm_roofline(wl, lm_us)
    log(f"[bench] {wl.name}: {elapsed * 1e3 / steps:.3f} ms/step, LM head {lm_us:.1f} us "
        f"({roof['achieved']:.0f} {roof['unit']}, {100 * roof['frac']:.1f}% of peak)")
    return {"workload": wl.name, "steps": steps, "ms_per_step": elapsed * 1e3 / steps,
            "blocks_per_s": wl.batch * steps / elapsed, "roofline": roof,
            "ms_per_step_rounds_min": min(rounds)}


def k_sweep(args, st):
    """Cost of K Jacobi passes (the latency-vs-K table of the paper's evaluation):
    ms per refine + verify at fixed K and with the early exit, the mean number of
    passes the early exit runs, and the share of sequences at a fixed point."""
    import numpy as np
    import torch
    wl = st.wl
    rows = []
    for K in range(1, 9):
        for early in (False, True):
            for _ in range(max(args.warmup, 2)):
                st.step(K, early)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(args.steps):
                st.step(K, early)
            torch.cuda.synchronize()
            dt = (time.perf_counter() - t0) / args.steps
            it = st.out.iters.cpu().numpy()
            rows.append({"K": K, "early_exit": early, "ms_per_step": dt * 1e3,
                         "blocks_per_s": wl.batch / dt, "iters_mean": float(np.mean(it)),
                         "fixed_point_before_K": float(np.mean(it < K))})
            log(f"[k-sweep] K={K} early_exit={early}: {dt * 1e3:.3f} ms/step, "
                f"iters {np.mean(it):.2f}")
    print(json.dumps({"k_sweep": rows, "workload": wl.name, "batch": wl.batch, "block": wl.B,
                      "steps": args.steps, "data": "synthetic"}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="qwen3-8b-bf16-B32-b64-mixed")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the measured HBM and MFMA peaks")
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the batch-1 and batch-32 LM-head measurements")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES")
    ap.add_argument("--layer", action="store_true",
                    help="time the context layer (the Qwen3-8B decoder layer over the block "
                         "and its context KV) on the workload's shapes and print that line "
                         "instead")
    ap.add_argument("--k-sweep", action="store_true",
                    help="time refine + verify for K = 1..8 passes, fixed K and with the "
                         "early exit, and print that table as one JSON line instead")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this path runs on one GPU; multi-GPU runs are not part of it "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE {world}).", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return

    import numpy as np
    import torch

    import synth

    wl = synth.BY_NAME[args.workload]
    if args.layer:
        layer_bench(args, wl)
        return
    st = Setup(wl)
    if args.k_sweep:
        k_sweep(args, st)
        st.close()
        return

    log(f"[bench] warmup {args.warmup}")
    for _ in range(args.warmup):
        st.step()
    torch.cuda.synchronize()

    # per-stage breakdown (all stages timed), outside the measured region
    st.ref.timing_enable(("prep", "lmhead", "select", "rspace", "read", "verify"), capacity=4096)
    for _ in range(3):
        st.step()
    breakdown = st.ref.timing_read()

    log(f"[bench] timing {args.steps} steps")
    elapsed, lm_us, rounds = timed_steps(st, args.steps)
    ms_step = elapsed * 1e3 / args.steps
    blocks_s = wl.batch * args.steps / elapsed
    roof = lm_roofline(wl, lm_us)
    achieved = roof["achieved"]
    if not args.no_peaks:
        from paper_2608_02438_amd.xpress import probe_hbm_read, probe_mfma_bf16
        log("[bench] measured peaks (HBM read stream, MFMA loop)")
        mp = measured_peaks(probe_hbm_read, probe_mfma_bf16)
        peak = mp["mfma_bf16_TFs"] if roof["bound"] == "mfma" else mp["hbm_read_GBs"]
        roof.update({"measured_peak": peak, "frac_of_measured": achieved / peak,
                     "measured_peaks": mp})
    n_acc = st.vout[0].cpu().numpy()
    log(f"[bench] {ms_step:.3f} ms/step, LM head {lm_us:.1f} us "
        f"({achieved:.0f} {roof['unit']}, {100 * roof['frac']:.1f}% of peak)")
    st.close()

    line = {
        "metric": METRIC, "value": blocks_s, "unit": "blocks/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic: seeded N(0,0.02^2) bf16 weights of the Qwen3-8B-shaped LM head and "
                "rank-256 refiner, N(0,1) drafter hidden states, uniform anchors",
        "config": {"workload": wl.name, "batch": wl.batch, "block": wl.B, "K": wl.K,
                   "H": wl.H, "V": wl.V, "r": wl.r, "temperature": wl.temp},
        "roofline": roof,
        "refined_tokens_per_s": blocks_s * wl.B,
        "stage_ms_per_step": {k: v[0] / 3 for k, v in breakdown.items()},
        "read_per_pass": read_per_pass(wl, breakdown),
        "rounds_ms_per_step": rounds,
        "ms_per_step_rounds_mean": sum(rounds) / len(rounds),
        "ms_per_step_rounds_min": min(rounds),
        "accepted_mean": float(np.mean(n_acc)),
        # tokens committed per second (accepted draft tokens plus the
        # correction or bonus token of each sequence): context only, the
        # synthetic targets fix the acceptance
        "committed_tokens_per_s": float(np.sum(n_acc + 1)) * args.steps / elapsed,
    }
    if not args.no_secondary and args.workload == "qwen3-8b-bf16-B32-b64-mixed":
        # the two kernel targets: the LM-head stream at batch 1 against HBM,
        # the LM-head GEMM at batch 32 against the bf16 matrix peak
        sec = {}
        for name in ("qwen3-8b-bf16-B16-b1-greedy", "qwen3-8b-bf16-B16-b32-greedy"):
            sec[name] = secondary(synth.BY_NAME[name], 20, 5)
        line["secondary"] = sec
        line["lmhead_hbm_frac_batch1"] = sec["qwen3-8b-bf16-B16-b1-greedy"]["roofline"]["frac"]
        line["lmhead_mfma_frac_batch32"] = sec["qwen3-8b-bf16-B16-b32-greedy"]["roofline"]["frac"]
    if not args.no_cpu:
        log("[bench] CPU oracle baseline (all threads)")
        line["cpu_baseline"] = cpu_baseline(wl, st.weights, st.inp)
        log("[bench] CPU oracle baseline (one thread)")
        line["cpu_baseline_1thread"] = cpu_baseline(wl, st.weights, st.inp, min_seconds=0.0,
                                                    threads=1)
    else:
        line["cpu_baseline"] = None
    print(json.dumps(line), flush=True)


LAYER_METRIC = ("context-layer forwards/sec (Qwen3-8B decoder layer over the drafted block "
                "and its context KV); % HBM peak")


def layer_bench(args, wl):
    """One step = one xp_layer_forward over the workload's batch of blocks with
    its context lengths.  The forward streams every weight once (it is
    HBM-bound at these position counts), so the roofline is the forward's
    algorithmic bytes (weights, the context K and V it reads, its inputs and
    outputs) over its time, against the HBM peak."""
    import numpy as np
    import torch

    import synth
    from paper_2608_02438_amd.xpress import LAYER_WEIGHT_NAMES, Layer, device_tensor

    log(f"[bench] context layer, workload {wl.name}: generating weights and the KV cache")
    weights = synth.make_layer_weights(wl)
    inp = synth.make_layer_inputs(wl)
    dw = {n: device_tensor(weights[n]) for n in LAYER_WEIGHT_NAMES}
    C_max = inp.k_cache.shape[1]
    layer = Layer(dw, wl.H, wl.n_heads, wl.n_kv_heads, wl.ffn, max_batch=wl.batch, max_B=wl.B,
                  max_ctx=C_max)
    x, kc, vc, cl = (device_tensor(a) for a in (inp.x, inp.k_cache, inp.v_cache, inp.ctx_len))
    M = wl.batch * wl.B
    h32 = torch.empty((wl.batch, wl.B, wl.H), dtype=torch.float32, device="cuda")
    hb = torch.empty((wl.batch, wl.B, wl.H), dtype=torch.bfloat16, device="cuda")
    for _ in range(args.warmup):
        layer.forward(x, kc, vc, cl, h_f32=h32, h_bf16=hb)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        layer.forward(x, kc, vc, cl, h_f32=h32, h_bf16=hb)
    e1.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / args.steps
    wbytes = sum(int(weights[n].size) * 2 for n in LAYER_WEIGHT_NAMES)
    kvbytes = int(np.sum(inp.ctx_len)) * wl.n_kv_heads * wl.head_dim * 2 * 2
    iobytes = M * wl.H * (2 + 4 + 2)
    nbytes = wbytes + kvbytes + iobytes
    gbs = nbytes / (ms * 1e-3) / 1e9
    log(f"[bench] layer {ms * 1e3:.1f} us per forward, {gbs:.0f} GB/s "
        f"({100 * gbs / HBM_PEAK_GBS:.1f}% of the HBM peak)")
    line = {
        "metric": LAYER_METRIC, "value": 1e3 / ms, "unit": "forwards/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: seeded N(0,0.02^2) bf16 projections, norm weights 1+N(0,0.1^2), "
                "N(0,1) hidden states and context K/V",
        "config": {"workload": wl.name + "+context-layer", "batch": wl.batch, "block": wl.B,
                   "H": wl.H, "heads": wl.n_heads, "kv_heads": wl.n_kv_heads,
                   "head_dim": wl.head_dim, "ffn": wl.ffn,
                   "ctx_len": [int(c) for c in inp.ctx_len[:8]]},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "xp_layer_forward (all of its kernels)",
                     "algorithmic_bytes_per_launch": nbytes, "weight_bytes": wbytes,
                     "kv_bytes": kvbytes, "launch_us": ms * 1e3},
        "wall_s": elapsed,
    }
    if not args.no_cpu:
        import oracle as O
        log("[bench] CPU oracle baseline of the layer (one block, all threads)")
        P = O.layer_ref.LayerParams.from_arrays(weights, wl.n_heads, wl.n_kv_heads, wl.head_dim)
        t = time.perf_counter()
        O.layer_ref.layer_forward(P, inp.x[:1], inp.k_cache[:1], inp.v_cache[:1],
                                  inp.ctx_len[:1])
        dt = time.perf_counter() - t
        line["cpu_baseline"] = {"value": 1.0 / dt, "unit": "blocks/s", "kind": "oracle",
                                "cores": os.cpu_count(),
                                "sample": "one block of the workload through the fp64 layer "
                                          "oracle (weights already widened)"}
    else:
        line["cpu_baseline"] = None
    layer.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
