"""Shared machinery of the GPU parity tests: build a problem, run the device
path through the C ABI, and check it against the oracle.

Exactness rules
  * token ids, iteration counts and acceptance lengths are integers: they must
    equal the oracle's, except where a decision is a near-tie that the device's
    fp32 arithmetic may legitimately resolve the other way;
  * a near-tie is judged against the oracle's own fp64 logits computed from the
    device's iterate (so one flipped token never excuses the rest of the block),
    with an element-wise bound E[k][v] on |l_device - l_exact|:
      greedy:  l[y_oracle] - l[y_device] <= E[y_oracle] + E[y_device];
      sampled: every weight e^(l - max) moves by a factor within e^(+-2 Emax), so
               the device token's CDF interval, widened by e^(+-4 Emax), must
               contain u (Emax = max_v E[k][v]);
  * E is not trusted blindly: the last pass's logits are compared element by
    element and must stay within E.

The bound E (fp32 unit roundoff u = 2^-24, probabilistic dot-product bound
lambda sqrt(n) u sum|terms| with lambda = 6, sum|w h| <= |w|_2 |h|_2):
    6 u sqrt(H) |W_lm[v]|_2 |h_k|_2           base readout s, H products
  + 6 u 16 (|W_r| |z_k|)[v]                    Read, r = 256 products
  + u |l[k][v]|                                final add and fp32 rounding
  + bf16: (|W_r| (c_k * ulp(z_k)))[v]           z elements whose fp64 value lies
          within 2^-16 |z| of a bf16 rounding midpoint may round the other way
          on the device (c = 1 there); every other z element rounds identically
    fp32: 2^-16 (|W_r| |z_k|)[v]                fp32 error of z itself
The 2^-16 relative budget for z covers the fp32 error of the stages that make
z (sums of up to H products); the device is far more accurate than that.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

import oracle as O
import synth
from synth import gen

U32 = 2.0 ** -24
Z_REL = 2.0 ** -16


@dataclass
class Problem:
    dtype: str
    H: int
    r: int
    V: int
    B: int
    batch: int
    K: int
    weights: dict
    inp: synth.Inputs
    seed_given: bool
    tau: np.ndarray | None = None       # [batch] float32 temperatures (None: 1)
    top_k: np.ndarray | None = None     # [batch] int32 top-k (None: no truncation)
    top_p: np.ndarray | None = None     # [batch] float32 top-p (None: no truncation)

    def T(self, b) -> float:
        return 1.0 if self.tau is None else float(self.tau[b])

    def filt(self, b):
        """(top_k, top_p) of sequence b as the device applies them: k outside
        [1, V) and p outside (0, 1) mean no truncation."""
        k = 0 if self.top_k is None else int(self.top_k[b])
        p = 1.0 if self.top_p is None else float(np.float32(self.top_p[b]))
        k = k if 0 < k < self.V else 0
        p = p if 0.0 < p < 1.0 else 1.0
        return k, p


def custom_problem(dtype, H, V, B, batch, K, sigmas=None, temp="greedy", seed=0,
                   seed_given=False, h_sigma=1.0, index=500, tau=None, top_k=None, top_p=None):
    """A problem with per-matrix weight scales (stress trajectories, ragged V)."""
    w = synth.scaled(synth.configs.QWEN_B1, index=index + seed, dtype=dtype, H=H, V=V, B=B,
                     batch=batch, K=K, temp=temp, h_sigma=h_sigma,
                     seed_mode="given" if seed_given else "base", p_match=0.6)
    sig = dict(W_lm=0.02, W_h=0.02, W_g=0.02, W_e=0.02, W_in=0.02, L=0.02, W_1=0.02, W_2=0.02,
               W_r=0.02)
    sig.update(sigmas or {})
    weights = {}
    for n, shape_fn in gen.WEIGHT_SHAPES.items():
        f = gen.normal_f32(w, n, shape_fn(w), sig[n])
        if n == "L":
            keep = np.tril(np.ones((B, B), bool), -1)
            f[:, ~keep] = 0.0
        weights[n] = gen.f32_to_bf16_bits(f) if dtype == "bf16" else f
    inp = synth.make_inputs(w)
    return Problem(dtype, H, 256, V, B, batch, K, weights, inp, seed_given, temperatures(tau, batch),
                   _per_seq(top_k, batch, np.int32), _per_seq(top_p, batch, np.float32))


def _per_seq(v, batch, dt):
    return None if v is None else np.broadcast_to(np.asarray(v, dtype=dt), (batch,)).copy()


def temperatures(tau, batch):
    """[batch] float32 temperatures from a scalar or a sequence (None stays None)."""
    if tau is None:
        return None
    return np.broadcast_to(np.asarray(tau, dtype=np.float32), (batch,)).copy()


def workload_problem(wl, batch=None, tau=None, top_k=None, top_p=None):
    weights = synth.make_weights(wl)
    inp = synth.make_inputs(wl, batch=batch)
    n = batch or wl.batch
    return Problem(wl.dtype, wl.H, wl.r, wl.V, wl.B, n, wl.K, weights, inp,
                   wl.seed_mode == "given", temperatures(tau, n), _per_seq(top_k, n, np.int32),
                   _per_seq(top_p, n, np.float32))


# ---------------------------------------------------------------------------
@dataclass
class DeviceRun:
    ids: np.ndarray
    iters: np.ndarray
    traj: np.ndarray
    logits: np.ndarray | None
    dev: dict = field(default_factory=dict)


def upload(prob: Problem):
    import torch
    from paper_2608_02438_amd.xpress import device_tensor
    i = prob.inp
    d = dict(hidden=device_tensor(i.h), anchor=device_tensor(i.anchor))
    d["seed_ids"] = device_tensor(i.seed_ids) if prob.seed_given else None
    sample_rows = bool(i.temp.any())
    d["temp"] = device_tensor(i.temp) if sample_rows else None
    d["u_draft"] = device_tensor(i.u_draft) if sample_rows else None
    d["r_accept"] = device_tensor(i.r_accept)
    d["u_res"] = device_tensor(i.u_res)
    d["target_logits"] = device_tensor(i.target_logits) if sample_rows else None
    d["temperature"] = device_tensor(prob.tau) if prob.tau is not None else None
    d["top_k"] = device_tensor(prob.top_k) if prob.top_k is not None else None
    d["top_p"] = device_tensor(prob.top_p) if prob.top_p is not None else None
    torch.cuda.synchronize()
    return d


def make_refiner(prob: Problem, max_batch=None):
    from paper_2608_02438_amd.xpress import refiner_from_arrays
    return refiner_from_arrays(prob.weights, prob.H, prob.r, prob.V, prob.B,
                               max_batch or prob.batch)


def run_device(ref, prob: Problem, dev: dict, K=None, early_exit=False, write_logits=True):
    import torch
    K = prob.K if K is None else K
    out = ref.refine_block(dev["hidden"], dev["anchor"], seed_ids=dev["seed_ids"],
                           temp=dev["temp"], u_draft=dev["u_draft"], K=K,
                           early_exit=early_exit, write_logits=write_logits, want_traj=True,
                           temperature=dev.get("temperature"), top_k=dev.get("top_k"),
                           top_p=dev.get("top_p"))
    torch.cuda.synchronize()
    return DeviceRun(ids=out.ids.cpu().numpy(), iters=out.iters.cpu().numpy(),
                     traj=out.traj.cpu().numpy(),
                     logits=out.logits.cpu().numpy() if write_logits else None)


# ---------------------------------------------------------------------------
@dataclass
class Tally:
    decisions: int = 0
    exact: int = 0
    excused: int = 0
    max_logit_err: float = 0.0
    max_err_over_bound: float = 0.0
    seq_exact: int = 0
    seqs: int = 0

    def add(self, o: "Tally"):
        for f in ("decisions", "exact", "excused", "seq_exact", "seqs"):
            setattr(self, f, getattr(self, f) + getattr(o, f))
        self.max_logit_err = max(self.max_logit_err, o.max_logit_err)
        self.max_err_over_bound = max(self.max_err_over_bound, o.max_err_over_bound)


def lm_row_norms(P):
    """|W_lm[v]|_2 for every vocabulary row (cached on the Params object)."""
    if getattr(P, "_lm_norm", None) is None:
        V = P.W_lm.shape[0]
        out = np.empty(V)
        for v0 in range(0, V, 8192):
            w = O.to_f64(P.W_lm[v0:v0 + 8192])
            out[v0:v0 + 8192] = np.sqrt(np.einsum("ij,ij->i", w, w))
        P._lm_norm = out
        P._abs_wr = np.abs(P.W_r)
    return P._lm_norm


def _bf16_spacing(x):
    _, e = np.frexp(x)
    return np.ldexp(1.0, np.maximum(e, -125) - 8)


def pass_logits(P, s_b, h_b, anchor, Y_prev):
    """Oracle logits of one pass from a given iterate (Y_prev None: the base logits),
    with the element-wise device error bound E of the module doc."""
    lmn = lm_row_norms(P)
    h64 = O.to_f64(h_b)
    H = h64.shape[1]
    if Y_prev is None:
        l = s_b
        Z = None
    else:
        st = O.fuse_static(P, h_b)
        x_prev = np.concatenate([[anchor], np.asarray(Y_prev, dtype=np.int64)[:-1]])
        Zraw = O.trans(P, O.mix(P.L, O.fuse(P, st, x_prev)))
        Z = O.round_bf16(Zraw) if P.round_z else Zraw
        l = s_b + O.read(P, Z)
    E = 6 * U32 * np.sqrt(H) * np.linalg.norm(h64, axis=1)[:, None] * lmn[None, :] + U32 * np.abs(l)
    if Z is not None:
        aw = P._abs_wr
        E += 6 * U32 * 16 * (np.abs(Z) @ aw.T)
        if P.round_z:
            sp = _bf16_spacing(Zraw)
            frac = Zraw / sp - np.floor(Zraw / sp)
            cand = np.abs(frac - 0.5) * sp <= Z_REL * np.abs(Zraw)
            E += (cand * sp) @ aw.T
        else:
            E += Z_REL * (np.abs(Z) @ aw.T)
    return l, E


def tempered_bound(l, E, T):
    """Bound on |x_device - l / T| when the device forms x as the fp32 product
    of l_device and the fp32 1/T: E / T plus two roundings of |l| / T."""
    return E / T + 2 * U32 * np.abs(l) / T


def filter_boundary(l, E, T, k, p):
    """Tokens at the truncation boundary whose membership the device error
    could flip (empty when the boundary is clear): top-k, the k-th and
    (k+1)-th largest scaled logits closer than twice the bound; top-p, the
    last kept and first dropped token when the mass before the first dropped
    one lies within the bound's relative effect (plus the device's 2^-44
    fixed-point mass units) of p times the top-k mass, or their logits are
    closer than twice the bound."""
    x = np.asarray(l, dtype=np.float64) / T
    ex = tempered_bound(l, E, T).max()
    V = x.shape[0]
    out = set()
    keep_k = np.ones(V, dtype=bool)
    if 0 < k < V:
        order = np.argsort(-x, kind="stable")
        a, b = order[k - 1], order[k]
        if x[a] - x[b] <= 4 * ex:
            out |= {int(v) for v in np.nonzero(np.abs(x - x[a]) <= 4 * ex)[0]}
        keep_k = x >= x[a]
    if p < 1.0:
        w = O.softmax_weights(l, T) * keep_k
        idx = np.nonzero(keep_k)[0]
        order = idx[np.lexsort((idx, -x[idx]))]
        before = np.concatenate([[0.0], np.cumsum(w[order])[:-1]])
        Zk = w.sum()
        n = int(np.sum(before < p * Zk))              # tokens kept
        if n < len(order):
            rel = np.expm1(4 * ex) + V * 2.0 ** -44 + 1e-12
            last, first_out = order[n - 1], order[n]
            if (abs(before[n] - p * Zk) <= rel * Zk
                    or x[last] - x[first_out] <= 4 * ex):
                out |= {int(last), int(first_out)}
    return out


def _decision_ok(l, E, y_dev, sample, u, T=1.0, k=0, p=1.0):
    y_o, _ = O.select(l, sample, u, T, k, p)
    if y_o == y_dev:
        return "exact"
    if not sample:
        ok = (l[y_o] - l[y_dev]) <= E[y_o] + E[y_dev]
    else:
        w = O.filtered_weights(l, T, k, p)
        if filter_boundary(l, E, T, k, p):
            # the device's kept set may legitimately differ at the boundary
            ok = bool(w[y_dev] > 0) or y_dev in filter_boundary(l, E, T, k, p)
        else:
            C = np.cumsum(w)
            Z = C[-1]
            lo = C[y_dev - 1] if y_dev > 0 else 0.0
            f = np.exp(4 * tempered_bound(l, E, T).max())
            ok = w[y_dev] > 0 and lo / f <= u * Z <= C[y_dev] * f
    return "excused" if ok else "wrong"


def check_sequence(P, s_b, h_b, anchor, seed, sample, u, K, traj, iters, logits, T=1.0,
                   abs_bar=None, k=0, p=1.0):
    """Validate one sequence's device trajectory; returns (Tally, final logits, final E).

    The final logits must lie within E of the oracle's element by element and,
    when ``abs_bar`` is given, within that absolute bar as well (the workloads'
    tolerance: 1e-5 for fp32, 2e-2 for bf16)."""
    B = s_b.shape[0]
    t = Tally(seqs=1)
    ref = O.refine_block(P, s_b, h_b, anchor, seed=seed, sample=sample, u=u, K=K,
                         early_exit=False, T=T, top_k=k, top_p=p)
    tro = ref.traj_padded(K)
    first = 0 if seed is None else 1
    exact_traj = np.array_equal(tro, traj)
    l_final = E_final = None
    for j in range(first, K + 1):
        if exact_traj and j < K:
            continue
        l, E = pass_logits(P, s_b, h_b, anchor, None if j == 0 else traj[j - 1])
        l_final, E_final = l, E
        if exact_traj:
            continue
        for q in range(B):
            r = _decision_ok(l[q], E[q], int(traj[j][q]), sample, float(u[q]), T, k, p)
            assert r != "wrong", f"pass {j} position {q}: device token {traj[j][q]} is not a valid selection"
            t.decisions += 1
            t.exact += r == "exact"
            t.excused += r == "excused"
    if exact_traj:
        n = (K + 1 - first) * B
        t.decisions = t.exact = n
        t.seq_exact = 1
    if l_final is None:                       # K = 0 with given seed ids
        l_final, E_final = pass_logits(P, s_b, h_b, anchor, None)
    it = next((j + 1 for j in range(K) if np.array_equal(traj[j + 1], traj[j])), K)
    assert int(iters) == it, f"iters {iters} != {it}"
    if logits is not None:
        err = np.abs(logits.astype(np.float64) - l_final)
        t.max_logit_err = float(err.max())
        t.max_err_over_bound = float((err / E_final).max())
        assert (err <= E_final).all(), (
            f"logit error {t.max_logit_err} exceeds its bound at "
            f"{np.unravel_index(np.argmax(err / E_final), err.shape)}")
        if abs_bar is not None:
            assert t.max_logit_err <= abs_bar, (
                f"logit error {t.max_logit_err} exceeds the absolute bar {abs_bar}")
    return t, l_final, E_final


def check_refine(prob: Problem, run: DeviceRun, seqs=None, P=None, s=None, abs_bar=None):
    """Check the chosen sequences of a device run; returns (Tally, final logits per seq).
    ``s`` (optional) holds the oracle's base logits of those sequences, in order."""
    P = P or O.Params.from_arrays(prob.weights, round_z=prob.dtype == "bf16")
    seqs = list(range(prob.batch)) if seqs is None else list(seqs)
    i = prob.inp
    if s is None:
        s = O.base_logits(P.W_lm, i.h[seqs].reshape(len(seqs) * prob.B, prob.H)).reshape(
            len(seqs), prob.B, -1)
    tot, finals = Tally(), {}
    for n, b in enumerate(seqs):
        seed = i.seed_ids[b] if prob.seed_given else None
        t, lf, Ef = check_sequence(P, s[n], i.h[b], int(i.anchor[b]), seed, bool(i.temp[b]),
                                   i.u_draft[b], run.traj.shape[0] - 1, run.traj[:, b],
                                   run.iters[b], None if run.logits is None else run.logits[b],
                                   prob.T(b), abs_bar=abs_bar, k=prob.filt(b)[0],
                                   p=prob.filt(b)[1])
        tot.add(t)
        finals[b] = (lf, Ef)
    return tot, finals


def check_verify(prob: Problem, run: DeviceRun, finals: dict, n_dev, next_dev, target_ids, seqs):
    """Greedy rows: exact.  Sampled rows: exact or a near-tie decision.

    With |l_device - l| <= E and |lse_device - lse| <= Emax the device's q moves
    by a factor within e^(+-2 Emax); the target p (fp32 logits, fp64 sums on
    both sides) by at most 1e-6 relative.  Truncated rows use the truncated
    q and p, and are also excused where a row's truncation boundary is itself
    a near-tie.
    """
    i = prob.inp
    excused = 0
    for b in seqs:
        y = run.ids[b]
        if not i.temp[b]:
            n, nx = O.verify_greedy(y, target_ids[b])
            assert (int(n_dev[b]), int(next_dev[b])) == (n, nx), f"seq {b}"
            continue
        lf, Ef = finals[b]
        T = prob.T(b)
        fk, fp = prob.filt(b)
        pl = i.target_logits[b].astype(np.float64)
        v = O.verify_sample(lf, y, pl, i.r_accept[b], float(i.u_res[b]), T, fk, fp)
        if (int(n_dev[b]), int(next_dev[b])) == (v.n, v.next):
            continue
        k = min(int(n_dev[b]), v.n)
        kq = min(k, prob.B - 1)
        tol = (np.exp(2 * tempered_bound(lf[kq], Ef[kq], T).max()) - 1 + 1e-6
               + 4 * U32 * np.abs(pl[k]).max() / T + prob.V * 2.0 ** -44)
        boundary = bool(filter_boundary(lf[kq], Ef[kq], T, fk, fp)) or bool(
            filter_boundary(pl[k], 4 * U32 * np.abs(pl[k]), T, fk, fp))
        if boundary:
            excused += 1
            continue
        if int(n_dev[b]) != v.n:
            assert v.accept_margins[k] <= tol, f"seq {b}: accept decision at {k} is not a near-tie"
        else:
            p = O.softmax(pl[k], T, fk, fp)
            res = np.maximum(p - O.softmax(lf[k], T, fk, fp), 0.0) if k < prob.B else p
            if not res.sum() > 0:
                res = p
            C = np.cumsum(res)
            t = int(next_dev[b])
            lo = C[t - 1] if t > 0 else 0.0
            uz = float(i.u_res[b]) * C[-1]
            assert lo - tol <= uz <= C[t] + tol, f"seq {b}: resample"
        excused += 1
    return excused
