"""fp64 CPU oracle of the xPress refine + verify path.

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the CPU-baseline
leg of the benchmark import this module.  The device path never imports, calls
or links it, and it shares no code with the device path: it takes plain numpy
arrays (bf16 bit patterns as uint16, or float32) and widens them itself.

What it computes, in the paper's order and notation (section 4):

* base readout   s_k = W_lm h_k                       (section 4.1, pipeline of Fig. 2a)
* global summary g = (1/B) sum_j h_j                  (section 4.1, below eq. correct)
* Fuse   a_k = W_in [W_h h_k || W_g g || W_e[x_{k-1}]]            (eq. fuse)
* Mix    c^(d) = (I_B + L^(d)) a^(d), L^(d) strictly lower        (eq. mix)
* Trans  z_k = c_k + W_2 sigma(W_1 c_k)                           (eq. mlp)
* Read   delta_k = W_r z_k                                        (eq. read)
* Correct l_k = s_k + delta_k ; p^r_k = softmax(l_k)              (eqs. correct, refined-dist)
* Jacobi refinement: Y0 from the base logits, then up to K parallel passes,
  stopping at the fixed point                                     (Algorithm 1, eq. jacobi-update)
* sequential decode y*_k = select(l_k(y*_{<k}))                    (Theorem 1)
* verification: greedy longest-prefix + bonus token, and speculative
  accept / reject with residual resampling                         (section 3.1; section 4.3 TV identity)

Readings where the paper is silent (each is listed with its reason in the
design notes): sigma is SiLU; no biases or norms; W_e and W_r are separate
matrices; the anchor x_0 is supplied per sequence; ties in argmax go to the
lowest index; at temperature 1 a position is selected by inverse-CDF sampling
of softmax(l_k) with one uniform u_k per position that stays fixed across
passes; the temperature-1 seed is the same inverse-CDF rule on softmax(s_k);
the refined distribution used for verification is the one of the pass that
produced the final token; for bf16 workloads z is the only activation rounded
to bf16 (before Read), everything else is exact fp64 here, selections
included (argmax and softmax on the fp64 logits).

Parity status: every function below is pinned by the CPU tests
(tests/test_oracle_*.py) except the exact logit values of a trained refiner,
which the paper does not print (no worked numerical example): "parity
unpinned" for absolute logit values beyond the identities and special cases
listed there.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

F64 = np.float64


# --------------------------------------------------------------------------
# storage widening and the bf16 rounding point
# --------------------------------------------------------------------------

def to_f64(x) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) or float32 to float64 exactly."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(F64)
    return x.astype(F64)


def round_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bf16 value, ties to even.

    bf16 keeps 8 significant bits: a normal value m * 2**e (0.5 <= |m| < 1) is
    rounded to a multiple of 2**(e-8); below 2**-126 the spacing stays 2**-133
    (subnormals).  Results beyond the largest finite bf16 become +-inf.
    """
    x = np.asarray(x, dtype=F64)
    _, e = np.frexp(x)
    e = np.maximum(e, -125)
    q = np.ldexp(np.rint(np.ldexp(x, 8 - e)), e - 8)
    big = np.abs(q) >= 2.0 ** 128
    if np.any(big):
        q = np.where(big, np.copysign(np.inf, x), q)
    return q


def silu(x):
    """SiLU, x * sigmoid(x).

    sigmoid is evaluated as 1 / (1 + e^-x) for x >= 0 and e^x / (1 + e^x) for
    x < 0, so that neither branch overflows nor cancels.
    """
    x = np.asarray(x, dtype=F64)
    e = np.exp(-np.abs(x))
    sig = np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))
    return x * sig


# --------------------------------------------------------------------------
# parameters
# --------------------------------------------------------------------------

@dataclass
class Params:
    """The refiner weights widened to fp64, plus the raw LM head.

    Shapes (row-major, rows are output units): W_lm [V][H], W_h and W_g [r][H],
    W_e [V][r] (row per token: the paper's r x V embedding, transposed),
    W_in [r][3r] with column blocks [h | g | token] in the order of eq. fuse,
    L [r][B][B] (only entries [d][k][i] with i < k are read), W_1 [2r][r],
    W_2 [r][2r], W_r [V][r].
    """
    W_lm: np.ndarray
    W_h: np.ndarray
    W_g: np.ndarray
    W_e: np.ndarray
    W_in: np.ndarray
    L: np.ndarray
    W_1: np.ndarray
    W_2: np.ndarray
    W_r: np.ndarray
    round_z: bool

    @staticmethod
    def from_arrays(w: dict, round_z: Optional[bool] = None) -> "Params":
        if round_z is None:
            round_z = w["W_r"].dtype == np.uint16
        return Params(W_lm=w["W_lm"], W_h=to_f64(w["W_h"]), W_g=to_f64(w["W_g"]),
                      W_e=to_f64(w["W_e"]), W_in=to_f64(w["W_in"]), L=to_f64(w["L"]),
                      W_1=to_f64(w["W_1"]), W_2=to_f64(w["W_2"]), W_r=to_f64(w["W_r"]),
                      round_z=bool(round_z))

    @property
    def r(self) -> int:
        return self.W_in.shape[0]

    @property
    def V(self) -> int:
        return self.W_r.shape[0]


# --------------------------------------------------------------------------
# base readout (A1) and the refiner stages
# --------------------------------------------------------------------------

def base_logits(W_lm, h, chunk: int = 8192) -> np.ndarray:
    """s_k = W_lm h_k for every row of ``h`` ([n][H]); returns [n][V] fp64.

    The target LM head reads the drafter hidden states out to the vocabulary
    (section 4.1, Fig. 2a).  The head is widened chunk by chunk to bound memory.
    """
    h64 = to_f64(h)
    V = W_lm.shape[0]
    s = np.empty((h64.shape[0], V), dtype=F64)
    for v0 in range(0, V, chunk):
        s[:, v0:v0 + chunk] = h64 @ to_f64(W_lm[v0:v0 + chunk]).T
    return s


def global_summary(h_block: np.ndarray) -> np.ndarray:
    """g = (1/B) sum_{j=1..B} h_j, the mean-pooled block summary (section 4.1)."""
    return h_block.mean(axis=0)


@dataclass
class Static:
    """Iteration-invariant part of Fuse: W_h h_k and W_g g (h, g fixed across passes)."""
    hh: np.ndarray      # [B][r]
    gg: np.ndarray      # [r]


def fuse_static(P: Params, h_block) -> Static:
    h64 = to_f64(h_block)
    g = global_summary(h64)
    return Static(hh=h64 @ P.W_h.T, gg=P.W_g @ g)


def fuse(P: Params, st: Static, x_prev) -> np.ndarray:
    """a_k = W_in [W_h h_k || W_g g || W_e[x_{k-1}]]   (eq. fuse).

    ``x_prev[k-1]`` is the token preceding position k: x_0 is the anchor and
    x_{k-1} (k >= 2) the current guess at position k-1.  Returns A as [B][r].
    """
    B = st.hh.shape[0]
    at = np.concatenate([st.hh, np.broadcast_to(st.gg, (B, P.r)),
                         P.W_e[np.asarray(x_prev, dtype=np.int64)]], axis=1)
    return at @ P.W_in.T


def mix(L: np.ndarray, A: np.ndarray) -> np.ndarray:
    """c^(d) = (I_B + L^(d)) a^(d) per channel d, L^(d) strictly lower  (eq. mix).

    Position k adds L[d][k][i] * a_{i,d} for every earlier position i < k; no
    entry with i >= k is read.
    """
    B = A.shape[0]
    C = A.copy()
    for k in range(B):
        for i in range(k):
            C[k] += L[:, k, i] * A[i]
    return C


def toeplitz_mixer(kappa: np.ndarray) -> np.ndarray:
    """The mixer of the Toeplitz remark (section 3): L^(d)_{k,j} = kappa[d][k-j].

    kappa is [r][B]; lag 0 is the identity of eq. mix, so kappa[:, 0] is never
    read.  Returns L [r][B][B] with L[d][k][j] = kappa[d][k - j] for j < k and 0
    on and above the diagonal, so Mix with it is a causal depthwise conv1d of
    kernel size B (kernel [1, kappa[d][1], ..., kappa[d][B-1]]).
    """
    kappa = np.asarray(kappa)
    r, B = kappa.shape
    L = np.zeros((r, B, B), dtype=kappa.dtype)
    for k in range(B):
        for j in range(k):
            L[:, k, j] = kappa[:, k - j]
    return L


def trans(P: Params, C: np.ndarray) -> np.ndarray:
    """z_k = c_k + W_2 sigma(W_1 c_k), sigma = SiLU   (eq. mlp)."""
    return C + silu(C @ P.W_1.T) @ P.W_2.T


def read(P: Params, Z: np.ndarray) -> np.ndarray:
    """delta_k = W_r z_k   (eq. read); returns [B][V]."""
    return Z @ P.W_r.T


def refiner(P: Params, st: Static, x_prev):
    """R_theta = Read . Trans . Mix . Fuse on one block; returns (delta, z)."""
    A = fuse(P, st, x_prev)
    C = mix(P.L, A)
    Z = trans(P, C)
    if P.round_z:
        Z = round_bf16(Z)
    return read(P, Z), Z


def fuse_mix_folded(W_in: np.ndarray, L: np.ndarray, At: np.ndarray) -> np.ndarray:
    """The folded Fuse-Mix operator of section 4.1 (low-overhead paragraph).

    c_k = sum_{j<=k} M_{k,j} at_j with M_{k,j} = diag(1[j=k] + 1[j<k] L_{k,j}) W_in,
    i.e. row d of W_in scaled by the channel-d mixing coefficient.  ``At`` holds
    the unfused inputs at_j = [W_h h_j || W_g g || W_e[x_{j-1}]] as [B][3r].
    """
    B = At.shape[0]
    r = W_in.shape[0]
    C = np.zeros((B, r), dtype=F64)
    for k in range(B):
        for j in range(k + 1):
            coef = np.ones(r) if j == k else L[:, k, j]
            C[k] += (coef[:, None] * W_in) @ At[j]
    return C


# --------------------------------------------------------------------------
# selection rules
# --------------------------------------------------------------------------

def select_greedy(l: np.ndarray):
    """argmax_v l_v with ties to the lowest index; returns (token, margin).

    The comparison is taken on the fp64 logits (np.argmax returns the first
    maximal index and treats -0 and +0 as equal).  The margin is the gap
    between the two largest logits.
    """
    l = np.asarray(l, dtype=F64)
    y = int(np.argmax(l))
    if l.shape[0] < 2:
        return y, np.inf
    top2 = np.partition(l, -2)[-2:]
    return y, float(top2[1] - top2[0])


def inverse_cdf(w: np.ndarray, u: float):
    """Smallest v with sum_{i<=v} w_i > u * sum(w); returns (token, margin).

    Falls back to the last v with w_v > 0 when rounding leaves no crossing.
    The margin is the distance from u * Z to the nearer edge of the chosen
    token's interval, divided by Z.
    """
    C = np.cumsum(w)
    Z = C[-1]
    t = float(u) * Z
    y = int(np.searchsorted(C, t, side="right"))
    if y >= w.shape[0]:
        y = int(np.nonzero(w > 0)[0][-1])
    lo = C[y - 1] if y > 0 else 0.0
    return y, float(min(t - lo, C[y] - t) / Z)


def softmax_weights(l: np.ndarray, T: float = 1.0) -> np.ndarray:
    """exp((l_v - max l) / T) in fp64: the unnormalised softmax of the
    logits at temperature T > 0."""
    l = np.asarray(l, dtype=F64)
    return np.exp((l - l.max()) / float(T))


def filtered_weights(l: np.ndarray, T: float = 1.0, top_k: int = 0,
                     top_p: float = 1.0) -> np.ndarray:
    """softmax_weights(l, T) restricted to the tokens the top-k and top-p
    truncations keep (zero elsewhere); top_k = 0 (or >= V) and top_p >= 1
    keep every token.

    Truncated sampling at temperature T (the filtered form of the sampling
    that verification keeps lossless, section 3.1), in this order:
    * top-k keeps every token whose scaled logit x = l / T is at least the
      k-th largest of them (counted with multiplicity, so ties with it stay);
    * top-p then orders the kept tokens by x descending, ties by lower index
      first, and keeps each token whose preceding mass in that order is
      below p times the total mass of the top-k set, i.e. the shortest
      prefix whose mass reaches p of it.
    """
    w = softmax_weights(l, T)
    V = w.shape[0]
    keep = np.ones(V, dtype=bool)
    x = np.asarray(l, dtype=F64) / float(T)
    if 0 < top_k < V:
        kth = np.sort(x)[V - top_k]
        keep &= x >= kth
    if top_p < 1.0:
        idx = np.nonzero(keep)[0]
        order = idx[np.lexsort((idx, -x[idx]))]          # x descending, then index ascending
        before = np.concatenate([[0.0], np.cumsum(w[order])[:-1]])
        keep_p = np.zeros(V, dtype=bool)
        keep_p[order[before < top_p * w[idx].sum()]] = True
        keep &= keep_p
    return np.where(keep, w, 0.0)


def select_sample(l: np.ndarray, u: float, T: float = 1.0, top_k: int = 0, top_p: float = 1.0):
    """Inverse-CDF sample of the (filtered) softmax(l / T) at the uniform u;
    returns (token, margin)."""
    return inverse_cdf(filtered_weights(l, T, top_k, top_p), u)


def select(l: np.ndarray, sample: bool, u: float, T: float = 1.0, top_k: int = 0,
           top_p: float = 1.0):
    return select_sample(l, u, T, top_k, top_p) if sample else select_greedy(l)


def softmax(l: np.ndarray, T: float = 1.0, top_k: int = 0, top_p: float = 1.0) -> np.ndarray:
    """The (filtered) softmax(l / T), normalised."""
    w = filtered_weights(l, T, top_k, top_p)
    return w / w.sum()


# --------------------------------------------------------------------------
# Jacobi refinement (Algorithm 1) and the sequential decode (Theorem 1)
# --------------------------------------------------------------------------

@dataclass
class Refined:
    ids: np.ndarray                 # [B] final block
    iters: int                      # passes run until the fixed-point test held (<= K)
    traj: List[np.ndarray]          # Y^(0) .. Y^(iters)
    margins: List[np.ndarray]       # margins of the decisions producing traj[j]
    logits: np.ndarray              # [B][V] l of the pass that produced ids (s if K = 0)
    z: Optional[np.ndarray] = None  # [B][r] z of that pass

    def traj_padded(self, K: int) -> np.ndarray:
        """Y^(0..K): past the fixed point every further pass reproduces it."""
        t = list(self.traj) + [self.traj[-1]] * (K + 1 - len(self.traj))
        return np.stack(t[:K + 1])


def refine_block(P: Params, s_b: np.ndarray, h_b, anchor: int, seed=None,
                 sample: bool = False, u=None, K: int = 6,
                 early_exit: bool = True, T: float = 1.0, top_k: int = 0,
                 top_p: float = 1.0) -> Refined:
    """Algorithm 1 for one sequence.

    Y^(0) is ``seed`` when given, otherwise each position's selection from the
    base logits s_k.  Pass j runs the refiner on Y^(j) (prefix x_0 = anchor,
    x_{k-1} = y^(j)_{k-1}), re-selects every position from s_k + delta_k in
    parallel, and stops once Y^(j+1) = Y^(j).  With ``early_exit`` False the
    loop always runs K passes, which must not change the result.  Sampled
    sequences draw from softmax(l / T), truncated by top_k / top_p.
    """
    B = s_b.shape[0]
    u = np.zeros(B) if u is None else np.asarray(u, dtype=F64)
    st = fuse_static(P, h_b)
    if seed is not None:
        Y = np.asarray(seed, dtype=np.int64).copy()
        mg = np.full(B, np.inf)
    else:
        sel = [select(s_b[k], sample, u[k], T, top_k, top_p) for k in range(B)]
        Y = np.array([t for t, _ in sel], dtype=np.int64)
        mg = np.array([m for _, m in sel])
    traj, margins = [Y.copy()], [mg]
    logits, zlast, iters = s_b, None, 0
    for j in range(K):
        x_prev = np.concatenate([[anchor], Y[:-1]])
        delta, Z = refiner(P, st, x_prev)
        l = s_b + delta
        sel = [select(l[k], sample, u[k], T, top_k, top_p) for k in range(B)]
        Yn = np.array([t for t, _ in sel], dtype=np.int64)
        traj.append(Yn.copy())
        margins.append(np.array([m for _, m in sel]))
        logits, zlast = l, Z
        converged = bool(np.array_equal(Yn, Y))
        Y = Yn
        if converged and iters == 0:
            iters = j + 1
            if early_exit:
                break
    if iters == 0:
        iters = K
    return Refined(ids=Y, iters=iters, traj=traj, margins=margins, logits=logits, z=zlast)


def sequential_decode(P: Params, s_b: np.ndarray, h_b, anchor: int,
                      sample: bool = False, u=None, T: float = 1.0, top_k: int = 0,
                      top_p: float = 1.0) -> np.ndarray:
    """y*_k = select(s_k + delta_k(x_0, y*_1..y*_{k-1})) for k = 1..B, in order.

    Positions after k are filled with token 0; by the causal structure of the
    refiner they do not affect position k.
    """
    B = s_b.shape[0]
    u = np.zeros(B) if u is None else np.asarray(u, dtype=F64)
    st = fuse_static(P, h_b)
    Y = np.zeros(B, dtype=np.int64)
    for k in range(B):
        x_prev = np.concatenate([[anchor], Y[:-1]])
        delta, _ = refiner(P, st, x_prev)
        Y[k], _ = select(s_b[k] + delta[k], sample, u[k], T, top_k, top_p)
    return Y


def pass_from(P: Params, s_b, h_b, anchor: int, Y_prev, sample: bool, u, T: float = 1.0,
              top_k: int = 0, top_p: float = 1.0):
    """One Jacobi pass from a given iterate: (new ids, margins, logits).

    Used to check a device trajectory decision by decision.
    """
    B = s_b.shape[0]
    u = np.zeros(B) if u is None else np.asarray(u, dtype=F64)
    st = fuse_static(P, h_b)
    x_prev = np.concatenate([[anchor], np.asarray(Y_prev, dtype=np.int64)[:-1]])
    delta, _ = refiner(P, st, x_prev)
    l = s_b + delta
    sel = [select(l[k], sample, u[k], T, top_k, top_p) for k in range(B)]
    return (np.array([t for t, _ in sel], dtype=np.int64),
            np.array([m for _, m in sel]), l)


# --------------------------------------------------------------------------
# verification (section 3.1)
# --------------------------------------------------------------------------

def verify_greedy(ids, target_ids):
    """Longest prefix n with y_i = t_i for all i <= n, and next = t_{n+1}.

    ``target_ids`` has B+1 entries: the target's greedy token after each
    prefix of the block, the last one being the bonus token.
    """
    B = len(ids)
    n = 0
    while n < B and int(ids[n]) == int(target_ids[n]):
        n += 1
    return n, int(target_ids[n])


@dataclass
class Verified:
    n: int
    next: int
    accept_margins: np.ndarray     # |r q - p| / max(p, r q) for each tested position
    resample_margin: float


def verify_sample(q_logits, ids, p_logits, r_accept, u_res, T: float = 1.0, top_k: int = 0,
                  top_p: float = 1.0) -> Verified:
    """Speculative accept / reject of a sampled block (section 3.1).

    For k = 1..B: accept y_k iff r_k * q_k(y_k) <= p_k(y_k), where q_k is the
    refined distribution the draft token was sampled from and p_k the target
    distribution after the same prefix, both at temperature T and truncated by
    the same top_k / top_p (so the emitted tokens follow the truncated target
    distribution).  At the first
    rejection the next token is an inverse-CDF sample (at u_res) of
    max(0, p_k - q_k), or of p_k if that residual has no mass.  If all B are
    accepted the bonus token is sampled from p_{B+1}.
    """
    B = len(ids)
    am = []
    for k in range(B):
        q = softmax(q_logits[k], T, top_k, top_p)
        p = softmax(p_logits[k], T, top_k, top_p)
        y = int(ids[k])
        rq = float(r_accept[k]) * q[y]
        den = max(p[y], rq)
        am.append(abs(rq - p[y]) / den if den > 0 else 0.0)   # 0 = 0: an exact tie
        if not rq <= p[y]:
            res = np.maximum(p - q, 0.0)
            if not res.sum() > 0:
                res = p
            t, m = inverse_cdf(res, u_res)
            return Verified(n=k, next=t, accept_margins=np.array(am), resample_margin=m)
    t, m = inverse_cdf(softmax(p_logits[B], T, top_k, top_p), u_res)
    return Verified(n=B, next=t, accept_margins=np.array(am), resample_margin=m)


# --------------------------------------------------------------------------
# whole-batch driver
# --------------------------------------------------------------------------

@dataclass
class BatchResult:
    seqs: List[int]
    refined: List[Refined] = field(default_factory=list)
    s: Optional[np.ndarray] = None          # [len(seqs)][B][V]


def refine_batch(P: Params, h, anchor, temp, u_draft, K: int, seed_ids=None,
                 seqs=None, early_exit: bool = True, temperature=None, top_k=None,
                 top_p=None) -> BatchResult:
    """Run Algorithm 1 on the chosen sequences of a batch (default: all);
    sampled sequences use temperature[b] (1 when None) and the truncations
    top_k[b], top_p[b] (none when None)."""
    bsz, B, H = h.shape
    seqs = list(range(bsz)) if seqs is None else list(seqs)
    s = base_logits(P.W_lm, h[seqs].reshape(len(seqs) * B, H)).reshape(len(seqs), B, -1)
    out = BatchResult(seqs=seqs, s=s)
    for i, b in enumerate(seqs):
        out.refined.append(refine_block(
            P, s[i], h[b], int(anchor[b]),
            seed=None if seed_ids is None else seed_ids[b],
            sample=bool(temp[b]), u=u_draft[b], K=K, early_exit=early_exit,
            T=1.0 if temperature is None else float(temperature[b]),
            top_k=0 if top_k is None else int(top_k[b]),
            top_p=1.0 if top_p is None else float(top_p[b])))
    return out
