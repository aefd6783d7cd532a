"""CPU oracle for the branch-cached DiT-MoE layer step (MoECa, Sec. 4).

TEST INFRASTRUCTURE ONLY.  This module is the slow, plain reference the GPU
library is checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it.  It shares no code,
header, table or helper with the HIP path, and the product never calls it.

What it computes, in the paper's order (Sec. 4.1-4.3):

1. schedule      full-computation step vs cache step (Sec. 4.1; refresh
                 cycle N from Sec. 5.1);
2. router        top-k routing result B_i^t = {(e_ip, w_ip)} (Sec. 4.1);
3. EMA           spatial activation statistic C_{e,i} (Sec. 4.3, EMA eq.);
4. entropy, tau  P_e(i), H_e, normalised H_e, tau_e (Sec. 4.3, entropy and
                 threshold eqs.);
5. match, score  q(p), Delta, o, s (Sec. 4.2, score eq.) and the margin
                 s - tau_e;
6. select        the recomputation set R_i^t (Sec. 4.2 threshold rule; a
                 per-sample refresh-ratio budget as the alternative mode);
7. slots         which cached slot each recomputed branch overwrites;
8. lists         per-expert lists of recomputed branches;
9. expert FFN    h = FFN_e(x_i) for recomputed branches (Sec. 2.3 MoE eq.);
10. combine      y_i (Sec. 4.1, output eq.), reused branches with the current
                 weight and the cached feature;
11. cache write  (e, w, h, ||h||) for recomputed branches and the attention
                 path for tokens with a recomputed branch (Sec. 4.1 sync
                 rule).

Arithmetic.  The paper fixes no precision.  Reductions and transcendentals
on the decision path (router logits, softmax, entropy, row norms) are done
in fp64 from exact inputs and rounded once to fp32; every other decision
quantity (EMA, threshold, score, margin) is the named fp32 operation in the
order written here (numpy fp32 arithmetic: correctly rounded, never fused).
The expert FFN runs in fp64 (library matmul) and its stored results are
rounded to the layer's activation dtype (bf16 or fp32), as is the GELU
intermediate.

Readings where the paper is silent or ambiguous:
R-1 gate = softmax over all experts, top-k, renormalised over the top-k
(``norm_topk``; the unnormalised form is a flag); R-2 entropy normalised by
log N; R-3 C is kept per sample; R-4 EMA updated every step (full steps
too), before the threshold, starting from 0; R-5 lambda1 = lambda2 = 1 by
default (the paper does not report them); R-6 the o denominator sums the
norms of all valid cached slots of the token; R-7 norms are of the stored
(rounded) rows; R-8 only recomputed branches are written back; R-9 reused
branches use the current weight; R-10 S_i = [R_i non-empty] drives the
attention refresh; R-11 strict s > tau with tau per expert; R-12 unmatched
branches take the free slots in ascending order; R-13 a fixed refresh cycle
(full iff t % N == 0 or the cache is invalid); R-14 ratio mode: all
unmatched plus the best matched by (margin desc, flat id asc) up to
K_b = floor(rho*N*k + 0.5) per sample; R-16 ties toward the lower expert id
and the lower flat id; R-17 tanh GELU; R-18 the layer returns y (the caller
adds the residual); R-20 round to nearest even; full steps place branch p
in slot p; R-24 shared experts (Sec. 2.3, shared-expert MoE eq.) are
ungated, evaluated for every token on every step and never cached; the
combine adds their outputs first (in expert order), then the routed
branches, in fp32; R-25 the gated (SwiGLU) expert FFN is
W_down (silu(W_gate x) * (W_up x)), silu(z) = z / (1 + exp(-z)), with the
gate and up rows interleaved in one up-projection matrix (row 2j gate j,
row 2j+1 up j) and the product rounded once to the stored dtype.

Pins: every function here is checked by ``tests/test_oracle_pins.py``
against closed forms, special cases that reduce to a library routine, a
constructed worked example, invariants and brute force.  Output quality
against the paper's trained models: parity unpinned (needs the trained
checkpoints).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

MODE_FULL = 0        # plain uncached MoE layer (the comparator)
MODE_THRESHOLD = 1   # paper's rule: recompute iff s > tau (or unmatched)
MODE_RATIO = 2       # per-sample refresh budget ranked by margin s - tau

BF16 = "bf16"
FP32 = "fp32"

F32 = np.float32
F64 = np.float64


# ---------------------------------------------------------------------------
# activation dtype: widening and rounding (round to nearest, ties to even)
# ---------------------------------------------------------------------------
_BF16_MAX = float.fromhex("0x1.fep127")


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of a stored tensor (bf16 bits or fp32) to fp64."""
    if dtype == BF16:
        u = np.asarray(a, dtype=np.uint16).astype(np.uint32) << 16
        return u.view(np.float32).astype(F64)
    return np.asarray(a, dtype=F32).astype(F64)


def to_f32(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of a stored tensor (bf16 bits or fp32) to fp32."""
    if dtype == BF16:
        u = np.asarray(a, dtype=np.uint16).astype(np.uint32) << 16
        return u.view(np.float32)
    return np.asarray(a, dtype=F32)


def round_act(v: np.ndarray, dtype: str) -> np.ndarray:
    """Round fp64 values to the activation dtype, nearest-even, one rounding.

    bf16 keeps 8 significant bits and fp32's exponent range.  The value is
    scaled by the bf16 quantum of its binade (a power of two, so exact),
    rounded to an integer with ties to even, and scaled back.
    """
    v = np.asarray(v, dtype=F64)
    if dtype == FP32:
        return v.astype(F32)
    out = np.empty(v.shape, dtype=F64)
    fin = np.isfinite(v)
    vf = v[fin]
    _, ex = np.frexp(vf)                      # vf = m * 2**ex, 0.5 <= |m| < 1
    ex = np.maximum(ex, -125)                 # below 2**-126 the quantum is fixed
    quantum = np.ldexp(1.0, ex - 8)           # 8 significant bits
    r = np.rint(vf / quantum) * quantum       # np.rint: ties to even
    r[np.abs(r) > _BF16_MAX] = np.inf * np.sign(r[np.abs(r) > _BF16_MAX])
    out[fin] = r
    out[~fin] = v[~fin]
    bits = out.astype(F32).view(np.uint32)    # exact: r is bf16-representable
    res = (bits >> 16).astype(np.uint16)
    res[np.isnan(out)] = 0x7FC0
    return res


# ---------------------------------------------------------------------------
# configuration and state
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class Policy:
    """Controller settings.  Defaults: tau0 = 0.80 (Sec. 5.4), beta = 0.65
    (Sec. 5.4), alpha = 0.6 (Tab. 4), refresh cycle N = 4 (Sec. 5.1)."""
    mode: int = MODE_THRESHOLD
    ratio: float = 0.3
    tau0: float = 0.80
    alpha: float = 0.6
    beta: float = 0.65
    lambda1: float = 1.0
    lambda2: float = 1.0
    lambda0: float = 1.0
    refresh_cycle: int = 4
    norm_topk: bool = True
    act: str = "gelu_tanh"


@dataclasses.dataclass
class Dims:
    d: int
    E: int
    k: int
    d_ff: int
    B: int
    N: int
    dtype: str = BF16
    n_shared: int = 0


class Weights:
    """Router and expert weights, ``out x in`` row-major, stored dtype."""

    def __init__(self, dims: Dims, W_r, b_r, W_up, W_down, W_sh_up=None, W_sh_down=None):
        self.dims = dims
        self.W_r = W_r
        self.b_r = None if b_r is None else np.asarray(b_r, dtype=F32)
        self.W_up = W_up
        self.W_down = W_down
        self.W_sh_up = W_sh_up      # (S, up rows, d) shared experts, or None
        self.W_sh_down = W_sh_down  # (S, d, d_ff)
        self._up64 = {}
        self._down64 = {}
        self.W_r64 = to_f64(W_r, dims.dtype)

    def up64(self, e: int) -> np.ndarray:
        if e not in self._up64:
            self._up64[e] = to_f64(self.W_up[e], self.dims.dtype)
        return self._up64[e]

    def down64(self, e: int) -> np.ndarray:
        if e not in self._down64:
            self._down64[e] = to_f64(self.W_down[e], self.dims.dtype)
        return self._down64[e]

    def shared_up64(self, s: int) -> np.ndarray:
        return to_f64(self.W_sh_up[s], self.dims.dtype)

    def shared_down64(self, s: int) -> np.ndarray:
        return to_f64(self.W_sh_down[s], self.dims.dtype)


class State:
    """Per-layer cache (Sec. 4.1) plus the expert statistic (Sec. 4.3).

    e_c, w_c, n_c : (B, N, k) cached expert id (-1 = empty), weight, row norm
    h_c           : (B, N, k, d) cached branch outputs, stored dtype
    C             : (B, E, N) fp32 spatial activation statistic
    A             : (B, N, d) attention-path cache, stored dtype, or None
    valid         : False until a full step has filled the cache
    """

    def __init__(self, dims: Dims, attention: bool = False):
        B, N, k, d, E = dims.B, dims.N, dims.k, dims.d, dims.E
        act = np.uint16 if dims.dtype == BF16 else F32
        self.e_c = np.full((B, N, k), -1, dtype=np.int32)
        self.w_c = np.zeros((B, N, k), dtype=F32)
        self.n_c = np.zeros((B, N, k), dtype=F32)
        self.h_c = np.zeros((B, N, k, d), dtype=act)
        self.C = np.zeros((B, E, N), dtype=F32)
        self.A = np.zeros((B, N, d), dtype=act) if attention else None
        self.valid = False

    def copy(self) -> "State":
        s = State.__new__(State)
        s.e_c, s.w_c, s.n_c = self.e_c.copy(), self.w_c.copy(), self.n_c.copy()
        s.h_c, s.C = self.h_c.copy(), self.C.copy()
        s.A = None if self.A is None else self.A.copy()
        s.valid = self.valid
        return s


# ---------------------------------------------------------------------------
# 1. schedule (Sec. 4.1 full/cache steps; Sec. 5.1 refresh cycle)
# ---------------------------------------------------------------------------
def is_full_step(policy: Policy, valid: bool, t: int) -> bool:
    if policy.mode == MODE_FULL or not valid:
        return True
    return policy.refresh_cycle > 0 and t % policy.refresh_cycle == 0


# ---------------------------------------------------------------------------
# 2. router (Sec. 4.1: B_i^t = {(e_ip, w_ip)}_{p=1..k})
# ---------------------------------------------------------------------------
def router_logits(x64: np.ndarray, W_r64: np.ndarray, b_r) -> tuple[np.ndarray, np.ndarray]:
    """l_{i,e} = x_i . W_r[e] (+ b_e): exact products summed in fp64, then
    rounded once to fp32.  Returns (fp64 sums, fp32 logits)."""
    l64 = x64 @ W_r64.T
    if b_r is not None:
        l64 = l64 + np.asarray(b_r, dtype=F32).astype(F64)
    return l64, l64.astype(F32)


def route(logits: np.ndarray, k: int, norm_topk: bool):
    """Top-k experts by descending fp32 logit (ties: lower expert id first)
    and their gate weights from a softmax over all experts, renormalised over
    the top-k when ``norm_topk``.  Softmax in fp64, weight rounded to fp32."""
    T, E = logits.shape
    order = np.argsort(-logits, axis=1, kind="stable")
    e = order[:, :k].astype(np.int32)
    lf = logits.astype(F64)
    z = np.exp(lf - lf.max(axis=1, keepdims=True))
    rows = np.arange(T)[:, None]
    zk = z[rows, e]
    den = zk.sum(axis=1) if norm_topk else z.sum(axis=1)
    w = (zk / den[:, None]).astype(F32)
    return e, w


# ---------------------------------------------------------------------------
# 3. EMA of expert spatial activation (Sec. 4.3, EMA eq.)
# ---------------------------------------------------------------------------
def ema_update(C: np.ndarray, e_t: np.ndarray, beta: float) -> np.ndarray:
    """C_{e,i} <- beta*C_{e,i} + (1-beta)*[e in B_i], per sample.

    fp32: first f32(beta*C), then f32(. + f32(1-beta)) where the indicator
    is one.  C: (B, E, N); e_t: (B, N, k)."""
    B, E, N = C.shape
    beta32 = F32(beta)
    c1 = F32(1.0) - beta32
    ind = np.zeros((B, E, N), dtype=bool)
    b_idx = np.repeat(np.arange(B), N * e_t.shape[2]).reshape(e_t.shape)
    i_idx = np.broadcast_to(np.arange(N)[None, :, None], e_t.shape)
    ind[b_idx, e_t, i_idx] = True
    Cn = (beta32 * C).astype(F32)
    return np.where(ind, (Cn + c1).astype(F32), Cn).astype(F32)


# ---------------------------------------------------------------------------
# 4. spatial-response entropy and expert-aware threshold (Sec. 4.3)
# ---------------------------------------------------------------------------
def normalized_entropy(C: np.ndarray) -> np.ndarray:
    """P_e(i) = C_{e,i} / sum_j C_{e,j};  H_e = -sum_i P log P  (fp64).

    Normalised as H_e / log N, clamped to [0, 1] and rounded to fp32.  An
    expert with an all-zero statistic, or N = 1, gets 0.  Shape (B, E)."""
    B, E, N = C.shape
    C64 = C.astype(F64)
    S = C64.sum(axis=2)
    H = np.zeros((B, E), dtype=F64)
    for b in range(B):
        for e in range(E):
            if S[b, e] == 0.0:
                continue
            P = C64[b, e] / S[b, e]
            P = P[P > 0.0]
            H[b, e] = -np.sum(P * np.log(P))
    if N <= 1:
        return np.zeros((B, E), dtype=F32)
    return np.clip(H / math.log(N), 0.0, 1.0).astype(F32)


def adaptive_threshold(Hbar: np.ndarray, tau0: float, alpha: float) -> np.ndarray:
    """tau_e = tau0 * (1 + alpha * (2*Hbar_e - 1)), fp32 operations."""
    two = F32(2.0) * Hbar
    centred = (two - F32(1.0)).astype(F32)
    scaled = (F32(alpha) * centred).astype(F32)
    return (F32(tau0) * (F32(1.0) + scaled).astype(F32)).astype(F32)


# ---------------------------------------------------------------------------
# 5. branch matching and recomputation score (Sec. 4.2)
# ---------------------------------------------------------------------------
def match(e_t: np.ndarray, e_c: np.ndarray):
    """q(p) = the cached slot holding the current expert e_p, or -1.

    e_t, e_c: (..., k).  Returns (matched bool, q int32)."""
    k = e_t.shape[-1]
    q = np.full(e_t.shape, -1, dtype=np.int32)
    for p in range(k):
        for slot in range(k):
            hit = (e_c[..., slot] == e_t[..., p]) & (e_c[..., slot] >= 0)
            q[..., p] = np.where(hit & (q[..., p] < 0), slot, q[..., p])
    return q >= 0, q


def score(w_t, w_c, n_c, e_c, q, matched, lambda1: float, lambda2: float,
          lambda0: float = 1.0):
    """Delta = |w_p - w_c[q]|,  o = n_c[q] / sum_{valid j} n_c[j],
    s = lambda0*w_p + lambda1*Delta + lambda2*o  (evaluated left to right in
    fp32; the score eq. of Sec. 4.2 has lambda0 = 1, and 0 drops the routing
    weight as in the score-signal ablation table of Sec. 5).

    The denominator is summed in fp64 and rounded once.  Unmatched branches
    get Delta = o = s = 0 (they are never scored).  Returns (Delta, o, s)."""
    qs = np.where(matched, q, 0)
    wc_q = np.take_along_axis(w_c, qs, axis=-1)
    nc_q = np.take_along_axis(n_c, qs, axis=-1)
    delta = np.abs((w_t - wc_q).astype(F32)).astype(F32)
    den = np.where(e_c >= 0, n_c.astype(F64), 0.0).sum(axis=-1).astype(F32)
    den_b = np.broadcast_to(den[..., None], w_t.shape)
    safe = np.where(den_b > 0, den_b, F32(1.0))
    o = np.where(den_b > 0, (nc_q / safe).astype(F32), F32(0.0)).astype(F32)
    s = ((F32(lambda0) * w_t).astype(F32) + (F32(lambda1) * delta).astype(F32)).astype(F32)
    s = (s + (F32(lambda2) * o).astype(F32)).astype(F32)
    zero = F32(0.0)
    return (np.where(matched, delta, zero), np.where(matched, o, zero),
            np.where(matched, s, zero))


def margins(s: np.ndarray, tau: np.ndarray, e_t: np.ndarray, matched) -> np.ndarray:
    """m = s - tau_{b, e_p} in fp32; +inf for unmatched branches.
    s, e_t: (B, N, k); tau: (B, E)."""
    B = s.shape[0]
    tau_p = tau[np.arange(B)[:, None, None], e_t]
    m = (s - tau_p).astype(F32)
    return np.where(matched, m, F32(np.inf)).astype(F32)


# ---------------------------------------------------------------------------
# 6. recomputation set (Sec. 4.2: unmatched -> recompute; s > tau)
# ---------------------------------------------------------------------------
def select_threshold(matched: np.ndarray, m: np.ndarray) -> np.ndarray:
    """R = unmatched  U  {matched with s > tau}  (s > tau  <=>  s - tau > 0)."""
    return (~matched) | (matched & (m > F32(0.0)))


def ratio_budget(ratio: float, N: int, k: int) -> int:
    """Per-sample branch budget K_b = floor(rho * N * k + 0.5), rho taken as
    the fp32 policy value widened to fp64."""
    return int(math.floor(float(F32(ratio)) * N * k + 0.5))


def select_ratio(matched: np.ndarray, m: np.ndarray, ratio: float) -> np.ndarray:
    """Per sample: every unmatched branch, plus the first max(0, K_b - |U_b|)
    matched branches ranked by margin descending, then flat id ascending."""
    B, N, k = matched.shape
    K = ratio_budget(ratio, N, k)
    mask = ~matched
    for b in range(B):
        mb = matched[b].reshape(-1)
        need = max(0, K - int((~mb).sum()))
        if need == 0:
            continue
        ids = np.flatnonzero(mb)                 # ascending flat ids
        keys = m[b].reshape(-1)[ids]
        order = np.lexsort((ids, -keys))         # margin desc, then id asc
        chosen = ids[order[:need]]
        flat = mask[b].reshape(-1)
        flat[chosen] = True
        mask[b] = flat.reshape(N, k)
    return mask


# ---------------------------------------------------------------------------
# 7. slot assignment
# ---------------------------------------------------------------------------
def assign_slots(matched: np.ndarray, q: np.ndarray, full: bool) -> np.ndarray:
    """sigma(p): the slot branch p occupies after this step.

    Full step: sigma(p) = p.  Cache step: matched branches keep their slot
    q(p); unmatched branches, in ascending p, take the slots no matched
    branch holds, in ascending slot order."""
    k = q.shape[-1]
    if full:
        return np.broadcast_to(np.arange(k, dtype=np.int32), q.shape).copy()
    flat_m = matched.reshape(-1, k)
    flat_q = q.reshape(-1, k)
    T = flat_m.shape[0]
    taken = np.zeros((T, k), dtype=bool)
    for p in range(k):
        rows = np.flatnonzero(flat_m[:, p])
        taken[rows, flat_q[rows, p]] = True
    free_sorted = np.argsort(taken, axis=1, kind="stable")   # free slots first, ascending
    unmatched_rank = np.cumsum(~flat_m, axis=1) - 1
    rank = np.where(flat_m, 0, unmatched_rank)
    free_pick = np.take_along_axis(free_sorted, rank, axis=1)
    sigma = np.where(flat_m, flat_q, free_pick).astype(np.int32)
    return sigma.reshape(q.shape)


# ---------------------------------------------------------------------------
# 8. per-expert lists of recomputed branches
# ---------------------------------------------------------------------------
def expert_lists(mask: np.ndarray, e_t: np.ndarray, E: int):
    """For each expert, the ascending flat ids f = (b*N + i)*k + p of the
    recomputed branches routed to it.  Returns (cnt[E], off[E+1], lst, pos)
    where pos[f] is f's index in lst or -1."""
    mf = mask.reshape(-1)
    ef = e_t.reshape(-1)
    parts = [np.flatnonzero(mf & (ef == e)).astype(np.int32) for e in range(E)]
    cnt = np.array([len(p) for p in parts], dtype=np.int32)
    off = np.zeros(E + 1, dtype=np.int32)
    off[1:] = np.cumsum(cnt)
    lst = np.concatenate(parts) if parts else np.zeros(0, np.int32)
    pos = np.full(mf.shape, -1, dtype=np.int32)
    pos[lst] = np.arange(lst.size, dtype=np.int32)
    return cnt, off, lst, pos


# ---------------------------------------------------------------------------
# 9. expert FFN (Sec. 2.3: FFN_e; GELU, or the gated SwiGLU form)
# ---------------------------------------------------------------------------
_SQRT_2_OVER_PI = math.sqrt(2.0 / math.pi)


def gelu(z: np.ndarray, kind: str) -> np.ndarray:
    """GELU in fp64: tanh form 0.5 z (1 + tanh(sqrt(2/pi)(z + 0.044715 z^3)))
    or the exact form 0.5 z (1 + erf(z / sqrt 2))."""
    if kind == "gelu_tanh":
        return 0.5 * z * (1.0 + np.tanh(_SQRT_2_OVER_PI * (z + 0.044715 * z ** 3)))
    if kind == "gelu_erf":
        from scipy.special import erf
        return 0.5 * z * (1.0 + erf(z / math.sqrt(2.0)))
    raise ValueError(kind)


def silu(z: np.ndarray) -> np.ndarray:
    """z * sigmoid(z) = z / (1 + exp(-z)) in fp64."""
    return z / (1.0 + np.exp(-z))


def expert_ffn(x_rows64: np.ndarray, Wup64: np.ndarray, Wdown64: np.ndarray,
               act: str, dtype: str) -> np.ndarray:
    """h = W_down . g(W_up . x): fp64 contractions, the activation and the
    output each rounded to the stored dtype.  Rows in, rows out.  For the
    gated form (``act == "swiglu"``) W_up holds 2 d_ff rows, gate and up
    interleaved, and g = silu(gate) * up."""
    z = x_rows64 @ Wup64.T
    if act == "swiglu":
        g = silu(z[:, 0::2]) * z[:, 1::2]
    else:
        g = gelu(z, act)
    g = to_f64(round_act(g, dtype), dtype)
    return round_act(g @ Wdown64.T, dtype)


def row_norms(h: np.ndarray, dtype: str) -> np.ndarray:
    """||h|| of stored rows: squares summed in fp64, sqrt, rounded to fp32."""
    h64 = to_f64(h, dtype)
    return np.sqrt(np.sum(h64 * h64, axis=-1)).astype(F32)


# ---------------------------------------------------------------------------
# 10. combine (Sec. 4.1 output eq.)
# ---------------------------------------------------------------------------
def combine(w_t: np.ndarray, hhat: np.ndarray, dtype: str, shared=()) -> np.ndarray:
    """y = sum_s h_s + sum_p f32(w_p * hhat_p), accumulated in fp32 (shared
    experts first, in order, then the branches in order), then rounded to
    the stored dtype.  w_t: (T, k); hhat: (T, k, d) stored; shared: stored
    (T, d) outputs of the shared experts."""
    T, k = w_t.shape
    y = np.zeros((T, hhat.shape[-1]), dtype=F32)
    for hs in shared:
        y = (y + to_f32(hs, dtype)).astype(F32)
    for p in range(k):
        prod = (w_t[:, p, None] * to_f32(hhat[:, p, :], dtype)).astype(F32)
        y = (y + prod).astype(F32)
    return round_act(y.astype(F64), dtype)


# ---------------------------------------------------------------------------
# the whole step
# ---------------------------------------------------------------------------
def step(dims: Dims, policy: Policy, W: Weights, state: State, x_t: np.ndarray,
         t: int, attn_in: np.ndarray | None = None, tokens=None,
         x_ffn: np.ndarray | None = None, forced: dict | None = None):
    """One layer step at sampling step ``t``.

    ``x_ffn`` (same shape and dtype as ``x_t``), when given, is the input of
    the expert FFNs while the router still reads ``x_t``: inside a block the
    routing input of a cache step is built from the cached attention feature
    and the recomputed branches read the refreshed one.

    ``state`` is not modified; the new state is returned.  ``tokens`` (flat
    token indices) limits the expert FFN, combine and row writes to those
    tokens (the decision path always runs over the whole batch); outputs and
    rows of other tokens are then left unset (``rec['evaluated']``).

    ``forced`` (test use only) replaces one rounded decision input by a value
    computed elsewhere and runs every later step of the method on it
    unchanged: ``"logits"`` (T, E) fp32 router logits, ``"Hbar"`` (B, E)
    fp32 normalised entropies.  Where an fp64 result lies at an fp32
    rounding tie either rounding is correct, so a checker adopts the other
    side's value there and still compares everything that follows.

    Returns ``(out, new_state, rec)``: ``out`` (B, N, d) stored dtype;
    ``rec`` a dict of every intermediate of the step.
    """
    B, N, k, d, E = dims.B, dims.N, dims.k, dims.d, dims.E
    dt = dims.dtype
    T = B * N
    full = is_full_step(policy, state.valid, t)
    uncached = policy.mode == MODE_FULL
    rec = {"full": full}

    # 2. router
    forced = forced or {}
    x64 = to_f64(x_t, dt).reshape(T, d)
    l64, logits = router_logits(x64, W.W_r64, W.b_r)
    if "logits" in forced:
        logits = np.asarray(forced["logits"], dtype=F32).reshape(T, E)
    e_flat, w_flat = route(logits, k, policy.norm_topk)
    e_t = e_flat.reshape(B, N, k)
    w_t = w_flat.reshape(B, N, k)
    rec.update(logits64=l64, logits=logits, e_t=e_t, w_t=w_t)

    new = state.copy()
    if not uncached:
        # 3-4. statistic and thresholds
        new.C = ema_update(state.C, e_t, policy.beta)
        Hbar = normalized_entropy(new.C)
        if "Hbar" in forced:
            Hbar = np.asarray(forced["Hbar"], dtype=F32).reshape(B, E)
        tau = adaptive_threshold(Hbar, policy.tau0, policy.alpha)
        rec.update(C=new.C, Hbar=Hbar, tau=tau)

    # 5-6. matching, scores, recomputation set
    if full:
        matched = np.zeros((B, N, k), dtype=bool)
        q = np.full((B, N, k), -1, dtype=np.int32)
        m = np.full((B, N, k), np.inf, dtype=F32)
        mask = np.ones((B, N, k), dtype=bool)
    else:
        matched, q = match(e_t, state.e_c)
        _, _, s = score(w_t, state.w_c, state.n_c, state.e_c, q, matched,
                        policy.lambda1, policy.lambda2, policy.lambda0)
        m = margins(s, tau, e_t, matched)
        rec["s"] = s
        if policy.mode == MODE_THRESHOLD:
            mask = select_threshold(matched, m)
        else:
            mask = select_ratio(matched, m, policy.ratio)
    S = mask.any(axis=2)
    sigma = assign_slots(matched, q, full)
    rec.update(matched=matched, q=q, m=m, mask=mask, S=S, sigma=sigma)

    # 8. lists
    cnt, off, lst, pos = expert_lists(mask, e_t, E)
    rec.update(cnt=cnt, off=off, lst=lst, pos=pos)

    # which tokens get FFN / combine / row writes
    evaluated = np.ones(T, dtype=bool) if tokens is None else np.zeros(T, dtype=bool)
    if tokens is not None:
        evaluated[np.asarray(tokens)] = True
    rec["evaluated"] = evaluated.reshape(B, N)

    # 9. expert FFN on the recomputed branches of evaluated tokens
    xf64 = x64 if x_ffn is None else to_f64(x_ffn, dt).reshape(T, d)
    act_t = np.uint16 if dt == BF16 else F32
    h_new = np.zeros((B * N * k, d), dtype=act_t)
    for e in range(E):
        f = lst[off[e]:off[e + 1]]
        f = f[evaluated[f // k]]
        if f.size == 0:
            continue
        h_new[f] = expert_ffn(xf64[f // k], W.up64(e), W.down64(e), policy.act, dt)
    h_new = h_new.reshape(B, N, k, d)
    rec["h_new"] = h_new

    # shared experts (Sec. 2.3 shared-expert eq.): every evaluated token
    ev = evaluated
    shared = [expert_ffn(xf64[ev], W.shared_up64(s_), W.shared_down64(s_), policy.act, dt)
              for s_ in range(dims.n_shared)]
    rec["h_shared"] = shared

    # 10. combine: recomputed -> new feature, reused -> cached feature q(p)
    hc_q = np.take_along_axis(state.h_c, np.where(matched, q, 0)[..., None], axis=2)
    hhat = np.where(mask[..., None], h_new, hc_q)
    out = np.zeros((T, d), dtype=act_t)
    out[ev] = combine(w_t.reshape(T, k)[ev], hhat.reshape(T, k, d)[ev], dt, shared)
    out = out.reshape(B, N, d)

    # 11. cache write (not for the uncached comparator)
    if not uncached:
        bb, ii, pp = np.nonzero(mask)
        ss = sigma[bb, ii, pp]
        new.e_c[bb, ii, ss] = e_t[bb, ii, pp]
        new.w_c[bb, ii, ss] = w_t[bb, ii, pp]
        okr = evaluated.reshape(B, N)[bb, ii]
        new.h_c[bb[okr], ii[okr], ss[okr]] = h_new[bb[okr], ii[okr], pp[okr]]
        norms = np.full(bb.shape, np.nan, dtype=F32)
        norms[okr] = row_norms(h_new[bb[okr], ii[okr], pp[okr]], dt)
        new.n_c[bb, ii, ss] = norms
        new.valid = True
        if new.A is not None and attn_in is not None:
            new.A[S] = attn_in[S]

    nm = int(matched.sum())
    reused = int((matched & ~mask).sum())
    rec["stats"] = {
        "n_recompute": int(mask.sum()),
        "n_unmatched": 0 if full else int((~matched).sum()),
        "n_matched": nm,
        "n_reused": reused,
        "n_sync": int(S.sum()),
        "reuse_over_match": (reused / nm) if nm else 0.0,
    }
    return out, new, rec


def uncached_layer(dims: Dims, W: Weights, x_t: np.ndarray, norm_topk: bool = True,
                   act: str = "gelu_tanh") -> np.ndarray:
    """The plain MoE layer output sum_s FFN_s(x) + sum_p w_p FFN_{e_p}(x)
    (Sec. 2.3), i.e. a step in the uncached comparator mode."""
    pol = Policy(mode=MODE_FULL, norm_topk=norm_topk, act=act)
    out, _, _ = step(dims, pol, W, State(dims), x_t, 0)
    return out
