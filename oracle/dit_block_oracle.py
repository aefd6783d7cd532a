"""CPU oracle for a stack of DiT-MoE blocks under branch-level caching.

TEST INFRASTRUCTURE ONLY.  Like ``moeca_oracle`` (whose layer step it
calls for the MoE sublayer), this module is the slow, plain reference the
GPU library is checked against.  Only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import it.  It shares no
code, header, table or helper with the HIP path.

What a block computes (Sec. 2.1, composition eq. and residual form; the MoE
FFN of Sec. 2.3):

    x1 = x  + g_a * a,   a = Attn(modulate(LN(x),  shift_a, scale_a))
    x' = x1 + g_m * y,   y = MoE (modulate(LN(x1), shift_m, scale_m))

with modulate(n, shift, scale) = n * (1 + scale) + shift and the six
per-sample vectors (shift_a, scale_a, g_a, shift_m, scale_m, g_m) given by
one linear map of SiLU(c) (AdaLN conditioned on the timestep and class
embedding c).  Attn is multi-head self-attention over the tokens of a
sample, softmax(q k^T / sqrt(d_h)) v per head, between a joint q/k/v
projection and an output projection.  The conditioning vector c comes from
a sinusoidal embedding of the timestep (cos of the first half of the
frequencies, then sin), a Linear-SiLU-Linear map, plus a class embedding row.

Caching across the block (Sec. 4.1).  The per-token cache holds the MoE
branch states (the layer oracle's State) and the attention feature a_i.  A
full-computation step runs the block as written above and overwrites both.
A cache step:

1. builds the routing input from the cached attention feature:
   x1_pre = x + g_a * a_cached, u_pre = modulate(LN(x1_pre), ...);
2. routes on u_pre, matches, scores and selects (Sec. 4.2-4.3), giving the
   recomputation sets R_i and the synchronised tokens S_i = [R_i non-empty];
3. refreshes the attention path of the tokens in S only (Sec. 4.1,
   synchronised update): their queries attend to the keys and values of
   every token of the sample at the current step; a_cached[S] is replaced,
   and x1 and u of those tokens are rebuilt from the new a;
4. runs the expert FFN of the recomputed branches on the rebuilt u (every
   token with a recomputed branch is in S) and combines (Sec. 4.1 output
   eq.) with the reused cached branches;
5. x' = x1 + g_m * y.
Tokens outside S keep their cached attention feature and every branch.

Readings where the paper is silent (listed with the layer's readings):
B-1 AdaLN as in the DiT convention: six d-vectors from Linear(SiLU(c)) in
    the order shift_a, scale_a, g_a, shift_m, scale_m, g_m; LayerNorm
    without affine parameters, eps 1e-6;
B-2 the attention feature a_i is the attention sublayer's output after
    its output projection and before its gate;
B-3 routing circularity: a cache step routes on the input built from the
    cached a_i (step 1), because the MoE sublayer's input depends on the
    attention output the cache is meant to skip; the recomputed branches
    then read the refreshed input (step 4);
B-4 a refreshed query attends to keys and values computed from every
    token's current input (the current sequence, not cached keys);
B-5 precision: the residual stream x, x1, x' and the AdaLN vectors are
    fp32; the attention input h, q/k/v, the attention output o, a, u and
    y are rounded to bf16 (round to nearest even) where they are produced;
    contractions, LayerNorm statistics and the softmax are fp64 here;
B-6 timestep embedding: 256 frequencies exp(-ln(10^4) j / 128), j < 128,
    of the timestep value, [cos, sin], then Linear-SiLU-Linear.

Pins: ``tests/test_block_oracle_pins.py`` (library attention and layer
norm, closed forms of the embedding, the zero-gate identity, bit-identity
of a cache step with an unchanged input, and a block written with torch's
own multi-head attention module).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

from . import moeca_oracle as mo

F32 = np.float32
F64 = np.float64
BF16 = mo.BF16

LN_EPS = 1e-6
FREQ_DIM = 256
MAX_PERIOD = 10000.0


def bf16_f64(a: np.ndarray) -> np.ndarray:
    return mo.to_f64(a, BF16)


def to_bf16(v: np.ndarray) -> np.ndarray:
    return mo.round_act(v, BF16)


# ---------------------------------------------------------------------------
# conditioning: timestep embedding and AdaLN vectors (Sec. 2.1 AdaLN)
# ---------------------------------------------------------------------------
def timestep_embedding(t: np.ndarray, dim: int = FREQ_DIM,
                       max_period: float = MAX_PERIOD) -> np.ndarray:
    """[cos(t f_j), sin(t f_j)], f_j = max_period^(-j / (dim/2)), fp64."""
    half = dim // 2
    f = np.exp(-math.log(max_period) * np.arange(half, dtype=F64) / half)
    arg = np.asarray(t, dtype=F64)[:, None] * f[None, :]
    return np.concatenate([np.cos(arg), np.sin(arg)], axis=1)


def cond_embed(t: np.ndarray, W1, b1, W2, b2, y_rows=None) -> np.ndarray:
    """c = W2 silu(W1 emb(t) + b1) + b2 (+ class row), fp32 (B, d).
    W1 (d, 256) and W2 (d, d) bf16 bits; biases fp32; y_rows (B, d) bf16."""
    e = timestep_embedding(t)
    h1 = e @ bf16_f64(W1).T + np.asarray(b1, F64)
    c = mo.silu(h1) @ bf16_f64(W2).T + np.asarray(b2, F64)
    if y_rows is not None:
        c = c + bf16_f64(y_rows)
    return c.astype(F32)


def adaln_f64(W_ada, b_ada, c: np.ndarray) -> np.ndarray:
    """The six modulation vectors per sample before their one rounding:
    (B, 6, d) fp64 from W_ada (6d, d) bf16 and b_ada (6d,) fp32 applied to
    SiLU(c)."""
    B, d = c.shape
    m = mo.silu(np.asarray(c, F64)) @ bf16_f64(W_ada).T + np.asarray(b_ada, F64)
    return m.reshape(B, 6, d)


def adaln(W_ada, b_ada, c: np.ndarray) -> np.ndarray:
    """The six modulation vectors per sample, rounded once to fp32: (B, 6, d)."""
    return adaln_f64(W_ada, b_ada, c).astype(F32)


# ---------------------------------------------------------------------------
# sublayer pieces
# ---------------------------------------------------------------------------
def layer_norm(x64: np.ndarray, eps: float = LN_EPS) -> np.ndarray:
    """(x - mean) / sqrt(var + eps) over the last axis, population variance."""
    mu = x64.mean(axis=-1, keepdims=True)
    var = ((x64 - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x64 - mu) / np.sqrt(var + eps)


def modulated_ln(x: np.ndarray, shift: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """bf16(LN(x) * (1 + scale) + shift); x (..., d) fp32, shift/scale (d,)
    or broadcastable fp32."""
    n = layer_norm(np.asarray(x, F64))
    return to_bf16(n * (1.0 + np.asarray(scale, F64)) + np.asarray(shift, F64))


def linear_bf16(a_bits: np.ndarray, W, b) -> np.ndarray:
    """bf16(a W^T + b) for bf16 rows a."""
    return to_bf16(bf16_f64(a_bits) @ bf16_f64(W).T + np.asarray(b, F64))


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, heads: int) -> np.ndarray:
    """Multi-head attention of one sample: q (nq, d), k and v (n, d) bf16
    bits, head h on columns h d_h .. (h+1) d_h - 1; bf16 (nq, d) out."""
    nq, d = q.shape
    dh = d // heads
    q64, k64, v64 = bf16_f64(q), bf16_f64(k), bf16_f64(v)
    out = np.empty((nq, d), dtype=F64)
    for h in range(heads):
        cols = slice(h * dh, (h + 1) * dh)
        s = q64[:, cols] @ k64[:, cols].T / math.sqrt(dh)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[:, cols] = p @ v64[:, cols]
    return to_bf16(out)


def gated_residual(x: np.ndarray, g: np.ndarray, f_bits: np.ndarray) -> np.ndarray:
    """fp32(x + g * f): x fp32, g fp32 (d,), f bf16 bits."""
    return (np.asarray(x, F64) + np.asarray(g, F64) * bf16_f64(f_bits)).astype(F32)


# ---------------------------------------------------------------------------
# block configuration, weights and state
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class BlockDims:
    d: int
    heads: int
    E: int
    k: int
    d_ff: int
    B: int
    N: int

    def layer(self) -> mo.Dims:
        return mo.Dims(self.d, self.E, self.k, self.d_ff, self.B, self.N, BF16)


class BlockWeights:
    """One block: AdaLN (6d, d) + (6d,), joint q/k/v projection (3d, d) +
    (3d,) with rows q (heads in order), k, v; output projection (d, d) + (d,);
    the MoE layer's weights.  Matrices are bf16 bits, biases fp32."""

    def __init__(self, W_ada, b_ada, W_qkv, b_qkv, W_o, b_o, moe: mo.Weights):
        self.W_ada, self.b_ada = W_ada, np.asarray(b_ada, F32)
        self.W_qkv, self.b_qkv = W_qkv, np.asarray(b_qkv, F32)
        self.W_o, self.b_o = W_o, np.asarray(b_o, F32)
        self.moe = moe


class BlockState:
    """The cached attention feature a (B, N, d) bf16 bits and the MoE
    layer's cache; valid once a full step has run."""

    def __init__(self, dims: BlockDims):
        self.a = np.zeros((dims.B, dims.N, dims.d), dtype=np.uint16)
        self.moe = mo.State(dims.layer())

    def copy(self) -> "BlockState":
        s = BlockState.__new__(BlockState)
        s.a = self.a.copy()
        s.moe = self.moe.copy()
        return s


# ---------------------------------------------------------------------------
# one block step
# ---------------------------------------------------------------------------
def attention_refresh(dims: BlockDims, W: BlockWeights, h: np.ndarray, sync: np.ndarray):
    """q for the tokens in ``sync`` (B, N) bool, k and v for every token,
    attention of the synchronised queries, output projection.  Returns
    (q, k, v, o, a) with rows of unsynchronised tokens zero in q, o, a."""
    B, N, d = dims.B, dims.N, dims.d
    Wq, Wk, Wv = W.W_qkv[:d], W.W_qkv[d:2 * d], W.W_qkv[2 * d:]
    bq, bk, bv = W.b_qkv[:d], W.b_qkv[d:2 * d], W.b_qkv[2 * d:]
    q = np.zeros((B, N, d), np.uint16)
    o = np.zeros((B, N, d), np.uint16)
    a = np.zeros((B, N, d), np.uint16)
    k = linear_bf16(h, Wk, bk)
    v = linear_bf16(h, Wv, bv)
    for b in range(B):
        rows = np.nonzero(sync[b])[0]
        if rows.size == 0:
            continue
        q[b, rows] = linear_bf16(h[b, rows], Wq, bq)
        o[b, rows] = attention(q[b, rows], k[b], v[b], dims.heads)
        a[b, rows] = linear_bf16(o[b, rows], W.W_o, W.b_o)
    return q, k, v, o, a


def block_step(dims: BlockDims, policy: mo.Policy, W: BlockWeights, state: BlockState,
               x: np.ndarray, mod: np.ndarray, t: int):
    """One block at sampling step ``t``: x (B, N, d) fp32 in, mod (B, 6, d)
    fp32 from ``adaln``.  Returns (x_out, new_state, rec) with every
    intermediate in ``rec``; ``state`` is not modified."""
    B, N, d = dims.B, dims.N, dims.d
    sa, ca, ga = mod[:, 0, None, :], mod[:, 1, None, :], mod[:, 2, None, :]
    sm, cm, gm = mod[:, 3, None, :], mod[:, 4, None, :], mod[:, 5, None, :]
    ld = dims.layer()
    full = mo.is_full_step(policy, state.moe.valid, t)
    rec = {"full": full}
    new = state.copy()

    h = modulated_ln(x, sa, ca)
    rec["h"] = h
    if full:
        sync = np.ones((B, N), dtype=bool)
        q, k, v, o, a = attention_refresh(dims, W, h, sync)
        x1 = gated_residual(x, ga, a)
        u = modulated_ln(x1, sm, cm)
        u_route = u
        y, new.moe, mrec = mo.step(ld, policy, W.moe, state.moe, u, t)
        new.a = a
    else:
        x1_pre = gated_residual(x, ga, state.a)
        u_route = modulated_ln(x1_pre, sm, cm)
        # the decision alone first (no token evaluated), then the refresh
        _, _, drec = mo.step(ld, policy, W.moe, state.moe, u_route, t,
                             tokens=np.zeros(0, dtype=np.int64))
        sync = drec["S"]
        q, k, v, o, a_new = attention_refresh(dims, W, h, sync)
        a = np.where(sync[..., None], a_new, state.a)
        x1 = np.where(sync[..., None], gated_residual(x, ga, a), x1_pre)
        u = np.where(sync[..., None], modulated_ln(x1, sm, cm), u_route)
        y, new.moe, mrec = mo.step(ld, policy, W.moe, state.moe, u_route, t, x_ffn=u)
        new.a = a
        rec["x1_pre"] = x1_pre
    x_out = gated_residual(x1, gm, y)
    rec.update(sync=sync, q=q, k=k, v=v, o=o, a=a, x1=x1, u=u, u_route=u_route, y=y,
               moe=mrec, x_out=x_out)
    return x_out, new, rec


def stack_step(dims: BlockDims, policy: mo.Policy, blocks: list, states: list,
               x: np.ndarray, c: np.ndarray, t: int):
    """Every block in order; returns (x_out, new_states, recs)."""
    new_states, recs = [], []
    for W, st in zip(blocks, states):
        mod = adaln(W.W_ada, W.b_ada, c)
        x, ns, rec = block_step(dims, policy, W, st, x, mod, t)
        rec["mod"] = mod
        new_states.append(ns)
        recs.append(rec)
    return x, new_states, recs
