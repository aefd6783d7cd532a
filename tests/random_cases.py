"""Seeded random layer configurations for the GPU parity sweep.

Each case draws a layer shape and a controller policy inside the limits
moeca_layer_create accepts (width and hidden width multiples of 64, 1 to 64
experts, k up to min(E, 8), up to 8 shared experts, GELU (tanh or erf) or
SwiGLU experts, bf16 or fp32), small enough that the oracle evaluates every
step whole in a second or two.  The draws are a plain function of the case
number, so a failing case is reproduced by its number alone.
"""
from __future__ import annotations

import math

import numpy as np

from paper_2606_15615_amd.synth import LayerShape

N_CASES = 40


def case(i: int):
    """(shape, mode, policy kwargs, steps, router bias) of case i."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([20261, i])))
    d = 64 * int(g.integers(1, 13))
    E = int(g.choice([1, 2, 3, 5, 8, 12, 16, 24, 33, 64]))
    k = int(g.choice([kk for kk in (1, 2, 3, 4, 6, 8) if kk <= E]))
    ffn = "swiglu" if g.random() < 0.3 else "gelu"
    d_ff = 64 * int(g.integers(1, 9))
    n_shared = int(g.choice([0, 0, 0, 1, 2])) if ffn == "swiglu" or g.random() < 0.3 else 0
    B = int(g.integers(1, 5)) if i % 3 else int(g.integers(1, 3))
    N = int(g.integers(1, 161)) if i % 3 else int(g.integers(161, 1200))
    dtype = "fp32" if i % 4 == 3 else "bf16"
    mode = str(g.choice(["ratio", "threshold", "full"], p=[0.5, 0.3, 0.2]))
    pol = dict(
        ratio=float(np.float32(g.choice([0.0, 1.0, g.uniform(0.02, 0.98)], p=[0.1, 0.1, 0.8]))),
        tau0=float(np.float32(g.uniform(0.05, 1.2))),
        alpha=float(np.float32(g.uniform(0.0, 0.95))),
        beta=float(np.float32(g.uniform(0.0, 0.95))),
        lambda1=float(np.float32(g.uniform(0.0, 2.0))),
        lambda2=float(np.float32(g.uniform(0.0, 2.0))),
        lambda0=float(np.float32(g.uniform(0.0, 2.0))),
        refresh_cycle=int(g.choice([0, 2, 3, 5])),
        norm_topk=bool(g.random() < 0.7),
    )
    if ffn == "gelu" and g.random() < 0.3:
        pol["act"] = "gelu_erf"
    bias = "zipf" if g.random() < 0.25 else None
    steps = int(g.integers(3, 6))
    shape = LayerShape(d=d, E=E, k=k, d_ff=d_ff, B=B, N=N, dtype=dtype, ffn=ffn,
                       n_shared=n_shared)
    return shape, mode, pol, steps, bias


N_PLAN_CASES = 12


def plan_case(j: int):
    """(shape, policy kwargs, steps, plan) of a ratio-mode case drawn so that
    its cache steps take the weight-streaming FFN plan (j even: few rows per
    expert, 2 E ceil(d_ff / 288) >= 256 column tiles) or the expert-wide up
    projection (j odd: a hidden width that is a multiple of 576 and 112-320
    recomputed rows per expert on average).  The first step is a full step."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([20262, j])))
    d = 64 * int(g.integers(2, 11))
    k = int(g.choice([1, 2, 4]))
    act = "gelu_erf" if g.random() < 0.3 else "gelu_tanh"
    if j % 2 == 0:
        E = int(g.choice([16, 32, 64]))
        nt_min = -(-128 // E)                       # column tiles of 288
        d_ff = 64 * int(g.integers(-(-(288 * (nt_min - 1) + 1) // 64), 288 * nt_min // 64 + 1))
        B = int(g.integers(1, 5))
        N = int(g.integers(max(k, 8), 256 * E // (B * k) + 1))
        hi = min(0.95, 112 * E / (B * N * k))
        ratio = float(np.float32(g.uniform(0.02, hi)))
        plan = 1
    else:
        E = int(g.choice([4, 8, 16]))
        d_ff = 576 * int(g.integers(1, 4))
        B = int(g.integers(1, 4))
        ratio = float(np.float32(g.uniform(0.2, 0.7)))
        # recomputed rows per expert between 150 and 300
        rows = int(g.integers(150, 301)) * E
        N = max(1, int(round(rows / (ratio * B * k))))
        plan = 2
    pol = dict(ratio=ratio, refresh_cycle=0, act=act,
               tau0=float(np.float32(g.uniform(0.2, 1.0))),
               alpha=float(np.float32(g.uniform(0.0, 0.9))),
               beta=float(np.float32(g.uniform(0.0, 0.9))),
               norm_topk=bool(g.random() < 0.7))
    steps = int(g.integers(3, 5))
    shape = LayerShape(d=d, E=E, k=k, d_ff=d_ff, B=B, N=N, dtype="bf16")
    return shape, pol, steps, plan


N_STACK_CASES = 12


def stack_case(i: int):
    """(stack shape, mode, policy kwargs, steps) of a small block stack: the
    head widths 8-96 in steps of 8 (d = heads x head width a multiple of 64,
    at most 1152), one or two blocks, ragged token counts."""
    from paper_2606_15615_amd.synth import StackShape
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([20263, i])))
    dh = 8 * (1 + (5 * i) % 12)                      # every head width once per 12 cases
    step = 64 // math.gcd(dh, 64)                     # heads: d = heads dh a multiple of 64
    heads = step * int(g.integers(1, max(1, 1152 // (dh * step)) + 1))
    d = dh * heads
    E = int(g.choice([2, 3, 4, 8, 12, 16]))
    k = int(g.choice([kk for kk in (1, 2, 4) if kk <= E]))
    d_ff = 64 * int(g.integers(1, 9))
    L = int(g.integers(1, 3))
    B = int(g.integers(1, 4))
    N = int(g.integers(1, 300))
    mode = str(g.choice(["ratio", "threshold", "full"], p=[0.5, 0.35, 0.15]))
    pol = dict(ratio=float(np.float32(g.uniform(0.0, 1.0))),
               tau0=float(np.float32(g.uniform(0.2, 1.0))),
               alpha=float(np.float32(g.uniform(0.0, 0.9))),
               beta=float(np.float32(g.uniform(0.0, 0.9))),
               refresh_cycle=int(g.choice([0, 2, 3])))
    steps = int(g.integers(2, 5))
    return StackShape(L=L, d=d, heads=heads, E=E, k=k, d_ff=d_ff, B=B, N=N), mode, pol, steps
