"""Pins of the block-stack oracle (``oracle/dit_block_oracle.py``) against
library routines, closed forms and invariants that do not use the oracle's
own formulas.  CPU only."""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

from oracle import dit_block_oracle as D
from oracle import moeca_oracle as O
from paper_2606_15615_amd.synth import (STACKS, StackShape, StackSynth, bf16_bits_to_fp32,
                                        fp32_to_bf16_bits)

TINY = StackShape(L=2, d=128, heads=2, E=4, k=2, d_ff=64, B=2, N=24)


def make_blocks(sh: StackShape, seed: int = 0):
    syn = StackSynth(sh, seed)
    dims = D.BlockDims(sh.d, sh.heads, sh.E, sh.k, sh.d_ff, sh.B, sh.N)
    blocks = []
    for l in range(sh.L):
        w = syn.block(l)
        moe = O.Weights(dims.layer(), w["W_r"], None, w["W_up"], w["W_down"])
        blocks.append(D.BlockWeights(w["W_ada"], w["b_ada"], w["W_qkv"], w["b_qkv"], w["W_o"],
                                     w["b_o"], moe))
    return syn, dims, blocks


def cond(syn: StackSynth, t_val: float) -> np.ndarray:
    e = syn.embedder()
    lab = syn.labels()
    return D.cond_embed(np.full(syn.shape.B, t_val, np.float32), e["W1"], e["b1"], e["W2"],
                        e["b2"], e["table"][lab])


def f64(bits):
    return bf16_bits_to_fp32(bits).astype(np.float64)


# ---- pieces against library routines -------------------------------------
def test_layer_norm_matches_torch():
    x = np.random.default_rng(0).standard_normal((7, 96)) * 3 + 1.5
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (96,), eps=1e-6).numpy()
    np.testing.assert_allclose(D.layer_norm(x), ref, rtol=0, atol=1e-12)


def test_attention_matches_torch_sdpa():
    g = np.random.default_rng(1)
    heads, dh, nq, n = 3, 72, 10, 37
    q, k, v = (fp32_to_bf16_bits(g.standard_normal((m, heads * dh), dtype=np.float32))
               for m in (nq, n, n))
    got = f64(D.attention(q, k, v, heads))
    tq, tk, tv = (torch.from_numpy(f64(a)).reshape(-1, heads, dh).transpose(0, 1) for a in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv)
    ref = ref.transpose(0, 1).reshape(nq, heads * dh).numpy()
    # the oracle rounds once to bf16: within half a bf16 ulp of the exact value
    assert np.all(np.abs(got - ref) <= np.abs(ref) * 2.0 ** -8 + 1e-30)


def test_attention_closed_forms():
    g = np.random.default_rng(2)
    d, n = 16, 9
    v = fp32_to_bf16_bits(g.standard_normal((n, d), dtype=np.float32))
    # identical keys: uniform weights, the output is the mean of the values
    k = np.tile(fp32_to_bf16_bits(g.standard_normal((1, d), dtype=np.float32)), (n, 1))
    q = fp32_to_bf16_bits(g.standard_normal((2, d), dtype=np.float32))
    out = f64(D.attention(q, k, v, 1))
    np.testing.assert_allclose(out, np.tile(f64(v).mean(0), (2, 1)), rtol=2 ** -8, atol=1e-6)
    # one key aligned with a large query dominates: the output is its value
    k2 = np.zeros((n, d), np.float32)
    k2[4, 0] = 1.0
    q2 = np.zeros((1, d), np.float32)
    q2[0, 0] = 400.0
    out2 = D.attention(fp32_to_bf16_bits(q2), fp32_to_bf16_bits(k2), v, 1)
    assert np.array_equal(out2[0], v[4])


def test_timestep_embedding_closed_form():
    t = np.array([0.0, 1.0, 250.0, 999.0])
    e = D.timestep_embedding(t)
    assert e.shape == (4, 256)
    np.testing.assert_array_equal(e[0], np.r_[np.ones(128), np.zeros(128)])
    np.testing.assert_allclose(e[:, 0], np.cos(t), atol=1e-15)      # f_0 = 1
    np.testing.assert_allclose(e[:, 128], np.sin(t), atol=1e-15)
    np.testing.assert_allclose(e[:, 64], np.cos(t / 100.0), atol=1e-15)  # f_64 = 10^-2


def test_cond_embed_matches_torch_modules():
    syn, _, _ = make_blocks(TINY)
    e = syn.embedder()
    lab = syn.labels()
    t = np.array([999.0, 17.0], np.float32)
    got = D.cond_embed(t, e["W1"], e["b1"], e["W2"], e["b2"], e["table"][lab])
    l1 = torch.nn.Linear(256, TINY.d, dtype=torch.float64)
    l2 = torch.nn.Linear(TINY.d, TINY.d, dtype=torch.float64)
    with torch.no_grad():
        l1.weight.copy_(torch.from_numpy(f64(e["W1"])))
        l1.bias.copy_(torch.from_numpy(e["b1"].astype(np.float64)))
        l2.weight.copy_(torch.from_numpy(f64(e["W2"])))
        l2.bias.copy_(torch.from_numpy(e["b2"].astype(np.float64)))
        half = 128
        f = torch.exp(-math.log(10000.0) * torch.arange(half, dtype=torch.float64) / half)
        arg = torch.from_numpy(t.astype(np.float64))[:, None] * f[None]
        emb = torch.cat([torch.cos(arg), torch.sin(arg)], dim=1)
        ref = l2(torch.nn.functional.silu(l1(emb))) + torch.from_numpy(f64(e["table"][lab]))
    np.testing.assert_allclose(got, ref.numpy().astype(np.float32), rtol=1e-6, atol=1e-6)


# ---- the block --------------------------------------------------------------
def torch_block(dims, W: D.BlockWeights, x: np.ndarray, mod: np.ndarray) -> np.ndarray:
    """The uncached block from torch's LayerNorm and MultiheadAttention
    modules (fp64), the layer oracle's uncached MoE layer for the MoE FFN."""
    d = dims.d
    mha = torch.nn.MultiheadAttention(d, dims.heads, batch_first=True, dtype=torch.float64)
    with torch.no_grad():
        mha.in_proj_weight.copy_(torch.from_numpy(f64(W.W_qkv)))
        mha.in_proj_bias.copy_(torch.from_numpy(W.b_qkv.astype(np.float64)))
        mha.out_proj.weight.copy_(torch.from_numpy(f64(W.W_o)))
        mha.out_proj.bias.copy_(torch.from_numpy(W.b_o.astype(np.float64)))
        m = torch.from_numpy(mod.astype(np.float64))
        xt = torch.from_numpy(x.astype(np.float64))
        ln = lambda z: torch.nn.functional.layer_norm(z, (d,), eps=1e-6)
        h = ln(xt) * (1 + m[:, 1, None]) + m[:, 0, None]
        a, _ = mha(h, h, h, need_weights=False)
        x1 = xt + m[:, 2, None] * a
        u = ln(x1) * (1 + m[:, 4, None]) + m[:, 3, None]
        u_bits = fp32_to_bf16_bits(u.numpy().astype(np.float32))
        y = O.uncached_layer(dims.layer(), W.moe, u_bits)
        return (x1 + m[:, 5, None] * torch.from_numpy(f64(y))).numpy()


def test_full_block_matches_torch_modules():
    syn, dims, blocks = make_blocks(TINY, seed=3)
    x = next(syn.trajectory(1))
    c = cond(syn, 999.0)
    mod = D.adaln(blocks[0].W_ada, blocks[0].b_ada, c)
    pol = O.Policy(mode=O.MODE_FULL)
    got, _, _ = D.block_step(dims, pol, blocks[0], D.BlockState(dims), x, mod, 0)
    ref = torch_block(dims, blocks[0], x, mod)
    # bf16 rounding of h, q, k, v, o, a, u, y on the oracle's side only
    err = np.abs(got - ref).max() / np.abs(ref).max()
    assert err < 2e-2, err


def test_zero_gates_give_identity():
    syn, dims, blocks = make_blocks(TINY, seed=4)
    W = blocks[0]
    W0 = D.BlockWeights(np.zeros_like(W.W_ada), np.zeros_like(W.b_ada), W.W_qkv, W.b_qkv,
                        W.W_o, W.b_o, W.moe)
    c = cond(syn, 500.0)
    mod = D.adaln(W0.W_ada, W0.b_ada, c)
    assert not mod.any()
    st = D.BlockState(dims)
    for t, x in enumerate(syn.trajectory(3)):
        out, st, _ = D.block_step(dims, O.Policy(mode=O.MODE_RATIO, ratio=0.3), W0, st, x, mod, t)
        np.testing.assert_array_equal(out, x)


@pytest.mark.parametrize("pol", [O.Policy(mode=O.MODE_RATIO, ratio=1.0),
                                 O.Policy(mode=O.MODE_RATIO, ratio=0.0),
                                 O.Policy(mode=O.MODE_THRESHOLD)])
def test_cache_step_with_unchanged_input_is_bit_identical(pol):
    """x and c unchanged since the full step: the cached attention feature
    is the fresh one, so the routing input, the routing and every reused or
    recomputed branch are the full step's, whatever the policy."""
    syn, dims, blocks = make_blocks(TINY, seed=5)
    x = next(syn.trajectory(1))
    c = cond(syn, 800.0)
    mod = D.adaln(blocks[0].W_ada, blocks[0].b_ada, c)
    out0, st, r0 = D.block_step(dims, pol, blocks[0], D.BlockState(dims), x, mod, 0)
    assert r0["full"]
    out1, st1, r1 = D.block_step(dims, pol, blocks[0], st, x, mod, 1)
    assert not r1["full"]
    np.testing.assert_array_equal(r1["u_route"], r0["u"])
    np.testing.assert_array_equal(out1, out0)
    if pol.mode == O.MODE_RATIO and pol.ratio == 0.0:
        assert not r1["sync"].any()            # every branch matched and reused
    if pol.mode == O.MODE_RATIO and pol.ratio == 1.0:
        assert r1["sync"].all()


def test_cache_step_refreshes_only_synchronised_tokens():
    syn, dims, blocks = make_blocks(TINY, seed=6)
    traj = list(syn.trajectory(2))
    c = cond(syn, 600.0)
    mod = D.adaln(blocks[0].W_ada, blocks[0].b_ada, c)
    pol = O.Policy(mode=O.MODE_RATIO, ratio=0.3)
    _, st, _ = D.block_step(dims, pol, blocks[0], D.BlockState(dims), traj[0], mod, 0)
    # a strongly changed input for a few tokens
    x = traj[1].copy()
    x[0, :5] += 3.0
    _, st1, r = D.block_step(dims, pol, blocks[0], st, x, mod, 1)
    S = r["sync"]
    assert S.any() and not S.all()
    np.testing.assert_array_equal(st1.a[~S], st.a[~S])
    np.testing.assert_array_equal(r["x1"][~S], r["x1_pre"][~S])
    np.testing.assert_array_equal(r["u"][~S], r["u_route"][~S])
    # refreshed tokens: the attention of their queries over every token
    dh = dims.d // dims.heads
    b, i = np.argwhere(S)[0]
    ref = D.attention(r["q"][b, i:i + 1], r["k"][b], r["v"][b], dims.heads)
    np.testing.assert_array_equal(r["o"][b, i], ref[0])
    assert dh * dims.heads == dims.d
    # a token with a recomputed branch is synchronised
    assert np.all(r["moe"]["mask"].any(axis=2) == S)


def test_stack_step_chains_blocks():
    syn, dims, blocks = make_blocks(TINY, seed=7)
    x = next(syn.trajectory(1))
    c = cond(syn, 999.0)
    pol = O.Policy(mode=O.MODE_RATIO, ratio=0.3)
    states = [D.BlockState(dims) for _ in blocks]
    out, _, recs = D.stack_step(dims, pol, blocks, states, x, c, 0)
    xb = x
    for W, st in zip(blocks, states):
        xb, _, _ = D.block_step(dims, pol, W, st, xb, D.adaln(W.W_ada, W.b_ada, c), 0)
    np.testing.assert_array_equal(out, xb)


def test_named_stacks_are_consistent():
    for sh in STACKS.values():
        assert sh.d % sh.heads == 0 and (sh.d // sh.heads) % 8 == 0 and sh.d % 64 == 0


def test_adaln_matches_torch_modules():
    syn, dims, blocks = make_blocks(TINY, seed=8)
    W = blocks[0]
    c = cond(syn, 321.0)
    got = D.adaln(W.W_ada, W.b_ada, c)
    lin = torch.nn.Linear(TINY.d, 6 * TINY.d, dtype=torch.float64)
    with torch.no_grad():
        lin.weight.copy_(torch.from_numpy(f64(W.W_ada)))
        lin.bias.copy_(torch.from_numpy(W.b_ada.astype(np.float64)))
        ref = lin(torch.nn.functional.silu(torch.from_numpy(c.astype(np.float64))))
    np.testing.assert_array_equal(got, ref.numpy().astype(np.float32).reshape(TINY.B, 6, TINY.d))


def test_full_refresh_cache_step_equals_full_step_for_refreshed_parts():
    """At ratio 1 every token is synchronised and every branch recomputed: the
    cache step's attention feature and rebuilt MoE input equal the full
    step's on the same input, and for each token every expert selected in
    both steps has the same cached row (the FFN of the rebuilt input)."""
    syn, dims, blocks = make_blocks(TINY, seed=9)
    traj = list(syn.trajectory(2))
    W = blocks[0]
    mod = D.adaln(W.W_ada, W.b_ada, cond(syn, 700.0))
    pol = O.Policy(mode=O.MODE_RATIO, ratio=1.0)
    _, st, _ = D.block_step(dims, pol, W, D.BlockState(dims), traj[0], mod, 0)
    x = traj[1].copy()
    x[:, :6] += 1.5          # a clearly changed input for some tokens
    _, st_c, rc = D.block_step(dims, pol, W, st, x, mod, 1)
    _, st_f, rf = D.block_step(dims, pol, W, D.BlockState(dims), x, mod, 0)
    assert not rc["full"] and rf["full"] and rc["sync"].all()
    np.testing.assert_array_equal(st_c.a, st_f.a)
    np.testing.assert_array_equal(rc["u"], rf["u"])
    np.testing.assert_array_equal(rc["x1"], rf["x1"])
    same = 0
    for b in range(dims.B):
        for i in range(dims.N):
            for e in set(st_c.moe.e_c[b, i]) & set(st_f.moe.e_c[b, i]):
                qc = int(np.flatnonzero(st_c.moe.e_c[b, i] == e)[0])
                qf = int(np.flatnonzero(st_f.moe.e_c[b, i] == e)[0])
                np.testing.assert_array_equal(st_c.moe.h_c[b, i, qc], st_f.moe.h_c[b, i, qf])
                same += 1
    assert same > dims.B * dims.N   # most tokens keep at least one expert
