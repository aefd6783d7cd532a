"""GPU parity of the DiT-MoE block stack (attention + AdaLN + the cached MoE
layer per block) against the block oracle.

Protocol (oracle-forced, per block): the oracle runs its own trajectory.
Before each block step its state (the cached attention feature and the MoE
layer's cache) is written into the GPU stack, the oracle's block input goes
in, the GPU runs that one block, and:
* the AdaLN vectors and, on cache steps, the routing input u and x1 of the
  tokens outside S are bit-exact (decision-path arithmetic on both sides),
  so every MoE decision of a cache step is compared bit for bit (the layer
  checks of ``gpu_harness.check_step``); the attention input h is within one
  bf16 ulp;
* the attention path (k, v, q, attention output, a, x1, the rebuilt u), the
  MoE output y and the block output are within the bf16 tolerance (max
  relative error 2e-2 over the tensor);
* on full steps the routing input comes from the GPU's own attention output,
  so routing is compared where the oracle's top-k is not within that
  tolerance of a tie.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import dit_block_oracle as D
from oracle import moeca_oracle as O
from paper_2606_15615_amd.synth import STACKS, StackShape, StackSynth
from gpu_harness import TOL, check_step, near_f32_tie, rel_err, say

pytestmark = pytest.mark.gpu

BF = "bf16"


class StackSetup:
    def __init__(self, sh: StackShape, mode="ratio", seed=0, T=5, **pol):
        import torch
        from paper_2606_15615_amd import _lib
        from paper_2606_15615_amd.layer import np_to_device
        from paper_2606_15615_amd.stack import MoecaStack
        self.sh = sh
        self.syn = StackSynth(sh, seed)
        self.dims = D.BlockDims(sh.d, sh.heads, sh.E, sh.k, sh.d_ff, sh.B, sh.N)
        omode = {"full": O.MODE_FULL, "threshold": O.MODE_THRESHOLD, "ratio": O.MODE_RATIO}[mode]
        gmode = {"full": _lib.MOECA_MODE_FULL, "threshold": _lib.MOECA_MODE_THRESHOLD,
                 "ratio": _lib.MOECA_MODE_RATIO}[mode]
        self.pol = O.Policy(mode=omode, **pol)
        self.S = MoecaStack(sh.L, sh.d, sh.heads, sh.E, sh.k, sh.d_ff, batch=sh.B, tokens=sh.N,
                            mode=gmode, ratio=self.pol.ratio, tau0=self.pol.tau0,
                            alpha=self.pol.alpha, beta=self.pol.beta,
                            refresh_cycle=self.pol.refresh_cycle)
        dev = self.S.device
        self.blocks, self.dev_w = [], []
        for l in range(sh.L):
            w = self.syn.block(l)
            moe = O.Weights(self.dims.layer(), w["W_r"], None, w["W_up"], w["W_down"])
            self.blocks.append(D.BlockWeights(w["W_ada"], w["b_ada"], w["W_qkv"], w["b_qkv"],
                                              w["W_o"], w["b_o"], moe))
            tw = {k_: np_to_device(v, dev) for k_, v in w.items()}
            self.S.set_block(l, tw["W_ada"], tw["b_ada"], tw["W_qkv"], tw["b_qkv"], tw["W_o"],
                             tw["b_o"], tw["W_r"], None, tw["W_up"], tw["W_down"])
            self.dev_w.append(tw)
        emb = self.syn.embedder()
        lab = self.syn.labels()
        self.tvals = self.syn.timestep_values(T)
        self.cs = [D.cond_embed(np.full(sh.B, tv, np.float32), emb["W1"], emb["b1"], emb["W2"],
                                emb["b2"], emb["table"][lab]) for tv in self.tvals]
        self.xs = list(self.syn.trajectory(T))
        self.x_dev = torch.zeros((sh.B, sh.N, sh.d), dtype=torch.float32, device=dev)
        self.c_dev = torch.zeros((sh.B, sh.d), dtype=torch.float32, device=dev)
        self.S.reset()
        torch.cuda.synchronize()

    def import_block(self, l: int, st: D.BlockState):
        T, d = self.sh.B * self.sh.N, self.sh.d
        self.S.write("a", st.a.reshape(T, d), l)
        lay = self.S.layer(l)
        m = st.moe
        lay.write("e_c", m.e_c.reshape(-1))
        lay.write("w_c", m.w_c.reshape(-1))
        lay.write("n_c", m.n_c.reshape(-1))
        lay.write("h_c", m.h_c.reshape(-1, d))
        lay.write("stat", m.C)
        lay.set_valid(m.valid)
        return lay


class _LayerView:
    """The attributes ``gpu_harness.check_step`` reads, for a block's layer."""

    def __init__(self, lay, dims: O.Dims):
        self.layer = lay
        self.dims = dims
        self.attention = False

        class _Sh:
            dtype = BF
        self.shape = _Sh()

    def gpu_state(self):
        st = O.State(self.dims)
        L = self.layer
        st.e_c = L.read("e_c").reshape(st.e_c.shape)
        st.w_c = L.read("w_c").reshape(st.w_c.shape)
        st.n_c = L.read("n_c").reshape(st.n_c.shape)
        st.h_c = L.read("h_c").reshape(st.h_c.shape)
        st.C = L.read("stat")
        return st


def topk_safe(logits64: np.ndarray, k: int, err: float) -> np.ndarray:
    """Tokens whose k + 1 largest logits are pairwise more than 2 err apart
    (the selected set and the branch order p are then both determined)."""
    s = np.sort(logits64, axis=1)[:, ::-1][:, :k + 1]
    return np.all(s[:, :-1] - s[:, 1:] > 2 * err, axis=1)


def tag0(l: int, t: int) -> str:
    return f"block {l} t={t}"


def check_block(SS: StackSetup, l: int, t: int, st_o: D.BlockState, x: np.ndarray):
    """Run block l of step t on the GPU from the oracle's state and input and
    compare; returns the oracle's (x_out, new state)."""
    import torch
    sh, dims = SS.sh, SS.dims
    B, N, d, k = sh.B, sh.N, sh.d, sh.k
    T = B * N
    lay = SS.import_block(l, st_o)
    SS.x_dev.copy_(torch.from_numpy(x))
    SS.c_dev.copy_(torch.from_numpy(SS.cs[t]))
    SS.S.step_blocks(SS.x_dev, SS.c_dev, t, l, 1)
    torch.cuda.synchronize()
    W = SS.blocks[l]
    # decision-path arithmetic: bit-exact.  The AdaLN vectors are fp64 sums
    # rounded once to fp32; where the oracle's fp64 value sits within fp64
    # rounding noise of an fp32 midpoint the other neighbour is as correct,
    # and both sides then go on from the GPU's vectors
    m64 = D.adaln_f64(W.W_ada, W.b_ada, SS.cs[t])
    mod = m64.astype(np.float32)
    g_mod = SS.S.read("mod")[l]
    off = g_mod != mod
    if off.any():
        tie = near_f32_tie(m64)
        assert np.all(tie[off]), f"{tag0(l, t)}: AdaLN vectors differ in {int(off.sum())} " \
            f"values, {int((off & ~tie).sum())} of them away from an fp32 rounding tie"
        nb = (g_mod[off] == np.nextafter(mod[off], np.float32(np.inf))) | \
             (g_mod[off] == np.nextafter(mod[off], np.float32(-np.inf)))
        assert np.all(nb), f"{tag0(l, t)}: an AdaLN value at a tie is not a neighbour"
        say(f"  {tag0(l, t)}: {int(off.sum())} AdaLN value(s) at an fp32 rounding tie")
        mod = g_mod
    x_out, st_new, rec = D.block_step(dims, SS.pol, W, st_o, x, mod, t)
    full = rec["full"]
    tag = f"block {l} t={t} {'full' if full else 'cache'}"
    say(f"  {tag}: |S| = {int(rec['sync'].sum())} of {T}")
    # the attention input is computed in fp32 (off the decision path): within
    # one bf16 ulp of the oracle's, or (where the modulation nearly cancels
    # the shift) within fp32 rounding of the terms
    g_h = SS.S.read("h").reshape(B, N, d)
    hg, ho = O.to_f64(g_h, BF), O.to_f64(rec["h"], BF)
    bound = np.abs(ho) * 2.0 ** -7 + 1e-5 * np.abs(ho).max()
    assert np.all(np.abs(hg - ho) <= bound), \
        f"{tag}: h off by {float(np.max(np.abs(hg - ho) - bound)):.3g} beyond the bound"
    g_u = SS.S.read("u").reshape(B, N, d)
    g_x1 = SS.S.read("x1").reshape(B, N, d)
    Sm = rec["sync"]
    if not full:
        assert np.array_equal(g_u, rec["u_route"]), \
            f"{tag}: routing input differs in {(g_u != rec['u_route']).sum()}"
        assert np.array_equal(g_x1[~Sm], rec["x1_pre"][~Sm]), f"{tag}: x1 outside S"

    # token lists
    soff = SS.S.read("soff")
    counts = Sm.sum(axis=1)
    assert np.array_equal(soff, np.r_[0, np.cumsum(counts)]), f"{tag}: sample offsets"
    slist = SS.S.read("slist")[:soff[-1]]
    assert np.array_equal(slist, np.flatnonzero(Sm.reshape(-1))), f"{tag}: token list"

    # attention path (tolerance)
    kv = SS.S.read("kv").reshape(B, N, 2 * d)
    tol = TOL[BF]
    for name, g, o in (("k", kv[..., :d], rec["k"]), ("v", kv[..., d:], rec["v"]),
                       ("q", SS.S.read("q").reshape(B, N, d)[Sm], rec["q"][Sm]),
                       ("o", SS.S.read("o").reshape(B, N, d)[Sm], rec["o"][Sm])):
        if g.size:
            e = rel_err(g, o, BF)
            assert e <= tol, f"{tag}: {name} rel err {e:.3g}"
    g_a = SS.S.read("a", l).reshape(B, N, d)
    assert np.array_equal(g_a[~Sm], st_o.a[~Sm]), f"{tag}: a of unsynchronised tokens changed"
    if Sm.any():
        e = rel_err(g_a[Sm], st_new.a[Sm], BF)
        assert e <= tol, f"{tag}: a rel err {e:.3g}"
        e = float(np.abs(g_x1[Sm] - rec["x1"][Sm]).max() / np.abs(rec["x1"]).max())
        assert e <= tol, f"{tag}: x1 rel err {e:.3g}"
        g_u2 = g_u if full else SS.S.read("u2").reshape(B, N, d)
        e = rel_err(g_u2[Sm], rec["u"][Sm], BF)
        assert e <= tol, f"{tag}: MoE input rel err {e:.3g}"

    # the MoE layer
    g_y = SS.S.read("y").reshape(B, N, d)
    mrec = rec["moe"]
    if not full:
        view = _LayerView(lay, dims.layer())
        rerun = lambda forced: O.step(dims.layer(), SS.pol, W.moe, st_o.moe, rec["u_route"], t,
                                      x_ffn=rec["u"], forced=forced)
        check_step(view, t, mrec, rec["y"], st_o.moe, st_new.moe, g_y,
                   uncached=SS.pol.mode == O.MODE_FULL, label=tag, rerun=rerun)
    else:
        lg = lay.read("logits")
        err = float(np.abs(lg.astype(np.float64) - mrec["logits64"]).max())
        safe = topk_safe(mrec["logits64"], k, err)
        e_t = lay.read("e_t").reshape(T, k)
        assert np.array_equal(e_t[safe], mrec["e_t"].reshape(T, k)[safe]), f"{tag}: routing"
        say(f"  {tag}: routing compared on {int(safe.sum())} of {T} tokens "
            f"(logit error {err:.2g})")
        # a token near a top-k tie may take other experts: y and the output
        # are compared on the others
        ok = safe.reshape(B, N)
        e = rel_err(g_y[ok], rec["y"][ok], BF)
        assert e <= tol, f"{tag}: y rel err {e:.3g}"

    # block output
    ok = np.ones((B, N), bool) if not full else safe.reshape(B, N)
    g_x = SS.x_dev.cpu().numpy()
    e = float(np.abs(g_x[ok] - x_out[ok]).max() / np.abs(x_out).max())
    assert e <= tol, f"{tag}: output rel err {e:.3g}"
    return x_out, st_new


def run_forced(SS: StackSetup, T: int):
    states = [D.BlockState(SS.dims) for _ in range(SS.sh.L)]
    for t in range(T):
        x = SS.xs[t]
        for l in range(SS.sh.L):
            x, states[l] = check_block(SS, l, t, states[l], x)


@pytest.mark.parametrize("mode,pol", [("ratio", {"ratio": 0.3}), ("threshold", {}),
                                      ("ratio", {"ratio": 1.0})])
def test_stack_tiny_forced(mode, pol):
    say(f"stack_tiny {mode} {pol}")
    SS = StackSetup(STACKS["stack_tiny"], mode=mode, T=5, **pol)
    run_forced(SS, 5)


@pytest.mark.parametrize("d,heads", [(512, 8), (640, 8), (384, 8)])
def test_stack_head_widths_ragged_forced(d, heads):
    """Head widths 64 (the other fixed tiling), 80 and 48 (the tilings with a
    run-time head width), 130 tokens: two query tiles and three key tiles
    with a ragged tail."""
    sh = StackShape(L=1, d=d, heads=heads, E=8, k=2, d_ff=256, B=2, N=130)
    say(f"head width {d // heads}, ragged")
    SS = StackSetup(sh, mode="ratio", seed=1, T=3, ratio=0.5)
    run_forced(SS, 3)


def test_stack_full_mode_forced():
    """The uncached comparator: every step is a full step."""
    say("stack_tiny full mode")
    SS = StackSetup(STACKS["stack_tiny"], mode="full", T=2)
    run_forced(SS, 2)


def test_stack_run_equals_block_by_block():
    """One call over both blocks (the residual folded into the next block's
    LayerNorm) gives the same bits as one call per block (the residual
    applied by the final pass)."""
    import torch
    sh = STACKS["stack_tiny"]
    A = StackSetup(sh, mode="ratio", seed=2, T=3, ratio=0.3)
    Bs = StackSetup(sh, mode="ratio", seed=2, T=3, ratio=0.3)
    xa = torch.zeros_like(A.x_dev)
    xb = torch.zeros_like(Bs.x_dev)
    for t in range(3):
        xa.copy_(torch.from_numpy(A.xs[t]))
        xb.copy_(torch.from_numpy(Bs.xs[t]))
        A.c_dev.copy_(torch.from_numpy(A.cs[t]))
        Bs.c_dev.copy_(torch.from_numpy(Bs.cs[t]))
        A.S.step(xa, A.c_dev, t)
        for l in range(sh.L):
            Bs.S.step_blocks(xb, Bs.c_dev, t, l, 1)
        torch.cuda.synchronize()
        assert torch.equal(xa, xb), f"t={t}"
        say(f"  t={t}: stack run == block by block")


def test_stack_graph_replay_equals_eager():
    """Steps replayed from HIP graphs (each block's k/v projection forked onto
    the stack's second stream and joined inside the graph) give the same bits
    as the same steps run eagerly; eager copies and synchronisations between
    the replays, every replay checked."""
    import torch
    sh = STACKS["stack_tiny"]
    A = StackSetup(sh, mode="ratio", seed=4, T=4, ratio=0.3)
    Bs = StackSetup(sh, mode="ratio", seed=4, T=4, ratio=0.3)
    for t in range(4):
        for S_ in (A, Bs):
            S_.x_dev.copy_(torch.from_numpy(S_.xs[t]))
            S_.c_dev.copy_(torch.from_numpy(S_.cs[t]))
        torch.cuda.synchronize()
        A.S.step(A.x_dev, A.c_dev, t)
        if t == 0:
            Bs.S.step(Bs.x_dev, Bs.c_dev, t)  # eager: the second stream is made here
        else:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                Bs.S.step(Bs.x_dev, Bs.c_dev, t)
            g.replay()
        torch.cuda.synchronize()
        assert torch.equal(A.x_dev, Bs.x_dev), f"t={t}"
        say(f"  t={t}: {'eager' if t == 0 else 'graph replay'} == eager")


def test_stack_embed_matches_oracle():
    import torch
    from paper_2606_15615_amd.layer import np_to_device
    sh = STACKS["stack_tiny"]
    SS = StackSetup(sh, T=1)
    emb = SS.syn.embedder()
    lab = SS.syn.labels()
    dev = SS.S.device
    tv = np.array([999.0, 3.5], np.float32)[:sh.B]
    lab_bad = lab.copy()
    lab_bad[-1] = sh.n_classes + 5   # outside the table: no class row
    for labels in (lab, lab_bad, None):
        c = torch.zeros((sh.B, sh.d), dtype=torch.float32, device=dev)
        ldev = None if labels is None else torch.from_numpy(labels.astype(np.int32)).to(dev)
        SS.S.embed(torch.from_numpy(tv).to(dev), ldev, np_to_device(emb["W1"], dev),
                   torch.from_numpy(emb["b1"]).to(dev), np_to_device(emb["W2"], dev),
                   torch.from_numpy(emb["b2"]).to(dev),
                   None if labels is None else np_to_device(emb["table"], dev), c)
        torch.cuda.synchronize()
        rows = None
        if labels is not None:
            ok = (labels >= 0) & (labels < sh.n_classes)
            rows = np.where(ok[:, None], emb["table"][np.clip(labels, 0, sh.n_classes - 1)], 0)
            rows = rows.astype(np.uint16)
        ref = D.cond_embed(tv, emb["W1"], emb["b1"], emb["W2"], emb["b2"], rows)
        got = c.cpu().numpy()
        np.testing.assert_allclose(got, ref, rtol=1e-5, atol=1e-6)


def test_stack_full_width_forced():
    """The dit28 block's attention shape (d = 1152, 16 heads of 72, 1024
    tokens: 16 key tiles, 8 query tiles) with small experts, a full step and
    two cache steps."""
    sh = StackShape(L=1, d=1152, heads=16, E=4, k=2, d_ff=256, B=2, N=1024)
    say("full width")
    SS = StackSetup(sh, mode="ratio", seed=3, T=3, ratio=0.3)
    run_forced(SS, 3)


@pytest.mark.timeout(600)
def test_stack_full_width_batch8_forced():
    """The benchmarked block's attention path at its full batch (d = 1152,
    16 heads of 72, 1024 tokens x 8, with small experts): the launch
    configuration of the timed stack, where a cache step's k/v projection
    (576 tiles) runs on the side stream with 24 blocks per XCD beside the
    decision kernels; a full step and two cache steps."""
    sh = StackShape(L=1, d=1152, heads=16, E=4, k=2, d_ff=256, B=8, N=1024)
    say("full width, batch 8")
    SS = StackSetup(sh, mode="ratio", seed=7, T=3, ratio=0.3)
    run_forced(SS, 3)


def test_stack_nothing_to_refresh_is_bit_identical():
    """A cache step whose input and conditioning equal the full step's, at
    ratio 0: every branch is matched and reused, no token is synchronised
    (the projections, attention and LN2 run over empty lists), and the
    output equals the full step's bit for bit, on the GPU as in the oracle."""
    import torch
    sh = StackShape(L=2, d=576, heads=8, E=4, k=2, d_ff=256, B=2, N=80)
    SS = StackSetup(sh, mode="ratio", seed=4, T=1, ratio=0.0)
    outs = []
    for t in range(2):
        SS.x_dev.copy_(torch.from_numpy(SS.xs[0]))
        SS.c_dev.copy_(torch.from_numpy(SS.cs[0]))
        SS.S.step(SS.x_dev, SS.c_dev, t)
        torch.cuda.synchronize()
        outs.append(SS.x_dev.clone())
        if t == 1:
            assert int(SS.S.read("soff")[-1]) == 0
            for l in range(sh.L):
                st = SS.S.layer(l).stats()
                assert st.n_recompute == 0 and st.n_sync == 0 and not st.full_step
    assert torch.equal(outs[0], outs[1])
    say("  nothing to refresh: cache step == full step")


def test_stack_single_token_single_head_forced():
    """One token per sample (attention over a single key: the output is
    that key's value) and one 64-wide head."""
    sh = StackShape(L=1, d=64, heads=1, E=4, k=2, d_ff=128, B=3, N=1)
    say("single token, single head")
    SS = StackSetup(sh, mode="ratio", seed=5, T=3, ratio=0.5)
    run_forced(SS, 3)


def test_stack_three_blocks_run_equals_block_by_block():
    import torch
    sh = StackShape(L=3, d=512, heads=8, E=8, k=2, d_ff=256, B=2, N=100)
    A = StackSetup(sh, mode="threshold", seed=6, T=3)
    Bs = StackSetup(sh, mode="threshold", seed=6, T=3)
    xa, xb = torch.zeros_like(A.x_dev), torch.zeros_like(Bs.x_dev)
    for t in range(3):
        xa.copy_(torch.from_numpy(A.xs[t]))
        xb.copy_(torch.from_numpy(Bs.xs[t]))
        A.c_dev.copy_(torch.from_numpy(A.cs[t]))
        Bs.c_dev.copy_(torch.from_numpy(Bs.cs[t]))
        A.S.step(xa, A.c_dev, t)
        Bs.S.step_blocks(xb, Bs.c_dev, t, 0, 2)   # blocks 0-1 in one call
        Bs.S.step_blocks(xb, Bs.c_dev, t, 2, 1)   # then block 2
        torch.cuda.synchronize()
        assert torch.equal(xa, xb), f"t={t}"


import random_cases


@pytest.mark.parametrize("i", range(random_cases.N_STACK_CASES))
def test_stack_random_configuration(i):
    """Seeded small stacks over every head width 8-96, one or two blocks,
    ragged token counts, every mode and drawn controller settings."""
    sh, mode, pol, T = random_cases.stack_case(i)
    say(f"stack case {i}: {sh} {mode} {pol} T={T}")
    SS = StackSetup(sh, mode=mode, seed=3000 + i, T=T, **pol)
    run_forced(SS, T)
