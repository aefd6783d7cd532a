"""GPU parity of the branch-cached MoE layer step against the CPU oracle.

Every test drives the HIP library through its C ABI (paper_2606_15615_amd
._lib via MoecaLayer) on seeded synthetic inputs and compares with the
oracle as described in tests/gpu_harness.py: decisions (logits, experts,
gate weights, statistic, thresholds, matching, margins, masks, slots, sync
mask, expert lists) bit for bit; rows and outputs within 2e-2 (bf16) or
1e-4 (fp32) max relative error.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

from oracle import moeca_oracle as O
from paper_2606_15615_amd.synth import LayerShape, WORKLOADS

from gpu_harness import (Setup, check_step, full_step_plan, oracle_rerun, run_forced, say,
                         rel_err)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_15615_amd import _lib
    _lib.load()   # fails loudly if the library is missing


# ---------------------------------------------------------------------------
# tiny fp32 layer (d=384, 8 experts, top-2, 1536 hidden, 256 tokens, 5 steps)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("mode,ratio", [("ratio", 0.0), ("ratio", 0.3), ("ratio", 1.0),
                                        ("threshold", 0.3)])
def test_tiny_fp32_trajectory(mode, ratio):
    S = Setup(WORKLOADS["tiny"], mode=mode, seed=1, T=5, ratio=ratio)
    infos = run_forced(S, 5, label=f"tiny {mode} {ratio}")
    say(f"  tiny {mode} {ratio}: {infos}")


# ---------------------------------------------------------------------------
# small bf16 layers with ragged token counts and a 64-multiple hidden width
# ---------------------------------------------------------------------------
RAGGED = LayerShape(d=256, E=6, k=2, d_ff=320, B=3, N=77, dtype="bf16")


@pytest.mark.parametrize("mode,ratio", [("threshold", 0.3), ("ratio", 0.3), ("ratio", 0.05)])
def test_ragged_bf16_trajectory(mode, ratio):
    S = Setup(RAGGED, mode=mode, seed=2, T=6, ratio=ratio)
    run_forced(S, 6, label=f"ragged {mode} {ratio}")


@pytest.mark.parametrize("shape", [
    LayerShape(d=128, E=4, k=4, d_ff=128, B=2, N=33, dtype="bf16"),    # k == E
    LayerShape(d=192, E=5, k=1, d_ff=256, B=2, N=40, dtype="bf16"),    # top-1
    LayerShape(d=64, E=3, k=2, d_ff=64, B=4, N=1, dtype="bf16"),       # one token per sample
    LayerShape(d=128, E=64, k=8, d_ff=128, B=1, N=50, dtype="fp32"),   # many experts, k = 8
])
def test_edge_shapes(shape):
    S = Setup(shape, mode="ratio", seed=3, T=5, ratio=0.4, refresh_cycle=3)
    run_forced(S, 5, label=f"edge {shape}")


def test_unnormalised_gate_erf_gelu_and_bias():
    shape = LayerShape(d=128, E=8, k=2, d_ff=192, B=2, N=64, dtype="fp32")
    S = Setup(shape, mode="threshold", seed=4, T=4, norm_topk=False, act="gelu_erf",
              bias="zipf", lambda1=0.5, lambda2=2.0, tau0=0.9, alpha=0.3, beta=0.5)
    run_forced(S, 4, label="variants")


WIDE = LayerShape(d=128, E=16, k=8, d_ff=128, B=2, N=1100, dtype="bf16")


@pytest.mark.parametrize("mode,ratio", [("ratio", 0.25), ("ratio", 0.02), ("threshold", 0.3),
                                        ("full", 0.3)])
def test_wide_decision_path(mode, ratio):
    """Samples of more than 8192 branches take the multi-block decision path
    (8800 branches here: eight full blocks and a partial one, 128 tokens per
    block): every decision bit for bit, refresh and cache steps."""
    S = Setup(WIDE, mode=mode, seed=18, T=4, ratio=ratio, refresh_cycle=3)
    run_forced(S, 4, label=f"wide {mode} {ratio}")


@pytest.mark.parametrize("mode,ratio", [("ratio", 0.3), ("threshold", 0.3)])
def test_one_block_many_branches_per_thread(mode, ratio):
    """k = 3 does not divide 1024, so 9000 branches per sample stay in one
    block per sample: nine branches per thread, the runtime-loop variant
    with the key halves in LDS."""
    shape = LayerShape(d=128, E=16, k=3, d_ff=128, B=1, N=3000, dtype="bf16")
    S = Setup(shape, mode=mode, seed=19, T=3, ratio=ratio, refresh_cycle=0)
    run_forced(S, 3, label=f"one-block {mode}")


@pytest.mark.parametrize("lams", [(1.0, 0.0, 0.0), (0.0, 1.0, 0.0), (0.0, 0.0, 1.0),
                                  (0.0, 1.0, 1.0), (0.5, 2.0, 0.25)])
def test_score_signal_ablations(lams):
    """Score-signal ablation (Sec. 5): s = lambda0 w + lambda1 Delta +
    lambda2 o with single signals, a pair and unequal weights, threshold
    mode (thresholds scaled so each variant recomputes a share)."""
    l0, l1, l2 = lams
    shape = LayerShape(d=128, E=8, k=2, d_ff=192, B=2, N=64, dtype="bf16")
    S = Setup(shape, mode="threshold", seed=17, T=4, lambda0=l0, lambda1=l1, lambda2=l2,
              tau0=0.3, alpha=0.6, refresh_cycle=0)
    run_forced(S, 4, label=f"score {lams}")


# ---------------------------------------------------------------------------
# uncached comparator, empty recomputation set, ratio 0 bit-exact combine
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("shape", [WORKLOADS["tiny"], RAGGED])
def test_uncached_mode(shape):
    S = Setup(shape, mode="full", seed=5, T=3)
    run_forced(S, 3, label="uncached")
    assert S.layer.stats().full_step == 1


@pytest.mark.parametrize("mode", ["ratio", "threshold"])
def test_nothing_recomputed_is_bit_exact(mode):
    """Same input as the refresh step: ratio 0 (or a huge threshold) reuses
    every branch; the output is then the combine of cached rows, which the
    GPU must reproduce bit for bit."""
    S = Setup(RAGGED, mode=mode, seed=6, T=1, ratio=0.0, tau0=1e6, refresh_cycle=0)
    st0 = O.State(S.dims, attention=True)
    out0, st1, _ = O.step(S.dims, S.pol, S.W, st0, S.xs[0], 0, attn_in=S.attn[0])
    S.import_state(st1)
    out_g = S.gpu_step(S.xs[0], 1, S.attn[0])
    rerun = oracle_rerun(S, st1, S.xs[0], 1, S.attn[0])
    out_o, st2, rec = rerun(None)
    assert rec["mask"].sum() == 0
    check_step(S, 1, rec, out_o, st1, st2, out_g, label="reuse-all", rerun=rerun)
    assert np.array_equal(out_g, out_o)
    assert np.array_equal(out_o, out0)


@pytest.mark.parametrize("N,E,k", [(40, 8, 2), (300, 8, 2), (2000, 8, 2), (2100, 16, 8)])
def test_all_branches_tied(N, E, k):
    """Every token carries the same input as at the refresh step, so every
    branch is matched and all branches of one slot tie on the margin.  The
    ratio selection must then take the lowest flat ids among the tied keys:
    ranked directly when at most 64 keys share the threshold's prefix (N=40),
    by the tie ballots after the fourth digit otherwise; one, eight and
    thirty-two branches per thread."""
    shape = LayerShape(d=128, E=E, k=k, d_ff=128, B=2, N=N, dtype="bf16")
    S = Setup(shape, mode="ratio", seed=11, T=1, ratio=0.3, refresh_cycle=0)
    x = np.repeat(S.xs[0][:, :1, :], N, axis=1)
    st0 = O.State(S.dims, attention=True)
    _, st1, _ = O.step(S.dims, S.pol, S.W, st0, x, 0, attn_in=S.attn[0])
    S.import_state(st1)
    out_g = S.gpu_step(x, 1, S.attn[0])
    rerun = oracle_rerun(S, st1, x, 1, S.attn[0])
    out_o, st2, rec = rerun(None)
    assert rec["matched"].all()
    assert all(len(np.unique(rec["m"][b])) <= k for b in range(2))  # one margin per slot
    assert 0 < rec["mask"].sum() < rec["mask"].size
    check_step(S, 1, rec, out_o, st1, st2, out_g, label=f"ties N={N} k={k}", rerun=rerun)


def test_reset_mid_trajectory():
    S = Setup(RAGGED, mode="ratio", seed=7, T=4, ratio=0.3, refresh_cycle=0)
    for t in range(3):
        S.gpu_step(S.xs[t], t, S.attn[t])
    assert S.layer.stats().full_step == 0
    S.layer.reset()
    out_g = S.gpu_step(S.xs[3], 3, S.attn[3])
    st0 = O.State(S.dims, True)
    rerun = oracle_rerun(S, st0, S.xs[3], 3, S.attn[3])
    out_o, st_new, rec = rerun(None)
    assert rec["full"] and S.layer.stats().full_step == 1
    check_step(S, 3, rec, out_o, st0, st_new, out_g, label="after reset", rerun=rerun)


def test_determinism():
    S = Setup(RAGGED, mode="ratio", seed=8, T=3, ratio=0.3, refresh_cycle=0)
    st = O.State(S.dims, attention=True)
    for t in range(2):
        _, st, _ = O.step(S.dims, S.pol, S.W, st, S.xs[t], t, attn_in=S.attn[t])
    outs = []
    for _ in range(2):
        S.import_state(st)
        outs.append((S.gpu_step(S.xs[2], 2, S.attn[2]), S.layer.read("h_c"),
                     S.layer.read("mask"), S.layer.read("list")))
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


def test_nonfinite_input_is_flagged():
    S = Setup(RAGGED, mode="ratio", seed=9, T=1, ratio=0.3)
    x = S.xs[0].copy()
    x[1, 5, 7] = 0x7FC0            # bf16 NaN
    S.gpu_step(x, 0, S.attn[0])
    assert S.layer.stats().nonfinite == 1
    S.gpu_step(S.xs[0], 1, S.attn[0])
    assert S.layer.stats().nonfinite == 0


# ---------------------------------------------------------------------------
# DiT-MoE-XL-like layer (d=1152, 16 experts, top-2, 4608 hidden), 256 tokens x 8
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("mode", ["ratio", "threshold"])
def test_xl256_trajectory(mode):
    S = Setup(WORKLOADS["xl256"], mode=mode, seed=10, T=5, ratio=0.3)
    infos = run_forced(S, 5, label=f"xl256 {mode}")
    say(f"  xl256 {mode}: {infos}")


# ---------------------------------------------------------------------------
# Full-size layers at their benchmarked shapes: decisions over the whole
# batch, outputs and rows on sampled tokens computed one by one by the
# oracle.  Step 0 is a full-computation step (Sec. 4.1: the cache is
# invalid), the later ones consecutive cache steps, each forced from the
# oracle's state.  The rows of tokens the oracle does not evaluate are given
# synthetic values and their norms after every step.
# ---------------------------------------------------------------------------
def sampled_tokens(shape, n, seed):
    rng = np.random.default_rng(seed)
    sample = np.sort(rng.choice(shape.tokens, size=n, replace=False))
    ev = np.zeros(shape.tokens, bool)
    ev[sample] = True
    return sample, ev.reshape(shape.B, shape.N)


def fill_unsampled(S, st, ev):
    fill = ~ev
    rows = S.sy.rows((int(fill.sum()), S.shape.k, S.shape.d), scale=0.05)
    st.h_c[fill] = rows
    st.n_c[fill] = O.row_norms(rows, S.shape.dtype)


def run_sampled(S, T, sample, ev, label):
    st = O.State(S.dims, attention=S.attention)
    infos = []
    for t in range(T):
        say(f"  [{label}] step {t}")
        S.import_state(st)
        a = None if S.attn is None else S.attn[t]
        out_g = S.gpu_step(S.xs[t], t, a)
        rerun = oracle_rerun(S, st, S.xs[t], t, a, tokens=sample)
        out_o, st_new, rec = rerun(None)
        assert rec["full"] == (t == 0)
        info = check_step(S, t, rec, out_o, st, st_new, out_g, evaluated=ev,
                          label=f"{label} t={t}", rerun=rerun)
        st = info.pop("state")
        fill_unsampled(S, st, ev)
        infos.append(info)
        say(f"  {label} t={t}: {info}")
    return infos


@pytest.mark.timeout(600)
@pytest.mark.parametrize("mode", ["ratio", "threshold"])
def test_xl1024_sampled(mode):
    """The benchmarked layer (d=1152, 16 experts, top-2, 4608 hidden, 1024
    tokens x 8, 30 % refresh): a refresh step over all 16384 branches (about
    1024 GEMM rows per expert), then three consecutive cache steps."""
    shape = WORKLOADS["xl1024"]
    S = Setup(shape, mode=mode, seed=11, T=4, ratio=0.3, refresh_cycle=0)
    sample, ev = sampled_tokens(shape, 48, 12)
    infos = run_sampled(S, 4, sample, ev, f"xl1024 {mode}")
    if mode == "ratio":
        for info in infos[1:]:
            assert abs(info["recompute_frac"] - 0.3) < 0.02
        # cache steps: about 307 rows per expert, the expert-wide up projection
        assert [i["ffn_plan"] for i in infos] == [full_step_plan(shape), 2, 2, 2]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("ratio,plan", [(0.05, 2), (0.6, 0)])
def test_xl1024_sampled_other_ratios(ratio, plan):
    """The benchmarked layer at a low and a high refresh ratio: the cache
    steps leave about 50 rows per expert plus the unmatched branches (the
    expert-wide up projection with few rows per tile) and about 600 (the
    128 x 256 tiles for both projections); a refresh step, then two cache
    steps."""
    shape = WORKLOADS["xl1024"]
    S = Setup(shape, mode="ratio", seed=13, T=3, ratio=ratio, refresh_cycle=0)
    sample, ev = sampled_tokens(shape, 32, 14)
    infos = run_sampled(S, 3, sample, ev, f"xl1024 rho={ratio}")
    for info in infos[1:]:
        assert info["recompute_frac"] >= ratio - 0.02
    assert [i["ffn_plan"] for i in infos] == [full_step_plan(S.shape), plan, plan]


@pytest.mark.timeout(600)
def test_xl256_sampled():
    """The layer at 256 tokens x 8 (d=1152, 16 experts, top-2, 4608 hidden,
    30 % refresh): its cache steps leave about 77 rows per expert and take
    the weight-streaming plan (128 x 288 tiles, the down projection in four
    K pieces added in order); a refresh step, then three cache steps."""
    shape = WORKLOADS["xl256"]
    S = Setup(shape, mode="ratio", seed=12, T=4, ratio=0.3, refresh_cycle=0)
    sample, ev = sampled_tokens(shape, 48, 13)
    infos = run_sampled(S, 4, sample, ev, "xl256 ratio")
    assert [i["ffn_plan"] for i in infos] == [full_step_plan(S.shape), 1, 1, 1]


# ---------------------------------------------------------------------------
# The weight-streaming plan at sizes the oracle evaluates whole: tiles that
# are exactly 288 wide, ragged N tiles and K pieces (37 k-tiles: 9, 9, 9,
# 10), and experts with more than one 128-row tile.
# ---------------------------------------------------------------------------
THIN_SHAPES = [
    (LayerShape(d=576, E=16, k=2, d_ff=2304, B=2, N=128, dtype="bf16"), 0.3),
    (LayerShape(d=640, E=16, k=2, d_ff=2368, B=2, N=100, dtype="bf16"), 0.3),
    (LayerShape(d=576, E=8, k=2, d_ff=4608, B=4, N=256, dtype="bf16"), 0.4),
]


@pytest.mark.parametrize("shape,ratio", THIN_SHAPES)
def test_thin_plan_trajectory(shape, ratio):
    S = Setup(shape, mode="ratio", seed=31, T=4, ratio=ratio, refresh_cycle=0)
    infos = run_forced(S, 4, label=f"thin {shape}")
    assert [i["ffn_plan"] for i in infos] == [full_step_plan(S.shape), 1, 1, 1]


# ---------------------------------------------------------------------------
# The expert-wide up projection at sizes the oracle evaluates whole: up to
# 384 rows of an expert in one tile by 144 columns; experts past 384 rows
# split into equal parts (the skewed shape has experts of a few rows and
# experts split in several parts), row counts that are not multiples of
# 16, and zero to three row tiles per wave.
# ---------------------------------------------------------------------------
WIDE_SHAPES = [
    (LayerShape(d=576, E=8, k=2, d_ff=1152, B=4, N=512, dtype="bf16"), 0.3, None),
    (LayerShape(d=512, E=8, k=2, d_ff=576, B=4, N=1024, dtype="bf16"), 0.29, None),
    (LayerShape(d=640, E=16, k=2, d_ff=1728, B=2, N=1000, dtype="bf16"), 0.6, None),
    (LayerShape(d=512, E=16, k=2, d_ff=576, B=2, N=1024, dtype="bf16"), 0.7, "zipf"),
]


@pytest.mark.parametrize("shape,ratio,bias", WIDE_SHAPES)
def test_wide_plan_trajectory(shape, ratio, bias):
    S = Setup(shape, mode="ratio", seed=41, T=4, ratio=ratio, refresh_cycle=0,
              **({} if bias is None else {"bias": bias, "drift": "bimodal"}))
    infos = run_forced(S, 4, label=f"wide {shape} {bias}")
    assert [i["ffn_plan"] for i in infos] == [full_step_plan(S.shape), 2, 2, 2]


# ---------------------------------------------------------------------------
# Skewed routing: 32 experts with a Zipf(1.2) router prior, bimodal token
# drift (90 % slow, 10 % fast), swept over refresh ratios.  Width reduced
# (d = 512, d_ff = 1024) so the oracle evaluates every branch; the same
# kernels run at the full width in the benchmark's ratio sweep.
# ---------------------------------------------------------------------------
SKEWED_SMALL = LayerShape(d=512, E=32, k=2, d_ff=1024, B=2, N=1024, dtype="bf16")


@pytest.mark.parametrize("ratio", [0.1, 0.5, 0.9])
def test_skewed_ratio_sweep(ratio):
    S = Setup(SKEWED_SMALL, mode="ratio", seed=14, T=4, ratio=ratio, refresh_cycle=0,
              bias="zipf", drift="bimodal")
    infos = run_forced(S, 4, label=f"skewed rho={ratio}")
    say(f"  skewed rho={ratio}: {infos}")


@pytest.mark.timeout(900)
def test_skewed_full_size_sampled():
    """The skewed-routing layer at its benchmarked size (d=3072, 32 experts,
    top-2, 8192 hidden, 4096 tokens x 2, Zipf(1.2) router prior, bimodal
    drift) at refresh ratios 0.1, 0.5 and 0.9: a refresh step and two cache
    steps each, outputs and rows on sampled tokens."""
    base = Setup(WORKLOADS["skewed"], mode="ratio", seed=22, T=3, ratio=0.1, refresh_cycle=0,
                 bias="zipf", drift="bimodal")
    sample, ev = sampled_tokens(base.shape, 24, 23)
    for ratio in (0.1, 0.5, 0.9):
        S = base if ratio == 0.1 else base.with_policy(ratio=ratio)
        infos = run_sampled(S, 3, sample, ev, f"skewed full rho={ratio}")
        for info in infos[1:]:
            assert info["recompute_frac"] >= ratio - 0.02
        if S is not base:
            S.release()


def test_skewed_threshold():
    S = Setup(SKEWED_SMALL, mode="threshold", seed=15, T=4, refresh_cycle=0, bias="zipf",
              drift="bimodal")
    infos = run_forced(S, 4, label="skewed threshold")
    say(f"  skewed threshold: {infos}")


def test_free_running_agreement():
    """Both sides run freely from a reset.  Stored rows legitimately differ
    in their last bf16 bits, so masks may drift apart over time; report the
    agreement and require the outputs to stay within tolerance while the
    masks agree."""
    S = Setup(WORKLOADS["xl256"], mode="ratio", seed=13, T=6, ratio=0.3)
    st = O.State(S.dims, attention=True)
    agree = []
    for t in range(6):
        out_g = S.gpu_step(S.xs[t], t, S.attn[t])
        out_o, st, rec = O.step(S.dims, S.pol, S.W, st, S.xs[t], t, attn_in=S.attn[t])
        mask = S.layer.read("mask").reshape(rec["mask"].shape).astype(bool)
        a = float((mask == rec["mask"]).mean())
        agree.append(a)
        if a == 1.0:
            assert rel_err(out_g, out_o, "bf16") <= 2e-2
    say(f"  free-running mask agreement per step: {agree}")
    assert min(agree) >= 0.99


# ---------------------------------------------------------------------------
# Fine-grained layer with shared experts (Sec. 2.3, shared-expert MoE eq.):
# gated (SwiGLU) experts, top-k over many small experts, always-on shared
# experts that are never cached, unnormalised gates.  The shapes cover the
# large-tile GEMM (>= 512 weight rows), the 128- and 64-wide tiles, the
# fp32 kernels, more than 64 GEMM groups, a GELU layer with a shared expert
# and the uncached comparator.
# ---------------------------------------------------------------------------
FINE_SHAPES = [
    LayerShape(d=512, E=16, k=4, d_ff=320, B=2, N=256, dtype="bf16", ffn="swiglu", n_shared=2),
    LayerShape(d=256, E=8, k=2, d_ff=128, B=2, N=77, dtype="bf16", ffn="swiglu", n_shared=1),
    LayerShape(d=192, E=6, k=3, d_ff=64, B=3, N=41, dtype="bf16", ffn="swiglu", n_shared=3),
    LayerShape(d=128, E=8, k=4, d_ff=64, B=2, N=50, dtype="fp32", ffn="swiglu", n_shared=2),
    LayerShape(d=256, E=64, k=8, d_ff=256, B=1, N=96, dtype="bf16", ffn="swiglu", n_shared=2),
    LayerShape(d=128, E=64, k=8, d_ff=64, B=1, N=60, dtype="fp32", ffn="swiglu", n_shared=8),
    LayerShape(d=256, E=6, k=2, d_ff=320, B=2, N=77, dtype="bf16", n_shared=1),
]


@pytest.mark.parametrize("shape", FINE_SHAPES)
def test_fine_shared_trajectory(shape):
    S = Setup(shape, mode="ratio", seed=16, T=5, ratio=0.25, refresh_cycle=3, norm_topk=False)
    infos = run_forced(S, 5, label=f"fine {shape}")
    say(f"  fine {shape}: {infos}")


def test_fine_shared_threshold_and_uncached():
    shape = FINE_SHAPES[0]
    S = Setup(shape, mode="threshold", seed=17, T=4, refresh_cycle=0, norm_topk=False)
    run_forced(S, 4, label="fine threshold")
    U = Setup(shape, mode="full", seed=18, T=2, norm_topk=False)
    run_forced(U, 2, label="fine uncached")


def test_fine_nothing_recomputed_still_runs_shared_experts():
    """Ratio 0 on a new input: every matched branch is reused, yet the
    output carries the shared experts of the new input."""
    shape = FINE_SHAPES[1]
    S = Setup(shape, mode="ratio", seed=19, T=2, ratio=0.0, refresh_cycle=0, norm_topk=False)
    st0 = O.State(S.dims, attention=True)
    _, st1, _ = O.step(S.dims, S.pol, S.W, st0, S.xs[0], 0, attn_in=S.attn[0])
    S.import_state(st1)
    out_g = S.gpu_step(S.xs[1], 1, S.attn[1])
    rerun = oracle_rerun(S, st1, S.xs[1], 1, S.attn[1])
    out_o, st2, rec = rerun(None)
    assert rec["mask"].sum() == (~rec["matched"]).sum()
    info = check_step(S, 1, rec, out_o, st1, st2, out_g, label="fine reuse", rerun=rerun)
    say(f"  fine reuse: {info}")


@pytest.mark.timeout(600)
def test_fine_sampled():
    """The benchmarked fine-grained layer (d=2048, 64 experts, top-8, 1408
    hidden SwiGLU, 2 shared experts, 4096 tokens x 4, 25 % refresh): a
    refresh step and two cache steps, outputs and rows on sampled tokens."""
    shape = WORKLOADS["fine"]
    S = Setup(shape, mode="ratio", seed=20, T=3, ratio=0.25, refresh_cycle=0, norm_topk=False)
    sample, ev = sampled_tokens(shape, 24, 21)
    run_sampled(S, 3, sample, ev, "fine sampled")


# ---------------------------------------------------------------------------
# Steps replayed from a HIP graph (the launch mode of the benchmark) against
# the oracle: one cache step captured once, then replayed from successive
# oracle states and inputs, with eager work between the replays.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("wl,mode", [("ragged", "ratio"), ("ragged", "threshold"),
                                     ("xl1024", "ratio")])
def test_graph_replayed_steps(wl, mode):
    import torch
    from paper_2606_15615_amd.layer import device_to_np, np_to_device
    shape = RAGGED if wl == "ragged" else WORKLOADS["xl1024"]
    T = 5
    S = Setup(shape, mode=mode, seed=24, T=T, ratio=0.3, refresh_cycle=0)
    sampled = wl != "ragged"
    sample, ev = sampled_tokens(shape, 32, 25) if sampled else (None, None)
    st = O.State(S.dims, attention=True)
    _, st, _ = O.step(S.dims, S.pol, S.W, st, S.xs[0], 0, attn_in=S.attn[0], tokens=sample)
    if sampled:
        fill_unsampled(S, st, ev)
    L = S.layer
    x_static = np_to_device(S.xs[1], L.device)
    S.import_state(st)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        L.step(x_static, 1, S.out)
    for t in range(1, T):
        say(f"  [graph {wl} {mode}] replay for step {t}")
        S.import_state(st)
        S.attn_in.copy_(np_to_device(S.attn[t], L.device))
        x_static.copy_(np_to_device(S.xs[t], L.device))
        S.out.zero_()
        g.replay()
        torch.cuda.synchronize()
        out_g = device_to_np(S.out, S.act_np)
        rerun = oracle_rerun(S, st, S.xs[t], t, S.attn[t], tokens=sample)
        out_o, st_new, rec = rerun(None)
        assert not rec["full"]
        info = check_step(S, t, rec, out_o, st, st_new, out_g, evaluated=ev,
                          label=f"graph {wl} {mode} t={t}", rerun=rerun)
        st = info.pop("state")
        if sampled:
            fill_unsampled(S, st, ev)
        say(f"  graph {wl} {mode} t={t}: {info}")


# ---------------------------------------------------------------------------
# A seeded sweep over layer configurations: shapes (widths, expert counts,
# top-k including 3 and 6, shared experts, SwiGLU, fp32), every mode and the
# controller settings drawn at random inside the documented limits
# ---------------------------------------------------------------------------
import random_cases


@pytest.mark.parametrize("i", range(random_cases.N_CASES))
def test_random_configuration(i):
    shape, mode, pol, T, bias = random_cases.case(i)
    say(f"  case {i}: {shape} {mode} {pol} T={T} bias={bias}")
    S = Setup(shape, mode=mode, seed=1000 + i, T=T, bias=bias, **pol)
    infos = run_forced(S, T, label=f"random {i}")
    say(f"  case {i}: {infos}")


@pytest.mark.parametrize("j", range(random_cases.N_PLAN_CASES))
def test_random_plan_configuration(j):
    """Seeded ratio-mode cases drawn to take the weight-streaming plan or the
    expert-wide up projection on every cache step (one multi-block decision
    among them: over 8192 branches per sample)."""
    shape, pol, T, plan = random_cases.plan_case(j)
    say(f"  plan case {j}: {shape} {pol} T={T} plan={plan}")
    S = Setup(shape, mode="ratio", seed=2000 + j, T=T, **pol)
    infos = run_forced(S, T, label=f"random plan {j}")
    say(f"  plan case {j}: {infos}")
    assert [i["ffn_plan"] for i in infos] == [full_step_plan(S.shape)] + [plan] * (T - 1)
