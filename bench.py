"""Benchmark: cached MoE-layer step on one MI355X.

A step is one pass of the whole branch-cached layer (router, statistic and
thresholds, matching and scores, selection, expert lists, grouped expert
FFN, combine with cache and attention write) over one batch of synthetic
input already resident in HBM.  The timed steps are cache steps at a 30%
per-sample branch budget; the full-recompute comparator (the uncached layer
through the same kernels) is timed on the same inputs.  Each phase runs
its K steps eagerly with HIP events between kernels (per-kernel times), then
replays the same K steps from one HIP graph (the headline time).  The
roofline object is for the longer of the two expert-FFN GEMM launches,
against the lower of its two roofs (MFMA peak, or arithmetic intensity x HBM
peak); its HBM traffic comes from the committed rocprofv3 counter summary,
and is null when the kernel source no longer matches the one the counters
were taken on.

    python bench.py [--steps K] [--warmup W] [--workload xl1024]
                    [--phase both|cached|full] [--no-cpu] [--no-graph]
                    [--sweep 0,0.1,...]   (extra cache-step timings per refresh ratio)
                    [--policy-study]      (threshold-mode controller study instead)

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "cached MoE-layer ms/step + MFMA TFLOP/s on recomputed branches, 30% refresh"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="xl1024")
    ap.add_argument("--ratio", type=float, default=None,
                    help="refresh ratio (default 0.3; 0.25 for the fine-grained layer)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--phase", choices=("both", "cached", "full"), default="both",
                    help="time the cache steps, the full-recompute comparator, or both")
    ap.add_argument("--no-graph", action="store_true",
                    help="time eager launches only (no HIP graph replay)")
    ap.add_argument("--sweep", default="",
                    help="comma-separated refresh ratios: also time cache steps at each one")
    ap.add_argument("--flush-mib", type=int, default=512,
                    help="MALL-flushed timing: write this many MiB between single timed steps (0: off)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--policy-study", action="store_true",
                    help="instead of the headline line: threshold-mode controller study (alpha, "
                         "tau0, beta sweeps and score-signal ablations) over --steps steps of the "
                         "synthetic trajectory, against the uncached layer; one JSON line")
    ap.add_argument("--blas-reference", action="store_true",
                    help="instead of the layer: time the vendor bf16 batched GEMM (torch.bmm) on "
                         "the per-expert shapes of the workload's two projections, as a reference "
                         "point for the grouped FFN kernel, and print one JSON line")
    return ap.parse_args()


def _oracle_timings(shape, ratio, seed, norm_topk, act, reps, threads):
    """The oracle, as it stands, over the whole batch of ``shape``, BLAS
    limited to ``threads`` threads: the weights widened to fp64 first
    (untimed), then the refresh step (a full-computation step: the cache
    starts invalid) and ``reps`` cache steps from the state it leaves.
    Returns (median cache ms, full ms)."""
    from threadpoolctl import threadpool_limits
    from oracle import moeca_oracle as O
    from paper_2606_15615_amd.synth import Synth
    sy = Synth(shape, seed)
    W = sy.weights()
    dims = O.Dims(shape.d, shape.E, shape.k, shape.d_ff, shape.B, shape.N, shape.dtype,
                  shape.n_shared)
    Wo = O.Weights(dims, *W, *(sy.shared_weights() or (None, None)))
    for e in range(shape.E):
        Wo.up64(e), Wo.down64(e)
    xs = list(sy.trajectory(reps + 1))
    pol = O.Policy(mode=O.MODE_RATIO, ratio=ratio, refresh_cycle=0, norm_topk=norm_topk, act=act)
    with threadpool_limits(limits=threads):
        t0 = time.perf_counter()
        _, st, rec = O.step(dims, pol, Wo, O.State(dims), xs[0], 0)
        full = time.perf_counter() - t0
        assert rec["full"]
        cache = []
        for j in range(reps):
            t0 = time.perf_counter()
            _, st, rec = O.step(dims, pol, Wo, st, xs[1 + j], 1 + j)
            cache.append(time.perf_counter() - t0)
            assert not rec["full"]
    return float(np.median(cache)) * 1e3, full * 1e3


def cpu_baseline(shape, ratio, seed, norm_topk, act, reps):
    """The oracle timed on this host's cores, over the whole batch of the
    benchmarked workload: the refresh step (a full-computation step) and the
    median of ``reps`` cache steps after it, with as many BLAS threads as
    the process may run on (sched_getaffinity).  The tiny fp32 layer (d=384,
    8 experts, 256 tokens) is timed the same way single-threaded."""
    from paper_2606_15615_amd.synth import WORKLOADS
    cores = len(os.sched_getaffinity(0))
    cache_ms, full_ms = _oracle_timings(shape, ratio, seed, norm_topk, act, reps, cores)
    tiny_cache, tiny_full = _oracle_timings(WORKLOADS["tiny"], ratio, seed, True, "gelu_tanh",
                                            3, 1)
    return {"value": round(cache_ms, 2), "unit": "ms/step", "cores": cores, "kind": "oracle",
            "sample": f"whole batch ({shape.B} x {shape.N} tokens): cache step at ratio {ratio} "
                      f"(median of {reps}) after the refresh step, which is timed as the full "
                      f"step",
            "full_ms_per_step": round(full_ms, 2),
            "tiny_fp32_single_thread": {"cache_ms": round(tiny_cache, 2),
                                        "full_ms": round(tiny_full, 2), "cores": 1}}


def blas_reference(shape, args):
    """The vendor bf16 GEMM (torch.bmm, hipBLASLt on ROCm) on dense per-expert
    problems with the grouped FFN's shapes: E experts x rows per expert
    (every branch on a full step, the ratio's share on a cache step), K = d
    (up) or d_ff (down).  No gather, scatter or activation: a reference for
    what a tuned library reaches on the same matrix shapes."""
    import torch
    dev = torch.device("cuda:0")
    full_rows = shape.B * shape.N * shape.k // shape.E
    cached_rows = int(round(full_rows * args.ratio))
    res = []
    cases = [(label, proj, shape.E, rows, K, Nn)
             for label, rows in (("full", full_rows), ("cached", cached_rows))
             for proj, K, Nn in (("up", shape.d, shape.up_rows), ("down", shape.d_ff, shape.d))]
    cases.append(("square", "-", 1, 8192, 8192, 8192))  # a large square product, for scale
    for label, proj, ne, rows, K, Nn in cases:
        a = torch.randn(ne, rows, K, device=dev, dtype=torch.bfloat16)
        w = torch.randn(ne, K, Nn, device=dev, dtype=torch.bfloat16).contiguous()
        for _ in range(3):
            torch.bmm(a, w)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 20
        e0.record()
        for _ in range(reps):
            torch.bmm(a, w)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        fl = 2.0 * ne * rows * K * Nn
        res.append({"step": label, "projection": proj, "experts": ne, "rows": rows,
                    "k": K, "n": Nn, "us": round(us, 1),
                    "tflops": round(fl / us / 1e6, 1),
                    "frac_bf16_peak": round(fl / us / 1e6 / PEAK_BF16_TFLOPS, 3)})
        del a, w
    return res


def kernel_traffic(kernel_src: str, summary: str, stage: str = "ffn_up"):
    """HBM bytes per launch of a GEMM stage (``ffn_up`` or ``ffn_down``) from
    the committed counter summary (FETCH_SIZE and WRITE_SIZE, scaled by the
    copy-kernel factors; keys ``<stage>.kernel_source_sha256`` and
    ``<stage>.hbm_bytes_per_launch``), or None when the kernel source changed
    since the counters were taken."""
    import hashlib
    try:
        vals = {}
        with open(summary) as f:
            for line in f:
                if "=" in line and not line.lstrip().startswith("#"):
                    k, v = line.split("=", 1)
                    vals[k.strip()] = v.strip()
        with open(kernel_src, "rb") as f:
            digest = hashlib.sha256(f.read()).hexdigest()
        if vals.get(f"{stage}.kernel_source_sha256") != digest:
            return None
        return float(vals[f"{stage}.hbm_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def bf16_bits_to_f32(t):
    """bf16 bit patterns held in an int16 tensor -> float32 values."""
    import torch
    return ((t.to(torch.int32) & 0xFFFF) << 16).view(torch.float32)


def policy_study(args, shape, make_layer, xs, out, _lib):
    """Threshold-mode controller study on the synthetic trajectory: the
    mechanisms behind the ablations of Sec. 5 (adaptive vs fixed threshold,
    tau0 and beta sweeps, score-signal ablation) and the reuse-over-match
    ratio of Fig. 8, measured as recompute share, reuse over match, time per
    step and output deviation from the uncached layer (the same kernels in
    MOECA_MODE_FULL) on the same inputs.  The paper's image-quality metrics
    need its trained models and datasets and are not reproduced; the output
    deviation is this study's stand-in.  Forced full steps every 4 steps
    (Sec. 5.1), tau0 0.8, alpha 0.6, beta 0.65, lambda 1 unless varied."""
    import torch
    T = len(xs)
    f32 = bf16_bits_to_f32 if shape.dtype == "bf16" else (lambda t: t.float())
    ref = []
    Lf = make_layer(_lib.MOECA_MODE_FULL, {})
    for t in range(T):
        Lf.step(xs[t], t, out)
        ref.append(f32(out).clone())
    Lf.close()
    base = dict(tau0=0.80, alpha=0.6, beta=0.65, lambda0=1.0, lambda1=1.0, lambda2=1.0)
    THR, RAT = _lib.MOECA_MODE_THRESHOLD, _lib.MOECA_MODE_RATIO
    configs = [("paper (adaptive, alpha 0.6)", {})]
    configs += [(f"fixed threshold (alpha 0)", dict(alpha=0.0))]
    configs += [(f"alpha {a}", dict(alpha=a)) for a in (0.4, 0.8)]
    configs += [(f"tau0 {v:.2f}", dict(tau0=v)) for v in (0.65, 0.70, 0.75, 0.85, 0.90, 0.95, 1.00)]
    configs += [(f"beta {v:.2f}", dict(beta=v)) for v in (0.45, 0.55, 0.75, 0.85)]
    signals = (("w only", (1, 0, 0)), ("Delta only", (0, 1, 0)), ("o only", (0, 0, 1)),
               ("w + Delta", (1, 1, 0)), ("w + o", (1, 0, 1)), ("Delta + o", (0, 1, 1)))
    for name, lam in signals:
        configs.append((f"score: {name}", dict(lambda0=float(lam[0]), lambda1=float(lam[1]),
                                               lambda2=float(lam[2]))))
    # the same ablation at an equal budget (ratio mode, 30 % of the branches
    # per sample): the output deviation then compares how well each score
    # ranks branches, at the same compute
    configs.append(("ratio 0.3, score: all", dict(mode=RAT, ratio=0.3)))
    for name, lam in signals:
        configs.append((f"ratio 0.3, score: {name}",
                        dict(mode=RAT, ratio=0.3, lambda0=float(lam[0]),
                             lambda1=float(lam[1]), lambda2=float(lam[2]))))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    rows = []
    for name, kw in configs:
        pol = dict(base, **kw)
        mode = pol.pop("mode", THR)
        L = make_layer(mode, pol)
        L.reset()
        rec, rom, err_l2, err_max = [], [], [], []
        for t in range(T):
            L.step(xs[t], t, out)
            st = L.stats()  # synchronises
            y = f32(out)
            r = ref[t]
            err_l2.append(float(torch.linalg.vector_norm(y - r) / torch.linalg.vector_norm(r)))
            err_max.append(float((y - r).abs().max() / r.abs().max()))
            if not st.full_step:
                rec.append(st.n_recompute / st.n_branches)
                rom.append(st.reuse_over_match)
        L.reset()
        torch.cuda.synchronize()
        e0.record()
        for t in range(T):
            L.step(xs[t], t, out)
        e1.record()
        torch.cuda.synchronize()
        L.close()
        rows.append({"config": name, "mode": "ratio" if mode == RAT else "threshold",
                     "ratio": pol.get("ratio"), **{k: pol[k] for k in base},
                     "recompute_share": round(float(np.mean(rec)), 4),
                     "reuse_over_match": round(float(np.mean(rom)), 4),
                     "reuse_over_match_per_step": [round(v, 4) for v in rom],
                     "rel_l2_err": round(float(np.mean(err_l2)), 5),
                     "max_rel_err": round(float(np.mean(err_max)), 5),
                     "ms_per_step": round(e0.elapsed_time(e1) / T, 4)})
        log(f"[policy] {name}: recompute {rows[-1]['recompute_share']:.3f} "
            f"reuse/match {rows[-1]['reuse_over_match']:.3f} l2 {rows[-1]['rel_l2_err']:.4f} "
            f"{rows[-1]['ms_per_step']:.3f} ms")
    return rows


def stack_bench(args):
    """The DiT-MoE block stack: one sampling step = the timestep/class
    embedding plus every block (attention, AdaLN, the branch-cached MoE
    layer).  Cache steps (ratio mode, refresh cycle off after the first
    full step) against the uncached comparator's full steps, both replayed
    from HIP graphs of K steps."""
    import torch
    from paper_2606_15615_amd import _lib
    from paper_2606_15615_amd.stack import MoecaStack
    from paper_2606_15615_amd.synth import STACKS, StackSynth

    _lib.load()  # fails loudly when the library is not built
    sh = STACKS[args.workload]
    ratio = 0.3 if args.ratio is None else args.ratio
    dev = torch.device("cuda:0")
    K, Wm = args.steps, args.warmup
    T = Wm + K
    log(f"[bench] stack {args.workload} {sh}; generating weights on the GPU")
    syn = StackSynth(sh, args.seed)
    weights = [syn.block_device(l, dev) for l in range(sh.L)]
    emb = syn.embedder_device(dev)
    labels = torch.from_numpy(syn.labels().astype(np.int32)).to(dev)
    tv = syn.timestep_values(T)
    t_rows = [torch.full((sh.B,), float(v), dtype=torch.float32, device=dev) for v in tv]
    xs = syn.trajectory_device(T, dev)
    x = torch.empty_like(xs[0])
    c = torch.empty((sh.B, sh.d), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()

    def make(mode):
        S = MoecaStack(sh.L, sh.d, sh.heads, sh.E, sh.k, sh.d_ff, batch=sh.B, tokens=sh.N,
                       mode=mode, ratio=ratio, refresh_cycle=0)
        for l, w in enumerate(weights):
            S.set_block(l, w["W_ada"], w["b_ada"], w["W_qkv"], w["b_qkv"], w["W_o"], w["b_o"],
                        w["W_r"], None, w["W_up"], w["W_down"])
        S.reset()
        return S

    def one(S, t):
        x.copy_(xs[t])
        S.embed(t_rows[t], labels, emb["W1"], emb["b1"], emb["W2"], emb["b2"], emb["table"], c)
        S.step(x, c, t)

    def run(S, t0, t1):
        for t in range(t0, t1):
            one(S, t)

    def measure(S, warm):
        S.reset()
        run(S, 0, warm)
        torch.cuda.synchronize()
        e0.record(stream)
        run(S, warm, T)
        e1.record(stream)
        torch.cuda.synchronize()
        ms_eager = e0.elapsed_time(e1) / K
        ms_graph, graphed = ms_eager, False
        if not args.no_graph:
            S.reset()
            run(S, 0, warm)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                run(S, warm, T)
            g.replay()
            torch.cuda.synchronize()
            S.reset()
            run(S, 0, warm)
            torch.cuda.synchronize()
            e0.record(stream)
            g.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            ms_graph, graphed = e0.elapsed_time(e1) / K, True
            del g
        # counts of the same steps
        S.reset()
        run(S, 0, warm)
        rec = syn_n = 0
        for t in range(warm, T):
            one(S, t)
            for l in range(sh.L):
                st = S.layer(l).stats()
                rec += st.n_recompute
                syn_n += st.n_sync
        return ms_eager, ms_graph, graphed, rec / K / sh.L, syn_n / K / sh.L

    c_eager = c_graph = f_eager = f_graph = None
    graphed, rec, syn_n = False, 0.0, 0.0
    if args.phase in ("both", "cached"):
        log("[bench] cache steps")
        S = make(_lib.MOECA_MODE_RATIO)
        c_eager, c_graph, graphed, rec, syn_n = measure(S, Wm)
        S.close()
        del S
    if args.phase in ("both", "full"):
        log("[bench] full steps (uncached comparator)")
        S = make(_lib.MOECA_MODE_FULL)
        f_eager, f_graph, g2, _, _ = measure(S, min(Wm, 2))
        graphed = graphed or g2
        S.close()

    def r4(v):
        return None if v is None else round(v, 4)
    branches = sh.B * sh.N * sh.k
    wl = (f"{args.workload}: {sh.L} DiT-MoE blocks d={sh.d}, {sh.heads} heads x {sh.d // sh.heads}, "
          f"E={sh.E} top-{sh.k} d_ff={sh.d_ff} GELU, {sh.N} tokens x batch {sh.B}, "
          f"timestep + class embedding, ratio mode rho={ratio}")
    value = c_graph if c_graph is not None else f_graph
    res = {"metric": "DiT-MoE stack sampling step (cache step)", "value": r4(value),
           "unit": "ms/step", "n_gpus": 1, "steps": K, "warmup": Wm, "higher_is_better": False,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "ms_per_step": r4(value), "launch": "hip_graph" if graphed else "eager",
           "eager_ms_per_step": r4(c_eager), "full_ms_per_step": r4(f_graph),
           "eager_full_ms_per_step": r4(f_eager),
           "cached_over_full": (round(c_graph / f_graph, 4)
                                if c_graph is not None and f_graph is not None else None),
           "refresh_ratio_actual": round(rec / branches, 4),
           "synchronized_token_frac": round(syn_n / (sh.B * sh.N), 4),
           "config": {"workload": wl, "batch": sh.B, "tokens": sh.N, "blocks": sh.L}}
    print(json.dumps(res), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); "
              "the library has no multi-GPU path", file=sys.stderr)
        sys.exit(2)
    from paper_2606_15615_amd.synth import STACKS
    if args.workload in STACKS:
        stack_bench(args)
        return
    import torch
    from paper_2606_15615_amd import _lib
    from paper_2606_15615_amd.layer import MoecaLayer, np_to_device
    from paper_2606_15615_amd.synth import WORKLOADS, Synth

    _lib.load()  # fails loudly when the library is not built
    shape = WORKLOADS[args.workload]
    fine = shape.n_shared > 0 or shape.ffn == "swiglu"
    if args.ratio is None:
        args.ratio = 0.25 if fine else 0.3
    if args.blas_reference:
        print(json.dumps({"reference": "torch.bmm bf16 (vendor BLAS)", "workload": args.workload,
                          "gemms": blas_reference(shape, args)}), flush=True)
        return
    act = "swiglu" if shape.ffn == "swiglu" else "gelu_tanh"
    norm_topk = not fine  # the fine-grained layer keeps the softmax gate values
    dev = torch.device("cuda:0")
    K, Wm = args.steps, args.warmup
    T = Wm + K
    do_cached = args.phase in ("both", "cached")
    do_full = args.phase in ("both", "full")
    log(f"[bench] workload {args.workload} {shape}; phase {args.phase}; generating inputs")
    # the skewed-routing layer: Zipf(1.2) router prior, bimodal token drift
    bias, drift = ("zipf", "bimodal") if args.workload == "skewed" else (None, "loguniform")
    sy = Synth(shape, args.seed)
    W = sy.weights(bias)
    dW = [np_to_device(W[0], dev), None if W[1] is None else np_to_device(W[1], dev),
          np_to_device(W[2], dev), np_to_device(W[3], dev)]
    del W
    Wsh = sy.shared_weights()
    dWsh = None if Wsh is None else [np_to_device(w, dev) for w in Wsh]
    del Wsh
    xs = [np_to_device(x, dev) for x in sy.trajectory(T, drift)]
    attn = np_to_device(next(sy.attention_trajectory(1, drift)), dev)
    attn_cache = torch.zeros_like(attn)
    out = torch.empty_like(xs[0])
    torch.cuda.synchronize()

    def make(mode, ratio=args.ratio):
        L = MoecaLayer(shape.d, shape.E, shape.k, shape.d_ff, batch=shape.B, tokens=shape.N,
                       mode=mode, ratio=ratio, refresh_cycle=0, dtype=shape.dtype, act=act,
                       norm_topk=norm_topk, n_shared=shape.n_shared)
        L.set_weights(*dW)
        if dWsh is not None:
            L.set_shared(*dWsh)
        L.bind_attention(attn, attn_cache)
        L.reset()
        return L

    stream = torch.cuda.current_stream()
    if args.policy_study:
        def make_policy_layer(mode, pol):
            L = MoecaLayer(shape.d, shape.E, shape.k, shape.d_ff, batch=shape.B,
                           tokens=shape.N, mode=mode, refresh_cycle=4, dtype=shape.dtype,
                           act=act, norm_topk=norm_topk, n_shared=shape.n_shared, **pol)
            L.set_weights(*dW)
            if dWsh is not None:
                L.set_shared(*dWsh)
            L.reset()
            return L
        rows = policy_study(args, shape, make_policy_layer, xs, out, _lib)
        print(json.dumps({"policy_study": rows, "workload": args.workload, "steps": T,
                          "data": "synthetic", "drift": drift}), flush=True)
        return

    def run(L, t0, t1):
        for t in range(t0, t1):
            L.step(xs[t], t, out)

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(L, t0, t1):
        torch.cuda.synchronize()
        e0.record(stream)
        run(L, t0, t1)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / (t1 - t0)

    def graph_timed(L, warm):
        """Capture the K steps in one HIP graph; replay it once untimed (the
        first replay also uploads the graph), rewind the layer to the same
        state (reset + the warm-up steps, eager), then time one replay."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            run(L, Wm, T)
        g.replay()
        torch.cuda.synchronize()
        L.reset()
        run(L, 0, warm)
        torch.cuda.synchronize()
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K

    def phase(L, warm):
        """Eager timed region with per-kernel events (the library records
        them on the launch stream between kernels), then the same K steps
        replayed from a HIP graph, then an untimed replay for the counts."""
        L.reset()
        run(L, 0, warm)                      # step 0 is the refresh step
        L.set_timing(True)
        ms_eager = timed(L, Wm, T)
        stage, n = L.timing()
        L.set_timing(False)
        # the entropy of the statistic runs inside the select kernel: the
        # statistic stage launches nothing, so its event pair is left out
        stage = {k: v / n for k, v in stage.items() if k != "stat"}
        ms_graph, graphed = ms_eager, False
        if not args.no_graph:
            try:
                L.reset()
                run(L, 0, warm)
                ms_graph = graph_timed(L, warm)
                graphed = True
            except Exception as exc:  # capture unsupported: report the eager numbers
                log(f"[bench] graph capture failed ({exc}); reporting eager timings")
        # the same steps once more, one at a time: counts, and (optionally)
        # each step timed alone after a write of flush_mib MiB, which leaves
        # none of the weights in the 256 MB MALL
        L.reset()
        run(L, 0, warm)
        torch.cuda.synchronize()
        rec, syn, flushed, plan = [], [], [], []
        for t in range(Wm, T):
            if flush is not None:
                flush.fill_(t & 0xff)
                e0.record(stream)
            L.step(xs[t], t, out)
            if flush is not None:
                e1.record(stream)
            st = L.stats()  # synchronises
            if flush is not None:
                flushed.append(e0.elapsed_time(e1))
            rec.append(st.n_recompute)
            syn.append(st.n_sync)
            plan.append(st.ffn_plan)
        ms_flushed = float(np.mean(flushed)) if flushed else None
        return ms_eager, ms_graph, graphed, stage, (rec, syn, ms_flushed, plan)

    flush = (torch.empty(args.flush_mib << 20, dtype=torch.uint8, device=dev)
             if args.flush_mib > 0 else None)
    res_c = res_f = None
    if do_cached:
        log("[bench] cache steps")
        cached = make(_lib.MOECA_MODE_RATIO)
        res_c = phase(cached, Wm)
        cached.close()
    if do_full:
        log("[bench] full recompute")
        full = make(_lib.MOECA_MODE_FULL)
        res_f = phase(full, min(Wm, 3))
        full.close()

    sweep = []
    for rho in [float(v) for v in args.sweep.split(",") if v.strip()]:
        log(f"[bench] sweep: cache steps at ratio {rho}")
        Ls = make(_lib.MOECA_MODE_RATIO, ratio=rho)
        ms_e, ms_g, graphed_s, stage_s, (rec_s, _, _, _) = phase(Ls, Wm)
        Ls.close()
        sweep.append({"ratio": rho, "ms_per_step": round(ms_g, 4),
                      "refresh_ratio_actual": round(float(np.mean(rec_s)) / (shape.tokens * shape.k), 4),
                      "ffn_ms": round(stage_s["ffn_up"] + stage_s["ffn_down"], 4)})

    if args.copy_mib:
        n = args.copy_mib * (1 << 20)
        a = torch.empty(n, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()

    branches = shape.B * shape.N * shape.k
    # flop per row of the up and the down projection (routed branch or
    # shared-expert token row); the shared experts add S * T rows per step
    up_flop = 2.0 * shape.d * shape.up_rows
    down_flop = 2.0 * shape.d * shape.d_ff
    shared_rows = shape.n_shared * shape.tokens
    peak = PEAK_BF16_TFLOPS if shape.dtype == "bf16" else PEAK_FP32_TFLOPS
    abytes = 2 if shape.dtype == "bf16" else 4
    wl = (f"{args.workload}: MoE layer d={shape.d}, E={shape.E}, top-{shape.k}, "
          f"d_ff={shape.d_ff} {'SwiGLU' if act == 'swiglu' else 'GELU'}"
          + (f", {shape.n_shared} shared experts" if shape.n_shared else "")
          + (", unnormalised top-k gates" if not norm_topk else "")
          + f", {shape.N} tokens x batch {shape.B}, ratio mode rho={args.ratio}"
          + (", Zipf(1.2) router prior, bimodal drift" if bias else ""))
    res = {"metric": METRIC, "unit": "ms/step", "n_gpus": 1, "steps": K, "warmup": Wm,
           "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
           "dtype": shape.dtype, "data": "synthetic",
           "config": {"workload": wl, "batch": shape.B, "tokens": shape.N, "phase": args.phase}}
    if res_c is not None:
        ms_eager, ms_graph, graphed, stage, (rec, syn, ms_flushed, plan) = res_c
        mean_rec = float(np.mean(rec))
        up_ms = stage["ffn_up"]
        down_ms = stage["ffn_down"]
        ffn_ms = up_ms + down_ms
        rows = mean_rec + shared_rows
        ffn_tf = rows * (up_flop + down_flop) / (ffn_ms * 1e-3) / 1e12
        # algorithmic HBM bytes of a cache step: expert weights (routed and
        # shared), inputs, cached rows, recomputed rows written, shared
        # outputs written and read, outputs (the attention refresh excluded)
        wbytes = (shape.E + shape.n_shared) * (shape.up_rows + shape.d_ff) * shape.d * abytes
        step_bytes = (wbytes + shape.tokens * shape.d * abytes * 2 + branches * shape.d * abytes
                      + 2 * shared_rows * shape.d * abytes)
        # per GEMM launch: flop (2 d d_ff per row) and algorithmic bytes (the
        # weights of every expert, which a cache step at these ratios reads
        # whole, and per row its input row read and its output row written)
        up_w = (shape.E + shape.n_shared) * shape.up_rows * shape.d * abytes
        down_w = (shape.E + shape.n_shared) * shape.d_ff * shape.d * abytes
        gemms = {
            "ffn_up": {"ms": up_ms, "flop": rows * up_flop,
                       "bytes": up_w + rows * (shape.d + shape.d_ff) * abytes},
            "ffn_down": {"ms": down_ms, "flop": rows * down_flop,
                         "bytes": down_w + rows * (shape.d_ff + shape.d) * abytes},
        }
        for g in gemms.values():
            g["tflops"] = g["flop"] / (g["ms"] * 1e-3) / 1e12
            g["gbs"] = g["bytes"] / (g["ms"] * 1e-3) / 1e9
            g["intensity"] = g["flop"] / g["bytes"]
        # the dominant kernel: the longer of the two GEMM launches; its roof
        # is the lower of the MFMA peak and intensity x HBM peak
        dom = max(gemms, key=lambda n: gemms[n]["ms"])
        g = gemms[dom]
        hbm_bound = g["intensity"] * PEAK_HBM_GBS / 1e3 < peak
        traffic = kernel_traffic(os.path.join(ROOT, "paper_2606_15615_amd", "csrc", "ffn.hip"),
                                 os.path.join(ROOT, "profiles", "xl1024_cached_counters.txt"),
                                 dom)
        if args.workload != "xl1024":
            traffic = None
        swiglu = act == "swiglu"
        thin = np.mean(np.array(plan) == 1) > 0.5
        wide = np.mean(np.array(plan) == 2) > 0.5
        kernel_names = {
            "ffn_up": ("gemm_bf16_big_kernel<0,3> (expert FFN up-projection + SwiGLU)" if swiglu
                       else "gemm_bf16_thin_kernel<0,0,1> (expert FFN up-projection + GELU, "
                            "weight-streaming tiles)" if thin
                       else "gemm_bf16_wide_kernel<0> (expert FFN up-projection + GELU, "
                            "expert-wide tiles)" if wide
                       else "gemm_bf16_big_kernel<0,0> (expert FFN up-projection + GELU)"),
            "ffn_down": ("gemm_bf16_thin_kernel<1,2,4> + reduce_partials_kernel<4> (expert FFN "
                         "down-projection, weight-streaming tiles in four K pieces)" if thin
                         else "gemm_bf16_big_kernel<1,2> (expert FFN down-projection, "
                              "scattered into the cache slots)"),
        }
        roof = {
            "bound": "hbm" if hbm_bound else "mfma",
            "kernel": kernel_names[dom],
            "achieved": round(g["gbs"] if hbm_bound else g["tflops"], 2),
            "peak": PEAK_HBM_GBS if hbm_bound else peak,
            "unit": "GB/s" if hbm_bound else "TFLOP/s",
            "frac": round(g["gbs"] / PEAK_HBM_GBS if hbm_bound else g["tflops"] / peak, 4),
            "traffic": None if traffic is None else int(traffic),
            "launch_ms": round(g["ms"], 4),
            "flop_per_launch": g["flop"],
            "bytes_per_launch": g["bytes"],
            "intensity_flop_per_byte": round(g["intensity"], 1),
            "ridge_flop_per_byte": round(peak * 1e3 / PEAK_HBM_GBS, 1),
            # the same launch against the MFMA peak
            "mfma_tflops": round(g["tflops"], 2),
            "mfma_frac": round(g["tflops"] / peak, 4),
        }
        res.update({
            "value": round(ms_graph, 4),
            "ms_per_step": round(ms_graph, 4),
            "launch": "hip_graph" if graphed else "eager",
            "eager_ms_per_step": round(ms_eager, 4),
            "flushed_ms_per_step": None if ms_flushed is None else round(ms_flushed, 4),
            "tflops_recomputed": round(ffn_tf, 2),
            "refresh_ratio_actual": round(mean_rec / branches, 4),
            "recomputed_branches": round(mean_rec, 1),
            "shared_expert_rows": shared_rows,
            "synchronized_tokens": round(float(np.mean(syn)), 1),
            # tiling of the expert FFN on the counted steps: 0 the 128 x 256
            # tiles, 1 the weight-streaming tiles, 2 the expert-wide
            # up-projection tiles
            "ffn_plan_steps": {str(v): int(c) for v, c in zip(*np.unique(plan, return_counts=True))},
            "stage_ms": {k: round(v, 4) for k, v in stage.items()},
            "step_hbm_frac": round(step_bytes / (ms_graph * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "gemm_launches": {n: {"ms": round(v["ms"], 4), "tflops": round(v["tflops"], 1),
                                  "mfma_frac": round(v["tflops"] / peak, 4),
                                  "gbs": round(v["gbs"], 1),
                                  "hbm_frac": round(v["gbs"] / PEAK_HBM_GBS, 4)}
                              for n, v in gemms.items()},
            "roofline": roof,
        })
    if res_f is not None:
        ms_eager_f, ms_graph_f, _, stage_f, (_, _, ms_flushed_f, _) = res_f
        res.update({"full_ms_per_step": round(ms_graph_f, 4),
                    "full_flushed_ms_per_step": None if ms_flushed_f is None else round(ms_flushed_f, 4),
                    "eager_full_ms_per_step": round(ms_eager_f, 4),
                    "full_stage_ms": {k: round(v, 4) for k, v in stage_f.items()}})
        if res_c is None:
            res.update({"value": round(ms_graph_f, 4), "ms_per_step": round(ms_graph_f, 4)})
    if res_c is not None and res_f is not None:
        res["cached_over_full"] = round(res_c[1] / res_f[1], 4)
        res["speedup_vs_full"] = round(res_f[1] / res_c[1], 3)
    if sweep:
        res["ratio_sweep"] = sweep
    if not args.no_cpu and res_c is not None:
        log("[bench] cpu baseline (oracle)")
        res["cpu_baseline"] = cpu_baseline(shape, args.ratio, args.seed, norm_topk, act,
                                           reps=1 if fine else 3)
        log(f"[bench] cpu baseline done: {res['cpu_baseline']}")
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
