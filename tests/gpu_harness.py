"""Helpers for the GPU parity tests.

Protocol (oracle-forced): the oracle runs its own trajectory from seeded
synthetic inputs.  Before each step its state is written into the GPU
layer's workspace, the GPU step runs, and every decision the step takes is
compared bit for bit with the oracle's; stored features and outputs are
compared within the floating-point tolerance (bf16 2e-2, fp32 1e-4, max
relative error over the tensor).  Inputs only ever flow oracle -> GPU.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from oracle import moeca_oracle as O
from paper_2606_15615_amd import _lib
from paper_2606_15615_amd.layer import MoecaLayer, device_to_np, np_to_device
from paper_2606_15615_amd.synth import LayerShape, Synth

TOL = {"bf16": 2e-2, "fp32": 1e-4}
MODE = {"full": _lib.MOECA_MODE_FULL, "threshold": _lib.MOECA_MODE_THRESHOLD,
        "ratio": _lib.MOECA_MODE_RATIO}
OMODE = {"full": O.MODE_FULL, "threshold": O.MODE_THRESHOLD, "ratio": O.MODE_RATIO}


def say(msg):
    print(msg, flush=True)


def full_step_plan(shape: LayerShape) -> int:
    """FFN tiling the library takes on a full step of this layer: the
    expert-wide up projection (2) when every branch leaves at most 320 rows
    per expert on average and the layer can take it (bf16, ungated, no
    shared experts, hidden width a multiple of 144), else the 128-row tiles
    (0)."""
    wide_capable = (shape.dtype == "bf16" and shape.n_shared == 0 and shape.ffn == "gelu"
                    and shape.d_ff % 144 == 0 and shape.tokens * shape.d < 2 ** 31)
    return 2 if wide_capable and shape.branches <= 320 * shape.E else 0


class Setup:
    """Seeded weights + trajectory, the oracle objects and a GPU layer."""

    def __init__(self, shape: LayerShape, mode="ratio", seed=0, T=4, attention=True,
                 bias=None, drift="loguniform", **pol):
        self.shape = shape
        self.mode = mode
        self.sy = Synth(shape, seed)
        W = self.sy.weights(bias)
        self.dims = O.Dims(shape.d, shape.E, shape.k, shape.d_ff, shape.B, shape.N, shape.dtype,
                           shape.n_shared)
        Wsh = self.sy.shared_weights()
        self.W = O.Weights(self.dims, *W, *(Wsh or (None, None)))
        if shape.ffn == "swiglu":
            pol.setdefault("act", "swiglu")
        self.xs = list(self.sy.trajectory(T, drift)) if T else []
        self.attn = list(self.sy.attention_trajectory(T)) if (T and attention) else None
        self.pol = O.Policy(mode=OMODE[mode], **pol)
        self.layer = self._new_layer()
        dev = self.layer.device
        self.dW = [np_to_device(W[0], dev),
                   None if W[1] is None else np_to_device(W[1], dev),
                   np_to_device(W[2], dev), np_to_device(W[3], dev)]
        self.dWsh = None if Wsh is None else [np_to_device(w, dev) for w in Wsh]
        self.attention = attention
        self._bind()

    def _new_layer(self):
        shape, pol = self.shape, self.pol
        return MoecaLayer(shape.d, shape.E, shape.k, shape.d_ff, batch=shape.B,
                          tokens=shape.N, mode=MODE[self.mode], dtype=shape.dtype,
                          ratio=pol.ratio, tau0=pol.tau0, alpha=pol.alpha, beta=pol.beta,
                          lambda1=pol.lambda1, lambda2=pol.lambda2, lambda0=pol.lambda0,
                          refresh_cycle=pol.refresh_cycle, norm_topk=pol.norm_topk,
                          act=pol.act, n_shared=shape.n_shared)

    def _bind(self):
        import torch
        shape, dev = self.shape, self.layer.device
        self.layer.set_weights(*self.dW)
        if self.dWsh is not None:
            self.layer.set_shared(*self.dWsh)
        self.act_np = np.uint16 if shape.dtype == "bf16" else np.float32
        tdt = torch.int16 if shape.dtype == "bf16" else torch.float32
        self.attn_in = torch.zeros((shape.B, shape.N, shape.d), dtype=tdt, device=dev)
        self.attn_cache = torch.zeros_like(self.attn_in)
        if self.attention:
            self.layer.bind_attention(self.attn_in, self.attn_cache)
        self.out = torch.zeros((shape.B, shape.N, shape.d), dtype=tdt, device=dev)
        self.layer.reset()

    def with_policy(self, **changes):
        """Another GPU layer on the same weights, inputs and oracle objects,
        with some policy fields changed."""
        import copy
        other = copy.copy(self)
        other.pol = dataclasses.replace(self.pol, **changes)
        other.layer = other._new_layer()
        other._bind()
        return other

    def release(self):
        """Destroy this setup's GPU layer and its workspace now."""
        import torch
        self.layer.close()
        self.layer = None
        torch.cuda.synchronize()

    # -- state transfer (oracle -> GPU) --------------------------------
    def import_state(self, st: O.State):
        import torch
        L = self.layer
        L.write("e_c", st.e_c.reshape(-1))
        L.write("w_c", st.w_c.reshape(-1))
        L.write("n_c", st.n_c.reshape(-1))
        L.write("h_c", st.h_c.reshape(-1, self.shape.d))
        L.write("stat", st.C)
        L.set_valid(st.valid)
        if self.attention and st.A is not None:
            self.attn_cache.copy_(np_to_device(st.A, L.device))
        torch.cuda.synchronize()

    def gpu_step(self, x_np, t, attn_np=None):
        import torch
        L = self.layer
        x = np_to_device(x_np, L.device)
        if attn_np is not None:
            self.attn_in.copy_(np_to_device(attn_np, L.device))
        L.step(x, t, self.out)
        torch.cuda.synchronize()
        return device_to_np(self.out, self.act_np)

    def gpu_state(self):
        L = self.layer
        st = O.State(self.dims, attention=self.attention)
        st.e_c = L.read("e_c").reshape(st.e_c.shape)
        st.w_c = L.read("w_c").reshape(st.w_c.shape)
        st.n_c = L.read("n_c").reshape(st.n_c.shape)
        st.h_c = L.read("h_c").reshape(st.h_c.shape)
        st.C = L.read("stat")
        if self.attention:
            st.A = device_to_np(self.attn_cache, self.act_np)
        return st


def near_f32_tie(v64: np.ndarray, rel=2.0 ** -40) -> np.ndarray:
    """True where an fp64 value sits within rounding noise of the midpoint
    between two fp32 numbers: either fp32 rounding of it is then correct."""
    r = v64.astype(np.float32)
    up = np.nextafter(r, np.float32(np.inf)).astype(np.float64)
    dn = np.nextafter(r, np.float32(-np.inf)).astype(np.float64)
    r64 = r.astype(np.float64)
    tol = rel * np.maximum(np.abs(v64), 1e-300)
    return (np.abs(v64 - (r64 + up) / 2) <= tol) | (np.abs(v64 - (r64 + dn) / 2) <= tol)


def rel_err(a, b, dtype) -> float:
    a64 = O.to_f64(a, dtype)
    b64 = O.to_f64(b, dtype)
    den = np.abs(b64).max()
    return float(np.abs(a64 - b64).max() / den) if den > 0 else float(np.abs(a64).max())


def entropy_tolerance(C: np.ndarray, Hbar: np.ndarray) -> np.ndarray:
    """Largest |difference| of two evaluations of the normalised entropy of
    the statistic C (B, E, N) that differ only in fp64 summation order and
    form: the library's (S log S - sum C log C) / S and the oracle's
    -sum P log P.  Each form carries at most gamma_n (S |log S| +
    sum |C log C|) / S of fp64 rounding error (n = N + 4 terms in a chain),
    the two together twice that; divided by log N; plus one fp32 ulp of the
    final rounding."""
    B, E, N = C.shape
    C64 = C.astype(np.float64)
    S = C64.sum(axis=2)
    with np.errstate(divide="ignore", invalid="ignore"):
        clc = np.where(C64 > 0, np.abs(C64 * np.log(np.where(C64 > 0, C64, 1.0))), 0.0).sum(axis=2)
        mag = np.where(S > 0, (S * np.abs(np.log(np.where(S > 0, S, 1.0))) + clc) / np.where(S > 0, S, 1.0), 0.0)
    gamma = (N + 4) * 2.0 ** -53
    logn = np.log(N) if N > 1 else 1.0
    ulp = np.spacing(np.maximum(np.abs(Hbar), np.float32(2.0 ** -126)).astype(np.float32)).astype(np.float64)
    return 2.0 * gamma * mag / logn + ulp


def check_step(S: Setup, t: int, rec: dict, out_o, st_old: O.State, st_new: O.State,
               out_g, evaluated=None, uncached=False, label="", rerun=None):
    """Compare one GPU step with the oracle's.  Returns a dict of metrics.

    ``rerun(forced)`` re-runs the oracle step with rounded decision inputs
    taken from the GPU (``O.step(..., forced=...)``).  Where a router logit
    or a normalised entropy lies at an fp32 rounding tie both roundings are
    correct; the checker then adopts the GPU's value and still compares
    every later decision bit for bit, every row and the output."""
    L = S.layer
    dims, dt = S.dims, S.shape.dtype
    B, N, k, E, d = dims.B, dims.N, dims.k, dims.E, dims.d
    tol = TOL[dt]
    info = {"label": label, "t": t, "ffn_plan": int(L.stats().ffn_plan)}
    forced = {}

    # router: logits bit-exact unless the oracle's fp64 sum is a near-tie
    lg = L.read("logits")
    diff = lg != rec["logits"]
    if diff.any():
        assert near_f32_tie(rec["logits64"][diff]).all(), \
            f"{label} t={t}: {int(diff.sum())} router logits differ away from a rounding tie"
        assert rerun is not None, f"{label} t={t}: logit tie and no way to re-run the oracle"
        info["logit_ties"] = int(diff.sum())
        say(f"  {label} t={t}: {int(diff.sum())} logits at an fp32 rounding tie; "
            "oracle re-run on the GPU's logits")
        forced["logits"] = lg
        out_o, st_new, rec = rerun(dict(forced))
    if not uncached:
        assert np.array_equal(L.read("stat"), rec["C"]), "EMA statistic"
        hb = L.read("hbar").reshape(rec["Hbar"].shape)
        hd = hb != rec["Hbar"]
        if hd.any():
            tolh = entropy_tolerance(rec["C"], rec["Hbar"])
            gap = np.abs(hb.astype(np.float64) - rec["Hbar"].astype(np.float64))
            assert (gap[hd] <= tolh[hd]).all(), \
                f"{label} t={t}: normalised entropy differs beyond the fp64 rounding bound"
            info["hbar_rounding"] = int(hd.sum())
            if not np.array_equal(L.read("tau").reshape(hb.shape), rec["tau"]):
                assert rerun is not None, f"{label} t={t}: entropy tie and no way to re-run"
                say(f"  {label} t={t}: {int(hd.sum())} normalised entropies differ by rounding; "
                    "oracle re-run on the GPU's values")
                forced["Hbar"] = hb
                out_o, st_new, rec = rerun(dict(forced))
                assert np.array_equal(L.read("logits"), rec["logits"])
        assert np.array_equal(L.read("tau").reshape(rec["tau"].shape), rec["tau"]), "thresholds"
    assert np.array_equal(L.read("e_t"), rec["e_t"].reshape(-1)), "e_t"
    assert np.array_equal(L.read("w_t"), rec["w_t"].reshape(-1)), "w_t"

    if not rec["full"]:
        q = L.read("q").reshape(B, N, k)
        assert np.array_equal(q, rec["q"]), "matching q(p)"
        m = L.read("margin").reshape(B, N, k)
        mm = rec["matched"]
        assert np.array_equal(m[mm], rec["m"][mm]), "margins"
    mask = L.read("mask").reshape(B, N, k).astype(bool)
    assert np.array_equal(mask, rec["mask"]), \
        f"mask: {int((mask != rec['mask']).sum())} branches differ"
    assert np.array_equal(L.read("sigma").reshape(B, N, k), rec["sigma"]), "slots"
    off = L.read("off")
    assert np.array_equal(off, rec["off"]), "expert offsets"
    assert np.array_equal(L.read("list")[:off[-1]], rec["lst"]), "expert lists"
    assert np.array_equal(L.read("pos"), rec["pos"]), "list positions"
    if not uncached:
        assert np.array_equal(L.read("sync").reshape(B, N).astype(bool), rec["S"]), "sync mask"

    ev = np.ones((B, N), bool) if evaluated is None else evaluated
    # layer output
    e = rel_err(out_g[ev], out_o[ev], dt)
    info["out_rel_err"] = e
    assert e <= tol, f"{label} t={t}: output rel err {e:.3g} > {tol}"

    if uncached:
        info["state"] = st_new
        return info
    g = S.gpu_state()
    assert np.array_equal(g.e_c, st_new.e_c), "cached expert ids"
    assert np.array_equal(g.w_c, st_new.w_c), "cached gate weights"
    written = np.zeros((B, N, k), bool)
    bb, ii, pp = np.nonzero(rec["mask"])
    written[bb, ii, rec["sigma"][bb, ii, pp]] = True
    keep = ~written
    assert np.array_equal(g.h_c[keep], st_old.h_c[keep]), "reused rows must be untouched"
    assert np.array_equal(g.n_c[keep], st_old.n_c[keep]), "reused norms must be untouched"
    wr = written & ev[..., None]
    if wr.any():
        er = rel_err(g.h_c[wr], st_new.h_c[wr], dt)
        info["row_rel_err"] = er
        assert er <= tol, f"recomputed rows rel err {er:.3g}"
        rows64 = O.to_f64(g.h_c[wr], dt)
        own = np.sqrt(np.sum(rows64 * rows64, axis=-1)).astype(np.float32)
        assert np.array_equal(g.n_c[wr], own), "norm must be that of the stored row"
        assert np.allclose(g.n_c[wr], st_new.n_c[wr], rtol=tol), "norms vs oracle"
    if S.attention:
        assert np.array_equal(g.A, st_new.A), "attention cache"
    sg = L.stats()
    so = rec["stats"]
    assert sg.n_recompute == so["n_recompute"] and sg.n_sync == so["n_sync"]
    assert sg.n_unmatched == so["n_unmatched"] and sg.n_matched == so["n_matched"]
    assert sg.full_step == int(rec["full"])
    info["recompute_frac"] = so["n_recompute"] / (B * N * k)
    info["state"] = st_new
    return info


def oracle_rerun(S: Setup, st: O.State, x, t: int, attn=None, tokens=None):
    """The oracle step from state ``st`` as a function of forced values."""
    return lambda forced: O.step(S.dims, S.pol, S.W, st, x, t, attn_in=attn, tokens=tokens,
                                 forced=forced)


def run_forced(S: Setup, T: int, label=""):
    """Oracle trajectory; every step checked from the oracle's own state."""
    st = O.State(S.dims, attention=S.attention)
    infos = []
    for t in range(T):
        say(f"  [{label}] step {t}")
        S.import_state(st)
        a = None if S.attn is None else S.attn[t]
        out_g = S.gpu_step(S.xs[t], t, a)
        rerun = oracle_rerun(S, st, S.xs[t], t, a)
        out_o, st_new, rec = rerun(None)
        info = check_step(S, t, rec, out_o, st, st_new, out_g,
                          uncached=S.pol.mode == O.MODE_FULL, label=label, rerun=rerun)
        infos.append(info)
        st = info.pop("state")   # the oracle state the step was compared against
    return infos
