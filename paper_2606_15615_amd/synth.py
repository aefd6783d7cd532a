"""Seeded synthetic inputs for the branch-cached MoE layer step.

This module only draws random numbers and stores them in the layouts the
library and the oracle take.  It holds none of the method's arithmetic
(no routing, scoring, selection, expert FFN or combine).  Both the GPU path
(tests, bench) and the CPU oracle (tests) read their inputs from here.

Workloads (paper Sec. 5.1: DiT-MoE / DSMoE at 256x256 px, 250 steps; the
latent is 32x32 with patch 2 -> 256 tokens, or 64x64 -> 1024 tokens):

* weights   ~ N(0, 1/d), router bias optional (log of a Zipf prior for the
  skewed stress layer);
* x_0       ~ N(0, 1);
* x_t       = sqrt(1 - a_i) * x_{t-1} + sqrt(a_i) * xi_t, with a per-token
  drift rate a_i (log-uniform in [1e-3, 1e-1], or bimodal);
* attn_in_t follows the same drift model from an independent stream.

The trained checkpoints and datasets the paper measures on are not
available; these inputs stand in for them with the same shapes.

bf16 tensors are returned as numpy ``uint16`` arrays holding the bf16 bit
patterns (round-to-nearest-even from the fp32 draw); fp32 tensors as
``float32``.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

BF16 = "bf16"
FP32 = "fp32"


def fp32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round an fp32 array to bf16 (nearest, ties to even); return the bits."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # no uint32 overflow: the largest non-NaN pattern is 0xFF800000 (-inf)
    r = (u >> 16) & np.uint32(1)
    r += u
    r += np.uint32(0x7FFF)
    r >>= 16
    out = r.astype(np.uint16)
    out[np.isnan(a)] = 0x7FC0
    return out


def bf16_bits_to_fp32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to fp32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass(frozen=True)
class LayerShape:
    """Shape of one routed MoE layer and of the token batch it serves."""
    d: int          # model width
    E: int          # routed experts
    k: int          # experts per token (top-k)
    d_ff: int       # expert hidden width
    B: int          # samples in the batch
    N: int          # tokens per sample
    dtype: str = BF16
    ffn: str = "gelu"   # "gelu" or "swiglu" (gated: 2 d_ff up-projection rows)
    n_shared: int = 0   # always-on shared experts (same width as the routed ones)

    @property
    def up_rows(self) -> int:
        return 2 * self.d_ff if self.ffn == "swiglu" else self.d_ff

    @property
    def tokens(self) -> int:
        return self.B * self.N

    @property
    def branches(self) -> int:
        return self.B * self.N * self.k


# Named workloads.  "xl256" and "xl1024" are the DiT-MoE-XL-like layer at a
# 32x32 and a 64x64 latent; "tiny" is the small fp32 parity layer; "skewed"
# is the Zipf-biased stress layer; "fine" the fine-grained layer with shared
# experts.
WORKLOADS = {
    "tiny": LayerShape(d=384, E=8, k=2, d_ff=1536, B=1, N=256, dtype=FP32),
    "xl256": LayerShape(d=1152, E=16, k=2, d_ff=4608, B=8, N=256, dtype=BF16),
    "xl1024": LayerShape(d=1152, E=16, k=2, d_ff=4608, B=8, N=1024, dtype=BF16),
    "skewed": LayerShape(d=3072, E=32, k=2, d_ff=8192, B=2, N=4096, dtype=BF16),
    # fine-grained layer: 64 small SwiGLU experts, top-8, two shared experts
    "fine": LayerShape(d=2048, E=64, k=8, d_ff=1408, B=4, N=4096, dtype=BF16, ffn="swiglu",
                       n_shared=2),
}


def _store(a32: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == BF16:
        return fp32_to_bf16_bits(a32)
    if dtype == FP32:
        return np.ascontiguousarray(a32, dtype=np.float32)
    raise ValueError(dtype)


class Synth:
    """Independent seeded streams for weights, trajectory, drift and attention."""

    def __init__(self, shape: LayerShape, seed: int = 0):
        self.shape = shape
        self.seed = seed
        ss = np.random.SeedSequence(seed)
        kids = ss.spawn(6)
        self._rng_w = np.random.Generator(np.random.PCG64(kids[0]))
        self._rng_x0 = np.random.Generator(np.random.PCG64(kids[1]))
        self._rng_a = np.random.Generator(np.random.PCG64(kids[2]))
        self._rng_xi = np.random.Generator(np.random.PCG64(kids[3]))
        self._rng_attn = np.random.Generator(np.random.PCG64(kids[4]))
        self._rng_misc = np.random.Generator(np.random.PCG64(kids[5]))
        self._drift = {}

    # ---- weights -------------------------------------------------------
    def weights(self, router_bias: str | None = None, zipf_s: float = 1.2):
        """Router and expert weights, ``out x in`` row-major, ~N(0, 1/d).

        Returns ``(W_r[E][d], b_r[E] or None, W_up[E][d_ff][d],
        W_down[E][d][d_ff])``; ``b_r`` is fp32.  ``router_bias="zipf"`` gives
        ``b_e = -s * ln(e + 1)`` (the log of a Zipf(s) prior over expert rank,
        rank = expert id).
        """
        s = self.shape
        std = 1.0 / math.sqrt(s.d)
        g = self._rng_w
        W_r = g.standard_normal((s.E, s.d), dtype=np.float32) * np.float32(std)
        W_up = g.standard_normal((s.E, s.up_rows, s.d), dtype=np.float32) * np.float32(std)
        W_down = g.standard_normal((s.E, s.d, s.d_ff), dtype=np.float32) * np.float32(std)
        b_r = None
        if router_bias == "zipf":
            b_r = (-zipf_s * np.log(np.arange(s.E, dtype=np.float64) + 1.0)).astype(np.float32)
        elif router_bias is not None:
            raise ValueError(router_bias)
        return (_store(W_r, s.dtype), b_r, _store(W_up, s.dtype), _store(W_down, s.dtype))

    def shared_weights(self):
        """Shared-expert weights ``(W_up[S][up_rows][d], W_down[S][d][d_ff])``
        ~N(0, 1/d) from their own stream, or None without shared experts.
        With a gated FFN the up-projection rows alternate gate / up."""
        s = self.shape
        if s.n_shared == 0:
            return None
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([self.seed, 7919])))
        std = np.float32(1.0 / math.sqrt(s.d))
        up = g.standard_normal((s.n_shared, s.up_rows, s.d), dtype=np.float32) * std
        down = g.standard_normal((s.n_shared, s.d, s.d_ff), dtype=np.float32) * std
        return _store(up, s.dtype), _store(down, s.dtype)

    # ---- trajectory ----------------------------------------------------
    def drift_rates(self, kind: str = "loguniform") -> np.ndarray:
        """Per-token drift rate a_i, shape (B, N), float64."""
        if kind in self._drift:
            return self._drift[kind]
        s = self.shape
        g = self._rng_a
        if kind == "loguniform":
            lo, hi = math.log(1e-3), math.log(1e-1)
            a = np.exp(g.uniform(lo, hi, size=(s.B, s.N)))
        elif kind == "bimodal":
            fast = g.random(size=(s.B, s.N)) < 0.1
            a = np.where(fast, 0.2, 1e-3)
        else:
            raise ValueError(kind)
        self._drift[kind] = a
        return a

    def trajectory(self, T: int, drift: str = "loguniform"):
        """Yield ``T`` layer inputs x_t, shape (B, N, d), in the layer dtype."""
        s = self.shape
        a = self.drift_rates(drift)[..., None].astype(np.float32)
        keep = np.sqrt(1.0 - a).astype(np.float32)
        mix = np.sqrt(a).astype(np.float32)
        x = self._rng_x0.standard_normal((s.B, s.N, s.d), dtype=np.float32)
        for t in range(T):
            if t > 0:
                xi = self._rng_xi.standard_normal((s.B, s.N, s.d), dtype=np.float32)
                x = keep * x + mix * xi
            yield _store(x, s.dtype)

    def attention_trajectory(self, T: int, drift: str = "loguniform"):
        """Yield ``T`` attention-path features, shape (B, N, d), layer dtype."""
        s = self.shape
        a = self.drift_rates(drift)[..., None].astype(np.float32)
        keep = np.sqrt(1.0 - a).astype(np.float32)
        mix = np.sqrt(a).astype(np.float32)
        g = self._rng_attn
        x = g.standard_normal((s.B, s.N, s.d), dtype=np.float32)
        for t in range(T):
            if t > 0:
                x = keep * x + mix * g.standard_normal((s.B, s.N, s.d), dtype=np.float32)
            yield _store(x, s.dtype)

    # ---- arbitrary cached rows ----------------------------------------
    def rows(self, shape, scale: float = 1.0) -> np.ndarray:
        """Random rows in the layer dtype (used to fill a cache directly)."""
        a = self._rng_misc.standard_normal(shape, dtype=np.float32) * np.float32(scale)
        return _store(a, self.shape.dtype)

    def integers(self, low, high, size) -> np.ndarray:
        return self._rng_misc.integers(low, high, size=size)

    def uniform(self, low, high, size) -> np.ndarray:
        return self._rng_misc.uniform(low, high, size=size)


# ---------------------------------------------------------------------------
# a stack of DiT-MoE blocks (attention + AdaLN + the MoE layer per block)
# ---------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class StackShape:
    """Shape of a stack of DiT-MoE blocks (bf16 weights and activations)."""
    L: int          # blocks
    d: int          # model width
    heads: int      # attention heads (head width d / heads)
    E: int
    k: int
    d_ff: int
    B: int
    N: int
    n_classes: int = 1000
    freq_dim: int = 256

    def layer(self) -> LayerShape:
        return LayerShape(d=self.d, E=self.E, k=self.k, d_ff=self.d_ff, B=self.B, N=self.N,
                          dtype=BF16)


# "dit28": 28 DiT-MoE-XL-like blocks at a 64x64 latent (1024 tokens, batch 8;
# 16 heads of 72); "stack_tiny": the two-block parity stack (ragged 80 tokens).
STACKS = {
    "dit28": StackShape(L=28, d=1152, heads=16, E=16, k=2, d_ff=4608, B=8, N=1024),
    "stack_tiny": StackShape(L=2, d=576, heads=8, E=4, k=2, d_ff=256, B=2, N=80),
}


class StackSynth:
    """Seeded weights and inputs of a block stack.

    Matrices ~N(0, 1/fan_in), biases ~N(0, 0.02^2) (fp32), the class table
    ~N(0, 1); every block draws from its own stream, so a block's weights do
    not depend on L.  Inputs: x_0 ~ N(0, 1) and the per-token drift model of
    the layer workloads (``Synth``), the diffusion timestep value decreasing
    over the steps, one class label per sample.
    """

    def __init__(self, shape: StackShape, seed: int = 0):
        self.shape = shape
        self.seed = seed
        self._layer = Synth(shape.layer(), seed)

    def _rng(self, *key) -> np.random.Generator:
        return np.random.Generator(np.random.PCG64(np.random.SeedSequence([self.seed, *key])))

    @staticmethod
    def _mat(g, rows, cols) -> np.ndarray:
        return fp32_to_bf16_bits(g.standard_normal((rows, cols), dtype=np.float32)
                                 * np.float32(1.0 / math.sqrt(cols)))

    @staticmethod
    def _bias(g, n) -> np.ndarray:
        return (g.standard_normal(n, dtype=np.float32) * np.float32(0.02)).astype(np.float32)

    def block(self, l: int) -> dict:
        """Weights of block l: W_ada (6d, d), b_ada, W_qkv (3d, d), b_qkv,
        W_o (d, d), b_o, W_r (E, d), W_up (E, d_ff, d), W_down (E, d, d_ff)."""
        s = self.shape
        g = self._rng(1000 + l)
        d = s.d
        out = {
            "W_ada": self._mat(g, 6 * d, d), "b_ada": self._bias(g, 6 * d),
            "W_qkv": self._mat(g, 3 * d, d), "b_qkv": self._bias(g, 3 * d),
            "W_o": self._mat(g, d, d), "b_o": self._bias(g, d),
            "W_r": self._mat(g, s.E, d),
        }
        up = g.standard_normal((s.E, s.d_ff, d), dtype=np.float32) * np.float32(1 / math.sqrt(d))
        out["W_up"] = fp32_to_bf16_bits(up)
        del up
        down = (g.standard_normal((s.E, d, s.d_ff), dtype=np.float32)
                * np.float32(1 / math.sqrt(s.d_ff)))
        out["W_down"] = fp32_to_bf16_bits(down)
        return out

    def embedder(self) -> dict:
        """Timestep/class embedder: W1 (d, freq_dim), b1, W2 (d, d), b2 and
        the class table (n_classes, d), bf16 matrices and fp32 biases."""
        s = self.shape
        g = self._rng(7)
        return {
            "W1": self._mat(g, s.d, s.freq_dim), "b1": self._bias(g, s.d),
            "W2": self._mat(g, s.d, s.d), "b2": self._bias(g, s.d),
            "table": fp32_to_bf16_bits(g.standard_normal((s.n_classes, s.d), dtype=np.float32)),
        }

    def labels(self) -> np.ndarray:
        return self._rng(8).integers(0, self.shape.n_classes, size=self.shape.B)

    @staticmethod
    def timestep_values(T: int, n_sampling: int = 250, t_max: float = 999.0) -> np.ndarray:
        """Diffusion timestep value of the first T steps of an n_sampling-step
        sampler (evenly spaced, decreasing from t_max; the paper's DiT-MoE
        runs sample in 250 steps, Sec. 5.1), float32."""
        i = np.arange(T, dtype=np.float64)
        return (t_max * (1.0 - i / n_sampling)).astype(np.float32)

    def trajectory(self, T: int, drift: str = "loguniform"):
        """Yield ``T`` stack inputs x_t, shape (B, N, d), fp32."""
        s = self.shape
        lay = self._layer
        a = lay.drift_rates(drift)[..., None].astype(np.float32)
        keep = np.sqrt(1.0 - a).astype(np.float32)
        mix = np.sqrt(a).astype(np.float32)
        g = self._rng(9)
        x = g.standard_normal((s.B, s.N, s.d), dtype=np.float32)
        for t in range(T):
            if t > 0:
                x = keep * x + mix * g.standard_normal((s.B, s.N, s.d), dtype=np.float32)
            yield x.copy()

    # ---- device-side draws (benchmarks of the full-size stack) -----------
    def _torch_gen(self, device, *key):
        import torch
        g = torch.Generator(device=device)
        g.manual_seed(int(np.random.SeedSequence([self.seed, *key]).generate_state(1)[0]))
        return g

    def block_device(self, l: int, device) -> dict:
        """Block l's weights drawn on the GPU by torch's seeded generator:
        the distributions of ``block`` (not its values), bf16 matrices as
        int16 bit patterns, fp32 biases."""
        import torch
        s = self.shape
        g = self._torch_gen(device, 2000 + l)

        def mat(*shape):
            a = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
            a *= 1.0 / math.sqrt(shape[-1])
            return a.to(torch.bfloat16).view(torch.int16)

        def bias(n):
            return torch.randn(n, generator=g, device=device, dtype=torch.float32) * 0.02

        d = s.d
        return {"W_ada": mat(6 * d, d), "b_ada": bias(6 * d), "W_qkv": mat(3 * d, d),
                "b_qkv": bias(3 * d), "W_o": mat(d, d), "b_o": bias(d), "W_r": mat(s.E, d),
                "W_up": mat(s.E, s.d_ff, d), "W_down": mat(s.E, d, s.d_ff)}

    def embedder_device(self, device) -> dict:
        import torch
        s = self.shape
        g = self._torch_gen(device, 3000)

        def mat(*shape, scale=None):
            a = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
            a *= scale if scale is not None else 1.0 / math.sqrt(shape[-1])
            return a.to(torch.bfloat16).view(torch.int16)
        return {"W1": mat(s.d, s.freq_dim),
                "b1": torch.randn(s.d, generator=g, device=device) * 0.02,
                "W2": mat(s.d, s.d), "b2": torch.randn(s.d, generator=g, device=device) * 0.02,
                "table": mat(s.n_classes, s.d, scale=1.0)}

    def trajectory_device(self, T: int, device, drift: str = "loguniform"):
        """``T`` stack inputs (B, N, d) fp32 drawn on the GPU: x_0 ~ N(0, 1),
        then the per-token drift model of ``trajectory``."""
        import torch
        s = self.shape
        a = torch.from_numpy(self._layer.drift_rates(drift)[..., None].astype(np.float32)).to(device)
        keep, mix = torch.sqrt(1.0 - a), torch.sqrt(a)
        g = self._torch_gen(device, 4000)
        x = torch.randn(s.B, s.N, s.d, generator=g, device=device)
        out = [x.clone()]
        for _ in range(1, T):
            x = keep * x + mix * torch.randn(s.B, s.N, s.d, generator=g, device=device)
            out.append(x.clone())
        return out
