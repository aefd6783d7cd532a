"""Python owner of a stack of branch-cached DiT-MoE blocks on a GPU.

Holds the library handle, the torch-allocated workspace and references to
the weight tensors, and forwards every call to the C ABI (``_lib``).  All
block arithmetic runs in the library's kernels.
"""
from __future__ import annotations

import numpy as np

from . import _lib
from .layer import MoecaLayer, _torch


class MoecaStack:
    """``MoecaStack(L, d, heads, E, k, d_ff, batch=B, tokens=N, ...)``: bf16."""

    def __init__(self, n_blocks, d, heads, E, k, d_ff, *, batch, tokens,
                 mode=_lib.MOECA_MODE_THRESHOLD, ratio=0.3, tau0=0.80, alpha=0.6, beta=0.65,
                 lambda1=1.0, lambda2=1.0, lambda0=1.0, refresh_cycle=4, act="gelu_tanh",
                 device="cuda:0"):
        torch = _torch()
        p = _lib.moeca_policy_default()
        p.mode, p.ratio, p.tau0, p.alpha, p.beta = mode, ratio, tau0, alpha, beta
        p.lambda0, p.lambda1, p.lambda2 = lambda0, lambda1, lambda2
        p.refresh_cycle = refresh_cycle
        p.act = {"gelu_tanh": _lib.MOECA_ACT_GELU_TANH, "gelu_erf": _lib.MOECA_ACT_GELU_ERF,
                 "swiglu": _lib.MOECA_ACT_SWIGLU}[act]
        p.dtype = _lib.MOECA_DTYPE_BF16
        p.batch, p.tokens = batch, tokens
        self.L, self.d, self.heads = n_blocks, d, heads
        self.E, self.k, self.d_ff, self.B, self.N = E, k, d_ff, batch, tokens
        self.device = torch.device(device)
        self.h = _lib.moeca_stack_create(n_blocks, d, heads, E, k, d_ff, p)
        nbytes = _lib.moeca_stack_workspace_bytes(self.h)
        self._ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        base = self._ws.data_ptr()
        shift = (-base) % 256
        self.workspace = self._ws[shift:shift + nbytes]
        _lib.moeca_stack_bind_workspace(self.h, base + shift, nbytes)
        self._keep = {}

    # -- binding ---------------------------------------------------------
    def set_block(self, l, W_ada, b_ada, W_qkv, b_qkv, W_o, b_o, W_r, b_r, W_up, W_down):
        ts = (W_ada, b_ada, W_qkv, b_qkv, W_o, b_o, W_r, b_r, W_up, W_down)
        self._keep[l] = ts
        w = _lib.moeca_block_weights(*[None if t is None else t.data_ptr() for t in ts])
        _lib.moeca_stack_set_block(self.h, l, w)

    # -- work ------------------------------------------------------------
    def _stream(self, stream):
        torch = _torch()
        s = stream if stream is not None else torch.cuda.current_stream(self.device)
        return s.cuda_stream

    def step(self, x, c, t, stream=None):
        """x (B, N, d) fp32 in/out, c (B, d) fp32."""
        _lib.moeca_stack_step(self.h, x.data_ptr(), c.data_ptr(), int(t), self._stream(stream))

    def step_blocks(self, x, c, t, first, count, stream=None):
        _lib.moeca_stack_step_blocks(self.h, x.data_ptr(), c.data_ptr(), int(t), first, count,
                                     self._stream(stream))

    def embed(self, t_values, labels, W1, b1, W2, b2, table, c, stream=None):
        n_classes = 0 if table is None else table.shape[0]
        _lib.moeca_stack_embed(self.h, t_values.data_ptr(),
                               None if labels is None else labels.data_ptr(), W1.data_ptr(),
                               b1.data_ptr(), W2.data_ptr(), b2.data_ptr(),
                               None if table is None else table.data_ptr(), n_classes,
                               c.data_ptr(), self._stream(stream))

    def reset(self, stream=None):
        _lib.moeca_stack_cache_reset(self.h, self._stream(stream))

    # -- inspection ------------------------------------------------------
    def _spec(self, name):
        T, d, B = self.B * self.N, self.d, self.B
        return {
            "mod": (np.float32, (self.L, B, 6, d)), "h": (np.uint16, (T, d)),
            "u": (np.uint16, (T, d)), "u2": (np.uint16, (T, d)), "q": (np.uint16, (T, d)),
            "kv": (np.uint16, (T, 2 * d)), "o": (np.uint16, (T, d)), "x1": (np.float32, (T, d)),
            "y": (np.uint16, (T, d)), "slist": (np.int32, (T,)), "soff": (np.int32, (B + 1,)),
            "a": (np.uint16, (T, d)),
        }[name]

    def buffer(self, name, l=0):
        off, nb = _lib.moeca_stack_debug_buffer(self.h, _lib.SBUF[name], l)
        return self.workspace[off:off + nb]

    def read(self, name, l=0) -> np.ndarray:
        torch = _torch()
        torch.cuda.synchronize(self.device)
        dt, shape = self._spec(name)
        raw = self.buffer(name, l).cpu().numpy()
        return raw.view(dt)[:int(np.prod(shape))].reshape(shape).copy()

    def write(self, name, arr, l=0) -> None:
        torch = _torch()
        dt, shape = self._spec(name)
        a = np.ascontiguousarray(np.asarray(arr).astype(dt, copy=False).reshape(shape))
        self.buffer(name, l)[:a.nbytes].copy_(
            torch.from_numpy(a.view(np.uint8).reshape(-1)).to(self.device))
        torch.cuda.synchronize(self.device)

    def layer(self, l) -> MoecaLayer:
        """A view of block l's MoE layer (statistics and state inspection)."""
        return MoecaLayer.attach(_lib.moeca_stack_layer(self.h, l), self.buffer("layer", l),
                                 self.d, self.E, self.k, self.d_ff, batch=self.B,
                                 tokens=self.N, device=str(self.device))

    def close(self):
        if getattr(self, "h", None):
            _lib.moeca_stack_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
