"""Python owner of one branch-cached MoE layer on a GPU.

Holds the library handle, the torch-allocated workspace and references to
the weight tensors, and forwards every call to the C ABI (``_lib``).  torch
provides device memory and the stream; all layer arithmetic runs in the
library's kernels.
"""
from __future__ import annotations

import numpy as np

from . import _lib


def _torch():
    import torch
    return torch


def np_to_device(a: np.ndarray, device):
    """Upload a numpy array; bf16 bit patterns (uint16) travel as int16."""
    torch = _torch()
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(device)


def device_to_np(t, like_dtype=None) -> np.ndarray:
    a = t.detach().cpu().numpy()
    if like_dtype is not None and a.dtype != like_dtype:
        a = a.view(like_dtype)
    return a


class MoecaLayer:
    """One layer: ``MoecaLayer(d, E, k, d_ff, batch=B, tokens=N, ...)``."""

    def __init__(self, d, E, k, d_ff, *, batch, tokens, mode=_lib.MOECA_MODE_THRESHOLD,
                 ratio=0.3, tau0=0.80, alpha=0.6, beta=0.65, lambda1=1.0, lambda2=1.0,
                 lambda0=1.0, refresh_cycle=4, norm_topk=True, act="gelu_tanh", dtype="bf16",
                 n_shared=0, device="cuda:0"):
        torch = _torch()
        p = _lib.moeca_policy_default()
        p.mode, p.ratio, p.tau0, p.alpha, p.beta = mode, ratio, tau0, alpha, beta
        p.lambda0, p.lambda1, p.lambda2 = lambda0, lambda1, lambda2
        p.refresh_cycle = refresh_cycle
        p.norm_topk = 1 if norm_topk else 0
        p.act = {"gelu_tanh": _lib.MOECA_ACT_GELU_TANH, "gelu_erf": _lib.MOECA_ACT_GELU_ERF,
                 "swiglu": _lib.MOECA_ACT_SWIGLU}[act]
        p.dtype = {"bf16": _lib.MOECA_DTYPE_BF16, "fp32": _lib.MOECA_DTYPE_FP32}[dtype]
        p.batch, p.tokens, p.n_shared = batch, tokens, n_shared
        self.d, self.E, self.k, self.d_ff, self.B, self.N = d, E, k, d_ff, batch, tokens
        self.n_shared = n_shared
        self.dtype = dtype
        self.act_np = np.uint16 if dtype == "bf16" else np.float32
        self.device = torch.device(device)
        self.h = _lib.moeca_layer_create(d, E, k, d_ff, p)
        nbytes = _lib.moeca_workspace_bytes(self.h)
        self._ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        base = self._ws.data_ptr()
        self._ws_shift = (-base) % 256
        self.workspace = self._ws[self._ws_shift:self._ws_shift + nbytes]
        _lib.moeca_bind_workspace(self.h, base + self._ws_shift, nbytes)
        self._keep = []

    @classmethod
    def attach(cls, handle, workspace, d, E, k, d_ff, *, batch, tokens, dtype="bf16",
               n_shared=0, device="cuda:0"):
        """A non-owning view of a layer created elsewhere (a block of a
        stack): ``workspace`` is the uint8 tensor slice the layer is bound to."""
        torch = _torch()
        self = cls.__new__(cls)
        self.d, self.E, self.k, self.d_ff, self.B, self.N = d, E, k, d_ff, batch, tokens
        self.n_shared, self.dtype = n_shared, dtype
        self.act_np = np.uint16 if dtype == "bf16" else np.float32
        self.device = torch.device(device)
        self.h = handle
        self.workspace = workspace
        self._owned = False
        return self

    # -- binding ---------------------------------------------------------
    def set_weights(self, W_r, b_r, W_up, W_down):
        self._keep = [W_r, b_r, W_up, W_down]
        _lib.moeca_layer_set_weights(self.h, W_r.data_ptr(),
                                     None if b_r is None else b_r.data_ptr(),
                                     W_up.data_ptr(), W_down.data_ptr())

    def set_shared(self, W_up_s, W_down_s):
        self._keep_shared = [W_up_s, W_down_s]
        _lib.moeca_layer_set_shared(self.h, W_up_s.data_ptr(), W_down_s.data_ptr())

    def bind_attention(self, attn_in, attn_cache):
        self._attn = (attn_in, attn_cache)
        _lib.moeca_bind_attention(self.h, None if attn_in is None else attn_in.data_ptr(),
                                  None if attn_cache is None else attn_cache.data_ptr())

    # -- work ------------------------------------------------------------
    def _stream(self, stream):
        torch = _torch()
        s = stream if stream is not None else torch.cuda.current_stream(self.device)
        return s.cuda_stream

    def step(self, x, t, out, stream=None):
        _lib.moeca_step(self.h, x.data_ptr(), int(t), out.data_ptr(), self._stream(stream))

    def reset(self, stream=None):
        _lib.moeca_cache_reset(self.h, self._stream(stream))

    def stats(self, stream=None):
        return _lib.moeca_get_stats(self.h, self._stream(stream))

    def set_valid(self, valid: bool):
        _lib.moeca_debug_set_valid(self.h, 1 if valid else 0)

    def set_timing(self, enable: bool):
        _lib.moeca_set_timing(self.h, 1 if enable else 0)

    def timing(self):
        ms, steps = _lib.moeca_get_timing(self.h, len(_lib.STAGES))
        return dict(zip(_lib.STAGES, ms)), steps

    # -- state inspection ------------------------------------------------
    def _spec(self, name):
        B, N, k, E, d = self.B, self.N, self.k, self.E, self.d
        nbr = (B * N * k,)
        table = {
            "e_c": (np.int32, nbr), "w_c": (np.float32, nbr), "n_c": (np.float32, nbr),
            "h_c": (self.act_np, (B * N * k, d)), "stat": (np.float32, (B, E, N)),
            "logits": (np.float32, (B * N, E)), "e_t": (np.int32, nbr), "w_t": (np.float32, nbr),
            "hbar": (np.float32, (B, E)), "tau": (np.float32, (B, E)),
            "margin": (np.float32, nbr), "q": (np.int32, nbr), "mask": (np.uint8, nbr),
            "sigma": (np.int32, nbr), "sync": (np.uint8, (B * N,)), "off": (np.int32, (E + 1,)),
            "list": (np.int32, nbr), "pos": (np.int32, nbr),
        }
        return table[name]

    def buffer(self, name):
        off, nb = _lib.moeca_debug_buffer(self.h, _lib.BUF[name])
        return self.workspace[off:off + nb]

    def read(self, name) -> np.ndarray:
        torch = _torch()
        torch.cuda.synchronize(self.device)
        dt, shape = self._spec(name)
        raw = self.buffer(name).cpu().numpy()
        return raw.view(dt).reshape(shape).copy()

    def write(self, name, arr) -> None:
        torch = _torch()
        dt, shape = self._spec(name)
        a = np.ascontiguousarray(np.asarray(arr).astype(dt, copy=False).reshape(shape))
        self.buffer(name).copy_(torch.from_numpy(a.view(np.uint8).reshape(-1)).to(self.device))
        torch.cuda.synchronize(self.device)

    def close(self):
        if getattr(self, "h", None) and getattr(self, "_owned", True):
            _lib.moeca_layer_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
