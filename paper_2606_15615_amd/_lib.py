"""ctypes binding of libmoeca.so (include/moeca.h): same names, argument
marshalling only.  Every step of the layer runs in the library's HIP
kernels; if the library is missing this module raises instead of falling
back to anything else."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoeca.so")

MOECA_OK = 0
MOECA_E_INVAL = -1
MOECA_E_STATE = -2
MOECA_E_HIP = -3

MOECA_MODE_FULL, MOECA_MODE_THRESHOLD, MOECA_MODE_RATIO = 0, 1, 2
MOECA_DTYPE_BF16, MOECA_DTYPE_FP32 = 0, 1
MOECA_ACT_GELU_TANH, MOECA_ACT_GELU_ERF, MOECA_ACT_SWIGLU = 0, 1, 2

BUF = {
    "e_c": 0, "w_c": 1, "n_c": 2, "h_c": 3, "stat": 4, "logits": 5, "e_t": 6, "w_t": 7,
    "hbar": 8, "tau": 9, "margin": 10, "q": 11, "mask": 12, "sigma": 13, "sync": 14,
    "off": 15, "list": 16, "pos": 17,
}
STAGES = ["router", "stat", "select", "lists", "ffn_up", "ffn_down", "combine"]
SBUF = {
    "mod": 0, "h": 1, "u": 2, "u2": 3, "q": 4, "kv": 5, "o": 6, "x1": 7, "y": 8, "slist": 9,
    "soff": 10, "a": 11, "layer": 12,
}


class moeca_policy(ctypes.Structure):
    _fields_ = [
        ("mode", ctypes.c_int32), ("ratio", ctypes.c_float), ("tau0", ctypes.c_float),
        ("alpha", ctypes.c_float), ("beta", ctypes.c_float), ("lambda1", ctypes.c_float),
        ("lambda2", ctypes.c_float), ("refresh_cycle", ctypes.c_int32),
        ("norm_topk", ctypes.c_int32), ("act", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("batch", ctypes.c_int32), ("tokens", ctypes.c_int32), ("n_shared", ctypes.c_int32),
        ("lambda0", ctypes.c_float),
    ]


class moeca_stats(ctypes.Structure):
    _fields_ = [
        ("n_branches", ctypes.c_int64), ("n_recompute", ctypes.c_int64),
        ("n_unmatched", ctypes.c_int64), ("n_matched", ctypes.c_int64),
        ("n_reused", ctypes.c_int64), ("n_sync", ctypes.c_int64),
        ("full_step", ctypes.c_int32), ("nonfinite", ctypes.c_int32),
        ("reuse_over_match", ctypes.c_double), ("expert_count", ctypes.c_int32 * 64),
        ("ffn_plan", ctypes.c_int32),
    ]


class moeca_block_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "W_ada", "b_ada", "W_qkv", "b_qkv", "W_o", "b_o", "W_r", "b_r", "W_up", "W_down")]


_vp = ctypes.c_void_p
_SIGS = {
    "moeca_policy_default": (None, [ctypes.POINTER(moeca_policy)]),
    "moeca_layer_create": (ctypes.c_void_p, [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                             ctypes.c_int, ctypes.POINTER(moeca_policy)]),
    "moeca_layer_destroy": (None, [ctypes.c_void_p]),
    "moeca_last_error": (ctypes.c_char_p, []),
    "moeca_layer_set_weights": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                               ctypes.c_void_p, ctypes.c_void_p]),
    "moeca_layer_set_shared": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_void_p]),
    "moeca_workspace_bytes": (ctypes.c_size_t, [ctypes.c_void_p]),
    "moeca_bind_workspace": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t]),
    "moeca_bind_attention": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "moeca_step": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                  ctypes.c_void_p, ctypes.c_void_p]),
    "moeca_forward_noalloc": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                             ctypes.c_void_p, ctypes.c_void_p]),
    "moeca_cache_reset": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p]),
    "moeca_get_stats": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(moeca_stats),
                                       ctypes.c_void_p]),
    "moeca_debug_buffer": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int,
                                          ctypes.POINTER(ctypes.c_size_t),
                                          ctypes.POINTER(ctypes.c_size_t)]),
    "moeca_debug_set_valid": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int]),
    "moeca_set_timing": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int]),
    "moeca_get_timing": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_double),
                                        ctypes.c_int, ctypes.POINTER(ctypes.c_int)]),
    "moeca_stack_create": (_vp, [ctypes.c_int] * 6 + [ctypes.POINTER(moeca_policy)]),
    "moeca_stack_destroy": (None, [_vp]),
    "moeca_stack_set_block": (ctypes.c_int, [_vp, ctypes.c_int,
                                             ctypes.POINTER(moeca_block_weights)]),
    "moeca_stack_workspace_bytes": (ctypes.c_size_t, [_vp]),
    "moeca_stack_bind_workspace": (ctypes.c_int, [_vp, _vp, ctypes.c_size_t]),
    "moeca_stack_step_blocks": (ctypes.c_int, [_vp, _vp, _vp, ctypes.c_int, ctypes.c_int,
                                               ctypes.c_int, _vp]),
    "moeca_stack_step": (ctypes.c_int, [_vp, _vp, _vp, ctypes.c_int, _vp]),
    "moeca_stack_cache_reset": (ctypes.c_int, [_vp, _vp]),
    "moeca_stack_layer": (_vp, [_vp, ctypes.c_int]),
    "moeca_stack_embed": (ctypes.c_int, [_vp] * 8 + [ctypes.c_int, _vp, _vp]),
    "moeca_stack_debug_buffer": (ctypes.c_int, [_vp, ctypes.c_int, ctypes.c_int,
                                                ctypes.POINTER(ctypes.c_size_t),
                                                ctypes.POINTER(ctypes.c_size_t)]),
}
EXPORTED = tuple(_SIGS)

_lib = None


def load() -> ctypes.CDLL:
    """Load libmoeca.so (built by ``__graft_entry__.build()``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


class MoecaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{msg} (code {code})")
        self.code = code


def _check(code: int) -> int:
    if code != MOECA_OK:
        raise MoecaError(code, load().moeca_last_error().decode())
    return code


def moeca_policy_default() -> moeca_policy:
    p = moeca_policy()
    load().moeca_policy_default(ctypes.byref(p))
    return p


def moeca_layer_create(d: int, E: int, k: int, d_ff: int, policy: moeca_policy) -> int:
    h = load().moeca_layer_create(d, E, k, d_ff, ctypes.byref(policy))
    if not h:
        raise MoecaError(MOECA_E_INVAL, load().moeca_last_error().decode())
    return h


def moeca_layer_destroy(h: int) -> None:
    load().moeca_layer_destroy(h)


def moeca_last_error() -> str:
    return load().moeca_last_error().decode()


def moeca_layer_set_weights(h, W_r, b_r, W_up, W_down) -> int:
    return _check(load().moeca_layer_set_weights(h, W_r, b_r, W_up, W_down))


def moeca_layer_set_shared(h, W_up_s, W_down_s) -> int:
    return _check(load().moeca_layer_set_shared(h, W_up_s, W_down_s))


def moeca_workspace_bytes(h) -> int:
    return load().moeca_workspace_bytes(h)


def moeca_bind_workspace(h, dev, nbytes) -> int:
    return _check(load().moeca_bind_workspace(h, dev, nbytes))


def moeca_bind_attention(h, attn_in, attn_cache) -> int:
    return _check(load().moeca_bind_attention(h, attn_in, attn_cache))


def moeca_step(h, x_t, t, out, stream) -> int:
    return _check(load().moeca_step(h, x_t, t, out, stream))


def moeca_forward_noalloc(h, x, samples, out, stream) -> int:
    return _check(load().moeca_forward_noalloc(h, x, samples, out, stream))


def moeca_cache_reset(h, stream) -> int:
    return _check(load().moeca_cache_reset(h, stream))


def moeca_get_stats(h, stream) -> moeca_stats:
    s = moeca_stats()
    _check(load().moeca_get_stats(h, ctypes.byref(s), stream))
    return s


def moeca_debug_buffer(h, which: int) -> tuple[int, int]:
    off, nb = ctypes.c_size_t(), ctypes.c_size_t()
    _check(load().moeca_debug_buffer(h, which, ctypes.byref(off), ctypes.byref(nb)))
    return off.value, nb.value


def moeca_debug_set_valid(h, valid: int) -> int:
    return _check(load().moeca_debug_set_valid(h, valid))


def moeca_set_timing(h, enable: int) -> int:
    return _check(load().moeca_set_timing(h, enable))


def moeca_get_timing(h, n: int = 7) -> tuple[list[float], int]:
    arr = (ctypes.c_double * n)()
    steps = ctypes.c_int()
    _check(load().moeca_get_timing(h, arr, n, ctypes.byref(steps)))
    return list(arr), steps.value


# ---- block stack -----------------------------------------------------------
def moeca_stack_create(n_blocks: int, d: int, heads: int, E: int, k: int, d_ff: int,
                       policy: moeca_policy) -> int:
    h = load().moeca_stack_create(n_blocks, d, heads, E, k, d_ff, ctypes.byref(policy))
    if not h:
        raise MoecaError(MOECA_E_INVAL, load().moeca_last_error().decode())
    return h


def moeca_stack_destroy(h) -> None:
    load().moeca_stack_destroy(h)


def moeca_stack_set_block(h, l: int, w: moeca_block_weights) -> int:
    return _check(load().moeca_stack_set_block(h, l, ctypes.byref(w)))


def moeca_stack_workspace_bytes(h) -> int:
    return load().moeca_stack_workspace_bytes(h)


def moeca_stack_bind_workspace(h, dev, nbytes) -> int:
    return _check(load().moeca_stack_bind_workspace(h, dev, nbytes))


def moeca_stack_step_blocks(h, x, c, t, first, count, stream) -> int:
    return _check(load().moeca_stack_step_blocks(h, x, c, t, first, count, stream))


def moeca_stack_step(h, x, c, t, stream) -> int:
    return _check(load().moeca_stack_step(h, x, c, t, stream))


def moeca_stack_cache_reset(h, stream) -> int:
    return _check(load().moeca_stack_cache_reset(h, stream))


def moeca_stack_layer(h, l: int) -> int:
    p = load().moeca_stack_layer(h, l)
    if not p:
        raise MoecaError(MOECA_E_INVAL, load().moeca_last_error().decode())
    return p


def moeca_stack_embed(h, t_values, labels, W1, b1, W2, b2, table, n_classes, c, stream) -> int:
    return _check(load().moeca_stack_embed(h, t_values, labels, W1, b1, W2, b2, table,
                                           n_classes, c, stream))


def moeca_stack_debug_buffer(h, which: int, l: int = 0) -> tuple[int, int]:
    off, nb = ctypes.c_size_t(), ctypes.c_size_t()
    _check(load().moeca_stack_debug_buffer(h, which, l, ctypes.byref(off), ctypes.byref(nb)))
    return off.value, nb.value
