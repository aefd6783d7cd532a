"""C-ABI contract, host side only: the library loads, exports every symbol
include/moeca.h declares, validates arguments and reports every error path
from the host, without launching GPU work."""
import ctypes
import json
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moeca.h")


@pytest.fixture(scope="module")
def L():
    from paper_2606_15615_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2606_15615_amd.build import build_library
        build_library()
    return _lib


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moeca_[a-z_]+)\s*\(", src)))


def test_header_declarations_are_exported(L):
    lib = L.load()
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(L.EXPORTED) == names


def test_policy_default_is_the_papers(L):
    with open(os.path.join(ROOT, "tests", "golden", "paper_hyperparams.json")) as f:
        hp = json.load(f)
    p = L.moeca_policy_default()
    assert p.mode == L.MOECA_MODE_THRESHOLD
    assert p.tau0 == pytest.approx(hp["tau0"]["value"])
    assert p.alpha == pytest.approx(hp["alpha"]["value"])
    assert p.beta == pytest.approx(hp["beta"]["value"])
    assert p.refresh_cycle == hp["refresh_cycle"]["value"]
    assert p.norm_topk == 1 and p.dtype == L.MOECA_DTYPE_BF16
    assert p.lambda0 == 1.0 and p.lambda1 == 1.0 and p.lambda2 == 1.0


def _pol(L, **kw):
    p = L.moeca_policy_default()
    p.batch, p.tokens = 2, 16
    for k, v in kw.items():
        setattr(p, k, v)
    return p


BAD_DIMS = [
    (0, 8, 2, 128), (100, 8, 2, 128), (64, 8, 2, 100), (64, 0, 1, 128), (64, 65, 2, 128),
    (64, 8, 0, 128), (64, 4, 5, 128), (64, 16, 9, 128), (32768, 8, 2, 128),
]


@pytest.mark.parametrize("dims", BAD_DIMS)
def test_create_rejects_bad_dims(L, dims):
    lib = L.load()
    h = lib.moeca_layer_create(*dims, ctypes.byref(_pol(L)))
    assert not h
    assert lib.moeca_last_error().decode() != ""


BAD_POLICY = [
    dict(mode=7), dict(dtype=3), dict(act=9), dict(ratio=-0.1), dict(ratio=1.5),
    dict(ratio=math.nan), dict(alpha=1.0), dict(alpha=-0.2), dict(beta=1.0), dict(beta=-0.1),
    dict(tau0=0.0), dict(tau0=math.inf), dict(lambda1=-1.0), dict(lambda2=math.nan),
    dict(lambda0=-0.5), dict(lambda0=math.inf),
    dict(refresh_cycle=-1), dict(norm_topk=2), dict(batch=0), dict(tokens=0),
    dict(batch=1 << 20, tokens=1 << 12), dict(n_shared=-1), dict(n_shared=9),
    dict(batch=1 << 14, tokens=1 << 14, n_shared=6),
]


def test_create_limits_tokens_times_k(L):
    """Above 32768 branches per sample the decision path needs k | 1024."""
    lib = L.load()
    assert not lib.moeca_layer_create(64, 8, 3, 128, ctypes.byref(_pol(L, tokens=11000)))
    assert "k in" in lib.moeca_last_error().decode()
    h = lib.moeca_layer_create(64, 8, 4, 128, ctypes.byref(_pol(L, tokens=11000)))
    assert h
    lib.moeca_layer_destroy(h)


@pytest.mark.parametrize("kw", BAD_POLICY)
def test_create_rejects_bad_policy(L, kw):
    lib = L.load()
    assert not lib.moeca_layer_create(64, 8, 2, 128, ctypes.byref(_pol(L, **kw)))
    assert lib.moeca_last_error().decode() != ""


def test_create_null_policy(L):
    lib = L.load()
    assert not lib.moeca_layer_create(64, 8, 2, 128, None)


def test_host_error_paths(L):
    lib = L.load()
    h = L.moeca_layer_create(128, 8, 2, 256, _pol(L, batch=3, tokens=50))
    try:
        nbytes = L.moeca_workspace_bytes(h)
        assert nbytes > 3 * 50 * 2 * (128 + 256) * 2
        fake = 1 << 40  # never dereferenced: every call below fails on the host
        assert lib.moeca_step(h, fake, 0, fake, None) == L.MOECA_E_STATE   # nothing bound
        assert lib.moeca_layer_set_weights(h, None, None, fake, fake) == L.MOECA_E_INVAL
        assert L.moeca_layer_set_weights(h, fake, None, fake, fake) == L.MOECA_OK
        assert lib.moeca_step(h, fake, 0, fake, None) == L.MOECA_E_STATE   # no workspace
        assert lib.moeca_cache_reset(h, None) == L.MOECA_E_STATE
        assert lib.moeca_bind_workspace(h, None, nbytes) == L.MOECA_E_INVAL
        assert lib.moeca_bind_workspace(h, fake + 8, nbytes) == L.MOECA_E_INVAL  # misaligned
        assert lib.moeca_bind_workspace(h, fake, nbytes - 1) == L.MOECA_E_INVAL  # too small
        assert "too small" in L.moeca_last_error()
        assert lib.moeca_bind_attention(h, fake, None) == L.MOECA_E_INVAL
        assert lib.moeca_bind_attention(h, None, None) == L.MOECA_OK
        assert L.moeca_bind_workspace(h, fake, nbytes) == L.MOECA_OK
        assert lib.moeca_step(h, None, 0, fake, None) == L.MOECA_E_INVAL
        assert lib.moeca_step(h, fake, -1, fake, None) == L.MOECA_E_INVAL
        assert lib.moeca_step(h, fake + 4, 0, fake, None) == L.MOECA_E_INVAL  # misaligned
        assert lib.moeca_layer_set_weights(h, fake + 2, None, fake, fake) == L.MOECA_E_INVAL
        assert lib.moeca_bind_attention(h, fake, fake + 8) == L.MOECA_E_INVAL
        with pytest.raises(L.MoecaError):
            L.moeca_debug_buffer(h, 99)
        # debug buffers: inside the workspace, 256-byte aligned, disjoint
        spans = sorted(L.moeca_debug_buffer(h, i) for i in range(len(L.BUF)))
        for (o1, b1), (o2, _) in zip(spans, spans[1:]):
            assert o1 % 256 == 0 and o1 + b1 <= o2
        assert spans[-1][0] + spans[-1][1] <= nbytes
        assert L.moeca_debug_buffer(h, L.BUF["h_c"])[1] == 3 * 50 * 2 * 128 * 2
        assert lib.moeca_get_stats(h, None, None) == L.MOECA_E_INVAL
        assert lib.moeca_get_timing(h, None, 8, None) == L.MOECA_E_INVAL
        assert L.moeca_set_timing(h, 0) == L.MOECA_OK
    finally:
        L.moeca_layer_destroy(h)
    lib.moeca_layer_destroy(None)  # no-op
    assert lib.moeca_workspace_bytes(None) == 0
    assert lib.moeca_debug_set_valid(None, 1) == L.MOECA_E_INVAL


def test_noalloc_forward_host_error_paths(L):
    """moeca_forward_noalloc refuses, on the host and before any device call:
    a NULL layer or buffer, misaligned buffers, sample counts outside
    [1, B], work whose intermediates exceed the library's 64 MiB array, and
    unbound weights."""
    lib = L.load()
    fake = 1 << 40  # never dereferenced
    assert lib.moeca_forward_noalloc(None, fake, 1, fake, None) == L.MOECA_E_INVAL
    big = L.moeca_layer_create(1152, 16, 2, 4608, _pol(L, batch=8, tokens=1024))
    try:
        assert lib.moeca_forward_noalloc(big, None, 1, fake, None) == L.MOECA_E_INVAL
        assert lib.moeca_forward_noalloc(big, fake, 1, fake + 8, None) == L.MOECA_E_INVAL
        assert lib.moeca_forward_noalloc(big, fake, 0, fake, None) == L.MOECA_E_INVAL
        assert lib.moeca_forward_noalloc(big, fake, 9, fake, None) == L.MOECA_E_INVAL
        assert "samples must be in [1, 8]" in L.moeca_last_error()
        # 8 and 3 samples of 1024 tokens exceed the array, 2 fit (then the
        # unbound weights are the next refusal)
        for n in (8, 3):
            assert lib.moeca_forward_noalloc(big, fake, n, fake, None) == L.MOECA_E_INVAL
            assert "bytes of scratch" in L.moeca_last_error()
        assert lib.moeca_forward_noalloc(big, fake, 2, fake, None) == L.MOECA_E_STATE
        assert "weights are not bound" in L.moeca_last_error()
    finally:
        L.moeca_layer_destroy(big)


def test_workspace_grows_with_the_layer(L):
    a = L.moeca_layer_create(1152, 16, 2, 4608, _pol(L, batch=8, tokens=256))
    b = L.moeca_layer_create(1152, 16, 2, 4608, _pol(L, batch=8, tokens=1024))
    c = L.moeca_layer_create(1152, 16, 2, 4608, _pol(L, batch=8, tokens=1024, dtype=1))
    try:
        wa, wb, wc = (L.moeca_workspace_bytes(h) for h in (a, b, c))
        # the 256-token layer (256 rows per expert on a full step) may stream
        # the weights with the thin plan: its workspace also holds the fp32
        # partial sums of the down projection's four K pieces
        part = 4 * (8 * 256 * 2) * 1152 * 4
        assert wa > part
        assert wb > 3.9 * (wa - part) and wc > 1.9 * wb
        # cache rows + FFN activation rows dominate: 16384 * (1152 + 4608) * 2 bytes
        assert wb >= 16384 * (1152 + 4608) * 2
    finally:
        for h in (a, b, c):
            L.moeca_layer_destroy(h)


def test_shared_experts_and_gated_ffn_host_paths(L):
    """Shared experts (Sec. 2.3, shared-expert MoE eq.) and the gated FFN:
    argument checks and workspace size, host only."""
    lib = L.load()
    fake = 1 << 40  # never dereferenced
    # the gated form doubles the up-projection rows: d_ff up to 32768
    assert not lib.moeca_layer_create(64, 8, 2, 32768 + 64,
                                      ctypes.byref(_pol(L, act=L.MOECA_ACT_SWIGLU)))
    h0 = L.moeca_layer_create(64, 8, 2, 32768 + 64, _pol(L))
    L.moeca_layer_destroy(h0)
    plain = L.moeca_layer_create(128, 8, 2, 192, _pol(L, batch=2, tokens=40))
    h = L.moeca_layer_create(128, 8, 2, 192, _pol(L, batch=2, tokens=40, n_shared=3,
                                                  act=L.MOECA_ACT_SWIGLU))
    try:
        # a layer without shared experts rejects shared weights
        assert lib.moeca_layer_set_shared(plain, fake, fake) == L.MOECA_E_INVAL
        assert "no shared experts" in L.moeca_last_error()
        # shared outputs [S][T][d] and S*T more intermediate rows [d_ff]
        extra = L.moeca_workspace_bytes(h) - L.moeca_workspace_bytes(plain)
        T = 2 * 40
        assert extra >= 3 * T * (128 + 192) * 2
        nbytes = L.moeca_workspace_bytes(h)
        assert L.moeca_layer_set_weights(h, fake, None, fake, fake) == L.MOECA_OK
        assert L.moeca_bind_workspace(h, fake, nbytes) == L.MOECA_OK
        assert lib.moeca_step(h, fake, 0, fake, None) == L.MOECA_E_STATE
        assert "shared" in L.moeca_last_error()
        assert lib.moeca_layer_set_shared(h, None, fake) == L.MOECA_E_INVAL
        assert lib.moeca_layer_set_shared(h, fake, fake + 8) == L.MOECA_E_INVAL
        assert L.moeca_layer_set_shared(h, fake, fake) == L.MOECA_OK
        # the public offsets view stays [E+1]
        assert L.moeca_debug_buffer(h, L.BUF["off"])[1] == (8 + 1) * 4
    finally:
        L.moeca_layer_destroy(h)
        L.moeca_layer_destroy(plain)


# ---- block stack ------------------------------------------------------------
@pytest.mark.parametrize("args,kw", [
    ((2, 1152, 16, 16, 2, 4608), {"dtype": 1}),          # fp32: the stack is bf16 only
    ((2, 1152, 16, 16, 2, 4608), {"n_shared": 1}),
    ((2, 4096, 32, 16, 2, 4608), {}),                    # d above 2048
    ((2, 1152, 7, 16, 2, 4608), {}),                     # heads do not divide d
    ((2, 1152, 12, 16, 2, 4608), {}),                    # head width 96 ok, see below
    ((2, 576, 6, 16, 2, 4608), {}),                      # head width 96
    ((2, 640, 5, 16, 2, 4608), {}),                      # head width 128
    ((2, 1152, 144, 16, 2, 4608), {}),                   # head width 8
    ((2, 1152, 96, 16, 2, 4608), {}),                    # head width 12
    ((0, 1152, 16, 16, 2, 4608), {}),
    ((2, 1152, 16, 16, 9, 4608), {}),                    # the layer's own limit on k
])
def test_stack_create_limits(L, args, kw):
    ok = {(2, 1152, 12), (2, 576, 6), (2, 1152, 144)}
    pol = _pol(L, batch=2, tokens=64)
    for f, v in kw.items():
        setattr(pol, f, v)
    h = L.load().moeca_stack_create(*args, ctypes.byref(pol))
    expect = not kw and args[:3] in ok
    assert bool(h) == expect, (args, kw, L.moeca_last_error())
    if h:
        assert L.moeca_stack_workspace_bytes(h) > 0
        L.moeca_stack_destroy(h)
    else:
        assert L.moeca_last_error() != ""


def test_stack_host_error_paths(L):
    lib = L.load()
    B, N, d, E, k, dff = 2, 80, 576, 4, 2, 256
    h = L.moeca_stack_create(3, d, 8, E, k, dff, _pol(L, batch=B, tokens=N))
    try:
        nbytes = L.moeca_stack_workspace_bytes(h)
        lay = L.moeca_layer_create(d, E, k, dff, _pol(L, batch=B, tokens=N))
        per_layer = L.moeca_workspace_bytes(lay)
        L.moeca_layer_destroy(lay)
        # three layers and attention caches, one FFN intermediate shared by the
        # blocks (they step one after another), the shared activations (x1 in two
        # buffers that alternate from block to block)
        mid = B * N * k * dff * 2
        assert nbytes >= 3 * (per_layer - mid + B * N * d * 2) + mid + B * N * d * (6 * 2 + 2 * 2 + 2 * 4)
        assert nbytes < 3 * (per_layer + B * N * d * 2) + B * N * d * (6 * 2 + 2 * 2 + 2 * 4)
        fake = 1 << 40  # never dereferenced
        W = L.moeca_block_weights(*([fake] * 10))
        assert lib.moeca_stack_step(h, fake, fake, 0, None) == L.MOECA_E_STATE  # no workspace
        assert lib.moeca_stack_cache_reset(h, None) == L.MOECA_E_STATE
        assert lib.moeca_stack_set_block(h, 3, ctypes.byref(W)) == L.MOECA_E_INVAL
        W.b_o = None
        assert lib.moeca_stack_set_block(h, 0, ctypes.byref(W)) == L.MOECA_E_INVAL
        W.b_o = fake + 2
        assert lib.moeca_stack_set_block(h, 0, ctypes.byref(W)) == L.MOECA_E_INVAL
        W.b_o, W.W_qkv = fake, fake + 8
        assert lib.moeca_stack_set_block(h, 0, ctypes.byref(W)) == L.MOECA_E_INVAL
        W.W_qkv, W.b_r = fake, None          # the router bias is optional
        assert L.moeca_stack_set_block(h, 0, W) == L.MOECA_OK
        assert lib.moeca_stack_bind_workspace(h, fake, nbytes - 1) == L.MOECA_E_INVAL
        assert lib.moeca_stack_bind_workspace(h, fake + 16, nbytes) == L.MOECA_E_INVAL
        assert L.moeca_stack_bind_workspace(h, fake, nbytes) == L.MOECA_OK
        # block 1 has no weights: a run over it is refused, block 0 alone is not checked here
        assert lib.moeca_stack_step(h, fake, fake, 0, None) == L.MOECA_E_STATE
        assert "block 1" in L.moeca_last_error()
        for first, count in ((-1, 1), (0, 0), (2, 2), (3, 1)):
            assert lib.moeca_stack_step_blocks(h, fake, fake, 0, first, count, None) == \
                L.MOECA_E_INVAL
        assert lib.moeca_stack_step_blocks(h, fake, fake, -1, 0, 1, None) == L.MOECA_E_INVAL
        assert lib.moeca_stack_step_blocks(h, fake + 4, fake, 0, 0, 1, None) == L.MOECA_E_INVAL
        assert lib.moeca_stack_step_blocks(h, None, fake, 0, 0, 1, None) == L.MOECA_E_INVAL
        assert lib.moeca_stack_embed(h, fake, fake, fake, fake, fake, fake, None, 0, fake,
                                     None) == L.MOECA_E_INVAL          # labels without a table
        assert lib.moeca_stack_embed(h, fake, None, fake + 8, fake, fake, fake, None, 0, fake,
                                     None) == L.MOECA_E_INVAL          # misaligned W1
        assert not lib.moeca_stack_layer(h, 3)
        assert lib.moeca_stack_layer(h, 2)
        # buffers: inside the workspace, aligned, disjoint, the right sizes
        spans = [L.moeca_stack_debug_buffer(h, i) for i in range(L.SBUF["a"])]
        spans += [L.moeca_stack_debug_buffer(h, L.SBUF[n], l) for n in ("a", "layer")
                  for l in range(3)]
        spans.sort()
        for (o1, b1), (o2, _) in zip(spans, spans[1:]):
            assert o1 % 256 == 0 and o1 + b1 <= o2
        assert spans[-1][0] + spans[-1][1] <= nbytes
        assert L.moeca_stack_debug_buffer(h, L.SBUF["kv"])[1] == B * N * 2 * d * 2
        assert L.moeca_stack_debug_buffer(h, L.SBUF["layer"], 1)[1] == per_layer - mid
        with pytest.raises(L.MoecaError):
            L.moeca_stack_debug_buffer(h, L.SBUF["a"], 3)
        with pytest.raises(L.MoecaError):
            L.moeca_stack_debug_buffer(h, 13)
    finally:
        L.moeca_stack_destroy(h)
    lib.moeca_stack_destroy(None)
    assert lib.moeca_stack_workspace_bytes(None) == 0
