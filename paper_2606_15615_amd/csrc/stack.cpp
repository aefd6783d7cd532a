// C ABI and host orchestration of a stack of DiT-MoE blocks (Sec. 2.1 block
// form) whose MoE sublayers are branch-cached layers (Sec. 4).
//
// Per block, a full step runs LN1 -> q/k/v projections -> attention -> the
// output projection (the new attention feature a) -> LN2 -> the MoE layer.
// A cache step runs LN1 (which also builds the routing input from the cached
// a) and the k/v projection of every token, then the MoE layer with the
// attention refresh of the synchronised tokens enqueued between its
// decision and its expert FFN (Sec. 4.1, synchronised update): the token
// list from the layer's sync flags, their q projection, attention, output
// projection (into the cached a) and LN2 of those tokens (the FFN input).
// The gated residual x' = x1 + g_m y is folded into the next block's LN1 and,
// after the last block of a run, applied by a final pass.  The k/v
// projection runs on a second stream that the stack makes on its first step
// outside a graph capture, forked after LN1 (and, on a full step, the token
// list) and joined before the attention.  Nothing here waits for the device or allocates device
// memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <new>
#include <string>
#include <vector>

#include "internal.h"
#include "moeca.h"

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

int fail(int code, const std::string& m) { return moeca::set_error(code, m); }

// Shared regions, in MOECA_SBUF_* order for the public ones.
enum Region {
  S_MOD, S_H, S_U, S_U2, S_Q, S_KV, S_O, S_X1, S_Y, S_SLIST, S_SOFF,
  S_IDENT, S_TAB, S_SC, S_EMB, S_H1, S_MID, S_X1B, S_COUNT
};

}  // namespace

struct moeca_stack {
  int L = 0, d = 0, heads = 0, B = 0, N = 0;
  std::vector<moeca_layer*> layers;
  std::vector<moeca_block_weights> w;
  std::vector<char> bound;
  size_t off[S_COUNT] = {};
  size_t bytes[S_COUNT] = {};
  std::vector<size_t> a_off;      // per block: cached attention feature
  std::vector<size_t> layer_off;  // per block: the MoE layer's workspace
  size_t total = 0;
  char* ws = nullptr;
  moeca::BlockBufs k{};
  // a second stream for the k/v projection of cache steps, made on the
  // first step that is not being captured, on that step's device
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_kv = nullptr;
  int side_dev = -1;
};

namespace {

void release_side(moeca_stack* S) {
  if (S->ev_kv) (void)hipEventDestroy(S->ev_kv);
  if (S->ev_fork) (void)hipEventDestroy(S->ev_fork);
  if (S->side) (void)hipStreamDestroy(S->side);
  S->side = nullptr;
  S->ev_fork = S->ev_kv = nullptr;
  S->side_dev = -1;
}

// True when the k/v projection of a cache step may run on the side stream:
// the side stream exists (or can be made now, outside a capture) on the
// current device.  Any failure leaves the single-stream order.
bool side_ready(moeca_stack* S, hipStream_t st) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  if (S->side != nullptr) return S->side_dev == dev;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(st, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) {
    (void)hipGetLastError();
    return false;
  }
  if (hipStreamCreateWithFlags(&S->side, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&S->ev_fork, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&S->ev_kv, hipEventDisableTiming) != hipSuccess) {
    (void)hipGetLastError();
    release_side(S);
    return false;
  }
  S->side_dev = dev;
  return true;
}

}  // namespace

extern "C" {

moeca_stack* moeca_stack_create(int n_blocks, int d, int heads, int E, int k, int d_ff,
                                const moeca_policy* p) {
  auto bad = [](const std::string& m) -> moeca_stack* {
    fail(MOECA_E_INVAL, m);
    return nullptr;
  };
  if (p == nullptr) return bad("policy is NULL");
  if (n_blocks < 1 || n_blocks > 4096) return bad("n_blocks must be in [1, 4096]");
  if (p->dtype != MOECA_DTYPE_BF16) return bad("the block stack is bf16 only");
  if (p->n_shared != 0) return bad("the block stack takes no shared experts");
  if (d <= 0 || d % 64 != 0 || d > moeca::kMaxWidth)
    return bad("d must be a positive multiple of 64, <= " + std::to_string(moeca::kMaxWidth));
  if (heads < 1 || d % heads != 0) return bad("heads must divide d");
  const int dh = d / heads;
  if (dh % 8 != 0 || dh > 96) return bad("the head width d / heads must be a multiple of 8, <= 96");
  auto* S = new (std::nothrow) moeca_stack();
  if (S == nullptr) return bad("out of host memory");
  S->L = n_blocks;
  S->d = d;
  S->heads = heads;
  S->B = p->batch;
  S->N = p->tokens;
  for (int l = 0; l < n_blocks; ++l) {
    moeca_layer* lay = moeca_layer_create(d, E, k, d_ff, p);
    if (lay == nullptr) {
      const std::string why = moeca_last_error();
      moeca_stack_destroy(S);
      return bad(why);
    }
    // the blocks step one after another: one FFN intermediate serves all
    moeca::layer_keep_mid_outside(lay);
    S->layers.push_back(lay);
  }
  S->w.assign(n_blocks, moeca_block_weights{});
  S->bound.assign(n_blocks, 0);

  const size_t T = size_t(S->B) * S->N;
  size_t b[S_COUNT];
  b[S_MOD] = size_t(n_blocks) * S->B * 6 * d * 4;
  b[S_H] = T * d * 2;
  b[S_U] = T * d * 2;
  b[S_U2] = T * d * 2;
  b[S_Q] = T * d * 2;
  b[S_KV] = T * 2 * d * 2;
  b[S_O] = T * d * 2;
  b[S_X1] = T * d * 4;
  b[S_X1B] = T * d * 4;  // x1 of every other block of a run
  b[S_Y] = T * d * 2;
  b[S_SLIST] = T * 4;
  b[S_SOFF] = size_t(S->B + 1) * 4;
  b[S_IDENT] = T * 4;
  b[S_TAB] = 8 * 4;
  b[S_SC] = size_t(S->B) * d * 8;
  b[S_EMB] = size_t(S->B) * moeca::kFreqDim * 8;
  b[S_H1] = size_t(S->B) * d * 8;
  b[S_MID] = moeca::layer_mid_bytes(S->layers[0]);
  size_t cur = 0;
  for (int i = 0; i < S_COUNT; ++i) {
    S->off[i] = cur;
    S->bytes[i] = b[i];
    cur = align_up(cur + b[i]);
  }
  for (int l = 0; l < n_blocks; ++l) {
    S->a_off.push_back(cur);
    cur = align_up(cur + T * d * 2);
    S->layer_off.push_back(cur);
    cur = align_up(cur + moeca_workspace_bytes(S->layers[l]));
  }
  S->total = cur;
  return S;
}

void moeca_stack_destroy(moeca_stack* S) {
  if (S == nullptr) return;
  for (moeca_layer* l : S->layers) moeca_layer_destroy(l);
  release_side(S);
  delete S;
}

int moeca_stack_set_block(moeca_stack* S, int l, const moeca_block_weights* w) {
  if (S == nullptr || w == nullptr) return fail(MOECA_E_INVAL, "stack and weights are required");
  if (l < 0 || l >= S->L) return fail(MOECA_E_INVAL, "block index out of range");
  if (w->W_ada == nullptr || w->b_ada == nullptr || w->W_qkv == nullptr || w->b_qkv == nullptr ||
      w->W_o == nullptr || w->b_o == nullptr)
    return fail(MOECA_E_INVAL, "W_ada, b_ada, W_qkv, b_qkv, W_o and b_o are required");
  if (!aligned16(w->W_ada) || !aligned16(w->W_qkv) || !aligned16(w->W_o) ||
      !aligned4(w->b_ada) || !aligned4(w->b_qkv) || !aligned4(w->b_o))
    return fail(MOECA_E_INVAL, "matrices must be 16-byte aligned, biases 4-byte");
  const int rc = moeca_layer_set_weights(S->layers[l], w->W_r, w->b_r, w->W_up, w->W_down);
  if (rc != MOECA_OK) return rc;
  S->w[l] = *w;
  S->bound[l] = 1;
  return MOECA_OK;
}

size_t moeca_stack_workspace_bytes(const moeca_stack* S) { return S ? S->total : 0; }

int moeca_stack_bind_workspace(moeca_stack* S, void* dev, size_t bytes) {
  if (S == nullptr) return fail(MOECA_E_INVAL, "stack is NULL");
  if (dev == nullptr) return fail(MOECA_E_INVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(dev) % kAlign != 0)
    return fail(MOECA_E_INVAL, "workspace must be 256-byte aligned");
  if (bytes < S->total)
    return fail(MOECA_E_INVAL, "workspace too small: need " + std::to_string(S->total) +
                                   " bytes, got " + std::to_string(bytes));
  char* w = static_cast<char*>(dev);
  for (int l = 0; l < S->L; ++l) {
    const int rc = moeca_bind_workspace(S->layers[l], w + S->layer_off[l],
                                        moeca_workspace_bytes(S->layers[l]));
    if (rc != MOECA_OK) return rc;
    moeca::layer_set_mid(S->layers[l], w + S->off[S_MID]);
  }
  moeca::BlockBufs& k = S->k;
  k.B = S->B;
  k.x = nullptr;
  k.x1 = reinterpret_cast<float*>(w + S->off[S_X1]);
  k.x1b = reinterpret_cast<float*>(w + S->off[S_X1B]);
  k.x1p = nullptr;
  k.h = reinterpret_cast<uint16_t*>(w + S->off[S_H]);
  k.u = reinterpret_cast<uint16_t*>(w + S->off[S_U]);
  k.u2 = reinterpret_cast<uint16_t*>(w + S->off[S_U2]);
  k.q = reinterpret_cast<uint16_t*>(w + S->off[S_Q]);
  k.kv = reinterpret_cast<uint16_t*>(w + S->off[S_KV]);
  k.o = reinterpret_cast<uint16_t*>(w + S->off[S_O]);
  k.y = reinterpret_cast<uint16_t*>(w + S->off[S_Y]);
  k.slist = reinterpret_cast<int32_t*>(w + S->off[S_SLIST]);
  k.soff = reinterpret_cast<int32_t*>(w + S->off[S_SOFF]);
  k.ident = reinterpret_cast<int32_t*>(w + S->off[S_IDENT]);
  k.tab = reinterpret_cast<int32_t*>(w + S->off[S_TAB]);
  S->ws = w;
  return MOECA_OK;
}

int moeca_stack_step_blocks(moeca_stack* S, float* x, const float* c, int t, int first,
                            int count, void* stream) {
  if (S == nullptr) return fail(MOECA_E_INVAL, "stack is NULL");
  if (x == nullptr || c == nullptr) return fail(MOECA_E_INVAL, "x and c are required");
  if (!aligned16(x) || !aligned16(c)) return fail(MOECA_E_INVAL, "x and c must be 16-byte aligned");
  if (t < 0) return fail(MOECA_E_INVAL, "t must be >= 0");
  if (first < 0 || count < 1 || first + count > S->L)
    return fail(MOECA_E_INVAL, "block range out of bounds");
  if (S->ws == nullptr) return fail(MOECA_E_STATE, "workspace is not bound");
  for (int l = first; l < first + count; ++l)
    if (!S->bound[l]) return fail(MOECA_E_STATE, "block " + std::to_string(l) + " has no weights");

  hipStream_t st = static_cast<hipStream_t>(stream);
  moeca::BlockBufs& k = S->k;
  k.x = x;
  const int d = S->d, N = S->N, H = S->heads, dh = d / H;
  const int T = S->B * N;
  char* w = S->ws;
  float* mod_all = reinterpret_cast<float*>(w + S->off[S_MOD]);
  double* sc = reinterpret_cast<double*>(w + S->off[S_SC]);
  const size_t mod_stride = size_t(S->B) * 6 * d;
  auto hip = [](hipError_t e, const char* what) -> int {
    if (e == hipSuccess) return MOECA_OK;
    return fail(MOECA_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
  };
  int rc;
  // SiLU(c), then the AdaLN vectors of every block of the run (they depend
  // on c only), kGemvBatch blocks per launch; the constant k/v row tables
  if ((rc = hip(moeca::launch_silu(c, S->B * d, sc, st), "silu")) != MOECA_OK) return rc;
  for (int l0 = first; l0 < first + count; l0 += moeca::kGemvBatch) {
    const int nm = std::min(moeca::kGemvBatch, first + count - l0);
    moeca::GemvBatch mats{};
    for (int i = 0; i < nm; ++i) {
      mats.W[i] = static_cast<const uint16_t*>(S->w[l0 + i].W_ada);
      mats.bias[i] = S->w[l0 + i].b_ada;
      mats.out[i] = mod_all + size_t(l0 + i) * mod_stride;
    }
    if ((rc = hip(moeca::launch_gemv(sc, S->B, d, mats, nm, 6 * d, nullptr, nullptr, 0, nullptr,
                                     st), "adaln")) != MOECA_OK)
      return rc;
  }
  if ((rc = hip(moeca::launch_slist(k, nullptr, N, d, st), "token list")) != MOECA_OK) return rc;
  const bool overlap = side_ready(S, st);

  for (int l = first; l < first + count; ++l) {
    const moeca_block_weights& W = S->w[l];
    moeca_layer* lay = S->layers[l];
    float* mod = mod_all + size_t(l) * mod_stride;
    const float* mod_prev = l > first ? mod_all + size_t(l - 1) * mod_stride : nullptr;
    auto* a = reinterpret_cast<uint16_t*>(w + S->a_off[l]);
    const auto* Wq = static_cast<const uint16_t*>(W.W_qkv);
    const uint16_t* Wkv = Wq + size_t(d) * d;
    const bool full = moeca::layer_full_step(lay, t);
    // x1 alternates between two buffers from block to block, so that a cache
    // step's LN2 can rebuild the listed tokens' x from the previous block's
    // x1 instead of LN1 storing x for every token
    float* const xa = reinterpret_cast<float*>(S->ws + S->off[S_X1]);
    float* const xb = reinterpret_cast<float*>(S->ws + S->off[S_X1B]);
    k.x1 = ((l - first) & 1) ? xb : xa;
    k.x1p = l > first ? (((l - first) & 1) ? xa : xb) : nullptr;

    if ((rc = hip(moeca::launch_ln_attn(k, T, N, d, mod, mod_prev, a, !full, st), "ln1")) !=
        MOECA_OK)
      return rc;
    // a full step lists every token first (the list call also rewrites the
    // whole-batch table that the k/v projection reads)
    if (full &&
        (rc = hip(moeca::launch_slist(k, nullptr, N, d, st), "token list")) != MOECA_OK)
      return rc;
    // keys and values of every token (tables of the whole batch), on the
    // side stream: what runs beside them on `stream` (a cache step's layer
    // decision and token list, the q projection of either step) reads no
    // k/v and writes nothing the projection reads, and fills the CUs its
    // last partial round of tiles leaves idle; the attention waits for it.
    const bool fork = overlap;
    if (fork) {
      if ((rc = hip(hipEventRecord(S->ev_fork, st), "fork")) != MOECA_OK ||
          (rc = hip(hipStreamWaitEvent(S->side, S->ev_fork, 0), "fork")) != MOECA_OK)
        return rc;
    }
    // On a cache step its persistent grid takes only as many blocks per XCD
    // as it needs to finish in the rounds of tiles it takes on every CU
    // (1024 x 8 tokens: 576 tiles, 72 per XCD, three rounds: 24 of an
    // XCD's 32 CUs), so that the decision kernels beside it find free CUs
    // (the one-block-per-sample decide kernel, 1024 threads, cannot share a
    // CU with a GEMM block) and the q projection starts on them.
    int kv_share = 0;
    if (fork && !full) {
      const int per_xcd =
          ((T + moeca::kProjTM - 1) / moeca::kProjTM * ((2 * d + moeca::kProjTN - 1) / moeca::kProjTN) +
           7) / 8;
      const int rounds = (per_xcd + moeca::cus_per_xcd() - 1) / moeca::cus_per_xcd();
      kv_share = std::max(1, (per_xcd + rounds - 1) / std::max(1, rounds));
    }
    rc = hip(moeca::launch_proj(k.h, Wkv, W.b_qkv + d, k.tab + 4, k.tab + 6, k.ident, d, 2 * d,
                                k.kv, fork ? S->side : st, kv_share),
             "kv projection");
    if (fork) {
      // the side stream's end is recorded even after a failed launch, so
      // that the main stream joins it on every path below
      const int rr = hip(hipEventRecord(S->ev_kv, S->side), "fork");
      if (rc == MOECA_OK) rc = rr;
    }
    // the main stream waits for the side stream once per block (every wait
    // is a barrier packet in the queue, which costs microseconds)
    bool joined = !fork;
    auto join = [&]() -> int {
      if (joined) return MOECA_OK;
      joined = true;
      return hip(hipStreamWaitEvent(st, S->ev_kv, 0), "join");
    };
    if (rc != MOECA_OK) {
      join();
      return rc;
    }
    // queries, attention, output projection and LN2 of the listed tokens
    auto refresh = [&](uint16_t* u_out) -> int {
      int r;
      if ((r = hip(moeca::launch_proj(k.h, Wq, W.b_qkv, k.tab, k.tab + 2, k.slist, d, d, k.q, st),
                   "q projection")) != MOECA_OK)
        return r;
      if ((r = join()) != MOECA_OK) return r;
      if ((r = hip(moeca::launch_attention(k, N, H, dh, st), "attention")) != MOECA_OK) return r;
      if ((r = hip(moeca::launch_proj(k.o, W.W_o, W.b_o, k.tab, k.tab + 2, k.slist, d, d, a, st),
                   "output projection")) != MOECA_OK)
        return r;
      return hip(moeca::launch_ln_mlp(k, T, N, d, mod, full ? nullptr : mod_prev, a, u_out, full,
                                      st),
                 "ln2");
    };
    if (full) {
      rc = refresh(k.u);
      if (rc == MOECA_OK) rc = moeca::layer_step(lay, k.u, k.u, t, k.y, st, {});
    } else {
      const uint8_t* sync = moeca::layer_buffers(lay).sync;
      rc = moeca::layer_step(lay, k.u, k.u2, t, k.y, st, [&]() -> int {
        const int r = hip(moeca::launch_slist(k, sync, N, d, st), "token list");
        return r != MOECA_OK ? r : refresh(k.u2);
      });
    }
    // the fork is joined on every path (a capture must end with it joined);
    // after the attention's wait this adds nothing
    const int rj = join();
    if (rc != MOECA_OK) return rc;
    if (rj != MOECA_OK) return rj;
  }
  const float* mod_last = mod_all + size_t(first + count - 1) * mod_stride;
  return hip(moeca::launch_ln_final(k, T, N, d, mod_last, st), "residual");
}

int moeca_stack_step(moeca_stack* S, float* x, const float* c, int t, void* stream) {
  if (S == nullptr) return fail(MOECA_E_INVAL, "stack is NULL");
  return moeca_stack_step_blocks(S, x, c, t, 0, S->L, stream);
}

int moeca_stack_cache_reset(moeca_stack* S, void* stream) {
  if (S == nullptr) return fail(MOECA_E_INVAL, "stack is NULL");
  if (S->ws == nullptr) return fail(MOECA_E_STATE, "workspace is not bound");
  for (moeca_layer* l : S->layers) {
    const int rc = moeca_cache_reset(l, stream);
    if (rc != MOECA_OK) return rc;
  }
  return MOECA_OK;
}

moeca_layer* moeca_stack_layer(moeca_stack* S, int l) {
  if (S == nullptr || l < 0 || l >= S->L) {
    fail(MOECA_E_INVAL, "bad stack or block index");
    return nullptr;
  }
  return S->layers[l];
}

int moeca_stack_embed(moeca_stack* S, const float* t_values, const int32_t* labels,
                      const void* W1, const float* b1, const void* W2, const float* b2,
                      const void* table, int n_classes, float* c, void* stream) {
  if (S == nullptr) return fail(MOECA_E_INVAL, "stack is NULL");
  if (t_values == nullptr || W1 == nullptr || b1 == nullptr || W2 == nullptr || b2 == nullptr ||
      c == nullptr)
    return fail(MOECA_E_INVAL, "t_values, W1, b1, W2, b2 and c are required");
  if (labels != nullptr && (table == nullptr || n_classes < 1))
    return fail(MOECA_E_INVAL, "labels need a class table and n_classes >= 1");
  if (!aligned16(W1) || !aligned16(W2) || !aligned16(c) || (table && !aligned16(table)) ||
      !aligned4(t_values) || !aligned4(b1) || !aligned4(b2) || !aligned4(labels))
    return fail(MOECA_E_INVAL, "matrices and c must be 16-byte aligned, vectors 4-byte");
  if (S->ws == nullptr) return fail(MOECA_E_STATE, "workspace is not bound");
  hipStream_t st = static_cast<hipStream_t>(stream);
  double* emb = reinterpret_cast<double*>(S->ws + S->off[S_EMB]);
  double* h1 = reinterpret_cast<double*>(S->ws + S->off[S_H1]);
  moeca::GemvBatch m1{}, m2{};
  m1.W[0] = static_cast<const uint16_t*>(W1);
  m1.bias[0] = b1;
  m2.W[0] = static_cast<const uint16_t*>(W2);
  m2.bias[0] = b2;
  m2.out[0] = c;
  hipError_t e = moeca::launch_sinusoid(t_values, S->B, emb, st);
  if (e == hipSuccess)
    e = moeca::launch_gemv(emb, S->B, moeca::kFreqDim, m1, 1, S->d, nullptr, nullptr, 0, h1, st);
  if (e == hipSuccess)
    e = moeca::launch_gemv(h1, S->B, S->d, m2, 1, S->d, labels ? table : nullptr, labels,
                           n_classes, nullptr, st);
  if (e != hipSuccess) return fail(MOECA_E_HIP, std::string("embed: ") + hipGetErrorString(e));
  return MOECA_OK;
}

int moeca_stack_debug_buffer(const moeca_stack* S, int which, int l, size_t* offset,
                             size_t* bytes) {
  if (S == nullptr || offset == nullptr || bytes == nullptr)
    return fail(MOECA_E_INVAL, "stack, offset and bytes are required");
  if (which < 0 || which >= MOECA_SBUF_COUNT) return fail(MOECA_E_INVAL, "unknown buffer id");
  if (which == MOECA_SBUF_A || which == MOECA_SBUF_LAYER) {
    if (l < 0 || l >= S->L) return fail(MOECA_E_INVAL, "block index out of range");
    if (which == MOECA_SBUF_A) {
      *offset = S->a_off[l];
      *bytes = size_t(S->B) * S->N * S->d * 2;
    } else {
      *offset = S->layer_off[l];
      *bytes = moeca_workspace_bytes(S->layers[l]);
    }
    return MOECA_OK;
  }
  *offset = S->off[which];
  *bytes = S->bytes[which];
  return MOECA_OK;
}

}  // extern "C"
