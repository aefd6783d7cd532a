// C ABI and host orchestration of the branch-cached MoE layer step.
//
// The host decides full vs cache step (Sec. 4.1; refresh cycle of Sec. 5.1)
// and enqueues the kernels on the caller's stream.  It never waits for the
// device inside a step and never allocates device memory: the caller binds
// the workspace, which this file only partitions.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "internal.h"
#include "moeca.h"

using moeca::Buffers;
using moeca::Shape;

namespace moeca {
LaunchEvents& launch_events() {
  thread_local LaunchEvents ev;
  return ev;
}
}  // namespace moeca

namespace {

thread_local std::string g_error;

int fail(int code, const std::string& msg) {
  g_error = msg;
  return code;
}

// Kernels read and write 16-byte vectors.
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr size_t kAlign = 256;
constexpr int kMaxTimedSteps = 512;
constexpr int kEventsPerStep = 2 * MOECA_STAGE_COUNT;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Workspace regions, in order.  Public ids come first (MOECA_BUF_*).
enum Region {
  R_E_C, R_W_C, R_N_C, R_H_C, R_STAT, R_LOGITS, R_E_T, R_W_T, R_HBAR, R_TAU, R_MARGIN, R_Q,
  R_MASK, R_SIGMA, R_SYNC, R_OFF, R_LIST, R_POS,
  R_CNT_BS, R_STATS_BS, R_RFLAGS, R_TILES, R_ROW_DST, R_ENT, R_CNT_CH, R_WIDE, R_MID, R_H_SH,
  R_PART, R_COUNT
};

struct Layout {
  size_t off[R_COUNT];
  size_t bytes[R_COUNT];
  size_t total;
};

// external_mid: the FFN intermediate lives outside this workspace (the
// blocks of a stack run one after another and share one).  partials: room
// for the down projection's partial sums of the weight-streaming plan
// (layers that can take it; not for the uncached forward of
// moeca_forward_noalloc, which never does).
Layout make_layout(const Shape& s, bool external_mid = false, bool partials = true) {
  const size_t nbr = static_cast<size_t>(s.branches());
  const size_t ntok = static_cast<size_t>(s.tokens());
  const size_t act = s.act_bytes();
  size_t b[R_COUNT];
  b[R_E_C] = nbr * 4;
  b[R_W_C] = nbr * 4;
  b[R_N_C] = nbr * 4;
  b[R_H_C] = nbr * s.d * act;
  b[R_STAT] = size_t(s.B) * s.E * s.N * 4;
  b[R_LOGITS] = ntok * s.E * 4;
  b[R_E_T] = nbr * 4;
  b[R_W_T] = nbr * 4;
  b[R_HBAR] = size_t(s.B) * s.E * 4;
  b[R_TAU] = size_t(s.B) * s.E * 4;
  b[R_MARGIN] = nbr * 4;
  b[R_Q] = nbr * 4;
  b[R_MASK] = nbr;
  b[R_SIGMA] = nbr * 4;
  b[R_SYNC] = ntok;
  b[R_OFF] = size_t(s.groups() + 1) * 4;
  b[R_LIST] = nbr * 4;
  b[R_POS] = nbr * 4;
  b[R_CNT_BS] = size_t(s.B) * s.E * 4;
  b[R_STATS_BS] = size_t(s.B) * 4 * 4;
  b[R_RFLAGS] = size_t(moeca::router_blocks(s)) * 4;
  b[R_TILES] = size_t(2) * (s.groups() + 1) * 4;
  b[R_ROW_DST] = nbr * 4;
  b[R_ENT] = size_t(s.B) * s.E * ((size_t(s.N) + 15) / 16) * 2 * 8;
  b[R_CNT_CH] = size_t(s.B) * ((size_t(s.N) * s.k + 1023) / 1024) * s.E * 4;
  b[R_WIDE] = size_t(s.B) * moeca::kWideWords * 4;
  b[R_MID] = external_mid ? 0 : size_t(s.mid_rows()) * s.d_ff * act;
  b[R_H_SH] = size_t(s.S) * ntok * s.d * act;
  b[R_PART] = partials && moeca::thin_capable(s)
                  ? size_t(moeca::kThinSplit) * size_t(s.mid_rows()) * s.d * 4
                  : 0;
  Layout L;
  size_t cur = 0;
  for (int i = 0; i < R_COUNT; ++i) {
    L.off[i] = cur;
    L.bytes[i] = b[i];
    cur = align_up(cur + b[i]);
  }
  L.total = cur;
  // the public view of the offsets covers the routed experts only
  L.bytes[R_OFF] = size_t(s.E + 1) * 4;
  return L;
}

// Device views of the regions of a workspace at w laid out as lay; the FFN
// intermediate at mid when it lives outside the workspace.
Buffers map_buffers(char* w, const Layout& lay, void* mid) {
  const size_t* o = lay.off;
  Buffers b{};
  b.e_c = reinterpret_cast<int32_t*>(w + o[R_E_C]);
  b.w_c = reinterpret_cast<float*>(w + o[R_W_C]);
  b.n_c = reinterpret_cast<float*>(w + o[R_N_C]);
  b.h_c = w + o[R_H_C];
  b.stat = reinterpret_cast<float*>(w + o[R_STAT]);
  b.ent = reinterpret_cast<double*>(w + o[R_ENT]);
  b.logits = reinterpret_cast<float*>(w + o[R_LOGITS]);
  b.e_t = reinterpret_cast<int32_t*>(w + o[R_E_T]);
  b.w_t = reinterpret_cast<float*>(w + o[R_W_T]);
  b.hbar = reinterpret_cast<float*>(w + o[R_HBAR]);
  b.tau = reinterpret_cast<float*>(w + o[R_TAU]);
  b.margin = reinterpret_cast<float*>(w + o[R_MARGIN]);
  b.q = reinterpret_cast<int32_t*>(w + o[R_Q]);
  b.mask = reinterpret_cast<uint8_t*>(w + o[R_MASK]);
  b.sigma = reinterpret_cast<int32_t*>(w + o[R_SIGMA]);
  b.sync = reinterpret_cast<uint8_t*>(w + o[R_SYNC]);
  b.off = reinterpret_cast<int32_t*>(w + o[R_OFF]);
  b.list = reinterpret_cast<int32_t*>(w + o[R_LIST]);
  b.pos = reinterpret_cast<int32_t*>(w + o[R_POS]);
  b.cnt_bs = reinterpret_cast<int32_t*>(w + o[R_CNT_BS]);
  b.cnt_ch = reinterpret_cast<int32_t*>(w + o[R_CNT_CH]);
  b.wide = reinterpret_cast<int32_t*>(w + o[R_WIDE]);
  b.stats_bs = reinterpret_cast<int32_t*>(w + o[R_STATS_BS]);
  b.rflags = reinterpret_cast<int32_t*>(w + o[R_RFLAGS]);
  b.tiles = reinterpret_cast<int32_t*>(w + o[R_TILES]);
  b.row_dst = reinterpret_cast<int32_t*>(w + o[R_ROW_DST]);
  b.mid = mid != nullptr ? mid : w + o[R_MID];
  b.h_sh = w + o[R_H_SH];
  b.part = lay.bytes[R_PART] != 0 ? reinterpret_cast<float*>(w + o[R_PART]) : nullptr;
  return b;
}

}  // namespace

struct moeca_layer {
  Shape shape;
  moeca_policy pol;
  Layout layout;
  const void* W_r = nullptr;
  const float* b_r = nullptr;
  const void* W_up = nullptr;
  const void* W_down = nullptr;
  const void* W_up_sh = nullptr;
  const void* W_down_sh = nullptr;
  char* ws = nullptr;
  Buffers buf{};
  const void* attn_in = nullptr;
  void* attn_cache = nullptr;
  bool valid = false;
  bool mid_outside = false;      // the FFN intermediate is not in ws
  void* external_mid = nullptr;  // its address when mid_outside
  bool last_full = false;
  int last_plan = 0;
  bool timing = false;
  std::vector<hipEvent_t> events;
  int timed_steps = 0;
};

extern "C" {

void moeca_policy_default(moeca_policy* p) {
  if (p == nullptr) return;
  std::memset(p, 0, sizeof(*p));
  p->mode = MOECA_MODE_THRESHOLD;
  p->ratio = 0.3f;
  p->tau0 = 0.80f;
  p->alpha = 0.6f;
  p->beta = 0.65f;
  p->lambda0 = 1.0f;
  p->lambda1 = 1.0f;
  p->lambda2 = 1.0f;
  p->refresh_cycle = 4;
  p->norm_topk = 1;
  p->act = MOECA_ACT_GELU_TANH;
  p->dtype = MOECA_DTYPE_BF16;
  p->batch = 1;
  p->tokens = 1;
  p->n_shared = 0;
}

const char* moeca_last_error(void) { return g_error.c_str(); }

moeca_layer* moeca_layer_create(int d, int E, int k, int d_ff, const moeca_policy* p) {
  g_error.clear();
  auto bad = [](const std::string& m) -> moeca_layer* {
    fail(MOECA_E_INVAL, m);
    return nullptr;
  };
  if (p == nullptr) return bad("policy is NULL");
  if (d <= 0 || d % 64 != 0 || d > 16384) return bad("d must be a positive multiple of 64, <= 16384");
  if (p->act != MOECA_ACT_GELU_TANH && p->act != MOECA_ACT_GELU_ERF &&
      p->act != MOECA_ACT_SWIGLU)
    return bad("unknown act");
  const int max_ff = p->act == MOECA_ACT_SWIGLU ? 32768 : 65536;
  if (d_ff <= 0 || d_ff % 64 != 0 || d_ff > max_ff)
    return bad("d_ff must be a positive multiple of 64, <= " + std::to_string(max_ff));
  if (E < 1 || E > 64) return bad("E must be in [1, 64]");
  if (k < 1 || k > 8 || k > E) return bad("k must be in [1, min(E, 8)]");
  if (p->n_shared < 0 || p->n_shared > 8) return bad("n_shared must be in [0, 8]");
  if (p->mode < MOECA_MODE_FULL || p->mode > MOECA_MODE_RATIO) return bad("unknown mode");
  if (p->dtype != MOECA_DTYPE_BF16 && p->dtype != MOECA_DTYPE_FP32) return bad("unknown dtype");
  if (!(p->ratio >= 0.0f && p->ratio <= 1.0f)) return bad("ratio must be in [0, 1]");
  if (!(p->tau0 > 0.0f) || !std::isfinite(p->tau0)) return bad("tau0 must be finite and > 0");
  if (!(p->alpha >= 0.0f && p->alpha < 1.0f)) return bad("alpha must be in [0, 1)");
  if (!(p->beta >= 0.0f && p->beta < 1.0f)) return bad("beta must be in [0, 1)");
  if (!(p->lambda1 >= 0.0f) || !std::isfinite(p->lambda1) || !(p->lambda2 >= 0.0f) ||
      !std::isfinite(p->lambda2) || !(p->lambda0 >= 0.0f) || !std::isfinite(p->lambda0))
    return bad("lambda0, lambda1, lambda2 must be finite and >= 0");
  if (p->refresh_cycle < 0) return bad("refresh_cycle must be >= 0");
  if (p->norm_topk != 0 && p->norm_topk != 1) return bad("norm_topk must be 0 or 1");
  if (p->batch < 1 || p->tokens < 1) return bad("batch and tokens must be >= 1");
  const int64_t nbr = int64_t(p->batch) * p->tokens * (k + p->n_shared);
  if (nbr >= (int64_t(1) << 31) - 1024) return bad("batch * tokens * (k + n_shared) too large");
  if (int64_t(p->tokens) * k > 32768 && 1024 % k != 0)
    return bad("tokens * k above 32768 needs k in {1, 2, 4, 8}");
  if (int64_t(p->batch) * p->tokens * d >= (int64_t(1) << 40)) return bad("batch too large");

  auto* L = new (std::nothrow) moeca_layer();
  if (L == nullptr) return bad("out of host memory");
  L->shape = Shape{d, E, k, d_ff, p->batch, p->tokens, p->dtype == MOECA_DTYPE_BF16};
  L->shape.S = p->n_shared;
  L->shape.swiglu = p->act == MOECA_ACT_SWIGLU;
  L->pol = *p;
  L->layout = make_layout(L->shape);
  return L;
}

void moeca_layer_destroy(moeca_layer* L) {
  if (L == nullptr) return;
  for (hipEvent_t e : L->events) (void)hipEventDestroy(e);
  delete L;
}

int moeca_layer_set_weights(moeca_layer* L, const void* W_r, const float* b_r, const void* W_up,
                            const void* W_down) {
  if (L == nullptr) return fail(MOECA_E_INVAL, "layer is NULL");
  if (W_r == nullptr || W_up == nullptr || W_down == nullptr)
    return fail(MOECA_E_INVAL, "W_r, W_up and W_down are required");
  if (!aligned16(W_r) || !aligned16(W_up) || !aligned16(W_down) ||
      (reinterpret_cast<uintptr_t>(b_r) & 3u) != 0)
    return fail(MOECA_E_INVAL, "weights must be 16-byte aligned (bias 4-byte)");
  L->W_r = W_r;
  L->b_r = b_r;
  L->W_up = W_up;
  L->W_down = W_down;
  return MOECA_OK;
}

int moeca_layer_set_shared(moeca_layer* L, const void* W_up_s, const void* W_down_s) {
  if (L == nullptr) return fail(MOECA_E_INVAL, "layer is NULL");
  if (L->shape.S == 0) return fail(MOECA_E_INVAL, "the layer has no shared experts");
  if (W_up_s == nullptr || W_down_s == nullptr)
    return fail(MOECA_E_INVAL, "W_up_s and W_down_s are required");
  if (!aligned16(W_up_s) || !aligned16(W_down_s))
    return fail(MOECA_E_INVAL, "shared weights must be 16-byte aligned");
  L->W_up_sh = W_up_s;
  L->W_down_sh = W_down_s;
  return MOECA_OK;
}

size_t moeca_workspace_bytes(const moeca_layer* L) { return L ? L->layout.total : 0; }

int moeca_bind_workspace(moeca_layer* L, void* dev, size_t bytes) {
  if (L == nullptr) return fail(MOECA_E_INVAL, "layer is NULL");
  if (dev == nullptr) return fail(MOECA_E_INVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(dev) % kAlign != 0)
    return fail(MOECA_E_INVAL, "workspace must be 256-byte aligned");
  if (bytes < L->layout.total)
    return fail(MOECA_E_INVAL, "workspace too small: need " + std::to_string(L->layout.total) +
                                   " bytes, got " + std::to_string(bytes));
  char* w = static_cast<char*>(dev);
  L->buf = map_buffers(w, L->layout, L->mid_outside ? L->external_mid : nullptr);
  L->ws = w;
  L->valid = false;
  return MOECA_OK;
}

int moeca_bind_attention(moeca_layer* L, const void* attn_in, void* attn_cache) {
  if (L == nullptr) return fail(MOECA_E_INVAL, "layer is NULL");
  if ((attn_in == nullptr) != (attn_cache == nullptr))
    return fail(MOECA_E_INVAL, "attn_in and attn_cache must both be set or both be NULL");
  if (!aligned16(attn_in) || !aligned16(attn_cache))
    return fail(MOECA_E_INVAL, "attention buffers must be 16-byte aligned");
  L->attn_in = attn_in;
  L->attn_cache = attn_cache;
  return MOECA_OK;
}

int moeca_step(moeca_layer* L, const void* x_t, int t, void* out, void* stream) {
  return moeca::layer_step(L, x_t, x_t, t, out, static_cast<hipStream_t>(stream), {});
}

int moeca_forward_noalloc(const moeca_layer* L, const void* x, int samples, void* out,
                          void* stream) {
  if (L == nullptr) return fail(MOECA_E_INVAL, "layer is NULL");
  if (x == nullptr || out == nullptr) return fail(MOECA_E_INVAL, "x and out are required");
  if (!aligned16(x) || !aligned16(out)) return fail(MOECA_E_INVAL, "x and out must be 16-byte aligned");
  if (samples < 1 || samples > L->shape.B)
    return fail(MOECA_E_INVAL, "samples must be in [1, " + std::to_string(L->shape.B) + "]");
  Shape s = L->shape;
  s.B = samples;
  const Layout lay = make_layout(s, false, false);
  if (lay.total > moeca::kNoallocScratchBytes)
    return fail(MOECA_E_INVAL, "this call needs " + std::to_string(lay.total) +
                                   " bytes of scratch; the library's array holds " +
                                   std::to_string(moeca::kNoallocScratchBytes) +
                                   " (use fewer samples per call, or moeca_step)");
  if (L->W_r == nullptr) return fail(MOECA_E_STATE, "weights are not bound");
  if (s.S > 0 && L->W_up_sh == nullptr)
    return fail(MOECA_E_STATE, "shared expert weights are not bound");
  void* base = nullptr;
  hipError_t e = moeca::noalloc_scratch(&base);
  if (e != hipSuccess)
    return fail(MOECA_E_HIP, std::string("scratch address: ") + hipGetErrorString(e));
  const Buffers b = map_buffers(static_cast<char*>(base), lay, nullptr);
  const moeca_policy& p = L->pol;
  const auto st = static_cast<hipStream_t>(stream);
  // the uncached layer: every branch recomputed, no statistic, no cache
  // metadata and no attention path (the MOECA_MODE_FULL step)
  if ((e = moeca::launch_router(s, x, L->W_r, L->b_r, p.norm_topk, p.beta, false, b, st)) ==
          hipSuccess &&
      (e = moeca::launch_decide(s, moeca::kSelFull, 0, p.lambda0, p.lambda1, p.lambda2, false,
                                p.tau0, p.alpha, b, st)) == hipSuccess &&
      (e = moeca::launch_lists(s, moeca::ffn_plan(s), b, st)) == hipSuccess &&
      (e = moeca::launch_ffn_up(s, x, L->W_up, L->W_up_sh, p.act, moeca::ffn_plan(s), b, st)) ==
          hipSuccess &&
      (e = moeca::launch_ffn_down(s, L->W_down, L->W_down_sh, moeca::ffn_plan(s), b, st)) ==
          hipSuccess)
    e = moeca::launch_combine(s, 0, out, nullptr, nullptr, b, st);
  if (e != hipSuccess) return fail(MOECA_E_HIP, std::string("launch: ") + hipGetErrorString(e));
  return MOECA_OK;
}

}  // extern "C"

namespace moeca {

int set_error(int code, const std::string& msg) { return fail(code, msg); }

size_t layer_mid_bytes(const moeca_layer* L) {
  const Shape& s = L->shape;
  return size_t(s.mid_rows()) * s.d_ff * s.act_bytes();
}

void layer_keep_mid_outside(moeca_layer* L) {
  L->mid_outside = true;
  L->layout = make_layout(L->shape, true);
  L->ws = nullptr;  // the layout changed: bind again
}

void layer_set_mid(moeca_layer* L, void* mid) {
  L->external_mid = mid;
  L->buf.mid = mid;
}

bool layer_full_step(const moeca_layer* L, int t) {
  const moeca_policy& p = L->pol;
  return p.mode == MOECA_MODE_FULL || !L->valid || (p.refresh_cycle > 0 && t % p.refresh_cycle == 0);
}

const Buffers& layer_buffers(const moeca_layer* L) { return L->buf; }

int layer_step(moeca_layer* L, const void* x_t, const void* x_ffn, int t, void* out,
               hipStream_t st, const std::function<int()>& between) {
  if (L == nullptr) return fail(MOECA_E_INVAL, "layer is NULL");
  if (x_t == nullptr || x_ffn == nullptr || out == nullptr)
    return fail(MOECA_E_INVAL, "x_t and out are required");
  if (t < 0) return fail(MOECA_E_INVAL, "t must be >= 0");
  if (!aligned16(x_t) || !aligned16(x_ffn) || !aligned16(out))
    return fail(MOECA_E_INVAL, "x_t and out must be 16-byte aligned");
  if (L->W_r == nullptr) return fail(MOECA_E_STATE, "weights are not bound");
  if (L->ws == nullptr) return fail(MOECA_E_STATE, "workspace is not bound");
  if (L->mid_outside && L->external_mid == nullptr)
    return fail(MOECA_E_STATE, "the FFN intermediate is not bound");
  if (L->shape.S > 0 && L->W_up_sh == nullptr)
    return fail(MOECA_E_STATE, "shared expert weights are not bound");
  const Shape& s = L->shape;
  const moeca_policy& p = L->pol;
  const bool uncached = p.mode == MOECA_MODE_FULL;
  const bool full = layer_full_step(L, t);

  const bool timed = L->timing && L->timed_steps < kMaxTimedSteps;
  hipEvent_t* ev = timed ? &L->events[size_t(L->timed_steps) * kEventsPerStep] : nullptr;
  // Each stage's kernel records its start and completion events with its
  // own dispatch (launch_kernel).  A stage that launches nothing records
  // both events back to back.
  int stage = 0;
  auto arm = [&]() {
    if (ev) {
      moeca::launch_events() = {ev[2 * stage], ev[2 * stage + 1]};
    }
  };
  auto check = [&](hipError_t e, const char* what) -> bool {
    if (ev) {
      moeca::LaunchEvents& le = moeca::launch_events();
      if (le.start != nullptr) {
        le = moeca::LaunchEvents{};
        if (e == hipSuccess) e = hipEventRecord(ev[2 * stage], st);
        if (e == hipSuccess) e = hipEventRecord(ev[2 * stage + 1], st);
      }
      ++stage;
    }
    if (e != hipSuccess) {
      fail(MOECA_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
      return false;
    }
    return true;
  };

  const Buffers& b = L->buf;
  arm();
  if (!check(moeca::launch_router(s, x_t, L->W_r, L->b_r, p.norm_topk, p.beta, !uncached, b, st),
             "router"))
    return MOECA_E_HIP;
  // the entropy and thresholds are derived inside the decide kernel; the
  // statistic stage launches nothing of its own
  arm();
  if (!check(hipSuccess, "entropy")) return MOECA_E_HIP;
  int sel = moeca::kSelFull;
  int budget = 0;
  if (!full) {
    sel = p.mode == MOECA_MODE_THRESHOLD ? moeca::kSelThreshold : moeca::kSelRatio;
    budget = static_cast<int>(std::floor(static_cast<double>(p.ratio) * s.N * s.k + 0.5));
  }
  arm();
  if (!check(moeca::launch_decide(s, sel, budget, p.lambda0, p.lambda1, p.lambda2, !uncached, p.tau0,
                                  p.alpha, b, st),
             "decide"))
    return MOECA_E_HIP;
  // ratio-mode cache steps whose budget leaves few rows per expert stream
  // the weights with the thin plan
  const bool thin = !full && p.mode == MOECA_MODE_RATIO &&
                    int64_t(budget) * s.B <= int64_t(moeca::kThinRows) * s.E &&
                    L->buf.part != nullptr;
  // and those that leave a few hundred take the expert-wide up projection,
  // as do full steps of that many rows per expert (every branch)
  const bool wide = (full ? int64_t(s.B) * s.N * s.k <= int64_t(moeca::kWideRows) * s.E
                          : p.mode == MOECA_MODE_RATIO &&
                                int64_t(budget) * s.B <= int64_t(moeca::kWideRows) * s.E);
  const moeca::FfnPlan plan = moeca::ffn_plan(s, thin, wide);
  arm();
  if (!check(moeca::launch_lists(s, plan, b, st), "lists")) return MOECA_E_HIP;
  if (between) {
    const int rc = between();
    if (rc != MOECA_OK) return rc;
  }
  arm();
  if (!check(moeca::launch_ffn_up(s, x_ffn, L->W_up, L->W_up_sh, p.act, plan, b, st), "ffn up"))
    return MOECA_E_HIP;
  arm();
  if (!check(moeca::launch_ffn_down(s, L->W_down, L->W_down_sh, plan, b, st), "ffn down"))
    return MOECA_E_HIP;
  arm();
  if (!check(moeca::launch_combine(s, uncached ? 0 : 1, out, L->attn_in, L->attn_cache, b, st),
             "combine"))
    return MOECA_E_HIP;
  if (timed) ++L->timed_steps;
  if (!uncached) L->valid = true;
  L->last_full = full;
  L->last_plan = plan.thin ? 1 : plan.wide_up ? 2 : 0;
  return MOECA_OK;
}

}  // namespace moeca

extern "C" {

int moeca_cache_reset(moeca_layer* L, void* stream) {
  if (L == nullptr) return fail(MOECA_E_INVAL, "layer is NULL");
  if (L->ws == nullptr) return fail(MOECA_E_STATE, "workspace is not bound");
  const hipError_t e = moeca::launch_reset(L->shape, L->buf, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(MOECA_E_HIP, std::string("reset: ") + hipGetErrorString(e));
  L->valid = false;
  return MOECA_OK;
}

int moeca_get_stats(moeca_layer* L, moeca_stats* out, void* stream) {
  if (L == nullptr || out == nullptr) return fail(MOECA_E_INVAL, "layer and out are required");
  if (L->ws == nullptr) return fail(MOECA_E_STATE, "workspace is not bound");
  const Shape& s = L->shape;
  hipStream_t st = static_cast<hipStream_t>(stream);
  std::vector<int32_t> sb(size_t(s.B) * 4), cb(size_t(s.B) * s.E),
      rf(size_t(moeca::router_blocks(s)));
  hipError_t e = hipMemcpyAsync(sb.data(), L->buf.stats_bs, sb.size() * 4, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(cb.data(), L->buf.cnt_bs, cb.size() * 4, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(rf.data(), L->buf.rflags, rf.size() * 4, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return fail(MOECA_E_HIP, std::string("stats: ") + hipGetErrorString(e));
  std::memset(out, 0, sizeof(*out));
  out->n_branches = s.branches();
  for (int b = 0; b < s.B; ++b) {
    out->n_recompute += sb[b * 4 + 0];
    out->n_unmatched += sb[b * 4 + 1];
    out->n_matched += sb[b * 4 + 2];
    out->n_sync += sb[b * 4 + 3];
    for (int x = 0; x < s.E; ++x) out->expert_count[x] += cb[size_t(b) * s.E + x];
  }
  out->n_reused = out->n_matched - (out->n_recompute - out->n_unmatched);
  if (L->last_full) out->n_reused = 0;
  out->reuse_over_match =
      out->n_matched > 0 ? double(out->n_reused) / double(out->n_matched) : 0.0;
  out->full_step = L->last_full ? 1 : 0;
  out->ffn_plan = L->last_plan;
  for (int32_t v : rf) out->nonfinite |= v;
  return MOECA_OK;
}

int moeca_debug_buffer(const moeca_layer* L, int which, size_t* offset, size_t* bytes) {
  if (L == nullptr || offset == nullptr || bytes == nullptr)
    return fail(MOECA_E_INVAL, "layer, offset and bytes are required");
  if (which < 0 || which >= MOECA_BUF_COUNT) return fail(MOECA_E_INVAL, "unknown buffer id");
  *offset = L->layout.off[which];
  *bytes = L->layout.bytes[which];
  return MOECA_OK;
}

int moeca_debug_set_valid(moeca_layer* L, int valid) {
  if (L == nullptr) return fail(MOECA_E_INVAL, "layer is NULL");
  L->valid = valid != 0;
  return MOECA_OK;
}

int moeca_set_timing(moeca_layer* L, int enable) {
  if (L == nullptr) return fail(MOECA_E_INVAL, "layer is NULL");
  for (hipEvent_t e : L->events) (void)hipEventDestroy(e);
  L->events.clear();
  L->timed_steps = 0;
  L->timing = false;
  if (!enable) return MOECA_OK;
  L->events.resize(size_t(kMaxTimedSteps) * kEventsPerStep);
  for (auto& e : L->events) {
    // timing-only events: no system-scope fence (cache writeback) at each
    // record, which would stretch the measured kernel intervals
    const hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
    if (r != hipSuccess) {
      e = nullptr;
      return fail(MOECA_E_HIP, std::string("event create: ") + hipGetErrorString(r));
    }
  }
  L->timing = true;
  return MOECA_OK;
}

int moeca_get_timing(moeca_layer* L, double* ms, int n, int* steps) {
  if (L == nullptr || ms == nullptr || steps == nullptr)
    return fail(MOECA_E_INVAL, "layer, ms and steps are required");
  if (n < 0 || n > MOECA_STAGE_COUNT) return fail(MOECA_E_INVAL, "n out of range");
  for (int i = 0; i < n; ++i) ms[i] = 0.0;
  *steps = L->timed_steps;
  if (!L->timing || L->timed_steps == 0) return MOECA_OK;
  const hipError_t e =
      hipEventSynchronize(L->events[size_t(L->timed_steps) * kEventsPerStep - 1]);
  if (e != hipSuccess) return fail(MOECA_E_HIP, std::string("timing: ") + hipGetErrorString(e));
  for (int sidx = 0; sidx < L->timed_steps; ++sidx) {
    hipEvent_t* ev = &L->events[size_t(sidx) * kEventsPerStep];
    for (int i = 0; i < n; ++i) {
      float v = 0.0f;
      const hipError_t r = hipEventElapsedTime(&v, ev[2 * i], ev[2 * i + 1]);
      if (r != hipSuccess)
        return fail(MOECA_E_HIP, std::string("elapsed: ") + hipGetErrorString(r));
      ms[i] += v;
    }
  }
  L->timed_steps = 0;
  return MOECA_OK;
}

}  // extern "C"
