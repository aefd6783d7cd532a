// Internal interface between the host orchestration (moeca.cpp) and the
// kernel launchers (*.hip).  Not part of the public C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <cstddef>
#include <cstdint>
#include <functional>
#include <string>

#include "moeca.h"

namespace moeca {

// Launch timing.  When `start` is set, the next kernel launched through
// launch_kernel records the two events as part of its own dispatch (its
// start and completion timestamps, with no marker packets in between), and
// the slot is cleared.  Per host thread.
struct LaunchEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};
LaunchEvents& launch_events();

template <typename... P, typename... A>
inline void launch_kernel(void (*kernel)(P...), dim3 grid, dim3 block, uint32_t shmem,
                          hipStream_t st, A... args) {
  LaunchEvents& ev = launch_events();
  if (ev.start != nullptr) {
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, st, ev.start, ev.stop, 0u,
                          static_cast<P>(args)...);
    ev = LaunchEvents{};
  } else {
    kernel<<<grid, block, shmem, st>>>(static_cast<P>(args)...);
  }
}

// A launch that records `start` before and/or `stop` after its dispatch
// (either may be null): the first and last kernels of a stage that launches
// several.
template <typename... P, typename... A>
inline void launch_kernel_ev(void (*kernel)(P...), dim3 grid, dim3 block, uint32_t shmem,
                             hipStream_t st, hipEvent_t start, hipEvent_t stop, A... args) {
  if (start != nullptr || stop != nullptr)
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, st, start, stop, 0u,
                          static_cast<P>(args)...);
  else
    kernel<<<grid, block, shmem, st>>>(static_cast<P>(args)...);
}

// Per-sample scratch words of the multi-block decision path: four 256-bin
// digit histograms, counters, and up to 64 ranked candidates.
constexpr int kWideWords = 1280;

struct Shape {
  int d, E, k, d_ff, B, N;
  bool bf16;
  int S = 0;            // shared experts
  bool swiglu = false;  // gated experts: 2 d_ff up-projection rows
  int64_t tokens() const { return int64_t(B) * N; }
  int64_t branches() const { return int64_t(B) * N * k; }
  size_t act_bytes() const { return bf16 ? 2 : 4; }
  int groups() const { return E + S; }                // grouped-GEMM groups
  int up_rows() const { return swiglu ? 2 * d_ff : d_ff; }
  int64_t mid_rows() const { return branches() + int64_t(S) * tokens(); }
};

// Device views of the workspace regions (see moeca_debug_buffer for the
// meaning of the public ones).
struct Buffers {
  int32_t* e_c;
  float* w_c;
  float* n_c;
  void* h_c;
  float* stat;      // [B][E][N]
  double* ent;      // [B][E][ceil(N/16)][2] per 16 positions of the statistic:
                    // sum C and sum C log C (the router writes them)
  float* logits;    // [B*N][E]
  int32_t* e_t;
  float* w_t;
  float* hbar;      // [B][E]
  float* tau;       // [B][E]
  float* margin;
  int32_t* q;
  uint8_t* mask;
  int32_t* sigma;
  uint8_t* sync;    // [B*N]
  int32_t* off;     // [E+S+1] group row offsets: routed experts into `list`,
                    // then the shared experts (T rows each) after them
  int32_t* list;
  int32_t* pos;
  int32_t* cnt_bs;  // [B][E] recomputed branches per sample and expert
  int32_t* cnt_ch;  // [B][RC][E] the same per chunk of 1024 branches (RC = ceil(N k / 1024))
  int32_t* stats_bs;// [B][4] recompute, unmatched, matched, sync per sample
  int32_t* rflags;  // router: one non-finite flag per block
  int32_t* tiles;   // [2][E+S+1] grouped-GEMM tile prefix per group (up, down)
  int32_t* row_dst; // [B*N*k] cache row of each listed branch: (f/k)*k + sigma(f)
  int32_t* wide;    // [B][kWideWords] per-sample scratch of the multi-block decision path
  void* mid;        // [B*N*k + S*T][d_ff] FFN activation of listed and shared rows
  void* h_sh;       // [S][T][d] shared experts' outputs
  float* part;      // [kThinSplit][B*N*k][d] fp32 partial sums of the down projection's
                    // K pieces (layers that may take the weight-streaming plan)
};

// Tiling of the grouped expert FFN: M tile (rows of one expert), N tile of
// the up and down projections, and the number of K pieces of the down
// projection.  The lists kernel turns the per-expert row counts into tile
// (unit) prefixes with the same plan.  thin: the weight-streaming kernel
// (128 x 288 tiles) for both projections, the down projection in
// kThinSplit K pieces whose fp32 partial sums are added in piece order.
struct FfnPlan {
  int tm;
  int tn_up;
  int tn_down;
  int split_down = 1;
  bool thin = false;
  bool wide_up = false;  // the up projection takes the expert-wide kernel
  int tm_up = 128;       // M tile of the up projection's tile table
};
constexpr int kThinSplit = 4;
// A ratio-mode cache step takes the thin plan when its budget leaves at most
// this many rows per expert on average (unmatched branches come on top).
constexpr int kThinRows = 112;
// A ratio-mode cache step with more rows per expert than that, and at most
// this many on average, takes the expert-wide up-projection tiles (all of
// an expert's rows, up to 384, by 144 columns); so does a full step with at
// most this many branches per expert on average.
constexpr int kWideRows = 320;
FfnPlan ffn_plan(const Shape& s, bool thin = false, bool wide = false);
// Layers that may take the wide up projection: bf16, no shared experts,
// ungated, d_ff a multiple of 144.
bool wide_capable(const Shape& s);
// Layers that may take the thin plan: bf16, no shared experts, ungated, at
// most 256 rows per expert on a full step, and enough 288-wide
// up-projection tiles for half the CUs.  Their workspace holds `part`.
bool thin_capable(const Shape& s);
int device_cus();

enum SelectMode { kSelFull = 0, kSelThreshold = 1, kSelRatio = 2 };

int router_blocks(const Shape& s);

hipError_t launch_router(const Shape& s, const void* x, const void* W_r, const float* b_r,
                         int norm_topk, float beta, bool update_stat, const Buffers& b,
                         hipStream_t st);
// with_stat: the router advanced the statistic in this step; the decide
// kernel then derives the entropy and thresholds first (hbar, tau).
hipError_t launch_decide(const Shape& s, int sel_mode, int budget, float lambda0, float lambda1,
                         float lambda2, bool with_stat, float tau0, float alpha,
                         const Buffers& b, hipStream_t st);
hipError_t launch_lists(const Shape& s, const FfnPlan& plan, const Buffers& b, hipStream_t st);
// act: MOECA_ACT_* of the policy.  W_*_sh: the shared experts (S > 0).
hipError_t launch_ffn_up(const Shape& s, const void* x, const void* W_up, const void* W_up_sh,
                         int act, const FfnPlan& plan, const Buffers& b, hipStream_t st);
// With plan.split_down > 1 this also adds the partial sums into the cache rows.
hipError_t launch_ffn_down(const Shape& s, const void* W_down, const void* W_down_sh,
                           const FfnPlan& plan, const Buffers& b, hipStream_t st);
hipError_t launch_combine(const Shape& s, int write_cache, void* out, const void* attn_in,
                          void* attn_cache, const Buffers& b, hipStream_t st);
hipError_t launch_reset(const Shape& s, const Buffers& b, hipStream_t st);

// ---- the entry point that allocates nothing (noalloc.hip) --------------
// Bytes of the library-owned device array every call of
// moeca_forward_noalloc on a GPU shares.
constexpr size_t kNoallocScratchBytes = size_t(64) << 20;
// The array's device address on the current device (looked up once per
// device with hipGetSymbolAddress).
hipError_t noalloc_scratch(void** out);

// ---- the MoE layer step, as used by a block (moeca.cpp) ----------------
// The step of moeca_step with the router reading x_route and the expert FFN
// reading x_ffn; `between`, when set, is called after the decision and the
// expert lists are enqueued and before the FFN (a nonzero return aborts the
// step with that code).
// Set this thread's moeca_last_error() text; returns code.
int set_error(int code, const std::string& msg);

int layer_step(moeca_layer* L, const void* x_route, const void* x_ffn, int t, void* out,
               hipStream_t st, const std::function<int()>& between);
bool layer_full_step(const moeca_layer* L, int t);
// Bytes of the layer's FFN intermediate (sized for a full step).
size_t layer_mid_bytes(const moeca_layer* L);
// Lay the workspace out without the FFN intermediate (moeca_workspace_bytes
// shrinks by layer_mid_bytes); layer_set_mid then gives its device address,
// after every moeca_bind_workspace.  Layers that never step concurrently
// (the blocks of a stack) share one intermediate.
void layer_keep_mid_outside(moeca_layer* L);
void layer_set_mid(moeca_layer* L, void* mid);
const Buffers& layer_buffers(const moeca_layer* L);

// ---- DiT block kernels (block.hip, ffn.hip) -----------------------------
constexpr int kFreqDim = 256;    // timestep embedding width
constexpr int kMaxWidth = 2048;  // largest block width d
constexpr int kProjTM = 128;     // projection GEMM tile: rows
constexpr int kProjTN = 256;     // and output columns

// Shared per-step activations of a block stack (device).
struct BlockBufs {
  int B;
  float* x;        // [T][d] residual stream (the caller's)
  float* x1;       // [T][d] this block's x1 (one of two buffers, alternating by block)
  float* x1b;      // [T][d] the other buffer
  const float* x1p;  // [T][d] the previous block's x1 in a multi-block run
  uint16_t* h;     // [T][d] attention input
  uint16_t* u;     // [T][d] MoE routing input
  uint16_t* u2;    // [T][d] rebuilt MoE input of synchronised tokens
  uint16_t* q;     // [T][d]
  uint16_t* kv;    // [T][2d]
  uint16_t* o;     // [T][d]
  uint16_t* y;     // [T][d]
  int32_t* slist;  // [T] synchronised tokens by sample
  int32_t* soff;   // [B+1]
  int32_t* ident;  // [T] identity row list
  int32_t* tab;    // [8] projection row offsets and tile counts (see launch_slist)
};

// dst[list[r]] = bf16(A[list[r]] . W^T + bias) for r < off[1]: one group of
// listed rows (tables off[2], tiles[2] on the device), K inputs, Nout outputs.
// blocks_per_xcd > 0 gives the persistent grid that many blocks per XCD
// instead of one per CU (the rest of the CUs stay free for kernels on another
// stream that run beside it).
hipError_t launch_proj(const void* A, const void* W, const float* bias, const int32_t* off,
                       const int32_t* tiles, const int32_t* list, int K, int Nout, void* dst,
                       hipStream_t st, int blocks_per_xcd = 0);
// CUs per XCD (the device's CU count over 8).
int cus_per_xcd();
hipError_t launch_sinusoid(const float* t_values, int B, double* e, hipStream_t st);
hipError_t launch_silu(const float* in, int n, double* out, hipStream_t st);
// Up to kGemvBatch matrices of one shape for one GEMV launch (by value).
constexpr int kGemvBatch = 32;
struct GemvBatch {
  const uint16_t* W[kGemvBatch];
  const float* bias[kGemvBatch];
  float* out[kGemvBatch];
};
// for each matrix m < n_mats: v[b][r] = W_m[r] . in[b] + bias_m[r]
// (+ table[labels[b]][r]) in fp64; out_m = fp32(v), or, with out64 set
// (one matrix), out64 = silu(v).  K a multiple of 32, at most kMaxWidth
// (hipErrorInvalidValue otherwise)
hipError_t launch_gemv(const double* in, int B, int K, const GemvBatch& mats, int n_mats,
                       int Nout, const void* table, const int32_t* labels, int n_classes,
                       double* out64, hipStream_t st);
// every token: [x = x1p + g_m(prev) y, stored on full steps;] h = LN(x) mod_a;
// [cached: x1 = x + g_a a, u = LN(x1) mod_m]
hipError_t launch_ln_attn(const BlockBufs& k, int T, int N, int d, const float* mod,
                          const float* mod_prev, const uint16_t* a, bool cached, hipStream_t st);
// listed tokens (slist, count soff[B]): [x = x1p + g_m(prev) y when mod_prev
// is set;] x1 = x + g_a a, u_out = LN(x1) mod_m (routing: u_out is a routing
// input and takes the decision-path arithmetic)
hipError_t launch_ln_mlp(const BlockBufs& k, int T, int N, int d, const float* mod,
                         const float* mod_prev, const uint16_t* a, uint16_t* u_out, bool routing,
                         hipStream_t st);
// every token: x = x1 + g_m y
hipError_t launch_ln_final(const BlockBufs& k, int T, int N, int d, const float* mod,
                           hipStream_t st);
// token lists from the sync flags (sync == NULL: every token) and the tables
hipError_t launch_slist(const BlockBufs& k, const uint8_t* sync, int N, int d, hipStream_t st);
hipError_t launch_attention(const BlockBufs& k, int N, int H, int dh, hipStream_t st);

}  // namespace moeca
