/*
 * moeca.h - branch-cached DiT-MoE layer step on AMD Instinct MI355X (gfx950).
 *
 * MoECa (Sec. 4) caches, per token i, the outputs of its k routed expert
 * branches C_i = {(e_q, w_q, h_q)} and the token's attention-path feature
 * a_i (Sec. 4.1).  At every denoising step the router runs (Sec. 4.1); the
 * current branches are matched to the cached ones and scored (Sec. 4.2);
 * only the branches in the recomputation set R_i go through their expert
 * FFN; the layer output combines recomputed and cached features with the
 * current gate weights (Sec. 4.1, output eq.); the cache and, for tokens with
 * a recomputed branch, the attention feature are refreshed in the same step
 * (Sec. 4.1, synchronised update).  Thresholds adapt per expert from an EMA
 * of its spatial activation and that statistic's entropy (Sec. 4.3).
 *
 * Conventions for every call below
 *  - Pointers named "device" point to memory on the current HIP device; the
 *    caller allocates and frees them and keeps them alive while the layer
 *    uses them.  The library never allocates device memory.
 *  - Activations and weights are bf16 (IEEE binary16-brain, stored as
 *    uint16) or fp32, as the policy's dtype says; gate weights, scores and
 *    statistics are fp32.  All arrays are dense, row-major, no padding.
 *  - "stream" is a hipStream_t passed as void* (NULL = the null stream).
 *  - Functions return MOECA_OK (0) or a negative error code and never throw;
 *    moeca_last_error() then describes the failure (thread-local string).
 *  - One host thread at a time per handle.  Handles are independent.
 */
#ifndef MOECA_H
#define MOECA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- error codes ------------------------------------------------------- */
#define MOECA_OK 0
#define MOECA_E_INVAL (-1) /* bad argument: NULL, size, range                */
#define MOECA_E_STATE (-2) /* weights or workspace not bound yet             */
#define MOECA_E_HIP (-3)   /* a HIP launch or copy reported an error         */

/* ---- policy ------------------------------------------------------------ */
enum {
  MOECA_MODE_FULL = 0,      /* uncached routed MoE layer (Sec. 2.3 MoE eq.);
                               the full-recompute comparator; no cache state */
  MOECA_MODE_THRESHOLD = 1, /* Sec. 4.2: recompute iff unmatched or s > tau  */
  MOECA_MODE_RATIO = 2      /* per sample: all unmatched branches plus the
                               best matched ones by margin s - tau, up to
                               K_b = floor(ratio * N * k + 0.5) branches     */
};
enum { MOECA_DTYPE_BF16 = 0, MOECA_DTYPE_FP32 = 1 };
enum {
  MOECA_ACT_GELU_TANH = 0, /* act(z) = 0.5 z (1 + tanh(sqrt(2/pi)(z + 0.044715 z^3)))   */
  MOECA_ACT_GELU_ERF = 1,  /* act(z) = 0.5 z (1 + erf(z / sqrt 2))                      */
  MOECA_ACT_SWIGLU = 2     /* gated expert: W_up has 2 d_ff rows, gate and up
                              interleaved (row 2j is gate j, row 2j+1 up j), and
                              the hidden value j is silu(gate_j) * up_j with
                              silu(z) = z / (1 + exp(-z)); the product is rounded
                              once to the activation dtype                     */
};

typedef struct moeca_policy {
  int32_t mode;          /* MOECA_MODE_*                                      */
  float ratio;           /* refresh ratio rho in [0, 1] (RATIO mode)          */
  float tau0;            /* base threshold tau_0 (Sec. 4.3), > 0; 0.80        */
  float alpha;           /* adaptation strength alpha in [0, 1); 0.6          */
  float beta;            /* EMA decay beta in [0, 1); 0.65                     */
  float lambda1;         /* weight of the drift term Delta (Sec. 4.2); 1.0    */
  float lambda2;         /* weight of the contribution term o (Sec. 4.2); 1.0 */
  int32_t refresh_cycle; /* forced full step when t % cycle == 0; 0 = never;
                            4 (Sec. 5.1)                                      */
  int32_t norm_topk;     /* 1: gate = softmax renormalised over the top-k     */
  int32_t act;           /* MOECA_ACT_*                                       */
  int32_t dtype;         /* MOECA_DTYPE_*                                     */
  int32_t batch;         /* B, samples per step, >= 1                         */
  int32_t tokens;        /* N, tokens per sample, >= 1                         */
  int32_t n_shared;      /* S, always-on shared experts (Sec. 2.3, shared-expert
                            MoE eq.), 0..8; they have the routed experts' shape
                            and activation, no gate, run on every token at
                            every step and are never cached                   */
  float lambda0;         /* weight of the routing weight w in the score
                            s = lambda0 w + lambda1 Delta + lambda2 o; 1.0 is
                            the score eq. of Sec. 4.2, 0 drops w (the
                            score-signal ablation of Sec. 5)                   */
} moeca_policy;

/* Fill *p with the paper's settings: THRESHOLD mode, tau0 0.80, alpha 0.6,
 * beta 0.65 (Sec. 5.4, Tab. 4), refresh cycle 4 (Sec. 5.1), lambda0 = 1,
 * lambda1 = lambda2 = 1 (not reported by the paper), ratio 0.3, bf16, tanh GELU,
 * renormalised top-k, batch 1, tokens 1, no shared experts.  NULL is
 * ignored. */
void moeca_policy_default(moeca_policy* p);

/* ---- layer handle ------------------------------------------------------ */
typedef struct moeca_layer moeca_layer;

/* Create a layer of width d, E routed experts, top-k routing and expert
 * hidden width d_ff (FFN_e(x) = W_down[e] act(W_up[e] x), Sec. 2.3).
 * Host only; the policy is copied.  Limits: 1 <= k <= min(E, 8), E <= 64,
 * 0 <= n_shared <= 8, d and d_ff multiples of 64, d <= 16384, d_ff <= 65536
 * (32768 with MOECA_ACT_SWIGLU), B*N*(k + n_shared) < 2^31.
 * Returns NULL on a bad argument (moeca_last_error() says which). */
moeca_layer* moeca_layer_create(int d, int E, int k, int d_ff, const moeca_policy* policy);

/* Release the handle.  Never frees caller memory.  NULL is a no-op. */
void moeca_layer_destroy(moeca_layer* layer);

/* Description of the last error on this thread ("" if none). */
const char* moeca_last_error(void);

/* Bind the weights (device, policy dtype, not copied):
 *   W_r    [E][d]        router (Sec. 4.1: B_i^t is its top-k)
 *   b_r    [E] fp32      optional router bias added to the logits, or NULL
 *   W_up   [E][U][d]     expert up-projections (out x in); U = d_ff, or
 *                        2 d_ff with MOECA_ACT_SWIGLU (gate/up interleaved)
 *   W_down [E][d][d_ff]  expert down-projections (out x in)
 * Host only.  MOECA_E_INVAL if a required pointer is NULL or a weight
 * pointer is not 16-byte aligned (the bias 4-byte). */
int moeca_layer_set_weights(moeca_layer* layer, const void* W_r, const float* b_r,
                            const void* W_up, const void* W_down);

/* Bind the shared experts' weights (Sec. 2.3, shared-expert MoE eq.;
 * device, policy dtype, not copied), required when n_shared > 0:
 *   W_up_s   [S][U][d]     up-projections, U as for W_up
 *   W_down_s [S][d][d_ff]  down-projections
 * Their outputs are added to every token's output without a gate.  Host
 * only.  MOECA_E_INVAL if the layer has no shared experts, a pointer is
 * NULL or not 16-byte aligned. */
int moeca_layer_set_shared(moeca_layer* layer, const void* W_up_s, const void* W_down_s);

/* Bytes of device workspace the layer needs: the branch cache (ids, gate
 * weights, norms and rows of B*N*k branches), the EMA statistic [B][E][N],
 * and per-step scratch (routing, scores, masks, expert lists, the FFN
 * intermediate, the shared experts' outputs).  0 if layer is NULL. */
size_t moeca_workspace_bytes(const moeca_layer* layer);

/* Bind caller-owned device memory of at least moeca_workspace_bytes() bytes,
 * 256-byte aligned.  Binding invalidates the cache: the next step is a full
 * step, and the statistic must be cleared with moeca_cache_reset() before
 * it (an unreset workspace holds undefined values).  MOECA_E_INVAL on NULL,
 * misalignment or a short buffer. */
int moeca_bind_workspace(moeca_layer* layer, void* dev, size_t bytes);

/* Optional attention path (Sec. 4.1, synchronised update).  attn_in and
 * attn_cache are device [B][N][d] in the policy dtype.  After each step,
 * attn_cache row i equals attn_in row i if token i had at least one
 * recomputed branch (every token on full steps), and is unchanged
 * otherwise.  attn_in is read when the step runs, so the caller may write
 * each step's features into the same buffer.  Both NULL unbinds; one NULL,
 * or a pointer that is not 16-byte aligned, is MOECA_E_INVAL. */
int moeca_bind_attention(moeca_layer* layer, const void* attn_in, void* attn_cache);

/* One layer step at sampling step t (0-based).
 *   x_t [B][N][d]  device, policy dtype: the MoE layer input u of Sec. 2.3
 *   out [B][N][d]  device, policy dtype: y_i of Sec. 4.1 (the routed sum,
 *                  plus the shared experts' outputs when n_shared > 0,
 *                  without the residual, which the caller adds)
 * The step is a full step when the cache is invalid, in FULL mode, or when
 * refresh_cycle > 0 and t % refresh_cycle == 0 (Sec. 4.1 / Sec. 5.1);
 * otherwise a cache step.  Enqueues work on the stream and returns without
 * waiting; it neither allocates nor synchronises.  Kernel faults surface at
 * the caller's next synchronisation.  x_t and out must not overlap the
 * workspace; both must be 16-byte aligned (else MOECA_E_INVAL).
 * MOECA_E_STATE if the weights, the workspace or (n_shared > 0) the shared
 * weights are unbound. */
int moeca_step(moeca_layer* layer, const void* x_t, int t, void* out, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the
 * uncached routed MoE layer, i.e. what moeca_step computes for a
 * MOECA_MODE_FULL layer (router, top-k gates, every branch through its
 * expert FFN, combine), over the first `samples` samples of N tokens.
 *   x   [samples][N][d]  device, policy dtype
 *   out [samples][N][d]  device, policy dtype
 * Needs only the bound weights (and shared weights when n_shared > 0): no
 * workspace, whatever the layer's mode, and the layer's cache and statistic
 * are neither read nor written.  Every intermediate lives in one
 * library-owned device array of 64 MiB per GPU, held from the library's
 * first use on that GPU until the process ends; this call allocates no
 * device or host memory and never synchronises.  A call whose intermediates
 * exceed that array (about samples * N * (k + n_shared) * (d + d_ff) * 2
 * bytes in bf16) is MOECA_E_INVAL with the sizes in moeca_last_error().
 * Every call on one GPU shares its array: calls that overlap on one GPU
 * (other streams, other threads) race and must be ordered by the caller.
 * MOECA_E_INVAL: NULL layer, x or out, unaligned x or out (16 bytes),
 * samples outside [1, B]; MOECA_E_STATE: weights unbound; MOECA_E_HIP: the
 * array's address could not be obtained or a launch failed. */
int moeca_forward_noalloc(const moeca_layer* layer, const void* x, int samples, void* out,
                          void* stream);

/* Enqueue a cache reset on the stream: every cached branch becomes empty,
 * the EMA statistic becomes zero, and the next step is a full step. */
int moeca_cache_reset(moeca_layer* layer, void* stream);

/* ---- statistics of the last step -------------------------------------- */
typedef struct moeca_stats {
  int64_t n_branches;      /* B * N * k                                        */
  int64_t n_recompute;     /* |R| summed over tokens                           */
  int64_t n_unmatched;     /* branches whose expert was not cached (0 on full) */
  int64_t n_matched;       /* branches matched to a cached slot (0 on full)    */
  int64_t n_reused;        /* matched and not recomputed                       */
  int64_t n_sync;          /* tokens whose attention feature was refreshed     */
  int32_t full_step;       /* 1 if the last step was a full step               */
  int32_t nonfinite;       /* 1 if a router logit was NaN or infinite          */
  double reuse_over_match; /* n_reused / n_matched (Sec. 5.4, Fig. 8); 0 if none */
  int32_t expert_count[64];/* recomputed branches per expert                  */
  int32_t ffn_plan;        /* tiling of the last step's expert FFN: 0 the
                              128 x 256 tiles, 1 the weight-streaming tiles
                              (few rows per expert), 2 the expert-wide
                              up-projection tiles (a few hundred rows per
                              expert) with the 128 x 256 down projection     */
} moeca_stats;

/* Copy the last step's statistics to *out.  Synchronises the stream. */
int moeca_get_stats(moeca_layer* layer, moeca_stats* out, void* stream);

/* ---- inspection (tests and benchmarks) --------------------------------- */
enum {
  MOECA_BUF_E_C = 0,    /* int32 [B*N*k]    cached expert id, -1 = empty      */
  MOECA_BUF_W_C = 1,    /* fp32  [B*N*k]    cached gate weight w^{t0}         */
  MOECA_BUF_N_C = 2,    /* fp32  [B*N*k]    norm of the cached row ||h^{t0}|| */
  MOECA_BUF_H_C = 3,    /* act   [B*N*k][d] cached branch outputs h^{t0}      */
  MOECA_BUF_STAT = 4,   /* fp32  [B][E][N]  EMA statistic C_{e,i}             */
  MOECA_BUF_LOGITS = 5, /* fp32  [B*N][E]   router logits of the last step    */
  MOECA_BUF_E_T = 6,    /* int32 [B*N*k]    current experts e_{i,p}           */
  MOECA_BUF_W_T = 7,    /* fp32  [B*N*k]    current gate weights w_{i,p}      */
  MOECA_BUF_HBAR = 8,   /* fp32  [B][E]     normalised entropy                */
  MOECA_BUF_TAU = 9,    /* fp32  [B][E]     thresholds tau_e                  */
  MOECA_BUF_MARGIN = 10,/* fp32  [B*N*k]    s - tau_e (+inf if unmatched)     */
  MOECA_BUF_Q = 11,     /* int32 [B*N*k]    matched slot q(p), -1 unmatched   */
  MOECA_BUF_MASK = 12,  /* uint8 [B*N*k]    1 = recomputed (p in R_i)         */
  MOECA_BUF_SIGMA = 13, /* int32 [B*N*k]    cache slot of branch p after step */
  MOECA_BUF_SYNC = 14,  /* uint8 [B*N]      S_i = [R_i non-empty]             */
  MOECA_BUF_OFF = 15,   /* int32 [E+1]      per-expert offsets into LIST (the
                           workspace keeps S more entries after it: the shared
                           experts' row ranges in the FFN intermediate)      */
  MOECA_BUF_LIST = 16,  /* int32 [B*N*k]    recomputed flat branch ids
                           f = (b*N + i)*k + p, grouped by expert, ascending  */
  MOECA_BUF_POS = 17,   /* int32 [B*N*k]    index of f in LIST, -1 if reused  */
  MOECA_BUF_COUNT = 18
};

/* Byte offset and size of an internal buffer inside the bound workspace, for
 * tests that read or overwrite layer state between steps (all prior work on
 * the stream must be complete).  Buffers 5-17 hold the last step's
 * decisions; their contents are unspecified before the first step.
 * MOECA_E_INVAL for an unknown id. */
int moeca_debug_buffer(const moeca_layer* layer, int which, size_t* offset, size_t* bytes);

/* Declare the cache valid (1) or invalid (0) after a test has written the
 * state buffers 0-4 directly.  Host only. */
int moeca_debug_set_valid(moeca_layer* layer, int valid);

/* ---- per-stage timing --------------------------------------------------- */
enum {
  MOECA_STAGE_ROUTER = 0,  /* router logits, top-k, gate; EMA statistic update */
  MOECA_STAGE_STAT = 1,    /* reserved: the entropy of the statistic and the
                              thresholds are computed at the start of the
                              SELECT stage's kernel; this stage launches
                              nothing and reads as 0                          */
  MOECA_STAGE_SELECT = 2,  /* matching, branch scores, recomputation set,
                              slots, sync mask                                */
  MOECA_STAGE_LISTS = 3,   /* per-expert compaction                            */
  MOECA_STAGE_FFN_UP = 4,  /* gathered up-projection + activation (routed and
                              shared experts in one grouped launch)           */
  MOECA_STAGE_FFN_DOWN = 5,/* down-projection into the cache rows (shared
                              experts: into their own output rows)            */
  MOECA_STAGE_COMBINE = 6, /* combine, norms, cache metadata, attention path   */
  MOECA_STAGE_COUNT = 7
};

/* Enable (1) or disable (0) HIP-event timing of each stage of each step on
 * the step's stream (at most 512 steps are kept).  Enabling creates the
 * events, disabling destroys them. */
int moeca_set_timing(moeca_layer* layer, int enable);

/* Sum of the per-stage times, in ms, over the steps recorded since timing
 * was enabled or last read, into ms[0..n-1] (n <= MOECA_STAGE_COUNT); a
 * stage skipped on a step contributes 0.  *steps receives the number of
 * steps.  Synchronises the recorded events and clears the record. */
int moeca_get_timing(moeca_layer* layer, double* ms, int n, int* steps);

/* ---- DiT-MoE block stack ----------------------------------------------
 * L DiT-MoE blocks (Sec. 2.1, composition eq. and residual form; the MoE FFN
 * of Sec. 2.3) under MoECa (Sec. 4.1).  Block l computes, per token,
 *   x1 = x  + g_a * a,  a = W_o Attn(h) + b_o,  h = LN(x)  * (1 + sc_a) + sh_a
 *   x' = x1 + g_m * y,  y = MoE(u),             u = LN(x1) * (1 + sc_m) + sh_m
 * where (sh_a, sc_a, g_a, sh_m, sc_m, g_m) are the six d-vectors of
 * W_ada SiLU(c) + b_ada (AdaLN conditioned on c, one c per sample), LN has
 * no affine parameters (eps 1e-6), and Attn is multi-head self-attention
 * over the tokens of a sample: [q k v] = W_qkv h + b_qkv, head j on columns
 * j d_h .. (j+1) d_h - 1, softmax(q k^T / sqrt(d_h)) v per head.
 *
 * Every block keeps the attention feature a_i of each token (Sec. 4.1) and
 * a MoE layer with its branch cache.  A full step runs the block as written
 * and refills both.  A cache step routes on u built from the cached a_i,
 * decides R_i and S_i = [R_i non-empty] (Sec. 4.2-4.3), recomputes the
 * attention feature of the tokens in S only (their queries against the keys
 * and values of every token of the sample at this step), rebuilds their x1
 * and u, and recomputes the branches in R_i on the rebuilt u (Sec. 4.1,
 * synchronised update); other tokens reuse a_i and their branches.  Full vs
 * cache step follows the policy as for moeca_step.
 *
 * Precision: x, x1, x' and the AdaLN vectors fp32; h, q, k, v, the
 * attention output, a, u and y bf16, rounded where produced; fp32
 * accumulation.  Limits: bf16 policy, n_shared = 0, d a multiple of 64 and
 * at most 2048, d_h = d / heads a multiple of 8 and at most 96, and the MoE
 * layer's limits. */
typedef struct moeca_stack moeca_stack;

/* Weights of one block: device, bf16 matrices (row-major, out x in) and
 * fp32 biases, not copied; matrices 16-byte aligned, biases 4-byte. */
typedef struct moeca_block_weights {
  const void* W_ada;  /* [6d][d] AdaLN rows: sh_a, sc_a, g_a, sh_m, sc_m, g_m */
  const float* b_ada; /* [6d]                                                  */
  const void* W_qkv;  /* [3d][d] rows q, then k, then v                         */
  const float* b_qkv; /* [3d]                                                  */
  const void* W_o;    /* [d][d] output projection                               */
  const float* b_o;   /* [d]                                                   */
  const void* W_r;    /* [E][d] router                                          */
  const float* b_r;   /* [E] router bias, or NULL                               */
  const void* W_up;   /* [E][U][d] as in moeca_layer_set_weights               */
  const void* W_down; /* [E][d][d_ff]                                          */
} moeca_block_weights;

/* Create a stack of n_blocks (1 to 4096) blocks of width d with `heads`
 * attention heads and the MoE layer (E, k, d_ff, policy) of
 * moeca_layer_create in each.  Host only; NULL on a bad argument (the
 * limits above, the layer's, or a non-bf16 policy or n_shared > 0). */
moeca_stack* moeca_stack_create(int n_blocks, int d, int heads, int E, int k, int d_ff,
                                const moeca_policy* policy);

/* Release the stack and its layers.  Never frees caller memory. */
void moeca_stack_destroy(moeca_stack* stack);

/* Bind block l's weights (0 <= l < n_blocks).  MOECA_E_INVAL on a NULL
 * required pointer (all but b_r) or misalignment. */
int moeca_stack_set_block(moeca_stack* stack, int l, const moeca_block_weights* w);

/* Device workspace: per block the cached attention features [B*N][d] and
 * the MoE layer's workspace; shared per-step activations (x1, h, u, the
 * rebuilt u, q, k/v, attention output, y), the AdaLN vectors of every block
 * and the token lists.  0 if stack is NULL. */
size_t moeca_stack_workspace_bytes(const moeca_stack* stack);

/* Bind caller-owned device memory (256-byte aligned, at least
 * moeca_stack_workspace_bytes()).  Invalidates every cache; clear them with
 * moeca_stack_cache_reset() before the first step. */
int moeca_stack_bind_workspace(moeca_stack* stack, void* dev, size_t bytes);

/* One step of blocks first .. first + count - 1 at sampling step t.
 *   x [B][N][d] fp32, device, in/out: the input of block `first`; on return
 *     the output of the last block run.  The stack also uses it for the
 *     residual stream between blocks.
 *   c [B][d] fp32, device: the conditioning vector of each sample.
 * Running all blocks is one model evaluation; a range lets a caller run
 * the stack in parts.  The step kind (full or cache) is decided per block
 * as in moeca_step.  Asynchronous on the stream; no device allocation.
 * Each block's k/v projection runs on a second stream owned by the stack (default priority, made on the first call that is not
 * inside a graph capture, on the current device), forked from `stream`
 * after the block's LayerNorm and joined back into it before the block's
 * attention: work enqueued on `stream` after the call sees the whole step,
 * and a graph captured from `stream` contains the fork.  Until that stream
 * exists, or on another device, everything runs on `stream`.
 * MOECA_E_INVAL on a bad range, NULL or misaligned pointers; MOECA_E_STATE
 * if a block's weights or the workspace are unbound. */
int moeca_stack_step_blocks(moeca_stack* stack, float* x, const float* c, int t, int first,
                            int count, void* stream);

/* moeca_stack_step_blocks over every block. */
int moeca_stack_step(moeca_stack* stack, float* x, const float* c, int t, void* stream);

/* Enqueue a reset of every block's caches; the next step is a full step. */
int moeca_stack_cache_reset(moeca_stack* stack, void* stream);

/* The MoE layer of block l (statistics, timing, inspection), owned by the
 * stack; NULL on a bad index. */
moeca_layer* moeca_stack_layer(moeca_stack* stack, int l);

/* Timestep and class conditioning (the DiT embedder): per sample
 *   c = W2 SiLU(W1 e(t) + b1) + b2 + table[label],
 * e(t) = [cos(t f_j), sin(t f_j)], f_j = 10^(-4 j / 128), j = 0..127.
 *   t_values [B] fp32 and labels [B] int32 (NULL: no class row) device;
 *   W1 [d][256], W2 [d][d], table [n_classes][d] bf16; b1, b2 [d] fp32;
 *   c [B][d] fp32 out.
 * A label outside [0, n_classes) adds no class row.  Uses the stack's
 * workspace for its intermediate; asynchronous. */
int moeca_stack_embed(moeca_stack* stack, const float* t_values, const int32_t* labels,
                      const void* W1, const float* b1, const void* W2, const float* b2,
                      const void* table, int n_classes, float* c, void* stream);

/* Shared activation buffers of the stack (values of the last block run). */
enum {
  MOECA_SBUF_MOD = 0,   /* fp32  [L][B][6][d] AdaLN vectors of every block     */
  MOECA_SBUF_H = 1,     /* bf16  [B*N][d]  attention input h                   */
  MOECA_SBUF_U = 2,     /* bf16  [B*N][d]  MoE routing input u                 */
  MOECA_SBUF_U2 = 3,    /* bf16  [B*N][d]  rebuilt u of the synchronised tokens
                           (the FFN input of a cache step; the same buffer as
                           U on a full step)                                  */
  MOECA_SBUF_Q = 4,     /* bf16  [B*N][d]  queries (rows of synchronised tokens) */
  MOECA_SBUF_KV = 5,    /* bf16  [B*N][2d] keys, then values                   */
  MOECA_SBUF_O = 6,     /* bf16  [B*N][d]  attention output before W_o (rows of
                           synchronised tokens)                               */
  MOECA_SBUF_X1 = 7,    /* fp32  [B*N][d]  x1                                  */
  MOECA_SBUF_Y = 8,     /* bf16  [B*N][d]  MoE output y                        */
  MOECA_SBUF_SLIST = 9, /* int32 [B*N]     synchronised tokens (flat ids
                           b*N + i), by sample, ascending                     */
  MOECA_SBUF_SOFF = 10, /* int32 [B+1]     start of each sample in SLIST       */
  MOECA_SBUF_A = 11,    /* bf16  [B*N][d]  cached attention feature a of block l */
  MOECA_SBUF_LAYER = 12,/* the MoE layer workspace of block l: the offsets of
                           moeca_debug_buffer on moeca_stack_layer(l) are
                           relative to its start                              */
  MOECA_SBUF_COUNT = 13
};

/* Byte offset and size of a stack buffer inside the bound workspace (l is
 * used by the per-block ids A and LAYER only).  MOECA_E_INVAL for an unknown
 * id or block. */
int moeca_stack_debug_buffer(const moeca_stack* stack, int which, int l, size_t* offset,
                             size_t* bytes);

#ifdef __cplusplus
}
#endif
#endif /* MOECA_H */
