// Kernels of the DiT-MoE block around the MoE layer (Sec. 2.1 block form):
// conditioning (timestep embedding, AdaLN vectors), LayerNorm with AdaLN
// modulation and the gated residuals, the list of synchronised tokens
// (Sec. 4.1, synchronised update) and multi-head self-attention of those
// tokens' queries over every token of the sample.  The q/k/v and output
// projections are the grouped GEMM's projection instantiation (ffn.hip).
#include <algorithm>
#include <cmath>

#include "common.h"
#include "internal.h"

namespace moeca {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_t;
typedef __attribute__((ext_vector_type(2))) unsigned int u32x2_t;
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
typedef __attribute__((ext_vector_type(4))) short v4i16_t;
typedef __attribute__((ext_vector_type(8))) short v8i16_t;

__device__ __forceinline__ uint32_t pack2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

__device__ __forceinline__ double silu64(double z) { return z / (1.0 + exp(-z)); }

// One correct rounding of an fp64 value to bf16 (nearest, ties to even).
// In fp32's normal range the fp64 significand is rounded to 8 bits in
// place (the carry may step the exponent) and the result converts to fp32
// exactly.  Elsewhere (zero, subnormal, overflow, inf, NaN): rounding to
// odd into fp32 first (truncate, then set the last bit if anything was
// dropped) keeps the second rounding from landing on a false tie.
__device__ __forceinline__ uint32_t f64_to_bf16(double v) {
  const double av = fabs(v);
  if (av >= 0x1p-126 && av < 0x1p127) {
    uint64_t b = static_cast<uint64_t>(__double_as_longlong(v));
    b += ((uint64_t(1) << 44) - 1) + ((b >> 45) & 1);
    b &= ~((uint64_t(1) << 45) - 1);
    return __float_as_uint(static_cast<float>(__longlong_as_double(static_cast<long long>(b)))) >>
           16;
  }
  uint32_t u = __float_as_uint(__double2float_rz(v));
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
  if (static_cast<double>(__uint_as_float(u)) != v && (u & 0x7fffffffu) < 0x7f800000u) u |= 1u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// fp32(x + g f) with one rounding of the exact value (a fused multiply-add;
// g f is exact).  An fp64 evaluation rounded to fp32 gives the same value
// except when its fp64 rounding lands exactly on an fp32 midpoint (about one
// value in 2^29).
__device__ __forceinline__ float gated_add(float x, float g, float f) { return fmaf(g, f, x); }

// ---------------------------------------------------------------------------
// conditioning
// ---------------------------------------------------------------------------
// e[b][j] = cos(t_b f_j) for j < 128, sin(t_b f_{j-128}) after, f_j =
// 10^(-4 j / 128); fp64 throughout.
__global__ void sinusoid_kernel(const float* __restrict__ t_values, int B,
                                double* __restrict__ e) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * kFreqDim) return;
  const int b = i / kFreqDim, j = i % kFreqDim, half = kFreqDim / 2;
  const int jj = j < half ? j : j - half;
  const double f = exp(-log(10000.0) * jj / half);
  const double arg = static_cast<double>(t_values[b]) * f;
  e[i] = j < half ? cos(arg) : sin(arg);
}

__global__ void silu_kernel(const float* __restrict__ in, int n, double* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = silu64(static_cast<double>(in[i]));
}

// v[b][r] = (sum_k W[r][k] in[b][k] + bias[r]) (+ table[labels[b]][r]) in
// fp64, then out = fp32(v), or out64 = silu(v) when out64 is set.  W rows
// are bf16 [Nout][K] (K a multiple of 32, at most kMaxWidth), in fp64
// [B][K].  One launch covers up to kGemvBatch matrices of the same shape
// (every block's AdaLN map at once).
//
// The products run on the fp64 matrix cores (v_mfma_f64_16x16x4f64), which
// here deliver several times the fp64 rate of the vector units: a wave
// takes 16 weight rows (the A operand) against up to kGemvSamples samples
// (the B operand; the other columns of the 16 are zero and discarded).
// Lane l loads 8 consecutive bf16 of weight row l % 16 at columns
// c + 8 (l / 16) of each 32-column block c and feeds them to 8 MFMAs in turn,
// MFMA u taking column c + 8 (l / 16) + u for k-row l / 16 in both operands,
// so that one 16-byte load serves 8 MFMAs, and kGemvDepth such loads are in
// flight per lane.  The samples' inputs are staged in LDS once per block
// (persistent blocks walk the 16-row tiles of all the matrices).  Four
// accumulator chains rotate over the MFMAs and are added in a fixed order
// (eight were slower).  The AdaLN vectors feed the routing input, so they
// take the decision path's arithmetic: an fp64 evaluation with one rounding.
constexpr int kGemvWaves = 8;
constexpr int kGemvSamples = 8;
constexpr int kGemvDepth = 8;  // 32-column blocks of weights in flight per wave

typedef __attribute__((ext_vector_type(4))) double f64x4_g;

__global__ __launch_bounds__(kGemvWaves * kWave) void gemv_kernel(
    const double* __restrict__ in, int B, int K, GemvBatch mats, int n_mats, int Nout,
    const uint16_t* __restrict__ table, const int32_t* __restrict__ labels, int n_classes,
    double* __restrict__ out64) {
  __shared__ __attribute__((aligned(16))) double s_in[kGemvSamples * kMaxWidth];  // 128 KB
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int n = lane & 15, g = lane >> 4;
  const int per_mat = (Nout + 15) / 16;
  const int tiles = per_mat * n_mats;
  const int nblk = K / 32;
  for (int b0 = 0; b0 < B; b0 += kGemvSamples) {
    const int nb = min(kGemvSamples, B - b0);
    __syncthreads();  // every wave is done with the previous samples' inputs
    for (int i = threadIdx.x; i < nb * K; i += kGemvWaves * kWave)
      s_in[i] = in[int64_t(b0) * K + i];
    __syncthreads();
    const bool has_col = n < nb;  // B column n is a staged sample
    const double* __restrict__ xin = s_in + (has_col ? n : 0) * K + 8 * g;
    for (int tt = blockIdx.x + gridDim.x * wv; tt < tiles; tt += gridDim.x * kGemvWaves) {
      const int m = tt / per_mat;
      const int r0 = (tt % per_mat) * 16;
      const uint16_t* __restrict__ wrow =
          mats.W[m] + int64_t(min(r0 + n, Nout - 1)) * K + 8 * g;
      f64x4_g acc[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] = f64x4_g{0.0, 0.0, 0.0, 0.0};
      u32x4_t raw[kGemvDepth];
#pragma unroll
      for (int d0 = 0; d0 < kGemvDepth; ++d0)
        if (d0 < nblk) raw[d0] = *reinterpret_cast<const u32x4_t*>(wrow + 32 * d0);
      for (int c0 = 0; c0 < nblk; c0 += kGemvDepth) {
#pragma unroll
        for (int d0 = 0; d0 < kGemvDepth; ++d0) {
          const int c = c0 + d0;
          if (c < nblk) {
            double wv8[8], xv[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              wv8[2 * e] = __uint_as_float(raw[d0][e] << 16);
              wv8[2 * e + 1] = __uint_as_float(raw[d0][e] & 0xffff0000u);
            }
            // the block kGemvDepth ahead reuses this register set
            if (c + kGemvDepth < nblk)
              raw[d0] = *reinterpret_cast<const u32x4_t*>(wrow + 32 * (c + kGemvDepth));
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
              const double2 t2 = *reinterpret_cast<const double2*>(xin + 32 * c + e);
              xv[e] = has_col ? t2.x : 0.0;
              xv[e + 1] = has_col ? t2.y : 0.0;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u)
              acc[u & 3] = __builtin_amdgcn_mfma_f64_16x16x4f64(wv8[u], xv[u], acc[u & 3], 0, 0, 0);
          }
        }
      }
      // lane l, register r: weight row r0 + 4 r + l / 16, sample l % 16
      const float* __restrict__ bias = mats.bias[m];
      float* __restrict__ out = mats.out[m];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = r0 + 4 * r + g;
        if (has_col && row < Nout) {
          const int b = b0 + n;
          double v = ((acc[0][r] + acc[1][r]) + (acc[2][r] + acc[3][r])) +
                     static_cast<double>(bias[row]);
          if (table != nullptr) {
            const int lab = labels[b];
            if (lab >= 0 && lab < n_classes) v += bf16_to_f32(table[int64_t(lab) * Nout + row]);
          }
          if (out64 != nullptr) out64[int64_t(b) * Nout + row] = silu64(v);
          else out[int64_t(b) * Nout + row] = static_cast<float>(v);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// LayerNorm + AdaLN modulation and the gated residuals, one wave per row
// ---------------------------------------------------------------------------
// d <= kMaxWidth: a lane holds float4 chunks lane + 64 j (j < NC) of the
// row; NC = ceil(d / 256) is a template parameter, so the registers held
// per lane (and the waves a CU keeps in flight) follow the width.
constexpr int kLnWaves = 4;
constexpr int kLnChunks = kMaxWidth / 4 / kWave;  // 8, the most

enum { kLnAttn = 0, kLnMlp = 1, kLnFinal = 2 };

struct LnArgs {
  float* x;                 // [T][d] residual stream (block input)
  float* x1;                // [T][d]
  const uint16_t* y;        // [T][d] MoE output of the previous block
  const uint16_t* a;        // [T][d] attention feature of this block
  uint16_t* h;              // [T][d] attention input
  uint16_t* u;              // [T][d] MoE input
  const float* mod;         // [B][6][d] this block's AdaLN vectors
  const float* mod_prev;    // [B][6][d] the previous block's (pending residual)
  const int32_t* rows;      // kLnMlp: the rows to process
  const int32_t* count;     // kLnMlp: device row count
  int T, N, d;
  int pending;              // x = x1 + g_m(prev) * y first (kLnAttn)
  int cached;               // kLnAttn on a cache step: also x1 and u from a
  int routing;              // kLnMlp: u is the routing input (a full step)
  const float* x1p;         // [T][d] the previous block's x1 (with pending)
};

template <int NC>
__device__ __forceinline__ void ln_stats(const float (&v)[NC][4], int n4, int lane, int d,
                                         double& mean, double& rstd) {
  double s = 0.0;
#pragma unroll
  for (int j = 0; j < NC; ++j)
    if (lane + kWave * j < n4)
#pragma unroll
      for (int e = 0; e < 4; ++e) s += v[j][e];
  const double mu = wave_sum_f64(s) / d;
  double q = 0.0;
#pragma unroll
  for (int j = 0; j < NC; ++j)
    if (lane + kWave * j < n4)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double t = v[j][e] - mu;
        q += t * t;
      }
  const double var = wave_sum_f64(q) / d;
  mean = mu;
  rstd = 1.0 / sqrt(var + 1e-6);
}

// bf16(LN(v) * (1 + scale) + shift) into row `dst` in fp32: the attention
// input (off the decision path)
template <int NC>
__device__ __forceinline__ void ln_store_f32(const float (&v)[NC][4], int n4, int lane,
                                             double mean, double rstd, const float* shift,
                                             const float* scale, uint16_t* dst) {
  const float mf = static_cast<float>(mean), rf = static_cast<float>(rstd);
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const int c = lane + kWave * j;
    if (c < n4) {
      const float4 sh = reinterpret_cast<const float4*>(shift)[c];
      const float4 sc = reinterpret_cast<const float4*>(scale)[c];
      const float z0 = fmaf((v[j][0] - mf) * rf, 1.0f + sc.x, sh.x);
      const float z1 = fmaf((v[j][1] - mf) * rf, 1.0f + sc.y, sh.y);
      const float z2 = fmaf((v[j][2] - mf) * rf, 1.0f + sc.z, sh.z);
      const float z3 = fmaf((v[j][3] - mf) * rf, 1.0f + sc.w, sh.w);
      reinterpret_cast<u32x2_t*>(dst)[c] = u32x2_t{pack2(z0, z1), pack2(z2, z3)};
    }
  }
}

// bf16(LN(v) * (1 + scale) + shift) into row `dst`, in fp64 and rounded
// once: this is the MoE routing input (decision-path arithmetic)
template <int NC>
__device__ __forceinline__ void ln_store(const float (&v)[NC][4], int n4, int lane,
                                         double mean, double rstd, const float* shift,
                                         const float* scale, uint16_t* dst) {
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const int c = lane + kWave * j;
    if (c < n4) {
      const float4 sh = reinterpret_cast<const float4*>(shift)[c];
      const float4 sc = reinterpret_cast<const float4*>(scale)[c];
      const float s4[4] = {sc.x, sc.y, sc.z, sc.w};
      const float h4[4] = {sh.x, sh.y, sh.z, sh.w};
      uint32_t z[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        z[e] = f64_to_bf16((static_cast<double>(v[j][e]) - mean) * rstd *
                               (1.0 + static_cast<double>(s4[e])) +
                           static_cast<double>(h4[e]));
      reinterpret_cast<u32x2_t*>(dst)[c] = u32x2_t{z[0] | (z[1] << 16), z[2] | (z[3] << 16)};
    }
  }
}

template <int MODE, int NC>
__global__ __launch_bounds__(kLnWaves * kWave) void ln_kernel(LnArgs p) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * kLnWaves + (threadIdx.x >> 6);
  int row;
  if constexpr (MODE == kLnMlp) {
    if (r >= *p.count) return;
    row = p.rows[r];
  } else {
    if (r >= p.T) return;
    row = r;
  }
  const int d = p.d, n4 = d / 4;
  const int b = row / p.N;
  const int64_t o = int64_t(row) * d;
  const float* m = p.mod + int64_t(b) * 6 * d;  // sh_a, sc_a, g_a, sh_m, sc_m, g_m
  float v[NC][4];

  if constexpr (MODE == kLnFinal) {
    const float* g = m + 5 * d;
#pragma unroll
    for (int j = 0; j < NC; ++j) {
      const int c = lane + kWave * j;
      if (c < n4) {
        const float4 x1 = reinterpret_cast<const float4*>(p.x1 + o)[c];
        const u32x2_t yy = reinterpret_cast<const u32x2_t*>(p.y + o)[c];
        const float4 gg = reinterpret_cast<const float4*>(g)[c];
        float4 r4;
        r4.x = gated_add(x1.x, gg.x, __uint_as_float(yy[0] << 16));
        r4.y = gated_add(x1.y, gg.y, __uint_as_float(yy[0] & 0xffff0000u));
        r4.z = gated_add(x1.z, gg.z, __uint_as_float(yy[1] << 16));
        r4.w = gated_add(x1.w, gg.w, __uint_as_float(yy[1] & 0xffff0000u));
        reinterpret_cast<float4*>(p.x + o)[c] = r4;
      }
    }
    return;
  }

  // the row's x: the block input, or the previous block's x1 + g_m y.  A
  // cache step does not store that x: LN2 rebuilds it for the listed
  // tokens from the same operands (a full step stores it for LN2)
  if (p.pending) {
    const float* gp = p.mod_prev + int64_t(b) * 6 * d + 5 * d;
#pragma unroll
    for (int j = 0; j < NC; ++j) {
      const int c = lane + kWave * j;
      if (c < n4) {
        const float4 x1 = reinterpret_cast<const float4*>(p.x1p + o)[c];
        const u32x2_t yy = reinterpret_cast<const u32x2_t*>(p.y + o)[c];
        const float4 gg = reinterpret_cast<const float4*>(gp)[c];
        v[j][0] = gated_add(x1.x, gg.x, __uint_as_float(yy[0] << 16));
        v[j][1] = gated_add(x1.y, gg.y, __uint_as_float(yy[0] & 0xffff0000u));
        v[j][2] = gated_add(x1.z, gg.z, __uint_as_float(yy[1] << 16));
        v[j][3] = gated_add(x1.w, gg.w, __uint_as_float(yy[1] & 0xffff0000u));
        if (MODE == kLnAttn && !p.cached)
          reinterpret_cast<float4*>(p.x + o)[c] = float4{v[j][0], v[j][1], v[j][2], v[j][3]};
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < NC; ++j) {
      const int c = lane + kWave * j;
      if (c < n4) {
        const float4 xx = reinterpret_cast<const float4*>(p.x + o)[c];
        v[j][0] = xx.x;
        v[j][1] = xx.y;
        v[j][2] = xx.z;
        v[j][3] = xx.w;
      }
    }
  }
  // the attention feature, requested together with x (it is used after the
  // first LayerNorm)
  const bool with_a = MODE == kLnMlp || p.cached;
  u32x2_t av[NC];
  if (with_a) {
#pragma unroll
    for (int j = 0; j < NC; ++j) {
      const int c = lane + kWave * j;
      if (c < n4) av[j] = reinterpret_cast<const u32x2_t*>(p.a + o)[c];
    }
  }
  double mean, rstd;
  if (MODE == kLnAttn) {
    ln_stats(v, n4, lane, d, mean, rstd);
    ln_store_f32(v, n4, lane, mean, rstd, m, m + d, p.h + o);
    if (!p.cached) return;
  }
  // x1 = x + g_a * a, then the MoE input from LN(x1)
  const float* ga = m + 2 * d;
#pragma unroll
  for (int j = 0; j < NC; ++j) {
    const int c = lane + kWave * j;
    if (c < n4) {
      const u32x2_t aa = av[j];
      const float4 gg = reinterpret_cast<const float4*>(ga)[c];
      v[j][0] = gated_add(v[j][0], gg.x, __uint_as_float(aa[0] << 16));
      v[j][1] = gated_add(v[j][1], gg.y, __uint_as_float(aa[0] & 0xffff0000u));
      v[j][2] = gated_add(v[j][2], gg.z, __uint_as_float(aa[1] << 16));
      v[j][3] = gated_add(v[j][3], gg.w, __uint_as_float(aa[1] & 0xffff0000u));
      reinterpret_cast<float4*>(p.x1 + o)[c] = float4{v[j][0], v[j][1], v[j][2], v[j][3]};
    }
  }
  ln_stats(v, n4, lane, d, mean, rstd);
  // a routing input (LN1 of a cache step, LN2 of a full step) takes the
  // decision-path arithmetic, so that the same input routes the same way on
  // either kind of step; the rebuilt FFN input of a cache step takes fp32
  if (MODE == kLnAttn || p.routing)
    ln_store(v, n4, lane, mean, rstd, m + 3 * d, m + 4 * d, p.u + o);
  else
    ln_store_f32(v, n4, lane, mean, rstd, m + 3 * d, m + 4 * d, p.u + o);
}

// ---------------------------------------------------------------------------
// synchronised tokens: per-sample ascending lists and the projection tables
// ---------------------------------------------------------------------------
// One 1024-thread block per sample.  all: every token (full steps); else
// sync[t] != 0.  Block b counts the flags of samples 0 .. b-1 (its base in
// the list), then lists its own tokens in ascending order.  Writes slist
// (flat token ids, by sample), soff[B + 1] and, from the last block,
// tab[0..3] = {0, nS, 0, tiles of nS rows x ntn_q} for the projections
// (128-row tiles); the full-list call also writes ident[t] = t and
// tab[4..7] = {0, T, 0, tiles of T rows x ntn_kv}.
constexpr int kListThreads = 1024;

__global__ __launch_bounds__(kListThreads) void slist_kernel(
    const uint8_t* __restrict__ sync, int all, int B, int N, int ntn_q, int ntn_kv,
    int32_t* __restrict__ slist, int32_t* __restrict__ soff, int32_t* __restrict__ ident,
    int32_t* __restrict__ tab) {
  __shared__ int s_wave[kListThreads / kWave];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int b = blockIdx.x;
  const int T = B * N;
  // the whole-batch list and table entries never change: written by the
  // full-list call only, so that a token-list call of a cache step writes
  // nothing that a k/v projection running beside it reads
  if (all)
    for (int i = tid; i < N; i += kListThreads) ident[b * N + i] = b * N + i;
  // base: the listed tokens of the samples before this one
  int base = 0;
  if (all) {
    base = b * N;
  } else {
    int mine = 0;
    for (int i = tid; i < b * N; i += kListThreads) mine += sync[i] != 0;
    // per-thread counts: sum over the block with a wave sum and the wave table
    const int ws = wave_sum_i32(mine);
    __syncthreads();
    if (lane == 0) s_wave[wv] = ws;
    __syncthreads();
    for (int w = 0; w < kListThreads / kWave; ++w) base += s_wave[w];
  }
  int run = base;
  for (int i0 = 0; i0 < N; i0 += kListThreads) {
    const int i = i0 + tid;
    const bool f = i < N && (all || sync[int64_t(b) * N + i] != 0);
    const uint64_t bal = __ballot(f);
    __syncthreads();
    if (lane == 0) s_wave[wv] = __popcll(bal);
    __syncthreads();
    int before = run, tot = 0;
    for (int w = 0; w < kListThreads / kWave; ++w) {
      if (w < wv) before += s_wave[w];
      tot += s_wave[w];
    }
    if (f) slist[before + __popcll(bal & ((1ull << lane) - 1ull))] = b * N + i;
    run += tot;
  }
  if (tid == 0) {
    soff[b] = base;
    if (b == B - 1) {
      const int ns = run;
      soff[B] = ns;
      tab[0] = 0;
      tab[1] = ns;
      tab[2] = 0;
      tab[3] = (ns + kProjTM - 1) / kProjTM * ntn_q;
      if (all) {
        tab[4] = 0;
        tab[5] = T;
        tab[6] = 0;
        tab[7] = (T + kProjTM - 1) / kProjTM * ntn_kv;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// multi-head attention of the listed queries (bf16 MFMA, fp32 softmax)
// ---------------------------------------------------------------------------
// Block: 4 waves, 128 listed queries of one (sample, head); wave w takes 32.
// Per tile of 64 keys the wave forms S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16 (keys as rows, queries as columns), so a lane
// owns one query (column lane & 31) and 16 of the 32 keys of each half
// tile: the online softmax (running max and sum per query) needs one lane
// exchange (l, l ^ 32) per tile.  The probabilities, rounded to bf16, are
// the B operand of O^T += V^T P^T, whose k order (keys) follows the S^T
// accumulator layout, so P never leaves registers.  K and V tiles land in
// LDS key-major, as they sit in memory, through direct global -> LDS loads
// (no register staging), in a two-stage ring (36 KB at d_h = 72), so three
// blocks share a CU (twelve waves): on a cache step the query tiles of the
// synchronised tokens then run in one round instead of two.  The V^T
// operand of p.v is read from the key-major V tile with the transposing
// LDS read.  Tile kt + 2's loads start after the barrier that ends tile
// kt's math and run under tile kt + 1's.  KS = ceil(d_h / 16) k-steps for
// q.k, OT = ceil(d_h / 32) output tiles of O^T; columns and rows past d_h
// are zero.  DH is d_h, a compile-time constant (every multiple of 8 up to
// 96 is instantiated), so the chunk index arithmetic of the tile loads has
// constant divisors.
constexpr int kAttnQ = 128;
constexpr int kAttnKeys = 64;
constexpr int kAttnThreads = 256;

template <int KS, int OT, int DH>
__global__ __launch_bounds__(kAttnThreads, 3) void attention_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kv,
    const int32_t* __restrict__ slist, const int32_t* __restrict__ soff, int B, int N, int H,
    int dh_arg, float scale_log2, uint16_t* __restrict__ o) {
  static_assert(DH % 8 == 0 && DH <= 96, "head width");
  constexpr int dh = DH;
  (void)dh_arg;
  constexpr int CPR = DH / 8;              // 16-byte chunks per head row
  // K and V rows in LDS (key-major, as in memory): KC chunks, an odd count,
  // so that the rows a read phase serves start on distinct bank groups; the
  // chunks past d_h hold whatever the loads put there and are never used
  constexpr int KC = CPR | 1;
  constexpr int KE = kAttnKeys * KC * 8;   // elements of one K (or V) stage
  constexpr int KI = KC;                   // DMA instructions per tile of K or V (64 chunks each)
  constexpr int KIW = (2 * KI + 3) / 4;    // per wave and tile, at most
  constexpr int kStg = 2;                  // LDS ring stages
  __shared__ __attribute__((aligned(16))) uint16_t sk[kStg * KE];
  __shared__ __attribute__((aligned(16))) uint16_t sv[kStg * KE];

  // (sample, head, query tile); the query tiles of one (sample, head) are
  // consecutive logical blocks on one XCD, so they share its L2 copy of K, V
  const int QT = (N + kAttnQ - 1) / kAttnQ;
  const int nblk = gridDim.x;
  const int L = nblk % 8 == 0 ? (blockIdx.x % 8) * (nblk / 8) + blockIdx.x / 8 : blockIdx.x;
  const int qt = L % QT;
  const int hh = (L / QT) % H;
  const int b = L / (QT * H);
  const int q0 = soff[b];
  const int nq = soff[b + 1] - q0;
  if (qt * kAttnQ >= nq) return;

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int n = lane & 31, hf = lane >> 5;
  const int d = H * dh;

  // the V^T rows past d_h of the p.v operand are zero, except that when
  // d_h is not a multiple of 32 the first of them is all ones, so that its
  // row of O^T accumulates the softmax denominator sum_k p_k (of the bf16 p
  // the p.v MFMAs use) with the same rescaling as O, and the VALU adds none
  constexpr bool kSumRow = DH % 32 != 0;

  // this lane's query and its fragments (B operand of S^T)
  const int qi = qt * kAttnQ + wv * 32 + n;
  const int tok = slist[q0 + min(qi, nq - 1)];
  const uint16_t* qrow = q + int64_t(tok) * d + hh * dh;
  bf16x8_t qf[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int c = 16 * s + 8 * hf;
    const u32x4_t w = c < dh ? *reinterpret_cast<const u32x4_t*>(qrow + c) : u32x4_t{0, 0, 0, 0};
    qf[s] = __builtin_bit_cast(bf16x8_t, w);
  }

  const int64_t row0 = int64_t(b) * N;
  // K and V: direct global -> LDS loads, key-major rows of KC chunks.  DMA
  // instruction i (wave i % 4) of a tile covers chunks 64 ii .. 64 ii + 63
  // of the K stage (i < KI, ii = i) or of the V stage (ii = i - KI), chunk
  // qc holding chunk qc % KC of key qc / KC (padding chunks load the key's
  // first chunk).
  const uint32_t sk0 = __builtin_amdgcn_readfirstlane(lds_addr(sk));
  const uint32_t sv0 = __builtin_amdgcn_readfirstlane(lds_addr(sv));
  const int kwv = __builtin_amdgcn_readfirstlane(wv);
  auto load_kv = [&](int kt, int st) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < KIW; ++u) {
      const int i = kwv + 4 * u;
      if (i < 2 * KI) {
        const bool isv = i >= KI;
        const int ii = isv ? i - KI : i;
        const int qc = 64 * ii + lane;
        const int key = min(kt * kAttnKeys + qc / KC, N - 1);
        const int c = qc % KC;
        const uint16_t* g =
            kv + (row0 + key) * (2 * d) + (isv ? d : 0) + hh * dh + (c < CPR ? c : 0) * 8;
        dma16(g, (isv ? sv0 : sk0) + (st * KE + ii * 512) * 2);
      }
    }
  };

  // softmax state in log2 units of the scaled scores.  m_run is the shift of
  // the exponentials, not always the running max: it moves only when a tile
  // brings a score more than kLazy above it, so p = 2^(s - m_run) stays
  // below 2^kLazy, and O (with the sum) is rescaled on few tiles instead of
  // nearly every one.  The normalised result is the same up to rounding.
  constexpr float kLazy = 8.0f;
  float m_run = -INFINITY, l_run = 0.0f;
  f32x16_t acc[OT];
#pragma unroll
  for (int t = 0; t < OT; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[t][v] = 0.0f;

  // q.k of tile kt: S^T for keys 32 t + (0..31)
  auto qk = [&](int kt, f32x16_t (&sacc)[2]) __attribute__((always_inline)) {
    const uint16_t* ks = sk + (kt % kStg) * KE;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) sacc[t][v] = 0.0f;
    // the two key halves alternate, so consecutive MFMAs are independent
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        // head dims past d_h (chunk CPR and above) are zero, as in q
        const int cc = 2 * s2 + hf;
        const bf16x8_t kf =
            cc < CPR ? *reinterpret_cast<const bf16x8_t*>(ks + ((32 * t + n) * KC + cc) * 8)
                     : bf16x8_t{};
        sacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s2], sacc[t], 0, 0, 0);
      }
  };
  // softmax of tile kt: keys past N masked (only a ragged last tile has
  // them), the running max and sum, O rescaled when some query's max moved,
  // then P (bf16) as the B operand fragments of the tile's four 16-key
  // k-steps; lane keys: 32 t + 8 (v / 4) + 4 hf + v % 4
  auto softmax = [&](int kt, f32x16_t (&sacc)[2], bf16x8_t (&pf)[4])
      __attribute__((always_inline)) {
    if ((kt + 1) * kAttnKeys > N) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kt * kAttnKeys + 32 * t + 8 * (v >> 2) + 4 * hf + (v & 3);
          if (key >= N) sacc[t][v] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[t][v]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave)) * scale_log2;
    const bool up = mx > m_run + kLazy;  // always on the first tile
    if (__ballot(up) != 0ull) {
      const float m_new = up ? mx : m_run;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);  // 0 on the first tile
      if constexpr (!kSumRow) l_run *= alpha;
#pragma unroll
      for (int t = 0; t < OT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[t][v] *= alpha;
      m_run = m_new;
    }
    float ps = 0.0f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sacc[t][v], scale_log2, -m_run));
        sacc[t][v] = p;
        if constexpr (!kSumRow) ps += p;
      }
    if constexpr (!kSumRow) l_run += ps;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const u32x4_t pw{pack2(sacc[t][8 * j], sacc[t][8 * j + 1]),
                         pack2(sacc[t][8 * j + 2], sacc[t][8 * j + 3]),
                         pack2(sacc[t][8 * j + 4], sacc[t][8 * j + 5]),
                         pack2(sacc[t][8 * j + 6], sacc[t][8 * j + 7])};
        pf[2 * t + j] = __builtin_bit_cast(bf16x8_t, pw);
      }
  };
  // O^T += V^T P^T for tile kt: fragment 2 t + j holds the keys
  // 32 t + 16 j + 4 hf + {0..3, 8..11}.  The V^T operand (lane: head dim
  // 32 ot + (lane & 31), those 8 keys) comes from the key-major V stage
  // through ds_read_b64_tr_b16: within a group of 16 lanes, lane i receives
  // element i % 4 of the 8-byte chunks that lanes 4 m + i / 4 (m = 0..3)
  // point at.  So lane 4 m + a of the group points at head dims
  // d0 + 4 a .. + 3 of key kb + m, and lane i (head dim d0 + i) receives
  // keys kb .. kb + 3, then kb + 8 .. kb + 11 from a second read.  Head dims
  // past d_h are replaced after the reads (their addresses are clamped).
  const int i16 = lane & 15;
  const int dl = 16 * ((lane >> 4) & 1);          // the group's first head dim in a tile
  typedef __attribute__((address_space(3))) v4i16_t* lp;
  auto pv = [&](int kt, const bf16x8_t (&pf)[4]) __attribute__((always_inline)) {
    const uint16_t* vs = sv + (kt % kStg) * KE;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int kb = 32 * t + 16 * j + 4 * hf + (i16 >> 2);  // key this lane points at
#pragma unroll
        for (int ot = 0; ot < OT; ++ot) {
          const int col = 32 * ot + dl + 4 * (i16 & 3);
          const uint16_t* vp = vs + kb * (KC * 8) + (col < DH ? col : 0);
          const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lp)(vp));
          const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lp)(vp + 8 * KC * 8));
          bf16x8_t vf = __builtin_bit_cast(
              bf16x8_t, v8i16_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
          if (32 * ot + 32 > DH) {
            const int dim = 32 * ot + dl + i16;  // this lane's head dim
            if (dim >= DH) {
              const uint32_t w = kSumRow && dim == DH ? 0x3F803F80u : 0u;  // bf16 ones or zeros
              vf = __builtin_bit_cast(bf16x8_t, u32x4_t{w, w, w, w});
            }
          }
          acc[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[2 * t + j], acc[ot], 0, 0, 0);
        }
      }
  };

  // Prologue: tiles 0 and 1 in their stages.  Iteration kt runs tile kt's
  // q.k, softmax and p.v on stage kt % 2, waits for tile kt + 1's loads
  // (issued in the previous iteration), and after the barrier (every wave
  // done with stage kt % 2) starts tile kt + 2's loads into it.
  const int nkt = (N + kAttnKeys - 1) / kAttnKeys;
  load_kv(0, 0);
  if (nkt > 1) load_kv(1, 1);
  wait_vmcnt<0>();
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    f32x16_t sacc[2];
    bf16x8_t pf[4];
    qk(kt, sacc);
    softmax(kt, sacc, pf);
    pv(kt, pf);
    wait_vmcnt<0>();
    __syncthreads();
    if (kt + 2 < nkt) load_kv(kt + 2, kt % kStg);
  }

  // normalise and store: lane holds head dims 32 ot + 8 g + 4 hf + (0..3);
  // the denominator: the ones row d_h of O^T (held by the lanes of half
  // (d_h % 8) / 4, register 4 ((d_h % 32) / 8) + d_h % 4 of tile d_h / 32),
  // or the two halves' running sums
  float l_tot;
  if constexpr (kSumRow) {
    constexpr int so = DH / 32, sr = 4 * ((DH % 32) / 8) + DH % 4, sh = (DH % 8) / 4;
    const float mine = acc[so][sr];
    const float other = __shfl_xor(mine, 32, kWave);
    l_tot = hf == sh ? mine : other;
  } else {
    l_tot = l_run + __shfl_xor(l_run, 32, kWave);
  }
  const float inv = 1.0f / l_tot;
  if (qi < nq) {
    uint16_t* orow = o + int64_t(tok) * d + hh * dh;
#pragma unroll
    for (int ot = 0; ot < OT; ++ot)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int m0 = 32 * ot + 8 * g + 4 * hf;
        if (m0 < dh)
          *reinterpret_cast<u32x2_t*>(orow + m0) =
              u32x2_t{pack2(acc[ot][4 * g] * inv, acc[ot][4 * g + 1] * inv),
                      pack2(acc[ot][4 * g + 2] * inv, acc[ot][4 * g + 3] * inv)};
      }
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_sinusoid(const float* t_values, int B, double* e, hipStream_t st) {
  const int n = B * kFreqDim;
  launch_kernel(&sinusoid_kernel, dim3((n + 255) / 256), dim3(256), 0, st, t_values, B, e);
  return hipGetLastError();
}

hipError_t launch_silu(const float* in, int n, double* out, hipStream_t st) {
  launch_kernel(&silu_kernel, dim3((n + 255) / 256), dim3(256), 0, st, in, n, out);
  return hipGetLastError();
}

hipError_t launch_gemv(const double* in, int B, int K, const GemvBatch& mats, int n_mats,
                       int Nout, const void* table, const int32_t* labels, int n_classes,
                       double* out64, hipStream_t st) {
  if (K % 32 != 0 || K > kMaxWidth || n_mats < 1 || n_mats > kGemvBatch)
    return hipErrorInvalidValue;
  // a small launch spreads its tiles over up to one block per CU (tile t
  // goes to block t mod blocks, wave t / blocks mod kGemvWaves)
  const int tiles = (Nout + 15) / 16 * n_mats;
  const int blocks = std::min(tiles, device_cus());
  launch_kernel(&gemv_kernel, dim3(blocks), dim3(kGemvWaves * kWave), 0,
                st, in, B, K, mats, n_mats, Nout, static_cast<const uint16_t*>(table), labels,
                n_classes, out64);
  return hipGetLastError();
}

// one wave per row; the instantiation holding ceil(d / 256) float4 chunks
// per lane
template <int MODE>
hipError_t launch_ln(const LnArgs& p, int T, int d, hipStream_t st) {
  const dim3 grid((T + kLnWaves - 1) / kLnWaves), block(kLnWaves * kWave);
  switch ((d / 4 + kWave - 1) / kWave) {
    case 1: launch_kernel(&ln_kernel<MODE, 1>, grid, block, 0, st, p); break;
    case 2: launch_kernel(&ln_kernel<MODE, 2>, grid, block, 0, st, p); break;
    case 3: launch_kernel(&ln_kernel<MODE, 3>, grid, block, 0, st, p); break;
    case 4: launch_kernel(&ln_kernel<MODE, 4>, grid, block, 0, st, p); break;
    case 5: launch_kernel(&ln_kernel<MODE, 5>, grid, block, 0, st, p); break;
    case 6: launch_kernel(&ln_kernel<MODE, 6>, grid, block, 0, st, p); break;
    case 7: launch_kernel(&ln_kernel<MODE, 7>, grid, block, 0, st, p); break;
    case 8: launch_kernel(&ln_kernel<MODE, 8>, grid, block, 0, st, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_ln_attn(const BlockBufs& k, int T, int N, int d, const float* mod,
                          const float* mod_prev, const uint16_t* a, bool cached,
                          hipStream_t st) {
  LnArgs p{k.x, k.x1, k.y, a, k.h, k.u, mod, mod_prev, nullptr, nullptr, T, N, d,
           mod_prev != nullptr ? 1 : 0, cached ? 1 : 0, 0, k.x1p};
  return launch_ln<kLnAttn>(p, T, d, st);
}

hipError_t launch_ln_mlp(const BlockBufs& k, int T, int N, int d, const float* mod,
                         const float* mod_prev, const uint16_t* a, uint16_t* u_out, bool routing,
                         hipStream_t st) {
  LnArgs p{k.x, k.x1, k.y, a, k.h, u_out, mod, mod_prev, k.slist, k.soff + k.B, T, N, d,
           mod_prev != nullptr ? 1 : 0, 1, routing ? 1 : 0, k.x1p};
  return launch_ln<kLnMlp>(p, T, d, st);
}

hipError_t launch_ln_final(const BlockBufs& k, int T, int N, int d, const float* mod,
                           hipStream_t st) {
  LnArgs p{k.x, k.x1, k.y, nullptr, nullptr, nullptr, mod, nullptr, nullptr, nullptr, T, N, d,
           0, 0, 0, nullptr};
  return launch_ln<kLnFinal>(p, T, d, st);
}

hipError_t launch_slist(const BlockBufs& k, const uint8_t* sync, int N, int d, hipStream_t st) {
  const int ntn_q = (d + kProjTN - 1) / kProjTN;
  const int ntn_kv = (2 * d + kProjTN - 1) / kProjTN;
  launch_kernel(&slist_kernel, dim3(k.B), dim3(kListThreads), 0, st, sync, sync == nullptr ? 1 : 0,
                k.B, N, ntn_q, ntn_kv, k.slist, k.soff, k.ident, k.tab);
  return hipGetLastError();
}

hipError_t launch_attention(const BlockBufs& k, int N, int H, int dh, hipStream_t st) {
  const int QT = (N + kAttnQ - 1) / kAttnQ;
  const dim3 grid(k.B * H * QT);
  const float scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(double(dh)));
  if (dh % 8 != 0 || dh > 96) return hipErrorInvalidValue;
#define MOECA_ATTN(DH)                                                                       \
  launch_kernel(&attention_kernel<((DH) + 15) / 16, ((DH) + 31) / 32, DH>, grid,               \
                dim3(kAttnThreads), 0, st, k.q, k.kv, k.slist, k.soff, k.B, N, H, dh,          \
                scale_log2, k.o)
  switch (dh / 8) {
    case 1: MOECA_ATTN(8); break;
    case 2: MOECA_ATTN(16); break;
    case 3: MOECA_ATTN(24); break;
    case 4: MOECA_ATTN(32); break;
    case 5: MOECA_ATTN(40); break;
    case 6: MOECA_ATTN(48); break;
    case 7: MOECA_ATTN(56); break;
    case 8: MOECA_ATTN(64); break;
    case 9: MOECA_ATTN(72); break;
    case 10: MOECA_ATTN(80); break;
    case 11: MOECA_ATTN(88); break;
    default: MOECA_ATTN(96); break;
  }
#undef MOECA_ATTN
  return hipGetLastError();
}

}  // namespace moeca
