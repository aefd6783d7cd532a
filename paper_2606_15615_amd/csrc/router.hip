// Router: logits, top-k experts and gate weights (Sec. 4.1, B_i^t).
//
// One wavefront per four tokens.  Lane l holds element pairs j = 2l + 128r of
// each token row; every W_r pair it loads and widens serves the four tokens.  For 16 experts at a time each lane accumulates the exact
// products x_j * W_r[e][j] (exact in fp64 for bf16 and fp32 inputs) in fp64;
// a transposing butterfly then reduces the 16 partial sums across the wave
// (each exchange halves the experts a lane carries), the sum (+ bias) is
// rounded once to fp32.  Top-k takes the largest logits, ties to the lower
// expert id; the gate is a softmax in fp64 over the top-k (renormalised) or
// over all experts, rounded once to fp32.
//
// The top-k and the gate are wave-parallel (lane e holds expert e).  The same
// kernel advances the expert statistic of its token (Sec. 4.3, EMA eq.): it
// knows which experts the token routes to.
//
// W_r is copied once per block into LDS when it fits (the benchmarked layer:
// 16 x 1152 bf16 = 36 KB), otherwise read from global memory (L2-resident).
#include "common.h"
#include "internal.h"

namespace moeca {
namespace {

constexpr int kRouterWaves = 4;
constexpr int kTokensPerWave = 4;  // tokens a wave accumulates together (reuses each W load)
constexpr int kTokensPerBlock = kRouterWaves * kTokensPerWave;
constexpr int kGroup = 16;
constexpr int kRowPairs = 9;  // element pairs per lane loaded at once: 1152 elements per chunk
constexpr size_t kLdsWBytes = 64 * 1024;

// A pair of consecutive elements widened to fp64.
template <typename T> struct Pair;
template <> struct Pair<uint16_t> {
  typedef uint32_t raw;
  static __device__ __forceinline__ raw load(const uint16_t* p) {
    return *reinterpret_cast<const uint32_t*>(p);
  }
  static __device__ __forceinline__ void widen(raw v, double& a, double& b) {
    a = static_cast<double>(__uint_as_float(v << 16));
    b = static_cast<double>(__uint_as_float(v & 0xffff0000u));
  }
};
template <> struct Pair<float> {
  typedef float2 raw;
  static __device__ __forceinline__ raw load(const float* p) {
    return *reinterpret_cast<const float2*>(p);
  }
  static __device__ __forceinline__ void widen(raw v, double& a, double& b) {
    a = static_cast<double>(v.x);
    b = static_cast<double>(v.y);
  }
};

// One stage of the transposing butterfly: lanes with bit O set keep the
// upper H sums and receive their partner's upper H; the others the lower H.
template <int H, int O>
__device__ __forceinline__ void transpose_stage(double (&v)[kGroup], bool upper) {
#pragma unroll
  for (int i = 0; i < H; ++i) {
    const double keep = upper ? v[i + H] : v[i];
    const double send = upper ? v[i] : v[i + H];
    v[i] = keep + __shfl_xor(send, O, kWave);
  }
}

// Reduce v[0..15] over the wave.  Afterwards lane l holds, in v[0], the full
// sum of expert g(l) = 8*b5 + 4*b4 + 2*b3 + b2 (b_i = bit i of l).
__device__ __forceinline__ void transpose_reduce16(double (&v)[kGroup], int lane) {
  transpose_stage<8, 32>(v, (lane & 32) != 0);
  transpose_stage<4, 16>(v, (lane & 16) != 0);
  transpose_stage<2, 8>(v, (lane & 8) != 0);
  transpose_stage<1, 4>(v, (lane & 4) != 0);
  v[0] += __shfl_xor(v[0], 2, kWave);
  v[0] += __shfl_xor(v[0], 1, kWave);
}

template <typename T, bool W_IN_LDS>
__global__ __launch_bounds__(kRouterWaves * kWave) void router_kernel(
    const T* __restrict__ x, const T* __restrict__ Wg, const float* __restrict__ bias,
    int64_t T_tokens, int d, int E, int k, int norm_topk, float* __restrict__ logits,
    int32_t* __restrict__ e_out, float* __restrict__ w_out, int32_t* __restrict__ rflags,
    float* __restrict__ C, int N, float beta) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ float s_logit[kRouterWaves][kTokensPerWave][64];
  __shared__ int s_bad;
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  if (threadIdx.x == 0) s_bad = 0;

  const T* W = Wg;
  if (W_IN_LDS) {
    T* ws = reinterpret_cast<T*>(smem);
    const int n16 = static_cast<int>(size_t(E) * d * sizeof(T) / 16);
    for (int i = threadIdx.x; i < n16; i += kRouterWaves * kWave)
      reinterpret_cast<uint4*>(ws)[i] = reinterpret_cast<const uint4*>(Wg)[i];
    W = ws;
  }
  __syncthreads();

  // this wave's tokens t0 .. t0 + kTokensPerWave - 1 (rows past the end re-read
  // the last token and are never written)
  const int64_t t0 = (int64_t(blockIdx.x) * kRouterWaves + wv) * kTokensPerWave;
  const T* xr[kTokensPerWave];
#pragma unroll
  for (int q = 0; q < kTokensPerWave; ++q) xr[q] = x + min(t0 + q, T_tokens - 1) * d;

  for (int e0 = 0; e0 < E; e0 += kGroup) {
    double acc[kTokensPerWave][kGroup];
#pragma unroll
    for (int q = 0; q < kTokensPerWave; ++q)
#pragma unroll
      for (int u = 0; u < kGroup; ++u) acc[q][u] = 0.0;
    // experts past E re-read row E-1 (branch-free); their sums are dropped
    const T* wrow[kGroup];
#pragma unroll
    for (int u = 0; u < kGroup; ++u) wrow[u] = W + int64_t(min(e0 + u, E - 1)) * d;
    // the rows in chunks of kRowPairs pairs per lane, each chunk loaded at once
    for (int c0 = 0; c0 < d; c0 += 2 * kWave * kRowPairs) {
      typename Pair<T>::raw xv[kTokensPerWave][kRowPairs];
#pragma unroll
      for (int r = 0; r < kRowPairs; ++r) {
        const int j = c0 + 2 * lane + 2 * kWave * r;
#pragma unroll
        for (int q = 0; q < kTokensPerWave; ++q)
          if (j < d) xv[q][r] = Pair<T>::load(xr[q] + j);
      }
#pragma unroll
      for (int r = 0; r < kRowPairs; ++r) {
        const int j = c0 + 2 * lane + 2 * kWave * r;
        if (j >= d) continue;
        typename Pair<T>::raw wr[kGroup];
#pragma unroll
        for (int u = 0; u < kGroup; ++u) wr[u] = Pair<T>::load(wrow[u] + j);
        double xa[kTokensPerWave], xb[kTokensPerWave];
#pragma unroll
        for (int q = 0; q < kTokensPerWave; ++q) Pair<T>::widen(xv[q][r], xa[q], xb[q]);
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
          double wa, wb;
          Pair<T>::widen(wr[u], wa, wb);
#pragma unroll
          for (int q = 0; q < kTokensPerWave; ++q) {
            acc[q][u] = fma(xa[q], wa, acc[q][u]);
            acc[q][u] = fma(xb[q], wb, acc[q][u]);
          }
        }
      }
    }
    const int ex = ((lane >> 5) & 1) * 8 + ((lane >> 4) & 1) * 4 + ((lane >> 3) & 1) * 2 +
                   ((lane >> 2) & 1);
#pragma unroll
    for (int q = 0; q < kTokensPerWave; ++q) {
      transpose_reduce16(acc[q], lane);
      if ((lane & 3) == 0 && e0 + ex < E) {
        double sm = acc[q][0];
        if (bias) sm += static_cast<double>(bias[e0 + ex]);
        s_logit[wv][q][e0 + ex] = static_cast<float>(sm);
      }
    }
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  bool bad = false;
  for (int q = 0; q < kTokensPerWave; ++q) {
    const int64_t t = t0 + q;
    if (t >= T_tokens) break;
    const bool is_e = lane < E;
    float lv = is_e ? s_logit[wv][q][lane] : -__builtin_huge_valf();
    if (is_e) logits[t * E + lane] = lv;
    if (is_e && !isfinite(lv)) bad = true;
    if (lv != lv) lv = -__builtin_huge_valf();  // a NaN logit never wins
    float mx = lv;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
    // top-k: k rounds of a wave argmax, ties to the lower expert id
    uint64_t taken = 0;
    int my_sel = 0;
    for (int p = 0; p < k; ++p) {
      const bool cand = is_e && !((taken >> lane) & 1ull);
      float cv = cand ? lv : -__builtin_huge_valf();
      int ci = cand ? lane : kWave;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const float ov = __shfl_xor(cv, o, kWave);
        const int oi = __shfl_xor(ci, o, kWave);
        if (ov > cv || (ov == cv && oi < ci)) {
          cv = ov;
          ci = oi;
        }
      }
      if (ci >= E) ci = __builtin_ctzll(~taken);  // defensive: cannot happen for k <= E
      if (lane == p) my_sel = ci;
      taken |= 1ull << ci;
    }
    // gate: softmax in fp64 over the top-k (renormalised) or all experts
    const double z = is_e ? exp(static_cast<double>(lv) - static_cast<double>(mx)) : 0.0;
    const bool in_den = norm_topk ? (((taken >> lane) & 1ull) != 0) : is_e;
    const double den = wave_sum_f64(in_den ? z : 0.0);
    const double zs = __shfl(z, my_sel, kWave);
    if (lane < k) {
      e_out[t * k + lane] = my_sel;
      w_out[t * k + lane] = static_cast<float>(zs / den);
    }
    // expert statistic C_{e,i} <- f32(f32(beta*C) + f32(1-beta)*[e in B_i])
    if (C != nullptr && is_e) {
      const int64_t b = t / N, i = t % N;
      float* cp = C + (b * E + lane) * N + i;
      float c = __fmul_rn(beta, *cp);
      if ((taken >> lane) & 1ull) c = __fadd_rn(c, __fsub_rn(1.0f, beta));
      *cp = c;
    }
  }
  if (bad) s_bad = 1;
  __syncthreads();
  if (threadIdx.x == 0) rflags[blockIdx.x] = s_bad;
}

template <typename T>
hipError_t launch_typed(const Shape& s, const void* x, const void* W_r, const float* b_r,
                        int norm_topk, float beta, bool update_stat, const Buffers& b,
                        hipStream_t st) {
  float* C = update_stat ? b.stat : nullptr;
  const dim3 grid(router_blocks(s)), block(kRouterWaves * kWave);
  const size_t wbytes = size_t(s.E) * s.d * sizeof(T);
  if (wbytes <= kLdsWBytes) {
    launch_kernel(
        &router_kernel<T, true>, grid, block, uint32_t(wbytes), st, static_cast<const T*>(x), static_cast<const T*>(W_r), b_r, s.tokens(), s.d, s.E, s.k,
        norm_topk, b.logits, b.e_t, b.w_t, b.rflags, C, s.N, beta);
  } else {
    launch_kernel(
        &router_kernel<T, false>, grid, block, 0, st, static_cast<const T*>(x), static_cast<const T*>(W_r), b_r, s.tokens(), s.d, s.E, s.k,
        norm_topk, b.logits, b.e_t, b.w_t, b.rflags, C, s.N, beta);
  }
  return hipGetLastError();
}

}  // namespace

int router_blocks(const Shape& s) {
  return static_cast<int>((s.tokens() + kTokensPerBlock - 1) / kTokensPerBlock);
}

hipError_t launch_router(const Shape& s, const void* x, const void* W_r, const float* b_r,
                         int norm_topk, float beta, bool update_stat, const Buffers& b,
                         hipStream_t st) {
  if (s.bf16)
    return launch_typed<uint16_t>(s, x, W_r, b_r, norm_topk, beta, update_stat, b, st);
  return launch_typed<float>(s, x, W_r, b_r, norm_topk, beta, update_stat, b, st);
}

}  // namespace moeca
