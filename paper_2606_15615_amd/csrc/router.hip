// Router: logits, top-k experts and gate weights (Sec. 4.1, B_i^t).
//
// One wavefront per token.  Lane l holds element pairs j = 2l + 128r of the
// token row.  For 16 experts at a time each lane accumulates the exact
// products x_j * W_r[e][j] (exact in fp64 for bf16 and fp32 inputs) in fp64;
// a transposing butterfly then reduces the 16 partial sums across the wave
// (each exchange halves the experts a lane carries), the sum (+ bias) is
// rounded once to fp32.  Top-k takes the largest logits, ties to the lower
// expert id; the gate is a softmax in fp64 over the top-k (renormalised) or
// over all experts, rounded once to fp32.
//
// W_r is copied once per block into LDS when it fits (the benchmarked layer:
// 16 x 1152 bf16 = 36 KB), otherwise read from global memory (L2-resident).
#include "common.h"
#include "internal.h"

namespace moeca {
namespace {

constexpr int kRouterWaves = 4;
constexpr int kTokensPerWave = 2;
constexpr int kTokensPerBlock = kRouterWaves * kTokensPerWave;
constexpr int kGroup = 16;
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
    int32_t* __restrict__ e_out, float* __restrict__ w_out, int32_t* __restrict__ rflags) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ float s_logit[kRouterWaves][64];
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

  bool bad = false;
  for (int it = 0; it < kTokensPerWave; ++it) {
    const int64_t t = int64_t(blockIdx.x) * kTokensPerBlock + it * kRouterWaves + wv;
    if (t >= T_tokens) break;
    const T* xr = x + t * d;
    for (int e0 = 0; e0 < E; e0 += kGroup) {
      double acc[kGroup];
#pragma unroll
      for (int u = 0; u < kGroup; ++u) acc[u] = 0.0;
      // experts past E re-read row E-1 (branch-free); their sums are dropped
      const T* wrow[kGroup];
#pragma unroll
      for (int u = 0; u < kGroup; ++u) wrow[u] = W + int64_t(min(e0 + u, E - 1)) * d;
      typename Pair<T>::raw xn = Pair<T>::load(xr + 2 * lane);
      for (int j = 2 * lane; j < d; j += 2 * kWave) {
        const typename Pair<T>::raw xc = xn;
        if (j + 2 * kWave < d) xn = Pair<T>::load(xr + j + 2 * kWave);
        typename Pair<T>::raw wr[kGroup];
#pragma unroll
        for (int u = 0; u < kGroup; ++u) wr[u] = Pair<T>::load(wrow[u] + j);
        double xa, xb;
        Pair<T>::widen(xc, xa, xb);
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
          double wa, wb;
          Pair<T>::widen(wr[u], wa, wb);
          acc[u] = fma(xa, wa, acc[u]);
          acc[u] = fma(xb, wb, acc[u]);
        }
      }
      transpose_reduce16(acc, lane);
      const int ex = ((lane >> 5) & 1) * 8 + ((lane >> 4) & 1) * 4 + ((lane >> 3) & 1) * 2 +
                     ((lane >> 2) & 1);
      if ((lane & 3) == 0 && e0 + ex < E) {
        double s = acc[0];
        if (bias) s += static_cast<double>(bias[e0 + ex]);
        s_logit[wv][e0 + ex] = static_cast<float>(s);
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (lane < E) logits[t * E + lane] = s_logit[wv][lane];
    if (lane == 0) {
      const float* l = s_logit[wv];
      float mx = l[0];
      for (int e = 0; e < E; ++e) {
        if (!isfinite(l[e])) bad = true;
        mx = fmaxf(mx, l[e]);
      }
      uint64_t taken = 0;
      int sel[8];
      for (int p = 0; p < k; ++p) {
        int best = -1;
        for (int e = 0; e < E; ++e) {
          if ((taken >> e) & 1ull) continue;
          if (best < 0 || l[e] > l[best]) best = e;
        }
        sel[p] = best;
        taken |= 1ull << best;
      }
      const double m64 = static_cast<double>(mx);
      double z[8];
      double den = 0.0;
      for (int p = 0; p < k; ++p) z[p] = exp(static_cast<double>(l[sel[p]]) - m64);
      if (norm_topk) {
        for (int p = 0; p < k; ++p) den += z[p];
      } else {
        for (int e = 0; e < E; ++e) den += exp(static_cast<double>(l[e]) - m64);
      }
      for (int p = 0; p < k; ++p) {
        e_out[t * k + p] = sel[p];
        w_out[t * k + p] = static_cast<float>(z[p] / den);
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  if (bad) s_bad = 1;
  __syncthreads();
  if (threadIdx.x == 0) rflags[blockIdx.x] = s_bad;
}

template <typename T>
hipError_t launch_typed(const Shape& s, const void* x, const void* W_r, const float* b_r,
                        int norm_topk, const Buffers& b, hipStream_t st) {
  const dim3 grid(router_blocks(s)), block(kRouterWaves * kWave);
  const size_t wbytes = size_t(s.E) * s.d * sizeof(T);
  if (wbytes <= kLdsWBytes) {
    router_kernel<T, true><<<grid, block, wbytes, st>>>(
        static_cast<const T*>(x), static_cast<const T*>(W_r), b_r, s.tokens(), s.d, s.E, s.k,
        norm_topk, b.logits, b.e_t, b.w_t, b.rflags);
  } else {
    router_kernel<T, false><<<grid, block, 0, st>>>(
        static_cast<const T*>(x), static_cast<const T*>(W_r), b_r, s.tokens(), s.d, s.E, s.k,
        norm_topk, b.logits, b.e_t, b.w_t, b.rflags);
  }
  return hipGetLastError();
}

}  // namespace

int router_blocks(const Shape& s) {
  return static_cast<int>((s.tokens() + kTokensPerBlock - 1) / kTokensPerBlock);
}

hipError_t launch_router(const Shape& s, const void* x, const void* W_r, const float* b_r,
                         int norm_topk, const Buffers& b, hipStream_t st) {
  if (s.bf16) return launch_typed<uint16_t>(s, x, W_r, b_r, norm_topk, b, st);
  return launch_typed<float>(s, x, W_r, b_r, norm_topk, b, st);
}

}  // namespace moeca
