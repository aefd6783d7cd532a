// Router: logits, top-k experts and gate weights (Sec. 4.1, B_i^t).
//
// One wavefront per token.  Each lane accumulates the exact products
// x_j * W_r[e][j] (exact in fp64 for bf16 and fp32 inputs) in fp64 for 16
// experts at a time, the wave reduces them with an xor butterfly, and the
// sum (+ bias) is rounded once to fp32.  Top-k takes the largest logits,
// ties to the lower expert id; the gate is a softmax in fp64, over the
// top-k (renormalised) or over all experts, rounded once to fp32.
#include "common.h"
#include "internal.h"

namespace moeca {
namespace {

constexpr int kRouterWaves = 4;
constexpr int kExpertGroup = 16;

template <typename T>
__device__ __forceinline__ double widen(T v) { return static_cast<double>(Act<T>::to_f32(v)); }

template <typename T>
__global__ __launch_bounds__(kRouterWaves * kWave) void router_kernel(
    const T* __restrict__ x, const T* __restrict__ W, const float* __restrict__ bias,
    int64_t T_tokens, int d, int E, int k, int norm_topk, float* __restrict__ logits,
    int32_t* __restrict__ e_out, float* __restrict__ w_out, int32_t* __restrict__ rflags) {
  __shared__ float s_logit[kRouterWaves][64];
  __shared__ int s_bad;
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  const int64_t t = int64_t(blockIdx.x) * kRouterWaves + wv;
  if (threadIdx.x == 0) s_bad = 0;
  __syncthreads();

  if (t < T_tokens) {
    const T* xr = x + t * d;
    for (int e0 = 0; e0 < E; e0 += kExpertGroup) {
      double acc[kExpertGroup];
#pragma unroll
      for (int u = 0; u < kExpertGroup; ++u) acc[u] = 0.0;
      for (int j = lane; j < d; j += kWave) {
        const double xv = widen(xr[j]);
#pragma unroll
        for (int u = 0; u < kExpertGroup; ++u) {
          if (e0 + u < E) acc[u] = fma(xv, widen(W[int64_t(e0 + u) * d + j]), acc[u]);
        }
      }
#pragma unroll
      for (int u = 0; u < kExpertGroup; ++u) {
        double s = wave_sum_f64(acc[u]);
        if (lane == u && e0 + u < E) {
          if (bias) s += static_cast<double>(bias[e0 + u]);
          s_logit[wv][e0 + u] = static_cast<float>(s);
        }
      }
    }
  }
  __syncthreads();

  if (t < T_tokens) {
    if (lane < E) logits[t * E + lane] = s_logit[wv][lane];
    if (lane == 0) {
      const float* l = s_logit[wv];
      bool bad = false;
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
      if (bad) s_bad = 1;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) rflags[blockIdx.x] = s_bad;
}

}  // namespace

int router_blocks(const Shape& s) {
  return static_cast<int>((s.tokens() + kRouterWaves - 1) / kRouterWaves);
}

hipError_t launch_router(const Shape& s, const void* x, const void* W_r, const float* b_r,
                         int norm_topk, const Buffers& b, hipStream_t st) {
  const dim3 grid(router_blocks(s)), block(kRouterWaves * kWave);
  if (s.bf16) {
    router_kernel<uint16_t><<<grid, block, 0, st>>>(
        static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(W_r), b_r, s.tokens(), s.d,
        s.E, s.k, norm_topk, b.logits, b.e_t, b.w_t, b.rflags);
  } else {
    router_kernel<float><<<grid, block, 0, st>>>(
        static_cast<const float*>(x), static_cast<const float*>(W_r), b_r, s.tokens(), s.d, s.E,
        s.k, norm_topk, b.logits, b.e_t, b.w_t, b.rflags);
  }
  return hipGetLastError();
}

}  // namespace moeca
