// Combine, cache metadata and attention-path refresh (Sec. 4.1).
//
//   y_i = sum_p f32(w_p * hhat_p), accumulated in fp32 in branch order, where
//   hhat_p is the cache row in slot sigma(p): the row the down projection
//   just wrote for a recomputed branch, the untouched cached row h_{q(p)} for
//   a reused one (reused branches use the current gate weight).
//   For each recomputed branch the slot's metadata becomes (e_p, w_p,
//   ||h||), the norm an fp64 sum of squares of the stored row rounded once.
//   Tokens with a recomputed branch copy their attention-path feature into
//   the attention cache (synchronised update).
//
// One wavefront per token; each lane handles groups of 8 consecutive
// elements (16 bytes of bf16).  Built without FMA contraction: the products
// and sums are the correctly rounded fp32 operations.
#include "common.h"
#include "internal.h"

#pragma clang fp contract(off)

namespace moeca {
namespace {

constexpr int kCombWaves = 4;

template <typename T> struct Vec8;
template <> struct Vec8<uint16_t> {
  static __device__ __forceinline__ void load(const uint16_t* p, float* v) {
    const uint4 raw = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      v[2 * u] = __uint_as_float(w[u] << 16);
      v[2 * u + 1] = __uint_as_float(w[u] & 0xffff0000u);
    }
  }
  static __device__ __forceinline__ void store(uint16_t* p, const float* v) {
    uint4 raw;
    raw.x = f32_to_bf16(v[0]) | (uint32_t(f32_to_bf16(v[1])) << 16);
    raw.y = f32_to_bf16(v[2]) | (uint32_t(f32_to_bf16(v[3])) << 16);
    raw.z = f32_to_bf16(v[4]) | (uint32_t(f32_to_bf16(v[5])) << 16);
    raw.w = f32_to_bf16(v[6]) | (uint32_t(f32_to_bf16(v[7])) << 16);
    *reinterpret_cast<uint4*>(p) = raw;
  }
  static __device__ __forceinline__ void copy(const uint16_t* src, uint16_t* dst) {
    *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(src);
  }
};
template <> struct Vec8<float> {
  static __device__ __forceinline__ void load(const float* p, float* v) {
    const float4 a = reinterpret_cast<const float4*>(p)[0];
    const float4 b = reinterpret_cast<const float4*>(p)[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
  static __device__ __forceinline__ void store(float* p, const float* v) {
    reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
    reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
  static __device__ __forceinline__ void copy(const float* src, float* dst) {
    reinterpret_cast<float4*>(dst)[0] = reinterpret_cast<const float4*>(src)[0];
    reinterpret_cast<float4*>(dst)[1] = reinterpret_cast<const float4*>(src)[1];
  }
};

template <typename T>
__global__ __launch_bounds__(kCombWaves * kWave) void combine_kernel(
    const float* __restrict__ w_t, const int32_t* __restrict__ e_t,
    const int32_t* __restrict__ sigma, const uint8_t* __restrict__ mask,
    const uint8_t* __restrict__ sync, T* __restrict__ h_c, int32_t* __restrict__ e_c,
    float* __restrict__ w_c, float* __restrict__ n_c, T* __restrict__ out,
    const T* __restrict__ attn_in, T* __restrict__ attn_cache, int64_t T_tokens, int d, int k,
    int write_cache) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t t = int64_t(blockIdx.x) * kCombWaves + threadIdx.x / kWave;
  if (t >= T_tokens) return;

  float wp[8];
  int slot[8];
  bool rec[8];
  for (int p = 0; p < k; ++p) {
    const int64_t f = t * k + p;
    wp[p] = w_t[f];
    slot[p] = sigma[f];
    rec[p] = mask[f] != 0;
  }
  double ss[8];
  for (int p = 0; p < k; ++p) ss[p] = 0.0;

  const int groups = d / 8;
  for (int g = lane; g < groups; g += kWave) {
    float acc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc[u] = 0.0f;
    for (int p = 0; p < k; ++p) {
      float h[8];
      Vec8<T>::load(h_c + (t * k + slot[p]) * d + g * 8, h);
#pragma unroll
      for (int u = 0; u < 8; ++u) acc[u] = __fadd_rn(acc[u], __fmul_rn(wp[p], h[u]));
      if (rec[p]) {
#pragma unroll
        for (int u = 0; u < 8; ++u) ss[p] += static_cast<double>(h[u]) * static_cast<double>(h[u]);
      }
    }
    Vec8<T>::store(out + t * d + g * 8, acc);
  }

  if (!write_cache) return;
  for (int p = 0; p < k; ++p) {
    if (!rec[p]) continue;  // uniform across the wave (one token per wave)
    const double s = wave_sum_f64(ss[p]);
    if (lane == 0) {
      const int64_t c = t * k + slot[p];
      n_c[c] = static_cast<float>(sqrt(s));
      e_c[c] = e_t[t * k + p];
      w_c[c] = wp[p];
    }
  }
  if (attn_in != nullptr && sync[t]) {
    for (int g = lane; g < groups; g += kWave)
      Vec8<T>::copy(attn_in + t * d + g * 8, attn_cache + t * d + g * 8);
  }
}

}  // namespace

hipError_t launch_combine(const Shape& s, int write_cache, void* out, const void* attn_in,
                          void* attn_cache, const Buffers& b, hipStream_t st) {
  const dim3 grid(static_cast<unsigned>((s.tokens() + kCombWaves - 1) / kCombWaves));
  const dim3 block(kCombWaves * kWave);
#define MOECA_COMBINE(KER, TT)                                                                 \
  launch_kernel(&KER, grid, block, 0, st, b.w_t, b.e_t, b.sigma, b.mask, b.sync,               \
                static_cast<TT*>(b.h_c), b.e_c, b.w_c, b.n_c, static_cast<TT*>(out),           \
                static_cast<const TT*>(attn_in), static_cast<TT*>(attn_cache), s.tokens(), s.d,  \
                s.k, write_cache)
  if (s.bf16) {
    MOECA_COMBINE(combine_kernel<uint16_t>, uint16_t);
  } else {
    MOECA_COMBINE(combine_kernel<float>, float);
  }
#undef MOECA_COMBINE
  return hipGetLastError();
}

}  // namespace moeca
