// Combine, cache metadata and attention-path refresh (Sec. 4.1).
//
//   y_i = sum_s h_s + sum_p f32(w_p * hhat_p), accumulated in fp32, shared
//   experts first (Sec. 2.3, shared-expert MoE eq.; no gate), then the
//   branches in order, where hhat_p is the cache row in slot sigma(p): the
//   row the down projection just wrote for a recomputed branch, the
//   untouched cached row h_{q(p)} for a reused one (reused branches use the
//   current gate weight).
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
    const T* __restrict__ attn_in, T* __restrict__ attn_cache, const T* __restrict__ h_sh,
    int S, int64_t T_tokens, int d, int k, int write_cache) {
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
    for (int sh = 0; sh < S; ++sh) {
      float h[8];
      Vec8<T>::load(h_sh + (sh * T_tokens + t) * d + g * 8, h);
#pragma unroll
      for (int u = 0; u < 8; ++u) acc[u] = __fadd_rn(acc[u], h[u]);
    }
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

// Fast path for k <= 2, d <= 512 GI and no shared experts (h_sh and S are
// not read): the token index is wave-uniform, so the branch metadata comes
// in by scalar loads; then every row load of the token (its k cache rows
// and, when synchronised, its attention row) is issued before any is used,
// so a token costs two dependent memory round trips.  Same arithmetic as
// above.
template <typename T> struct Raw8;
template <> struct Raw8<uint16_t> {
  typedef __attribute__((ext_vector_type(4))) unsigned int v;
  // the combine reads each cached row and attention row once per step:
  // non-temporal loads, so that they do not displace the step's other data
  static __device__ __forceinline__ v load(const uint16_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const v*>(p));
  }
  static __device__ __forceinline__ void store(uint16_t* p, v x) { *reinterpret_cast<v*>(p) = x; }
  static __device__ __forceinline__ void widen(v x, float* f) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      f[2 * u] = __uint_as_float(x[u] << 16);
      f[2 * u + 1] = __uint_as_float(x[u] & 0xffff0000u);
    }
  }
  static __device__ __forceinline__ v narrow(const float* f) {
    v x;
#pragma unroll
    for (int u = 0; u < 4; ++u)
      x[u] = f32_to_bf16(f[2 * u]) | (uint32_t(f32_to_bf16(f[2 * u + 1])) << 16);
    return x;
  }
};
template <> struct Raw8<float> {
  typedef __attribute__((ext_vector_type(8))) float v;
  static __device__ __forceinline__ v load(const float* p) {
    return *reinterpret_cast<const v*>(p);
  }
  static __device__ __forceinline__ void store(float* p, v x) { *reinterpret_cast<v*>(p) = x; }
  static __device__ __forceinline__ void widen(v x, float* f) {
#pragma unroll
    for (int u = 0; u < 8; ++u) f[u] = x[u];
  }
  static __device__ __forceinline__ v narrow(const float* f) {
    v x;
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = f[u];
    return x;
  }
};

template <typename T, int K, int GI>
__global__ __launch_bounds__(kCombWaves * kWave) void combine_fast_kernel(
    const float* __restrict__ w_t, const int32_t* __restrict__ e_t,
    const int32_t* __restrict__ sigma, const uint8_t* __restrict__ mask,
    const uint8_t* __restrict__ sync, T* __restrict__ h_c, int32_t* __restrict__ e_c,
    float* __restrict__ w_c, float* __restrict__ n_c, T* __restrict__ out,
    const T* __restrict__ attn_in, T* __restrict__ attn_cache, const T* __restrict__ h_sh,
    int S, int64_t T_tokens, int d, int k, int write_cache) {
  typedef typename Raw8<T>::v raw;
  const int lane = threadIdx.x & (kWave - 1);
  const int t = __builtin_amdgcn_readfirstlane(
      static_cast<int>(blockIdx.x) * kCombWaves + static_cast<int>(threadIdx.x) / kWave);
  if (t >= T_tokens) return;
  const int groups = d / 8;

  float wp[K];
  int slot[K];
  bool rec[K];
#pragma unroll
  for (int p = 0; p < K; ++p) {
    const int64_t f = int64_t(t) * K + p;
    wp[p] = w_t[f];
    slot[p] = sigma[f];
    rec[p] = mask[f] != 0;
  }
  const bool syn = write_cache && attn_in != nullptr && sync[t] != 0;

  raw h[K][GI];
  raw a[GI];
#pragma unroll
  for (int p = 0; p < K; ++p) {
    const T* row = h_c + (int64_t(t) * K + slot[p]) * d;
#pragma unroll
    for (int gi = 0; gi < GI; ++gi) {
      const int g = lane + kWave * gi;
      if (g < groups) h[p][gi] = Raw8<T>::load(row + g * 8);
    }
  }
  if (syn) {
#pragma unroll
    for (int gi = 0; gi < GI; ++gi) {
      const int g = lane + kWave * gi;
      if (g < groups) a[gi] = Raw8<T>::load(attn_in + int64_t(t) * d + g * 8);
    }
  }

  double ss[K];
#pragma unroll
  for (int p = 0; p < K; ++p) ss[p] = 0.0;
#pragma unroll
  for (int gi = 0; gi < GI; ++gi) {
    const int g = lane + kWave * gi;
    if (g >= groups) continue;
    float acc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc[u] = 0.0f;
#pragma unroll
    for (int p = 0; p < K; ++p) {
      float hv[8];
      Raw8<T>::widen(h[p][gi], hv);
#pragma unroll
      for (int u = 0; u < 8; ++u) acc[u] = __fadd_rn(acc[u], __fmul_rn(wp[p], hv[u]));
      if (rec[p]) {
#pragma unroll
        for (int u = 0; u < 8; ++u)
          ss[p] += static_cast<double>(hv[u]) * static_cast<double>(hv[u]);
      }
    }
    Raw8<T>::store(out + int64_t(t) * d + g * 8, Raw8<T>::narrow(acc));
    if (syn) Raw8<T>::store(attn_cache + int64_t(t) * d + g * 8, a[gi]);
  }

  if (!write_cache) return;
#pragma unroll
  for (int p = 0; p < K; ++p) {
    if (!rec[p]) continue;  // uniform across the wave (one token per wave)
    const double sq = wave_sum_f64(ss[p]);
    if (lane == 0) {
      const int64_t c = int64_t(t) * K + slot[p];
      n_c[c] = static_cast<float>(sqrt(sq));
      e_c[c] = e_t[int64_t(t) * K + p];
      w_c[c] = wp[p];
    }
  }
}

// bf16 layers outside the fast path (k up to 8, shared experts): one wave
// per token as in combine_kernel, but for each 16-byte group every row load
// (the S shared rows, the k cache rows and, when synchronised, the attention
// row) is issued before any is used.  Same arithmetic and order.
template <int KMAX, int SMAX>
__global__ __launch_bounds__(kCombWaves * kWave) void combine_wide_kernel(
    const float* __restrict__ w_t, const int32_t* __restrict__ e_t,
    const int32_t* __restrict__ sigma, const uint8_t* __restrict__ mask,
    const uint8_t* __restrict__ sync, uint16_t* __restrict__ h_c, int32_t* __restrict__ e_c,
    float* __restrict__ w_c, float* __restrict__ n_c, uint16_t* __restrict__ out,
    const uint16_t* __restrict__ attn_in, uint16_t* __restrict__ attn_cache,
    const uint16_t* __restrict__ h_sh, int S, int64_t T_tokens, int d, int k,
    int write_cache) {
  typedef Raw8<uint16_t>::v raw;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t t = __builtin_amdgcn_readfirstlane(
      static_cast<int>(blockIdx.x) * kCombWaves + static_cast<int>(threadIdx.x) / kWave);
  if (t >= T_tokens) return;
  const int groups = d / 8;

  float wp[KMAX];
  int slot[KMAX];
  bool rec[KMAX];
#pragma unroll
  for (int p = 0; p < KMAX; ++p) {
    wp[p] = 0.0f;
    slot[p] = 0;
    rec[p] = false;
    if (p < k) {
      const int64_t f = t * k + p;
      wp[p] = w_t[f];
      slot[p] = sigma[f];
      rec[p] = mask[f] != 0;
    }
  }
  const bool syn = write_cache && attn_in != nullptr && sync[t] != 0;
  double ss[KMAX];
#pragma unroll
  for (int p = 0; p < KMAX; ++p) ss[p] = 0.0;

  for (int g = lane; g < groups; g += kWave) {
    raw hs[SMAX], hk[KMAX], av;
#pragma unroll
    for (int sh = 0; sh < SMAX; ++sh)
      if (sh < S) hs[sh] = Raw8<uint16_t>::load(h_sh + (sh * T_tokens + t) * d + g * 8);
#pragma unroll
    for (int p = 0; p < KMAX; ++p)
      if (p < k) hk[p] = Raw8<uint16_t>::load(h_c + (t * k + slot[p]) * d + g * 8);
    if (syn) av = Raw8<uint16_t>::load(attn_in + t * d + g * 8);
    float acc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc[u] = 0.0f;
#pragma unroll
    for (int sh = 0; sh < SMAX; ++sh) {
      if (sh < S) {
        float h[8];
        Raw8<uint16_t>::widen(hs[sh], h);
#pragma unroll
        for (int u = 0; u < 8; ++u) acc[u] = __fadd_rn(acc[u], h[u]);
      }
    }
#pragma unroll
    for (int p = 0; p < KMAX; ++p) {
      if (p < k) {
        float h[8];
        Raw8<uint16_t>::widen(hk[p], h);
#pragma unroll
        for (int u = 0; u < 8; ++u) acc[u] = __fadd_rn(acc[u], __fmul_rn(wp[p], h[u]));
        if (rec[p]) {
#pragma unroll
          for (int u = 0; u < 8; ++u)
            ss[p] += static_cast<double>(h[u]) * static_cast<double>(h[u]);
        }
      }
    }
    Raw8<uint16_t>::store(out + t * d + g * 8, Raw8<uint16_t>::narrow(acc));
    if (syn) Raw8<uint16_t>::store(attn_cache + t * d + g * 8, av);
  }

  if (!write_cache) return;
#pragma unroll
  for (int p = 0; p < KMAX; ++p) {
    if (p >= k || !rec[p]) continue;  // uniform across the wave (one token per wave)
    const double sq = wave_sum_f64(ss[p]);
    if (lane == 0) {
      const int64_t c = t * k + slot[p];
      n_c[c] = static_cast<float>(sqrt(sq));
      e_c[c] = e_t[t * k + p];
      w_c[c] = wp[p];
    }
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
                static_cast<const TT*>(attn_in), static_cast<TT*>(attn_cache),                 \
                static_cast<const TT*>(b.h_sh), s.S, s.tokens(), s.d, s.k, write_cache)
  const int gi = (s.d / 8 + kWave - 1) / kWave;  // 8-element groups per lane
  const bool fast = s.k <= 2 && gi <= 4 && s.S == 0 && s.tokens() < (int64_t(1) << 31);
#define MOECA_FAST(TT, KK)                                                           \
  switch (gi) {                                                                      \
    case 1: MOECA_COMBINE((combine_fast_kernel<TT, KK, 1>), TT); break;              \
    case 2: MOECA_COMBINE((combine_fast_kernel<TT, KK, 2>), TT); break;              \
    case 3: MOECA_COMBINE((combine_fast_kernel<TT, KK, 3>), TT); break;              \
    default: MOECA_COMBINE((combine_fast_kernel<TT, KK, 4>), TT); break;             \
  }
  if (fast && s.bf16) {
    if (s.k == 1) { MOECA_FAST(uint16_t, 1) } else { MOECA_FAST(uint16_t, 2) }
  } else if (fast) {
    if (s.k == 1) { MOECA_FAST(float, 1) } else { MOECA_FAST(float, 2) }
  } else if (s.bf16 && s.tokens() < (int64_t(1) << 31)) {
    MOECA_COMBINE((combine_wide_kernel<8, 8>), uint16_t);
  } else if (s.bf16) {
    MOECA_COMBINE(combine_kernel<uint16_t>, uint16_t);
  } else {
    MOECA_COMBINE(combine_kernel<float>, float);
  }
#undef MOECA_FAST
#undef MOECA_COMBINE
  return hipGetLastError();
}

}  // namespace moeca
