// Router: logits, top-k experts and gate weights (Sec. 4.1, B_i^t), and the
// EMA of the expert statistic (Sec. 4.3, EMA eq.).
//
// Logits.  A block takes 16 consecutive positions of one sample (the last
// chunk of a sample may hold fewer).  The dot products x_i . W_r[e] run on
// the fp64 matrix cores (v_mfma_f64_16x16x4f64: 16 tokens x 16 experts x 4
// k per instruction).  Every product of two bf16 (or two fp32) values is
// exact in fp64, so this is the exact-product, fp64-accumulated sum the
// decision path asks for; the sum (+ bias) is rounded once to fp32.  The four
// waves split d into four ranges.  Lane l feeds token l % 16 (A operand) and
// expert l % 16 (B operand) at MFMA k-row l / 16; the k-rows interleave in
// runs of one load vector, so a row's four lanes read a contiguous segment
// of both the token row and the expert row with each load.  Four accumulator
// chains (two with more than 32 experts) rotate to hide the MFMA latency;
// the chains and then the four waves' partial sums are added in a fixed
// order (deterministic).
//
// Loads are software-pipelined: a wave's share of d is walked in chunks,
// the next chunk's loads issued before the current chunk's MFMAs.
//
// Epilogue.  Wave w takes the four tokens 4w + g (g = l / 16), one per
// 16-lane group, lane l % 16 holding experts l % 16 + 16 q.  Top-k: k rounds
// of a group argmax (ties to the lower expert id, NaN never wins); gate: a
// softmax in fp64 over the top-k (renormalised) or over all experts, rounded
// once to fp32, written by the lane that holds the selected expert.  The
// 16-lane reductions use DPP row permutations (quad swaps, half-row and row
// mirrors), so every lane of the group ends with the same value.  The
// statistic C[b][e][i] of the token's experts is read at kernel start and
// updated here: C <- f32(f32(beta C) + f32(1 - beta) [e in B_i]).  For the
// entropy of the statistic the block also writes, per expert, the fp64 sums
// over its positions of C and of C log C (log in fp64 of the stored value,
// the product rounded once; positions with C = 0 add nothing), in a fixed
// order: token pairs within a wave by lane exchange, then the four waves.
#include "common.h"
#include "internal.h"

namespace moeca {
namespace {

constexpr int kRouterWaves = 4;
constexpr int kTokensPerBlock = 16;

typedef __attribute__((ext_vector_type(4))) double f64x4_t;
typedef __attribute__((ext_vector_type(4))) unsigned int r_u32x4_t;
typedef __attribute__((ext_vector_type(2))) unsigned int r_u32x2_t;
typedef __attribute__((ext_vector_type(4))) float r_f32x4_t;

// VW consecutive elements of a row: one 8- or 16-byte load, widened to fp64.
template <typename T, int VW> struct Vec;
template <> struct Vec<uint16_t, 8> {
  typedef r_u32x4_t raw;
  static __device__ __forceinline__ raw load(const uint16_t* p) {
    return *reinterpret_cast<const r_u32x4_t*>(p);
  }
  static __device__ __forceinline__ void widen(raw r, double (&v)[8]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      v[2 * u] = static_cast<double>(__uint_as_float(r[u] << 16));
      v[2 * u + 1] = static_cast<double>(__uint_as_float(r[u] & 0xffff0000u));
    }
  }
};
template <> struct Vec<uint16_t, 4> {
  typedef r_u32x2_t raw;
  static __device__ __forceinline__ raw load(const uint16_t* p) {
    return *reinterpret_cast<const r_u32x2_t*>(p);
  }
  static __device__ __forceinline__ void widen(raw r, double (&v)[4]) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      v[2 * u] = static_cast<double>(__uint_as_float(r[u] << 16));
      v[2 * u + 1] = static_cast<double>(__uint_as_float(r[u] & 0xffff0000u));
    }
  }
};
template <> struct Vec<float, 4> {
  typedef r_f32x4_t raw;
  static __device__ __forceinline__ raw load(const float* p) {
    return *reinterpret_cast<const r_f32x4_t*>(p);
  }
  static __device__ __forceinline__ void widen(raw r, double (&v)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = static_cast<double>(r[u]);
  }
};

// Row max and row argmax (ties to the lower id).
__device__ __forceinline__ float row_max(float v) {
  v = fmaxf(v, dpp_f32<kDppRow[0]>(v));
  v = fmaxf(v, dpp_f32<kDppRow[1]>(v));
  v = fmaxf(v, dpp_f32<kDppRow[2]>(v));
  return fmaxf(v, dpp_f32<kDppRow[3]>(v));
}
template <int CTRL>
__device__ __forceinline__ void argmax_dpp(float& v, int& i) {
  const float ov = dpp_f32<CTRL>(v);
  const int oi = dpp_i32<CTRL>(i);
  if (ov > v || (ov == v && oi < i)) {
    v = ov;
    i = oi;
  }
}
__device__ __forceinline__ void row_argmax(float& v, int& i) {
  argmax_dpp<kDppRow[0]>(v, i);
  argmax_dpp<kDppRow[1]>(v, i);
  argmax_dpp<kDppRow[2]>(v, i);
  argmax_dpp<kDppRow[3]>(v, i);
}

template <typename T, int VW, int NG>
__global__ __launch_bounds__(kRouterWaves * kWave) void router_kernel(
    const T* __restrict__ x, const T* __restrict__ Wg, const float* __restrict__ bias,
    int d, int E, int k, int norm_topk, float* __restrict__ logits,
    int32_t* __restrict__ e_out, float* __restrict__ w_out, int32_t* __restrict__ rflags,
    float* __restrict__ C, double* __restrict__ ent, int N, float beta) {
  __shared__ double s_part[kRouterWaves][NG][4][kWave];
  __shared__ double s_ent[kRouterWaves][NG][2][16];
  __shared__ int s_bad;
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  const int n = lane & 15, g = lane >> 4;
  // block = (sample, chunk of 16 positions): it never spans two samples
  const int nch = (N + kTokensPerBlock - 1) / kTokensPerBlock;
  const int64_t sb = blockIdx.x / nch;
  const int chunk = blockIdx.x % nch;
  const int64_t t0 = sb * N + int64_t(chunk) * kTokensPerBlock;
  const int nlive = min(kTokensPerBlock, N - chunk * kTokensPerBlock);
  if (threadIdx.x == 0) s_bad = 0;

  // the epilogue token of this lane, and its statistic values (read early)
  const bool live = g + 4 * wv < nlive;
  const int64_t si = live ? int64_t(chunk) * kTokensPerBlock + g + 4 * wv : 0;
  const int64_t te = sb * N + si;
  float c_old[NG];
#pragma unroll
  for (int q = 0; q < NG; ++q) {
    const int e = 16 * q + n;
    c_old[q] = (C != nullptr && live && e < E) ? C[(sb * E + e) * N + si] : 0.0f;
  }

  // ---- logits on the fp64 matrix cores ------------------------------------
  // The wave's quarter of d is walked in groups of 4 VW elements; within a
  // group, MFMA k-row g takes elements g VW .. g VW + VW - 1, so the four
  // lanes of a row read one contiguous 4 VW-element segment per load.
  const int nv = d / (16 * VW);  // vectors per lane
  const int64_t kbase = int64_t(wv) * (d >> 2) + int64_t(g) * VW;
  const T* xp = x + (t0 + min(n, nlive - 1)) * d + kbase;  // A: token row n
  const T* wp[NG];
#pragma unroll
  for (int q = 0; q < NG; ++q) wp[q] = Wg + int64_t(min(16 * q + n, E - 1)) * d + kbase;

  // independent accumulator chains per expert group: four, or two when the
  // expert groups alone give enough independent MFMAs (and registers for
  // two waves per SIMD are wanted)
  constexpr int NCH = NG >= 3 ? 2 : 4;
  f64x4_t acc[NCH][NG];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int q = 0; q < NG; ++q) acc[c][q] = f64x4_t{0.0, 0.0, 0.0, 0.0};
  // chunks of CH vectors, double-buffered: the next chunk's loads are issued
  // before the current chunk's MFMAs
  constexpr int CH = NG == 1 ? 3 : 2;
  typedef typename Vec<T, VW>::raw Raw;
  Raw xa[CH], wa[CH][NG], xb[CH], wb[CH][NG];
  auto load = [&](Raw (&xr)[CH], Raw (&wr)[CH][NG], int c0) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      if (c0 + c < nv) {
        const int64_t o = int64_t(c0 + c) * 4 * VW;
        xr[c] = Vec<T, VW>::load(xp + o);
#pragma unroll
        for (int q = 0; q < NG; ++q) wr[c][q] = Vec<T, VW>::load(wp[q] + o);
      }
    }
  };
  auto compute = [&](const Raw (&xr)[CH], const Raw (&wr)[CH][NG], int c0) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      if (c0 + c >= nv) continue;
      double xv[VW];
      Vec<T, VW>::widen(xr[c], xv);
#pragma unroll
      for (int q = 0; q < NG; ++q) {
        double wv2[VW];
        Vec<T, VW>::widen(wr[c][q], wv2);
#pragma unroll
        for (int u = 0; u < VW; ++u)
          acc[u % NCH][q] =
              __builtin_amdgcn_mfma_f64_16x16x4f64(xv[u], wv2[u], acc[u % NCH][q], 0, 0, 0);
      }
    }
  };
  load(xa, wa, 0);
  for (int c0 = 0; c0 < nv; c0 += 2 * CH) {
    if (c0 + CH < nv) load(xb, wb, c0 + CH);
    compute(xa, wa, c0);
    if (c0 + 2 * CH < nv) load(xa, wa, c0 + 2 * CH);
    if (c0 + CH < nv) compute(xb, wb, c0 + CH);
  }
  // lane l, register r of a 16 x 16 result: token 4 r + l / 16, expert l % 16
#pragma unroll
  for (int q = 0; q < NG; ++q)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      s_part[wv][q][r][lane] = NCH == 4
                                   ? (acc[0][q][r] + acc[1][q][r]) + (acc[2 % NCH][q][r] + acc[3 % NCH][q][r])
                                   : acc[0][q][r] + acc[1][q][r];
  __syncthreads();

  // ---- epilogue: tokens 4 wv + g, register r = wv of every wave's partial --
  float lv[NG];  // fp32 logits of experts 16 q + n (-inf where e >= E)
  bool bad = false;
#pragma unroll
  for (int q = 0; q < NG; ++q) {
    const int e = 16 * q + n;
    double sm = s_part[0][q][wv][lane];
#pragma unroll
    for (int w2 = 1; w2 < kRouterWaves; ++w2) sm += s_part[w2][q][wv][lane];
    if (e < E) {
      if (bias) sm += static_cast<double>(bias[e]);
      lv[q] = static_cast<float>(sm);
      if (live) logits[te * E + e] = lv[q];
      if (!isfinite(lv[q])) bad = true;
      if (lv[q] != lv[q]) lv[q] = -__builtin_huge_valf();  // a NaN logit never wins
    } else {
      lv[q] = -__builtin_huge_valf();
    }
  }
  // group max over the token's experts (softmax shift)
  float mx = lv[0];
#pragma unroll
  for (int q = 1; q < NG; ++q) mx = fmaxf(mx, lv[q]);
  mx = row_max(mx);

  // top-k: k rounds of a group argmax over the untaken experts
  uint64_t taken = 0;
  int sel[8];
  for (int p = 0; p < k; ++p) {
    float cv = -__builtin_huge_valf();
    int ci = 1 << 20;
#pragma unroll
    for (int q = 0; q < NG; ++q) {  // ascending ids: a later equal value never replaces
      const int e = 16 * q + n;
      if (e < E && !((taken >> e) & 1ull) && (ci == (1 << 20) || lv[q] > cv)) {
        cv = lv[q];
        ci = e;
      }
    }
    row_argmax(cv, ci);
    if (ci >= E) ci = __builtin_ctzll(~taken);  // defensive: cannot happen for k <= E
    sel[p] = ci;
    taken |= 1ull << ci;
  }

  // gate: softmax in fp64 over the top-k (renormalised) or all experts; the
  // lane holding a selected expert writes its id and weight
  double z[NG];
  double part = 0.0;
#pragma unroll
  for (int q = 0; q < NG; ++q) {
    const int e = 16 * q + n;
    const bool in_den = e < E && (norm_topk ? ((taken >> e) & 1ull) != 0 : true);
    z[q] = in_den ? exp(static_cast<double>(lv[q]) - static_cast<double>(mx)) : 0.0;
    part += z[q];
  }
  part = row_sum_f64(part);
  if (live) {
    for (int p = 0; p < k; ++p) {
#pragma unroll
      for (int q = 0; q < NG; ++q) {
        if (sel[p] == 16 * q + n) {
          e_out[te * k + p] = sel[p];
          w_out[te * k + p] = static_cast<float>(z[q] / part);
        }
      }
    }
  }

  // expert statistic C_{e,i} <- f32(f32(beta*C) + f32(1-beta)*[e in B_i]),
  // and for the entropy of the statistic (Sec. 4.3) this chunk's sums
  // sum_i C_i and sum_i C_i log C_i per expert (fp64, exact products of
  // the stored fp32 value and its fp64 logarithm; C_i = 0 adds 0): the
  // token pairs (g, g ^ 1), then (g, g ^ 2), then the four waves in order
  if (C != nullptr) {
    double sv[NG], av[NG];
#pragma unroll
    for (int q = 0; q < NG; ++q) {
      const int e = 16 * q + n;
      sv[q] = 0.0;
      av[q] = 0.0;
      if (e < E && live) {
        float c = __fmul_rn(beta, c_old[q]);
        if ((taken >> e) & 1ull) c = __fadd_rn(c, __fsub_rn(1.0f, beta));
        C[(sb * E + e) * N + si] = c;
        if (c > 0.0f) {
          const double cd = static_cast<double>(c);
          sv[q] = cd;
          av[q] = __dmul_rn(cd, log(cd));
        }
      }
      sv[q] += __shfl_xor(sv[q], 16, kWave);
      av[q] += __shfl_xor(av[q], 16, kWave);
      sv[q] += __shfl_xor(sv[q], 32, kWave);
      av[q] += __shfl_xor(av[q], 32, kWave);
      if (g == 0) {
        s_ent[wv][q][0][n] = sv[q];
        s_ent[wv][q][1][n] = av[q];
      }
    }
  }
  if (bad && live) s_bad = 1;
  __syncthreads();
  if (threadIdx.x == 0) rflags[blockIdx.x] = s_bad;
  if (C != nullptr && wv == 0 && g < 2) {
    // lane (g, n): sum (g = 0) or sum of C log C (g = 1) of experts 16 q + n
#pragma unroll
    for (int q = 0; q < NG; ++q) {
      const int e = 16 * q + n;
      if (e < E)
        ent[((sb * E + e) * nch + chunk) * 2 + g] =
            (s_ent[0][q][g][n] + s_ent[1][q][g][n]) + (s_ent[2][q][g][n] + s_ent[3][q][g][n]);
    }
  }
}

template <typename T, int VW>
hipError_t launch_vw(const Shape& s, const void* x, const void* W_r, const float* b_r,
                     int norm_topk, float beta, float* C, double* ent, const Buffers& b,
                     hipStream_t st) {
  const dim3 grid(router_blocks(s)), block(kRouterWaves * kWave);
  const int ng = (s.E + 15) / 16;
#define MOECA_ROUTER(NGV)                                                                 \
  launch_kernel(&router_kernel<T, VW, NGV>, grid, block, 0, st, static_cast<const T*>(x), \
                static_cast<const T*>(W_r), b_r, s.d, s.E, s.k, norm_topk,                \
                b.logits, b.e_t, b.w_t, b.rflags, C, ent, s.N, beta)
  switch (ng) {
    case 1: MOECA_ROUTER(1); break;
    case 2: MOECA_ROUTER(2); break;
    case 3: MOECA_ROUTER(3); break;
    case 4: MOECA_ROUTER(4); break;
    default: return hipErrorInvalidValue;
  }
#undef MOECA_ROUTER
  return hipGetLastError();
}

}  // namespace

int router_blocks(const Shape& s) {
  return s.B * ((s.N + kTokensPerBlock - 1) / kTokensPerBlock);
}

// d is a multiple of 64 (checked at layer creation), so each lane's quarter
// (d / 16 elements) is a multiple of 4; bf16 rows use 16-byte loads when it
// is a multiple of 8.  E <= 64 and k <= 8 (four expert groups of 16 lanes).
hipError_t launch_router(const Shape& s, const void* x, const void* W_r, const float* b_r,
                         int norm_topk, float beta, bool update_stat, const Buffers& b,
                         hipStream_t st) {
  if (s.d % 64 != 0 || s.E > 64 || s.k > 8 || s.k > s.E) return hipErrorInvalidValue;
  float* C = update_stat ? b.stat : nullptr;
  double* ent = update_stat ? b.ent : nullptr;
  if (s.bf16) {
    if ((s.d / 16) % 8 == 0)
      return launch_vw<uint16_t, 8>(s, x, W_r, b_r, norm_topk, beta, C, ent, b, st);
    return launch_vw<uint16_t, 4>(s, x, W_r, b_r, norm_topk, beta, C, ent, b, st);
  }
  return launch_vw<float, 4>(s, x, W_r, b_r, norm_topk, beta, C, ent, b, st);
}

}  // namespace moeca
