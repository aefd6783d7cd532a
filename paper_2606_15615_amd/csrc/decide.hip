// Decision path of a cache step: expert statistic and thresholds (Sec. 4.3),
// branch matching and score (Sec. 4.2), the recomputation set (Sec. 4.2),
// slot assignment and the sync mask (Sec. 4.1), and the per-expert lists of
// recomputed branches that drive the grouped expert FFN.
//
// Everything here decides integers (masks, slots, list order), so the
// arithmetic is fixed: fp32 operations are the correctly rounded intrinsics
// in the order the method states them (this file is built without FMA
// contraction), and reductions are fp64 sums of exact values rounded once.
// No atomic operation decides an order: counts use integer atomics only.
#include "common.h"
#include "internal.h"

#pragma clang fp contract(off)

namespace moeca {
namespace {

// ---------------------------------------------------------------------------
// EMA statistic, normalised entropy and per-expert threshold, one block per
// (sample, expert).
//   C_{e,i} <- f32(f32(beta*C) + f32(1-beta)*[e in B_i])     (Sec. 4.3 EMA eq.)
//   P(i) = C_i / sum C,  H = -sum P log P,  Hbar = clamp(H / log N, 0, 1)
//   tau_e = tau0 * (1 + alpha * (2*Hbar - 1))                 (Sec. 4.3)
// ---------------------------------------------------------------------------
constexpr int kStatThreads = 256;

__global__ __launch_bounds__(kStatThreads) void stat_kernel(
    const int32_t* __restrict__ e_t, float* __restrict__ C, int N, int E, int k, float beta,
    float tau0, float alpha, float* __restrict__ hbar, float* __restrict__ tau) {
  __shared__ double s_red[kStatThreads / kWave];
  const int b = blockIdx.x / E;
  const int e = blockIdx.x % E;
  float* Cr = C + (int64_t(b) * E + e) * N;
  const int32_t* eb = e_t + int64_t(b) * N * k;
  const float c1 = __fsub_rn(1.0f, beta);

  double part = 0.0;
  for (int i = threadIdx.x; i < N; i += kStatThreads) {
    bool hit = false;
    for (int p = 0; p < k; ++p) hit |= (eb[int64_t(i) * k + p] == e);
    float c = __fmul_rn(beta, Cr[i]);
    if (hit) c = __fadd_rn(c, c1);
    Cr[i] = c;
    part += static_cast<double>(c);
  }
  const double S = block_sum_f64<kStatThreads / kWave>(part, s_red);

  double hpart = 0.0;
  if (S > 0.0) {
    for (int i = threadIdx.x; i < N; i += kStatThreads) {
      const float c = Cr[i];
      if (c > 0.0f) {
        const double P = static_cast<double>(c) / S;
        hpart -= P * log(P);
      }
    }
  }
  const double H = block_sum_f64<kStatThreads / kWave>(hpart, s_red);

  if (threadIdx.x == 0) {
    float hb = 0.0f;
    if (N > 1 && S > 0.0) {
      double v = H / log(static_cast<double>(N));
      v = v < 0.0 ? 0.0 : (v > 1.0 ? 1.0 : v);
      hb = static_cast<float>(v);
    }
    const float centred = __fsub_rn(__fmul_rn(2.0f, hb), 1.0f);
    const float scaled = __fmul_rn(alpha, centred);
    hbar[b * E + e] = hb;
    tau[b * E + e] = __fmul_rn(tau0, __fadd_rn(1.0f, scaled));
  }
}

// ---------------------------------------------------------------------------
// Matching and branch score, one thread per branch (cache steps only).
//   q(p): cached slot with the same expert, or -1           (Sec. 4.2)
//   Delta = |w_p - w_c[q]|,  o = n_c[q] / f32(sum_j n_c[j]),
//   s = (w_p + lambda1*Delta) + lambda2*o,  m = s - tau_{b,e_p}
// ---------------------------------------------------------------------------
constexpr int kScoreThreads = 256;

__global__ __launch_bounds__(kScoreThreads) void score_kernel(
    const int32_t* __restrict__ e_t, const float* __restrict__ w_t,
    const int32_t* __restrict__ e_c, const float* __restrict__ w_c,
    const float* __restrict__ n_c, const float* __restrict__ tau, int64_t nbr, int N, int E,
    int k, float lambda1, float lambda2, int32_t* __restrict__ q_out,
    float* __restrict__ margin) {
  const int64_t f = int64_t(blockIdx.x) * kScoreThreads + threadIdx.x;
  if (f >= nbr) return;
  const int64_t tok = f / k;
  const int b = static_cast<int>(tok / N);
  const int e = e_t[f];
  const float w = w_t[f];
  const int32_t* ec = e_c + tok * k;
  const float* wc = w_c + tok * k;
  const float* nc = n_c + tok * k;
  int q = -1;
  double den = 0.0;
  for (int j = 0; j < k; ++j) {
    const int ej = ec[j];
    if (ej >= 0) den += static_cast<double>(nc[j]);
    if (q < 0 && ej >= 0 && ej == e) q = j;
  }
  float m = __int_as_float(0x7f800000);  // +inf: unmatched, always recomputed
  if (q >= 0) {
    const float denf = static_cast<float>(den);
    const float delta = fabsf(__fsub_rn(w, wc[q]));
    const float o = denf > 0.0f ? __fdiv_rn(nc[q], denf) : 0.0f;
    float s = __fadd_rn(w, __fmul_rn(lambda1, delta));
    s = __fadd_rn(s, __fmul_rn(lambda2, o));
    m = __fsub_rn(s, tau[b * E + e]);
  }
  q_out[f] = q;
  margin[f] = m;
}

// ---------------------------------------------------------------------------
// Recomputation set, slots, sync mask and per-expert counts; one block per
// sample.
//   full step : R = all, sigma(p) = p
//   threshold : R = unmatched U {m > 0}                    (Sec. 4.2)
//   ratio     : R = unmatched U the first max(0, K_b - |U|) matched branches
//               by (m desc, flat id asc), found with an MSB-first radix select
//               on the 64-bit key (order(m) << 32 | ~id): keys are unique, so
//               exactly that many keys are >= the selected one.
//   slots     : matched p keep q(p); unmatched p (ascending) take the free
//               slots in ascending order
// ---------------------------------------------------------------------------
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;

__device__ __forceinline__ uint64_t branch_key(float m, int j) {
  return (static_cast<uint64_t>(f32_order_key(m)) << 32) | static_cast<uint32_t>(~j);
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(
    const int32_t* __restrict__ q, const float* __restrict__ margin,
    const int32_t* __restrict__ e_t, int N, int E, int k, int mode, int budget,
    uint8_t* __restrict__ mask, int32_t* __restrict__ sigma, uint8_t* __restrict__ sync,
    int32_t* __restrict__ cnt_bs, int32_t* __restrict__ stats_bs) {
  __shared__ int s_hist[256];
  __shared__ int s_wtot[kSelWaves];
  __shared__ int s_cnt[64];
  __shared__ int s_unmatched, s_matched, s_recompute, s_sync;
  __shared__ unsigned long long s_prefix;
  __shared__ int s_remaining;

  const int b = blockIdx.x;
  const int nb = N * k;
  const int64_t base = int64_t(b) * nb;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wv = tid / kWave;

  if (tid < 64) s_cnt[tid] = 0;
  if (tid == 0) {
    s_unmatched = 0;
    s_matched = 0;
    s_recompute = 0;
    s_sync = 0;
    s_prefix = 0ull;
  }
  __syncthreads();

  // 1. count unmatched / matched branches of the sample
  if (mode != kSelFull) {
    int u = 0;
    for (int j = tid; j < nb; j += kSelThreads) u += (q[base + j] < 0) ? 1 : 0;
    u = wave_sum_i32(u);
    if (lane == 0) atomicAdd(&s_unmatched, u);
    __syncthreads();
    if (tid == 0) s_matched = nb - s_unmatched;
    __syncthreads();
  }

  // 2. ratio mode: find the key of the need-th best matched branch
  int need = 0;
  bool take_all_matched = false;
  if (mode == kSelRatio) {
    need = budget - s_unmatched;
    if (need < 0) need = 0;
    if (need >= s_matched) take_all_matched = true;
    if (need > 0 && !take_all_matched) {
      if (tid == 0) s_remaining = need;
      __syncthreads();
      for (int shift = 56; shift >= 0; shift -= 8) {
        // prefix and remaining are read here and written only after the two
        // barriers below, so every thread sees this pass's values.
        const uint64_t prefix = s_prefix;
        const int rem = s_remaining;
        if (tid < 256) s_hist[tid] = 0;
        __syncthreads();
        const uint64_t hi_mask = (shift == 56) ? 0ull : (~0ull << (shift + 8));
        for (int j = tid; j < nb; j += kSelThreads) {
          if (q[base + j] < 0) continue;
          const uint64_t key = branch_key(margin[base + j], j);
          if (((key ^ prefix) & hi_mask) == 0ull)
            atomicAdd(&s_hist[(key >> shift) & 255ull], 1);
        }
        __syncthreads();
        // suffix sums over the 256 bins (bin 255 first) by the first 4 waves
        int h = 0, incl = 0;
        if (tid < 256) {
          const int bin = 255 - tid;  // tid 0 holds the top bin
          h = s_hist[bin];
          incl = h;
#pragma unroll
          for (int o = 1; o < kWave; o <<= 1) {
            const int v = __shfl_up(incl, o, kWave);
            if (lane >= o) incl += v;
          }
          if (lane == kWave - 1) s_wtot[wv] = incl;
        }
        __syncthreads();
        if (tid < 256) {
          for (int w2 = 0; w2 < wv; ++w2) incl += s_wtot[w2];
          const int excl = incl - h;
          if (h > 0 && excl < rem && rem <= incl) {
            s_prefix = prefix | (static_cast<uint64_t>(255 - tid) << shift);
            s_remaining = rem - excl;
          }
        }
        __syncthreads();
      }
    }
  }
  const uint64_t thr = s_prefix;

  // 3. mask
  for (int j = tid; j < nb; j += kSelThreads) {
    bool r;
    if (mode == kSelFull) {
      r = true;
    } else {
      const bool matched = q[base + j] >= 0;
      if (!matched) {
        r = true;
      } else if (mode == kSelThreshold) {
        r = margin[base + j] > 0.0f;
      } else if (take_all_matched) {
        r = true;
      } else if (need == 0) {
        r = false;
      } else {
        r = branch_key(margin[base + j], j) >= thr;
      }
    }
    mask[base + j] = r ? 1 : 0;
    if (r) atomicAdd(&s_cnt[e_t[base + j]], 1);
  }
  __syncthreads();

  // 4. per token: sync flag and slots
  int rec = 0, syn = 0;
  for (int i = tid; i < N; i += kSelThreads) {
    const int64_t t0 = base + int64_t(i) * k;
    bool any = false;
    uint32_t taken = 0;
    if (mode != kSelFull) {
      for (int p = 0; p < k; ++p) {
        const int qp = q[t0 + p];
        if (qp >= 0) taken |= 1u << qp;
      }
    }
    for (int p = 0; p < k; ++p) {
      const bool r = mask[t0 + p] != 0;
      any |= r;
      rec += r ? 1 : 0;
      int sg;
      if (mode == kSelFull) {
        sg = p;
      } else {
        const int qp = q[t0 + p];
        if (qp >= 0) {
          sg = qp;
        } else {
          sg = 0;
          while ((taken >> sg) & 1u) ++sg;
          taken |= 1u << sg;
        }
      }
      sigma[t0 + p] = sg;
    }
    sync[int64_t(b) * N + i] = any ? 1 : 0;
    syn += any ? 1 : 0;
  }
  rec = wave_sum_i32(rec);
  syn = wave_sum_i32(syn);
  if (lane == 0) {
    atomicAdd(&s_recompute, rec);
    atomicAdd(&s_sync, syn);
  }
  __syncthreads();
  if (tid < E) cnt_bs[b * E + tid] = s_cnt[tid];
  if (tid == 0) {
    stats_bs[b * 4 + 0] = s_recompute;
    stats_bs[b * 4 + 1] = (mode == kSelFull) ? 0 : s_unmatched;
    stats_bs[b * 4 + 2] = (mode == kSelFull) ? 0 : s_matched;
    stats_bs[b * 4 + 3] = s_sync;
  }
}

// ---------------------------------------------------------------------------
// Per-expert lists of recomputed branches, ascending flat id within each
// expert; one block per sample.  Each block derives its write base per
// expert from the [B][E] count table, then walks its branches in flat order
// in chunks of 1024 and ranks them with wave ballots (stable, no atomics).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kSelThreads) void lists_kernel(
    const uint8_t* __restrict__ mask, const int32_t* __restrict__ e_t,
    const int32_t* __restrict__ cnt_bs, int B, int N, int E, int k, int tm, int nt_up,
    int nt_down, int32_t* __restrict__ off, int32_t* __restrict__ tiles,
    int32_t* __restrict__ list, int32_t* __restrict__ pos) {
  __shared__ int s_base[64];
  __shared__ int s_run[64];
  __shared__ int s_wcnt[kSelWaves][64];
  const int b = blockIdx.x;
  const int nb = N * k;
  const int64_t base = int64_t(b) * nb;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wv = tid / kWave;

  // per expert: total count and count in samples before this one
  if (tid < E) {
    int tot = 0, below = 0;
    for (int b2 = 0; b2 < B; ++b2) {
      const int c = cnt_bs[b2 * E + tid];
      tot += c;
      if (b2 < b) below += c;
    }
    s_base[tid] = below;
    s_run[tid] = tot;
  }
  __syncthreads();
  if (tid == 0) {
    int acc = 0, tu = 0, td = 0;
    for (int e = 0; e < E; ++e) {
      const int tot = s_run[e];
      if (b == 0) {
        off[e] = acc;
        tiles[e] = tu;
        tiles[E + 1 + e] = td;
      }
      s_base[e] += acc;
      s_run[e] = 0;
      acc += tot;
      const int mt = (tot + tm - 1) / tm;
      tu += mt * nt_up;
      td += mt * nt_down;
    }
    if (b == 0) {
      off[E] = acc;
      tiles[E] = tu;
      tiles[2 * E + 1] = td;
    }
  }
  __syncthreads();

  for (int c0 = 0; c0 < nb; c0 += kSelThreads) {
    const int j = c0 + tid;
    const bool in = j < nb;
    const bool sel = in && mask[base + j] != 0;
    const int e = sel ? e_t[base + j] : -1;
    int rank = 0;
    for (int ee = 0; ee < E; ++ee) {
      const uint64_t bal = __ballot(e == ee);
      if (lane == 0) s_wcnt[wv][ee] = __popcll(bal);
      if (e == ee) rank = lane_rank(bal);
    }
    __syncthreads();
    if (sel) {
      int before = 0;
      for (int w2 = 0; w2 < wv; ++w2) before += s_wcnt[w2][e];
      const int idx = s_base[e] + s_run[e] + before + rank;
      list[idx] = static_cast<int32_t>(base + j);
      pos[base + j] = idx;
    } else if (in) {
      pos[base + j] = -1;
    }
    __syncthreads();
    if (tid < E) {
      int tot = 0;
      for (int w2 = 0; w2 < kSelWaves; ++w2) tot += s_wcnt[w2][tid];
      s_run[tid] += tot;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Cache reset: empty slots, zero statistic.
// ---------------------------------------------------------------------------
__global__ void reset_kernel(int32_t* __restrict__ e_c, float* __restrict__ w_c,
                             float* __restrict__ n_c, int64_t nbr, float* __restrict__ C,
                             int64_t nstat) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < nbr; i += stride) {
    e_c[i] = -1;
    w_c[i] = 0.0f;
    n_c[i] = 0.0f;
  }
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < nstat; i += stride)
    C[i] = 0.0f;
}

}  // namespace

hipError_t launch_stat(const Shape& s, float beta, float tau0, float alpha, const Buffers& b,
                       hipStream_t st) {
  stat_kernel<<<dim3(s.B * s.E), dim3(kStatThreads), 0, st>>>(b.e_t, b.stat, s.N, s.E, s.k,
                                                                beta, tau0, alpha, b.hbar, b.tau);
  return hipGetLastError();
}

hipError_t launch_score(const Shape& s, float lambda1, float lambda2, const Buffers& b,
                        hipStream_t st) {
  const int64_t n = s.branches();
  const dim3 grid(static_cast<unsigned>((n + kScoreThreads - 1) / kScoreThreads));
  score_kernel<<<grid, dim3(kScoreThreads), 0, st>>>(b.e_t, b.w_t, b.e_c, b.w_c, b.n_c, b.tau,
                                                      n, s.N, s.E, s.k, lambda1, lambda2, b.q,
                                                      b.margin);
  return hipGetLastError();
}

hipError_t launch_select(const Shape& s, int sel_mode, int budget, const Buffers& b,
                         hipStream_t st) {
  select_kernel<<<dim3(s.B), dim3(kSelThreads), 0, st>>>(b.q, b.margin, b.e_t, s.N, s.E, s.k,
                                                         sel_mode, budget, b.mask, b.sigma,
                                                         b.sync, b.cnt_bs, b.stats_bs);
  return hipGetLastError();
}

hipError_t launch_lists(const Shape& s, const FfnPlan& plan, const Buffers& b, hipStream_t st) {
  lists_kernel<<<dim3(s.B), dim3(kSelThreads), 0, st>>>(
      b.mask, b.e_t, b.cnt_bs, s.B, s.N, s.E, s.k, plan.tm, s.d_ff / plan.tn_up,
      s.d / plan.tn_down, b.off, b.tiles, b.list, b.pos);
  return hipGetLastError();
}

hipError_t launch_reset(const Shape& s, const Buffers& b, hipStream_t st) {
  reset_kernel<<<dim3(256), dim3(256), 0, st>>>(b.e_c, b.w_c, b.n_c, s.branches(), b.stat,
                                                 int64_t(s.B) * s.E * s.N);
  return hipGetLastError();
}

}  // namespace moeca
