// Decision path of a cache step: entropy-based thresholds (Sec. 4.3),
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
// Thresholds, matching, branch scores, recomputation set, slots, sync mask
// and per-expert counts; one block per sample, each thread holding up to R
// of the sample's branches (j = tid + 1024 r) in registers.
//   entropy (when the router advanced the statistic C in this step; one
//   wave per expert, fixed-order fp64 sums, Sec. 4.3):
//     S = sum_i C_i,  H = -sum_{C_i > 0} (C_i / S) (log C_i - log S),
//     Hbar = clamp(H / log N, 0, 1),  tau_e = tau0 * (1 + alpha * (2*Hbar - 1))
//   with log C_i stored by the router; log(C_i / S) is formed as the
//   difference of the two logarithms, so one occupied position gives H = 0
//   exactly.
//   q(p): cached slot with the same expert, or -1           (Sec. 4.2)
//   Delta = |w_p - w_c[q]|,  o = n_c[q] / f32(sum_j n_c[j]),
//   s = (w_p + lambda1*Delta) + lambda2*o,  m = s - tau_{b,e_p}
//   full step : R = all, sigma(p) = p
//   threshold : R = unmatched U {m > 0}                    (Sec. 4.2)
//   ratio     : R = unmatched U the first max(0, K_b - |U|) matched branches
//               by (m desc, flat id asc): an MSB-first radix select on the
//               order-preserving 32-bit key of m, then the lowest flat ids
//               among the keys equal to the selected one.
//   slots     : matched p keep q(p); unmatched p (ascending) take the free
//               slots in ascending order
// ---------------------------------------------------------------------------
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;

template <int R>
__global__ __launch_bounds__(kSelThreads) void decide_kernel(
    const int32_t* __restrict__ e_t, const float* __restrict__ w_t,
    const int32_t* __restrict__ e_c, const float* __restrict__ w_c,
    const float* __restrict__ n_c, const float* __restrict__ C, const double* __restrict__ logc,
    int with_stat, float tau0, float alpha, float* __restrict__ hbar, float* __restrict__ tau,
    int N, int E, int k, int mode, int budget, float lambda1, float lambda2,
    int32_t* __restrict__ q_out,
    float* __restrict__ margin, uint8_t* __restrict__ mask, int32_t* __restrict__ sigma,
    uint8_t* __restrict__ sync, int32_t* __restrict__ cnt_bs, int32_t* __restrict__ stats_bs) {
  extern __shared__ __attribute__((aligned(16))) unsigned char s_dyn[];
  int8_t* s_q = reinterpret_cast<int8_t*>(s_dyn);            // [N*k] matched slot or -1
  uint8_t* s_mask = reinterpret_cast<uint8_t*>(s_dyn) + N * k; // [N*k]
  __shared__ int s_hist[2][256];
  __shared__ int s_cnt[64];
  __shared__ float s_tau[64];
  __shared__ int s_tcnt[R][kSelWaves];
  __shared__ int s_unmatched, s_recompute, s_sync;
  __shared__ unsigned s_bin;
  __shared__ int s_remaining;

  const int b = blockIdx.x;
  const int nb = N * k;
  const int64_t base = int64_t(b) * nb;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wv = tid / kWave;

  if (tid < 64) {
    s_cnt[tid] = 0;
    if (tid < E && !with_stat) s_tau[tid] = tau[b * E + tid];
  }
  if (with_stat) {
    // 0. entropy of the statistic and the threshold, one wave per expert
    for (int e = wv; e < E; e += kSelWaves) {
      const float* Cr = C + (int64_t(b) * E + e) * N;
      const double* Lr = logc + (int64_t(b) * E + e) * N;
      // positions lane + 64 v of each 1024-position chunk, all loads of a
      // chunk (C and log C) issued together; four partial sums per lane
      constexpr int PER = 16;
      double s4[4] = {0.0, 0.0, 0.0, 0.0};
      double h4[4] = {0.0, 0.0, 0.0, 0.0};
      float c[PER];
      double lc[PER];
      auto load_chunk = [&](int i0) __attribute__((always_inline)) {
#pragma unroll
        for (int v = 0; v < PER; ++v) {
          const int i = i0 + lane + v * kWave;
          c[v] = i < N ? Cr[i] : 0.0f;
          lc[v] = i < N ? Lr[i] : 0.0;
        }
      };
      for (int i0 = 0; i0 < N; i0 += PER * kWave) {
        load_chunk(i0);
#pragma unroll
        for (int v = 0; v < PER; ++v) s4[v & 3] += static_cast<double>(c[v]);
      }
      const double S = wave_sum_f64((s4[0] + s4[1]) + (s4[2] + s4[3]));
      if (S > 0.0) {
        const double logS = log(S);
        for (int i0 = 0; i0 < N; i0 += PER * kWave) {
          if (N > PER * kWave) load_chunk(i0);  // a single chunk is still in registers
#pragma unroll
          for (int v = 0; v < PER; ++v)
            if (c[v] > 0.0f) h4[v & 3] -= (static_cast<double>(c[v]) / S) * (lc[v] - logS);
        }
      }
      const double Hs = wave_sum_f64((h4[0] + h4[1]) + (h4[2] + h4[3]));
      if (lane == 0) {
        float hb = 0.0f;
        if (N > 1 && S > 0.0) {
          double v = Hs / log(static_cast<double>(N));
          v = v < 0.0 ? 0.0 : (v > 1.0 ? 1.0 : v);
          hb = static_cast<float>(v);
        }
        const float centred = __fsub_rn(__fmul_rn(2.0f, hb), 1.0f);
        const float th = __fmul_rn(tau0, __fadd_rn(1.0f, __fmul_rn(alpha, centred)));
        hbar[b * E + e] = hb;
        tau[b * E + e] = th;
        s_tau[e] = th;
      }
    }
  }
  if (tid < 256) s_hist[0][tid] = 0;
  if (tid == 0) {
    s_unmatched = 0;
    s_recompute = 0;
    s_sync = 0;
  }
  __syncthreads();

  // 1. matching and scores (cache steps); every operand of a branch is
  // loaded before any is used
  int qv[R];
  float mv[R];
  int ev[R];
  int unmatched = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = tid + kSelThreads * r;
    qv[r] = -1;
    mv[r] = __int_as_float(0x7f800000);  // +inf: unmatched, always recomputed
    ev[r] = 0;
    if (j < nb) {
      const int64_t f = base + j;
      const int e = e_t[f];
      ev[r] = e;
      if (mode != kSelFull) {
        const int64_t c0 = base + (j / k) * k;  // the token's first slot
        const float w = w_t[f];
        int ejs[8];
        float ncs[8], wcs[8];
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          if (jj < k) {
            ejs[jj] = e_c[c0 + jj];
            ncs[jj] = n_c[c0 + jj];
            wcs[jj] = w_c[c0 + jj];
          }
        }
        int q = -1;
        double den = 0.0;
        float ncq = 0.0f, wcq = 0.0f;
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          if (jj < k) {
            if (ejs[jj] >= 0) den += static_cast<double>(ncs[jj]);
            if (q < 0 && ejs[jj] >= 0 && ejs[jj] == e) {
              q = jj;
              ncq = ncs[jj];
              wcq = wcs[jj];
            }
          }
        }
        if (q >= 0) {
          const float denf = static_cast<float>(den);
          const float delta = fabsf(__fsub_rn(w, wcq));
          const float o = denf > 0.0f ? __fdiv_rn(ncq, denf) : 0.0f;
          float sc = __fadd_rn(w, __fmul_rn(lambda1, delta));
          sc = __fadd_rn(sc, __fmul_rn(lambda2, o));
          mv[r] = __fsub_rn(sc, s_tau[e]);
        } else {
          ++unmatched;
        }
        qv[r] = q;
        q_out[f] = q;
        margin[f] = mv[r];
      }
    }
  }
  if (mode != kSelFull) {
    unmatched = wave_sum_i32(unmatched);
    if (lane == 0) atomicAdd(&s_unmatched, unmatched);
  }
  __syncthreads();
  const int n_unmatched = s_unmatched;
  const int n_matched = mode == kSelFull ? 0 : nb - n_unmatched;

  // 2. ratio mode: the need-th best matched branch.  Four 8-bit radix
  // passes (most significant first) find the margin key T with fewer than
  // `need` matched keys above it and at least `need` at or above it; of the
  // keys equal to T the lowest flat ids are taken (rank by ballots).
  int need = 0;
  bool take_all_matched = false;
  uint32_t thr = 0;
  int tie_rem = 0;
  bool tie_take[R];
#pragma unroll
  for (int r = 0; r < R; ++r) tie_take[r] = false;
  if (mode == kSelRatio) {
    need = budget - n_unmatched;
    if (need < 0) need = 0;
    if (need >= n_matched) take_all_matched = true;
    if (need > 0 && !take_all_matched) {
      uint32_t mk[R];
#pragma unroll
      for (int r = 0; r < R; ++r) mk[r] = f32_order_key(mv[r]);
      uint32_t prefix = 0;
      int rem = need;
#pragma unroll
      for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        int* hist = s_hist[pass & 1];
        const uint32_t hi_mask = pass == 0 ? 0u : (~0u << (shift + 8));
        // histogram of this digit over the matched keys that share the
        // prefix: the (at most two) most frequent bins of a wave are added
        // once by one lane, the remaining lanes add their own
#pragma unroll
        for (int r = 0; r < R; ++r) {
          bool part = qv[r] >= 0 && ((mk[r] ^ prefix) & hi_mask) == 0u;
          const int bin = static_cast<int>((mk[r] >> shift) & 255u);
#pragma unroll
          for (int it = 0; it < 2; ++it) {
            const uint64_t todo = __ballot(part);
            if (todo == 0ull) break;
            const int leader = __builtin_ctzll(todo);
            const int lb = __builtin_amdgcn_readlane(bin, leader);
            const uint64_t same = __ballot(part && bin == lb);
            if (lane == leader) atomicAdd(&hist[lb], __popcll(same));
            if (bin == lb) part = false;
          }
          if (part) atomicAdd(&hist[bin], 1);
        }
        __syncthreads();
        if (wv == 0) {
          // lane l holds bins 255 - 4l .. 252 - 4l (descending)
          int c[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) c[u] = hist[255 - 4 * lane - u];
          const int tot = c[0] + c[1] + c[2] + c[3];
          int incl = tot;
#pragma unroll
          for (int o = 1; o < kWave; o <<= 1) {
            const int v = __shfl_up(incl, o, kWave);
            if (lane >= o) incl += v;
          }
          int run = incl - tot;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            if (c[u] > 0 && run < rem && rem <= run + c[u]) {
              s_bin = static_cast<unsigned>(255 - 4 * lane - u);
              s_remaining = rem - run;
            }
            run += c[u];
          }
        } else if (wv == 1) {
#pragma unroll
          for (int u = 0; u < 4; ++u) s_hist[(pass + 1) & 1][4 * lane + u] = 0;
        }
        __syncthreads();
        prefix |= static_cast<uint32_t>(s_bin) << shift;
        rem = s_remaining;
      }
      thr = prefix;
      tie_rem = rem;
      // keys equal to T: take the tie_rem lowest flat ids (j = tid + 1024 r,
      // so the order is r-major, then wave, then lane)
      uint64_t tb[R];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        tb[r] = __ballot(qv[r] >= 0 && mk[r] == thr);
        if (lane == 0) s_tcnt[r][wv] = __popcll(tb[r]);
      }
      __syncthreads();
      int before = 0;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        int in_r = 0, below = 0;
        for (int w2 = 0; w2 < kSelWaves; ++w2) {
          const int c = s_tcnt[r][w2];
          in_r += c;
          if (w2 < wv) below += c;
        }
        const bool flag = ((tb[r] >> lane) & 1ull) != 0;
        tie_take[r] = flag && before + below + lane_rank(tb[r]) < tie_rem;
        before += in_r;
      }
    }
  }

  // 3. mask and per-expert counts
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = tid + kSelThreads * r;
    bool rc = false;
    if (j < nb) {
      if (mode == kSelFull || qv[r] < 0) {
        rc = true;
      } else if (mode == kSelThreshold) {
        rc = mv[r] > 0.0f;
      } else if (take_all_matched) {
        rc = true;
      } else if (need == 0) {
        rc = false;
      } else {
        const uint32_t mk = f32_order_key(mv[r]);
        rc = mk > thr || tie_take[r];
      }
      mask[base + j] = rc ? 1 : 0;
      s_mask[j] = rc ? 1 : 0;
      s_q[j] = static_cast<int8_t>(qv[r]);
      if (rc) atomicAdd(&s_cnt[ev[r]], 1);
    }
  }
  __syncthreads();

  // 4. per token: sync flag and slots
  int rec = 0, syn = 0;
  for (int i = tid; i < N; i += kSelThreads) {
    bool any = false;
    uint32_t taken = 0;
    if (mode != kSelFull) {
      for (int p = 0; p < k; ++p) {
        const int qp = s_q[i * k + p];
        if (qp >= 0) taken |= 1u << qp;
      }
    }
    for (int p = 0; p < k; ++p) {
      const bool rc = s_mask[i * k + p] != 0;
      any |= rc;
      rec += rc ? 1 : 0;
      int sg;
      if (mode == kSelFull) {
        sg = p;
      } else {
        const int qp = s_q[i * k + p];
        if (qp >= 0) {
          sg = qp;
        } else {
          sg = 0;
          while ((taken >> sg) & 1u) ++sg;
          taken |= 1u << sg;
        }
      }
      sigma[base + int64_t(i) * k + p] = sg;
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
    stats_bs[b * 4 + 1] = mode == kSelFull ? 0 : n_unmatched;
    stats_bs[b * 4 + 2] = n_matched;
    stats_bs[b * 4 + 3] = s_sync;
  }
}

// ---------------------------------------------------------------------------
// Per-expert lists of recomputed branches, ascending flat id within each
// expert; one block per sample, each thread holding up to R of the sample's
// branches (j = tid + 1024 r).  All inputs are loaded first.  Wave 0 turns the
// [B][E] count table into this sample's write base per expert (and, in block
// 0, the expert offsets and the GEMM tile tables); each wave counts and ranks
// its selected branches per expert with ballots; after one barrier every
// branch knows its place: branches of earlier r, then of earlier waves, then
// of lower lanes come first (stable, no atomics).
// ---------------------------------------------------------------------------
// Group table entries E..E+S: the shared experts (Sec. 2.3, shared-expert
// MoE eq.) follow the routed ones in the FFN's grouped GEMM, T rows each (every
// token, in token order), so their offsets and tile prefixes continue the
// routed totals (o rows, tu / td tiles).  Tile tables: up at [0, E+S],
// down at [E+S+1, 2(E+S)+1].
__device__ __forceinline__ void write_shared_groups(int32_t* __restrict__ off,
                                                    int32_t* __restrict__ tiles, int E, int S,
                                                    int T, int tm, int nt_up, int nt_down, int o,
                                                    int tu, int td) {
  const int mts = (T + tm - 1) / tm;
  for (int s2 = 0; s2 <= S; ++s2) {
    off[E + s2] = o + s2 * T;
    tiles[E + s2] = tu + s2 * mts * nt_up;
    tiles[E + S + 1 + E + s2] = td + s2 * mts * nt_down;
  }
}

template <int R>
__global__ __launch_bounds__(kSelThreads) void lists_kernel(
    const uint8_t* __restrict__ mask, const int32_t* __restrict__ e_t,
    const int32_t* __restrict__ cnt_bs, int B, int N, int E, int S, int k, int tm, int nt_up,
    int nt_down, const int32_t* __restrict__ sigma, int32_t* __restrict__ off,
    int32_t* __restrict__ tiles, int32_t* __restrict__ list, int32_t* __restrict__ pos,
    int32_t* __restrict__ row_dst) {
  __shared__ int s_base[64];
  __shared__ int s_wcnt[R][kSelWaves][64];
  const int b = blockIdx.x;
  const int nb = N * k;
  const int64_t base = int64_t(b) * nb;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wv = tid / kWave;

  int ev[R], sg[R];
  bool sel[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = tid + kSelThreads * r;
    sel[r] = false;
    ev[r] = -1;
    sg[r] = 0;
    if (j < nb) {
      sel[r] = mask[base + j] != 0;
      ev[r] = e_t[base + j];
      sg[r] = sigma[base + j];
    }
  }
  if (wv == 0) {
    // lane e: expert e's total over all samples and over the samples before b
    int tot = 0, below = 0;
    if (lane < E) {
      for (int b2 = 0; b2 < B; ++b2) {
        const int c = cnt_bs[b2 * E + lane];
        tot += c;
        if (b2 < b) below += c;
      }
    }
    const int mt = (tot + tm - 1) / tm;
    int o = tot, tu = mt * nt_up, td = mt * nt_down;  // inclusive scans over experts
#pragma unroll
    for (int dd = 1; dd < kWave; dd <<= 1) {
      const int vo = __shfl_up(o, dd, kWave);
      const int vu = __shfl_up(tu, dd, kWave);
      const int vd = __shfl_up(td, dd, kWave);
      if (lane >= dd) {
        o += vo;
        tu += vu;
        td += vd;
      }
    }
    if (lane < E) s_base[lane] = o - tot + below;
    if (b == 0 && lane < E) {
      // exclusive prefixes per expert; the last expert also writes the
      // prefixes of the shared experts and the totals
      off[lane] = o - tot;
      tiles[lane] = tu - mt * nt_up;
      tiles[E + S + 1 + lane] = td - mt * nt_down;
      if (lane == E - 1) write_shared_groups(off, tiles, E, S, B * N, tm, nt_up, nt_down, o, tu, td);
    }
  }
  int rk[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    rk[r] = 0;
    for (int ee = 0; ee < E; ++ee) {
      const bool mine = sel[r] && ev[r] == ee;
      const uint64_t bal = __ballot(mine);
      if (lane == ee) s_wcnt[r][wv][ee] = __popcll(bal);
      if (mine) rk[r] = lane_rank(bal);
    }
  }
  __syncthreads();

#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = tid + kSelThreads * r;
    if (j >= nb) continue;
    const int64_t f = base + j;
    if (!sel[r]) {
      pos[f] = -1;
      continue;
    }
    const int e = ev[r];
    int before = 0;
    for (int r2 = 0; r2 < r; ++r2)
      for (int w2 = 0; w2 < kSelWaves; ++w2) before += s_wcnt[r2][w2][e];
    for (int w2 = 0; w2 < wv; ++w2) before += s_wcnt[r][w2][e];
    const int idx = s_base[e] + before + rk[r];
    list[idx] = static_cast<int32_t>(f);
    pos[f] = idx;
    row_dst[idx] = static_cast<int32_t>((f / k) * k + sg[r]);
  }
}

// ---------------------------------------------------------------------------
// Per-expert lists for samples of more than 8192 branches (the register
// version below would not fit its count table in LDS): ascending flat id
// within each expert; one block per sample.  Each block derives its write base per
// expert from the [B][E] count table, then walks its branches in flat order
// in chunks of 1024 and ranks them with wave ballots (stable, no atomics).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kSelThreads) void lists_chunked_kernel(
    const uint8_t* __restrict__ mask, const int32_t* __restrict__ e_t,
    const int32_t* __restrict__ cnt_bs, int B, int N, int E, int S, int k, int tm, int nt_up,
    int nt_down, const int32_t* __restrict__ sigma, int32_t* __restrict__ off,
    int32_t* __restrict__ tiles, int32_t* __restrict__ list, int32_t* __restrict__ pos,
    int32_t* __restrict__ row_dst) {
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
        tiles[E + S + 1 + e] = td;
      }
      s_base[e] += acc;
      s_run[e] = 0;
      acc += tot;
      const int mt = (tot + tm - 1) / tm;
      tu += mt * nt_up;
      td += mt * nt_down;
    }
    if (b == 0) write_shared_groups(off, tiles, E, S, B * N, tm, nt_up, nt_down, acc, tu, td);
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
      const int64_t f = base + j;
      list[idx] = static_cast<int32_t>(f);
      pos[f] = idx;
      row_dst[idx] = static_cast<int32_t>((f / k) * k + sigma[f]);
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

hipError_t launch_decide(const Shape& s, int sel_mode, int budget, float lambda1, float lambda2,
                         bool with_stat, float tau0, float alpha, const Buffers& b,
                         hipStream_t st) {
  const int nb = s.N * s.k;
  const size_t lds = size_t(2) * nb;
  if (lds > 64 * 1024) return hipErrorInvalidValue;
#define MOECA_DECIDE(RR)                                                                      \
  launch_kernel(&decide_kernel<RR>, dim3(s.B), dim3(kSelThreads), uint32_t(lds), st, b.e_t,   \
                b.w_t, b.e_c, b.w_c, b.n_c, b.stat, b.logc, with_stat ? 1 : 0, tau0, alpha,   \
                b.hbar, b.tau, s.N, s.E, s.k, sel_mode, budget, lambda1, lambda2, b.q,        \
                b.margin, b.mask, b.sigma, b.sync, b.cnt_bs, b.stats_bs)
  if (nb <= 2 * kSelThreads) {
    MOECA_DECIDE(2);
  } else if (nb <= 8 * kSelThreads) {
    MOECA_DECIDE(8);
  } else if (nb <= 32 * kSelThreads) {
    MOECA_DECIDE(32);
  } else {
    return hipErrorInvalidValue;
  }
#undef MOECA_DECIDE
  return hipGetLastError();
}

hipError_t launch_lists(const Shape& s, const FfnPlan& plan, const Buffers& b, hipStream_t st) {
  const int nb = s.N * s.k;
  const int nt_up = (s.up_rows() + plan.tn_up - 1) / plan.tn_up;
  const int nt_down = (s.d + plan.tn_down - 1) / plan.tn_down;
#define MOECA_LISTS(KER)                                                                       \
  launch_kernel(&KER, dim3(s.B), dim3(kSelThreads), 0, st, b.mask, b.e_t, b.cnt_bs, s.B, s.N, \
                s.E, s.S, s.k, plan.tm, nt_up, nt_down, b.sigma, b.off, b.tiles, b.list,      \
                b.pos, b.row_dst)
  if (nb <= 2 * kSelThreads) {
    MOECA_LISTS(lists_kernel<2>);
  } else if (nb <= 8 * kSelThreads) {
    MOECA_LISTS(lists_kernel<8>);
  } else {
    MOECA_LISTS(lists_chunked_kernel);
  }
#undef MOECA_LISTS
  return hipGetLastError();
}

hipError_t launch_reset(const Shape& s, const Buffers& b, hipStream_t st) {
  launch_kernel(&reset_kernel, dim3(256), dim3(256), 0, st, b.e_c, b.w_c, b.n_c, s.branches(),
                b.stat, int64_t(s.B) * s.E * s.N);
  return hipGetLastError();
}

}  // namespace moeca
