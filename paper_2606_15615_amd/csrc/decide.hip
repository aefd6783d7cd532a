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
#include <algorithm>
#include <cmath>

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
//     S = sum_i C_i,  A = sum_i C_i log C_i  (the router's sums per chunk of
//     16 positions, then over the chunks),
//     H = -(1/S) sum_{C_i > 0} C_i (log C_i - log S) = (S log S - A) / S,
//     Hbar = clamp(H / log N, 0, 1),  tau_e = tau0 * (1 + alpha * (2*Hbar - 1))
//   with log N from the host's libm.  One occupied position gives H = 0
//   exactly: S log S and A are then the same rounded product.
//   q(p): cached slot with the same expert, or -1           (Sec. 4.2)
//   Delta = |w_p - w_c[q]|,  o = n_c[q] / f32(sum_j n_c[j]),
//   s = (lambda0*w_p + lambda1*Delta) + lambda2*o,  m = s - tau_{b,e_p}
//   (lambda0 = 1 is the score eq.; other values serve the score-signal
//   ablation of Sec. 5)
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

// Matching and score of one branch (Sec. 4.2): q(p) = the first of the
// token's k cached slots (expert ej, norm nc, gate weight wc) that holds the
// branch's expert e, or -1; for a matched branch the margin
// m = ((lambda0 w + lambda1 Delta) + lambda2 o) - tau_e, with the norm sum of
// o accumulated in fp64 and rounded once.  m is left alone when unmatched.
__device__ __forceinline__ int match_score(int e, float w, const int* ej, const float* nc,
                                           const float* wc, int k, float tau_e, float lambda0,
                                           float lambda1, float lambda2, float& m) {
  int q = -1;
  double den = 0.0;
  float ncq = 0.0f, wcq = 0.0f;
#pragma unroll
  for (int jj = 0; jj < 8; ++jj) {
    if (jj < k) {
      if (ej[jj] >= 0) den += static_cast<double>(nc[jj]);
      if (q < 0 && ej[jj] >= 0 && ej[jj] == e) {
        q = jj;
        ncq = nc[jj];
        wcq = wc[jj];
      }
    }
  }
  if (q >= 0) {
    const float denf = static_cast<float>(den);
    const float delta = fabsf(__fsub_rn(w, wcq));
    const float o = denf > 0.0f ? __fdiv_rn(ncq, denf) : 0.0f;
    float sc = __fadd_rn(__fmul_rn(lambda0, w), __fmul_rn(lambda1, delta));
    sc = __fadd_rn(sc, __fmul_rn(lambda2, o));
    m = __fsub_rn(sc, tau_e);
  }
  return q;
}

// Slots of one token's k branches (Sec. 4.1): a matched branch keeps its
// slot q(p), unmatched ones (ascending p) take the free slots in ascending
// order; on full steps branch p takes slot p.  sq / sm: the token's matched
// slots and recompute flags; writes the k slots to sg and returns whether
// any branch of the token is recomputed (its sync flag), adding the
// recomputed count to rec.
__device__ __forceinline__ bool token_slots(const int8_t* sq, const uint8_t* sm, int k, bool full,
                                            int32_t* __restrict__ sg, int& rec) {
  bool any = false;
  uint32_t taken = 0;
  if (!full) {
    for (int p = 0; p < k; ++p) {
      const int qp = sq[p];
      if (qp >= 0) taken |= 1u << qp;
    }
  }
  for (int p = 0; p < k; ++p) {
    const bool rc = sm[p] != 0;
    any |= rc;
    rec += rc ? 1 : 0;
    int slot;
    if (full) {
      slot = p;
    } else {
      const int qp = sq[p];
      if (qp >= 0) {
        slot = qp;
      } else {
        slot = 0;
        while ((taken >> slot) & 1u) ++slot;
        taken |= 1u << slot;
      }
    }
    sg[p] = slot;
  }
  return any;
}
// Ratio mode: once a digit leaves at most this many keys sharing the
// threshold's prefix, one wave ranks them directly.
constexpr int kDirect = 64;

template <int R>
__global__ __launch_bounds__(kSelThreads) void decide_kernel(
    const int32_t* __restrict__ e_t, const float* __restrict__ w_t,
    const int32_t* __restrict__ e_c, const float* __restrict__ w_c,
    const float* __restrict__ n_c, const double* __restrict__ ent,
    int with_stat, double log_n, float tau0, float alpha, float* __restrict__ hbar,
    float* __restrict__ tau,
    int N, int E, int k, int mode, int budget, float lambda0, float lambda1, float lambda2,
    int32_t* __restrict__ q_out,
    float* __restrict__ margin, uint8_t* __restrict__ mask, int32_t* __restrict__ sigma,
    uint8_t* __restrict__ sync, int32_t* __restrict__ cnt_bs, int32_t* __restrict__ stats_bs,
    int32_t* __restrict__ cnt_ch) {
  extern __shared__ __attribute__((aligned(16))) unsigned char s_dyn[];
  int8_t* s_q = reinterpret_cast<int8_t*>(s_dyn);            // [N*k] matched slot or -1
  uint8_t* s_mask = reinterpret_cast<uint8_t*>(s_dyn) + N * k; // [N*k]
  __shared__ int s_hist[3][256];
  __shared__ int s_cnt[64];
  __shared__ int s_cntr[R][64];  // per 1024-branch chunk of the sample
  __shared__ float s_tau[64];
  __shared__ int s_tcnt[R][kSelWaves];
  // with more than 8 branches per thread: the high 16 bits of each branch's
  // margin key, so that most key decisions need no global read
  __shared__ uint16_t s_k16[R <= 8 ? 1 : R * kSelThreads];
  __shared__ int s_unmatched, s_recompute, s_sync;
  __shared__ uint32_t s_ckey[kDirect];  // ratio mode: the candidates of the last digit
  __shared__ int s_cj[kDirect];
  __shared__ int s_csel[kDirect];
  __shared__ int s_ncand;

  const int b = blockIdx.x;
  const int nb = N * k;
  const int64_t base = int64_t(b) * nb;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wv = tid / kWave;

  // operands of branch j = tid + 1024 r: its expert and gate weight, and the
  // k cached slots of its token (expert, norm, gate weight)
  struct BranchIn {
    int e;
    float w;
    int ej[8];
    float nc[8], wc[8];
  };
  auto load_branch = [&](int r, BranchIn& in) __attribute__((always_inline)) {
    const int j = tid + kSelThreads * r;
    if (j >= nb) return;
    const int64_t f = base + j;
    in.e = e_t[f];
    if (mode == kSelFull) return;
    in.w = w_t[f];
    const int64_t c0 = base + (j / k) * k;  // the token's first slot
    if (k == 8 || k == 4) {
      // 16-byte vectors: the token's slots start at a multiple of k entries
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if (h * 4 < k) {
          const int4 ev = *reinterpret_cast<const int4*>(e_c + c0 + 4 * h);
          const float4 nv = *reinterpret_cast<const float4*>(n_c + c0 + 4 * h);
          const float4 wv4 = *reinterpret_cast<const float4*>(w_c + c0 + 4 * h);
          in.ej[4 * h] = ev.x; in.ej[4 * h + 1] = ev.y; in.ej[4 * h + 2] = ev.z; in.ej[4 * h + 3] = ev.w;
          in.nc[4 * h] = nv.x; in.nc[4 * h + 1] = nv.y; in.nc[4 * h + 2] = nv.z; in.nc[4 * h + 3] = nv.w;
          in.wc[4 * h] = wv4.x; in.wc[4 * h + 1] = wv4.y; in.wc[4 * h + 2] = wv4.z; in.wc[4 * h + 3] = wv4.w;
        }
      }
    } else {
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        if (jj < k) {
          in.ej[jj] = e_c[c0 + jj];
          in.nc[jj] = n_c[c0 + jj];
          in.wc[jj] = w_c[c0 + jj];
        }
      }
    }
  };
  // with two branches per thread their loads are issued before the entropy
  // phase, whose own round trip then covers theirs
  constexpr bool kPre = R <= 2;
  BranchIn pre[kPre ? R : 1];
  if constexpr (kPre) {
#pragma unroll
    for (int r = 0; r < R; ++r) load_branch(r, pre[r]);
  }

  for (int i = tid; i < R * 64; i += kSelThreads) (&s_cntr[0][0])[i] = 0;
  if (tid < 64) {
    s_cnt[tid] = 0;
    if (tid < E && !with_stat) s_tau[tid] = tau[b * E + tid];
  }
  if (with_stat) {
    // 0. entropy of the statistic and the threshold, one wave per expert:
    // the router's per-chunk sums, lane-strided then across the wave
    const int nch = (N + 15) / 16;
    for (int e = wv; e < E; e += kSelWaves) {
      const double* P = ent + (int64_t(b) * E + e) * nch * 2;
      double sp = 0.0, ap = 0.0;
      for (int c = lane; c < nch; c += kWave) {
        sp += P[2 * c];
        ap += P[2 * c + 1];
      }
      const double S = wave_sum_f64(sp);
      const double A = wave_sum_f64(ap);
      if (lane == 0) {
        float hb = 0.0f;
        if (N > 1 && S > 0.0) {
          // H = -(1/S) sum_i C_i (log C_i - log S) = (S log S - A) / S; with
          // one occupied position S log S and A are the same product
          const double Hs = (S * log(S) - A) / S;
          double v = Hs / log_n;
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
  if (tid < 512) (&s_hist[0][0])[tid] = 0;
  if (tid == 0) {
    s_unmatched = 0;
    s_recompute = 0;
    s_sync = 0;
    s_ncand = 0;
  }
  __syncthreads();

  // 1. matching and scores (cache steps); every operand of a branch is
  // loaded before any is used
  // per branch: margin and the packed (matched slot + 1) | expert << 4,
  // kept in registers while a thread holds at most 8 branches.  With more
  // (up to 32) nothing per branch stays in registers and the per-branch
  // loops are runtime loops: the later passes read the margin back from the
  // margin buffer this thread wrote (the values stay in L2), the slot from
  // its LDS copy s_q and the expert from e_t.
  constexpr bool kMvRegs = R <= 8;
  // unroll factor of the per-branch loops (by four when they are runtime
  // loops, so that a few branches' loads are in flight together)
  constexpr int kU = kMvRegs ? R : 4;
  float mv[kMvRegs ? R : 1];
  int qe[kMvRegs ? R : 1];
  // outside the sample (j >= nb) a branch reads as unmatched with margin +inf
  auto mval = [&](int r) __attribute__((always_inline)) -> float {
    if constexpr (kMvRegs) {
      return mv[r];
    } else {
      const int j = tid + kSelThreads * r;
      return j < nb ? margin[base + j] : __int_as_float(0x7f800000);
    }
  };
  auto key_full = [&](int r) __attribute__((always_inline)) -> uint32_t {
    return f32_order_key(mval(r));
  };
  // (key & msk) compared with t (t has no bits outside msk; msk keeps the
  // high bits): -1, 0 or 1.  With the key halves in LDS the low half is
  // read only when the high halves are equal.
  auto cmp_masked = [&](int r, uint32_t msk, uint32_t t) __attribute__((always_inline)) -> int {
    if constexpr (kMvRegs) {
      const uint32_t mk = key_full(r) & msk;
      return mk > t ? 1 : (mk < t ? -1 : 0);
    } else {
      const int j = tid + kSelThreads * r;
      const uint32_t hm = msk & 0xFFFF0000u;
      const uint32_t h = (j < nb ? static_cast<uint32_t>(s_k16[j]) << 16 : 0xFF800000u) & hm;
      if (h != (t & hm)) return h > (t & hm) ? 1 : -1;
      if ((msk & 0xFFFFu) == 0u) return 0;
      const uint32_t mk = key_full(r) & msk;
      return mk > t ? 1 : (mk < t ? -1 : 0);
    }
  };
  auto q_of = [&](int r) __attribute__((always_inline)) -> int {
    if constexpr (kMvRegs) {
      return (qe[r] & 15) - 1;
    } else {
      const int j = tid + kSelThreads * r;
      return j < nb ? static_cast<int>(s_q[j]) : -1;
    }
  };
  auto e_of = [&](int r) __attribute__((always_inline)) -> int {
    if constexpr (kMvRegs) return qe[r] >> 4;
    else return e_t[base + tid + kSelThreads * r];
  };
  int unmatched = 0;
#pragma unroll kU
  for (int r = 0; r < R; ++r) {
    const int j = tid + kSelThreads * r;
    float m = __int_as_float(0x7f800000);  // +inf: unmatched, always recomputed
    int qv = 0;                           // packed: slot -1, expert 0
    if (j < nb) {
      const int64_t f = base + j;
      BranchIn in;
      if constexpr (kPre) in = pre[r];
      else load_branch(r, in);
      const int e = in.e;
      qv = e << 4;
      if (mode != kSelFull) {
        const int q = match_score(e, in.w, in.ej, in.nc, in.wc, k, s_tau[e], lambda0, lambda1,
                                  lambda2, m);
        if (q < 0) ++unmatched;
        qv = (e << 4) | (q + 1);
        q_out[f] = q;
        margin[f] = m;
      }
    }
    if constexpr (kMvRegs) {
      mv[r] = m;
      qe[r] = qv;
    } else if (j < nb) {
      s_q[j] = static_cast<int8_t>((qv & 15) - 1);
      s_k16[j] = static_cast<uint16_t>(f32_order_key(m) >> 16);
    }
    // keep the scheduler from hoisting the loads of every branch at once
    // (a thread holds up to 32 branches, each with up to 3 k slot loads):
    // groups of four branches, pairs when a thread holds many
    if (kMvRegs ? (r & 3) == 3 : (r & 1) == 1) __builtin_amdgcn_sched_barrier(0);
  }
  if (mode != kSelFull) {
    unmatched = wave_sum_i32(unmatched);
    if (lane == 0) atomicAdd(&s_unmatched, unmatched);
  }
  __syncthreads();
  const int n_unmatched = s_unmatched;
  const int n_matched = mode == kSelFull ? 0 : nb - n_unmatched;

  // 2. ratio mode: the need-th best matched branch.  8-bit radix passes
  // (most significant first) narrow the margin key T down: after a pass the
  // prefix P of T is known, with fewer than `need` matched keys above it and
  // rem of the keys sharing it still to take.  When at most kDirect keys
  // share P, one wave ranks them by (key desc, flat id asc) and takes the
  // first rem (direct); otherwise, after the fourth pass, the keys equal to
  // T are ties and the lowest flat ids among them are taken (ballots).
  int need = 0;
  bool take_all_matched = false;
  bool direct = false;
  uint32_t thr = 0;
  uint32_t dmask = ~0u;   // key bits compared with thr
  int tie_rem = 0;
  uint32_t tie_bits = 0;  // bit r: branch r is one of the taken ties
  if (mode == kSelRatio) {
    need = budget - n_unmatched;
    if (need < 0) need = 0;
    if (need >= n_matched) take_all_matched = true;
    if (need > 0 && !take_all_matched) {
      uint32_t prefix = 0;
      int rem = need;
#pragma unroll
      for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        int* hist = s_hist[pass % 3];
        const uint32_t hi_mask = pass == 0 ? 0u : (~0u << (shift + 8));
        // histogram of this digit over the matched keys that share the
        // prefix: the (at most two) most frequent bins of a wave are added
        // once by one lane, the remaining lanes add their own
#pragma unroll kU
        for (int r = 0; r < R; ++r) {
          bool part = q_of(r) >= 0 && cmp_masked(r, hi_mask, prefix) == 0;
          int bin = 0;
          if (part) {
            if constexpr (!kMvRegs) {
              if (shift >= 16) {
                const int j = tid + kSelThreads * r;
                bin = static_cast<int>((static_cast<uint32_t>(s_k16[j]) >> (shift - 16)) & 255u);
              } else {
                bin = static_cast<int>((key_full(r) >> shift) & 255u);
              }
            } else {
              bin = static_cast<int>((key_full(r) >> shift) & 255u);
            }
          }
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
        // one barrier per pass: every wave scans the histogram itself; the
        // last wave clears the buffer of pass + 2 (three buffers in turn:
        // that one was last read by the scans of pass - 1, which every wave
        // finished before this barrier, and is next written after the
        // barrier of pass + 1)
        __syncthreads();
        if (wv == kSelWaves - 1 && pass + 2 < 4) {
#pragma unroll
          for (int u = 0; u < 4; ++u) s_hist[(pass + 2) % 3][4 * lane + u] = 0;
        }
        // lane l holds bins 255 - 4l .. 252 - 4l (descending); the lane whose
        // run of bins reaches rem names the digit and what remains of rem
        int c[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) c[u] = hist[255 - 4 * lane - u];
        const int tot = c[0] + c[1] + c[2] + c[3];
        int run = wave_incl_scan_i32(tot) - tot;
        int fbin = 0, frem = 0, fcnt = 0;
        bool found = false;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (c[u] > 0 && run < rem && rem <= run + c[u]) {
            found = true;
            fbin = 255 - 4 * lane - u;
            frem = rem - run;
            fcnt = c[u];
          }
          run += c[u];
        }
        const int leader = __builtin_ctzll(__ballot(found));
        prefix |= static_cast<uint32_t>(__builtin_amdgcn_readlane(fbin, leader)) << shift;
        rem = __builtin_amdgcn_readlane(frem, leader);
        if (__builtin_amdgcn_readlane(fcnt, leader) <= kDirect) {
          direct = true;  // the same decision in every wave
          dmask = ~0u << shift;
          break;
        }
      }
      thr = prefix;
      tie_rem = rem;
    }
    if (direct) {
      // the keys sharing the prefix (candidate index kept in s_mask[j],
      // free until step 3), ranked by wave 0; the order of the appends does
      // not matter
#pragma unroll kU
      for (int r = 0; r < R; ++r) {
        const int j = tid + kSelThreads * r;
        if (q_of(r) >= 0 && cmp_masked(r, dmask, thr) == 0) {
          const int ci = atomicAdd(&s_ncand, 1);
          s_ckey[ci] = key_full(r);
          s_cj[ci] = j;
          s_mask[j] = static_cast<uint8_t>(ci);
        }
      }
      __syncthreads();
      if (wv == 0) {
        const int nc = s_ncand;
        const uint32_t ki = lane < nc ? s_ckey[lane] : 0u;
        const int ji = lane < nc ? s_cj[lane] : 0;
        int rank = 0;
        for (int t = 0; t < nc; ++t) {
          const uint32_t kt = __builtin_amdgcn_readlane(ki, t);
          const int jt = __builtin_amdgcn_readlane(ji, t);
          rank += (kt > ki || (kt == ki && jt < ji)) ? 1 : 0;
        }
        if (lane < nc) s_csel[lane] = rank < tie_rem ? 1 : 0;
      }
      __syncthreads();
    } else if (need > 0 && !take_all_matched) {
      // keys equal to T: take the tie_rem lowest flat ids (j = tid + 1024 r,
      // so the order is r-major, then wave, then lane)
#pragma unroll kU
      for (int r = 0; r < R; ++r) {
        const uint64_t tb = __ballot(q_of(r) >= 0 && cmp_masked(r, ~0u, thr) == 0);
        if (lane == 0) s_tcnt[r][wv] = __popcll(tb);
      }
      __syncthreads();
      int before = 0;
#pragma unroll kU
      for (int r = 0; r < R; ++r) {
        int in_r = 0, below = 0;
        for (int w2 = 0; w2 < kSelWaves; ++w2) {
          const int c = s_tcnt[r][w2];
          in_r += c;
          if (w2 < wv) below += c;
        }
        const uint64_t tb = __ballot(q_of(r) >= 0 && cmp_masked(r, ~0u, thr) == 0);
        const bool flag = ((tb >> lane) & 1ull) != 0;
        if (flag && before + below + lane_rank(tb) < tie_rem) tie_bits |= 1u << r;
        before += in_r;
      }
    }
  }

  // 3. mask and per-expert counts
#pragma unroll kU
  for (int r = 0; r < R; ++r) {
    const int j = tid + kSelThreads * r;
    bool rc = false;
    if (j < nb) {
      if (mode == kSelFull || q_of(r) < 0) {
        rc = true;
      } else if (mode == kSelThreshold) {
        rc = cmp_masked(r, ~0u, 0x80000000u) > 0;  // m > 0 (+0 and -0 have this key)
      } else if (take_all_matched) {
        rc = true;
      } else if (need == 0) {
        rc = false;
      } else if (direct) {
        const int c = cmp_masked(r, dmask, thr);
        rc = c > 0 || (c == 0 && s_csel[s_mask[j]] != 0);
      } else {
        rc = cmp_masked(r, ~0u, thr) > 0 || ((tie_bits >> r) & 1u) != 0;
      }
      mask[base + j] = rc ? 1 : 0;
      s_mask[j] = rc ? 1 : 0;
      if constexpr (kMvRegs) s_q[j] = static_cast<int8_t>(q_of(r));
      if (rc) {
        atomicAdd(&s_cnt[e_of(r)], 1);
        atomicAdd(&s_cntr[r][e_of(r)], 1);
      }
    }
  }
  __syncthreads();

  // 4. per token: sync flag and slots
  int rec = 0, syn = 0;
  for (int i = tid; i < N; i += kSelThreads) {
    const bool any = token_slots(s_q + i * k, s_mask + i * k, k, mode == kSelFull,
                                 sigma + base + int64_t(i) * k, rec);
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
  // per-chunk counts [B][RC][E] for the lists kernel (RC chunks of 1024 branches)
  const int rc_n = (nb + kSelThreads - 1) / kSelThreads;
  for (int i = tid; i < rc_n * E; i += kSelThreads)
    cnt_ch[(int64_t(b) * rc_n + i / E) * E + i % E] = s_cntr[i / E][i % E];
  if (tid == 0) {
    stats_bs[b * 4 + 0] = s_recompute;
    stats_bs[b * 4 + 1] = mode == kSelFull ? 0 : n_unmatched;
    stats_bs[b * 4 + 2] = n_matched;
    stats_bs[b * 4 + 3] = s_sync;
  }
}

// Group table entries E..E+S: the shared experts (Sec. 2.3, shared-expert
// MoE eq.) follow the routed ones in the FFN's grouped GEMM, T rows each (every
// token, in token order), so their offsets and tile prefixes continue the
// routed totals (o rows, tu / td tiles).  Tile tables: up at [0, E+S],
// down at [E+S+1, 2(E+S)+1].
__device__ __forceinline__ void write_shared_groups(int32_t* __restrict__ off,
                                                    int32_t* __restrict__ tiles, int E, int S,
                                                    int T, int tm_up, int tm, int nt_up,
                                                    int nt_down, int o, int tu, int td) {
  const int mts_up = (T + tm_up - 1) / tm_up;
  const int mts = (T + tm - 1) / tm;
  for (int s2 = 0; s2 <= S; ++s2) {
    off[E + s2] = o + s2 * T;
    tiles[E + s2] = tu + s2 * mts_up * nt_up;
    tiles[E + S + 1 + E + s2] = td + s2 * mts * nt_down;
  }
}

// ---------------------------------------------------------------------------
// Per-expert lists of recomputed branches, ascending flat id within each
// expert; one 1024-thread block per chunk of 1024 consecutive branches of a
// sample (chunk c of sample b covers flat ids b N k + 1024 c ..).  Every
// block reads the [B][RC][E] chunk count table written by the decide kernel
// and derives, per expert, the total (-> expert offsets, block 0 also writes
// them and the GEMM tile tables) and the count in the chunks before its own
// in flat order (-> its write base).  Within the chunk each wave ranks its
// selected branches per expert with ballots; branches of earlier waves, then
// of lower lanes come first (stable, no atomics).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kSelThreads) void lists_kernel(
    const uint8_t* __restrict__ mask, const int32_t* __restrict__ e_t,
    const int32_t* __restrict__ cnt_ch, int B, int N, int E, int S, int k, int tm_up, int tm,
    int nt_up, int nt_down, const int32_t* __restrict__ sigma, int32_t* __restrict__ off,
    int32_t* __restrict__ tiles, int32_t* __restrict__ list, int32_t* __restrict__ pos,
    int32_t* __restrict__ row_dst) {
  __shared__ int s_part_tot[kSelThreads];
  __shared__ int s_part_bef[kSelThreads];
  __shared__ int s_base[64];
  __shared__ int s_wcnt[kSelWaves][64];
  const int nb = N * k;
  const int rc_n = (nb + kSelThreads - 1) / kSelThreads;
  const int b = blockIdx.x / rc_n;
  const int c = blockIdx.x % rc_n;
  const int my = blockIdx.x;  // flat chunk index (b rc_n + c)
  const int nchunks = B * rc_n;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wv = tid / kWave;

  // this block's branch, loaded first
  const int j = c * kSelThreads + tid;
  const int64_t f = int64_t(b) * nb + j;
  const bool in = j < nb;
  const bool sel = in && mask[f] != 0;
  const int ev = sel ? e_t[f] : -1;
  const int sg = sel ? sigma[f] : 0;

  // per expert: total over all chunks and count in the chunks before this one
  // thread (e0, part) for part < parts; E <= 64
  const int parts = min(kSelThreads / E, nchunks);
  const int e0 = tid % E, part = tid / E;
  int tot = 0, bef = 0;
  if (part < parts) {
    for (int ch = part; ch < nchunks; ch += parts) {
      const int v = cnt_ch[int64_t(ch) * E + e0];
      tot += v;
      if (ch < my) bef += v;
    }
  }
  s_part_tot[tid] = tot;
  s_part_bef[tid] = bef;
  __syncthreads();
  if (wv == 0) {
    int t = 0, bf = 0;
    if (lane < E) {
#pragma unroll 4
      for (int pp = 0; pp < parts; ++pp) {
        t += s_part_tot[pp * E + lane];
        bf += s_part_bef[pp * E + lane];
      }
    }
    const int mt_up = (t + tm_up - 1) / tm_up;
    const int mt = (t + tm - 1) / tm;
    // inclusive scans over experts
    const int o = wave_incl_scan_i32(t);
    const int tu = wave_incl_scan_i32(mt_up * nt_up);
    const int td = wave_incl_scan_i32(mt * nt_down);
    if (lane < E) s_base[lane] = o - t + bf;
    if (my == 0 && lane < E) {
      // exclusive prefixes per expert; the last expert also writes the
      // prefixes of the shared experts and the totals
      off[lane] = o - t;
      tiles[lane] = tu - mt_up * nt_up;
      tiles[E + S + 1 + lane] = td - mt * nt_down;
      if (lane == E - 1)
        write_shared_groups(off, tiles, E, S, B * N, tm_up, tm, nt_up, nt_down, o, tu, td);
    }
  }
  int rk = 0;
  for (int ee = 0; ee < E; ++ee) {
    const bool mine = ev == ee;
    const uint64_t bal = __ballot(mine);
    if (lane == ee) s_wcnt[wv][ee] = __popcll(bal);
    if (mine) rk = lane_rank(bal);
  }
  __syncthreads();
  if (!in) return;
  if (!sel) {
    pos[f] = -1;
    return;
  }
  int before = 0;
  for (int w2 = 0; w2 < wv; ++w2) before += s_wcnt[w2][ev];
  const int idx = s_base[ev] + before + rk;
  list[idx] = static_cast<int32_t>(f);
  pos[f] = idx;
  row_dst[idx] = static_cast<int32_t>((f / k) * k + sg);
}

// ---------------------------------------------------------------------------
// Multi-block decision path for samples of more than 8192 branches (k a
// divisor of 1024): the decisions of decide_kernel with a sample spread over
// ceil(N k / 1024) blocks of one branch per thread; block (b, c) takes the
// flat ids c 1024 + tid of sample b, whole tokens.  The steps that need the
// whole sample meet at kernel boundaries:
//   wide_prep   entropy and thresholds, one wave per (sample, expert); clears
//               the per-sample scratch, the expert counts and the statistics
//   wide_score  matching, scores and margins; unmatched counts; in ratio
//               steps the histogram of the first radix digit, in threshold
//               and full steps the whole decision
//   wide_pass p (ratio steps, p = 1, 2, 3) every block derives the digits so
//               far from the histograms, then adds its keys to the histogram
//               of digit p, or, right after the digit that left at most
//               kDirect keys sharing the prefix, appends those keys and their
//               flat ids to the sample's candidate list
//   wide_final  the ratio decision: the candidates ranked by (key desc, flat
//               id asc), or, with more equal keys than kDirect after the
//               fourth digit, the keys equal to the threshold ranked by flat
//               id; then mask, counts, slots and sync
// Scratch per sample (kWideWords ints): four 256-bin histograms, counters
// (0: unmatched, 3: candidates), candidate keys and flat ids.
// ---------------------------------------------------------------------------
constexpr int kWsCtr = 1024, kWsCKey = 1032, kWsCJ = 1096;

// The digit of a radix pass from its 256-bin histogram h (keys descending
// from bin 255): the bin holding the rem-th key, what remains of rem inside
// it, and the bin's count.  Wave-wide; every lane gets the same values.
__device__ __forceinline__ void digit_select(const int* h, int rem, int& bin, int& nrem,
                                             int& cnt) {
  const int lane = threadIdx.x & (kWave - 1);
  int c[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) c[u] = h[255 - 4 * lane - u];
  const int tot = c[0] + c[1] + c[2] + c[3];
  int run = wave_incl_scan_i32(tot) - tot;
  int fbin = 0, frem = 0, fcnt = 0;
  bool found = false;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (c[u] > 0 && run < rem && rem <= run + c[u]) {
      found = true;
      fbin = 255 - 4 * lane - u;
      frem = rem - run;
      fcnt = c[u];
    }
    run += c[u];
  }
  const int leader = __builtin_ctzll(__ballot(found));
  bin = __builtin_amdgcn_readlane(fbin, leader);
  nrem = __builtin_amdgcn_readlane(frem, leader);
  cnt = __builtin_amdgcn_readlane(fcnt, leader);
}

// The ratio selection of a sample as far as the first `upto` digit
// histograms take it.
struct WideChain {
  int need = 0;
  bool take_all = false;
  bool active = false;     // a threshold key has to be found
  uint32_t prefix = 0;     // digits found so far
  uint32_t dmask = 0;      // their bits
  int rem = 0;             // keys still to take among those sharing prefix
  int digits = 0;
  int direct_at = -1;      // digit after which at most kDirect keys remain
};

__device__ __forceinline__ WideChain wide_chain(const int32_t* ws, int budget, int nb, int upto) {
  WideChain ch;
  const int n_unmatched = ws[kWsCtr + 0];
  const int n_matched = nb - n_unmatched;
  ch.need = budget - n_unmatched;
  if (ch.need < 0) ch.need = 0;
  ch.take_all = ch.need >= n_matched;
  ch.active = ch.need > 0 && !ch.take_all;
  ch.rem = ch.need;
  if (!ch.active) return ch;
  for (int p = 0; p < upto; ++p) {
    int bin, nrem, cnt;
    digit_select(ws + 256 * p, ch.rem, bin, nrem, cnt);
    const int shift = 24 - 8 * p;
    ch.prefix |= static_cast<uint32_t>(bin) << shift;
    ch.dmask = ~0u << shift;
    ch.rem = nrem;
    ch.digits = p + 1;
    if (cnt <= kDirect && p < 3) {
      ch.direct_at = p;
      break;
    }
  }
  return ch;
}

// Adds the block's keys to a 256-bin histogram in LDS (the at most two most
// frequent bins of a wave by one lane each), then to the global one.
__device__ __forceinline__ void wide_hist(int* s_h, bool part, int bin, int32_t* gh) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const uint64_t todo = __ballot(part);
    if (todo == 0ull) break;
    const int leader = __builtin_ctzll(todo);
    const int lb = __builtin_amdgcn_readlane(bin, leader);
    const uint64_t same = __ballot(part && bin == lb);
    if (lane == leader) atomicAdd(&s_h[lb], __popcll(same));
    if (bin == lb) part = false;
  }
  if (part) atomicAdd(&s_h[bin], 1);
  __syncthreads();
  if (threadIdx.x < 256 && s_h[threadIdx.x] != 0) atomicAdd(&gh[threadIdx.x], s_h[threadIdx.x]);
}

__global__ __launch_bounds__(kSelThreads) void wide_prep_kernel(
    const double* __restrict__ ent, int with_stat, double log_n, float tau0, float alpha,
    float* __restrict__ hbar, float* __restrict__ tau, int B, int N, int E,
    int32_t* __restrict__ ws, int32_t* __restrict__ cnt_bs, int32_t* __restrict__ stats_bs) {
  const int64_t gt = int64_t(blockIdx.x) * kSelThreads + threadIdx.x;
  const int64_t gs = int64_t(gridDim.x) * kSelThreads;
  for (int64_t i = gt; i < int64_t(B) * kWideWords; i += gs) ws[i] = 0;
  for (int64_t i = gt; i < int64_t(B) * E; i += gs) cnt_bs[i] = 0;
  for (int64_t i = gt; i < int64_t(B) * 4; i += gs) stats_bs[i] = 0;
  if (!with_stat) return;
  // entropy of the statistic and tau (Sec. 4.3), as in decide_kernel
  const int lane = threadIdx.x & (kWave - 1);
  const int row = blockIdx.x * kSelWaves + threadIdx.x / kWave;  // b E + e
  if (row >= B * E) return;
  const int nch = (N + 15) / 16;
  const double* P = ent + int64_t(row) * nch * 2;
  double sp = 0.0, ap = 0.0;
  for (int c = lane; c < nch; c += kWave) {
    sp += P[2 * c];
    ap += P[2 * c + 1];
  }
  const double S = wave_sum_f64(sp);
  const double A = wave_sum_f64(ap);
  if (lane == 0) {
    float hb = 0.0f;
    if (N > 1 && S > 0.0) {
      const double Hs = (S * log(S) - A) / S;
      double v = Hs / log_n;
      v = v < 0.0 ? 0.0 : (v > 1.0 ? 1.0 : v);
      hb = static_cast<float>(v);
    }
    const float centred = __fsub_rn(__fmul_rn(2.0f, hb), 1.0f);
    hbar[row] = hb;
    tau[row] = __fmul_rn(tau0, __fadd_rn(1.0f, __fmul_rn(alpha, centred)));
  }
}

// Mask, counts, slots and sync of one block (one branch per thread, whole
// tokens), as steps 3 and 4 of decide_kernel.
__device__ __forceinline__ void wide_finish(int b, int c, int j, bool in, bool rc, int q, int e,
                                            int mode, int N, int E, int k, int nb,
                                            uint8_t* __restrict__ mask,
                                            int32_t* __restrict__ sigma,
                                            uint8_t* __restrict__ sync,
                                            int32_t* __restrict__ cnt_bs,
                                            int32_t* __restrict__ cnt_ch,
                                            int32_t* __restrict__ stats_bs) {
  __shared__ int8_t s_q[kSelThreads];
  __shared__ uint8_t s_m[kSelThreads];
  __shared__ int s_cnt[64];
  __shared__ int s_rs[2];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int64_t base = int64_t(b) * nb;
  if (tid < 64) s_cnt[tid] = 0;
  if (tid < 2) s_rs[tid] = 0;
  __syncthreads();
  if (in) {
    mask[base + j] = rc ? 1 : 0;
    if (rc) atomicAdd(&s_cnt[e], 1);
  }
  s_m[tid] = in && rc ? 1 : 0;
  s_q[tid] = static_cast<int8_t>(in ? q : -1);
  __syncthreads();
  // tokens of the block: t_local = tid < 1024 / k, token c (1024 / k) + t_local
  const int tpb = kSelThreads / k;
  const int i = c * tpb + tid;
  int rec = 0, syn = 0;
  if (tid < tpb && i < N) {
    const bool any = token_slots(s_q + tid * k, s_m + tid * k, k, mode == kSelFull,
                                 sigma + base + int64_t(c) * kSelThreads + int64_t(tid) * k, rec);
    sync[int64_t(b) * N + i] = any ? 1 : 0;
    syn = any ? 1 : 0;
  }
  rec = wave_sum_i32(rec);
  syn = wave_sum_i32(syn);
  if (lane == 0 && (rec | syn) != 0) {
    atomicAdd(&s_rs[0], rec);
    atomicAdd(&s_rs[1], syn);
  }
  __syncthreads();
  const int rc_n = (nb + kSelThreads - 1) / kSelThreads;
  if (tid < E) {
    cnt_ch[(int64_t(b) * rc_n + c) * E + tid] = s_cnt[tid];
    if (s_cnt[tid] != 0) atomicAdd(&cnt_bs[b * E + tid], s_cnt[tid]);
  }
  if (tid == 0) {
    atomicAdd(&stats_bs[b * 4 + 0], s_rs[0]);
    atomicAdd(&stats_bs[b * 4 + 3], s_rs[1]);
  }
}

__global__ __launch_bounds__(kSelThreads) void wide_score_kernel(
    const int32_t* __restrict__ e_t, const float* __restrict__ w_t,
    const int32_t* __restrict__ e_c, const float* __restrict__ w_c,
    const float* __restrict__ n_c, const float* __restrict__ tau, int N, int E, int k,
    int mode, float lambda0, float lambda1, float lambda2, int32_t* __restrict__ q_out,
    float* __restrict__ margin, int32_t* __restrict__ ws, uint8_t* __restrict__ mask,
    int32_t* __restrict__ sigma, uint8_t* __restrict__ sync, int32_t* __restrict__ cnt_bs,
    int32_t* __restrict__ cnt_ch, int32_t* __restrict__ stats_bs) {
  __shared__ float s_tau[64];
  __shared__ int s_h[256];
  __shared__ int s_un, s_mt;
  const int nb = N * k;
  const int rc_n = (nb + kSelThreads - 1) / kSelThreads;
  const int b = blockIdx.x / rc_n, c = blockIdx.x % rc_n;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int j = c * kSelThreads + tid;
  const bool in = j < nb;
  const int64_t f = int64_t(b) * nb + j;
  if (tid < 256) s_h[tid] = 0;
  if (tid < E) s_tau[tid] = tau[b * E + tid];
  if (tid == 0) {
    s_un = 0;
    s_mt = 0;
  }
  __syncthreads();
  int e = 0, q = -1;
  float m = __int_as_float(0x7f800000);  // +inf: unmatched
  if (in) {
    e = e_t[f];
    if (mode != kSelFull) {
      const float w = w_t[f];
      const int64_t c0 = int64_t(b) * nb + (j / k) * k;
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
      q = match_score(e, w, ejs, ncs, wcs, k, s_tau[e], lambda0, lambda1, lambda2, m);
      q_out[f] = q;
      margin[f] = m;
    }
  }
  if (mode != kSelFull) {
    const int un = wave_sum_i32(in && q < 0 ? 1 : 0);
    const int mt = wave_sum_i32(in && q >= 0 ? 1 : 0);
    if (lane == 0 && un != 0) atomicAdd(&s_un, un);
    if (lane == 0 && mt != 0) atomicAdd(&s_mt, mt);
  }
  __syncthreads();
  // one device atomic per block and counter (the blocks of a sample share
  // its counters)
  if (mode != kSelFull && tid == 0) {
    if (s_un != 0) {
      atomicAdd(&ws[int64_t(b) * kWideWords + kWsCtr + 0], s_un);
      atomicAdd(&stats_bs[b * 4 + 1], s_un);
    }
    if (s_mt != 0) atomicAdd(&stats_bs[b * 4 + 2], s_mt);
  }
  if (mode == kSelRatio) {
    const uint32_t mk = f32_order_key(m);
    wide_hist(s_h, in && q >= 0, static_cast<int>(mk >> 24), ws + int64_t(b) * kWideWords);
    return;
  }
  const bool rc = mode == kSelFull || q < 0 || m > 0.0f;
  wide_finish(b, c, j, in, rc, q, e, mode, N, E, k, nb, mask, sigma, sync, cnt_bs, cnt_ch,
              stats_bs);
}

__global__ __launch_bounds__(kSelThreads) void wide_pass_kernel(
    int pass, const int32_t* __restrict__ q_out, const float* __restrict__ margin, int N,
    int k, int budget, int32_t* __restrict__ ws) {
  __shared__ int s_h[256];
  const int nb = N * k;
  const int rc_n = (nb + kSelThreads - 1) / kSelThreads;
  const int b = blockIdx.x / rc_n, c = blockIdx.x % rc_n;
  const int tid = threadIdx.x;
  int32_t* w = ws + int64_t(b) * kWideWords;
  const WideChain ch = wide_chain(w, budget, nb, pass);
  if (!ch.active || (ch.direct_at >= 0 && ch.direct_at < pass - 1)) return;  // block-uniform
  const int j = c * kSelThreads + tid;
  const int64_t f = int64_t(b) * nb + j;
  const bool matched = j < nb && q_out[f] >= 0;
  const uint32_t mk = matched ? f32_order_key(margin[f]) : 0u;
  const bool share = matched && (mk & ch.dmask) == ch.prefix;
  if (ch.direct_at == pass - 1) {
    // at most kDirect keys share the prefix: append them
    if (share) {
      const int ci = atomicAdd(&w[kWsCtr + 3], 1);  // below kDirect by the count above
      if (ci < kDirect) {
        w[kWsCKey + ci] = static_cast<int32_t>(mk);
        w[kWsCJ + ci] = j;
      }
    }
    return;
  }
  if (tid < 256) s_h[tid] = 0;
  __syncthreads();
  const int shift = 24 - 8 * pass;
  wide_hist(s_h, share, static_cast<int>((mk >> shift) & 255u), w + 256 * pass);
}

__global__ __launch_bounds__(kSelThreads) void wide_final_kernel(
    const int32_t* __restrict__ e_t, const int32_t* __restrict__ q_out,
    const float* __restrict__ margin, int N, int E, int k, int budget,
    int32_t* __restrict__ ws, uint8_t* __restrict__ mask, int32_t* __restrict__ sigma,
    uint8_t* __restrict__ sync, int32_t* __restrict__ cnt_bs, int32_t* __restrict__ cnt_ch,
    int32_t* __restrict__ stats_bs) {
  __shared__ int s_csel[kDirect];
  __shared__ int s_cjl[kDirect];
  __shared__ int s_wt[kSelWaves];
  __shared__ int s_before;
  const int nb = N * k;
  const int rc_n = (nb + kSelThreads - 1) / kSelThreads;
  const int b = blockIdx.x / rc_n, c = blockIdx.x % rc_n;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wv = tid / kWave;
  const int32_t* w = ws + int64_t(b) * kWideWords;
  const WideChain ch = wide_chain(w, budget, nb, 4);
  const int j = c * kSelThreads + tid;
  const bool in = j < nb;
  const int64_t base = int64_t(b) * nb;
  const int64_t f = base + j;
  const int q = in ? q_out[f] : -1;
  const int e = in ? e_t[f] : 0;
  const uint32_t mk = in && q >= 0 ? f32_order_key(margin[f]) : 0u;
  bool rc = in && (q < 0 || ch.take_all);
  if (ch.active && ch.direct_at >= 0) {
    if (wv == 0) {
      // rank the candidates by (key desc, flat id asc)
      const int nc = min(w[kWsCtr + 3], kDirect);
      const uint32_t ki = lane < nc ? static_cast<uint32_t>(w[kWsCKey + lane]) : 0u;
      const int ji = lane < nc ? w[kWsCJ + lane] : -1;
      int rank = 0;
      for (int t = 0; t < nc; ++t) {
        const uint32_t kt = __builtin_amdgcn_readlane(ki, t);
        const int jt = __builtin_amdgcn_readlane(ji, t);
        rank += (kt > ki || (kt == ki && jt < ji)) ? 1 : 0;
      }
      if (lane < kDirect) {
        s_csel[lane] = lane < nc && rank < ch.rem ? 1 : 0;
        s_cjl[lane] = ji;
      }
    }
    __syncthreads();
    if (in && q >= 0) {
      const uint32_t hm = mk & ch.dmask;
      if (hm > ch.prefix) {
        rc = true;
      } else if (hm == ch.prefix) {
        for (int t = 0; t < kDirect; ++t)
          if (s_cjl[t] == j) rc = s_csel[t] != 0;
      }
    }
  } else if (ch.active) {
    // threshold key T = prefix (all four digits); the keys equal to T rank by
    // flat id: those in the sample's earlier blocks, then within the block
    if (tid == 0) s_before = 0;
    __syncthreads();
    int cnt = 0;
    for (int jj = tid; jj < c * kSelThreads; jj += kSelThreads) {
      const int64_t ff = base + jj;
      if (q_out[ff] >= 0 && f32_order_key(margin[ff]) == ch.prefix) ++cnt;
    }
    cnt = wave_sum_i32(cnt);
    if (lane == 0 && cnt != 0) atomicAdd(&s_before, cnt);
    const bool tie = in && q >= 0 && mk == ch.prefix;
    const uint64_t tb = __ballot(tie);
    if (lane == 0) s_wt[wv] = __popcll(tb);
    __syncthreads();
    int below = s_before;
    for (int w2 = 0; w2 < wv; ++w2) below += s_wt[w2];
    if (in && q >= 0) rc = mk > ch.prefix || (tie && below + lane_rank(tb) < ch.rem);
  }
  wide_finish(b, c, j, in, rc, q, e, kSelRatio, N, E, k, nb, mask, sigma, sync, cnt_bs, cnt_ch,
              stats_bs);
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

hipError_t launch_decide(const Shape& s, int sel_mode, int budget, float lambda0, float lambda1,
                         float lambda2, bool with_stat, float tau0, float alpha,
                         const Buffers& b, hipStream_t st) {
  const int nb = s.N * s.k;
  const double log_n = std::log(static_cast<double>(s.N));  // the entropy's normaliser
  if (nb > 8 * kSelThreads && kSelThreads % s.k == 0 && s.E <= 64) {
    // multi-block path: the stage's start event goes with the first launch,
    // its stop event with the last
    const LaunchEvents ev = launch_events();
    launch_events() = LaunchEvents{};
    const int rc_n = (nb + kSelThreads - 1) / kSelThreads;
    const int grid = s.B * rc_n;
    const int prep = std::max((s.B * s.E + kSelWaves - 1) / kSelWaves,
                              (s.B * kWideWords + kSelThreads - 1) / kSelThreads);
    const bool ratio = sel_mode == kSelRatio;
    launch_kernel_ev(&wide_prep_kernel, dim3(prep), dim3(kSelThreads), 0, st, ev.start, nullptr,
                     b.ent, with_stat ? 1 : 0, log_n, tau0, alpha, b.hbar, b.tau, s.B, s.N, s.E,
                     b.wide, b.cnt_bs, b.stats_bs);
    launch_kernel_ev(&wide_score_kernel, dim3(grid), dim3(kSelThreads), 0, st, nullptr,
                     ratio ? nullptr : ev.stop, b.e_t, b.w_t, b.e_c, b.w_c, b.n_c, b.tau, s.N,
                     s.E, s.k, sel_mode, lambda0, lambda1, lambda2, b.q, b.margin, b.wide,
                     b.mask, b.sigma, b.sync, b.cnt_bs, b.cnt_ch, b.stats_bs);
    if (ratio) {
      for (int pass = 1; pass < 4; ++pass)
        launch_kernel_ev(&wide_pass_kernel, dim3(grid), dim3(kSelThreads), 0, st, nullptr,
                         nullptr, pass, b.q, b.margin, s.N, s.k, budget, b.wide);
      launch_kernel_ev(&wide_final_kernel, dim3(grid), dim3(kSelThreads), 0, st, nullptr,
                       ev.stop, b.e_t, b.q, b.margin, s.N, s.E, s.k, budget, b.wide, b.mask,
                       b.sigma, b.sync, b.cnt_bs, b.cnt_ch, b.stats_bs);
    }
    return hipGetLastError();
  }
  const size_t lds = size_t(2) * nb;
  if (lds > 64 * 1024) return hipErrorInvalidValue;
#define MOECA_DECIDE(RR)                                                                      \
  launch_kernel(&decide_kernel<RR>, dim3(s.B), dim3(kSelThreads), uint32_t(lds), st, b.e_t,   \
                b.w_t, b.e_c, b.w_c, b.n_c, b.ent, with_stat ? 1 : 0, log_n, tau0,            \
                alpha,                                                                        \
                b.hbar, b.tau, s.N, s.E, s.k, sel_mode, budget, lambda0, lambda1, lambda2,    \
                b.q,                                                                          \
                b.margin, b.mask, b.sigma, b.sync, b.cnt_bs, b.stats_bs, b.cnt_ch)
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
  // units of the down projection per M tile: N tiles times K pieces
  const int nt_down = (s.d + plan.tn_down - 1) / plan.tn_down * plan.split_down;
  const int rc_n = (nb + kSelThreads - 1) / kSelThreads;
  if (s.E > 64) return hipErrorInvalidValue;
  launch_kernel(&lists_kernel, dim3(s.B * rc_n), dim3(kSelThreads), 0, st, b.mask, b.e_t,
                b.cnt_ch, s.B, s.N, s.E, s.S, s.k, plan.tm_up, plan.tm, nt_up, nt_down, b.sigma, b.off,
                b.tiles, b.list, b.pos, b.row_dst);
  return hipGetLastError();
}

hipError_t launch_reset(const Shape& s, const Buffers& b, hipStream_t st) {
  launch_kernel(&reset_kernel, dim3(256), dim3(256), 0, st, b.e_c, b.w_c, b.n_c, s.branches(),
                b.stat, int64_t(s.B) * s.E * s.N);
  return hipGetLastError();
}

}  // namespace moeca
