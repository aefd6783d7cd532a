// Grouped expert FFN on the recomputed branches (Sec. 4.1: only R_i goes
// through FFN_e; Sec. 2.3: FFN_e(x) = W_down[e] act(W_up[e] x)).
//
// The per-expert lists (ascending flat branch ids, grouped by expert) define
// a grouped GEMM with a device-side row count per expert.  The grid is sized
// on the host for the worst case and every block derives its tile from the
// per-expert offsets, so no count ever travels to the host.
//
//   up   : mid[r]  = act(x[token(r)] . W_up[e]^T)     gathered rows -> rows
//   down : h_c[slot(r)] = mid[r] . W_down[e]^T        rows -> cache rows
//
// The down projection writes each recomputed branch straight into the cache
// slot it will occupy: reused slots are never touched, so the combine reads
// every branch feature from the cache.
//
// Shared experts (Sec. 2.3, shared-expert MoE eq.) are S more groups of the
// same grouped GEMM, after the E routed ones: group E+s has every token as
// its rows (in token order), its own weights, and its down projection writes
// h_sh[s][token].  With the gated activation (SwiGLU) the up-projection rows
// alternate gate / up, so a lane's four consecutive accumulator columns hold
// two (gate, up) pairs and the epilogue emits silu(gate) * up for both:
// the intermediate is d_ff wide for either activation.
//
// bf16 path: v_mfma_f32_32x32x16_bf16 with fp32 accumulation; 256 threads
// as 2x2 waves, block tile TM x TN, k-tile 64, LDS double buffered with
// padded rows; the activation is applied to the fp32 accumulator and the
// result rounded to bf16.  Tile order: expert-major, then N tile, then M tile,
// and consecutive logical tiles sit on the same XCD, so the M tiles sharing a
// weight slice run together and the expert's gathered rows stay in that
// XCD's L2.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "internal.h"
#include "moeca.h"

namespace moeca {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_t;  // 16 bytes, a native vector
typedef __attribute__((ext_vector_type(2))) unsigned int u32x2_t;

// kProj: a dense projection of listed token rows (the attention path of a
// block): row r reads token list[r] and writes row list[r] of the output.
enum { kUp = 0, kDown = 1, kProj = 2 };
constexpr int kXcds = 8;

// Activation of the up projection.  tanh GELU:
//   0.5 z (1 + tanh(u)) = z / (1 + exp(-2u)),  u = sqrt(2/pi) (z + 0.044715 z^3),
// with exp(-2u) = 2^(-2u log2 e) from the hardware exp2 (about 1 ulp) and a
// hardware reciprocal; the erf form uses erff.  kActSwiglu marks the gated
// epilogue (silu below), which pairs columns instead of mapping each one.
enum { kActGeluTanh = 0, kActGeluErf = 1, kActNone = 2, kActSwiglu = 3, kActBias = 4 };

// silu(z) = z / (1 + exp(-z)), exp(-z) = 2^(-z log2 e) by the hardware exp2.
__device__ __forceinline__ float silu_f(float z) {
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z));
}

template <int ACT>
__device__ __forceinline__ float act_fn(float z) {
  if constexpr (ACT == kActGeluTanh) {
    const float u = 0.7978845608028654f * (z + 0.044715f * z * z * z);
    return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-2.8853900817779268f * u));
  } else if constexpr (ACT == kActGeluErf) {
    return 0.5f * z * (1.0f + erff(z * 0.7071067811865476f));
  } else {
    return z;
  }
}

struct Tile {
  int e, r0, rows, n0;
};

// Logical tile L -> (group, first row, row count, first column); e = -1 if
// this block has no tile.  Tiles per group: ceil(cnt_e / TM) * NT.
template <int TM>
__device__ Tile decode_tile(const int32_t* __restrict__ off, int G, int NT) {
  int total = 0;
  for (int e = 0; e < G; ++e) total += ((off[e + 1] - off[e] + TM - 1) / TM) * NT;
  const int per = (total + kXcds - 1) / kXcds;
  const int xcd = blockIdx.x % kXcds;
  const int slot = blockIdx.x / kXcds;
  const int L = xcd * per + slot;
  Tile t{-1, 0, 0, 0};
  if (slot >= per || L >= total) return t;
  int acc = 0;
  for (int e = 0; e < G; ++e) {
    const int cnt = off[e + 1] - off[e];
    const int mt = (cnt + TM - 1) / TM;
    const int tiles = mt * NT;
    if (L < acc + tiles) {
      const int local = L - acc;
      const int m = local % mt;
      t.e = e;
      t.r0 = off[e] + m * TM;
      t.rows = min(TM, cnt - m * TM);
      t.n0 = (local / mt);
      return t;
    }
    acc += tiles;
  }
  return t;
}

// Group of logical tile L: the number of group tile prefixes <= L, minus
// one, from two ballots (groups 0-63 in toff0, 64-127 in toff1: lane l holds
// the prefixes of groups l and 64 + l, INT_MAX past the last group); also
// returns the group's first tile.
__device__ __forceinline__ int tile_group(int L, int toff0, int toff1, int& first) {
  const int n0 = __popcll(__ballot(toff0 <= L));
  const int n1 = __popcll(__ballot(toff1 <= L));
  const int e = n0 + n1 - 1;
  first = e < 64 ? __shfl(toff0, e, 64) : __shfl(toff1, e - 64, 64);
  return e;
}

// Row table entry r of a tile of group e (first list row r0, `rows` rows):
// the A-operand source row and the output row (-1: padding, never stored;
// padding rows re-read the tile's first row).  Routed groups (e < E): up
// reads token list[r]/k and writes intermediate row r; down reads
// intermediate row r and writes cache row row_dst[r].  Shared groups: up
// reads token r - off[e] and writes intermediate row r; down reads
// intermediate row r and writes shared-output row r - off[E].
template <int KIND>
__device__ __forceinline__ void group_row(int e, int E, int r0, int rows, int r, int k,
                                          const int32_t* __restrict__ off,
                                          const int32_t* __restrict__ list,
                                          const int32_t* __restrict__ row_dst, int& src,
                                          int& dst) {
  const int rr = r < rows ? r : 0;
  if (KIND == kProj) {
    src = list[r0 + rr];
    dst = r < rows ? list[r0 + r] : -1;
  } else if (e < E) {
    if (KIND == kUp) {
      src = list[r0 + rr] / k;
      dst = r < rows ? r0 + r : -1;
    } else {
      src = r0 + rr;
      dst = r < rows ? row_dst[r0 + r] : -1;
    }
  } else {
    if (KIND == kUp) {
      src = r0 + rr - off[e];
      dst = r < rows ? r0 + r : -1;
    } else {
      src = r0 + rr;
      dst = r < rows ? r0 + r - off[E] : -1;
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA grouped GEMM, persistent.
//
// The grid holds a fixed number of blocks per CU.  Logical tiles (expert-
// major, then N tile, then M tile; prefix per expert in `tile_off`) are split
// into eight contiguous ranges, one per XCD (block b runs on XCD b % 8), and
// the blocks of an XCD walk their range with a stride.  A block finds the
// expert of a tile with one ballot over the per-expert prefixes.
//
// Main loop: k-tile 64, two LDS buffers, global loads issued two k-tiles
// ahead into two register sets, one barrier per k-tile.  Epilogue: the tile
// goes through LDS and leaves as 16-byte row segments.
// ---------------------------------------------------------------------------
constexpr int kTK = 64;
constexpr int kLdsRow = kTK + 8;  // padded row (bf16 elements): 144 bytes
constexpr int kGemmThreads = 256;

// Global -> registers: LA rows of A and LB rows of W, 16 bytes each.
template <int LA, int LB>
__device__ __forceinline__ void gload(u32x4_t (&R)[LA + LB], const uint16_t* const (&ap)[LA],
                                      const uint16_t* const (&bp)[LB], int koff) {
#pragma unroll
  for (int i = 0; i < LA; ++i) R[i] = *reinterpret_cast<const u32x4_t*>(ap[i] + koff);
#pragma unroll
  for (int i = 0; i < LB; ++i) R[LA + i] = *reinterpret_cast<const u32x4_t*>(bp[i] + koff);
}

// Registers -> one LDS buffer (row r of the tile at r * kLdsRow).
template <int LA, int LB>
__device__ __forceinline__ void lstore(const u32x4_t (&R)[LA + LB], uint16_t* as, uint16_t* bs,
                                       int lrow, int lcol) {
#pragma unroll
  for (int i = 0; i < LA; ++i)
    *reinterpret_cast<u32x4_t*>(&as[(lrow + 32 * i) * kLdsRow + lcol]) = R[i];
#pragma unroll
  for (int i = 0; i < LB; ++i)
    *reinterpret_cast<u32x4_t*>(&bs[(lrow + 32 * i) * kLdsRow + lcol]) = R[LA + i];
}

// One k-tile of MFMAs on an LDS buffer: the wave's FM x FN 32x32 tiles.
template <int FM, int FN>
__device__ __forceinline__ void mfma_ktile(f32x16_t (&acc)[FM][FN], const uint16_t* as,
                                           const uint16_t* bs, int arow0, int brow0, int frow,
                                           int fk) {
#pragma unroll
  for (int ks = 0; ks < kTK / 16; ++ks) {
    bf16x8_t fa[FM], fb[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
      fa[i] = *reinterpret_cast<const bf16x8_t*>(
          &as[(arow0 + i * 32 + frow) * kLdsRow + ks * 16 + fk]);
#pragma unroll
    for (int j = 0; j < FN; ++j)
      fb[j] = *reinterpret_cast<const bf16x8_t*>(
          &bs[(brow0 + j * 32 + frow) * kLdsRow + ks * 16 + fk]);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
  }
}

template <int TM, int TN, int KIND, int ACT>
__global__ __launch_bounds__(kGemmThreads, 2) void gemm_bf16_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ W,
    const uint16_t* __restrict__ Wsh, const int32_t* __restrict__ off,
    const int32_t* __restrict__ tile_off, const int32_t* __restrict__ list,
    const int32_t* __restrict__ row_dst, int E, int G, int k, int K, int Nout,
    uint16_t* __restrict__ dst, uint16_t* __restrict__ dst_sh) {
  constexpr int WM = TM / 2, WN = TN / 2;  // wave tile (2 x 2 waves)
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int LA = TM / 32, LB = TN / 32;  // 16-byte loads per thread per k-tile
  constexpr int CROW = TN + 8;               // epilogue LDS row (bf16 elements)
  constexpr bool kGated = ACT == kActSwiglu;
  constexpr int OTN = kGated ? TN / 2 : TN;  // output columns per tile
  static_assert(TM * CROW <= 2 * TM * kLdsRow, "epilogue tile must fit in As");
  __shared__ __attribute__((aligned(16))) uint16_t As[2 * TM * kLdsRow];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2 * TN * kLdsRow];
  __shared__ int s_src[TM];
  __shared__ int s_dst[TM];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = tid >> 6;
  const int wm = wv >> 1, wn = wv & 1;
  const int total = tile_off[G];
  const int per = (total + kXcds - 1) / kXcds;
  const int lo = (blockIdx.x % kXcds) * per;
  const int hi = min(total, lo + per);
  const int stride = gridDim.x / kXcds;
  const int toff0 = lane < G ? tile_off[lane] : 0x7fffffff;
  const int toff1 = lane + 64 < G ? tile_off[lane + 64] : 0x7fffffff;
  const int Nw = kGated ? Nout / 2 : Nout;  // output row width

  const int lrow = tid >> 3;       // 0..31
  const int lcol = (tid & 7) * 8;  // element offset of this thread's 16 bytes
  const int frow = lane & 31;
  const int fk = (lane >> 5) * 8;
  const int KT = K / kTK;

  for (int L = lo + static_cast<int>(blockIdx.x) / kXcds; L < hi; L += stride) {
    int e_base;
    const int e = tile_group(L, toff0, toff1, e_base);
    const int o0 = off[e];
    const int cnt = off[e + 1] - o0;
    const int mt = (cnt + TM - 1) / TM;
    const int local = L - e_base;
    const int m = local % mt;
    const int r0 = o0 + m * TM;
    const int rows = min(TM, cnt - m * TM);
    const int n0 = (local / mt) * TN;
    const uint16_t* Wg = e < E ? W + int64_t(e) * Nout * K : Wsh + int64_t(e - E) * Nout * K;
    uint16_t* const og = e < E ? dst : dst_sh;

    for (int r = tid; r < TM; r += kGemmThreads)
      group_row<KIND>(e, E, r0, rows, r, k, off, list, row_dst, s_src[r], s_dst[r]);
    __syncthreads();

    const uint16_t* a_ptr[LA];
    const uint16_t* b_ptr[LB];
#pragma unroll
    for (int i = 0; i < LA; ++i) a_ptr[i] = A + int64_t(s_src[lrow + 32 * i]) * K + lcol;
#pragma unroll
    for (int i = 0; i < LB; ++i) b_ptr[i] = Wg + int64_t(n0 + lrow + 32 * i) * K + lcol;

    f32x16_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    u32x4_t R0[LA + LB], R1[LA + LB];
    uint16_t* const as0 = As;
    uint16_t* const as1 = As + TM * kLdsRow;
    uint16_t* const bs0 = Bs;
    uint16_t* const bs1 = Bs + TN * kLdsRow;
    const int arow0 = wm * WM, brow0 = wn * WN;

    // prologue: tile 0 in LDS buffer 0, tile 1 in R1, tile 2 in R0
    gload<LA, LB>(R0, a_ptr, b_ptr, 0);
    if (KT > 1) gload<LA, LB>(R1, a_ptr, b_ptr, kTK);
    lstore<LA, LB>(R0, as0, bs0, lrow, lcol);
    if (KT > 2) gload<LA, LB>(R0, a_ptr, b_ptr, 2 * kTK);
    __syncthreads();
    for (int kt = 0; kt < KT; kt += 2) {
      mfma_ktile<FM, FN>(acc, as0, bs0, arow0, brow0, frow, fk);          // tile kt
      if (kt + 1 < KT) {
        lstore<LA, LB>(R1, as1, bs1, lrow, lcol);                          // tile kt+1
        if (kt + 3 < KT) gload<LA, LB>(R1, a_ptr, b_ptr, (kt + 3) * kTK);
      }
      __syncthreads();
      if (kt + 1 < KT) {
        mfma_ktile<FM, FN>(acc, as1, bs1, arow0, brow0, frow, fk);        // tile kt+1
        if (kt + 2 < KT) {
          lstore<LA, LB>(R0, as0, bs0, lrow, lcol);                        // tile kt+2
          if (kt + 4 < KT) gload<LA, LB>(R0, a_ptr, b_ptr, (kt + 4) * kTK);
        }
        __syncthreads();
      }
    }

    // epilogue: activation, bf16, through LDS (reusing As), 16-byte stores.
    // D layout of a 32x32 MFMA tile: lane holds column (lane & 31) and rows
    // 8*(r/4) + 4*(lane/32) + (r%4) for r = 0..15.  Gated: the (gate, up)
    // pair of an output column sits in lanes 2c and 2c+1.
    uint16_t* cs = As;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int mr = wm * WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          const int nc = wn * WN + j * 32 + (lane & 31);
          const float v = acc[i][j][r];
          if constexpr (kGated) {
            const float up = __shfl_xor(v, 1, kWave);
            if ((lane & 1) == 0) cs[mr * CROW + (nc >> 1)] = f32_to_bf16(silu_f(v) * up);
          } else {
            cs[mr * CROW + nc] = f32_to_bf16(act_fn<ACT>(v));
          }
        }
    __syncthreads();
    constexpr int CPR = OTN / 8;  // 16-byte chunks per row
    const int on0 = kGated ? n0 / 2 : n0;
    for (int c = tid; c < TM * CPR; c += kGemmThreads) {
      const int mr = c / CPR;
      const int cc = (c % CPR) * 8;
      const int drow = s_dst[mr];
      if (drow >= 0)
        *reinterpret_cast<u32x4_t*>(og + int64_t(drow) * Nw + on0 + cc) =
            *reinterpret_cast<const u32x4_t*>(&cs[mr * CROW + cc]);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA grouped GEMM, large tile: 128 x 256 per block, 8 waves (two per
// SIMD) of 64 x 64 (four MFMA tiles each, accumulators in AGPRs), k-tile 64, a
// three-stage LDS ring filled by direct global -> LDS loads
// (global_load_lds_dwordx4: a wave's 64 x 16 bytes land contiguously at a
// wave-uniform LDS address), one barrier per k-tile.  Within a k-tile each
// wave reads the next 16-wide k-step's fragments while the current step's
// MFMAs run.  The epilogue applies the activation and writes packed bf16
// straight from the accumulators.  Each 128-byte tile row keeps its eight
// 16-byte chunks XOR-swizzled by ((row >> 1) & 7): a ds_read_b128 is served
// 16 lanes (256 bytes) at a time, and with this swizzle the 16 rows of a
// group land on distinct 16-byte bank groups.  N need not be a multiple of
// 256: weight rows past N are clamped and their columns dropped.  Used when
// the output width is at least 512.
// ---------------------------------------------------------------------------
constexpr int kBigTM = 128;
constexpr int kBigTN = 256;
constexpr int kBigWaves = 8;
constexpr int kBigThreads = kBigWaves * kWave;
constexpr int kStages = 3;
constexpr int kTileA = kBigTM * kTK;          // bf16 elements of one A stage (16 KB)
constexpr int kTileB = kBigTN * kTK;          // 32 KB
constexpr int kStageElems = kTileA + kTileB;  // 48 KB
constexpr int kLoadsA = kBigTM / 8 / kBigWaves;  // DMA instructions per wave per stage (A)
constexpr int kLoadsB = kBigTN / 8 / kBigWaves;  // (B)
constexpr int kLoadsPerStage = kLoadsA + kLoadsB;
static_assert(kProjTM == kBigTM && kProjTN == kBigTN, "projection tables use the big tile");

__device__ __forceinline__ void s_waitcnt_vm(int n) {
  // gfx9 encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] << 14
  if (n == 0) __builtin_amdgcn_s_waitcnt(0x0F70);
  else __builtin_amdgcn_s_waitcnt(0x0F70 | kLoadsPerStage);
}


// MFMA operand fragments of one 16-wide k-step: weights are the A operand
// (32 output columns x 16 k), token rows the B operand (16 k x 32 rows), so
// a lane's accumulator holds four consecutive output columns of one row.
template <int FN, int FM>
struct Frags {
  bf16x8_t w[FN];
  bf16x8_t x[FM];
};

template <int FN, int FM>
__device__ __forceinline__ void read_frags(Frags<FN, FM>& f, const uint16_t* xs,
                                           const uint16_t* ws, int xrow0, int wrow0, int ks,
                                           int lane) {
  const int rr = lane & 31;
  // swizzled chunk: ((row >> 1) & 7) == ((lane >> 1) & 7) for rows 32-aligned + (lane & 31)
  const int pos = (2 * ks + (lane >> 5)) ^ ((lane >> 1) & 7);
#pragma unroll
  for (int i = 0; i < FN; ++i)
    f.w[i] = *reinterpret_cast<const bf16x8_t*>(ws + ((wrow0 + i * 32 + rr) * 8 + pos) * 8);
#pragma unroll
  for (int j = 0; j < FM; ++j)
    f.x[j] = *reinterpret_cast<const bf16x8_t*>(xs + ((xrow0 + j * 32 + rr) * 8 + pos) * 8);
}

template <int FN, int FM>
__device__ __forceinline__ void mfma_step(f32x16_t (&acc)[FN][FM], const Frags<FN, FM>& f) {
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.w[i], f.x[j], acc[i][j], 0, 0, 0);
}

// One k-tile (four k-steps) on a swizzled stage, the next step's fragment
// reads interleaved with the current step's MFMAs; hook(ks) runs after
// k-step ks's MFMAs are issued.
template <int FN, int FM, typename Hook>
__device__ __forceinline__ void mfma_ktile_pipe(f32x16_t (&acc)[FN][FM], const uint16_t* xs,
                                                const uint16_t* ws, int xrow0, int wrow0,
                                                int lane, Hook&& hook) {
  constexpr int KS = kTK / 16;
  Frags<FN, FM> cur, nxt;
  read_frags(cur, xs, ws, xrow0, wrow0, 0, lane);
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    if (ks + 1 < KS) read_frags(nxt, xs, ws, xrow0, wrow0, ks + 1, lane);
    mfma_step(acc, cur);
    hook(ks);
    if (ks + 1 < KS) cur = nxt;
  }
  // schedule: first step's reads, then per step one MFMA per read of the
  // next step, the step's remaining MFMAs, and the last step's MFMAs
  __builtin_amdgcn_sched_group_barrier(0x100, FN + FM, 0);
#pragma unroll
  for (int ks = 0; ks + 1 < KS; ++ks) {
#pragma unroll
    for (int r = 0; r < FN + FM; ++r) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, FN * FM - (FN + FM), 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, FN * FM, 0);
}

typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

// Four fp32 -> four bf16 (hardware round to nearest even), packed in 8 bytes.
__device__ __forceinline__ u32x2_t pack4_bf16(float a, float b, float c, float d) {
  const bf16x2_t lo = __builtin_convertvector(f32x2_t{a, b}, bf16x2_t);
  const bf16x2_t hi = __builtin_convertvector(f32x2_t{c, d}, bf16x2_t);
  return u32x2_t{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
}

// One tile of the persistent walk: group, first list row, rows, first
// output column.
struct BigTile {
  int e, r0, rows, n0;
};

__device__ __forceinline__ BigTile big_tile(int L, int toff0, int toff1,
                                            const int32_t* __restrict__ off) {
  BigTile t;
  int e_base;
  t.e = tile_group(L, toff0, toff1, e_base);
  const int o0 = off[t.e];
  const int cnt = off[t.e + 1] - o0;
  const int mt = (cnt + kBigTM - 1) / kBigTM;
  const int local = L - e_base;
  const int m = local % mt;
  t.r0 = o0 + m * kBigTM;
  t.rows = min(kBigTM, cnt - m * kBigTM);
  t.n0 = (local / mt) * kBigTN;
  return t;
}

// Two fp32 -> two bf16 (hardware round to nearest even), packed in 4 bytes.
__device__ __forceinline__ uint32_t pack2_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

template <int KIND, int ACT>
__global__ __launch_bounds__(kBigThreads, 1) void gemm_bf16_big_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ W,
    const uint16_t* __restrict__ Wsh, const int32_t* __restrict__ off,
    const int32_t* __restrict__ tile_off, const int32_t* __restrict__ list,
    const int32_t* __restrict__ row_dst, int E, int G, int k, int K, int Nout,
    const float* __restrict__ bias, uint16_t* __restrict__ dst, uint16_t* __restrict__ dst_sh) {
  constexpr int TM = kBigTM, TN = kBigTN;
  constexpr bool kGated = ACT == kActSwiglu;
  constexpr int FM = 2, FN = 2;  // wave tile: 64 rows x 64 columns
  constexpr int WN = TN / (FN * 32);  // waves along N
  static_assert(kBigWaves == (TM / (FM * 32)) * WN, "wave grid must cover the tile");
  static_assert(WN == 4 && kBigWaves == 8, "the wave rotation below assumes 2 x 4 waves");
  __shared__ __attribute__((aligned(16))) uint16_t lds[kStages * kStageElems];
  __shared__ int s_src[TM];
  __shared__ int s_dst[TM];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = tid >> 6;
  // waves w and w + 4 share a SIMD; the second row of waves is rotated by
  // two columns so that each SIMD holds one wave of either row half and one
  // of either column half: a tile with only its first 64 rows, or only its
  // first 128 columns, still keeps every SIMD busy with one wave
  const int wm = wv / WN, wn = (wv + 2 * wm) % WN;
  const int total = tile_off[G];
  const int per = (total + kXcds - 1) / kXcds;
  const int lo = (blockIdx.x % kXcds) * per;
  const int hi = min(total, lo + per);
  const int stride = gridDim.x / kXcds;
  const int toff0 = lane < G ? tile_off[lane] : 0x7fffffff;
  const int toff1 = lane + 64 < G ? tile_off[lane + 64] : 0x7fffffff;
  const int KT = K / kTK;
  const int Nw = kGated ? Nout / 2 : Nout;  // output row width
  // Logical chunk this lane fetches.  DMA instruction i covers rows 8i..8i+7
  // (lane l: row 8i + l/8, stored position l & 7); the stored position is
  // chunk ^ ((row >> 1) & 7) = chunk ^ (4 (i & 1) + l / 16), and
  // i = wv + kBigWaves u has the parity of wv.
  const int chunk = (lane & 7) ^ (4 * (wv & 1) + (lane >> 4));
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(lds) + wv * 1024);

  const uint16_t* ga[kLoadsA];
  const uint16_t* gb[kLoadsB];
  // publish a tile's row table, then point this lane's loads at it
  auto start_tile = [&](const BigTile& t, int src, int dstr) __attribute__((always_inline)) {
    if (tid < TM) {
      s_src[tid] = src;
      s_dst[tid] = dstr;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kLoadsA; ++u) {
      const int r = 8 * (wv + kBigWaves * u) + (lane >> 3);
      ga[u] = A + int64_t(s_src[r]) * K + chunk * 8;
    }
    const uint16_t* Wg = t.e < E ? W + int64_t(t.e) * Nout * K : Wsh + int64_t(t.e - E) * Nout * K;
#pragma unroll
    for (int u = 0; u < kLoadsB; ++u) {
      const int r = 8 * (wv + kBigWaves * u) + (lane >> 3);
      const int n = min(t.n0 + r, Nout - 1);
      gb[u] = Wg + int64_t(n) * K + chunk * 8;
    }
  };
  // this wave's loads p0 .. p1 - 1 of k-tile kt into stage st (token rows
  // first, then weight rows)
  auto issue_part = [&](int kt, int st, int p0, int p1) __attribute__((always_inline)) {
    const uint32_t base = lds0 + st * (kStageElems * 2);
#pragma unroll
    for (int u = 0; u < kLoadsA; ++u)
      if (u >= p0 && u < p1) dma16(ga[u] + kt * kTK, base + u * kBigWaves * 1024);
#pragma unroll
    for (int u = 0; u < kLoadsB; ++u)
      if (kLoadsA + u >= p0 && kLoadsA + u < p1)
        dma16(gb[u] + kt * kTK, base + kTileA * 2 + u * kBigWaves * 1024);
  };
  auto issue = [&](int kt, int st) __attribute__((always_inline)) {
    issue_part(kt, st, 0, kLoadsPerStage);
  };

  int L = lo + static_cast<int>(blockIdx.x) / kXcds;
  if (L >= hi) return;
  BigTile cur = big_tile(L, toff0, toff1, off);
  {
    int src = 0, dstr = -1;
    if (tid < TM) group_row<KIND>(cur.e, E, cur.r0, cur.rows, tid, k, off, list, row_dst, src, dstr);
    start_tile(cur, src, dstr);
  }
  issue(0, 0);
  if (KT > 1) issue(1, 1);

  for (;;) {
    // the next tile's metadata and row table entries, loaded now and used
    // only after this tile's k-loop (which ends with every load complete)
    const int Ln = L + stride;
    const bool has_next = Ln < hi;
    BigTile nxt = cur;
    int nsrc = 0, ndst = -1;
    if (has_next) {
      nxt = big_tile(Ln, toff0, toff1, off);
      if (tid < TM)
        group_row<KIND>(nxt.e, E, nxt.r0, nxt.rows, tid, k, off, list, row_dst, nsrc, ndst);
    }

    f32x16_t acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
      for (int j = 0; j < FM; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    // a wave whose 64 x 64 sub-tile lies wholly past the tile's rows or the
    // output width skips its MFMAs (it still loads its share and syncs)
    const bool active = wm * FM * 32 < cur.rows && cur.n0 + wn * FN * 32 < Nout;
    int st = 0;
    for (int kt = 0; kt < KT; ++kt) {
      // this wave's loads of tile kt have landed once at most one later
      // tile's loads are outstanding; the barrier then publishes every
      // wave's loads and retires all reads of the stage refilled next
      if (kt + 1 < KT) s_waitcnt_vm(kLoadsPerStage);
      else s_waitcnt_vm(0);
      __builtin_amdgcn_s_barrier();
      const bool more = kt + 2 < KT;
      const int nst = st == 0 ? 2 : st - 1;
      const uint16_t* base = lds + st * kStageElems;
      if (more) issue(kt + 2, nst);
      if (active)
        mfma_ktile_pipe<FN, FM>(acc, base, base + kTileA, wm * FM * 32, wn * FN * 32, lane,
                                [](int) {});
      st = st == 2 ? 0 : st + 1;
    }

    // destination rows of this wave's accumulators, then hand the LDS over
    // to the next tile and start its loads before this tile's epilogue
    int drow[FM];
#pragma unroll
    for (int j = 0; j < FM; ++j) drow[j] = s_dst[wm * FM * 32 + j * 32 + (lane & 31)];
    __syncthreads();
    if (has_next) {
      start_tile(nxt, nsrc, ndst);
      issue(0, 0);
      if (KT > 1) issue(1, 1);
    }

    // epilogue: per 32 x 32 tile the lane holds row (lane & 31) and columns
    // 8q + 4h + s (q, s = 0..3, h = lane >> 5).  Activation and bf16 rounding, then
    // the lane pair (l, l ^ 32) exchanges runs so that lane h holds columns
    // 16p + 8h .. +7 (p = 0, 1) and each store writes 16 bytes (a 32-byte row
    // segment per lane pair).  Gated: two (gate, up) pairs -> two outputs.
    const int h = lane >> 5;
    const int c0 = cur.n0 + wn * FN * 32;
    uint16_t* const og = cur.e < E ? dst : dst_sh;
#pragma unroll
    for (int j = 0; j < FM; ++j) {
#pragma unroll
      for (int i = 0; i < FN; ++i) {
        const f32x16_t& a = acc[i][j];
        if constexpr (kGated) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int c = c0 + i * 32 + 8 * q + 4 * h;
            if (drow[j] >= 0 && c < Nout)
              *reinterpret_cast<uint32_t*>(og + int64_t(drow[j]) * Nw + (c >> 1)) =
                  pack2_bf16(silu_f(a[4 * q]) * a[4 * q + 1], silu_f(a[4 * q + 2]) * a[4 * q + 3]);
          }
        } else {
          uint32_t pk[4][2];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if constexpr (ACT == kActBias) {
              // columns c .. c + 3 of the bias (clamped: masked columns are not stored)
              const int c = c0 + i * 32 + 8 * q + 4 * h;
              float bv[4];
#pragma unroll
              for (int s2 = 0; s2 < 4; ++s2) bv[s2] = bias[min(c + s2, Nout - 1)];
              pk[q][0] = pack2_bf16(a[4 * q] + bv[0], a[4 * q + 1] + bv[1]);
              pk[q][1] = pack2_bf16(a[4 * q + 2] + bv[2], a[4 * q + 3] + bv[3]);
            } else {
              pk[q][0] = pack2_bf16(act_fn<ACT>(a[4 * q]), act_fn<ACT>(a[4 * q + 1]));
              pk[q][1] = pack2_bf16(act_fn<ACT>(a[4 * q + 2]), act_fn<ACT>(a[4 * q + 3]));
            }
          }
#pragma unroll
          for (int p = 0; p < 2; ++p) {
            // h = 0 keeps run 2p and sends run 2p + 1; h = 1 keeps 2p + 1 and sends 2p
            const uint32_t r0 = __shfl_xor(h ? pk[2 * p][0] : pk[2 * p + 1][0], 32, kWave);
            const uint32_t r1 = __shfl_xor(h ? pk[2 * p][1] : pk[2 * p + 1][1], 32, kWave);
            const uint32_t k0 = h ? pk[2 * p + 1][0] : pk[2 * p][0];
            const uint32_t k1 = h ? pk[2 * p + 1][1] : pk[2 * p][1];
            const int c = c0 + i * 32 + 16 * p + 8 * h;
            if (drow[j] >= 0 && c < Nout)
              *reinterpret_cast<u32x4_t*>(og + int64_t(drow[j]) * Nw + c) =
                  h ? u32x4_t{r0, r1, k0, k1} : u32x4_t{k0, k1, r0, r1};
          }
        }
      }
    }
    if (!has_next) break;
    L = Ln;
    cur = nxt;
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA grouped GEMM for weight-streaming steps: few rows per expert, so
// every weight byte is used by one tile and the step is bound by how fast
// the CUs pull the weights in.  The tile is 128 rows x 288 columns, so that
// an expert's up-projection rows split into equal tiles that give every CU
// about one (16 experts x 4608 rows: 256 tiles); the down projection splits
// K into SPLIT equal pieces (units), each writing its fp32 partial sums to
// part[piece][row][column], which reduce_partials_kernel adds in piece
// order.  8 waves (two per SIMD) of 32 rows x 144 columns, each 2 x 9
// v_mfma_f32_16x16x32_bf16 tiles (weights the A operand, token rows the B
// operand: a lane holds four consecutive output columns of one row), on the
// large kernel's three-stage direct-to-LDS ring of 64-wide k-tiles with the
// same XOR-swizzled 16-byte chunks.  A stage holds 128 token rows and 288
// weight rows (52 KB): 36 DMA instructions of 8 weight rows, so waves 0-3
// issue five and waves 4-7 four.  Units are numbered expert-major, then k
// piece, then N tile, then M tile, and walked like the large kernel's
// tiles (contiguous ranges per XCD): the units that share a k piece of an
// expert's rows run together on one XCD.  The weight rows, used by one unit
// each, are loaded with the non-temporal hint (the token rows, shared by an
// expert's N tiles, are not).
// ---------------------------------------------------------------------------
constexpr int kThinTM = 128;
constexpr int kThinTN = 288;
constexpr int kThinWaves = 8;
constexpr int kThinThreads = kThinWaves * kWave;
constexpr int kThinTileA = kThinTM * kTK;            // 16 KB
constexpr int kThinTileB = kThinTN * kTK;            // 36 KB
constexpr int kThinStage = kThinTileA + kThinTileB;  // 52 KB
constexpr int kThinLoadsA = kThinTM / 8 / kThinWaves;                     // 2 per wave
constexpr int kThinInstB = kThinTN / 8;                                   // 36
constexpr int kThinLoadsB = (kThinInstB + kThinWaves - 1) / kThinWaves;   // 5 (waves 0-3), 4
static_assert(kThinInstB % kThinWaves == kThinWaves / 2, "waves 0-3 issue one more weight load");

typedef __attribute__((ext_vector_type(4))) float f32x4_t;


template <int KIND, int ACT, int SPLIT>
__global__ __launch_bounds__(kThinThreads, 1) void gemm_bf16_thin_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ W,
    const int32_t* __restrict__ off, const int32_t* __restrict__ tile_off,
    const int32_t* __restrict__ list, const int32_t* __restrict__ row_dst, int E, int k, int K,
    int Nout, int64_t part_rows, uint16_t* __restrict__ dst, float* __restrict__ part) {
  constexpr int TM = kThinTM, TN = kThinTN;
  constexpr int FM = 2, FN = 9;  // 16 x 16 accumulator tiles of a wave
  static_assert(KIND != kDown || ACT == kActNone, "the down projection has no activation");
  static_assert(SPLIT == 1 || KIND == kDown, "only the down projection splits K");
  __shared__ __attribute__((aligned(16))) uint16_t lds[kStages * kThinStage];
  __shared__ int s_src[TM];
  __shared__ int s_dst[TM];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = tid >> 6;
  const int wm = wv >> 1, wn = wv & 1;  // 4 x 2 waves
  const int G = E;
  const int total = tile_off[G];
  const int per = (total + kXcds - 1) / kXcds;
  const int lo = (blockIdx.x % kXcds) * per;
  const int hi = min(total, lo + per);
  const int stride = gridDim.x / kXcds;
  const int toff0 = lane < G ? tile_off[lane] : 0x7fffffff;
  const int toff1 = lane + 64 < G ? tile_off[lane + 64] : 0x7fffffff;
  const int KT = K / kTK;
  const int NT = (Nout + TN - 1) / TN;
  // waves issuing kThinLoadsB weight loads (wave-uniform: from readfirstlane)
  const bool five = __builtin_amdgcn_readfirstlane(wv) < kThinInstB % kThinWaves;
  // stored chunk position: chunk ^ ((row >> 1) & 7) with row = 8 i + lane / 8
  // and i = wv + 8 u (the parity of wv), as in the large kernel
  const int chunk = (lane & 7) ^ (4 * (wv & 1) + (lane >> 4));
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(lds) + wv * 1024);

  struct Unit {
    int e, r0, rows, n0, ks, kt0, kt1;
  };
  auto unit = [&](int L) __attribute__((always_inline)) {
    Unit u;
    int e_base;
    u.e = tile_group(L, toff0, toff1, e_base);
    const int o0 = off[u.e];
    const int cnt = off[u.e + 1] - o0;
    const int mt = (cnt + TM - 1) / TM;
    const int local = L - e_base;
    const int m = local % mt;
    const int rest = local / mt;
    u.ks = rest / NT;
    u.r0 = o0 + m * TM;
    u.rows = min(TM, cnt - m * TM);
    u.n0 = (rest % NT) * TN;
    u.kt0 = u.ks * KT / SPLIT;
    u.kt1 = (u.ks + 1) * KT / SPLIT;
    // the unit is the same for every lane (the group comes from a ballot):
    // say so, so that the k-loop and the stage addresses stay scalar
    u.e = __builtin_amdgcn_readfirstlane(u.e);
    u.r0 = __builtin_amdgcn_readfirstlane(u.r0);
    u.rows = __builtin_amdgcn_readfirstlane(u.rows);
    u.n0 = __builtin_amdgcn_readfirstlane(u.n0);
    u.ks = __builtin_amdgcn_readfirstlane(u.ks);
    u.kt0 = __builtin_amdgcn_readfirstlane(u.kt0);
    u.kt1 = __builtin_amdgcn_readfirstlane(u.kt1);
    return u;
  };

  const uint16_t* ga[kThinLoadsA];
  const uint16_t* gb[kThinLoadsB];
  auto start_unit = [&](const Unit& t, int src, int dstr) __attribute__((always_inline)) {
    if (tid < TM) {
      s_src[tid] = src;
      s_dst[tid] = dstr;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kThinLoadsA; ++u) {
      const int r = 8 * (wv + kThinWaves * u) + (lane >> 3);
      ga[u] = A + int64_t(s_src[r]) * K + chunk * 8;
    }
    const uint16_t* Wg = W + int64_t(t.e) * Nout * K;
#pragma unroll
    for (int u = 0; u < kThinLoadsB; ++u) {
      const int r = 8 * (wv + kThinWaves * u) + (lane >> 3);
      const int n = min(t.n0 + min(r, TN - 1), Nout - 1);  // rows past the tile or N: clamped
      gb[u] = Wg + int64_t(n) * K + chunk * 8;
    }
  };
  auto issue = [&](int kt, int st) __attribute__((always_inline)) {
    const uint32_t base = lds0 + st * (kThinStage * 2);
#pragma unroll
    for (int u = 0; u < kThinLoadsA; ++u) dma16(ga[u] + kt * kTK, base + u * kThinWaves * 1024);
#pragma unroll
    for (int u = 0; u < kThinLoadsB; ++u)
      if (u + 1 < kThinLoadsB || five)
        dma16_nt(gb[u] + kt * kTK, base + kThinTileA * 2 + u * kThinWaves * 1024);
  };
  // this wave's loads of the oldest stage in flight have landed once at most
  // one later stage's loads are outstanding
  auto wait_stage = [&](bool last) __attribute__((always_inline)) {
    if (last) wait_vmcnt<0>();
    else if (five) wait_vmcnt<kThinLoadsA + kThinLoadsB>();
    else wait_vmcnt<kThinLoadsA + kThinLoadsB - 1>();
  };

  int L = lo + static_cast<int>(blockIdx.x) / kXcds;
  if (L >= hi) return;
  Unit cur = unit(L);
  {
    int src = 0, dstr = -1;
    if (tid < TM) group_row<KIND>(cur.e, E, cur.r0, cur.rows, tid, k, off, list, row_dst, src, dstr);
    start_unit(cur, src, dstr);
  }
  if (cur.kt0 < cur.kt1) issue(cur.kt0, 0);
  if (cur.kt0 + 1 < cur.kt1) issue(cur.kt0 + 1, 1);

  for (;;) {
    const int Ln = L + stride;
    const bool has_next = Ln < hi;
    Unit nxt = cur;
    int nsrc = 0, ndst = -1;
    if (has_next) {
      nxt = unit(Ln);
      if (tid < TM) group_row<KIND>(nxt.e, E, nxt.r0, nxt.rows, tid, k, off, list, row_dst, nsrc, ndst);
    }

    f32x4_t acc[FN][FM];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int i = 0; i < FM; ++i) acc[j][i] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    // a wave whose rows lie wholly past the unit's rows, or whose columns
    // past N, skips its MFMAs (it still loads its share and syncs)
    const bool active = wm * 32 < cur.rows && cur.n0 + wn * 144 < Nout;
    int st = 0;
    for (int kt = cur.kt0; kt < cur.kt1; ++kt) {
      wait_stage(kt + 1 >= cur.kt1);
      __builtin_amdgcn_s_barrier();
      if (kt + 2 < cur.kt1) issue(kt + 2, st == 0 ? 2 : st - 1);
      const uint16_t* xs = lds + st * kThinStage;
      const uint16_t* ws = xs + kThinTileA;
      if (active) {
#pragma unroll
        for (int s2 = 0; s2 < kTK / 32; ++s2) {
          const int c = 4 * s2 + (lane >> 4);  // logical 16-byte chunk of this lane
          bf16x8_t xa[FM], wb[FN];
#pragma unroll
          for (int i = 0; i < FM; ++i) {
            const int row = wm * 32 + i * 16 + (lane & 15);
            xa[i] = *reinterpret_cast<const bf16x8_t*>(xs + (row * 8 + (c ^ ((row >> 1) & 7))) * 8);
          }
#pragma unroll
          for (int j = 0; j < FN; ++j) {
            const int row = wn * 144 + j * 16 + (lane & 15);
            wb[j] = *reinterpret_cast<const bf16x8_t*>(ws + (row * 8 + (c ^ ((row >> 1) & 7))) * 8);
          }
#pragma unroll
          for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int i = 0; i < FM; ++i)
              acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wb[j], xa[i], acc[j][i], 0, 0, 0);
        }
      }
      st = st == 2 ? 0 : st + 1;
    }

    // destination rows of this wave's accumulators; then the LDS goes to the
    // next unit, whose first loads start before this unit's epilogue
    int drow[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i) drow[i] = s_dst[wm * 32 + i * 16 + (lane & 15)];
    __syncthreads();
    if (has_next) {
      start_unit(nxt, nsrc, ndst);
      if (nxt.kt0 < nxt.kt1) issue(nxt.kt0, 0);
      if (nxt.kt0 + 1 < nxt.kt1) issue(nxt.kt0 + 1, 1);
    }

    // epilogue: lane holds columns c .. c + 3 of row (lane & 15) of each
    // 16 x 16 tile, c = n0 + 144 wn + 16 j + 4 (lane >> 4)
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int r = wm * 32 + i * 16 + (lane & 15);
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int c = cur.n0 + wn * 144 + j * 16 + 4 * (lane >> 4);
        if (c >= Nout || r >= cur.rows) continue;
        const f32x4_t& a = acc[j][i];
        if constexpr (SPLIT > 1) {
          *reinterpret_cast<f32x4_t*>(part + (int64_t(cur.ks) * part_rows + cur.r0 + r) * Nout + c) = a;
        } else {
          const u32x2_t v{pack2_bf16(act_fn<ACT>(a[0]), act_fn<ACT>(a[1])),
                          pack2_bf16(act_fn<ACT>(a[2]), act_fn<ACT>(a[3]))};
          *reinterpret_cast<u32x2_t*>(dst + int64_t(drow[i]) * Nout + c) = v;
        }
      }
    }
    if (!has_next) break;
    L = Ln;
    cur = nxt;
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA up-projection for cache steps with a few hundred rows per
// expert: a tile takes all of an expert's listed rows (up to 384; more are
// split into equal parts) by 144 output columns.  On such a step every
// weight byte is loaded by one tile only, each CU gets about two tiles (16
// experts x 4608 columns: 512 tiles), and the token rows an expert's 32
// tiles share are read from L2.  8 waves (two per SIMD), wave w taking the
// 16-row tiles w, w + 8, w + 16 (a tile with fewer rows stays balanced: the
// waves of a SIMD, w and w + 4, interleave) and all 144 columns, as up to
// 3 x 9 v_mfma_f32_16x16x32_bf16 tiles (weights the A operand, token rows
// the B operand: a lane holds four consecutive output columns of one row).
// Two-stage ring of 64-wide k-tiles (2 x 66 KB) filled by direct global ->
// LDS loads with the large kernel's XOR-swizzled 16-byte chunks; the next
// k-tile's loads go out one between each weight fragment's MFMAs (issued
// in one burst they hold the wave at the load queue, away from its MFMAs),
// and loads of row groups wholly past the tile's rows are skipped.  The
// weight rows (one tile each) are loaded with the non-temporal hint.
// ---------------------------------------------------------------------------
constexpr int kWideTM = 384;
constexpr int kWideTN = 144;
constexpr int kWideWaves = 8;
constexpr int kWideThreads = kWideWaves * kWave;
constexpr int kWideTileA = kWideTM * kTK;                                // 48 KB
constexpr int kWideTileB = kWideTN * kTK;                                // 18 KB
constexpr int kWideStage = kWideTileA + kWideTileB;                      // 66 KB
constexpr int kWideInstA = kWideTM / 8;                                  // 48 DMA instructions
constexpr int kWideInstB = kWideTN / 8;                                  // 18
constexpr int kWideLoadsA = (kWideInstA + kWideWaves - 1) / kWideWaves;  // 6
constexpr int kWideLoadsB = (kWideInstB + kWideWaves - 1) / kWideWaves;  // 3 (waves 0-1), 2
static_assert(2 * kWideStage * 2 <= 163840, "two stages within the LDS");

// One 64-wide k-tile of a wide-kernel wave: its NR row tiles with rows
// (16 rows: w + 8 r) against the FN column tiles, the token-row fragments of
// a 32-wide k step held, the weight fragments read one at a time; hook(q)
// runs after the q-th weight fragment's MFMAs (q = 0 .. 2 FN - 1), so that
// the caller can spread work over the k-tile.
template <int NR, int FN, typename Hook>
__device__ __forceinline__ void wide_ktile(f32x4_t (&acc)[FN][NR], const uint16_t* xs,
                                           const uint16_t* ws, int wv, int lane, Hook&& hook) {
#pragma unroll
  for (int s2 = 0; s2 < kTK / 32; ++s2) {
    const int c = 4 * s2 + (lane >> 4);  // logical 16-byte chunk of this lane
    bf16x8_t xa[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const int row = 16 * (wv + kWideWaves * r) + (lane & 15);
      xa[r] = *reinterpret_cast<const bf16x8_t*>(xs + (row * 8 + (c ^ ((row >> 1) & 7))) * 8);
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int row = j * 16 + (lane & 15);
      const bf16x8_t wb =
          *reinterpret_cast<const bf16x8_t*>(ws + (row * 8 + (c ^ ((row >> 1) & 7))) * 8);
#pragma unroll
      for (int r = 0; r < NR; ++r)
        acc[j][r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wb, xa[r], acc[j][r], 0, 0, 0);
      hook(s2 * FN + j);
    }
  }
}

template <int ACT>
__global__ __launch_bounds__(kWideThreads, 1) void gemm_bf16_wide_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ W,
    const int32_t* __restrict__ off, const int32_t* __restrict__ tile_off,
    const int32_t* __restrict__ list, int E, int k, int K, int Nout,
    uint16_t* __restrict__ dst) {
  constexpr int FR = kWideTM / 16 / kWideWaves;  // 16-row tiles per wave (3)
  constexpr int FN = kWideTN / 16;               // 16-column tiles (9)
  static_assert(FR == 3, "the row-tile dispatch below covers zero to three");
  static_assert(kWideLoadsA + kWideLoadsB <= 2 * FN, "one load per weight fragment");
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * kWideStage];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int kwv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int total = tile_off[E];
  const int per = (total + kXcds - 1) / kXcds;
  const int lo = (blockIdx.x % kXcds) * per;
  const int hi = min(total, lo + per);
  const int stride = gridDim.x / kXcds;
  const int toff0 = lane < E ? tile_off[lane] : 0x7fffffff;
  const int toff1 = lane + 64 < E ? tile_off[lane + 64] : 0x7fffffff;
  const int KT = K / kTK;
  // stored chunk position: chunk ^ ((row >> 1) & 7) with row = 8 i + lane / 8
  // and i = wv + 8 u (the parity of wv), as in the large kernel
  const int chunk = (lane & 7) ^ (4 * (kwv & 1) + (lane >> 4));
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_addr(lds) + kwv * 1024);

  for (int L = lo + static_cast<int>(blockIdx.x) / kXcds; L < hi; L += stride) {
    int e_base;
    const int e = __builtin_amdgcn_readfirstlane(tile_group(L, toff0, toff1, e_base));
    const int o0 = off[e];
    const int cnt = off[e + 1] - o0;
    const int mt = (cnt + kWideTM - 1) / kWideTM;
    const int local = __builtin_amdgcn_readfirstlane(L - e_base);
    const int m = local % mt;
    // part m of mt equal parts of the expert's rows (at most kWideTM each)
    const int r0 = __builtin_amdgcn_readfirstlane(o0 + m * cnt / mt);
    const int rows = __builtin_amdgcn_readfirstlane(o0 + (m + 1) * cnt / mt - r0);
    const int n0 = __builtin_amdgcn_readfirstlane((local / mt) * kWideTN);

    // byte offset of each of this lane's A loads (its token row); rows past
    // the tile re-read its first row and are never stored.  Loads take a
    // wave-uniform base and these 32-bit offsets, so few registers hold them.
    uint32_t aoff[kWideLoadsA];
#pragma unroll
    for (int u = 0; u < kWideLoadsA; ++u) {
      const int r = 8 * (kwv + kWideWaves * u) + (lane >> 3);
      aoff[u] = static_cast<uint32_t>(((list[r0 + (r < rows ? r : 0)] / k) * K + chunk * 8) * 2);
    }
    const uint16_t* wg = W + (int64_t(e) * Nout + n0) * K;  // wave-uniform
    const uint32_t woff = static_cast<uint32_t>(((8 * kwv + (lane >> 3)) * K + chunk * 8) * 2);
    // the p-th of this wave's loads of k-tile kt into stage st (p <
    // kWideLoadsA: token rows, then weight rows)
    auto issue_one = [&](int kt, int st, int p) __attribute__((always_inline)) {
      const uint32_t base = lds0 + st * (kWideStage * 2);
      if (p < kWideLoadsA) {
        const int i = kwv + kWideWaves * p;
        if (8 * i < rows) dma16_s(A + kt * kTK, aoff[p], base + p * kWideWaves * 1024);
      } else {
        const int u = p - kWideLoadsA;
        if (kwv + kWideWaves * u < kWideInstB)
          dma16_s_nt(wg + int64_t(u) * (8 * kWideWaves) * K + kt * kTK, woff,
                  base + kWideTileA * 2 + u * kWideWaves * 1024);
      }
    };
    auto issue = [&](int kt, int st) __attribute__((always_inline)) {
#pragma unroll
      for (int p = 0; p < kWideLoadsA + kWideLoadsB; ++p) issue_one(kt, st, p);
    };

    // The tile for a wave with NR row tiles that hold rows (w + 8 r, r < NR):
    // k-loop and epilogue, one instantiation per NR so that each has its
    // accumulators in fixed registers and straight-line MFMAs.  Every wave
    // issues its loads and meets every barrier, NR = 0 included.
    auto run = [&](auto nr_c) __attribute__((always_inline)) {
      constexpr int NR = decltype(nr_c)::value;
      constexpr int NA = NR > 0 ? NR : 1;
      f32x4_t acc[FN][NA];
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < NA; ++r) acc[j][r] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
      issue(0, 0);
      for (int kt = 0; kt < KT; ++kt) {
        // this wave's loads of stage kt & 1 have landed; after the barrier so
        // have every wave's, and every wave is done with the other stage
        wait_vmcnt<0>();
        __builtin_amdgcn_s_barrier();
        const bool more = kt + 1 < KT;
        if constexpr (NR > 0) {
          const uint16_t* xs = lds + (kt & 1) * kWideStage;
          wide_ktile<NR, FN>(acc, xs, xs + kWideTileA, kwv, lane, [&](int q) {
            if (more && q < kWideLoadsA + kWideLoadsB) issue_one(kt + 1, (kt + 1) & 1, q);
          });
        } else {
          if (more) issue(kt + 1, (kt + 1) & 1);
        }
      }
      __syncthreads();  // every wave done with the LDS before a next tile's loads

      // epilogue: the lane holds columns 16 j + 4 g .. + 3 (g = lane >> 4) of
      // row (lane & 15) of each 16 x 16 tile.  Activation and bf16 rounding;
      // then lanes l and l ^ 16 exchange runs so that for each pair of column
      // tiles (2 p, 2 p + 1) lane g writes 16 bytes: columns 8 (g / 2) .. + 7
      // of tile 2 p + (g & 1).  The ninth tile is written in 8-byte runs.
      const int g = lane >> 4, h = g & 1;
#pragma unroll
      for (int r = 0; r < NR; ++r) {
        const int row = 16 * (kwv + kWideWaves * r) + (lane & 15);
        const bool ok = row < rows;
        uint16_t* orow = dst + int64_t(r0 + row) * Nout + n0;
        u32x2_t pk[FN];
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const f32x4_t& a = acc[j][r];
          pk[j] = u32x2_t{pack2_bf16(act_fn<ACT>(a[0]), act_fn<ACT>(a[1])),
                          pack2_bf16(act_fn<ACT>(a[2]), act_fn<ACT>(a[3]))};
        }
#pragma unroll
        for (int p = 0; p < FN / 2; ++p) {
          const u32x2_t keep = h ? pk[2 * p + 1] : pk[2 * p];
          const u32x2_t send = h ? pk[2 * p] : pk[2 * p + 1];
          const uint32_t q0 = __shfl_xor(send[0], 16, kWave);
          const uint32_t q1 = __shfl_xor(send[1], 16, kWave);
          const int col = 16 * (2 * p + h) + 4 * (g - h);
          if (ok)
            *reinterpret_cast<u32x4_t*>(orow + col) =
                h ? u32x4_t{q0, q1, keep[0], keep[1]} : u32x4_t{keep[0], keep[1], q0, q1};
        }
        if constexpr (FN % 2 == 1) {
          if (ok) *reinterpret_cast<u32x2_t*>(orow + 16 * (FN - 1) + 4 * g) = pk[FN - 1];
        }
      }
    };
    // this wave's row tiles with rows (wave-uniform)
    const int nr = __builtin_amdgcn_readfirstlane(((rows + 15) / 16 - kwv + kWideWaves - 1) / kWideWaves);
    switch (nr) {
      case 3: run(std::integral_constant<int, 3>{}); break;
      case 2: run(std::integral_constant<int, 2>{}); break;
      case 1: run(std::integral_constant<int, 1>{}); break;
      default: run(std::integral_constant<int, 0>{}); break;
    }
  }
}

// h_c[row_dst[r]] = bf16(((part[0][r] + part[1][r]) + ...) + part[S-1][r])
// for the listed rows r < off[E] (the down projection's K pieces, added in
// piece order); one wave per row, 16 bytes of bf16 per lane and step.
template <int SPLIT>
__global__ __launch_bounds__(256) void reduce_partials_kernel(
    const float* __restrict__ part, int64_t part_rows, const int32_t* __restrict__ off,
    const int32_t* __restrict__ row_dst, int E, int d, uint16_t* __restrict__ h_c) {
  const int lane = threadIdx.x & (kWave - 1);
  const int r = static_cast<int>(blockIdx.x) * 4 + static_cast<int>(threadIdx.x) / kWave;
  if (r >= off[E]) return;
  const int64_t drow = row_dst[r];
  for (int g = lane; g < d / 8; g += kWave) {
    f32x4_t s0 = *reinterpret_cast<const f32x4_t*>(part + int64_t(r) * d + g * 8);
    f32x4_t s1 = *reinterpret_cast<const f32x4_t*>(part + int64_t(r) * d + g * 8 + 4);
#pragma unroll
    for (int p = 1; p < SPLIT; ++p) {
      const float* q = part + (int64_t(p) * part_rows + r) * d + g * 8;
      const f32x4_t a0 = *reinterpret_cast<const f32x4_t*>(q);
      const f32x4_t a1 = *reinterpret_cast<const f32x4_t*>(q + 4);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        s0[u] = __fadd_rn(s0[u], a0[u]);
        s1[u] = __fadd_rn(s1[u], a1[u]);
      }
    }
    *reinterpret_cast<u32x4_t*>(h_c + drow * d + g * 8) =
        u32x4_t{pack2_bf16(s0[0], s0[1]), pack2_bf16(s0[2], s0[3]), pack2_bf16(s1[0], s1[1]),
                pack2_bf16(s1[2], s1[3])};
  }
}

// ---------------------------------------------------------------------------
// fp32 grouped GEMM (fp32 layers): 64 x 64 block tile (token rows by output
// columns), 16-wide k-steps through LDS, four waves of 32 x 32 on the fp32
// matrix cores (v_mfma_f32_32x32x2_f32, fp32 products accumulated in fp32).
// ---------------------------------------------------------------------------
constexpr int kF32T = 64;
constexpr int kF32K = 16;

template <int KIND, int ACT>
__global__ __launch_bounds__(256) void gemm_f32_kernel(
    const float* __restrict__ A, const float* __restrict__ W, const float* __restrict__ Wsh,
    const int32_t* __restrict__ off, const int32_t* __restrict__ list,
    const int32_t* __restrict__ row_dst, int E, int G, int k, int K, int Nout,
    float* __restrict__ dst, float* __restrict__ dst_sh) {
  constexpr bool kGated = ACT == kActSwiglu;
  __shared__ float As[kF32K][kF32T + 4];  // token rows, k-major
  __shared__ float Bs[kF32K][kF32T + 4];  // weight rows, k-major
  __shared__ int s_src[kF32T];
  __shared__ int s_dst[kF32T];
  __shared__ int s_tile[4];
  const int tid = threadIdx.x;
  if (tid == 0) {
    const Tile t = decode_tile<kF32T>(off, G, Nout / kF32T);
    s_tile[0] = t.e;
    s_tile[1] = t.r0;
    s_tile[2] = t.rows;
    s_tile[3] = t.n0 * kF32T;
  }
  __syncthreads();
  const int e = s_tile[0];
  if (e < 0) return;
  const int r0 = s_tile[1], rows = s_tile[2], n0 = s_tile[3];
  if (tid < kF32T) group_row<KIND>(e, E, r0, rows, tid, k, off, list, row_dst, s_src[tid], s_dst[tid]);
  __syncthreads();
  // tile loads: thread -> row lr, k columns lk .. lk + 3 of the 16-wide k-step
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  const float* Wg = e < E ? W + int64_t(e) * Nout * K : Wsh + int64_t(e - E) * Nout * K;
  float* const og = e < E ? dst : dst_sh;
  const float* ap = A + int64_t(s_src[lr]) * K + lk;
  const float* bp = Wg + int64_t(n0 + lr) * K + lk;
  // MFMA: wave w computes outputs 32 (w & 1) .. + 31 (weights, the A operand)
  // by tokens 32 (w >> 1) .. + 31 (the B operand) with v_mfma_f32_32x32x2_f32;
  // lane l supplies output / token (l & 31) at k-row l >> 5 of each 2-wide
  // k-step and holds D[8 (v / 4) + 4 (l >> 5) + v % 4][l & 31] in acc[v]:
  // four consecutive outputs of one token per group v / 4
  const int lane = tid & 63, wv = tid >> 6;
  const int wo = (wv & 1) * 32, wt = (wv >> 1) * 32;
  const int lc = lane & 31, lh = lane >> 5;
  typedef __attribute__((ext_vector_type(16))) float f32x16_v;
  f32x16_v acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
  for (int k0 = 0; k0 < K; k0 += kF32K) {
    const float4 va = *reinterpret_cast<const float4*>(ap + k0);
    const float4 vb = *reinterpret_cast<const float4*>(bp + k0);
    As[lk + 0][lr] = va.x;
    As[lk + 1][lr] = va.y;
    As[lk + 2][lr] = va.z;
    As[lk + 3][lr] = va.w;
    Bs[lk + 0][lr] = vb.x;
    Bs[lk + 1][lr] = vb.y;
    Bs[lk + 2][lr] = vb.z;
    Bs[lk + 3][lr] = vb.w;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kF32K; kk += 2)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(Bs[kk + lh][wo + lc], As[kk + lh][wt + lc], acc,
                                                 0, 0, 0);
    __syncthreads();
  }
  const int drow = s_dst[wt + lc];
  if (drow < 0) return;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int c = n0 + wo + 8 * q + 4 * lh;  // outputs c .. c + 3
    if constexpr (kGated) {  // columns (gate, up, gate, up) -> two outputs
      *reinterpret_cast<float2*>(og + int64_t(drow) * (Nout / 2) + c / 2) =
          make_float2(silu_f(acc[4 * q]) * acc[4 * q + 1], silu_f(acc[4 * q + 2]) * acc[4 * q + 3]);
    } else {
      *reinterpret_cast<float4*>(og + int64_t(drow) * Nout + c) =
          make_float4(act_fn<ACT>(acc[4 * q]), act_fn<ACT>(acc[4 * q + 1]),
                      act_fn<ACT>(acc[4 * q + 2]), act_fn<ACT>(acc[4 * q + 3]));
    }
  }
}

int max_tiles(const Shape& s, int TM, int NT) {
  const int64_t mt = (s.mid_rows() + TM - 1) / TM + s.groups();
  const int64_t g = mt * NT;
  return static_cast<int>((g + kXcds - 1) / kXcds * kXcds);
}

constexpr int kBlocksPerCu = 2;

// Grouped GEMM over the E routed groups (weights W, outputs dst) and the S
// shared groups (weights Wsh, outputs dst_sh) with Nout weight rows and K
// inputs per group.
template <int KIND, int ACT>
hipError_t launch_gemm(const Shape& s, const FfnPlan& plan, const void* A, const void* W,
                       const void* Wsh, int K, int Nout, const Buffers& b, void* dst, void* dst_sh,
                       hipStream_t st) {
  const int G = s.groups();
  if (KIND == kUp && plan.wide_up) {
    // bf16, ungated, no shared experts (wide_capable)
    if constexpr (ACT == kActSwiglu || ACT == kActBias || KIND != kUp) {
      return hipErrorInvalidValue;
    } else {
      launch_kernel(&gemm_bf16_wide_kernel<ACT>, dim3(device_cus()), dim3(kWideThreads), 0, st,
                    static_cast<const uint16_t*>(A), static_cast<const uint16_t*>(W), b.off,
                    b.tiles, b.list, s.E, s.k, K, Nout, static_cast<uint16_t*>(dst));
      return hipGetLastError();
    }
  }
  if (plan.thin) {
    // bf16, ungated, no shared experts (thin_capable)
    if constexpr (ACT == kActSwiglu || ACT == kActBias) {
      return hipErrorInvalidValue;
    } else {
      const int32_t* toff = b.tiles + (KIND == kUp ? 0 : G + 1);
      const auto* a = static_cast<const uint16_t*>(A);
      const auto* w = static_cast<const uint16_t*>(W);
      const int64_t rows = s.mid_rows();
      if (KIND == kDown && plan.split_down == kThinSplit && b.part != nullptr) {
        // the stage's start event goes with the GEMM, its stop event with
        // the addition of the partial sums
        const LaunchEvents ev = launch_events();
        launch_events() = LaunchEvents{};
        launch_kernel_ev(&gemm_bf16_thin_kernel<kDown, kActNone, kThinSplit>, dim3(device_cus()),
                         dim3(kThinThreads), 0, st, ev.start, nullptr, a, w, b.off, toff, b.list,
                         b.row_dst, s.E, s.k, K, Nout, rows, static_cast<uint16_t*>(nullptr),
                         b.part);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        launch_kernel_ev(&reduce_partials_kernel<kThinSplit>,
                         dim3(static_cast<unsigned>((rows + 3) / 4)), dim3(256), 0, st, nullptr,
                         ev.stop, static_cast<const float*>(b.part), rows, b.off, b.row_dst, s.E,
                         s.d, static_cast<uint16_t*>(b.h_c));
      } else if (KIND == kDown) {
        launch_kernel(&gemm_bf16_thin_kernel<kDown, kActNone, 1>, dim3(device_cus()),
                      dim3(kThinThreads), 0, st, a, w, b.off, toff, b.list, b.row_dst, s.E, s.k,
                      K, Nout, rows, static_cast<uint16_t*>(dst), static_cast<float*>(nullptr));
      } else {
        launch_kernel(&gemm_bf16_thin_kernel<kUp, ACT, 1>, dim3(device_cus()),
                      dim3(kThinThreads), 0, st, a, w, b.off, toff, b.list, b.row_dst, s.E, s.k,
                      K, Nout, rows, static_cast<uint16_t*>(dst), static_cast<float*>(nullptr));
      }
      return hipGetLastError();
    }
  }
  if (s.bf16) {
    const int tn = KIND == kUp ? plan.tn_up : plan.tn_down;
    const int32_t* toff = b.tiles + (KIND == kUp ? 0 : G + 1);
    const int grid = device_cus() * kBlocksPerCu;  // multiple of 8
    const auto* a = static_cast<const uint16_t*>(A);
    const auto* w = static_cast<const uint16_t*>(W);
    const auto* wsh = static_cast<const uint16_t*>(Wsh);
    auto* o = static_cast<uint16_t*>(dst);
    auto* osh = static_cast<uint16_t*>(dst_sh);
    if (tn == kBigTN) {
      launch_kernel(&gemm_bf16_big_kernel<KIND, ACT>, dim3(device_cus()), dim3(kBigThreads), 0, st,
          a, w, wsh, b.off, toff, b.list, b.row_dst, s.E, G, s.k, K, Nout,
          static_cast<const float*>(nullptr), o, osh);
    } else if (tn == 128) {
      launch_kernel(&gemm_bf16_kernel<128, 128, KIND, ACT>, dim3(grid), dim3(kGemmThreads), 0, st,
          a, w, wsh, b.off, toff, b.list, b.row_dst, s.E, G, s.k, K, Nout, o, osh);
    } else {
      launch_kernel(&gemm_bf16_kernel<128, 64, KIND, ACT>, dim3(grid), dim3(kGemmThreads), 0, st,
          a, w, wsh, b.off, toff, b.list, b.row_dst, s.E, G, s.k, K, Nout, o, osh);
    }
  } else {
    launch_kernel(&gemm_f32_kernel<KIND, ACT>, dim3(max_tiles(s, kF32T, Nout / kF32T)), dim3(256),
        0, st, static_cast<const float*>(A), static_cast<const float*>(W),
        static_cast<const float*>(Wsh), b.off, b.list, b.row_dst, s.E, G, s.k, K, Nout,
        static_cast<float*>(dst), static_cast<float*>(dst_sh));
  }
  return hipGetLastError();
}

}  // namespace

// Weight-row counts of at least 512 take the large 128 x 256 tile (a
// partial last N tile is masked); smaller ones the 128 x 128 / 128 x 64
// tiles; the thin plan the 128 x 288 tile; the wide plan the expert-wide
// 384 x 144 up-projection tile (the down projection keeps the large tile).
FfnPlan ffn_plan(const Shape& s, bool thin, bool wide) {
  auto tn = [](int n) { return n >= 512 ? kBigTN : (n % 128 == 0 ? 128 : 64); };
  FfnPlan p;
  p.tm = p.tm_up = 128;
  if (thin && thin_capable(s)) {
    p.thin = true;
    p.tn_up = p.tn_down = kThinTN;
    p.split_down = kThinSplit;
    return p;
  }
  p.tn_up = tn(s.up_rows());
  p.tn_down = tn(s.d);
  if (wide && wide_capable(s)) {
    p.wide_up = true;
    p.tm_up = kWideTM;
    p.tn_up = kWideTN;
  }
  return p;
}

bool wide_capable(const Shape& s) {
  return s.bf16 && s.S == 0 && !s.swiglu && s.E <= 64 && s.up_rows() % kWideTN == 0 &&
         s.d % kTK == 0 && s.tokens() * s.d < (int64_t(1) << 31);
}

bool thin_capable(const Shape& s) {
  const int nt = (s.up_rows() + kThinTN - 1) / kThinTN;
  return s.bf16 && s.S == 0 && !s.swiglu && s.E <= 64 && s.branches() <= int64_t(256) * s.E &&
         2 * s.E * nt >= device_cus();
}

int cus_per_xcd() { return device_cus() / kXcds; }

int device_cus() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        n > 0)
      cus = (n + kXcds - 1) / kXcds * kXcds;
    else
      cus = 256;
  }
  return cus;
}

hipError_t launch_ffn_up(const Shape& s, const void* x, const void* W_up, const void* W_up_sh,
                         int act, const FfnPlan& plan, const Buffers& b, hipStream_t st) {
  const int n = s.up_rows();
  if (act == MOECA_ACT_SWIGLU)
    return launch_gemm<kUp, kActSwiglu>(s, plan, x, W_up, W_up_sh, s.d, n, b, b.mid, b.mid, st);
  if (act == MOECA_ACT_GELU_ERF)
    return launch_gemm<kUp, kActGeluErf>(s, plan, x, W_up, W_up_sh, s.d, n, b, b.mid, b.mid, st);
  return launch_gemm<kUp, kActGeluTanh>(s, plan, x, W_up, W_up_sh, s.d, n, b, b.mid, b.mid, st);
}

hipError_t launch_ffn_down(const Shape& s, const void* W_down, const void* W_down_sh,
                           const FfnPlan& plan, const Buffers& b, hipStream_t st) {
  return launch_gemm<kDown, kActNone>(s, plan, b.mid, W_down, W_down_sh, s.d_ff, s.d, b, b.h_c,
                                      b.h_sh, st);
}

hipError_t launch_proj(const void* A, const void* W, const float* bias, const int32_t* off,
                       const int32_t* tiles, const int32_t* list, int K, int Nout, void* dst,
                       hipStream_t st, int blocks_per_xcd) {
  if (K % kTK != 0 || Nout < 1 || blocks_per_xcd < 0) return hipErrorInvalidValue;
  // the grid stays a multiple of the XCD count (block b runs on XCD b % 8)
  const int grid = blocks_per_xcd > 0 ? kXcds * std::min(blocks_per_xcd, cus_per_xcd())
                                      : device_cus();
  const auto* w = static_cast<const uint16_t*>(W);
  launch_kernel(&gemm_bf16_big_kernel<kProj, kActBias>, dim3(grid), dim3(kBigThreads), 0,
                st, static_cast<const uint16_t*>(A), w, w, off, tiles, list,
                static_cast<const int32_t*>(nullptr), 1, 1, 1, K, Nout, bias,
                static_cast<uint16_t*>(dst), static_cast<uint16_t*>(dst));
  return hipGetLastError();
}

}  // namespace moeca
