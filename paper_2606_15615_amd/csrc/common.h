// Device helpers shared by the MoECa kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace moeca {

constexpr int kWave = 64;

// ---- bf16 storage ---------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t u) {
  return __uint_as_float(static_cast<uint32_t>(u) << 16);
}

// fp32 -> bf16, round to nearest, ties to even; NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

template <typename T> struct Act;
template <> struct Act<uint16_t> {
  static __device__ __forceinline__ float to_f32(uint16_t v) { return bf16_to_f32(v); }
  static __device__ __forceinline__ uint16_t from_f32(float v) { return f32_to_bf16(v); }
};
template <> struct Act<float> {
  static __device__ __forceinline__ float to_f32(float v) { return v; }
  static __device__ __forceinline__ float from_f32(float v) { return v; }
};

// ---- direct global -> LDS loads ---------------------------------------------
// 16 bytes per lane, global -> LDS at the wave-uniform LDS byte address
// `lds` (lane l lands at lds + 16 l).  Issued as inline assembly so that the
// compiler does not treat it as an LDS store: it would otherwise wait for
// every outstanding DMA before each LDS read.  The kernel orders the
// accesses itself with s_waitcnt vmcnt and s_barrier (loads complete in
// order, so the compiler's own vmcnt waits stay conservative).  m0 is
// reserved by the compiler, which may not preserve it around the statement:
// this is safe because no kernel here has other m0 uses (the generated code
// contains no m0 access besides these statements).
__device__ __forceinline__ void dma16(const uint16_t* g, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off"
      :
      : "s"(lds), "v"(g)
      : "memory", "m0");
}

// The same load with a wave-uniform 64-bit base (SGPRs) and a per-lane
// 32-bit byte offset: the lane reads base + voff.
__device__ __forceinline__ void dma16_s(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2"
      :
      : "s"(lds), "v"(voff), "s"(base)
      : "memory", "m0");
}

// The same two loads with the non-temporal hint, for a stream whose every
// byte feeds one tile (the expert weights of the weight-streaming and
// expert-wide tilings): its lines are not kept for reuse, so the stream
// neither displaces the step's other data from the caches nor, on a miss in
// the last-level cache, forces that cache's dirty lines out to HBM before
// it can be served.  Not for operands that several tiles share through L2.
__device__ __forceinline__ void dma16_nt(const uint16_t* g, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off nt"
      :
      : "s"(lds), "v"(g)
      : "memory", "m0");
}

__device__ __forceinline__ void dma16_s_nt(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2 nt"
      :
      : "s"(lds), "v"(voff), "s"(base)
      : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const void*)p));
}

// Wait until at most N vector memory operations of this wave are in flight
// (gfx9 encoding of s_waitcnt, N < 16; expcnt and lgkmcnt not waited for).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

// ---- lane exchange within 16-lane rows (DPP) -------------------------------
// Row permutations: xor 1, xor 2, half-row mirror, row mirror.  Applied in
// this order, a commutative reduction leaves every lane of the row with the
// same result (each step combines two lanes that already agree).
constexpr int kDppRow[4] = {0xB1, 0x4E, 0x141, 0x140};

template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(dpp_i32<CTRL>(__float_as_int(v)));
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const int lo = dpp_i32<CTRL>(static_cast<int>(u & 0xffffffffu));
  const int hi = dpp_i32<CTRL>(static_cast<int>(u >> 32));
  return __builtin_bit_cast(double, (uint64_t(uint32_t(hi)) << 32) | uint32_t(lo));
}

__device__ __forceinline__ double row_sum_f64(double v) {
  v += dpp_f64<kDppRow[0]>(v);
  v += dpp_f64<kDppRow[1]>(v);
  v += dpp_f64<kDppRow[2]>(v);
  return v + dpp_f64<kDppRow[3]>(v);
}
__device__ __forceinline__ int row_sum_i32(int v) {
  v += dpp_i32<kDppRow[0]>(v);
  v += dpp_i32<kDppRow[1]>(v);
  v += dpp_i32<kDppRow[2]>(v);
  return v + dpp_i32<kDppRow[3]>(v);
}

// ---- wave reductions: every lane ends with the same value -----------------
// Row sums (DPP), then the four row results in a fixed order,
// (row0 + row1) + (row2 + row3).
__device__ __forceinline__ double wave_sum_f64(double v) {
  v = row_sum_f64(v);
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  double r[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(u & 0xffffffffu), 16 * q);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(u >> 32), 16 * q);
    r[q] = __builtin_bit_cast(double, (uint64_t(hi) << 32) | lo);
  }
  return (r[0] + r[1]) + (r[2] + r[3]);
}

__device__ __forceinline__ int wave_sum_i32(int v) {
  v = row_sum_i32(v);
  return (__builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16)) +
         (__builtin_amdgcn_readlane(v, 32) + __builtin_amdgcn_readlane(v, 48));
}

// Inclusive prefix sum over the wave's lanes (integers): a Hillis-Steele
// scan inside each 16-lane row (row shifts by 1, 2, 4, 8; lanes shifted in
// from outside the row read 0), then the totals of the rows before.
__device__ __forceinline__ int wave_incl_scan_i32(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, true);
  const int row = (threadIdx.x & (kWave - 1)) >> 4;
  const int t0 = __builtin_amdgcn_readlane(v, 15);
  const int t1 = __builtin_amdgcn_readlane(v, 31);
  const int t2 = __builtin_amdgcn_readlane(v, 47);
  return v + (row > 0 ? t0 : 0) + (row > 1 ? t1 : 0) + (row > 2 ? t2 : 0);
}

// Block-wide fp64 sum for blocks of NW waves; every thread gets the result.
// `scratch` must hold NW doubles; the call contains two barriers.
template <int NW>
__device__ __forceinline__ double block_sum_f64(double v, double* scratch) {
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  v = wave_sum_f64(v);
  if (lane == 0) scratch[w] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int i = 0; i < NW; ++i) s += scratch[i];
  __syncthreads();
  return s;
}

// Number of set bits of `mask` below this lane.
__device__ __forceinline__ int lane_rank(uint64_t mask) {
  const int lane = threadIdx.x & (kWave - 1);
  return __popcll(mask & ((1ull << lane) - 1ull));
}

// fp32 -> uint32 whose unsigned order is the numeric order (-0 and +0 equal).
__device__ __forceinline__ uint32_t f32_order_key(float f) {
  uint32_t u = __float_as_uint(f + 0.0f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace moeca
