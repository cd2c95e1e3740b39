// Small device helpers shared by the gfx950 kernels: bf16 unpacking and
// wave64 reductions / scans built on DPP and lane-swap instructions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fva {

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Orders LDS traffic of one wavefront without a workgroup barrier.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Lane exchanges without LDS: DPP moves inside rows of 16 lanes (kCtrl is
// the DPP control word) and the gfx950 row-swap instructions across rows.
template <int kCtrl>
__device__ __forceinline__ uint32_t dpp_move(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kCtrl, 0xF, 0xF, false);
}
// Lanes whose source lane i - n lies before the start of their row read 0.
template <int kN>
__device__ __forceinline__ uint32_t dpp_row_shr(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x110 + kN, 0xF, 0xF, true);
}

__device__ __forceinline__ uint64_t u64_of(double v) { return (uint64_t)__double_as_longlong(v); }
__device__ __forceinline__ uint64_t u64_of(uint64_t v) { return v; }
template <typename T>
__device__ __forceinline__ T from_u64(uint64_t b);
template <>
__device__ __forceinline__ double from_u64<double>(uint64_t b) { return __longlong_as_double((long long)b); }
template <>
__device__ __forceinline__ uint64_t from_u64<uint64_t>(uint64_t b) { return b; }
__device__ __forceinline__ uint64_t join64(uint32_t lo, uint32_t hi) { return ((uint64_t)hi << 32) | lo; }

// All-lane reduction of a 64-bit value with a commutative op as a butterfly:
// partners l^1, l^2 (quad permutes), mirror within 8 and within 16 lanes,
// then rows l^16 and l^32. Both partners of every step combine the same two
// operands, so all 64 lanes end with the same bits (also for fp64 sums). The
// result is returned through the scalar unit.
template <typename T, typename Op>
__device__ __forceinline__ T wave_allreduce(T v, Op op) {
  auto step_dpp = [&](auto mover) {
    const uint64_t b = u64_of(v);
    v = op(v, from_u64<T>(join64(mover((uint32_t)b), mover((uint32_t)(b >> 32)))));
  };
  step_dpp([](uint32_t x) { return dpp_move<0xB1>(x); });   // lane ^ 1
  step_dpp([](uint32_t x) { return dpp_move<0x4E>(x); });   // lane ^ 2
  step_dpp([](uint32_t x) { return dpp_move<0x141>(x); });  // 7 - lane within 8
  step_dpp([](uint32_t x) { return dpp_move<0x140>(x); });  // 15 - lane within 16
  {
    const uint64_t b = u64_of(v);
    const auto lo = __builtin_amdgcn_permlane16_swap((uint32_t)b, (uint32_t)b, false, false);
    const auto hi = __builtin_amdgcn_permlane16_swap((uint32_t)(b >> 32), (uint32_t)(b >> 32), false, false);
    v = op(from_u64<T>(join64(lo[0], hi[0])), from_u64<T>(join64(lo[1], hi[1])));
  }
  {
    const uint64_t b = u64_of(v);
    const auto lo = __builtin_amdgcn_permlane32_swap((uint32_t)b, (uint32_t)b, false, false);
    const auto hi = __builtin_amdgcn_permlane32_swap((uint32_t)(b >> 32), (uint32_t)(b >> 32), false, false);
    v = op(from_u64<T>(join64(lo[0], hi[0])), from_u64<T>(join64(lo[1], hi[1])));
  }
  const uint64_t b = u64_of(v);
  return from_u64<T>(join64(__builtin_amdgcn_readfirstlane((uint32_t)b),
                            __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32))));
}

__device__ __forceinline__ double wave_max(double v) {
  return wave_allreduce(v, [](double a, double b) { return fmax(a, b); });
}
__device__ __forceinline__ double wave_min(double v) {
  return wave_allreduce(v, [](double a, double b) { return fmin(a, b); });
}
__device__ __forceinline__ double wave_sum(double v) {
  return wave_allreduce(v, [](double a, double b) { return a + b; });
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  return wave_allreduce(v, [](uint64_t a, uint64_t b) { return a + b; });
}

// 64-bit lane value of lane `src` (wave-uniform) through the scalar unit.
__device__ __forceinline__ uint64_t lane_u64(uint64_t v, int src) {
  return join64(__builtin_amdgcn_readlane((uint32_t)v, src), __builtin_amdgcn_readlane((uint32_t)(v >> 32), src));
}

// Inclusive prefix sum over lanes 0..63: Hillis-Steele steps 1, 2, 4, 8
// inside each row of 16 lanes, then the totals of the rows below are added.
__device__ __forceinline__ uint64_t wave_incl_scan_u64(uint64_t v, int lane) {
  v += join64(dpp_row_shr<1>((uint32_t)v), dpp_row_shr<1>((uint32_t)(v >> 32)));
  v += join64(dpp_row_shr<2>((uint32_t)v), dpp_row_shr<2>((uint32_t)(v >> 32)));
  v += join64(dpp_row_shr<4>((uint32_t)v), dpp_row_shr<4>((uint32_t)(v >> 32)));
  v += join64(dpp_row_shr<8>((uint32_t)v), dpp_row_shr<8>((uint32_t)(v >> 32)));
  const uint64_t r0 = lane_u64(v, 15), r1 = lane_u64(v, 31), r2 = lane_u64(v, 47);
  const int row = lane >> 4;
  return v + (row == 0 ? 0ull : row == 1 ? r0 : row == 2 ? r0 + r1 : r0 + r1 + r2);
}

__device__ __forceinline__ int wave_incl_scan_i32(int v, int lane) {
  v += (int)dpp_row_shr<1>((uint32_t)v);
  v += (int)dpp_row_shr<2>((uint32_t)v);
  v += (int)dpp_row_shr<4>((uint32_t)v);
  v += (int)dpp_row_shr<8>((uint32_t)v);
  const int r0 = __builtin_amdgcn_readlane(v, 15), r1 = __builtin_amdgcn_readlane(v, 31),
            r2 = __builtin_amdgcn_readlane(v, 47);
  const int row = lane >> 4;
  return v + (row == 0 ? 0 : row == 1 ? r0 : row == 2 ? r0 + r1 : r0 + r1 + r2);
}

// Number of set bits of `mask` below this lane.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

}  // namespace fva
