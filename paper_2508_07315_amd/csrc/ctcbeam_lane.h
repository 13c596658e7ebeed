// Cross-lane building blocks of the gfx950 decode kernels (wave64): lane
// reads, DPP / permlane exchanges, wave prefix sums, bitonic steps, the
// transcript hash and the candidate order key.  Included by both kernel
// sources (the general decoder and the small-beam decoder).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ctcbeam {
namespace detail {

constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ uint64_t mix_token(uint64_t h, uint32_t c) {
  uint64_t z = h + (static_cast<uint64_t>(c) + 1ull) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Order key: larger is better; (x desc, idx asc); -0 and +0 compare equal.
__device__ __forceinline__ uint64_t order_key(float x, uint32_t idx) {
  const float y = x + 0.0f;
  uint32_t u = __float_as_uint(y);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<uint64_t>(u) << 32) | static_cast<uint64_t>(0xFFFFFFFFu - idx);
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const uint32_t lane = threadIdx.x & 63u;
  return lane == 0 ? 0ull : (~0ull >> (64u - lane));
}

__device__ __forceinline__ int rdlane(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ uint32_t rdlane(uint32_t v, int l) {
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), l));
}
__device__ __forceinline__ float rdlane(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

// ---- cross-lane exchange on gfx950 without the LDS crossbar ----
// DPP row/quad patterns for distances 1..8 and the gfx950 permlane swaps for
// 16 and 32.  update_dpp with bound_ctrl off returns `old` (0) for lanes whose
// source lies outside the row.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), CTRL, 0xF, 0xF, false));
}
// DPP move for patterns whose source lane is valid for every lane
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_full(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(v), CTRL, 0xF, 0xF, false));
}
// per-lane predicate from a compile-time lane mask (an SGPR constant used as
// the select mask, no per-lane arithmetic)
__device__ __forceinline__ bool lane_in(uint64_t mask) { return __builtin_amdgcn_inverse_ballot_w64(mask); }
// the same, with the constant materialised where it is used: loops with many
// such masks would otherwise keep them all live in SGPRs across the loop
template <uint64_t M>
__device__ __forceinline__ bool lane_in_here() {
  uint32_t lo, hi;
  asm volatile("s_mov_b32 %0, %1" : "=s"(lo) : "i"(static_cast<uint32_t>(M)));
  asm volatile("s_mov_b32 %0, %1" : "=s"(hi) : "i"(static_cast<uint32_t>(M >> 32)));
  return __builtin_amdgcn_inverse_ballot_w64((static_cast<uint64_t>(hi) << 32) | lo);
}
constexpr uint64_t kLanesBit2 = 0xF0F0F0F0F0F0F0F0ull;   // lane & 4
constexpr uint64_t kLanesBit4 = 0xFFFF0000FFFF0000ull;   // lane & 16
constexpr uint64_t kLanesBit5 = 0xFFFFFFFF00000000ull;   // lane & 32
constexpr uint64_t kLanesGe16 = 0xFFFFFFFFFFFF0000ull;
constexpr uint64_t kLanesGe48 = 0xFFFF000000000000ull;
template <int CTRL>
__device__ __forceinline__ float dpp_movf(float v, float old) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]
constexpr int kDppRowShl4 = 0x104;
constexpr int kDppRowShr1 = 0x111;
constexpr int kDppRowShr2 = 0x112;
constexpr int kDppRowShr4 = 0x114;
constexpr int kDppRowShr8 = 0x118;
constexpr int kDppRowRor8 = 0x128;
// rotation by D within each 16-lane row (D = 0: the value itself)
template <int D>
__device__ __forceinline__ uint32_t dpp_row_ror(uint32_t v) {
  if constexpr (D == 0) return v;
  else return dpp_full<0x120 + D>(v);
}

// value of lane (lane ^ j); j must be a compile-time power of two <= 32 after
// unrolling
__device__ __forceinline__ uint32_t xor_lane(uint32_t v, int j, int lane) {
  (void)lane;
  switch (j) {
    case 1: return dpp_full<kDppQuadXor1>(v);
    case 2: return dpp_full<kDppQuadXor2>(v);
    case 4: {
      const uint32_t up = dpp_mov<kDppRowShl4>(v);
      const uint32_t dn = dpp_mov<kDppRowShr4>(v);
      return lane_in(kLanesBit2) ? dn : up;
    }
    case 8: return dpp_full<kDppRowRor8>(v);
    case 16: {
      const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
      return lane_in(kLanesBit4) ? static_cast<uint32_t>(r[0]) : static_cast<uint32_t>(r[1]);
    }
    default: {
      const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
      return lane_in(kLanesBit5) ? static_cast<uint32_t>(r[0]) : static_cast<uint32_t>(r[1]);
    }
  }
}
__device__ __forceinline__ float xor_lane(float v, int j, int lane) {
  return __uint_as_float(xor_lane(__float_as_uint(v), j, lane));
}

// inclusive prefix sum over the wave
__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
  v += static_cast<int>(dpp_mov<kDppRowShr1>(static_cast<uint32_t>(v)));
  v += static_cast<int>(dpp_mov<kDppRowShr2>(static_cast<uint32_t>(v)));
  v += static_cast<int>(dpp_mov<kDppRowShr4>(static_cast<uint32_t>(v)));
  v += static_cast<int>(dpp_mov<kDppRowShr8>(static_cast<uint32_t>(v)));
  (void)lane;
  const int r0 = __builtin_amdgcn_readlane(v, 15);
  const int r1 = __builtin_amdgcn_readlane(v, 31);
  const int r2 = __builtin_amdgcn_readlane(v, 47);
  v += lane_in(kLanesGe16) ? r0 : 0;
  v += lane_in(kLanesBit5) ? r1 : 0;
  v += lane_in(kLanesGe48) ? r2 : 0;
  return v;
}

// maximum over each 16-lane row, valid in the row's last lane
__device__ __forceinline__ float fmax_sel(float a, float b) { return (b > a) ? b : a; }
__device__ __forceinline__ float fmin_sel(float a, float b) { return (b < a) ? b : a; }
__device__ __forceinline__ float row_max_last(float v) {
  const float ni = -__builtin_huge_valf();
  v = fmax_sel(v, dpp_movf<kDppRowShr1>(v, ni));
  v = fmax_sel(v, dpp_movf<kDppRowShr2>(v, ni));
  v = fmax_sel(v, dpp_movf<kDppRowShr4>(v, ni));
  v = fmax_sel(v, dpp_movf<kDppRowShr8>(v, ni));
  return v;
}

// lanes that keep the larger value in the bitonic step (k, j) of a sort of
// groups of N lanes, descending
constexpr uint64_t bitonic_max_lanes(int k, int j, int N) {
  uint64_t m = 0;
  for (int l = 0; l < 64; ++l) {
    const bool desc = (l & k) == 0 || k == N;
    const bool lower = (l & j) == 0;
    if (lower == desc) m |= 1ull << l;
  }
  return m;
}

// one compare-exchange step (k, j) of the bitonic sort of groups of N lanes
template <int N, int k, int j>
__device__ __forceinline__ float bitonic_step(float v, int lane) {
  const float o = xor_lane(v, j, lane);
  return ((o > v) == lane_in_here<bitonic_max_lanes(k, j, N)>()) ? o : v;
}
template <int N, int k, int j>
__device__ __forceinline__ float bitonic_merge(float v, int lane) {
  v = bitonic_step<N, k, j>(v, lane);
  if constexpr (j > 1) v = bitonic_merge<N, k, j / 2>(v, lane);
  return v;
}
template <int N, int k>
__device__ __forceinline__ float bitonic_levels(float v, int lane) {
  v = bitonic_merge<N, k, k / 2>(v, lane);
  if constexpr (k < N) v = bitonic_levels<N, k * 2>(v, lane);
  return v;
}

// Recombination probes at distances D = 1..DMAX: lane j against lane j-D of
// its 16-lane row.  Lanes shifted in from outside the row read all ones.
template <int D, int DMAX>
__device__ __forceinline__ bool recomb_shifts(uint32_t klo, uint32_t khi) {
  constexpr int kCtrl = 0x110 + D;  // row_shr:D
  const uint32_t ol = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(-1, static_cast<int>(klo), kCtrl, 0xF, 0xF, false));
  const uint32_t oh = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(-1, static_cast<int>(khi), kCtrl, 0xF, 0xF, false));
  bool m = ((static_cast<uint64_t>(oh) << 32) | ol) == ((static_cast<uint64_t>(khi) << 32) | klo);
  if constexpr (D < DMAX) m = m || recomb_shifts<D + 1, DMAX>(klo, khi);
  return m;
}

// Count, per lane, the values of its 16-lane row at least as large as its own
// (the lane itself included): 15 rotations, no dependent sort.
template <int D>
__device__ __forceinline__ uint32_t ge_count_step(float v, uint32_t n) {
  const float o = __uint_as_float(dpp_row_ror<D>(__float_as_uint(v)));
  return n + (o >= v ? 1u : 0u);
}
__device__ __forceinline__ uint32_t row_ge_count(float v) {
  uint32_t n = 1u;
  n = ge_count_step<1>(v, n);
  n = ge_count_step<2>(v, n);
  n = ge_count_step<3>(v, n);
  n = ge_count_step<4>(v, n);
  n = ge_count_step<5>(v, n);
  n = ge_count_step<6>(v, n);
  n = ge_count_step<7>(v, n);
  n = ge_count_step<8>(v, n);
  n = ge_count_step<9>(v, n);
  n = ge_count_step<10>(v, n);
  n = ge_count_step<11>(v, n);
  n = ge_count_step<12>(v, n);
  n = ge_count_step<13>(v, n);
  n = ge_count_step<14>(v, n);
  n = ge_count_step<15>(v, n);
  return n;
}

// Bitonic sort of one value per lane within groups of N lanes, descending.
template <int N>
__device__ __forceinline__ float wave_sort_desc(float v, int lane) {
  return bitonic_levels<N, 2>(v, lane);
}

}  // namespace detail
}  // namespace ctcbeam
