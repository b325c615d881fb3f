// Wave64 building blocks for gfx950 (CDNA4): lane masks, prefix counts, DPP
// reductions and 64-bit bitonic compare-exchange.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gorio {

constexpr int kWave = 64;
constexpr uint64_t kInfKey = ~0ull;

__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

__device__ __forceinline__ uint64_t ballot(bool p) { return (uint64_t)__ballot(p); }

// Number of set bits of `mask` in lanes below this one.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint32_t readlane(uint32_t v, int lane) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int lane) {
  uint32_t lo = readlane((uint32_t)v, lane);
  uint32_t hi = readlane((uint32_t)(v >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint32_t first_lane_value(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}

// Cross-lane exchange with lane ^ m (ds_bpermute through the LDS crossbar).
__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int m) {
  int src = (lane_id() ^ m) << 2;
  uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)(uint32_t)v);
  uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)(uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Value of lane - 1 (lane 0 gets `fill`).
__device__ __forceinline__ uint64_t shfl_up1_64(uint64_t v, uint64_t fill) {
  int l = lane_id();
  int src = ((l + 63) & 63) << 2;
  uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)(uint32_t)v);
  uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)(uint32_t)(v >> 32));
  uint64_t r = ((uint64_t)hi << 32) | lo;
  return l == 0 ? fill : r;
}

// Value of lane + 1 (lane 63 gets `fill`).
__device__ __forceinline__ uint64_t shfl_down1_64(uint64_t v, uint64_t fill) {
  int l = lane_id();
  int src = ((l + 1) & 63) << 2;
  uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)(uint32_t)v);
  uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)(uint32_t)(v >> 32));
  uint64_t r = ((uint64_t)hi << 32) | lo;
  return l == kWave - 1 ? fill : r;
}

// Sum over each aligned group of 8 lanes; every lane of the group gets the total.
// quad_perm [1,0,3,2] (0xB1), quad_perm [2,3,0,1] (0x4E), row_half_mirror (0x141).
__device__ __forceinline__ int sum8(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
  return v;
}

// Eight rounds of per-group partials reduced at once: v[j] is this lane's
// partial of round j; every group of 8 lanes sums each round, and lane gl of
// the group receives round gl's total.  Three butterfly stages; at each, a
// lane keeps the half of its rounds whose index bit matches its own lane bit
// and adds the partner's other half (partner = the lane with that bit
// flipped: row_half_mirror for bit 2, quad_perm for bits 1 and 0).  21
// instructions for 8 totals instead of 8 sum8 calls and 8 selects.
__device__ __forceinline__ int transpose_sum8(const int (&v)[8]) {
  const int gl = lane_id() & 7;
  const bool b2 = gl & 4, b1 = gl & 2, b0 = gl & 1;
  int w[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int keep = b2 ? v[j + 4] : v[j], send = b2 ? v[j] : v[j + 4];
    w[j] = keep + __builtin_amdgcn_update_dpp(0, send, 0x141, 0xF, 0xF, false);
  }
  int u[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int keep = b1 ? w[j + 2] : w[j], send = b1 ? w[j] : w[j + 2];
    u[j] = keep + __builtin_amdgcn_update_dpp(0, send, 0x4E, 0xF, 0xF, false);
  }
  const int keep = b0 ? u[1] : u[0], send = b0 ? u[0] : u[1];
  return keep + __builtin_amdgcn_update_dpp(0, send, 0xB1, 0xF, 0xF, false);
}

// Sum over the whole wave, result in every lane (used off the hot path).
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  for (int m = 1; m < kWave; m <<= 1) v += shfl_xor64(v, m);
  return v;
}

__device__ __forceinline__ uint64_t min64(uint64_t a, uint64_t b) { return a < b ? a : b; }
__device__ __forceinline__ uint64_t max64(uint64_t a, uint64_t b) { return a < b ? b : a; }

// ---------------------------------------------------------------------------
// Bitonic networks over P = 64 * KPL keys held as v[r] at element r*64 + lane.
// ---------------------------------------------------------------------------

// Value of lane ^ M for M <= 8 by DPP (quad_perm, half-row mirror, row
// rotate), without the LDS crossbar.  Every lane's source exists, so the
// moves need no old value.  (Distances 16 and 32 use v_permlane16/32_swap in
// exchange_lanes.)
template <int M>
__device__ __forceinline__ uint32_t xor_lanes(uint32_t v) {
  const int iv = (int)v;
  if constexpr (M == 1) {
    return (uint32_t)__builtin_amdgcn_mov_dpp(iv, 0xB1, 0xF, 0xF, false);  // quad_perm [1,0,3,2]
  } else if constexpr (M == 2) {
    return (uint32_t)__builtin_amdgcn_mov_dpp(iv, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
  } else if constexpr (M == 4) {
    int t = __builtin_amdgcn_mov_dpp(iv, 0x141, 0xF, 0xF, false);          // i -> 7 - i in 8
    return (uint32_t)__builtin_amdgcn_mov_dpp(t, 0x1B, 0xF, 0xF, false);   // reverse each quad
  } else {
    static_assert(M == 8, "lane distance");
    return (uint32_t)__builtin_amdgcn_mov_dpp(iv, 0x128, 0xF, 0xF, false); // row_ror:8
  }
}

template <int M>
__device__ __forceinline__ uint64_t xor_lanes64(uint64_t v) {
  uint32_t lo = xor_lanes<M>((uint32_t)v);
  uint32_t hi = xor_lanes<M>((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Value of lane - 1 for a whole wave (DPP wave_shr:1); lane 0 gets `fill`.
__device__ __forceinline__ uint64_t wave_shr1_64(uint64_t v, uint64_t fill) {
  uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)fill, (int)(uint32_t)v, 0x138, 0xF, 0xF, false);
  uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)(fill >> 32), (int)(uint32_t)(v >> 32), 0x138,
                                                      0xF, 0xF, false);
  return ((uint64_t)hi << 32) | lo;
}

// Lanes (bit l of register r's mask) that keep the smaller key of their pair
// at the stage with partner distance J inside blocks of K: element
// e = r * 64 + l sorts upward when ((e & K) == 0) != DESC and is the lower of
// its pair when (e & J) == 0.
template <int KPL>
struct LaneMasks {
  uint64_t m[KPL];
};
template <int KPL, int J, int K, bool DESC>
__host__ __device__ constexpr LaneMasks<KPL> keep_min_lanes() {
  LaneMasks<KPL> x{};
  for (int r = 0; r < KPL; ++r) {
    uint64_t m = 0;
    for (int l = 0; l < kWave; ++l) {
      const int e = r * kWave + l;
      if ((((e & K) == 0) != DESC) == ((e & J) == 0)) m |= 1ull << l;
    }
    x.m[r] = m;
  }
  return x;
}

// m ^ (HI:LO) by two scalar XORs with literal operands.  Written as
// instructions so that the constants are not hoisted out of loops into
// registers (which then spill to VGPR lanes).
template <uint32_t LO, uint32_t HI>
__device__ __forceinline__ uint64_t xor_mask(uint64_t m) {
  uint32_t lo = (uint32_t)m, hi = (uint32_t)(m >> 32);
  if constexpr (LO != 0) asm volatile("s_xor_b32 %0, %0, %1" : "+s"(lo) : "i"(LO));
  if constexpr (HI != 0) asm volatile("s_xor_b32 %0, %0, %1" : "+s"(hi) : "i"(HI));
  return ((uint64_t)hi << 32) | lo;
}

// One compare-exchange of a lane pair at distance J < 64.  Each lane sees
// both keys of its pair, (a, b) = (lower lane's, upper lane's), and takes b
// when (b < a) equals its keep-min bit (KEEP_MIN), else a: one 64-bit
// compare whose lane mask is XORed with the constant, then two selects.
template <int J, uint64_t KEEP_MIN>
__device__ __forceinline__ uint64_t exchange_lanes(uint64_t v) {
  constexpr uint64_t kFlip = ~KEEP_MIN;  // take b where lt ^ flip is set
  if constexpr (J >= 16) {
    // permlane swap: the first result holds the pair's lower element in every
    // lane, the second its upper element
    const int vl = (int)(uint32_t)v, vh = (int)(uint32_t)(v >> 32);
    const auto lo = J == 16 ? __builtin_amdgcn_permlane16_swap(vl, vl, false, false)
                            : __builtin_amdgcn_permlane32_swap(vl, vl, false, false);
    const auto hi = J == 16 ? __builtin_amdgcn_permlane16_swap(vh, vh, false, false)
                            : __builtin_amdgcn_permlane32_swap(vh, vh, false, false);
    const uint64_t a = ((uint64_t)(uint32_t)hi[0] << 32) | (uint32_t)lo[0];
    const uint64_t b = ((uint64_t)(uint32_t)hi[1] << 32) | (uint32_t)lo[1];
    const uint64_t t = xor_mask<(uint32_t)kFlip, (uint32_t)(kFlip >> 32)>(ballot(b < a));
    return __builtin_amdgcn_inverse_ballot_w64(t) ? b : a;
  } else {
    // the partner's value o stands in for the other element: the lower lane
    // sees (v, o), the upper (o, v), and "take o" covers both
    const uint64_t o = xor_lanes64<J>(v);
    const uint64_t t = xor_mask<(uint32_t)kFlip, (uint32_t)(kFlip >> 32)>(ballot(o < v));
    return __builtin_amdgcn_inverse_ballot_w64(t) ? o : v;
  }
}

template <int KPL, int J, int K, bool DESC, int R>
__device__ __forceinline__ void exchange_registers_from(uint64_t (&v)[KPL]) {
  v[R] = exchange_lanes<J, keep_min_lanes<KPL, J, K, DESC>().m[R]>(v[R]);
  if constexpr (R + 1 < KPL) exchange_registers_from<KPL, J, K, DESC, R + 1>(v);
}

// One stage with partner distance J of the network over blocks of K.
template <int KPL, int J, int K, bool DESC>
__device__ __forceinline__ void bitonic_stage(uint64_t (&v)[KPL]) {
  if constexpr (J >= kWave) {
    constexpr LaneMasks<KPL> km = keep_min_lanes<KPL, J, K, DESC>();
    constexpr int rj = J / kWave;
#pragma unroll
    for (int r = 0; r < KPL; ++r) {
      if (r & rj) continue;
      // both elements sort the same way (the block direction is uniform per register)
      const bool up = (km.m[r] & 1ull) != 0;
      const uint64_t a = v[r], b = v[r | rj];
      const bool lt = b < a;
      v[r] = (lt == up) ? b : a;
      v[r | rj] = (lt == up) ? a : b;
    }
  } else {
    exchange_registers_from<KPL, J, K, DESC, 0>(v);
  }
}

template <int KPL, int J, int K, bool DESC>
__device__ __forceinline__ void bitonic_stages(uint64_t (&v)[KPL]) {
  bitonic_stage<KPL, J, K, DESC>(v);
  if constexpr (J > 1) bitonic_stages<KPL, J / 2, K, DESC>(v);
}

template <int KPL, int K, bool DESC>
__device__ __forceinline__ void bitonic_sort_from(uint64_t (&v)[KPL]) {
  bitonic_stages<KPL, K / 2, K, DESC>(v);
  if constexpr (K < KPL * kWave) bitonic_sort_from<KPL, 2 * K, DESC>(v);
}

// Full sort of P = 64 * KPL keys held as v[r] at element r * 64 + lane
// (ascending unless DESC).
template <int KPL, bool DESC>
__device__ __forceinline__ void bitonic_sort(uint64_t (&v)[KPL]) {
  bitonic_sort_from<KPL, 2, DESC>(v);
}

// Sorts a bitonic sequence of P keys ascending.
template <int KPL>
__device__ __forceinline__ void bitonic_merge_up(uint64_t (&v)[KPL]) {
  bitonic_stages<KPL, KPL * kWave / 2, 2 * KPL * kWave, false>(v);
}

}  // namespace gorio
