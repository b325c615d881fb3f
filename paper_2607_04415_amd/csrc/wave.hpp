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

// Value of lane ^ M, M a power of two below 64, without the LDS crossbar:
// DPP for M <= 8 (quad_perm, half-row mirror, row rotate), the gfx950
// v_permlane16/32_swap for 16 and 32.
template <int M>
__device__ __forceinline__ uint32_t xor_lanes(uint32_t v) {
  const int iv = (int)v;
  if constexpr (M == 1) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, iv, 0xB1, 0xF, 0xF, false);  // quad_perm [1,0,3,2]
  } else if constexpr (M == 2) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, iv, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
  } else if constexpr (M == 4) {
    int t = __builtin_amdgcn_update_dpp(0, iv, 0x141, 0xF, 0xF, false);          // i -> 7 - i in 8
    return (uint32_t)__builtin_amdgcn_update_dpp(0, t, 0x1B, 0xF, 0xF, false);   // reverse each quad
  } else if constexpr (M == 8) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, iv, 0x128, 0xF, 0xF, false); // row_ror:8
  } else if constexpr (M == 16) {
    auto r = __builtin_amdgcn_permlane16_swap(iv, iv, false, false);
    return (uint32_t)(((lane_id() >> 4) & 1) ? r[0] : r[1]);
  } else {
    static_assert(M == 32, "lane distance");
    auto r = __builtin_amdgcn_permlane32_swap(iv, iv, false, false);
    return (uint32_t)(lane_id() >= 32 ? r[0] : r[1]);
  }
}

template <int M>
__device__ __forceinline__ uint64_t xor_lanes64(uint64_t v) {
  uint32_t lo = xor_lanes<M>((uint32_t)v);
  uint32_t hi = xor_lanes<M>((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t xor_lanes64_rt(uint64_t v, int m) {
  switch (m) {
    case 1: return xor_lanes64<1>(v);
    case 2: return xor_lanes64<2>(v);
    case 4: return xor_lanes64<4>(v);
    case 8: return xor_lanes64<8>(v);
    case 16: return xor_lanes64<16>(v);
    default: return xor_lanes64<32>(v);
  }
}

// Value of lane - 1 for a whole wave (DPP wave_shr:1); lane 0 gets `fill`.
__device__ __forceinline__ uint64_t wave_shr1_64(uint64_t v, uint64_t fill) {
  uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)fill, (int)(uint32_t)v, 0x138, 0xF, 0xF, false);
  uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)(fill >> 32), (int)(uint32_t)(v >> 32), 0x138,
                                                      0xF, 0xF, false);
  return ((uint64_t)hi << 32) | lo;
}

// One compare-exchange stage with partner distance j.  Element e keeps the
// smaller key when (e is the lower of the pair) == (its block sorts upward).
// j and k are compile-time constants after unrolling.
template <int KPL>
__device__ __forceinline__ void bitonic_stage(uint64_t (&v)[KPL], int j, int k, bool descending) {
  const int l = lane_id();
  if (j >= kWave) {
    const int rj = j / kWave;
#pragma unroll
    for (int r = 0; r < KPL; ++r) {
      if (r & rj) continue;
      const int e = r * kWave + l;
      bool up = ((e & k) == 0) != descending;
      uint64_t a = v[r], b = v[r | rj];
      v[r] = up ? min64(a, b) : max64(a, b);
      v[r | rj] = up ? max64(a, b) : min64(a, b);
    }
  } else {
#pragma unroll
    for (int r = 0; r < KPL; ++r) {
      const int e = r * kWave + l;
      bool up = ((e & k) == 0) != descending;
      bool lower = (l & j) == 0;
      uint64_t o = xor_lanes64_rt(v[r], j);
      v[r] = (lower == up) ? min64(v[r], o) : max64(v[r], o);
    }
  }
}

// Full sort of P keys (ascending unless `descending`).
template <int KPL>
__device__ __forceinline__ void bitonic_sort(uint64_t (&v)[KPL], bool descending) {
  constexpr int P = KPL * kWave;
#pragma unroll
  for (int k = 2; k <= P; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) bitonic_stage<KPL>(v, j, k, descending);
  }
}

// Sorts a bitonic sequence of P keys ascending.
template <int KPL>
__device__ __forceinline__ void bitonic_merge_up(uint64_t (&v)[KPL]) {
  constexpr int P = KPL * kWave;
#pragma unroll
  for (int j = P >> 1; j > 0; j >>= 1) bitonic_stage<KPL>(v, j, 2 * P, false);
}

}  // namespace gorio
