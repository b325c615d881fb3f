// Frontier and distance helpers shared by the resident and paged search
// kernels: uint8 vector lanes, exact squared-L2 partials, and the register
// frontier (sorted keys, insertion by rank, bitonic merge with dedupe).
#pragma once

#include "common.hpp"

namespace gorio {

// Lane layout for distance evaluation: 8 groups of 8 lanes; group g handles
// one vector per round, lane gl of the group holds dwords [gl*VDW, gl*VDW+VDW).
// EXACT: the vector is exactly 8 * VDW dwords (no per-dword bound checks, and
// 16-B loads when VDW is a multiple of 4; records are 4-B aligned).
template <int VDW, bool EXACT>
struct U8Vec {
  uint32_t w[VDW];

  __device__ __forceinline__ void load(const uint8_t *rec, int gl, uint32_t dwords) {
    const uint32_t *p = reinterpret_cast<const uint32_t *>(rec) + gl * VDW;
    if constexpr (EXACT && VDW % 4 == 0) {
#pragma unroll
      for (int t = 0; t < VDW; t += 4) {
        uint4 u;
        __builtin_memcpy(&u, __builtin_assume_aligned(p + t, 4), 16);
        w[t] = u.x; w[t + 1] = u.y; w[t + 2] = u.z; w[t + 3] = u.w;
      }
    } else if constexpr (EXACT) {
#pragma unroll
      for (int t = 0; t < VDW; ++t) w[t] = p[t];
    } else {
#pragma unroll
      for (int t = 0; t < VDW; ++t) w[t] = (uint32_t)(gl * VDW + t) < dwords ? p[t] : 0u;
    }
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int t = 0; t < VDW; ++t) w[t] = 0u;
  }
};

// Partial of sum (x.x - 2 q.x) over this lane's dwords (both dot products
// accumulate through v_dot4_u32_u8's addend; no overflow: VDW * 4 * 255^2 < 2^31).
template <int VDW, bool EXACT>
__device__ __forceinline__ int partial_u8(const U8Vec<VDW, EXACT> &q, const U8Vec<VDW, EXACT> &x) {
  uint32_t xx = 0, qx = 0;
#pragma unroll
  for (int t = 0; t < VDW; ++t) {
    xx = __builtin_amdgcn_udot4(x.w[t], x.w[t], xx, false);
    qx = __builtin_amdgcn_udot4(q.w[t], x.w[t], qx, false);
  }
  return (int)xx - 2 * (int)qx;
}

__device__ __forceinline__ uint32_t key_id(uint64_t key) { return (uint32_t)(key >> 1) & 0x7FFFFFFFu; }

// Key at frontier slot e (uniform e).
template <int KPL>
__device__ __forceinline__ uint64_t frontier_at(const uint64_t (&F)[KPL], uint32_t e) {
  uint64_t v = kInfKey;
#pragma unroll
  for (int r = 0; r < KPL; ++r)
    if ((uint32_t)r == e / kWave) v = readlane64(F[r], e % kWave);
  return v;
}

// Insert one key c (wave-uniform) by rank: slots at or above its rank move up
// by one, the last slot falls off.  A key whose node is already in F is
// dropped, so repeated evaluations never duplicate a frontier entry.
template <int KPL>
__device__ __forceinline__ void insert_key(uint64_t (&F)[KPL], uint64_t c) {
  uint32_t rank = 0;
  bool dup = false;
#pragma unroll
  for (int r = 0; r < KPL; ++r) {
    rank += (uint32_t)__popcll(ballot(F[r] < c));
    dup |= ballot(F[r] != kInfKey && (F[r] >> 1) == (c >> 1)) != 0;
  }
  if (dup || rank >= (uint32_t)(KPL * kWave)) return;
  uint64_t prev[KPL];
#pragma unroll
  for (int r = 0; r < KPL; ++r) {
    uint64_t fill = r == 0 ? kInfKey : readlane64(F[r == 0 ? 0 : r - 1], kWave - 1);
    prev[r] = wave_shr1_64(F[r], fill);
  }
  const uint32_t l = lane_id();
#pragma unroll
  for (int r = 0; r < KPL; ++r) {
    const uint32_t e = r * kWave + l;
    F[r] = e < rank ? F[r] : (e == rank ? c : prev[r]);
  }
}

// Slow path after the visited filter forgot a node: a candidate may repeat a
// frontier node or another candidate.  Merge without truncating (2P slots:
// F ascending then C descending is bitonic), drop all but the last copy of
// each node (the copy carrying the expanded bit sorts last), re-sort, keep P.
template <int KPL>
__device__ __forceinline__ void merge_dedupe(uint64_t (&F)[KPL], uint64_t c_desc) {
  uint64_t big[2 * KPL];
#pragma unroll
  for (int r = 0; r < KPL; ++r) {
    big[r] = F[r];
    big[KPL + r] = kInfKey;
  }
  big[2 * KPL - 1] = c_desc;
  bitonic_merge_up<2 * KPL>(big);
  uint64_t next[2 * KPL];
#pragma unroll
  for (int r = 0; r < 2 * KPL; ++r) {
    uint64_t fill = r + 1 < 2 * KPL ? readlane64(big[r + 1 < 2 * KPL ? r + 1 : r], 0) : kInfKey;
    next[r] = shfl_down1_64(big[r], fill);
  }
#pragma unroll
  for (int r = 0; r < 2 * KPL; ++r)
    if (big[r] != kInfKey && next[r] != kInfKey && (next[r] >> 1) == (big[r] >> 1)) big[r] = kInfKey;
  bitonic_sort<2 * KPL, false>(big);
#pragma unroll
  for (int r = 0; r < KPL; ++r) F[r] = big[r];
}


// Up to this many keys below the L-th frontier key are inserted one by one;
// more go through the sorting network (measured on the 1M uint8 index, 64-key
// chunks: 6, 12, 32 -> 0.848, 0.836, 0.846 ms per 10k-query launch).
constexpr uint32_t kInsertMax = 12;

// Sort-and-merge path for a one-register frontier, kept out of line: it is
// rare after the first iterations, and one copy keeps the kernel small.
static __device__ __noinline__ uint64_t sort_merge_1(uint64_t f, uint64_t key, bool forgot) {
  uint64_t F[1] = {f};
  uint64_t cc[1] = {key};
  bitonic_sort<1, true>(cc);
  if (!forgot) {
    F[0] = min64(F[0], cc[0]);
    bitonic_merge_up<1>(F);
  } else {
    merge_dedupe<1>(F, cc[0]);
  }
  return F[0];
}

// Merge one key per lane (kInfKey = none) into F: keys at or above F's L-th
// key cannot enter; a few survivors are inserted by rank, more are sorted
// and bitonic-merged (with dedupe once the visited filter has forgotten a
// node).  Slots past L are cleared.
template <int KPL>
__device__ __forceinline__ void merge_keys(uint64_t (&F)[KPL], uint64_t key, bool forgot, uint32_t L) {
  const uint64_t thr = frontier_at<KPL>(F, L - 1);
  const bool pass = key < thr;
  uint64_t pm = ballot(pass);
  if (pm == 0) return;
  if (!pass) key = kInfKey;
  if ((uint32_t)__popcll(pm) <= kInsertMax) {
    while (pm) {
      const int lane = __builtin_ctzll(pm);
      pm &= pm - 1;
      insert_key<KPL>(F, readlane64(key, lane));
    }
  } else if constexpr (KPL == 1) {
    F[0] = sort_merge_1(F[0], key, forgot);
  } else {
    uint64_t cc[1] = {key};
    bitonic_sort<1, true>(cc);
    if (!forgot) {
      // no node can repeat: the P smallest of F and C are min(F, C reversed)
      F[KPL - 1] = min64(F[KPL - 1], cc[0]);
      bitonic_merge_up<KPL>(F);
    } else {
      merge_dedupe<KPL>(F, cc[0]);
    }
  }
  const uint32_t l = lane_id();
#pragma unroll
  for (int r = 0; r < KPL; ++r)
    if ((uint32_t)(r * kWave + l) >= L) F[r] = kInfKey;
}

}  // namespace gorio
