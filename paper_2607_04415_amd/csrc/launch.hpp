// Kernel launchers.  Each dtype's kernel variants are instantiated in a
// translation unit of their own (resident_u8.hip, resident_f32.hip,
// paged_u8.hip, paged_f32.hip) so that they compile in parallel.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>

#include "search_paged.hpp"
#include "search_resident.hpp"

namespace gorio {

// Resident search: one wave per query at a time, at most `grid` workgroups
// (queries past the grid are handed out by the kernel's counter).
hipError_t launch_resident_u8(const ResidentParams &p, int grid, hipStream_t s);
hipError_t launch_resident_f32(const ResidentParams &p, int grid, hipStream_t s);

// Paged search: the persistent kernel (fill waves + query waves).  With
// grid == pp.fill_waves it runs only the fill waves.
hipError_t launch_paged_u8(const PagedParams &pp, int grid, hipStream_t s);
hipError_t launch_paged_f32(const PagedParams &pp, int grid, hipStream_t s);

// Host-scheduled lanes: one workgroup per listed lane, or (no list) the
// persistent launch of fill waves, the run ring's tail mirror and executors.
hipError_t launch_rounds_u8(const PagedParams &pp, const RoundParams &rp, int grid, hipStream_t s);
hipError_t launch_rounds_f32(const PagedParams &pp, const RoundParams &rp, int grid, hipStream_t s);

// 32-bit words of one lane's saved state for a search with frontier size L.
inline uint32_t lane_state_words(uint32_t L) {
  const size_t b = L <= 64 ? sizeof(QSlot<1>) : L <= 128 ? sizeof(QSlot<2>) : sizeof(QSlot<4>);
  return (uint32_t)((b + 3) / 4);
}

// Visited tables of the resident kernel: 16-bit entries (2^M::kHtLog2 of
// them) when every id fits that table's domain, else 8192 32-bit entries.
using ResidentHtLarge = VisitedLds<13>;

namespace detail {

// One workgroup per wave slot the device holds at once, but at most
// `grid_waves_per_simd` per SIMD (queries beyond the grid are taken from the
// kernel's counter), and at most `grid`.
template <auto Kernel, int grid_waves_per_simd>
hipError_t launch_resident_grid(const ResidentParams &p, int grid, hipStream_t s) {
  static int slots = 0;  // per kernel
  if (slots == 0) {
    constexpr int kSimdsPerCu = 4;
    int dev = 0, cus = 0, per_cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(Kernel), kWave, 0);
    if (e != hipSuccess) return e;
    slots = std::max(1, cus * std::min(per_cu, kSimdsPerCu * grid_waves_per_simd));
  }
  Kernel<<<std::min(grid, slots), kWave, 0, s>>>(p);
  return hipGetLastError();
}

template <int KPL, class M, bool N2S>
hipError_t resident_t(const ResidentParams &p, int grid, hipStream_t s) {
  using Small = VisitedLds16<M::kHtLog2>;
  constexpr int kGrid = M::kGridWavesPerSimd;
  if (p.n <= Small::kMaxId) return launch_resident_grid<search_resident<KPL, M, Small, N2S>, kGrid>(p, grid, s);
  return launch_resident_grid<search_resident<KPL, M, ResidentHtLarge, N2S>, kGrid>(p, grid, s);
}

// frontier slots per lane (L <= 64 KPL) and node_to_slot presence
template <class M>
hipError_t resident(const ResidentParams &p, int grid, hipStream_t s) {
  if constexpr (M::kLocators) {  // identity placement only
    if (p.L <= 64) return resident_t<1, M, false>(p, grid, s);
    if (p.L <= 128) return resident_t<2, M, false>(p, grid, s);
    return resident_t<4, M, false>(p, grid, s);
  } else {
    const bool n2s = p.geom.node_to_slot != nullptr;
    if (p.L <= 64) return n2s ? resident_t<1, M, true>(p, grid, s) : resident_t<1, M, false>(p, grid, s);
    if (p.L <= 128) return n2s ? resident_t<2, M, true>(p, grid, s) : resident_t<2, M, false>(p, grid, s);
    return n2s ? resident_t<4, M, true>(p, grid, s) : resident_t<4, M, false>(p, grid, s);
  }
}

template <int KPL, class M, bool N2S>
hipError_t paged_t(const PagedParams &pp, int grid, hipStream_t s) {
  const size_t lds = pp.oversub * sizeof(QSlot<KPL>);
  auto k = search_paged<KPL, M, N2S>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(k),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  k<<<grid, kWave, lds, s>>>(pp);
  return hipGetLastError();
}

template <class M>
hipError_t paged(const PagedParams &pp, int grid, hipStream_t s) {
  const bool n2s = pp.geom.node_to_slot != nullptr;
  if (pp.L <= 64) return n2s ? paged_t<1, M, true>(pp, grid, s) : paged_t<1, M, false>(pp, grid, s);
  if (pp.L <= 128) return n2s ? paged_t<2, M, true>(pp, grid, s) : paged_t<2, M, false>(pp, grid, s);
  return n2s ? paged_t<4, M, true>(pp, grid, s) : paged_t<4, M, false>(pp, grid, s);
}

template <int KPL, class M, bool N2S>
hipError_t rounds_t(const PagedParams &pp, const RoundParams &rp, int grid, hipStream_t s) {
  paged_round<KPL, M, N2S><<<grid, kWave, sizeof(QSlot<KPL>), s>>>(pp, rp);
  return hipGetLastError();
}

template <class M>
hipError_t rounds(const PagedParams &pp, const RoundParams &rp, int grid, hipStream_t s) {
  const bool n2s = pp.geom.node_to_slot != nullptr;
  if (pp.L <= 64) return n2s ? rounds_t<1, M, true>(pp, rp, grid, s) : rounds_t<1, M, false>(pp, rp, grid, s);
  if (pp.L <= 128) return n2s ? rounds_t<2, M, true>(pp, rp, grid, s) : rounds_t<2, M, false>(pp, rp, grid, s);
  return n2s ? rounds_t<4, M, true>(pp, rp, grid, s) : rounds_t<4, M, false>(pp, rp, grid, s);
}

}  // namespace detail
}  // namespace gorio
