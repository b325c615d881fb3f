// Launchers of the GPU resume-queue search (paged_queue in search_paged.hpp):
// fill waves, then executor waves, one persistent launch per search.  Each
// dtype instantiates them in its paged translation unit.
#pragma once

#include <hip/hip_runtime.h>

#include "search_paged.hpp"

namespace gorio {

hipError_t launch_queue_u8(const PagedParams &pp, const RoundParams &rp, const RunQueue &qp, int grid,
                           hipStream_t s);
hipError_t launch_queue_f32(const PagedParams &pp, const RoundParams &rp, const RunQueue &qp, int grid,
                            hipStream_t s);

namespace detail {

template <int KPL, class M, bool N2S>
hipError_t queue_t(const PagedParams &pp, const RoundParams &rp, const RunQueue &qp, int grid, hipStream_t s) {
  paged_queue<KPL, M, N2S><<<grid, kWave, sizeof(QSlot<KPL>), s>>>(pp, rp, qp);
  return hipGetLastError();
}

template <class M>
hipError_t queue(const PagedParams &pp, const RoundParams &rp, const RunQueue &qp, int grid, hipStream_t s) {
  const bool n2s = pp.geom.node_to_slot != nullptr;
  if (pp.L <= 64) return n2s ? queue_t<1, M, true>(pp, rp, qp, grid, s) : queue_t<1, M, false>(pp, rp, qp, grid, s);
  if (pp.L <= 128) return n2s ? queue_t<2, M, true>(pp, rp, qp, grid, s) : queue_t<2, M, false>(pp, rp, qp, grid, s);
  return n2s ? queue_t<4, M, true>(pp, rp, qp, grid, s) : queue_t<4, M, false>(pp, rp, qp, grid, s);
}

}  // namespace detail
}  // namespace gorio
