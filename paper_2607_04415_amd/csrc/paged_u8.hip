// Paged search kernels for uint8 rows (same variant choice as the resident ones).
#include "launch.hpp"
#include "queue_launch.hpp"

namespace gorio {

hipError_t launch_paged_u8(const PagedParams &pp, int grid, hipStream_t s) {
  if (pp.D == 128) return detail::paged<MetricU8<4, true>>(pp, grid, s);
  const uint32_t vdw = (pp.D / 4 + 7) / 8;
  if (vdw <= 1) return detail::paged<MetricU8<1, false>>(pp, grid, s);
  if (vdw <= 4) return detail::paged<MetricU8<4, false>>(pp, grid, s);
  return detail::paged<MetricU8<16, false>>(pp, grid, s);
}

hipError_t launch_rounds_u8(const PagedParams &pp, const RoundParams &rp, int grid, hipStream_t s) {
  if (pp.D == 128) return detail::rounds<MetricU8<4, true>>(pp, rp, grid, s);
  const uint32_t vdw = (pp.D / 4 + 7) / 8;
  if (vdw <= 1) return detail::rounds<MetricU8<1, false>>(pp, rp, grid, s);
  if (vdw <= 4) return detail::rounds<MetricU8<4, false>>(pp, rp, grid, s);
  return detail::rounds<MetricU8<16, false>>(pp, rp, grid, s);
}

hipError_t launch_queue_u8(const PagedParams &pp, const RoundParams &rp, const RunQueue &qp, int grid,
                           hipStream_t s) {
  if (pp.D == 128) return detail::queue<MetricU8<4, true>>(pp, rp, qp, grid, s);
  const uint32_t vdw = (pp.D / 4 + 7) / 8;
  if (vdw <= 1) return detail::queue<MetricU8<1, false>>(pp, rp, qp, grid, s);
  if (vdw <= 4) return detail::queue<MetricU8<4, false>>(pp, rp, qp, grid, s);
  return detail::queue<MetricU8<16, false>>(pp, rp, qp, grid, s);
}

}  // namespace gorio
