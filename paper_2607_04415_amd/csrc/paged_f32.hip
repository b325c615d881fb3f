// Paged search kernels for float32 rows (same variant choice as the resident ones).
#include "launch.hpp"
#include "queue_launch.hpp"

namespace gorio {

hipError_t launch_paged_f32(const PagedParams &pp, int grid, hipStream_t s) {
  if (pp.D == 96) return detail::paged<MetricF32<24, true>>(pp, grid, s);
  return detail::paged<MetricF32<64, false>>(pp, grid, s);
}

hipError_t launch_rounds_f32(const PagedParams &pp, const RoundParams &rp, int grid, hipStream_t s) {
  if (pp.D == 96) return detail::rounds<MetricF32<24, true>>(pp, rp, grid, s);
  return detail::rounds<MetricF32<64, false>>(pp, rp, grid, s);
}

hipError_t launch_queue_f32(const PagedParams &pp, const RoundParams &rp, const RunQueue &qp, int grid,
                            hipStream_t s) {
  if (pp.D == 96) return detail::queue<MetricF32<24, true>>(pp, rp, qp, grid, s);
  return detail::queue<MetricF32<64, false>>(pp, rp, qp, grid, s);
}

}  // namespace gorio
