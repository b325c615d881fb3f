// Resident search kernels for float32 rows.
#include "launch.hpp"

namespace gorio {

// 96-d rows get the exact variant (24 16-B loads per lane at once); others
// the generic dword loop (D <= 256).
hipError_t launch_resident_f32(const ResidentParams &p, int grid, hipStream_t s) {
  if (p.D == 96) return detail::resident<MetricF32<24, true>>(p, grid, s);
  return detail::resident<MetricF32<64, false>>(p, grid, s);
}

}  // namespace gorio
