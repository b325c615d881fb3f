// Resident search kernels for uint8 rows.
#include "launch.hpp"

namespace gorio {

// 128-d rows get the exact 16-B-per-lane variant (candidates kept as
// 16-byte locators when the pages allow it); others the generic one with 1,
// 4 or 16 dwords per lane.
hipError_t launch_resident_u8(const ResidentParams &p, int grid, hipStream_t s) {
  if (p.D == 128) {
    if (p.geom.units16 != 0 && p.geom.node_to_slot == nullptr)
      return detail::resident<MetricU8<4, true, true>>(p, grid, s);
    return detail::resident<MetricU8<4, true>>(p, grid, s);
  }
  const uint32_t vdw = (p.D / 4 + 7) / 8;
  if (vdw <= 1) return detail::resident<MetricU8<1, false>>(p, grid, s);
  if (vdw <= 4) return detail::resident<MetricU8<4, false>>(p, grid, s);
  return detail::resident<MetricU8<16, false>>(p, grid, s);
}

}  // namespace gorio
