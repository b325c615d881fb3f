// Locality-aware node placement (host code): a node_to_slot permutation that
// puts graph neighbours in the same page.
//
// Graph pages are the unit of I/O (GORIO Sec. 3.1); which nodes share a page
// decides how many pages a search touches.  Disk-resident ANNS work that the
// paper builds on (DiskANN, Starling; Sec. 6) places neighbours together for
// this reason.  The rule here: visit nodes breadth-first from the entry
// (neighbours in adjacency order); when a visited node has no slot yet, give
// it the next slot, then fill the rest of its page with its own neighbours
// that have no slot yet, in adjacency order (near edges come first).  Nodes
// the walk never reaches follow in id order.  Deterministic; O(n R).
#include <cstdint>
#include <vector>

#include "../../include/gorio.h"

namespace gorio {
gorio_status fail(gorio_status st, const char *fmt, ...);  // gorio.hip: sets the thread's last error
}

extern "C" gorio_status gorio_locality_order(const uint32_t *graph, uint64_t n, uint32_t R, uint32_t entry,
                                             uint32_t records_per_page, uint32_t *node_to_slot) {
  using gorio::fail;
  if (!graph || !node_to_slot) return fail(GORIO_EINVAL, "graph and node_to_slot must be non-NULL");
  if (n == 0 || n >= (1ull << 31)) return fail(GORIO_EINVAL, "n=%llu outside [1, 2^31)", (unsigned long long)n);
  if (R == 0 || R > 256) return fail(GORIO_EINVAL, "R=%u outside [1, 256]", R);
  if (records_per_page == 0) return fail(GORIO_EINVAL, "records_per_page must be >= 1");
  if (entry >= n) return fail(GORIO_EINVAL, "entry %u >= n", entry);
  for (uint64_t i = 0; i < n * R; ++i)
    if (graph[i] != UINT32_MAX && graph[i] >= n)
      return fail(GORIO_EINVAL, "graph id %u at row %llu is >= n", graph[i], (unsigned long long)(i / R));

  const uint32_t kNone = UINT32_MAX;
  std::vector<uint32_t> slot(n, kNone);
  std::vector<uint8_t> seen(n, 0);
  std::vector<uint32_t> queue;
  queue.reserve(n);
  uint32_t next = 0;
  auto place = [&](uint32_t v) {
    slot[v] = next++;
  };
  auto place_with_neighbours = [&](uint32_t u) {
    place(u);
    const uint32_t *row = graph + (uint64_t)u * R;
    for (uint32_t j = 0; j < R && next % records_per_page != 0; ++j) {
      const uint32_t v = row[j];
      if (v != UINT32_MAX && slot[v] == kNone) place(v);
    }
  };
  queue.push_back(entry);
  seen[entry] = 1;
  for (size_t h = 0; h < queue.size(); ++h) {
    const uint32_t u = queue[h];
    if (slot[u] == kNone) place_with_neighbours(u);
    const uint32_t *row = graph + (uint64_t)u * R;
    for (uint32_t j = 0; j < R; ++j) {
      const uint32_t v = row[j];
      if (v != UINT32_MAX && !seen[v]) {
        seen[v] = 1;
        queue.push_back(v);
      }
    }
  }
  for (uint64_t v = 0; v < n; ++v)
    if (slot[v] == kNone) slot[v] = next++;
  for (uint64_t v = 0; v < n; ++v) node_to_slot[v] = slot[v];
  return GORIO_OK;
}
