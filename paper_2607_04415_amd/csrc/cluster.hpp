// Nearest-centroid assignment shared by the cluster placement helper and the
// paged search's query ordering (cluster.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/gorio.h"

namespace gorio {

constexpr uint32_t kMaxClusters = 65536;

// out[i] = nearest of the K centroids c (K x D float32, cc[k] = |c_k|^2) to
// vector i of v (count x D, uint8 or float32); device pointers, async on s.
hipError_t launch_nearest_centroid(gorio_dtype dt, const void *v, uint64_t count, uint32_t D, const float *c,
                                   const float *cc, uint32_t K, uint32_t *out, hipStream_t s);

// cc[k] = |c_k|^2 (host).
void centroid_norms(const float *c, uint32_t K, uint32_t D, float *cc);

// Stable counting sort of [0, count) by key (< K): order[j] = j-th index.
void order_by_key(const uint32_t *key, uint64_t count, uint32_t K, uint32_t *order);

}  // namespace gorio
