// Cluster placement and query ordering for paged search (host entry points
// and their kernels).
//
// Pages are the unit of remote I/O (GORIO Sec. 3.1), so which nodes share a
// page, and which queries run at the same time, decide how often a fetched
// page is used again before the clock hand evicts it.  The disk-resident ANNS
// work the paper builds on studies page layout and graph locality (Sec. 6);
// the paper's future work asks for miss coalescing across queries (Sec. 7.2).
// Here: a few Lloyd iterations of k-means on the GPU give K centroids; nodes
// are placed cluster by cluster (node_to_slot), and a paged search admits its
// queries cluster by cluster, so the queries in flight at any time read a
// small set of clusters' pages, which the cache then holds.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <thread>
#include <vector>

#include "../../include/gorio.h"
#include "cluster.hpp"

namespace gorio {
gorio_status fail(gorio_status st, const char *fmt, ...);

// Nearest centroid of each vector: argmin_k (|c_k|^2 - 2 x . c_k), float32
// arithmetic, d in order, ties to the smaller k.  One thread per vector;
// every lane of a wave reads the same centroid element (a broadcast).  With
// the dimension known at compile time (DC > 0) the vector is held in
// registers and each centroid is read once per wave through scalar loads.
template <typename T, int DC>
__global__ __launch_bounds__(256) void nearest_centroid(const T *v, uint64_t count, uint32_t D, const float *c,
                                                        const float *cc, uint32_t K, uint32_t *out) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= count) return;
  const T *x = v + i * D;
  float best = 0.0f;
  uint32_t arg = 0;
  if constexpr (DC > 0) {
    float xr[DC];
#pragma unroll
    for (int d = 0; d < DC; ++d) xr[d] = (float)x[d];
    for (uint32_t k = 0; k < K; ++k) {
      const float *ck = c + (uint64_t)k * DC;
      float dot = 0.0f;
#pragma unroll
      for (int d = 0; d < DC; ++d) dot += xr[d] * ck[d];
      const float s = cc[k] - 2.0f * dot;
      if (k == 0 || s < best) {
        best = s;
        arg = k;
      }
    }
  } else {
    for (uint32_t k = 0; k < K; ++k) {
      const float *ck = c + (uint64_t)k * D;
      float dot = 0.0f;
      for (uint32_t d = 0; d < D; ++d) dot += (float)x[d] * ck[d];
      const float s = cc[k] - 2.0f * dot;
      if (k == 0 || s < best) {
        best = s;
        arg = k;
      }
    }
  }
  out[i] = arg;
}

template <typename T>
hipError_t launch_nearest_centroid_t(const T *v, uint64_t count, uint32_t D, const float *c, const float *cc,
                                     uint32_t K, uint32_t *out, hipStream_t s) {
  const int block = 256;
  const unsigned grid = (unsigned)((count + block - 1) / block);
  switch (D) {
    case 32: nearest_centroid<T, 32><<<grid, block, 0, s>>>(v, count, D, c, cc, K, out); break;
    case 64: nearest_centroid<T, 64><<<grid, block, 0, s>>>(v, count, D, c, cc, K, out); break;
    case 96: nearest_centroid<T, 96><<<grid, block, 0, s>>>(v, count, D, c, cc, K, out); break;
    case 128: nearest_centroid<T, 128><<<grid, block, 0, s>>>(v, count, D, c, cc, K, out); break;
    default: nearest_centroid<T, 0><<<grid, block, 0, s>>>(v, count, D, c, cc, K, out); break;
  }
  return hipGetLastError();
}

hipError_t launch_nearest_centroid(gorio_dtype dt, const void *v, uint64_t count, uint32_t D, const float *c,
                                   const float *cc, uint32_t K, uint32_t *out, hipStream_t s) {
  if (count == 0) return hipSuccess;
  if (dt == GORIO_U8)
    return launch_nearest_centroid_t(static_cast<const uint8_t *>(v), count, D, c, cc, K, out, s);
  return launch_nearest_centroid_t(static_cast<const float *>(v), count, D, c, cc, K, out, s);
}

void centroid_norms(const float *c, uint32_t K, uint32_t D, float *cc) {
  for (uint32_t k = 0; k < K; ++k) {
    float s = 0.0f;
    for (uint32_t d = 0; d < D; ++d) s += c[(uint64_t)k * D + d] * c[(uint64_t)k * D + d];
    cc[k] = s;
  }
}

void order_by_key(const uint32_t *key, uint64_t count, uint32_t K, uint32_t *order) {
  std::vector<uint64_t> start(K + 1, 0);
  for (uint64_t i = 0; i < count; ++i) ++start[key[i] + 1];
  for (uint32_t k = 0; k < K; ++k) start[k + 1] += start[k];
  for (uint64_t i = 0; i < count; ++i) order[start[key[i]]++] = (uint32_t)i;
}

}  // namespace gorio

using namespace gorio;

#define HIP_OR_FAIL(expr)                                                                  \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess)                                                                  \
      return fail(e_ == hipErrorOutOfMemory ? GORIO_ENOMEM : GORIO_EDEVICE, "%s: %s", #expr, \
                  hipGetErrorString(e_));                                                  \
  } while (0)

namespace {
struct Buf {
  void *p = nullptr;
  ~Buf() { if (p) (void)hipFree(p); }
  hipError_t alloc(size_t bytes) { return hipMalloc(&p, bytes ? bytes : 4); }
};
struct StreamGuard {
  hipStream_t s = nullptr;
  ~StreamGuard() { if (s) (void)hipStreamDestroy(s); }
};
}  // namespace

extern "C" gorio_status gorio_cluster_order(gorio_dtype dtype, const void *vectors, uint64_t n, uint32_t D,
                                            uint32_t clusters, uint32_t iterations, uint32_t *node_to_slot,
                                            float *centroids) {
  if (!vectors || !node_to_slot || !centroids) return fail(GORIO_EINVAL, "vectors, node_to_slot and centroids must be non-NULL");
  if (dtype != GORIO_U8 && dtype != GORIO_F32) return fail(GORIO_EINVAL, "unknown dtype %d", (int)dtype);
  if (n == 0 || n >= (1ull << 31)) return fail(GORIO_EINVAL, "n=%llu outside [1, 2^31)", (unsigned long long)n);
  if (D == 0 || D > 1024) return fail(GORIO_EINVAL, "D=%u outside [1, 1024]", D);
  if (clusters == 0 || clusters > kMaxClusters || clusters > n)
    return fail(GORIO_EINVAL, "clusters=%u outside [1, min(n, %u)]", clusters, kMaxClusters);
  if (iterations > 64) return fail(GORIO_EINVAL, "iterations=%u above 64", iterations);
  const uint32_t K = clusters;
  const size_t eb = dtype == GORIO_U8 ? 1 : 4;
  StreamGuard sg;
  HIP_OR_FAIL(hipStreamCreateWithFlags(&sg.s, hipStreamNonBlocking));
  Buf d_v, d_c, d_cc, d_key;
  HIP_OR_FAIL(d_v.alloc(n * D * eb));
  HIP_OR_FAIL(d_c.alloc((size_t)K * D * 4));
  HIP_OR_FAIL(d_cc.alloc((size_t)K * 4));
  HIP_OR_FAIL(d_key.alloc(n * 4));
  HIP_OR_FAIL(hipMemcpyAsync(d_v.p, vectors, n * D * eb, hipMemcpyHostToDevice, sg.s));

  // initial centroids: the vectors of nodes i * n / K (distinct ids)
  std::vector<float> c((size_t)K * D), cc(K);
  auto elem = [&](uint64_t i, uint32_t d) -> double {
    return dtype == GORIO_U8 ? (double)static_cast<const uint8_t *>(vectors)[i * D + d]
                             : (double)static_cast<const float *>(vectors)[i * D + d];
  };
  for (uint32_t k = 0; k < K; ++k) {
    const uint64_t i = (uint64_t)k * n / K;
    for (uint32_t d = 0; d < D; ++d) c[(size_t)k * D + d] = (float)elem(i, d);
  }
  std::vector<uint32_t> key(n);
  // Lloyd updates on the host: 16 threads sum fixed node ranges in float64,
  // then the partial sums are added in range order (the same result on any
  // machine)
  const uint32_t nt = 16;
  std::vector<std::vector<double>> sums(nt, std::vector<double>((size_t)K * D));
  std::vector<std::vector<uint64_t>> cnts(nt, std::vector<uint64_t>(K));
  auto accumulate = [&](uint32_t t) {
    std::vector<double> &sum = sums[t];
    std::vector<uint64_t> &cnt = cnts[t];
    std::fill(sum.begin(), sum.end(), 0.0);
    std::fill(cnt.begin(), cnt.end(), 0);
    const uint64_t i0 = n * t / nt, i1 = n * (t + 1) / nt;
    for (uint64_t i = i0; i < i1; ++i) {
      const uint32_t k = key[i];
      ++cnt[k];
      double *sk = sum.data() + (size_t)k * D;
      if (dtype == GORIO_U8) {
        const uint8_t *x = static_cast<const uint8_t *>(vectors) + i * D;
        for (uint32_t d = 0; d < D; ++d) sk[d] += x[d];
      } else {
        const float *x = static_cast<const float *>(vectors) + i * D;
        for (uint32_t d = 0; d < D; ++d) sk[d] += x[d];
      }
    }
  };
  for (uint32_t it = 0;; ++it) {
    centroid_norms(c.data(), K, D, cc.data());
    HIP_OR_FAIL(hipMemcpyAsync(d_c.p, c.data(), c.size() * 4, hipMemcpyHostToDevice, sg.s));
    HIP_OR_FAIL(hipMemcpyAsync(d_cc.p, cc.data(), cc.size() * 4, hipMemcpyHostToDevice, sg.s));
    HIP_OR_FAIL(launch_nearest_centroid(dtype, d_v.p, n, D, static_cast<float *>(d_c.p),
                                        static_cast<float *>(d_cc.p), K, static_cast<uint32_t *>(d_key.p), sg.s));
    HIP_OR_FAIL(hipMemcpyAsync(key.data(), d_key.p, n * 4, hipMemcpyDeviceToHost, sg.s));
    HIP_OR_FAIL(hipStreamSynchronize(sg.s));
    if (it == iterations) break;
    // each centroid becomes the mean of its members (an empty cluster keeps
    // its centroid)
    std::vector<std::thread> pool;
    for (uint32_t t = 1; t < nt; ++t) pool.emplace_back(accumulate, t);
    accumulate(0);
    for (auto &th : pool) th.join();
    for (uint32_t k = 0; k < K; ++k) {
      uint64_t cnt = 0;
      for (uint32_t t = 0; t < nt; ++t) cnt += cnts[t][k];
      if (!cnt) continue;
      for (uint32_t d = 0; d < D; ++d) {
        double sd = 0.0;
        for (uint32_t t = 0; t < nt; ++t) sd += sums[t][(size_t)k * D + d];
        c[(size_t)k * D + d] = (float)(sd / (double)cnt);
      }
    }
  }
  // cluster by cluster, id order inside a cluster
  std::vector<uint32_t> order(n);
  order_by_key(key.data(), n, K, order.data());
  for (uint64_t s = 0; s < n; ++s) node_to_slot[order[s]] = (uint32_t)s;
  memcpy(centroids, c.data(), c.size() * 4);
  return GORIO_OK;
}
