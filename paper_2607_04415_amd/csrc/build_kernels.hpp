// Index construction on the GPU: page packing, layout checks and the medoid
// entry rule.
#pragma once

#include "common.hpp"

namespace gorio {

// Byte fill (the packed page array starts zeroed: page tails are zero).
__global__ void fill_u32(uint32_t *dst, uint64_t words, uint32_t value) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words;
       i += (uint64_t)gridDim.x * blockDim.x)
    dst[i] = value;
}

// node_to_slot must be a permutation of [0, n): count out-of-range or repeated slots.
__global__ void check_permutation(const uint32_t *node_to_slot, uint32_t n, uint32_t *seen_bits,
                                  unsigned int *bad) {
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    uint32_t s = node_to_slot[i];
    if (s >= n) { atomicAdd(bad, 1u); continue; }
    uint32_t bit = 1u << (s & 31);
    uint32_t old = atomicOr(&seen_bits[s >> 5], bit);
    if (old & bit) atomicAdd(bad, 1u);
  }
}

// One wave per node: copy the vector, compact the real edges (UINT32_MAX =
// no edge) in order, pad with UINT32_MAX, store the degree.  Ids >= n that
// are not UINT32_MAX are counted in *bad.
__global__ __launch_bounds__(256) void pack_records(const uint8_t *vectors, uint32_t vec_bytes,
                                                    const uint32_t *graph, uint32_t R, uint32_t n,
                                                    PageGeom geom, uint8_t *pages, unsigned int *bad) {
  const int l = lane_id();
  const uint32_t waves = gridDim.x * (blockDim.x / kWave);
  for (uint32_t v = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave; v < n; v += waves) {
    const uint32_t s = slot_of(geom, v);
    const uint32_t *src = reinterpret_cast<const uint32_t *>(vectors + (uint64_t)v * vec_bytes);
    uint32_t *dst = reinterpret_cast<uint32_t *>(pages + vec_offset(geom, s));
    for (uint32_t w = l; w < vec_bytes / 4; w += kWave) dst[w] = src[w];
    uint8_t *adj = pages + adj_offset(geom, s);
    uint32_t *ids = reinterpret_cast<uint32_t *>(adj + 4);
    uint32_t deg = 0;
    for (uint32_t j0 = 0; j0 < R; j0 += kWave) {
      uint32_t j = j0 + l;
      uint32_t id = j < R ? graph[(uint64_t)v * R + j] : kNoEdge;
      bool real = id != kNoEdge;
      if (real && id >= n) atomicAdd(bad, 1u);
      uint64_t m = ballot(real);
      if (real) ids[deg + lanes_below(m)] = id;
      deg += (uint32_t)__popcll(m);
    }
    for (uint32_t j = deg + l; j < R; j += kWave) ids[j] = kNoEdge;
    if (l == 0) *reinterpret_cast<uint32_t *>(adj) = deg;
  }
}

// ---- medoid -----------------------------------------------------------------
// uint8: exact column sums (any order gives the same integers).
__global__ __launch_bounds__(256) void column_sums_u8(const uint8_t *x, uint32_t n, uint32_t D,
                                                      uint32_t rows_per_block,
                                                      unsigned long long *sums) {
  const uint32_t r0 = blockIdx.x * rows_per_block;
  const uint32_t r1 = min(n, r0 + rows_per_block);
  for (uint32_t d = threadIdx.x; d < D; d += blockDim.x) {
    unsigned long long s = 0;
    for (uint32_t i = r0; i < r1; ++i) s += x[(uint64_t)i * D + d];
    atomicAdd(&sums[d], s);
  }
}

// float32: one thread per dimension sums in node order in float64.
__global__ void column_sums_f32_ordered(const float *x, uint32_t n, uint32_t D, double *sums) {
  const uint32_t d = blockIdx.x * blockDim.x + threadIdx.x;
  if (d >= D) return;
  double s = 0.0;
  uint32_t i = 0;
  for (; i + 8 <= n; i += 8) {
    float v[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) v[t] = x[(uint64_t)(i + t) * D + d];
#pragma unroll
    for (int t = 0; t < 8; ++t) s = __dadd_rn(s, (double)v[t]);
  }
  for (; i < n; ++i) s = __dadd_rn(s, (double)x[(uint64_t)i * D + d]);
  sums[d] = s;
}

// key = (distance bits << 32) | id, minimised with one atomic per block.
__device__ __forceinline__ void block_min_key(uint64_t key, unsigned long long *best) {
  __shared__ uint64_t part[256 / kWave];
  for (int m = 1; m < kWave; m <<= 1) key = min64(key, shfl_xor64(key, m));
  if (lane_id() == 0) part[threadIdx.x / kWave] = key;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t b = part[0];
    for (uint32_t w = 1; w < blockDim.x / kWave; ++w) b = min64(b, part[w]);
    atomicMin(best, (unsigned long long)b);
  }
}

__global__ __launch_bounds__(256) void nearest_to_centroid_u8(const uint8_t *x, uint32_t n, uint32_t D,
                                                              const unsigned long long *sums,
                                                              unsigned long long *best) {
  __shared__ uint8_t c[512];
  for (uint32_t d = threadIdx.x; d < D; d += blockDim.x)
    c[d] = (uint8_t)((sums[d] + n / 2) / n);
  __syncthreads();
  uint64_t key = kInfKey;
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    uint32_t s = 0;
    for (uint32_t d = 0; d < D; ++d) {
      int t = (int)c[d] - (int)x[(uint64_t)i * D + d];
      s += (uint32_t)(t * t);
    }
    key = min64(key, ((uint64_t)s << 32) | i);
  }
  block_min_key(key, best);
}

__global__ __launch_bounds__(256) void nearest_to_centroid_f32(const float *x, uint32_t n, uint32_t D,
                                                               const double *sums,
                                                               unsigned long long *best) {
  __shared__ float c[256];
  for (uint32_t d = threadIdx.x; d < D; d += blockDim.x) c[d] = (float)(sums[d] / (double)n);
  __syncthreads();
  uint64_t key = kInfKey;
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    float acc = 0.0f;
    for (uint32_t d = 0; d < D; ++d) {
      float t = __fsub_rn(c[d], x[(uint64_t)i * D + d]);
      acc = __fadd_rn(acc, __fmul_rn(t, t));
    }
    key = min64(key, ((uint64_t)__float_as_uint(acc) << 32) | i);
  }
  block_min_key(key, best);
}

}  // namespace gorio
