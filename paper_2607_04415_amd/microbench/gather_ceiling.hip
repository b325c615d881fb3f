// Practical ceiling of the resident search's dominant traffic: random 128-byte
// vector reads from 4 KB pages, with no search around them.
//
// Vector v sits at page (v / rpp) * page_bytes + (v % rpp) * vec_stride (the
// vectors-first page layout).  Each wave reads `per_wave` vectors whose ids
// are drawn uniformly (fixed seed), 8 lanes x 16 bytes per vector, ROUNDS
// rounds of 8 vectors in flight, through a 16-byte-stride buffer resource,
// the same instructions as the search's gather.  The grid is `waves`
// one-wave workgroups at four waves per SIMD.  Prints one JSON line with the
// best of 5 timed launches per depth.
//
// With vector_bytes > 128 (a multiple of 128, e.g. 384 for 96 float32s) the
// line also holds two whole-vector patterns over the same ids: "by_lines"
// (8 lanes per vector, each lane 16 bytes of every 128, 8 vectors per
// round, 8 rounds in flight) and "lane_per_vector" (each lane reads its own
// whole vector as vector_bytes / 16 separate 16-byte loads).  Rates count
// vector_bytes per vector.
//
//   gather_ceiling [n_vectors rpp page_bytes vec_stride waves per_wave vector_bytes]
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#define CHECK(x)                                                                   \
  do {                                                                             \
    hipError_t e_ = (x);                                                           \
    if (e_ != hipSuccess) {                                                        \
      fprintf(stderr, "gather_ceiling: %s at line %d\n", hipGetErrorString(e_), __LINE__); \
      return 1;                                                                    \
    }                                                                              \
  } while (0)

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ u32x4_t buffer_load_b128(__amdgpu_buffer_rsrc_t rsrc, int vindex, int voffset, int soffset,
                                    int aux) __asm("llvm.amdgcn.struct.ptr.buffer.load.v4i32");

template <int ROUNDS>
__global__ __launch_bounds__(64, 4) void gather(const uint8_t *pages, uint32_t units, const uint32_t *loc,
                                                uint32_t per_wave, uint32_t *sink) {
  const int l = threadIdx.x, g = l >> 3, gl = l & 7;
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(pages), (short)16, (int)units, 0x00020000);
  const uint32_t *my = loc + (uint64_t)blockIdx.x * per_wave;
  uint32_t acc = 0;
  for (uint32_t v0 = 0; v0 < per_wave; v0 += ROUNDS * 8) {
    u32x4_t x[ROUNDS];
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) x[r] = buffer_load_b128(rs, (int)(my[v0 + r * 8 + g] + gl), 0, 0, 0);
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) acc = __builtin_amdgcn_udot4(x[r].x ^ x[r].z, x[r].y ^ x[r].w, acc, false);
  }
  if (acc == 0x9E3779B9u) sink[blockIdx.x * 64 + l] = acc;  // keeps the loads
}

// Whole vectors of J 128-byte lines, 8 lanes per vector.
template <int J>
__global__ __launch_bounds__(64, 2) void gather_lines(const uint8_t *pages, uint32_t units, const uint32_t *loc,
                                                      uint32_t per_wave, uint32_t *sink) {
  const int l = threadIdx.x, g = l >> 3, gl = l & 7;
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(pages), (short)16, (int)units, 0x00020000);
  const uint32_t *my = loc + (uint64_t)blockIdx.x * per_wave;
  uint32_t acc = 0;
  for (uint32_t v0 = 0; v0 < per_wave; v0 += 64) {
    u32x4_t x[8][J];
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
      for (int j = 0; j < J; ++j) x[r][j] = buffer_load_b128(rs, (int)(my[v0 + r * 8 + g] + gl + 8 * j), 0, 0, 0);
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
      for (int j = 0; j < J; ++j) acc = __builtin_amdgcn_udot4(x[r][j].x ^ x[r][j].z, x[r][j].y ^ x[r][j].w, acc, false);
  }
  if (acc == 0x9E3779B9u) sink[blockIdx.x * 64 + l] = acc;
}

// Whole vectors of J 128-byte lines, one lane per vector.
template <int J>
__global__ __launch_bounds__(64, 2) void gather_lane_per_vector(const uint8_t *pages, uint32_t units,
                                                                const uint32_t *loc, uint32_t per_wave,
                                                                uint32_t *sink) {
  const int l = threadIdx.x;
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(pages), (short)16, (int)units, 0x00020000);
  const uint32_t *my = loc + (uint64_t)blockIdx.x * per_wave;
  uint32_t acc = 0;
  for (uint32_t v0 = 0; v0 < per_wave; v0 += 64) {
    u32x4_t x[8 * J];
    const uint32_t u = my[v0 + l];
#pragma unroll
    for (int i = 0; i < 8 * J; ++i) x[i] = buffer_load_b128(rs, (int)(u + i), 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 8 * J; ++i) acc = __builtin_amdgcn_udot4(x[i].x ^ x[i].z, x[i].y ^ x[i].w, acc, false);
  }
  if (acc == 0x9E3779B9u) sink[blockIdx.x * 64 + l] = acc;
}

template <int J>
void launch_whole(bool by_lines, uint32_t waves, const uint8_t *pages, uint32_t units, const uint32_t *loc,
                  uint32_t per_wave, uint32_t *sink) {
  if (by_lines) gather_lines<J><<<waves, 64>>>(pages, units, loc, per_wave, sink);
  else gather_lane_per_vector<J><<<waves, 64>>>(pages, units, loc, per_wave, sink);
}

int main(int argc, char **argv) {
  const uint64_t n = argc > 1 ? strtoull(argv[1], nullptr, 10) : 1000000;
  const uint64_t rpp = argc > 2 ? strtoull(argv[2], nullptr, 10) : 10;
  const uint64_t page_bytes = argc > 3 ? strtoull(argv[3], nullptr, 10) : 4096;
  const uint64_t vec_stride = argc > 4 ? strtoull(argv[4], nullptr, 10) : 128;
  const uint32_t waves = argc > 5 ? (uint32_t)strtoul(argv[5], nullptr, 10) : 4096;
  const uint32_t per_wave = argc > 6 ? (uint32_t)strtoul(argv[6], nullptr, 10) : 10240;
  const uint64_t vector_bytes = argc > 7 ? strtoull(argv[7], nullptr, 10) : 128;
  const uint64_t num_pages = (n + rpp - 1) / rpp;
  const uint64_t units = num_pages * page_bytes / 16;
  if (n == 0 || rpp == 0 || page_bytes % 16 || vec_stride % 16 || vec_stride < 128 || rpp * vec_stride > page_bytes ||
      units >= (1ull << 31) || per_wave == 0 || per_wave % 256 || waves == 0 || vector_bytes % 128 ||
      vector_bytes == 0 || vector_bytes > 512 || vector_bytes > vec_stride) {
    fprintf(stderr, "gather_ceiling: unsupported geometry\n");
    return 2;
  }
  const uint64_t nvec = (uint64_t)per_wave * waves;
  std::vector<uint32_t> loc(nvec);
  std::mt19937_64 rng(20260);
  for (auto &x : loc) {
    const uint64_t v = rng() % n;
    x = (uint32_t)(((v / rpp) * page_bytes + (v % rpp) * vec_stride) / 16);  // every unit read stays in the page
  }
  uint8_t *d_pages = nullptr;
  uint32_t *d_loc = nullptr, *d_sink = nullptr;
  CHECK(hipMalloc(&d_pages, num_pages * page_bytes));
  CHECK(hipMemset(d_pages, 1, num_pages * page_bytes));
  CHECK(hipMalloc(&d_loc, nvec * 4));
  CHECK(hipMemcpy(d_loc, loc.data(), nvec * 4, hipMemcpyHostToDevice));
  CHECK(hipMalloc(&d_sink, (size_t)waves * 64 * 4));
  hipEvent_t a, b;
  CHECK(hipEventCreate(&a));
  CHECK(hipEventCreate(&b));
  printf("{\"vectors\": %llu, \"waves\": %u, \"vector_bytes\": 128", (unsigned long long)nvec, waves);
  for (int rounds : {8, 16, 32}) {
    float best = 1e30f;
    for (int it = 0; it < 6; ++it) {
      CHECK(hipEventRecord(a));
      if (rounds == 8) gather<8><<<waves, 64>>>(d_pages, (uint32_t)units, d_loc, per_wave, d_sink);
      if (rounds == 16) gather<16><<<waves, 64>>>(d_pages, (uint32_t)units, d_loc, per_wave, d_sink);
      if (rounds == 32) gather<32><<<waves, 64>>>(d_pages, (uint32_t)units, d_loc, per_wave, d_sink);
      CHECK(hipGetLastError());
      CHECK(hipEventRecord(b));
      CHECK(hipEventSynchronize(b));
      float ms = 0;
      CHECK(hipEventElapsedTime(&ms, a, b));
      if (it > 0 && ms < best) best = ms;
    }
    printf(", \"rounds_%d\": {\"ms\": %.4f, \"gbs\": %.1f}", rounds, best, nvec * 128.0 / (best * 1e-3) / 1e9);
  }
  if (vector_bytes > 128) {
    const int J = (int)(vector_bytes / 128);
    for (int by_lines = 1; by_lines >= 0; --by_lines) {
      float best = 1e30f;
      for (int it = 0; it < 6; ++it) {
        CHECK(hipEventRecord(a));
        switch (J) {
          case 2: launch_whole<2>(by_lines, waves, d_pages, (uint32_t)units, d_loc, per_wave, d_sink); break;
          case 3: launch_whole<3>(by_lines, waves, d_pages, (uint32_t)units, d_loc, per_wave, d_sink); break;
          default: launch_whole<4>(by_lines, waves, d_pages, (uint32_t)units, d_loc, per_wave, d_sink); break;
        }
        CHECK(hipGetLastError());
        CHECK(hipEventRecord(b));
        CHECK(hipEventSynchronize(b));
        float ms = 0;
        CHECK(hipEventElapsedTime(&ms, a, b));
        if (it > 0 && ms < best) best = ms;
      }
      printf(", \"%s\": {\"vector_bytes\": %llu, \"ms\": %.4f, \"gbs\": %.1f}",
             by_lines ? "by_lines" : "lane_per_vector", (unsigned long long)vector_bytes, best,
             nvec * (double)vector_bytes / (best * 1e-3) / 1e9);
    }
  }
  printf("}\n");
  (void)hipFree(d_pages);
  (void)hipFree(d_loc);
  (void)hipFree(d_sink);
  return 0;
}
