// C ABI of the paged graph beam-search library (declared in include/gorio.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cstdio>
#include <thread>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/gorio.h"
#include "build_kernels.hpp"
#include "cluster.hpp"
#include "index.hpp"
#include "launch.hpp"
#include "queue_launch.hpp"

#if defined(__x86_64__)
#include <immintrin.h>
#define GORIO_CPU_PAUSE() _mm_pause()
#else
#define GORIO_CPU_PAUSE() std::this_thread::yield()
#endif

using namespace gorio;

// ---------------------------------------------------------------------------
// errors
// ---------------------------------------------------------------------------
static thread_local std::string g_last_error;

gorio_status gorio::fail(gorio_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

extern "C" const char *gorio_last_error(void) { return g_last_error.c_str(); }

#define HIP_OR_FAIL(expr)                                                                  \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess)                                                                  \
      return fail(e_ == hipErrorOutOfMemory ? GORIO_ENOMEM : GORIO_EDEVICE, "%s: %s", #expr, \
                  hipGetErrorString(e_));                                                  \
  } while (0)

namespace {

struct DeviceGuard {
  int prev = -1;
  bool ok = true;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

// Device buffer freed on scope exit unless released.
struct DevBuf {
  void *p = nullptr;
  ~DevBuf() { if (p) (void)hipFree(p); }
  hipError_t alloc(size_t bytes) { return hipMalloc(&p, bytes ? bytes : 4); }
  void *release() { void *r = p; p = nullptr; return r; }
  template <class T> T *as() const { return static_cast<T *>(p); }
};

bool is_device_pointer(const void *ptr) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, ptr) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeDevice || a.isManaged;
}

int env_int(const char *name, int dflt) {
  const char *v = getenv(name);
  return v && *v ? atoi(v) : dflt;
}

uint32_t vec_bytes_of(gorio_dtype dt, uint32_t D) { return dt == GORIO_U8 ? D : 4u * D; }

int grid_for(uint64_t items, int per_block, int cap = 65536) {
  uint64_t g = (items + per_block - 1) / per_block;
  return (int)std::max<uint64_t>(1, std::min<uint64_t>(g, cap));
}

}  // namespace

// ---------------------------------------------------------------------------
// build
// ---------------------------------------------------------------------------
extern "C" gorio_status gorio_build_index(gorio_dtype dtype, const void *vectors, uint64_t n, uint32_t D,
                                          const uint32_t *graph, uint32_t R,
                                          const gorio_page_layout *layout, uint32_t entry,
                                          gorio_index **out) {
  if (!out) return fail(GORIO_EINVAL, "out is NULL");
  *out = nullptr;
  if (dtype != GORIO_U8 && dtype != GORIO_F32) return fail(GORIO_EINVAL, "unknown dtype %d", (int)dtype);
  if (!vectors || !graph) return fail(GORIO_EINVAL, "vectors and graph must be non-NULL");
  if (n == 0 || n >= (1ull << 31)) return fail(GORIO_EINVAL, "n=%llu outside [1, 2^31)", (unsigned long long)n);
  if (R == 0 || R > 256) return fail(GORIO_EINVAL, "R=%u outside [1, 256]", R);
  if (dtype == GORIO_U8 && (D == 0 || D % 4 != 0 || D > 512))
    return fail(GORIO_EINVAL, "uint8 D=%u must be a multiple of 4 in [4, 512]", D);
  if (dtype == GORIO_F32 && (D == 0 || D > 256)) return fail(GORIO_EINVAL, "float32 D=%u outside [1, 256]", D);
  if (entry != UINT32_MAX && entry >= n) return fail(GORIO_EINVAL, "entry %u >= n", entry);

  const uint32_t vb = vec_bytes_of(dtype, D);
  const uint32_t arrangement = layout ? layout->arrangement : (uint32_t)GORIO_LAYOUT_DEFAULT;
  if (arrangement > (uint32_t)GORIO_LAYOUT_CONTIGUOUS)
    return fail(GORIO_EINVAL, "arrangement=%u is not a gorio_arrangement", arrangement);
  const bool vfirst = arrangement != (uint32_t)GORIO_LAYOUT_CONTIGUOUS;
  // vectors first: each vector slot is rounded up to 16 bytes
  const uint32_t min_rec = (vfirst ? ((vb + 15u) & ~15u) : vb) + 4 + 4 * R;
  uint32_t page_bytes = layout && layout->page_bytes ? layout->page_bytes : 4096;
  uint32_t rec_bytes = layout && layout->record_bytes ? layout->record_bytes : min_rec;
  if (page_bytes % 16 != 0) return fail(GORIO_EINVAL, "page_bytes=%u is not a multiple of 16", page_bytes);
  if (rec_bytes < min_rec || rec_bytes % 4 != 0)
    return fail(GORIO_EINVAL, "record_bytes=%u must be a multiple of 4 and >= %u", rec_bytes, min_rec);
  uint32_t rpp = layout && layout->records_per_page ? layout->records_per_page : page_bytes / rec_bytes;
  if (rpp == 0 || (uint64_t)rpp * rec_bytes > page_bytes)
    return fail(GORIO_EINVAL, "%u records of %u bytes do not fit a %u-byte page", rpp, rec_bytes, page_bytes);
  const uint32_t *n2s_host = layout ? layout->node_to_slot : nullptr;

  int dev = 0;
  HIP_OR_FAIL(hipGetDevice(&dev));
  auto ix = std::make_unique<gorio_index>();
  ix->device = dev;
  ix->dtype = dtype;
  ix->n = n;
  ix->D = D;
  ix->R = R;
  ix->vec_bytes = vb;
  ix->page_bytes = page_bytes;
  ix->rec_bytes = rec_bytes;
  ix->rpp = rpp;
  ix->vectors_first = vfirst;
  ix->num_pages = (n + rpp - 1) / rpp;

  HIP_OR_FAIL(hipStreamCreateWithFlags(&ix->stream, hipStreamNonBlocking));
  HIP_OR_FAIL(hipEventCreate(&ix->ev_start));
  HIP_OR_FAIL(hipEventCreate(&ix->ev_stop));
  HIP_OR_FAIL(hipEventCreateWithFlags(&ix->ev_done, hipEventDisableTiming));
  HIP_OR_FAIL(hipMalloc(&ix->d_stats, sizeof(unsigned long long) * 2 * kStatWords));
  hipStream_t s = ix->stream;
  fill_u32<<<1, 64, 0, s>>>(reinterpret_cast<uint32_t *>(ix->d_stats), 4 * kStatWords, 0u);

  DevBuf d_vec, d_graph, d_flags;
  HIP_OR_FAIL(d_vec.alloc((size_t)n * vb));
  HIP_OR_FAIL(d_graph.alloc((size_t)n * R * 4));
  HIP_OR_FAIL(d_flags.alloc(64));
  HIP_OR_FAIL(hipMemcpyAsync(d_vec.p, vectors, (size_t)n * vb, hipMemcpyHostToDevice, s));
  HIP_OR_FAIL(hipMemcpyAsync(d_graph.p, graph, (size_t)n * R * 4, hipMemcpyHostToDevice, s));
  unsigned int *bad = d_flags.as<unsigned int>();
  unsigned long long *best = reinterpret_cast<unsigned long long *>(d_flags.as<char>() + 8);
  fill_u32<<<1, 64, 0, s>>>(d_flags.as<uint32_t>(), 16, 0u);
  fill_u32<<<1, 64, 0, s>>>(reinterpret_cast<uint32_t *>(best), 2, 0xFFFFFFFFu);

  if (n2s_host) {
    HIP_OR_FAIL(hipMalloc(&ix->d_node_to_slot, (size_t)n * 4));
    HIP_OR_FAIL(hipMemcpyAsync(ix->d_node_to_slot, n2s_host, (size_t)n * 4, hipMemcpyHostToDevice, s));
    DevBuf bits;
    const uint64_t words = (n + 31) / 32;
    HIP_OR_FAIL(bits.alloc(words * 4));
    fill_u32<<<grid_for(words, 256), 256, 0, s>>>(bits.as<uint32_t>(), words, 0u);
    check_permutation<<<grid_for(n, 256), 256, 0, s>>>(ix->d_node_to_slot, (uint32_t)n,
                                                       bits.as<uint32_t>(), bad);
    unsigned int h_bad = 0;
    HIP_OR_FAIL(hipMemcpyAsync(&h_bad, bad, 4, hipMemcpyDeviceToHost, s));
    HIP_OR_FAIL(hipStreamSynchronize(s));
    if (h_bad) return fail(GORIO_EINVAL, "node_to_slot is not a permutation of [0, n)");
  }

  // pack into HBM
  const uint64_t index_bytes = ix->num_pages * (uint64_t)page_bytes;
  HIP_OR_FAIL(hipMalloc(&ix->d_pages, index_bytes));
  fill_u32<<<grid_for(index_bytes / 4, 256), 256, 0, s>>>(reinterpret_cast<uint32_t *>(ix->d_pages),
                                                          index_bytes / 4, 0u);
  PageGeom geom = ix->geom();
  pack_records<<<grid_for(n, 4), 256, 0, s>>>(d_vec.as<uint8_t>(), vb, d_graph.as<uint32_t>(), R,
                                              (uint32_t)n, geom, ix->d_pages, bad);
  HIP_OR_FAIL(hipGetLastError());

  // entry node
  if (entry == UINT32_MAX) {
    DevBuf sums;
    HIP_OR_FAIL(sums.alloc(sizeof(double) * D));
    fill_u32<<<1, 256, 0, s>>>(sums.as<uint32_t>(), 2ull * D, 0u);
    if (dtype == GORIO_U8) {
      const uint32_t rows = 4096;
      column_sums_u8<<<grid_for(n, rows, 1 << 30), 256, 0, s>>>(
          d_vec.as<uint8_t>(), (uint32_t)n, D, rows, sums.as<unsigned long long>());
      nearest_to_centroid_u8<<<grid_for(n, 256, 2048), 256, 0, s>>>(
          d_vec.as<uint8_t>(), (uint32_t)n, D, sums.as<unsigned long long>(), best);
    } else {
      column_sums_f32_ordered<<<(D + 63) / 64, 64, 0, s>>>(d_vec.as<float>(), (uint32_t)n, D,
                                                           sums.as<double>());
      nearest_to_centroid_f32<<<grid_for(n, 256, 2048), 256, 0, s>>>(d_vec.as<float>(), (uint32_t)n, D,
                                                                    sums.as<double>(), best);
    }
    HIP_OR_FAIL(hipGetLastError());
    unsigned long long h_best = 0;
    HIP_OR_FAIL(hipMemcpyAsync(&h_best, best, 8, hipMemcpyDeviceToHost, s));
    HIP_OR_FAIL(hipStreamSynchronize(s));
    ix->entry = (uint32_t)(h_best & 0xFFFFFFFFu);
  } else {
    ix->entry = entry;
  }
  unsigned int h_bad = 0;
  HIP_OR_FAIL(hipMemcpyAsync(&h_bad, bad, 4, hipMemcpyDeviceToHost, s));
  HIP_OR_FAIL(hipStreamSynchronize(s));
  if (h_bad) return fail(GORIO_EINVAL, "graph holds %u ids >= n that are not UINT32_MAX", h_bad);
  if (ix->entry >= n) return fail(GORIO_EDEVICE, "entry selection failed");

  ix->resident = true;
  *out = ix.release();
  return GORIO_OK;
}

// ---------------------------------------------------------------------------
// paged mode: memory
// ---------------------------------------------------------------------------
namespace {
constexpr uint32_t kMaxPendingPerQuery = 32;  // page requests one query keeps outstanding

uint32_t next_pow2(uint64_t v) {
  uint32_t p = 1;
  while (p < v) p <<= 1;
  return p;
}

template <class T>
hipError_t host_ring(T **h, T **d, size_t count) {
  hipError_t e = hipHostMalloc(reinterpret_cast<void **>(h), count * sizeof(T),
                               hipHostMallocCoherent | hipHostMallocMapped);
  if (e != hipSuccess) return e;
  memset(*h, 0, count * sizeof(T));
  return hipHostGetDevicePointer(reinterpret_cast<void **>(d), *h, 0);
}
}  // namespace

gorio_status gorio_index::make_paged(uint64_t slots) {
  using namespace gorio;
  if (slots < 2ull * kMaxPendingPerQuery)
    return fail(GORIO_EINVAL, "a paged cache needs at least %u slots (asked for %llu)",
                2 * kMaxPendingPerQuery, (unsigned long long)slots);
  if (slots * (uint64_t)page_bytes > 0x7FFFF000ull)
    return fail(GORIO_EUNSUPPORTED, "a paged cache is limited to 2 GiB (asked for %llu slots)",
                (unsigned long long)slots);
  if (resident) {
    hipError_t e = hipHostMalloc(reinterpret_cast<void **>(&h_backing), index_bytes(), hipHostMallocDefault);
    if (e != hipSuccess)
      return fail(GORIO_ENOMEM, "pinned backing store of %llu bytes failed", (unsigned long long)index_bytes());
    e = hipMemcpy(h_backing, d_pages, index_bytes(), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail(GORIO_EDEVICE, "page download failed: %s", hipGetErrorString(e));
    (void)hipFree(d_pages);
    d_pages = nullptr;
    resident = false;
  }
  if (paged) paged->release();
  paged = std::make_unique<PagedState>();
  PagedState &P = *paged;
  P.slots = slots;
  P.ctrl_stride = (uint32_t)std::max(1, std::min(32, env_int("GORIO_CTRL_STRIDE", (int)PagedState::kCtrlStride)));
  HIP_OR_FAIL(hipMalloc(&P.d_cache, slots * (uint64_t)page_bytes));
  HIP_OR_FAIL(hipMalloc(&P.d_slot_word, slots * sizeof(unsigned long long)));
  HIP_OR_FAIL(hipMalloc(&P.d_page_slot, num_pages * sizeof(uint32_t)));
  HIP_OR_FAIL(hipMalloc(&P.d_ctrl, PagedState::kCtrlWords * PagedState::kCtrlStride * sizeof(unsigned long long)));
  // Every descriptor and every unconsumed completion belongs to a LOADING
  // slot, so no ring ever holds more than `slots` live entries.
  P.ring_cap = next_pow2(2 * slots + 1024);
  P.cq_cap = next_pow2(slots + 1024);
  HIP_OR_FAIL(host_ring(&P.h_mq, &P.d_mq, P.ring_cap));
  HIP_OR_FAIL(host_ring(&P.h_cq, &P.d_cq, (size_t)P.cq_cap * PagedState::kMaxRings));
  HIP_OR_FAIL(host_ring(&P.h_cq_tail, &P.d_cq_tail, (size_t)PagedState::kTailStride * PagedState::kMaxRings));
  HIP_OR_FAIL(host_ring(&P.h_abort, &P.d_abort, 16));
  cache_slots = slots;
  gorio_status st = reset_cache();
  if (st != GORIO_OK) return st;
  P.proxy.start(P.h_mq, P.ring_cap - 1, P.h_cq, P.cq_cap - 1, P.h_cq_tail, PagedState::kTailStride);
  return GORIO_OK;
}

// Empty the cache (every slot EMPTY, no page mapped).
gorio_status gorio_index::reset_cache() {
  using namespace gorio;
  PagedState &P = *paged;
  fill_u32<<<grid_for(P.slots * 2, 256), 256, 0, stream>>>(reinterpret_cast<uint32_t *>(P.d_slot_word),
                                                           P.slots * 2, 0u);
  fill_u32<<<grid_for(num_pages, 256), 256, 0, stream>>>(P.d_page_slot, num_pages, 0xFFFFFFFFu);
  fill_u32<<<1, 256, 0, stream>>>(reinterpret_cast<uint32_t *>(P.d_ctrl), 2 * PagedState::kCtrlWords * PagedState::kCtrlStride, 0u);
  HIP_OR_FAIL(hipGetLastError());
  HIP_OR_FAIL(hipStreamSynchronize(stream));
  return GORIO_OK;
}

// ---------------------------------------------------------------------------
// cache / backing configuration
// ---------------------------------------------------------------------------
extern "C" gorio_status gorio_set_cache(gorio_index *ix, uint64_t bytes) {
  if (!ix) return fail(GORIO_EINVAL, "index is NULL");
  DeviceGuard dg(ix->device);
  if (bytes >= ix->index_bytes()) return ix->make_resident();
  return ix->make_paged(bytes / ix->page_bytes);
}

extern "C" gorio_status gorio_set_query_order(gorio_index *ix, const float *centroids, uint32_t clusters) {
  if (!ix) return fail(GORIO_EINVAL, "index is NULL");
  if (clusters > kMaxClusters) return fail(GORIO_EINVAL, "clusters=%u above %u", clusters, kMaxClusters);
  if (clusters > 0 && !centroids) return fail(GORIO_EINVAL, "centroids must be non-NULL");
  DeviceGuard dg(ix->device);
  if (ix->d_centroids) (void)hipFree(ix->d_centroids);
  if (ix->d_centroid_norms) (void)hipFree(ix->d_centroid_norms);
  ix->d_centroids = ix->d_centroid_norms = nullptr;
  ix->order_clusters = 0;
  if (clusters == 0) return GORIO_OK;
  std::vector<float> cc(clusters);
  centroid_norms(centroids, clusters, ix->D, cc.data());
  HIP_OR_FAIL(hipMalloc(&ix->d_centroids, (size_t)clusters * ix->D * 4));
  HIP_OR_FAIL(hipMalloc(&ix->d_centroid_norms, (size_t)clusters * 4));
  HIP_OR_FAIL(hipMemcpy(ix->d_centroids, centroids, (size_t)clusters * ix->D * 4, hipMemcpyHostToDevice));
  HIP_OR_FAIL(hipMemcpy(ix->d_centroid_norms, cc.data(), (size_t)clusters * 4, hipMemcpyHostToDevice));
  ix->order_clusters = clusters;
  return GORIO_OK;
}

extern "C" gorio_status gorio_set_backing(gorio_index *ix, double latency_us, uint32_t max_outstanding,
                                          uint32_t oversub, int blocking) {
  if (!ix) return fail(GORIO_EINVAL, "index is NULL");
  if (!(latency_us >= 0.0) || latency_us > 1e7) return fail(GORIO_EINVAL, "latency_us=%g out of range", latency_us);
  if (oversub < 1 || oversub > 16) return fail(GORIO_EINVAL, "oversub=%u outside [1, 16]", oversub);
  if (blocking < 0 || blocking > 3) return fail(GORIO_EINVAL, "mode (blocking) must be 0, 1, 2 or 3");
  ix->latency_us = latency_us;
  ix->max_outstanding = max_outstanding ? max_outstanding : 4096;
  ix->oversub = oversub;
  ix->blocking = blocking;
  return GORIO_OK;
}

extern "C" gorio_status gorio_set_scheduler(gorio_index *ix, uint32_t query_waves, uint32_t max_pending) {
  if (!ix) return fail(GORIO_EINVAL, "index is NULL");
  if (query_waves > 65536) return fail(GORIO_EINVAL, "query_waves=%u above 65536", query_waves);
  if (max_pending > 256) return fail(GORIO_EINVAL, "max_pending=%u above 256", max_pending);
  ix->query_waves = query_waves;
  ix->max_pending = max_pending;
  return GORIO_OK;
}

// ---------------------------------------------------------------------------
// search
// ---------------------------------------------------------------------------
namespace {

// Host-scheduled lanes (the GustANN-style comparison point of Sec. 5.1, over
// the same page cache, miss descriptors and proxy): the calling thread owns
// the query schedule.  It keeps `lanes` query lanes, starts queries in free
// lanes in admission order, and hands the lanes it deems runnable to the GPU:
// by default to one persistent launch whose executor waves take them from a
// ring in host memory, else (GORIO_HOST_EXECUTOR=0) in round kernels, up to
// GORIO_ROUND_FLIGHTS in flight on streams of their own.  Each lane's report
// ends with a sequence number, so a lane is retired as soon as its turn is
// over.  A lane is runnable when one of the cache slots it reported waiting
// for has been filled -- the fill waves publish, per completion ring, how many
// completions they have copied, and the host reads the filled {page, slot}
// entries back from the ring -- or, for a lane that could not issue all of
// its requests, when any page has been filled, or at once when its turn ended
// while it could still proceed.  A slot filled while the lane's turn ran is
// caught by comparing when the host saw that fill with when the lane was
// handed over.  A lane not woken within a few milliseconds is run anyway, so
// a missed wake costs time, never progress.
gorio_status run_host_rounds(gorio_index *ix, PagedParams &pp, uint32_t lanes, const std::vector<uint32_t> &order,
                             hipStream_t s, double limit_s, bool &timed_out) {
  using Clock = std::chrono::steady_clock;
  constexpr int kMaxFlights = PagedState::kMaxFlights;
  // round kernels in flight at once (each on a stream of its own)
  const int flights = std::max(1, std::min(kMaxFlights, env_int("GORIO_ROUND_FLIGHTS", 2)));
  // the lanes' turns are run by one persistent launch that takes them from a
  // ring the host writes (the default), or by a launch per round
  const bool executor = env_int("GORIO_HOST_EXECUTOR", 1) != 0;
  // a turn ends when the lane parks; a launch per round also ends it after two
  // passes that found pages ready, since the round waits for its slowest lane
  pp.turn_passes = (uint32_t)std::max(0, env_int("GORIO_TURN_PASSES", executor ? 0 : 2));
  PagedState &P = *ix->paged;
  const uint32_t words = lane_state_words(pp.L);
  if ((uint64_t)lanes * words > P.lane_state_words) {
    if (P.d_lane_state) (void)hipFree(P.d_lane_state);
    P.d_lane_state = nullptr;
    P.lane_state_words = 0;
    HIP_OR_FAIL(hipMalloc(&P.d_lane_state, (uint64_t)lanes * words * 4));
    P.lane_state_words = (uint64_t)lanes * words;
  }
  if (lanes > P.round_cap) {
    if (P.h_round) (void)hipHostFree(P.h_round);
    if (P.h_lane_out) (void)hipHostFree(P.h_lane_out);
    P.h_round = P.d_round = nullptr;
    P.h_lane_out = P.d_lane_out = nullptr;
    P.round_cap = 0;
    HIP_OR_FAIL(host_ring(&P.h_round, &P.d_round, 2 * kMaxFlights * (size_t)lanes));
    HIP_OR_FAIL(host_ring(&P.h_lane_out, &P.d_lane_out, lanes));
    P.round_cap = lanes;
  }
  if (!P.h_fill_head)
    HIP_OR_FAIL(host_ring(&P.h_fill_head, &P.d_fill_head, (size_t)PagedState::kMaxRings * PagedState::kTailStride));
  if (!P.fill_stream) HIP_OR_FAIL(hipStreamCreateWithFlags(&P.fill_stream, hipStreamNonBlocking));
  for (int i = 1; i < flights; ++i)
    if (!P.round_stream[i]) HIP_OR_FAIL(hipStreamCreateWithFlags(&P.round_stream[i], hipStreamNonBlocking));
  for (int i = 0; i < flights; ++i)
    if (!P.ev_round[i]) HIP_OR_FAIL(hipEventCreateWithFlags(&P.ev_round[i], hipEventDisableTiming));
  if (!P.ev_fill) HIP_OR_FAIL(hipEventCreateWithFlags(&P.ev_fill, hipEventDisableTiming));
  const uint32_t rings = std::max(1u, pp.fill_waves);
  for (uint32_t r = 0; r < rings; ++r)
    __atomic_store_n(P.h_fill_head + (size_t)r * PagedState::kTailStride, 0ull, __ATOMIC_RELEASE);
  pp.fill_head = P.d_fill_head;
  hipStream_t rstream[kMaxFlights];
  RoundParams rp[kMaxFlights] = {};
  uint32_t *h_lanes[kMaxFlights], *h_admit[kMaxFlights];
  for (int i = 0; i < flights; ++i) {
    rstream[i] = i == 0 ? s : P.round_stream[i];
    rp[i].lanes = P.d_round + (size_t)2 * i * lanes;
    rp[i].admit = P.d_round + (size_t)(2 * i + 1) * lanes;
    rp[i].state = P.d_lane_state;
    rp[i].state_words = words;
    rp[i].out = P.d_lane_out;
    h_lanes[i] = P.h_round + (size_t)2 * i * lanes;
    h_admit[i] = P.h_round + (size_t)(2 * i + 1) * lanes;
  }

  // fill waves in a kernel of their own, and the second round stream, both
  // after the control words were reset on s.  The fill kernel leaves after
  // about two milliseconds and is launched again (from the ring positions it
  // published) as soon as it has: no kernel of this mode waits on the GPU
  // for work of another stream, so progress does not depend on how the
  // runtime maps streams to hardware queues (streams that share a queue run
  // one after another).
  int clock_khz = 0;
  HIP_OR_FAIL(hipDeviceGetAttribute(&clock_khz, hipDeviceAttributeWallClockRate, ix->device));
  const int budget_us = std::max(50, env_int("GORIO_FILL_BUDGET_US", 2000));
  pp.fill_budget = (unsigned long long)std::max(1.0, (double)clock_khz * budget_us / 1000.0);
  HIP_OR_FAIL(hipEventRecord(ix->ev_start, s));
  HIP_OR_FAIL(hipStreamWaitEvent(P.fill_stream, ix->ev_start, 0));
  for (int i = 1; i < flights; ++i) HIP_OR_FAIL(hipStreamWaitEvent(P.round_stream[i], ix->ev_start, 0));
  // persistent launch: fill waves and executor waves in one kernel on s
  uint64_t runq_tail = 0;
  if (executor) {
    uint32_t cap = 1;
    while (cap < 2 * lanes + 64) cap <<= 1;
    if (cap > P.runq_cap) {
      if (P.h_runq) (void)hipHostFree(P.h_runq);
      P.h_runq = P.d_runq = nullptr;
      P.runq_cap = 0;
      HIP_OR_FAIL(host_ring(&P.h_runq, &P.d_runq, cap));
      P.runq_cap = cap;
    }
    if (!P.h_runq_ctl) HIP_OR_FAIL(host_ring(&P.h_runq_ctl, &P.d_runq_ctl, (size_t)PagedState::kTailStride));
    memset(P.h_runq, 0, P.runq_cap * sizeof(unsigned long long));
    __atomic_store_n(P.h_runq_ctl, 0ull, __ATOMIC_RELEASE);
    RoundParams rx = {};
    rx.state = P.d_lane_state;
    rx.state_words = words;
    rx.out = P.d_lane_out;
    rx.runq = P.d_runq;
    rx.runq_tail = P.d_runq_ctl;
    rx.runq_head = P.ctrl(PagedState::kNextQuery);  // zeroed with the other control words
    rx.runq_tail_seen = P.ctrl(PagedState::kRunqTailSeen);
    rx.runq_mask = P.runq_cap - 1;
    rx.out_lanes = lanes;
    int cus = 0;
    HIP_OR_FAIL(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, ix->device));
    const int execs = (int)std::min<uint64_t>(lanes, (uint64_t)cus * 4);
    pp.fill_budget = 0;  // the fill waves stay until every query is done
    const int grid = (int)pp.fill_waves + 1 + execs;  // fill waves, the tail mirror, executors
    const hipError_t le = ix->dtype == GORIO_F32 ? launch_rounds_f32(pp, rx, grid, s)
                                                 : launch_rounds_u8(pp, rx, grid, s);
    if (le != hipSuccess) return fail(GORIO_EDEVICE, "executor launch failed: %s", hipGetErrorString(le));
    const hipError_t re = hipEventRecord(P.ev_round[0], s);
    if (re != hipSuccess) {
      // the launch leaves on the abort flag; it is over before the caller
      // stops the proxy it would wait on
      __atomic_store_n(P.h_abort, 1u, __ATOMIC_RELEASE);
      (void)hipStreamSynchronize(s);
      return fail(GORIO_EDEVICE, "hipEventRecord: %s", hipGetErrorString(re));
    }
  }
  auto push_lane = [&](uint32_t lane, uint32_t q) {  // q = kNone: go on with the lane's query
    const unsigned long long e = ((unsigned long long)(q == kNone ? 0u : q + 1u) << 32) | (lane + 1u);
    __atomic_store_n(&P.h_runq[runq_tail & (P.runq_cap - 1)], e, __ATOMIC_RELAXED);
    ++runq_tail;
  };
  bool fill_busy = false;
  auto launch_fill = [&]() -> hipError_t {
    hipError_t le = ix->dtype == GORIO_F32 ? launch_paged_f32(pp, (int)pp.fill_waves, P.fill_stream)
                                           : launch_paged_u8(pp, (int)pp.fill_waves, P.fill_stream);
    if (le == hipSuccess) le = hipEventRecord(P.ev_fill, P.fill_stream);
    fill_busy = le == hipSuccess;
    return le;
  };
  if (!executor) {
    const hipError_t le = launch_fill();
    if (le != hipSuccess) return fail(GORIO_EDEVICE, "fill kernel launch failed: %s", hipGetErrorString(le));
  }

  enum : uint8_t { kFree = 0, kRunnable = 1, kWaiting = 2, kRunning = 3 };
  const uint64_t nq = pp.nq;
  std::vector<uint8_t> lstate(lanes, kFree);
  std::vector<uint32_t> epoch(lanes, 0);
  std::vector<Clock::time_point> since(lanes);
  std::vector<uint32_t> runq, freeq;
  runq.reserve(lanes);
  freeq.reserve(lanes);
  for (uint32_t l = lanes; l-- > 0;) freeq.push_back(l);
  using Waiter = std::pair<uint32_t, uint32_t>;  // lane, its park epoch
  std::vector<std::vector<Waiter>> waiters(P.slots);
  std::vector<Waiter> any_fill;
  std::vector<uint64_t> ring_head(rings, 0);
  // fill_seq counts the polls that found filled pages; slot_seq[s] is its
  // value when a fill of slot s was last seen
  uint64_t fill_seq = 0;
  std::vector<uint64_t> slot_seq(P.slots, 0);
  const uint64_t cq_cap = P.cq_cap;
  auto wake = [&](uint32_t lane, uint32_t ep) {
    if (lstate[lane] == kWaiting && epoch[lane] == ep) {
      lstate[lane] = kRunnable;
      runq.push_back(lane);
    }
  };
  auto poll_fills = [&]() {
    bool progress = false;
    for (uint32_t r = 0; r < rings; ++r) {
      const uint64_t fh = __atomic_load_n(P.h_fill_head + (size_t)r * PagedState::kTailStride, __ATOMIC_ACQUIRE);
      uint64_t &h = ring_head[r];
      if (fh <= h) continue;
      if (!progress) ++fill_seq;
      progress = true;
      if (fh - h > cq_cap) h = fh - cq_cap;  // entries already reused by the proxy: the fallback wakes them
      const unsigned long long *ring = P.h_cq + (size_t)r * cq_cap;
      for (; h < fh; ++h) {
        const uint32_t slot = (uint32_t)__atomic_load_n(&ring[h & (cq_cap - 1)], __ATOMIC_RELAXED);
        if (slot >= P.slots) continue;
        slot_seq[slot] = fill_seq;
        for (const Waiter &w : waiters[slot]) wake(w.first, w.second);
        waiters[slot].clear();
      }
    }
    if (progress && !any_fill.empty()) {
      for (const Waiter &w : any_fill) wake(w.first, w.second);
      any_fill.clear();
    }
    return progress;
  };
  struct Flight {
    bool busy = false;
    uint32_t n = 0;
    Clock::time_point t0;
  } fl[kMaxFlights];
  // A lane is retired as soon as its report says its turn is over (the
  // sequence number it publishes last), not when its launch ends: a round
  // lasts as long as its slowest lane, and the others go on meanwhile.
  std::vector<uint64_t> lane_fill_seq(lanes, 0);  // fill_seq when the lane's round was launched
  std::vector<uint32_t> out_seq(lanes);           // the last sequence number seen per lane
  for (uint32_t l = 0; l < lanes; ++l) out_seq[l] = __atomic_load_n(&P.h_lane_out[l].seq, __ATOMIC_ACQUIRE);
  std::vector<uint32_t> running;
  running.reserve(lanes);

  const auto t0 = Clock::now();
  auto last_sweep = t0;
  const auto stale = std::chrono::milliseconds(4);
  uint64_t admitted = 0, finished = 0;
  // scheduler counters (printed to stderr with GORIO_ROUNDS_STATS=1)
  uint64_t n_rounds = 0, n_lane_runs = 0, n_idle = 0, n_stale = 0, n_early = 0;
  double round_us = 0.0;
  const uint32_t min_round = std::max(1u, lanes / (4u * (uint32_t)flights));
  gorio_status st = GORIO_OK;
  // the lane's turn is over: act on its report
  auto retire_lane = [&](uint32_t lane, Clock::time_point done_at) {
    ++n_lane_runs;
    const LaneOut &o = P.h_lane_out[lane];
    if (o.code == kLaneIdle) ++n_idle;
    if (o.code == kLaneDone) {
      ++finished;
      lstate[lane] = kFree;
      freeq.push_back(lane);
      return;
    }
    const uint32_t ep = ++epoch[lane];
    bool now = o.code == kLaneYield;  // its turn ended while it could still proceed
    const uint32_t nw = std::min(o.nwait, kLaneWaitCap);
    for (uint32_t j = 0; j < nw && !now; ++j) {
      const uint32_t w = o.wait[j];
      if (w >= P.slots) continue;
      if (slot_seq[w] > lane_fill_seq[lane]) now = true;  // filled while the lane ran
      else waiters[w].push_back({lane, ep});
    }
    if (!now && (o.retry || nw == 0)) {
      if (fill_seq > lane_fill_seq[lane]) now = true;
      else any_fill.push_back({lane, ep});
    }
    if (now) {
      if (o.code != kLaneYield) ++n_early;
      lstate[lane] = kRunnable;
      runq.push_back(lane);
    } else {
      lstate[lane] = kWaiting;
      since[lane] = done_at;
    }
  };
  // lanes whose turn is over, whatever their launch is doing
  auto reap = [&]() {
    bool any = false;
    const auto done_at = Clock::now();
    for (size_t k = 0; k < running.size();) {
      const uint32_t lane = running[k];
      const uint32_t sq = __atomic_load_n(&P.h_lane_out[lane].seq, __ATOMIC_ACQUIRE);
      if (sq == out_seq[lane]) {
        ++k;
        continue;
      }
      out_seq[lane] = sq;
      running[k] = running.back();
      running.pop_back();
      retire_lane(lane, done_at);
      any = true;
    }
    return any;
  };

  while (finished < nq) {
    const auto now = Clock::now();
    if (std::chrono::duration<double>(now - t0).count() > limit_s) {
      timed_out = true;
      __atomic_store_n(P.h_abort, 1u, __ATOMIC_RELEASE);
      break;
    }
    if (now - last_sweep > std::chrono::milliseconds(1)) {  // lanes no fill has woken
      last_sweep = now;
      for (uint32_t l = 0; l < lanes; ++l)
        if (lstate[l] == kWaiting && now - since[l] > stale) {
          wake(l, epoch[l]);
          ++n_stale;
        }
    }
    bool acted = reap();
    if (executor) {
      const hipError_t q = hipEventQuery(P.ev_round[0]);
      if (q != hipErrorNotReady) {
        // the launch leaves once every query is done, possibly before the
        // last reports were read here
        if (q == hipSuccess) {
          reap();
          if (finished >= nq) break;
        }
        st = fail(GORIO_EDEVICE, "executor launch ended with %llu of %llu queries done%s%s",
                  (unsigned long long)finished, (unsigned long long)nq, q == hipSuccess ? "" : ": ",
                  q == hipSuccess ? "" : hipGetErrorString(q));
        break;
      }
      acted |= poll_fills();
      if (!runq.empty() || (!freeq.empty() && admitted < nq)) {
        for (uint32_t lane : runq) {
          lstate[lane] = kRunning;
          lane_fill_seq[lane] = fill_seq;
          running.push_back(lane);
          push_lane(lane, kNone);
        }
        runq.clear();
        while (!freeq.empty() && admitted < nq) {
          const uint32_t lane = freeq.back();
          freeq.pop_back();
          lstate[lane] = kRunning;
          lane_fill_seq[lane] = fill_seq;
          running.push_back(lane);
          push_lane(lane, order.empty() ? (uint32_t)admitted : order[admitted]);
          ++admitted;
        }
        __atomic_store_n(P.h_runq_ctl, (unsigned long long)runq_tail, __ATOMIC_RELEASE);
        acted = true;
      }
      if (!acted)
        for (int i = 0; i < 16; ++i) GORIO_CPU_PAUSE();
      continue;
    }
    for (int i = 0; i < flights; ++i) {
      if (!fl[i].busy) continue;
      const hipError_t q = hipEventQuery(P.ev_round[i]);
      if (q == hipErrorNotReady) continue;
      if (q != hipSuccess) {
        st = fail(GORIO_EDEVICE, "round failed: %s", hipGetErrorString(q));
        break;
      }
      // the launch is over (its lanes reported before it ended): its stream
      // and lane list are free again
      ++n_rounds;
      round_us += std::chrono::duration<double, std::micro>(Clock::now() - fl[i].t0).count();
      fl[i].busy = false;
      acted = true;
    }
    if (st != GORIO_OK) break;
    if (fill_busy) {
      const hipError_t q = hipEventQuery(P.ev_fill);
      if (q == hipSuccess) {
        fill_busy = false;
      } else if (q != hipErrorNotReady) {
        st = fail(GORIO_EDEVICE, "fill kernel failed: %s", hipGetErrorString(q));
        break;
      }
    }
    if (!fill_busy) {
      const hipError_t le = launch_fill();
      if (le != hipSuccess) {
        st = fail(GORIO_EDEVICE, "fill kernel launch failed: %s", hipGetErrorString(le));
        break;
      }
    }
    acted |= poll_fills();
    int busy = 0;
    for (int i = 0; i < flights; ++i) busy += fl[i].busy ? 1 : 0;
    for (int i = 0; i < flights; ++i) {
      if (fl[i].busy) continue;
      const uint64_t avail = runq.size() + std::min<uint64_t>(freeq.size(), nq - admitted);
      // with another round running, wait for a worthwhile number of lanes
      if (avail == 0 || (busy > 0 && avail < min_round)) break;
      uint32_t n = 0;
      for (uint32_t lane : runq) {
        h_lanes[i][n] = lane;
        h_admit[i][n] = kNone;
        lstate[lane] = kRunning;
        ++n;
      }
      runq.clear();
      while (!freeq.empty() && admitted < nq) {
        const uint32_t lane = freeq.back();
        freeq.pop_back();
        h_lanes[i][n] = lane;
        h_admit[i][n] = order.empty() ? (uint32_t)admitted : order[admitted];
        lstate[lane] = kRunning;
        ++admitted;
        ++n;
      }
      for (uint32_t k = 0; k < n; ++k) {
        lane_fill_seq[h_lanes[i][k]] = fill_seq;
        running.push_back(h_lanes[i][k]);
      }
      fl[i].t0 = Clock::now();
      const hipError_t le = ix->dtype == GORIO_F32 ? launch_rounds_f32(pp, rp[i], (int)n, rstream[i])
                                                   : launch_rounds_u8(pp, rp[i], (int)n, rstream[i]);
      if (le != hipSuccess) {
        st = fail(GORIO_EDEVICE, "round launch failed: %s", hipGetErrorString(le));
        break;
      }
      const hipError_t re = hipEventRecord(P.ev_round[i], rstream[i]);
      if (re != hipSuccess) {
        st = fail(GORIO_EDEVICE, "hipEventRecord: %s", hipGetErrorString(re));
        break;
      }
      fl[i].busy = true;
      fl[i].n = n;
      ++busy;
      acted = true;
    }
    if (st != GORIO_OK) break;
    if (!acted)
      for (int i = 0; i < 16; ++i) GORIO_CPU_PAUSE();
  }
  if (st != GORIO_OK || timed_out) __atomic_store_n(P.h_abort, 1u, __ATOMIC_RELEASE);
  if (executor) {
    // every wave of the launch leaves once every query is done (or on abort)
    for (;;) {
      const hipError_t q = hipEventQuery(P.ev_round[0]);
      if (q == hipSuccess) break;
      if (q != hipErrorNotReady) return fail(GORIO_EDEVICE, "executor launch failed: %s", hipGetErrorString(q));
      if (!timed_out && std::chrono::duration<double>(Clock::now() - t0).count() > limit_s) {
        timed_out = true;
        __atomic_store_n(P.h_abort, 1u, __ATOMIC_RELEASE);
      }
      std::this_thread::sleep_for(std::chrono::microseconds(50));
    }
    if (env_int("GORIO_ROUNDS_STATS", 0))
      fprintf(stderr, "[gorio rounds] lanes %u, executor, lane turns %llu (%llu not runnable), woken at report %llu, "
              "stale wakes %llu, %.3f s in all\n", lanes, (unsigned long long)n_lane_runs,
              (unsigned long long)n_idle, (unsigned long long)n_early, (unsigned long long)n_stale,
              std::chrono::duration<double>(Clock::now() - t0).count());
    HIP_OR_FAIL(hipEventRecord(ix->ev_stop, s));
    return st;
  }
  // rounds still in flight (after an error or the watchdog) finish: every lane
  // turn is bounded and stops at once on the abort flag
  for (int i = 0; i < flights; ++i)
    if (fl[i].busy) (void)hipEventSynchronize(P.ev_round[i]);
  if (env_int("GORIO_ROUNDS_STATS", 0))
    fprintf(stderr, "[gorio rounds] lanes %u, rounds %llu, lane runs %llu (%.1f per round, %llu not runnable), "
            "woken at retirement %llu, stale wakes %llu, %.1f us per round (launch to retirement), %.3f s in all\n",
            lanes, (unsigned long long)n_rounds, (unsigned long long)n_lane_runs,
            n_rounds ? (double)n_lane_runs / n_rounds : 0.0, (unsigned long long)n_idle,
            (unsigned long long)n_early, (unsigned long long)n_stale, n_rounds ? round_us / n_rounds : 0.0,
            std::chrono::duration<double>(Clock::now() - t0).count());
  // the last fill kernel leaves once every query is done (or on abort)
  HIP_OR_FAIL(hipEventRecord(P.ev_fill, P.fill_stream));
  for (;;) {
    const hipError_t q = hipEventQuery(P.ev_fill);
    if (q == hipSuccess) break;
    if (q != hipErrorNotReady) return fail(GORIO_EDEVICE, "fill kernel failed: %s", hipGetErrorString(q));
    if (!timed_out && std::chrono::duration<double>(Clock::now() - t0).count() > limit_s) {
      timed_out = true;
      __atomic_store_n(P.h_abort, 1u, __ATOMIC_RELEASE);
    }
    std::this_thread::sleep_for(std::chrono::microseconds(50));
  }
  HIP_OR_FAIL(hipStreamWaitEvent(s, P.ev_fill, 0));
  for (int i = 1; i < flights; ++i) {
    HIP_OR_FAIL(hipEventRecord(P.ev_round[i], P.round_stream[i]));
    HIP_OR_FAIL(hipStreamWaitEvent(s, P.ev_round[i], 0));
  }
  HIP_OR_FAIL(hipEventRecord(ix->ev_stop, s));
  return st;
}

// GPU resume queue (mode 3): one persistent launch of fill waves and
// executor waves; the fill waves queue the lanes parked on the slots they
// fill and the executors run the queued lanes' turns (paged_queue).  The
// host only runs the proxy and the watchdog.
gorio_status run_gpu_queue(gorio_index *ix, PagedParams &pp, uint32_t lanes, hipStream_t s, double limit_s,
                           bool &timed_out) {
  PagedState &P = *ix->paged;
  const uint32_t words = lane_state_words(pp.L);
  if ((uint64_t)lanes * words > P.lane_state_words) {
    if (P.d_lane_state) (void)hipFree(P.d_lane_state);
    P.d_lane_state = nullptr;
    P.lane_state_words = 0;
    HIP_OR_FAIL(hipMalloc(&P.d_lane_state, (uint64_t)lanes * words * 4));
    P.lane_state_words = (uint64_t)lanes * words;
  }
  if (lanes > P.lane_out_q_cap) {
    if (P.d_lane_out_q) (void)hipFree(P.d_lane_out_q);
    P.d_lane_out_q = nullptr;
    P.lane_out_q_cap = 0;
    HIP_OR_FAIL(hipMalloc(&P.d_lane_out_q, (size_t)lanes * sizeof(LaneOut)));
    P.lane_out_q_cap = lanes;
  }
  // one buffer of 64-bit words: a waiter set per cache slot, the run queue,
  // its head, its tail and the lane counter (each on a 256-byte line of its
  // own), then the lanes' state words
  const uint32_t wset = (lanes + 63) / 64;
  uint32_t cap = 1;
  while (cap < 2 * lanes + 64) cap <<= 1;
  const uint64_t line = PagedState::kCtrlStride;
  const uint64_t o_rq = P.slots * (uint64_t)wset, o_ctl = o_rq + cap, o_st = o_ctl + 3 * line;
  const uint64_t total = o_st + (lanes + 1) / 2;
  if (total > P.queue_words) {
    if (P.d_queue) (void)hipFree(P.d_queue);
    P.d_queue = nullptr;
    P.queue_words = 0;
    HIP_OR_FAIL(hipMalloc(&P.d_queue, total * sizeof(unsigned long long)));
    P.queue_words = total;
  }
  fill_u32<<<grid_for(total * 2, 256), 256, 0, s>>>(reinterpret_cast<uint32_t *>(P.d_queue), total * 2, 0u);
  const uint64_t out_words = (uint64_t)lanes * sizeof(LaneOut) / 4;
  fill_u32<<<grid_for(out_words, 256), 256, 0, s>>>(reinterpret_cast<uint32_t *>(P.d_lane_out_q), out_words, 0u);
  HIP_OR_FAIL(hipGetLastError());
  RunQueue qp;
  qp.lanes = lanes;
  qp.words = wset;
  qp.waiters = P.d_queue;
  qp.rq = P.d_queue + o_rq;
  qp.rq_mask = cap - 1;
  qp.rq_head = P.d_queue + o_ctl;
  qp.rq_tail = P.d_queue + o_ctl + line;
  qp.next_lane = reinterpret_cast<unsigned int *>(P.d_queue + o_ctl + 2 * line);
  qp.lane_st = reinterpret_cast<uint32_t *>(P.d_queue + o_st);
  RoundParams rx = {};
  rx.state = P.d_lane_state;
  rx.state_words = words;
  rx.out = P.d_lane_out_q;
  rx.out_lanes = lanes;
  pp.fill_head = nullptr;
  pp.fill_budget = 0;
  pp.turn_passes = 0;  // a turn runs until the lane parks
  int cus = 0;
  HIP_OR_FAIL(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, ix->device));
  const int execs = (int)std::min<uint64_t>(lanes, (uint64_t)cus * 4);
  const int grid = (int)pp.fill_waves + execs;
  HIP_OR_FAIL(hipEventRecord(ix->ev_start, s));
  const hipError_t le = ix->dtype == GORIO_F32 ? launch_queue_f32(pp, rx, qp, grid, s)
                                               : launch_queue_u8(pp, rx, qp, grid, s);
  if (le != hipSuccess) return fail(GORIO_EDEVICE, "queue launch failed: %s", hipGetErrorString(le));
  const hipError_t re = hipEventRecord(ix->ev_stop, s);
  if (re != hipSuccess) {  // the launch leaves on the abort flag, before the proxy stops
    __atomic_store_n(P.h_abort, 1u, __ATOMIC_RELEASE);
    (void)hipStreamSynchronize(s);
    return fail(GORIO_EDEVICE, "hipEventRecord: %s", hipGetErrorString(re));
  }
  // watchdog: the waves poll the abort flag (through its device mirror)
  const auto t0 = std::chrono::steady_clock::now();
  for (;;) {
    const hipError_t q = hipEventQuery(ix->ev_stop);
    if (q == hipSuccess) break;
    if (q != hipErrorNotReady) return fail(GORIO_EDEVICE, "queue search failed: %s", hipGetErrorString(q));
    const double el = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
    if (!timed_out && el > limit_s) {
      timed_out = true;
      __atomic_store_n(P.h_abort, 1u, __ATOMIC_RELEASE);
    }
    std::this_thread::sleep_for(std::chrono::microseconds(200));
  }
  return GORIO_OK;
}

// Paged search: reset the per-search rings and counters, fill in the kernel
// parameters, arm the proxy, then run either the persistent kernel (GPU
// scheduler, split-phase or blocking) or host-scheduled lanes, under a
// watchdog.
gorio_status run_paged(gorio_index *ix, const ResidentParams &rp, hipStream_t s, bool &timed_out) {
  PagedState &P = *ix->paged;
  const bool host_rounds = ix->blocking == 2;
  const bool gpu_queue = ix->blocking == 3;
  const bool blocking = ix->blocking == 1;
  const bool lanes_mode = host_rounds || gpu_queue;  // query state in HBM, turns run by executors
  const uint32_t oversub = (blocking || lanes_mode) ? 1u : ix->oversub;
  int dev = 0, cus = 0;
  HIP_OR_FAIL(hipGetDevice(&dev));
  HIP_OR_FAIL(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  // concurrent queries: each may hold max_pending pins, kept within half the
  // cache so the clock always finds victims for the rest
  const uint32_t pend_dflt = ix->max_pending ? ix->max_pending : kMaxPendingPerQuery;
  const uint32_t max_pending = (uint32_t)std::max(1, std::min(256, env_int("GORIO_MAX_PENDING", (int)pend_dflt)));
  const uint64_t q_cache = std::max<uint64_t>(1, P.slots / (2ull * max_pending));
  const uint64_t wave_cap = ix->query_waves ? ix->query_waves : (uint64_t)cus * 8;
  const uint64_t q_live = std::min<uint64_t>({wave_cap * oversub, q_cache, rp.nq, lanes_mode ? 8192ull : ~0ull});
  // persistent kernel: query waves; host rounds: lanes
  const int qwaves = (int)std::max<uint64_t>(1, (q_live + oversub - 1) / oversub);
  // waves that only copy arriving pages, each from a completion ring of its
  // own, so the fill rate does not depend on how many queries run at once
  // and no two waves contend for completions (host rounds need them)
  int fwaves = std::max(0, std::min((int)PagedState::kMaxRings, env_int("GORIO_FILL_WAVES", 32)));
  if (lanes_mode) fwaves = std::max(fwaves, 1);
  const uint32_t rings = (uint32_t)std::max(1, fwaves);
  const uint64_t ht_entries = (uint64_t)qwaves * oversub << kPagedHtLog2;
  if (ht_entries > P.ht_pool_entries) {
    if (P.d_ht_pool) (void)hipFree(P.d_ht_pool);
    P.d_ht_pool = nullptr;
    P.ht_pool_entries = 0;
    HIP_OR_FAIL(hipMalloc(&P.d_ht_pool, ht_entries * sizeof(uint32_t)));
    P.ht_pool_entries = ht_entries;
  }
  // per-search reset: rings empty, indices zero (the clock hand and the cached
  // pages stay: a warm cache carries over to the next search)
  memset(P.h_mq, 0, P.ring_cap * sizeof(unsigned long long));
  for (uint32_t r = 0; r < rings; ++r) __atomic_store_n(P.h_cq_tail + (size_t)r * PagedState::kTailStride, 0ull, __ATOMIC_RELEASE);
  __atomic_store_n(P.h_abort, 0u, __ATOMIC_RELEASE);
  fill_u32<<<1, 256, 0, s>>>(reinterpret_cast<uint32_t *>(P.ctrl(PagedState::kMqTail)),
                             2 * (PagedState::kCtrlWords - PagedState::kMqTail) * PagedState::kCtrlStride, 0u);

  PagedParams pp;
  pp.cache.data = P.d_cache;
  pp.cache.slot_word = P.d_slot_word;
  pp.cache.page_slot = P.d_page_slot;
  pp.cache.clock_hand = P.ctrl(PagedState::kClock);
  pp.cache.slots = (uint32_t)P.slots;
  pp.cache.page_bytes = ix->page_bytes;
  pp.cache.mq = P.d_mq;
  pp.cache.mq_mask = P.ring_cap - 1;
  pp.cache.mq_tail = P.ctrl(PagedState::kMqTail);
  pp.geom = rp.geom;
  pp.n = rp.n;
  pp.D = rp.D;
  pp.R = rp.R;
  pp.Rdiv = rp.Rdiv;
  pp.entry = rp.entry;
  pp.num_pages = (uint32_t)ix->num_pages;
  uint8_t *d_backing = nullptr;
  HIP_OR_FAIL(hipHostGetDevicePointer(reinterpret_cast<void **>(&d_backing), ix->h_backing, 0));
  pp.backing = d_backing;
  pp.cq = P.d_cq;
  pp.cq_mask = P.cq_cap - 1;
  pp.cq_tail = P.d_cq_tail;
  pp.tail_stride = PagedState::kTailStride;
  pp.cq_head = P.ctrl(PagedState::kCqHead);
  pp.tail_seen = P.ctrl(PagedState::kTailSeen);
  pp.poll_lock = reinterpret_cast<unsigned int *>(P.ctrl(PagedState::kPollLock));
  pp.abort_flag = P.d_abort;
  pp.abort_seen = reinterpret_cast<unsigned int *>(P.ctrl(PagedState::kAbortSeen));
  pp.queries = rp.queries;
  pp.nq = rp.nq;
  pp.k = rp.k;
  pp.L = rp.L;
  pp.W = rp.W;
  pp.next_query = reinterpret_cast<unsigned int *>(P.ctrl(PagedState::kNextQuery));
  // admission order: cluster by cluster of the queries' nearest centroids
  DevBuf d_key, d_order;
  std::vector<uint32_t> order;
  pp.order = nullptr;
  if (ix->order_clusters > 0) {
    HIP_OR_FAIL(d_key.alloc((size_t)rp.nq * 4));
    HIP_OR_FAIL(d_order.alloc((size_t)rp.nq * 4));
    HIP_OR_FAIL(launch_nearest_centroid(ix->dtype, rp.queries, rp.nq, ix->D, ix->d_centroids, ix->d_centroid_norms,
                                        ix->order_clusters, d_key.as<uint32_t>(), s));
    std::vector<uint32_t> key(rp.nq);
    order.resize(rp.nq);
    HIP_OR_FAIL(hipMemcpyAsync(key.data(), d_key.p, (size_t)rp.nq * 4, hipMemcpyDeviceToHost, s));
    HIP_OR_FAIL(hipStreamSynchronize(s));
    order_by_key(key.data(), rp.nq, ix->order_clusters, order.data());
    HIP_OR_FAIL(hipMemcpyAsync(d_order.p, order.data(), (size_t)rp.nq * 4, hipMemcpyHostToDevice, s));
    pp.order = d_order.as<uint32_t>();
  }
  pp.done_queries = reinterpret_cast<unsigned int *>(P.ctrl(PagedState::kDoneQueries));
  pp.fill_head = nullptr;
  pp.fill_budget = 0;  // host rounds set their own
  pp.fill_waves = (uint32_t)fwaves;
  pp.out_ids = rp.out_ids;
  pp.out_dists = rp.out_dists;
  pp.ht_pool = P.d_ht_pool;
  pp.oversub = oversub;
  pp.max_pending = max_pending;
  pp.blocking = blocking ? 1 : 0;
  pp.turn_passes = 0;  // host rounds set their own
  pp.stats = rp.stats;

  // test hooks: random extra delay per request (completions leave out of
  // order) and a proxy that never completes (the watchdog must end the search)
  const char *jit = getenv("GORIO_PROXY_JITTER_US");
  P.proxy.begin(ix->latency_us, ix->max_outstanding, rings, jit ? atof(jit) : 0.0,
                env_int("GORIO_PROXY_HOLD", 0) != 0);
  const double limit_s = env_int("GORIO_WATCHDOG_S", 120);
  gorio_status st = GORIO_OK;
  if (host_rounds) {
    st = run_host_rounds(ix, pp, (uint32_t)q_live, order, s, limit_s, timed_out);
  } else if (gpu_queue) {
    st = run_gpu_queue(ix, pp, (uint32_t)q_live, s, limit_s, timed_out);
  } else {
    const int grid = qwaves + fwaves;
    HIP_OR_FAIL(hipEventRecord(ix->ev_start, s));
    const hipError_t le = ix->dtype == GORIO_F32 ? launch_paged_f32(pp, grid, s) : launch_paged_u8(pp, grid, s);
    if (le != hipSuccess) {
      P.proxy.end();
      return fail(GORIO_EDEVICE, "paged search launch failed: %s", hipGetErrorString(le));
    }
    const hipError_t re = hipEventRecord(ix->ev_stop, s);
    if (re != hipSuccess) {  // the kernel leaves on the abort flag, before the proxy stops
      __atomic_store_n(P.h_abort, 1u, __ATOMIC_RELEASE);
      (void)hipStreamSynchronize(s);
      P.proxy.end();
      (void)ix->reset_cache();
      return fail(GORIO_EDEVICE, "hipEventRecord: %s", hipGetErrorString(re));
    }
    // watchdog: the kernel polls the abort flag (through its device mirror)
    const auto t0 = std::chrono::steady_clock::now();
    for (;;) {
      hipError_t q = hipEventQuery(ix->ev_stop);
      if (q == hipSuccess) break;
      if (q != hipErrorNotReady) {
        P.proxy.end();
        (void)ix->reset_cache();
        return fail(GORIO_EDEVICE, "paged search failed: %s", hipGetErrorString(q));
      }
      const double el = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
      if (!timed_out && el > limit_s) {
        timed_out = true;
        __atomic_store_n(P.h_abort, 1u, __ATOMIC_RELEASE);
      }
      std::this_thread::sleep_for(std::chrono::microseconds(200));
    }
  }
  P.proxy.end();
  if (st != GORIO_OK) {
    // a search that failed part way leaves pins and LOADING slots behind, as an
    // aborted one does; the first error is the one reported
    const std::string msg = gorio_last_error();
    (void)ix->reset_cache();
    return fail(st, "%s", msg.c_str());
  }
  if (timed_out) {
    gorio_status rs = ix->reset_cache();  // pins and LOADING slots of aborted queries
    if (rs != GORIO_OK) return rs;
  }
  return GORIO_OK;
}

}  // namespace

extern "C" gorio_status gorio_search(gorio_index *ix, const void *queries, uint64_t nq, uint32_t k,
                                     uint32_t L, uint32_t W, uint32_t *ids, void *dists,
                                     gorio_stats *stats, void *stream) {
  const auto t0 = std::chrono::steady_clock::now();
  if (!ix) return fail(GORIO_EINVAL, "index is NULL");
  if (k == 0 || L < k || L > 256) return fail(GORIO_EINVAL, "need 1 <= k <= L <= 256 (k=%u L=%u)", k, L);
  if (W == 0 || W > L) return fail(GORIO_EINVAL, "need 1 <= W <= L (W=%u L=%u)", W, L);
  if (nq >= (1ull << 31)) return fail(GORIO_EINVAL, "nq=%llu too large", (unsigned long long)nq);
  if (stats) memset(stats, 0, sizeof *stats);
  if (nq == 0) return GORIO_OK;
  if (!queries || !ids || !dists) return fail(GORIO_EINVAL, "queries, ids and dists must be non-NULL");
  if (!ix->resident && W > (uint32_t)kPagedMaxW)
    return fail(GORIO_EUNSUPPORTED, "paged search supports W <= %d (W=%u)", kPagedMaxW, W);

  DeviceGuard dg(ix->device);
  if (!dg.ok) return fail(GORIO_EDEVICE, "cannot select device %d", ix->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  {
    // each search takes its query tickets from a base kept on the host, so a
    // captured search would replay with a stale base
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    HIP_OR_FAIL(hipStreamIsCapturing(s, &cap));
    if (cap != hipStreamCaptureStatusNone)
      return fail(GORIO_EUNSUPPORTED, "gorio_search cannot be captured into a graph; use gorio_search_noalloc");
  }

  const size_t qbytes = (size_t)nq * ix->vec_bytes;
  const size_t obytes = (size_t)nq * k * 4;
  const bool q_dev = is_device_pointer(queries);
  const bool i_dev = is_device_pointer(ids);
  const bool d_dev = is_device_pointer(dists);
  const void *d_q = queries;
  uint32_t *d_ids = ids;
  void *d_dists = dists;
  if (!q_dev || !i_dev || !d_dev) {
    // host buffers go through the index's staging buffer (grown when a batch
    // needs more; the last search that used it has returned, so it is idle)
    auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
    const size_t need = (q_dev ? 0 : up(qbytes)) + (i_dev ? 0 : up(obytes)) + (d_dev ? 0 : up(obytes));
    if (need > ix->stage_bytes) {
      if (ix->d_stage) (void)hipFree(ix->d_stage);
      ix->d_stage = nullptr;
      ix->stage_bytes = 0;
      HIP_OR_FAIL(hipMalloc(&ix->d_stage, need));
      ix->stage_bytes = need;
    }
    uint8_t *at = ix->d_stage;
    if (!q_dev) {
      HIP_OR_FAIL(hipMemcpyAsync(at, queries, qbytes, hipMemcpyHostToDevice, s));
      d_q = at;
      at += up(qbytes);
    }
    if (!i_dev) {
      d_ids = reinterpret_cast<uint32_t *>(at);
      at += up(obytes);
    }
    if (!d_dev) d_dists = at;
  }

  // the previous search of this index finishes before this one uses the
  // counters they share: by stream order, or by waiting for the event it
  // recorded last
  if (ix->ev_done_recorded && !follows_last_search(ix, s)) HIP_OR_FAIL(hipStreamWaitEvent(s, ix->ev_done, 0));
  // the counters only grow; a search that reports them reports the growth
  if (stats)
    HIP_OR_FAIL(hipMemcpyAsync(ix->d_stats + kStatWords, ix->d_stats, kStatWords * sizeof(unsigned long long),
                               hipMemcpyDeviceToDevice, s));

  ResidentParams p;
  p.pages = ix->d_pages;
  p.geom = ix->geom();
  p.n = (uint32_t)ix->n;
  p.D = ix->D;
  p.R = ix->R;
  p.Rdiv = make_fastdiv(ix->R);
  p.entry = ix->entry;
  p.queries = d_q;
  p.nq = (uint32_t)nq;
  p.k = k;
  p.L = L;
  p.W = W;
  p.out_ids = d_ids;
  p.out_dists = static_cast<uint32_t *>(d_dists);
  p.stats = ix->d_stats;
  p.next_query = ix->d_stats + kStatNextQuery;
  p.next_base = ix->next_base;

  gorio_status st;
  bool timed_out = false;
  if (ix->resident) {
    const int grid = (int)std::min<uint64_t>(nq, 1u << 30);
    if (stats) HIP_OR_FAIL(hipEventRecord(ix->ev_start, s));
    HIP_OR_FAIL(ix->dtype == GORIO_F32 ? launch_resident_f32(p, grid, s) : launch_resident_u8(p, grid, s));
    ix->next_base += nq;  // every query takes one ticket
    if (stats) HIP_OR_FAIL(hipEventRecord(ix->ev_stop, s));
  } else {
    st = run_paged(ix, p, s, timed_out);
    if (st != GORIO_OK) return st;
  }

  if (!i_dev) HIP_OR_FAIL(hipMemcpyAsync(ids, d_ids, obytes, hipMemcpyDeviceToHost, s));
  if (!d_dev) HIP_OR_FAIL(hipMemcpyAsync(dists, d_dists, obytes, hipMemcpyDeviceToHost, s));
  unsigned long long h_cnt[2 * kStatWords] = {};  // counters after, then before
  if (stats) HIP_OR_FAIL(hipMemcpyAsync(h_cnt, ix->d_stats, sizeof h_cnt, hipMemcpyDeviceToHost, s));
  HIP_OR_FAIL(hipEventRecord(ix->ev_done, s));
  ix->ev_done_recorded = true;
  ix->last_stream = s;
  if (stats || !i_dev || !d_dev || !q_dev) HIP_OR_FAIL(hipStreamSynchronize(s));
  if (stats) {
    float ms = 0.f;
    HIP_OR_FAIL(hipEventElapsedTime(&ms, ix->ev_start, ix->ev_stop));
    stats->kernel_ms = ms;
    auto grown = [&](int w) { return h_cnt[w] - h_cnt[kStatWords + w]; };
    stats->evaluations = grown(kStatEval);
    stats->reevaluations = grown(kStatReeval);
    stats->expansions = grown(kStatExp);
    stats->iterations = grown(kStatIter);
    stats->hits = grown(kStatHit);
    stats->misses = grown(kStatMiss);
    stats->pages_served = grown(kStatServed);
    stats->bytes_served = grown(kStatServed) * ix->page_bytes;
    stats->parks = grown(kStatPark);
    stats->resumes = grown(kStatResume);
    stats->proxy_peak = ix->paged ? ix->paged->proxy.max_in_flight() : 0;
    stats->wall_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
  }
  if (timed_out) return fail(GORIO_ETIMEOUT, "paged search did not finish within the watchdog limit");
  return GORIO_OK;
}

// ---------------------------------------------------------------------------
// info / pages / free
// ---------------------------------------------------------------------------
extern "C" gorio_status gorio_index_info_get(const gorio_index *ix, gorio_index_info *info) {
  if (!ix || !info) return fail(GORIO_EINVAL, "NULL argument");
  info->dtype = ix->dtype;
  info->n = ix->n;
  info->D = ix->D;
  info->R = ix->R;
  info->page_bytes = ix->page_bytes;
  info->record_bytes = ix->rec_bytes;
  info->records_per_page = ix->rpp;
  info->vectors_first = ix->vectors_first ? 1 : 0;
  info->num_pages = ix->num_pages;
  info->index_bytes = ix->index_bytes();
  info->entry = ix->entry;
  info->resident = ix->resident ? 1 : 0;
  info->cache_slots = ix->resident ? ix->num_pages : ix->cache_slots;
  info->device = ix->device;
  return GORIO_OK;
}

extern "C" gorio_status gorio_copy_pages(const gorio_index *ix, uint64_t first, uint64_t count, void *dst) {
  if (!ix || (!dst && count)) return fail(GORIO_EINVAL, "NULL argument");
  if (first > ix->num_pages || count > ix->num_pages - first) return fail(GORIO_EINVAL, "page range out of bounds");
  if (count == 0) return GORIO_OK;
  DeviceGuard dg(ix->device);
  const size_t off = first * ix->page_bytes, bytes = count * ix->page_bytes;
  if (ix->resident) {
    HIP_OR_FAIL(hipMemcpy(dst, ix->d_pages + off, bytes, hipMemcpyDeviceToHost));
  } else {
    memcpy(dst, ix->h_backing + off, bytes);
  }
  return GORIO_OK;
}

extern "C" void gorio_free_index(gorio_index *ix) {
  if (!ix) return;
  {
    DeviceGuard dg(ix->device);
    ix->release_all();
  }
  delete ix;
}
