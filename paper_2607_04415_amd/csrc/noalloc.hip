// gorio_search_noalloc: the resident search for callers that cannot allocate
// device memory.  Its only scratch memory (the kernel's counters and its query
// counter) is a file-scope device array, one copy per GPU.
#include <hip/hip_runtime.h>

#include <cstring>
#include <mutex>

#include "../../include/gorio.h"
#include "index.hpp"
#include "launch.hpp"

using namespace gorio;

namespace {

// Scratch of every gorio_search_noalloc call on a GPU: kStatWords 64-bit
// words (128 bytes) -- the resident kernel's statistics and the counter that
// hands out queries past the first grid.  The size does not depend on the
// batch.  Host code never uses this name as an address: it takes the per-device
// address that hipGetSymbolAddress returns.
constexpr uint32_t kScratchWords = kStatWords;
__device__ __align__(256) unsigned long long scratch[kScratchWords];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned long long *g_scratch[kMaxDevices] = {};

// Device address of `scratch` on device `dev` (current), looked up on the
// first call on that device and kept.
gorio_status scratch_of(int dev, unsigned long long **out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(GORIO_EUNSUPPORTED, "device %d above %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(GORIO_EDEVICE, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch[dev] = static_cast<unsigned long long *>(ptr);
  }
  *out = g_scratch[dev];
  return GORIO_OK;
}

// Zero the scratch words before a search (a kernel, not a memset node).
__global__ void zero_words(unsigned long long *w, uint32_t n) {
  for (uint32_t i = threadIdx.x; i < n; i += blockDim.x) w[i] = 0ull;
}

bool on_device(const void *ptr) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, ptr) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeDevice || a.isManaged;
}

}  // namespace

extern "C" gorio_status gorio_search_noalloc(gorio_index *ix, const void *queries, uint64_t nq, uint32_t k,
                                             uint32_t L, uint32_t W, uint32_t *ids, void *dists,
                                             gorio_stats *stats, void *stream) {
  if (!ix) return fail(GORIO_EINVAL, "index is NULL");
  if (k == 0 || L < k || L > 256) return fail(GORIO_EINVAL, "need 1 <= k <= L <= 256 (k=%u L=%u)", k, L);
  if (W == 0 || W > L) return fail(GORIO_EINVAL, "need 1 <= W <= L (W=%u L=%u)", W, L);
  if (nq >= (1ull << 31)) return fail(GORIO_EINVAL, "nq=%llu too large", (unsigned long long)nq);
  if (stats) memset(stats, 0, sizeof *stats);
  if (nq == 0) return GORIO_OK;
  if (!ix->resident)
    return fail(GORIO_EUNSUPPORTED, "gorio_search_noalloc runs resident indexes only (this one is paged)");
  if (!queries || !ids || !dists) return fail(GORIO_EINVAL, "queries, ids and dists must be non-NULL");

  int prev = -1;
  if (hipGetDevice(&prev) != hipSuccess) return fail(GORIO_EDEVICE, "hipGetDevice failed");
  if (prev != ix->device && hipSetDevice(ix->device) != hipSuccess)
    return fail(GORIO_EDEVICE, "cannot select device %d", ix->device);
  struct Restore {
    int prev, dev;
    ~Restore() { if (prev >= 0 && prev != dev) (void)hipSetDevice(prev); }
  } restore{prev, ix->device};

  if (!on_device(queries) || !on_device(ids) || !on_device(dists))
    return fail(GORIO_EINVAL, "gorio_search_noalloc needs device pointers for queries, ids and dists");
  unsigned long long *sc = nullptr;
  gorio_status st = scratch_of(ix->device, &sc);
  if (st != GORIO_OK) return st;

  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipSuccess;
#define NOALLOC_HIP(expr)                                                                   \
  do {                                                                                      \
    e = (expr);                                                                             \
    if (e != hipSuccess) return fail(GORIO_EDEVICE, "%s: %s", #expr, hipGetErrorString(e)); \
  } while (0)
  // Under graph capture the graph orders the work: no event is recorded or
  // waited for (the caller orders replays with its other work), and no
  // statistics (they need a synchronisation).  Otherwise the call follows
  // the previous search of this index, as gorio_search does.
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  NOALLOC_HIP(hipStreamIsCapturing(s, &cap));
  const bool capturing = cap != hipStreamCaptureStatusNone;
  if (capturing && stats)
    return fail(GORIO_EINVAL, "gorio_search_noalloc under graph capture takes no statistics (pass NULL)");
  if (!capturing && ix->ev_done_recorded && !follows_last_search(ix, s))
    NOALLOC_HIP(hipStreamWaitEvent(s, ix->ev_done, 0));
  zero_words<<<1, 64, 0, s>>>(sc, kScratchWords);
  NOALLOC_HIP(hipGetLastError());

  ResidentParams p;
  p.pages = ix->d_pages;
  p.geom = ix->geom();
  p.n = (uint32_t)ix->n;
  p.D = ix->D;
  p.R = ix->R;
  p.Rdiv = make_fastdiv(ix->R);
  p.entry = ix->entry;
  p.queries = queries;
  p.nq = (uint32_t)nq;
  p.k = k;
  p.L = L;
  p.W = W;
  p.out_ids = ids;
  p.out_dists = static_cast<uint32_t *>(dists);
  p.stats = sc;
  p.next_query = sc + kStatNextQuery;
  p.next_base = 0;  // cleared above
  const int grid = (int)std::min<uint64_t>(nq, 1u << 30);
  if (stats) NOALLOC_HIP(hipEventRecord(ix->ev_start, s));
  NOALLOC_HIP(ix->dtype == GORIO_F32 ? launch_resident_f32(p, grid, s) : launch_resident_u8(p, grid, s));
  if (stats) NOALLOC_HIP(hipEventRecord(ix->ev_stop, s));
  unsigned long long h[kScratchWords] = {};
  if (stats) NOALLOC_HIP(hipMemcpyAsync(h, sc, sizeof h, hipMemcpyDeviceToHost, s));
  if (!capturing) {
    NOALLOC_HIP(hipEventRecord(ix->ev_done, s));
    ix->ev_done_recorded = true;
    ix->last_stream = s;
  }
  if (stats) {
    NOALLOC_HIP(hipStreamSynchronize(s));
    float ms = 0.f;
    NOALLOC_HIP(hipEventElapsedTime(&ms, ix->ev_start, ix->ev_stop));
    stats->kernel_ms = ms;
    stats->evaluations = h[kStatEval];
    stats->reevaluations = h[kStatReeval];
    stats->expansions = h[kStatExp];
    stats->iterations = h[kStatIter];
  }
#undef NOALLOC_HIP
  return GORIO_OK;
}
