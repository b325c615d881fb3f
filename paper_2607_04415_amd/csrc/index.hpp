// The library-owned index object behind gorio_index*.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdint>
#include <memory>

#include "../../include/gorio.h"
#include "common.hpp"

namespace gorio {

gorio_status fail(gorio_status st, const char *fmt, ...);

enum StatWord : int {
  kStatEval = 0,
  kStatReeval,
  kStatExp,
  kStatIter,
  kStatHit,
  kStatMiss,
  kStatServed,
  kStatPark,
  kStatResume,
  kStatWords = 16
};

}  // namespace gorio

struct gorio_index {
  int device = 0;
  gorio_dtype dtype = GORIO_U8;
  uint64_t n = 0;
  uint32_t D = 0, R = 0, vec_bytes = 0;
  uint32_t page_bytes = 4096, rec_bytes = 0, rpp = 0;
  uint64_t num_pages = 0;
  uint32_t entry = 0;
  uint32_t *d_node_to_slot = nullptr;

  bool resident = true;
  uint8_t *d_pages = nullptr;    // resident mode: packed pages in HBM
  uint8_t *h_backing = nullptr;  // paged mode: packed pages in pinned host memory
  uint64_t cache_slots = 0;

  double latency_us = 0.0;
  uint32_t max_outstanding = 4096;
  uint32_t oversub = 1;
  int blocking = 0;

  hipStream_t stream = nullptr;  // library-internal work (build, mode switches)
  hipEvent_t ev_start = nullptr, ev_stop = nullptr;
  unsigned long long *d_stats = nullptr;

  uint64_t index_bytes() const { return num_pages * (uint64_t)page_bytes; }

  gorio::PageGeom geom() const {
    gorio::PageGeom g;
    g.page_bytes = page_bytes;
    g.record_bytes = rec_bytes;
    g.vec_bytes = vec_bytes;
    g.rpp = gorio::make_fastdiv(rpp);
    g.node_to_slot = d_node_to_slot;
    return g;
  }

  // All pages to HBM (from the backing store if paged).
  gorio_status make_resident() {
    if (resident) return GORIO_OK;
    hipError_t e = hipMalloc(&d_pages, index_bytes());
    if (e != hipSuccess) return gorio::fail(GORIO_ENOMEM, "hipMalloc of %llu page bytes failed",
                                            (unsigned long long)index_bytes());
    e = hipMemcpy(d_pages, h_backing, index_bytes(), hipMemcpyHostToDevice);
    if (e != hipSuccess) return gorio::fail(GORIO_EDEVICE, "page upload failed: %s", hipGetErrorString(e));
    (void)hipHostFree(h_backing);
    h_backing = nullptr;
    cache_slots = 0;
    resident = true;
    return GORIO_OK;
  }

  // Pages to the pinned host backing store; the HBM copy is released.
  gorio_status make_paged(uint64_t slots) {
    if (slots == 0) return gorio::fail(GORIO_EINVAL, "a paged cache needs at least one slot");
    if (resident) {
      hipError_t e = hipHostMalloc(reinterpret_cast<void **>(&h_backing), index_bytes(), hipHostMallocDefault);
      if (e != hipSuccess) return gorio::fail(GORIO_ENOMEM, "pinned backing store of %llu bytes failed",
                                              (unsigned long long)index_bytes());
      e = hipMemcpy(h_backing, d_pages, index_bytes(), hipMemcpyDeviceToHost);
      if (e != hipSuccess) return gorio::fail(GORIO_EDEVICE, "page download failed: %s", hipGetErrorString(e));
      (void)hipFree(d_pages);
      d_pages = nullptr;
      resident = false;
    }
    cache_slots = slots;
    return GORIO_OK;
  }

  void release_all() {
    if (d_pages) (void)hipFree(d_pages);
    if (h_backing) (void)hipHostFree(h_backing);
    if (d_node_to_slot) (void)hipFree(d_node_to_slot);
    if (d_stats) (void)hipFree(d_stats);
    if (ev_start) (void)hipEventDestroy(ev_start);
    if (ev_stop) (void)hipEventDestroy(ev_stop);
    if (stream) (void)hipStreamDestroy(stream);
    d_pages = nullptr;
    h_backing = nullptr;
    d_node_to_slot = nullptr;
    d_stats = nullptr;
    ev_start = ev_stop = nullptr;
    stream = nullptr;
  }
};
