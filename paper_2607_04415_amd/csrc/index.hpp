// The library-owned index object behind gorio_index*.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdint>
#include <memory>

#include "../../include/gorio.h"
#include "common.hpp"
#include "proxy.hpp"

namespace gorio {

gorio_status fail(gorio_status st, const char *fmt, ...);

struct LaneOut;  // search_paged.hpp: a host-scheduled lane's report

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
  kStatNextQuery,  // resident kernel: query tickets (grows by nq per launch)
  kStatMalformed,  // paged kernel: completion entries it could not use
  kStatWords = 16
};

// Device and host memory of the paged mode (one per index, sized by set_cache).
struct PagedState {
  uint64_t slots = 0;
  uint8_t *d_cache = nullptr;                 // slots * page_bytes
  unsigned long long *d_slot_word = nullptr;  // slots
  uint32_t *d_page_slot = nullptr;            // num_pages
  // device control words (one allocation): clock hand, descriptor tail, shared
  // completion head and tail mirror, poll lock, abort mirror, next query (or,
  // for host-scheduled lanes, run-ring entries taken), finished queries,
  // run-ring tail mirror
  unsigned long long *d_ctrl = nullptr;
  // host rings (coherent pinned memory) and their device-visible addresses
  unsigned long long *h_mq = nullptr, *d_mq = nullptr;
  unsigned long long *h_cq = nullptr, *d_cq = nullptr;
  unsigned long long *h_cq_tail = nullptr, *d_cq_tail = nullptr;
  unsigned int *h_abort = nullptr, *d_abort = nullptr;
  uint32_t ring_cap = 0;   // descriptor ring entries
  uint32_t cq_cap = 0;     // entries of each completion ring
  // completion rings: one per fill wave (or one shared ring when query waves
  // serve completions themselves); tails 128 bytes apart
  static constexpr uint32_t kMaxRings = 64;
  static constexpr uint32_t kTailStride = 16;  // u64 words
  uint32_t *d_ht_pool = nullptr;
  uint64_t ht_pool_entries = 0;
  // host-scheduled lanes: lane states (HBM), the round's lane list and the
  // lanes' reports (host memory the kernels read and write), and how far each
  // completion ring has been filled (written by the fill waves)
  // round kernels in flight at once: flight 0 on the search's stream, flight
  // i > 0 on round_stream[i]
  static constexpr int kMaxFlights = 8;
  hipStream_t fill_stream = nullptr, round_stream[kMaxFlights] = {};
  hipEvent_t ev_round[kMaxFlights] = {}, ev_fill = nullptr;
  uint32_t *d_lane_state = nullptr;
  uint64_t lane_state_words = 0;
  uint32_t *h_round = nullptr, *d_round = nullptr;   // 2 x round_cap: lanes, then admissions
  uint32_t round_cap = 0;
  LaneOut *h_lane_out = nullptr, *d_lane_out = nullptr;
  unsigned long long *h_fill_head = nullptr, *d_fill_head = nullptr;
  // host-scheduled lanes run by a persistent launch: the run ring the host
  // writes and the kernel reads, and its tail (entries written)
  unsigned long long *h_runq = nullptr, *d_runq = nullptr;
  uint32_t runq_cap = 0;
  unsigned long long *h_runq_ctl = nullptr, *d_runq_ctl = nullptr;
  // GPU resume queue: waiter sets, run queue, its counters and the lanes'
  // states in one device buffer, and the lanes' reports in HBM
  unsigned long long *d_queue = nullptr;
  uint64_t queue_words = 0;
  LaneOut *d_lane_out_q = nullptr;
  uint32_t lane_out_q_cap = 0;
  Proxy proxy;

  enum Ctrl {
    kClock = 0, kMqTail, kCqHead, kTailSeen, kPollLock, kAbortSeen, kNextQuery, kDoneQueries, kRunqTailSeen,
    kCtrlWords = 9
  };
  // each control word on its own 256-byte line: they are hot atomics of
  // different waves and must not serialize on one L2 channel
  static constexpr uint32_t kCtrlStride = 32;  // u64 words
  uint32_t ctrl_stride = kCtrlStride;
  unsigned long long *ctrl(int w) const { return d_ctrl + (size_t)w * ctrl_stride; }

  void release() {
    proxy.stop();
    if (d_cache) (void)hipFree(d_cache);
    if (d_slot_word) (void)hipFree(d_slot_word);
    if (d_page_slot) (void)hipFree(d_page_slot);
    if (d_ctrl) (void)hipFree(d_ctrl);
    if (d_ht_pool) (void)hipFree(d_ht_pool);
    if (d_lane_state) (void)hipFree(d_lane_state);
    if (h_round) (void)hipHostFree(h_round);
    if (h_lane_out) (void)hipHostFree(h_lane_out);
    if (h_fill_head) (void)hipHostFree(h_fill_head);
    if (h_runq) (void)hipHostFree(h_runq);
    if (h_runq_ctl) (void)hipHostFree(h_runq_ctl);
    if (d_queue) (void)hipFree(d_queue);
    if (d_lane_out_q) (void)hipFree(d_lane_out_q);
    if (fill_stream) (void)hipStreamDestroy(fill_stream);
    for (hipStream_t &r : round_stream)
      if (r) (void)hipStreamDestroy(r);
    for (hipEvent_t &e : ev_round)
      if (e) (void)hipEventDestroy(e);
    if (ev_fill) (void)hipEventDestroy(ev_fill);
    if (h_mq) (void)hipHostFree(h_mq);
    if (h_cq) (void)hipHostFree(h_cq);
    if (h_cq_tail) (void)hipHostFree(h_cq_tail);
    if (h_abort) (void)hipHostFree(h_abort);
    d_cache = nullptr;
    d_slot_word = nullptr;
    d_page_slot = nullptr;
    d_ctrl = nullptr;
    d_ht_pool = nullptr;
    d_lane_state = nullptr;
    lane_state_words = 0;
    h_round = d_round = nullptr;
    round_cap = 0;
    h_lane_out = d_lane_out = nullptr;
    h_fill_head = d_fill_head = nullptr;
    h_runq = d_runq = nullptr;
    runq_cap = 0;
    h_runq_ctl = d_runq_ctl = nullptr;
    d_queue = nullptr;
    queue_words = 0;
    d_lane_out_q = nullptr;
    lane_out_q_cap = 0;
    fill_stream = nullptr;
    for (int i = 0; i < kMaxFlights; ++i) {
      round_stream[i] = nullptr;
      ev_round[i] = nullptr;
    }
    ev_fill = nullptr;
    h_mq = d_mq = h_cq = d_cq = h_cq_tail = d_cq_tail = nullptr;
    h_abort = d_abort = nullptr;
    slots = 0;
    ring_cap = 0;
    cq_cap = 0;
    ht_pool_entries = 0;
  }
  ~PagedState() { release(); }
};

}  // namespace gorio

struct gorio_index {
  int device = 0;
  gorio_dtype dtype = GORIO_U8;
  uint64_t n = 0;
  uint32_t D = 0, R = 0, vec_bytes = 0;
  uint32_t page_bytes = 4096, rec_bytes = 0, rpp = 0;
  bool vectors_first = false;   // page layout: all vectors of a page, then all adjacency blocks
  uint64_t num_pages = 0;
  uint32_t entry = 0;
  uint32_t *d_node_to_slot = nullptr;

  bool resident = true;
  uint8_t *d_pages = nullptr;    // resident mode: packed pages in HBM
  uint8_t *h_backing = nullptr;  // paged mode: packed pages in pinned host memory
  uint64_t cache_slots = 0;

  std::unique_ptr<gorio::PagedState> paged;

  double latency_us = 0.0;
  uint32_t max_outstanding = 4096;
  uint32_t oversub = 1;
  int blocking = 0;
  // paged scheduler shape (gorio_set_scheduler); 0 = the library's choice
  uint32_t query_waves = 0;   // waves that run queries
  uint32_t max_pending = 0;   // page requests one query keeps outstanding

  // paged searches admit their queries cluster by cluster (gorio_set_query_order)
  uint32_t order_clusters = 0;
  float *d_centroids = nullptr;       // order_clusters x D float32
  float *d_centroid_norms = nullptr;  // order_clusters

  hipStream_t stream = nullptr;  // library-internal work (build, mode switches)
  hipEvent_t ev_start = nullptr, ev_stop = nullptr;
  // Recorded after the last operation of every search on the stream it used.
  // The next search makes its own stream wait for it, so searches of one index
  // issued on different streams never share the counters below at once.
  hipEvent_t ev_done = nullptr;
  bool ev_done_recorded = false;
  hipStream_t last_stream = nullptr;  // stream of the last search (its ev_done)
  // Counters (kStatWords 64-bit words) that only grow, then a snapshot of
  // them taken before a search that reports statistics (it reports the
  // difference).  next_base is the query-ticket counter's value when the next
  // resident launch starts.
  unsigned long long *d_stats = nullptr;
  uint64_t next_base = 0;
  // device staging for searches handed host buffers: grow-only, used by one
  // search at a time (such a search returns only after its copies)
  uint8_t *d_stage = nullptr;
  size_t stage_bytes = 0;

  uint64_t index_bytes() const { return num_pages * (uint64_t)page_bytes; }

  gorio::PageGeom geom() const {
    gorio::PageGeom g;
    g.page_bytes = page_bytes;
    g.record_bytes = rec_bytes;
    g.vec_bytes = vec_bytes;
    if (vectors_first) {
      g.vec_stride = (vec_bytes + 15u) & ~15u;
      g.adj_base = rpp * g.vec_stride;
      g.adj_stride = rec_bytes - g.vec_stride;
    } else {
      g.vec_stride = rec_bytes;
      g.adj_base = vec_bytes;
      g.adj_stride = rec_bytes;
    }
    g.rpp = gorio::make_fastdiv(rpp);
    g.node_to_slot = d_node_to_slot;
    // a buffer instruction's offset (index x stride) is a 32-bit byte offset:
    // locators address at most the first 4 GiB of the pages
    const uint64_t units = index_bytes() / 16;
    const bool loc16 = g.vec_stride % 16 == 0 && page_bytes % 16 == 0 && index_bytes() <= (1ull << 32);
    g.units16 = loc16 ? (uint32_t)units : 0u;
    g.page16 = gorio::make_fastdiv(loc16 ? page_bytes / 16 : 1u);
    g.vec16 = gorio::make_fastdiv(loc16 ? g.vec_stride / 16 : 1u);
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
    if (paged) paged->release();
    paged.reset();
    cache_slots = 0;
    resident = true;
    return GORIO_OK;
  }

  // Pages to the pinned host backing store (the HBM copy is released) and an
  // empty HBM cache of `slots` pages.  Defined in gorio.hip.
  gorio_status make_paged(uint64_t slots);
  gorio_status reset_cache();

  void release_all() {
    if (paged) paged->release();
    paged.reset();
    if (d_pages) (void)hipFree(d_pages);
    if (h_backing) (void)hipHostFree(h_backing);
    if (d_node_to_slot) (void)hipFree(d_node_to_slot);
    if (d_stats) (void)hipFree(d_stats);
    if (d_stage) (void)hipFree(d_stage);
    if (d_centroids) (void)hipFree(d_centroids);
    if (d_centroid_norms) (void)hipFree(d_centroid_norms);
    if (ev_start) (void)hipEventDestroy(ev_start);
    if (ev_stop) (void)hipEventDestroy(ev_stop);
    if (ev_done) (void)hipEventDestroy(ev_done);
    if (stream) (void)hipStreamDestroy(stream);
    d_pages = nullptr;
    h_backing = nullptr;
    d_node_to_slot = nullptr;
    d_stats = nullptr;
    d_stage = nullptr;
    stage_bytes = 0;
    d_centroids = d_centroid_norms = nullptr;
    order_clusters = 0;
    ev_start = ev_stop = ev_done = nullptr;
    ev_done_recorded = false;
    stream = nullptr;
  }
};

// True when stream order alone puts a search on `s` after the index's last
// search: the same stream, and one that is never destroyed (the null stream or
// the per-thread stream).  A created stream's handle is given to the next
// stream created once it is destroyed, so on any other handle the search waits
// for the last search's event.
inline bool follows_last_search(const gorio_index *ix, hipStream_t s) {
  return ix->last_stream == s && (s == nullptr || s == hipStreamPerThread);
}
