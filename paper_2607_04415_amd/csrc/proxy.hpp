// Host transport proxy (GORIO Sec. 3.3 and Sec. 4, "CPU transport proxy").
//
// One thread stands in for the paper's SPDK NVMe-oF workers.  It only moves
// page-level descriptors: it takes {page, slot} descriptors that GPU waves
// publish into a ring in coherent pinned memory, holds each one until its
// injected service latency has elapsed (the stand-in for a remote read), and
// publishes it to a completion ring the GPU polls (one ring per GPU fill wave).  It never looks at query
// state.  It batches both directions and caps the requests it holds in flight.
// The page bytes themselves are copied by GPU waves from the pinned backing
// store into the HBM slot, standing in for the RNIC's direct placement.
#pragma once

#include <atomic>
#include <cstdint>
#include <thread>

namespace gorio {

class Proxy {
 public:
  Proxy() = default;
  ~Proxy() { stop(); }
  Proxy(const Proxy &) = delete;
  Proxy &operator=(const Proxy &) = delete;

  // Rings live in host memory that both sides can access; capacities are powers of two.
  // Completions are dealt round-robin over the completion rings of a search:
  // ring r is cq + r * (cq_mask + 1), its publish index cq_tail[r * tail_stride].
  void start(unsigned long long *mq, uint32_t mq_mask, unsigned long long *cq, uint32_t cq_mask,
             unsigned long long *cq_tail, uint32_t tail_stride);
  // Reset ring indices and counters for a new search and begin serving over
  // `rings` completion rings (the caller has zeroed their tails).
  // Fault injection for tests: jitter_us adds a uniform random delay in
  // [0, jitter_us] to each request, so completions leave out of request
  // order; hold keeps every request in flight (none completes).
  void begin(double latency_us, uint32_t max_outstanding, uint32_t rings, double jitter_us = 0.0,
             bool hold = false);
  // Stop serving (the search ended); descriptors in flight are dropped.
  void end();
  void stop();

  uint64_t requests() const { return requests_.load(std::memory_order_relaxed); }
  uint64_t completed() const { return completed_.load(std::memory_order_relaxed); }
  uint64_t max_in_flight() const { return max_in_flight_.load(std::memory_order_relaxed); }

 private:
  void loop();

  unsigned long long *mq_ = nullptr, *cq_ = nullptr, *cq_tail_ = nullptr;
  uint32_t mq_mask_ = 0, cq_mask_ = 0, tail_stride_ = 1;
  std::atomic<uint32_t> rings_{1};
  std::atomic<bool> quit_{false}, active_{false}, idle_{true};
  std::atomic<uint64_t> epoch_{0};
  std::atomic<uint64_t> latency_ns_{0}, jitter_ns_{0};
  std::atomic<bool> hold_{false};
  std::atomic<uint32_t> max_outstanding_{4096};
  std::atomic<uint64_t> requests_{0}, completed_{0}, max_in_flight_{0};
  std::thread th_;
};

}  // namespace gorio
