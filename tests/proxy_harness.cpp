// CPU harness for the transport proxy: host threads play the GPU side of the
// descriptor and completion rings.  Checks that every descriptor is completed
// exactly once, never before its injected latency, and that the proxy never
// holds more requests than its cap.  Prints one JSON line with the result.
//
//   proxy_harness <requests> <latency_us> <max_outstanding> <slots> <producers> <rings> <jitter_us>
//
// With several completion rings, one consumer thread per ring plays the GPU
// fill wave that owns that ring.
#include <atomic>
#include <chrono>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <thread>
#include <vector>

#include "../paper_2607_04415_amd/csrc/proxy.hpp"

using clk = std::chrono::steady_clock;

static uint64_t now_ns() {
  return (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(clk::now().time_since_epoch()).count();
}

int main(int argc, char **argv) {
  const uint64_t requests = argc > 1 ? strtoull(argv[1], nullptr, 10) : 200000;
  const double latency_us = argc > 2 ? atof(argv[2]) : 0.0;
  const uint32_t cap = argc > 3 ? (uint32_t)atoi(argv[3]) : 4096;
  const uint32_t slots = argc > 4 ? (uint32_t)atoi(argv[4]) : 10000;
  const int producers = argc > 5 ? atoi(argv[5]) : 4;
  const uint32_t rings = argc > 6 ? (uint32_t)atoi(argv[6]) : 1;
  const double jitter_us = argc > 7 ? atof(argv[7]) : 0.0;
  const uint32_t tail_stride = 8;  // tails on separate 64-byte lines

  uint32_t ring = 1;
  while (ring < 2 * slots + 1024) ring <<= 1;
  std::vector<unsigned long long> mq(ring, 0), cq((size_t)ring * rings, 0);
  std::vector<unsigned long long> cq_tail((size_t)rings * tail_stride, 0);

  gorio::Proxy proxy;
  proxy.start(mq.data(), ring - 1, cq.data(), ring - 1, cq_tail.data(), tail_stride);
  proxy.begin(latency_us, cap, rings, jitter_us);

  // slot s is "LOADING" while in flight; a producer may only use a free slot,
  // as the GPU may only publish a descriptor for a slot it claimed
  std::vector<std::atomic<uint8_t>> busy(slots);
  std::vector<std::atomic<uint64_t>> issued_at(slots);
  std::vector<std::atomic<uint32_t>> done_count(requests);
  for (auto &b : busy) b.store(0);
  for (auto &d : done_count) d.store(0);
  std::atomic<uint64_t> next_req{0}, mq_tail{0}, completed{0}, early{0}, bad{0}, reordered{0};

  auto producer = [&](int id) {
    uint32_t s = (uint32_t)id;
    for (;;) {
      const uint64_t r = next_req.fetch_add(1);
      if (r >= requests) return;
      // find a free slot (the claim)
      for (;;) {
        s = (s + 1) % slots;
        uint8_t z = 0;
        if (busy[s].compare_exchange_strong(z, 1)) break;
      }
      issued_at[s].store(now_ns(), std::memory_order_relaxed);
      const uint64_t t = mq_tail.fetch_add(1);
      // descriptor: (request + 1) << 32 | slot  (the "page" field carries the request id)
      __atomic_store_n(&mq[t & (ring - 1)], ((r + 1) << 32) | s, __ATOMIC_RELEASE);
    }
  };

  auto consumer = [&](uint32_t r0) {
    uint64_t head = 0, last_issue = 0;
    const unsigned long long *q = cq.data() + (size_t)r0 * ring;
    while (completed.load() < requests) {
      const uint64_t t = __atomic_load_n(&cq_tail[(size_t)r0 * tail_stride], __ATOMIC_ACQUIRE);
      for (; head < t; ++head) {
        const unsigned long long e = __atomic_load_n(&q[head & (ring - 1)], __ATOMIC_RELAXED);
        const uint64_t r = (e >> 32) - 1;
        const uint32_t s = (uint32_t)e;
        if (r >= requests || s >= slots) { bad.fetch_add(1); continue; }
        const uint64_t at = issued_at[s].load(std::memory_order_relaxed);
        // completed well before a request issued earlier on this ring
        if (at + 20000 < last_issue) reordered.fetch_add(1);
        last_issue = at > last_issue ? at : last_issue;
        const uint64_t waited = now_ns() - at;
        if (waited + 2000 < (uint64_t)(latency_us * 1000.0)) early.fetch_add(1);
        done_count[r].fetch_add(1);
        busy[s].store(0);  // the fill made the slot READY; it can be reused
        completed.fetch_add(1);
      }
      std::this_thread::yield();
    }
  };

  const uint64_t t0 = now_ns();
  std::vector<std::thread> th;
  for (int i = 0; i < producers; ++i) th.emplace_back(producer, i);
  std::vector<std::thread> cons;
  for (uint32_t r = 0; r < rings; ++r) cons.emplace_back(consumer, r);
  for (auto &x : th) x.join();
  for (auto &x : cons) x.join();
  const double secs = (now_ns() - t0) * 1e-9;
  proxy.end();
  proxy.stop();

  uint64_t twice = 0, missing = 0;
  for (uint64_t r = 0; r < requests; ++r) {
    const uint32_t c = done_count[r].load();
    if (c == 0) ++missing;
    if (c > 1) ++twice;
  }
  printf("{\"requests\": %llu, \"seconds\": %.4f, \"per_second\": %.0f, \"missing\": %llu, "
         "\"duplicated\": %llu, \"early\": %llu, \"bad\": %llu, \"max_in_flight\": %llu, \"cap\": %u, "
         "\"reordered\": %llu}\n",
         (unsigned long long)requests, secs, requests / secs, (unsigned long long)missing,
         (unsigned long long)twice, (unsigned long long)early.load(), (unsigned long long)bad.load(),
         (unsigned long long)proxy.max_in_flight(), cap, (unsigned long long)reordered.load());
  return (missing || twice || early.load() || bad.load() || proxy.max_in_flight() > cap) ? 1 : 0;
}
