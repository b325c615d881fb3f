// Host transport proxy: descriptor intake, deadline queue, completion publish.
#include "proxy.hpp"

#include <chrono>
#include <deque>
#include <functional>
#include <queue>
#include <utility>
#include <vector>

#if defined(__x86_64__)
#include <immintrin.h>
#define GORIO_PAUSE() _mm_pause()
#else
#define GORIO_PAUSE() std::this_thread::yield()
#endif

namespace gorio {

namespace {
uint64_t now_ns() {
  return (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(
             std::chrono::steady_clock::now().time_since_epoch())
      .count();
}
}  // namespace

void Proxy::start(unsigned long long *mq, uint32_t mq_mask, unsigned long long *cq, uint32_t cq_mask,
                  unsigned long long *cq_tail, uint32_t tail_stride) {
  stop();
  mq_ = mq;
  mq_mask_ = mq_mask;
  cq_ = cq;
  cq_mask_ = cq_mask;
  cq_tail_ = cq_tail;
  tail_stride_ = tail_stride ? tail_stride : 1;
  quit_.store(false);
  active_.store(false);
  th_ = std::thread([this] { loop(); });
}

void Proxy::begin(double latency_us, uint32_t max_outstanding, uint32_t rings, double jitter_us, bool hold) {
  rings_.store(rings ? rings : 1);
  latency_ns_.store((uint64_t)(latency_us * 1000.0));
  jitter_ns_.store(jitter_us > 0.0 ? (uint64_t)(jitter_us * 1000.0) : 0);
  hold_.store(hold);
  max_outstanding_.store(max_outstanding ? max_outstanding : 4096);
  requests_.store(0);
  completed_.store(0);
  max_in_flight_.store(0);
  epoch_.fetch_add(1);
  active_.store(true, std::memory_order_release);
}

void Proxy::end() {
  active_.store(false, std::memory_order_release);
  // wait until the thread has left its serving iteration: nothing it does can
  // land in the rings after this returns
  while (th_.joinable() && !idle_.load(std::memory_order_acquire)) std::this_thread::yield();
}

void Proxy::stop() {
  if (th_.joinable()) {
    quit_.store(true);
    th_.join();
  }
}

void Proxy::loop() {
  // (descriptor, due time); latency is the same for every request, so FIFO
  // order is deadline order
  std::deque<std::pair<unsigned long long, uint64_t>> fifo;
  // with jitter, requests leave by due time: (due time, descriptor), earliest first
  using Due = std::pair<uint64_t, unsigned long long>;
  std::priority_queue<Due, std::vector<Due>, std::greater<Due>> heap;
  uint64_t rng = 0x9E3779B97F4A7C15ull;  // SplitMix64 state for the jitter draws
  std::vector<uint64_t> tails;  // completions published per ring
  uint64_t head = 0, dealt = 0, epoch = ~0ull;
  uint32_t rings = 1;
  while (!quit_.load(std::memory_order_relaxed)) {
    if (!active_.load(std::memory_order_acquire)) {
      idle_.store(true, std::memory_order_release);
      std::this_thread::sleep_for(std::chrono::microseconds(50));
      continue;
    }
    idle_.store(false, std::memory_order_release);
    if (!active_.load(std::memory_order_acquire)) continue;  // end() raced with the flag above
    if (epoch != epoch_.load()) {  // a new search: rings were reset by the host
      epoch = epoch_.load();
      fifo.clear();
      heap = decltype(heap)();
      rings = rings_.load();
      tails.assign(rings, 0);
      head = dealt = 0;
    }
    const uint64_t lat = latency_ns_.load(std::memory_order_relaxed);
    const uint64_t jitter = jitter_ns_.load(std::memory_order_relaxed);
    const bool hold = hold_.load(std::memory_order_relaxed);
    const uint32_t cap = max_outstanding_.load(std::memory_order_relaxed);
    uint32_t intake = 0;
    while (fifo.size() + heap.size() < cap) {
      unsigned long long *slot = &mq_[head & mq_mask_];
      const unsigned long long e = __atomic_load_n(slot, __ATOMIC_ACQUIRE);
      if (e == 0) break;
      __atomic_store_n(slot, 0ull, __ATOMIC_RELAXED);
      ++head;
      fifo.emplace_back(e, 0);
      ++intake;
    }
    // the clock is read after the intake, so no request is due before it was
    // published plus the latency
    const uint64_t now = now_ns();
    for (size_t i = fifo.size() - intake; i < fifo.size(); ++i) fifo[i].second = now + lat;
    if (jitter) {  // move the new requests into the due-time heap with their random delay
      while (!fifo.empty()) {
        uint64_t z = (rng += 0x9E3779B97F4A7C15ull);
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        z ^= z >> 31;
        heap.emplace(fifo.front().second + z % (jitter + 1), fifo.front().first);
        fifo.pop_front();
      }
    }
    const size_t in_flight = fifo.size() + heap.size();
    if (intake) {
      requests_.fetch_add(intake, std::memory_order_relaxed);
      if (in_flight > max_in_flight_.load(std::memory_order_relaxed))
        max_in_flight_.store(in_flight, std::memory_order_relaxed);
    }
    uint32_t done = 0;
    while (!hold && !fifo.empty() && fifo.front().second <= now) {
      const uint32_t r = (uint32_t)(dealt++ % rings);
      cq_[(uint64_t)r * (cq_mask_ + 1) + (tails[r]++ & cq_mask_)] = fifo.front().first;
      fifo.pop_front();
      ++done;
    }
    while (!hold && !heap.empty() && heap.top().first <= now) {
      const uint32_t r = (uint32_t)(dealt++ % rings);
      cq_[(uint64_t)r * (cq_mask_ + 1) + (tails[r]++ & cq_mask_)] = heap.top().second;
      heap.pop();
      ++done;
    }
    if (done) {
      // publish every ring that received completions (entries before tails)
      const uint32_t touched = done < rings ? done : rings;
      for (uint32_t i = 0; i < touched; ++i) {
        const uint32_t r = (uint32_t)((dealt - 1 - i) % rings);
        __atomic_store_n(&cq_tail_[(uint64_t)r * tail_stride_], (unsigned long long)tails[r], __ATOMIC_RELEASE);
      }
      completed_.fetch_add(done, std::memory_order_relaxed);
    }
    if (!intake && !done) GORIO_PAUSE();
  }
}

}  // namespace gorio
