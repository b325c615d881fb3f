// The GPU resume queue's transitions on the CPU: resume_queue.hpp compiled
// for the host and driven by threads that play its two sides (GORIO Sec. 3.1,
// Fig. 1: a ready table feeding a resume queue).
//
//   executor threads  take a queued lane (or a lane that never ran) and run a
//                     "turn": if none of the pages the lane waits for is ready
//                     (a wake that found nothing) it parks on them again;
//                     otherwise it counts one step, and after `steps` steps the
//                     lane is done; else it requests 1..max_waits new pages
//                     (fresh slots, LOADING) and parks on them, or now and then
//                     queues itself again (a lane that can go on)
//   filler threads    take requests in a random order after a random delay,
//                     mark the slot READY, fence, and queue the lanes parked
//                     on it
//
// Checked: every lane finishes (no stretch of `stall_s` seconds without a
// finished step: a lost wake stalls the run); a lane taken from the queue is
// QUEUED (never queued twice, never taken while parked or running); no lane
// is run by two executors at once; at the end the queue is empty and every
// waiter set is clear.
//
// HIP's atomic functions are supplied below with sequentially consistent host
// atomics: this checks the transitions' logic and their interleavings, not
// the GPU memory model's orderings.
//
// usage: queue_harness lanes executors fillers steps max_waits seed stall_s [pause_us [withdraw [control]]]
// withdraw 0: a resumed lane keeps its bits in the other slots it parked on
// (they wake it again for nothing).  control 1 (the negative control, which
// the stall check must catch): a parked lane does not look at its slots again
// after setting its bits, so a fill that took the waiter set before the bit
// was set loses the wake.
// Prints one JSON line; a broken invariant exits with status 1.
#include <atomic>
#include <chrono>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <mutex>
#include <thread>
#include <vector>

#define __device__
#define __forceinline__ inline
#define __HIP_MEMORY_SCOPE_AGENT 0
#define __hip_atomic_load(p, order, scope) __atomic_load_n((p), __ATOMIC_SEQ_CST)
#define __hip_atomic_store(p, v, order, scope) __atomic_store_n((p), (v), __ATOMIC_SEQ_CST)
template <class T, class U> inline T atomicAdd(T *p, U v) { return __atomic_fetch_add(p, (T)v, __ATOMIC_SEQ_CST); }
template <class T, class U> inline T atomicOr(T *p, U v) { return __atomic_fetch_or(p, (T)v, __ATOMIC_SEQ_CST); }
template <class T, class U> inline T atomicAnd(T *p, U v) { return __atomic_fetch_and(p, (T)v, __ATOMIC_SEQ_CST); }
template <class T, class U> inline T atomicExch(T *p, U v) { return __atomic_exchange_n(p, (T)v, __ATOMIC_SEQ_CST); }
template <class T, class U, class V> inline T atomicCAS(T *p, U expected, V desired) {
  T e = (T)expected;
  __atomic_compare_exchange_n(p, &e, (T)desired, false, __ATOMIC_SEQ_CST, __ATOMIC_SEQ_CST);
  return e;
}
#define GORIO_QUEUE_FENCE_ACQ() std::atomic_thread_fence(std::memory_order_acquire)
#define GORIO_QUEUE_FENCE_REL() std::atomic_thread_fence(std::memory_order_release)
#define GORIO_QUEUE_FENCE_SEQ() std::atomic_thread_fence(std::memory_order_seq_cst)
#define GORIO_QUEUE_SLEEP() std::this_thread::yield()

// Delays at the transitions' pause points (pause_us > 0): a thread sleeps
// there now and then, so that other threads run whole transitions in between.
static double g_pause_us = 0.0;
static bool g_withdraw = true;
static int g_control = 0;
static thread_local uint64_t t_pause_rng = 0x853c49e6748fea9bull;
static inline void queue_pause() {
  if (g_pause_us <= 0.0) return;
  t_pause_rng = t_pause_rng * 6364136223846793005ull + 1442695040888963407ull;
  if ((t_pause_rng >> 59) == 0)  // 1 in 32
    std::this_thread::sleep_for(std::chrono::nanoseconds((int64_t)(g_pause_us * 1000)));
}
#define GORIO_QUEUE_PAUSE(where) queue_pause()

#include "../paper_2607_04415_amd/csrc/resume_queue.hpp"

using namespace gorio;
using clk = std::chrono::steady_clock;

static uint64_t splitmix64(uint64_t x) {
  x += 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  return x ^ (x >> 31);
}

struct Lane {
  std::vector<uint32_t> waits;   // slots of the pages it waits for (its executor's only)
  uint32_t steps = 0;
  uint64_t rng = 0;
};

int main(int argc, char **argv) {
  if (argc < 8) {
    fprintf(stderr, "usage: queue_harness lanes executors fillers steps max_waits seed stall_s [pause_us]\n");
    return 2;
  }
  const uint32_t lanes = (uint32_t)atoi(argv[1]);
  const int executors = atoi(argv[2]), fillers = atoi(argv[3]);
  const uint32_t steps = (uint32_t)atoi(argv[4]), max_waits = (uint32_t)atoi(argv[5]);
  const uint64_t seed = strtoull(argv[6], nullptr, 10);
  const double stall_s = atof(argv[7]);
  g_pause_us = argc > 8 ? atof(argv[8]) : 0.0;
  g_withdraw = argc > 9 ? atoi(argv[9]) != 0 : true;
  g_control = argc > 10 ? atoi(argv[10]) : 0;

  const uint64_t slots = (uint64_t)lanes * steps * max_waits + 1;
  const uint32_t words = (lanes + 63) / 64;
  uint32_t cap = 1;
  while (cap < 2 * lanes + 64) cap <<= 1;
  std::vector<unsigned long long> waiters(slots * words, 0), rq(cap, 0);
  std::vector<uint32_t> lane_st(lanes, kLsRunning), slot_ready(slots, 0);
  std::vector<std::atomic<int>> owner(lanes);
  for (auto &o : owner) o = 0;
  unsigned long long rq_head = 0, rq_tail = 0;
  unsigned int next_lane = 0;
  RunQueue q{lanes, words, waiters.data(), lane_st.data(), rq.data(), cap - 1, &rq_head, &rq_tail, &next_lane};

  std::vector<Lane> L(lanes);
  for (uint32_t i = 0; i < lanes; ++i) L[i].rng = splitmix64(seed * 1000003 + i);
  std::atomic<uint64_t> next_slot{1}, done_lanes{0}, done_steps{0};
  std::atomic<uint64_t> n_self{0}, n_woken{0}, n_spurious{0}, n_requeue{0};
  std::atomic<bool> stop_all{false}, failed{false}, stalled{false};
  auto stop = [&]() { return stop_all.load() || done_lanes.load() >= lanes; };
  auto fail = [&](const char *what, uint64_t a, uint64_t b) {
    if (!failed.exchange(true)) fprintf(stderr, "FAIL: %s (%llu, %llu)\n", what, (unsigned long long)a,
                                        (unsigned long long)b);
    stop_all = true;
  };

  // requests: slot ids the fillers complete in a random order after a delay
  std::mutex req_mu;
  std::vector<std::pair<uint64_t, clk::time_point>> requests;

  auto executor = [&](int id) {
    uint64_t rng = splitmix64(seed ^ (0xE0000 + id));
    while (!stop()) {
      uint32_t lane = queue_take(q, stop);
      if (lane != kNoLane) {
        // taken from the queue: it must be QUEUED
        const uint32_t st = __atomic_load_n(&lane_st[lane], __ATOMIC_SEQ_CST);
        if (st != kLsQueued) { fail("lane taken from the queue is not QUEUED", lane, st); break; }
      } else {
        lane = take_fresh_lane(q);
        if (lane == kNoLane) { std::this_thread::yield(); continue; }
      }
      if (lane >= lanes) { fail("lane out of range", lane, lanes); break; }
      if (owner[lane].exchange(1) != 0) { fail("lane run by two executors at once", lane, 0); break; }
      lane_running(q, lane);
      Lane &ln = L[lane];
      // a lane taken from the queue leaves the waiter sets it parked in (unless
      // withdraw is off: then stale bits wake it again for nothing)
      if (g_withdraw)
        for (uint32_t s : ln.waits) park_withdraw(q, lane, s);
      // the turn
      bool any_ready = ln.waits.empty();
      for (uint32_t s : ln.waits) any_ready |= __atomic_load_n(&slot_ready[s], __ATOMIC_SEQ_CST) != 0;
      if (!any_ready) {
        n_spurious++;
      } else {
        ln.waits.clear();
        ++ln.steps;
        done_steps++;
        if (ln.steps >= steps) {
          owner[lane] = 0;
          done_lanes++;
          continue;
        }
        ln.rng = splitmix64(ln.rng);
        if ((ln.rng & 15) == 0) {  // it can go on: queue it again
          owner[lane] = 0;
          GORIO_QUEUE_FENCE_REL();
          requeue_lane(q, lane, stop);
          n_requeue++;
          continue;
        }
        const uint32_t nw = 1 + (uint32_t)((ln.rng >> 8) % max_waits);
        std::lock_guard<std::mutex> g(req_mu);
        for (uint32_t j = 0; j < nw; ++j) {
          const uint64_t s = next_slot++;
          if (s >= slots) { fail("slot pool exhausted", s, slots); break; }
          ln.waits.push_back((uint32_t)s);
          rng = splitmix64(rng);
          requests.push_back({s, clk::now() + std::chrono::microseconds(rng % 50)});
        }
      }
      // park on the lane's waits, from a copy taken before the lane can be
      // woken (another executor may run it from then on)
      const std::vector<uint32_t> waits = ln.waits;
      owner[lane] = 0;
      park_begin(q, lane);
      GORIO_QUEUE_FENCE_REL();
      for (uint32_t s : waits) park_wait_on(q, lane, s);
      GORIO_QUEUE_FENCE_SEQ();
      if (g_control == 1) continue;  // negative control: no second look
      bool ready = false;
      for (uint32_t s : waits) ready |= __atomic_load_n(&slot_ready[s], __ATOMIC_SEQ_CST) != 0;
      if (ready && park_recheck_wake(q, lane, stop)) n_self++;
    }
  };

  auto filler = [&](int id) {
    uint64_t rng = splitmix64(seed ^ (0xF0000 + id));
    while (!stop()) {
      uint64_t s = 0;
      {
        std::lock_guard<std::mutex> g(req_mu);
        if (!requests.empty()) {
          rng = splitmix64(rng);
          const size_t i = rng % requests.size();
          if (requests[i].second <= clk::now()) {
            s = requests[i].first;
            requests[i] = requests.back();
            requests.pop_back();
          }
        }
      }
      if (s == 0) { std::this_thread::yield(); continue; }
      __atomic_store_n(&slot_ready[s], 1u, __ATOMIC_SEQ_CST);
      GORIO_QUEUE_FENCE_SEQ();
      n_woken += wake_waiters(q, (uint32_t)s, stop);
    }
  };

  std::vector<std::thread> th;
  for (int i = 0; i < executors; ++i) th.emplace_back(executor, i);
  for (int i = 0; i < fillers; ++i) th.emplace_back(filler, i);
  // watchdog: progress in finished steps
  uint64_t last = 0;
  auto last_t = clk::now();
  while (!stop()) {
    std::this_thread::sleep_for(std::chrono::milliseconds(20));
    const uint64_t d = done_steps.load();
    if (d != last) { last = d; last_t = clk::now(); }
    else if (std::chrono::duration<double>(clk::now() - last_t).count() > stall_s) {
      size_t parked = 0, queued = 0;
      for (uint32_t i = 0; i < lanes; ++i) {
        parked += __atomic_load_n(&lane_st[i], __ATOMIC_SEQ_CST) == kLsParked;
        queued += __atomic_load_n(&lane_st[i], __ATOMIC_SEQ_CST) == kLsQueued;
      }
      fprintf(stderr, "stalled: %zu lanes parked, %zu queued\n", parked, queued);
      stalled = true;
      stop_all = true;
    }
  }
  for (auto &t : th) t.join();
  if (failed) return 1;
  // end state (a finished run): every lane done, nothing left in the queue
  size_t left = 0;
  for (uint32_t i = 0; i < cap; ++i) left += rq[i] != 0;
  if (!stalled && (done_lanes.load() != lanes || left != 0 || rq_head != rq_tail)) {
    fprintf(stderr, "FAIL: %llu of %u lanes done, %zu queue entries left\n", (unsigned long long)done_lanes.load(),
            lanes, left);
    return 1;
  }
  printf("{\"stalled\": %s, \"lanes_done\": %llu, \"steps\": %llu, \"woken\": %llu, \"self_woken\": %llu, "
         "\"spurious\": %llu, \"requeued\": %llu, \"slots_used\": %llu}\n",
         stalled ? "true" : "false", (unsigned long long)done_lanes.load(), (unsigned long long)done_steps.load(),
         (unsigned long long)n_woken.load(), (unsigned long long)n_self.load(), (unsigned long long)n_spurious.load(),
         (unsigned long long)n_requeue.load(), (unsigned long long)next_slot.load() - 1);
  return 0;
}
