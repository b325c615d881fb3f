// The page cache's slot state machine on the CPU: the transitions of
// paper_2607_04415_amd/csrc/slot_state.hpp, compiled for the host, driven by
// threads that play the two sides of the paged search (GORIO Sec. 3.2).
//
//   query threads  each runs queries one after another, as a query slot of a
//                  wave does: it walks the query's page accesses, keeps up to
//                  max_pending of them outstanding (acquire_page: hit, join of
//                  a LOADING page, or claim + miss descriptor), parks when no
//                  slot can be taken, reads a page once its slot is READY and
//                  then unpins it
//   fill threads   take miss descriptors from the ring in order (as the proxy
//                  and fill waves do), wait the injected latency, write the
//                  page's stamp into the slot, and mark the slot READY
//
// Checked: a page read through a pinned slot is the page that was asked for,
// both right after the slot turned READY and again just before the unpin (a
// slot refilled while pinned fails this); every query finishes, with no
// stretch of `stall_s` seconds without a completed access; at the end no pin
// is left, no slot is LOADING, every READY slot is the one its page maps to,
// and every descriptor was consumed.
//
// HIP's atomic functions are supplied below with sequentially consistent host
// atomics: this checks the transitions' logic and their interleavings, not
// the GPU memory model's orderings (those are the business of the coherent
// buffer operations and waits in page_cache.hpp).
//
// usage: slot_harness slots pages queries_in_flight max_pending queries
//                     accesses fillers latency_us seed stall_s [control [pause_us]]
// control (negative controls, which the stamp check must catch): 1 = a query
// unpins before it reads the page; 2 = a fill marks the slot READY before it
// writes the page.  pause_us > 0 makes a thread sleep that long, now and then,
// at the state machine's pause points (between a lookup and its pin).
#include <atomic>
#include <chrono>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <thread>
#include <vector>

#define __device__
#define __forceinline__ inline
#define __HIP_MEMORY_SCOPE_AGENT 0
#define __HIP_MEMORY_SCOPE_SYSTEM 0
#define __hip_atomic_load(p, order, scope) __atomic_load_n((p), __ATOMIC_SEQ_CST)
#define __hip_atomic_store(p, v, order, scope) __atomic_store_n((p), (v), __ATOMIC_SEQ_CST)
template <class T, class U> inline T atomicAdd(T *p, U v) { return __atomic_fetch_add(p, (T)v, __ATOMIC_SEQ_CST); }
template <class T, class U> inline T atomicSub(T *p, U v) { return __atomic_fetch_sub(p, (T)v, __ATOMIC_SEQ_CST); }
template <class T, class U> inline T atomicAnd(T *p, U v) { return __atomic_fetch_and(p, (T)v, __ATOMIC_SEQ_CST); }
template <class T, class U> inline T atomicOr(T *p, U v) { return __atomic_fetch_or(p, (T)v, __ATOMIC_SEQ_CST); }
template <class T, class U, class V> inline T atomicCAS(T *p, U expected, V desired) {
  T e = (T)expected;
  __atomic_compare_exchange_n(p, &e, (T)desired, false, __ATOMIC_SEQ_CST, __ATOMIC_SEQ_CST);
  return e;
}

// Delays at the state machine's pause points (pause_us > 0): a thread sleeps
// there now and then, so that other threads run whole transitions in between.
static double g_pause_us = 0.0;
static thread_local uint64_t t_pause_rng = 0x853c49e6748fea9bull;
static inline void slot_pause() {
  if (g_pause_us <= 0.0) return;
  t_pause_rng = t_pause_rng * 6364136223846793005ull + 1442695040888963407ull;
  if ((t_pause_rng >> 59) == 0)  // 1 in 32
    std::this_thread::sleep_for(std::chrono::nanoseconds((int64_t)(g_pause_us * 1000)));
}
#define GORIO_SLOT_PAUSE(where) slot_pause()

#include "../paper_2607_04415_amd/csrc/slot_state.hpp"

using namespace gorio;
using clk = std::chrono::steady_clock;

static uint64_t splitmix64(uint64_t x) {
  x += 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  return x ^ (x >> 31);
}

int main(int argc, char **argv) {
  if (argc < 11) {
    fprintf(stderr, "usage: %s slots pages queries_in_flight max_pending queries accesses fillers "
                    "latency_us seed stall_s [control [pause_us]]\n", argv[0]);
    return 2;
  }
  const uint32_t slots = (uint32_t)atoi(argv[1]);
  const uint32_t pages = (uint32_t)atoi(argv[2]);
  const int live = atoi(argv[3]);
  const uint32_t max_pending = (uint32_t)atoi(argv[4]);
  const uint64_t queries = (uint64_t)atoll(argv[5]);
  const uint32_t accesses = (uint32_t)atoi(argv[6]);
  const int fillers = atoi(argv[7]);
  const double latency_us = atof(argv[8]);
  const uint64_t seed = (uint64_t)atoll(argv[9]);
  const double stall_s = atof(argv[10]);
  const int control = argc > 11 ? atoi(argv[11]) : 0;
  const bool read_after_unpin = control == 1, ready_before_bytes = control == 2;
  g_pause_us = argc > 12 ? atof(argv[12]) : 0.0;
  if (slots == 0 || pages == 0 || live <= 0 || max_pending == 0 || fillers <= 0) return 2;

  uint32_t ring = 1;
  while (ring < 2 * slots + 64) ring <<= 1;
  std::vector<unsigned long long> slot_word(slots, 0), mq(ring, 0);
  std::vector<uint32_t> page_slot(pages, kNone), stamp(slots, 0);
  unsigned long long clock_hand = 0, mq_tail = 0;
  CacheView c{};
  c.slot_word = slot_word.data();
  c.page_slot = page_slot.data();
  c.clock_hand = &clock_hand;
  c.slots = slots;
  c.page_bytes = 4096;
  c.mq = mq.data();
  c.mq_mask = ring - 1;
  c.mq_tail = &mq_tail;

  std::atomic<uint64_t> next_query{0}, done_queries{0}, mq_head{0};
  std::atomic<uint64_t> hits{0}, joins{0}, misses{0}, noslot{0}, served{0}, bad{0}, completed{0};
  std::atomic<bool> stop{false}, stalled{false};
  std::atomic<int64_t> last_progress{clk::now().time_since_epoch().count()};
  const uint32_t hot = pages < 16 ? pages : 16;           // the entry's neighbourhood
  const uint32_t region = pages / 8 > 0 ? pages / 8 : 1;  // a query's cluster

  auto check_read = [&](uint32_t s, uint32_t page) {
    if (__atomic_load_n(&stamp[s], __ATOMIC_SEQ_CST) != page + 1) bad.fetch_add(1);
  };

  auto query_side = [&](int t) {
    struct Pending { uint32_t page, slot; };
    std::vector<Pending> pend;
    while (!stop.load()) {
      const uint64_t q = next_query.fetch_add(1);
      if (q >= queries) break;
      const uint64_t qs = splitmix64(seed ^ (q * 0x100000001B3ull));
      const uint32_t base = (uint32_t)(qs % pages);
      uint32_t i = 0;
      pend.clear();
      while ((i < accesses || !pend.empty()) && !stop.load()) {
        bool progress = false;
        // start accesses while fewer than max_pending are outstanding
        while (i < accesses && pend.size() < max_pending) {
          const uint64_t r = splitmix64(qs + i);
          uint32_t page;
          switch (r & 3) {
            case 0: page = (uint32_t)((r >> 8) % hot); break;
            case 1: page = (base + (uint32_t)((r >> 8) % region)) % pages; break;
            default: page = (uint32_t)((r >> 8) % pages); break;
          }
          uint32_t s = kNone;
          bool issued = false;
          const uint32_t a = acquire_page(c, page, true, s, issued);
          if (a == kAcqNoSlot) { noslot.fetch_add(1); break; }  // park; retried later
          ++i;
          if (a == kAcqReady) {
            hits.fetch_add(1);
            if (read_after_unpin) {
              unpin(c, s);
              std::this_thread::sleep_for(std::chrono::microseconds(20));
              check_read(s, page);
            } else {
              check_read(s, page);
              if ((r >> 40) % 8 == 0) std::this_thread::yield();  // hold the pin a while
              check_read(s, page);
              unpin(c, s);
            }
            progress = true;
            completed.fetch_add(1);
          } else {
            (issued ? misses : joins).fetch_add(1);
            pend.push_back({page, s});
          }
        }
        // resume the accesses whose slots are READY
        for (size_t k = 0; k < pend.size();) {
          if (slot_ready(c, pend[k].slot)) {
            check_read(pend[k].slot, pend[k].page);
            std::this_thread::yield();
            check_read(pend[k].slot, pend[k].page);
            unpin(c, pend[k].slot);
            pend[k] = pend.back();
            pend.pop_back();
            progress = true;
            completed.fetch_add(1);
          } else {
            ++k;
          }
        }
        if (progress)
          last_progress.store(clk::now().time_since_epoch().count());
        else
          std::this_thread::yield();
      }
      for (const Pending &p : pend) {  // only on stop
        if (stalled.load()) {
          const uint64_t w = __atomic_load_n(&slot_word[p.slot], __ATOMIC_SEQ_CST);
          fprintf(stderr, "stuck: page %u slot %u state %llu page-in-slot %u pins %llu page_slot[page] %u\n",
                  p.page, p.slot, (unsigned long long)sw_state(w), sw_page(w), (unsigned long long)sw_pins(w),
                  __atomic_load_n(&page_slot[p.page], __ATOMIC_SEQ_CST));
        }
        unpin(c, p.slot);
      }
      done_queries.fetch_add(1);
    }
    (void)t;
  };

  auto fill_side = [&](int f) {
    uint64_t rng = splitmix64(seed + 1000 + f);
    while (!stop.load()) {
      const uint64_t h = mq_head.load();
      if (h >= __atomic_load_n(&mq_tail, __ATOMIC_SEQ_CST)) {
        if (done_queries.load() >= queries) break;
        std::this_thread::yield();
        continue;
      }
      uint64_t expect = h;
      if (!mq_head.compare_exchange_strong(expect, h + 1)) continue;
      unsigned long long e;
      while ((e = __atomic_load_n(&mq[h & (ring - 1)], __ATOMIC_SEQ_CST)) == 0) {
        if (stop.load()) return;
        std::this_thread::yield();
      }
      __atomic_store_n(&mq[h & (ring - 1)], 0ull, __ATOMIC_SEQ_CST);
      const uint32_t page = (uint32_t)(e >> 32) - 1u, s = (uint32_t)e;
      if (page >= pages || s >= slots) { bad.fetch_add(1); continue; }
      const uint64_t w = __atomic_load_n(&slot_word[s], __ATOMIC_SEQ_CST);
      if (sw_state(w) != kLoading || sw_page(w) != page) bad.fetch_add(1);  // a fill owns its slot
      if (latency_us > 0) {
        rng = splitmix64(rng);
        const double us = latency_us * (0.5 + (double)(rng % 1000) / 1000.0);
        std::this_thread::sleep_for(std::chrono::nanoseconds((int64_t)(us * 1000)));
      }
      if (ready_before_bytes) {
        mark_ready(c, s);
        std::this_thread::sleep_for(std::chrono::microseconds(20));
        __atomic_store_n(&stamp[s], page + 1, __ATOMIC_SEQ_CST);
      } else {
        __atomic_store_n(&stamp[s], page + 1, __ATOMIC_SEQ_CST);
        mark_ready(c, s);
      }
      served.fetch_add(1);
    }
  };

  const auto t0 = clk::now();
  std::vector<std::thread> th;
  for (int f = 0; f < fillers; ++f) th.emplace_back(fill_side, f);
  for (int t = 0; t < live; ++t) th.emplace_back(query_side, t);
  while (done_queries.load() < queries) {
    std::this_thread::sleep_for(std::chrono::milliseconds(20));
    const double idle =
        std::chrono::duration<double>(clk::now().time_since_epoch() -
                                      clk::duration(last_progress.load())).count();
    if (idle > stall_s) {
      stalled.store(true);
      stop.store(true);
      break;
    }
  }
  stop.store(true);
  for (auto &x : th) x.join();
  const double secs = std::chrono::duration<double>(clk::now() - t0).count();

  // final state
  uint64_t pins_left = 0, loading_left = 0, unmapped_ready = 0, map_errors = 0;
  for (uint32_t s = 0; s < slots; ++s) {
    const uint64_t w = slot_word[s];
    pins_left += sw_pins(w);
    if (sw_state(w) == kLoading) ++loading_left;
    if (sw_state(w) == kReady && page_slot[sw_page(w)] != s) ++unmapped_ready;
  }
  for (uint32_t p = 0; p < pages; ++p) {
    const uint32_t s = page_slot[p];
    if (s == kNone) continue;
    if (s >= slots || sw_page(slot_word[s]) != p || sw_state(slot_word[s]) == kEmpty) ++map_errors;
    else if (stamp[s] != p + 1) ++map_errors;
  }
  printf("{\"queries\": %llu, \"completed_accesses\": %llu, \"hits\": %llu, \"joins\": %llu, "
         "\"misses\": %llu, \"served\": %llu, \"noslot\": %llu, \"bad_reads\": %llu, \"stalled\": %s, "
         "\"pins_left\": %llu, \"loading_left\": %llu, \"unmapped_ready\": %llu, \"map_errors\": %llu, "
         "\"descriptors_left\": %llu, \"seconds\": %.3f}\n",
         (unsigned long long)done_queries.load(), (unsigned long long)completed.load(),
         (unsigned long long)hits.load(), (unsigned long long)joins.load(), (unsigned long long)misses.load(),
         (unsigned long long)served.load(), (unsigned long long)noslot.load(), (unsigned long long)bad.load(),
         stalled.load() ? "true" : "false", (unsigned long long)pins_left, (unsigned long long)loading_left,
         (unsigned long long)unmapped_ready, (unsigned long long)map_errors,
         (unsigned long long)(mq_tail - mq_head.load()), secs);
  return 0;
}
