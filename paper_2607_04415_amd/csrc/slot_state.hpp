// The HBM page cache's slot state machine (GORIO Sec. 3.2: GPU page cache,
// per-slot ready table, lock-free request descriptors).
//
// This header holds every transition of a cache slot and nothing else. It is
// written against the HIP atomic functions alone (atomicAdd/Sub/And/Or/CAS,
// __hip_atomic_load/store), so that a host build which supplies those
// functions compiles the same code: the CPU harness under tests/ runs these
// transitions from many threads to check that a pinned slot is never
// refilled and that every request completes. Page bytes, and the coherent
// buffer operations that move them, are in page_cache.hpp.
//
// slot_word[s] packs one cache slot's whole state so that one atomic decides
// every transition:
//   bits  0..23  pins     waves currently using or waiting on the slot
//   bit   24     ref      clock reference bit (set by a hit, or by a lookup that
//                         joins a page still LOADING: the page is used more than once)
//   bits 25..26  state    EMPTY / LOADING / READY
//   bits 32..63  page id
// page_slot[p] maps a page to its slot (kNone if not cached).
//
// Transitions:
//   pin      atomicAdd(+1); valid if the returned word still names the page in
//            LOADING or READY, else undone with atomicSub(1) and the lookup retried
//   claim    the clock hand walks the slots; an unpinned READY/EMPTY slot
//            with a clear ref bit is CAS-ed to (page, LOADING, pins=1); the
//            slot's old page is unmapped, then page_slot[page] is CAS-ed from
//            kNone (losing that race gives the slot back and joins the winner)
//   fill     after the page bytes are written and those stores have
//            completed, atomicAdd turns LOADING into READY (mark_ready); the
//            page arrives unreferenced, so a page read once (most pages a
//            random edge brings in) is the clock's first victim, and a page
//            that is hit keeps its slot for another sweep
//   unpin    atomicSub(1)
#pragma once

#include <cstdint>

namespace gorio {

constexpr uint32_t kNone = 0xFFFFFFFFu;
constexpr uint64_t kPinMask = (1ull << 24) - 1;
constexpr uint64_t kRefBit = 1ull << 24;
constexpr int kStateShift = 25;
constexpr uint64_t kStateMask = 3ull << kStateShift;
constexpr uint64_t kEmpty = 0, kLoading = 1, kReady = 2;

__device__ __forceinline__ uint64_t sw_state(uint64_t w) { return (w & kStateMask) >> kStateShift; }
__device__ __forceinline__ uint32_t sw_page(uint64_t w) { return (uint32_t)(w >> 32); }
__device__ __forceinline__ uint64_t sw_pins(uint64_t w) { return w & kPinMask; }

struct CacheView {
  uint8_t *data;                   // slots * page_bytes, HBM
  unsigned long long *slot_word;   // slots
  uint32_t *page_slot;             // num_pages
  unsigned long long *clock_hand;
  uint32_t slots;
  uint64_t page_bytes;
  // miss descriptors -> proxy: ring in host memory, reserved by a device counter
  unsigned long long *mq;
  uint32_t mq_mask;
  unsigned long long *mq_tail;
};

__device__ __forceinline__ uint64_t load_word(const unsigned long long *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Result of looking a page up for one record access.
enum : uint32_t { kAcqReady = 0, kAcqWait = 1, kAcqNoSlot = 2 };

// A point where a host test may stretch the time between two steps of a
// transition (the CPU harness delays a thread there to widen races); empty in
// the library.
#ifndef GORIO_SLOT_PAUSE
#define GORIO_SLOT_PAUSE(where)
#endif
enum : int { kPauseAfterLookup = 0, kPauseAfterClaim = 1, kPauseBeforeGiveBack = 2 };

// Publish a miss descriptor {page, slot} to the proxy (8 bytes, nonzero).
__device__ __forceinline__ void publish_miss(const CacheView &c, uint32_t page, uint32_t slot) {
  const unsigned long long t = atomicAdd(c.mq_tail, 1ull);
  const unsigned long long e = ((unsigned long long)(page + 1) << 32) | slot;
  __hip_atomic_store(&c.mq[t & c.mq_mask], e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Find a victim slot with the clock hand and claim it for `page` in LOADING
// state with one pin.  Returns kNone if no slot can be taken now.
__device__ __forceinline__ uint32_t claim_slot(const CacheView &c, uint32_t page) {
  const uint64_t fresh = ((uint64_t)page << 32) | (kLoading << kStateShift) | 1ull;
  // bounded walk: a failed claim parks the request and the query retries later
  const uint32_t walk = 2 * c.slots + 8;
  const uint32_t max_tries = walk < 512u ? walk : 512u;
  for (uint32_t tries = 0; tries < max_tries; ++tries) {
    const uint32_t s = (uint32_t)(atomicAdd(c.clock_hand, 1ull) % c.slots);
    const uint64_t w = load_word(&c.slot_word[s]);
    const uint64_t st = sw_state(w);
    if (sw_pins(w) != 0 || st == kLoading) continue;
    if (w & kRefBit) {
      atomicAnd(&c.slot_word[s], ~(unsigned long long)kRefBit);
      continue;
    }
    if (atomicCAS(&c.slot_word[s], (unsigned long long)w, (unsigned long long)fresh) != w) continue;
    if (st == kReady) atomicCAS(&c.page_slot[sw_page(w)], s, kNone);
    return s;
  }
  return kNone;
}

// One record access to `page`: on return the slot is pinned unless kAcqNoSlot.
// `allow_claim` false: do not start new page requests (only hit or join).
// `issued` is set when this call published the page's miss descriptor.
__device__ __forceinline__ uint32_t acquire_page(const CacheView &c, uint32_t page, bool allow_claim,
                                                 uint32_t &slot_out, bool &issued) {
  issued = false;
  for (int attempt = 0; attempt < 64; ++attempt) {
    const uint32_t s = __hip_atomic_load(&c.page_slot[page], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (s != kNone) {
      GORIO_SLOT_PAUSE(kPauseAfterLookup);
      const uint64_t old = atomicAdd(&c.slot_word[s], 1ull);
      const uint64_t st = sw_state(old);
      if (sw_page(old) == page && (st == kLoading || st == kReady)) {
        // The lookup may be stale: the slot can have been evicted and claimed
        // again for this same page by a wave that then loses the race to map
        // it and gives the slot back, unfilled.  A LOADING slot is joined only
        // while the page maps to it (only that claim's successful map can make
        // it so, and a pinned slot is never claimed again); a READY slot is
        // always mapped.  The load is issued after the pin has returned.
        if (st == kLoading &&
            __hip_atomic_load(&c.page_slot[page], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != s) {
          atomicSub(&c.slot_word[s], 1ull);
          continue;
        }
        if (!(old & kRefBit)) atomicOr(&c.slot_word[s], (unsigned long long)kRefBit);
        slot_out = s;
        return st == kReady ? kAcqReady : kAcqWait;
      }
      atomicSub(&c.slot_word[s], 1ull);
      continue;
    }
    if (!allow_claim) return kAcqNoSlot;
    const uint32_t ns = claim_slot(c, page);
    if (ns == kNone) return kAcqNoSlot;
    GORIO_SLOT_PAUSE(kPauseAfterClaim);
    if (atomicCAS(&c.page_slot[page], kNone, ns) != kNone) {
      // another wave mapped the page first: give the slot back in one atomic
      // (LOADING -> EMPTY and our pin dropped; pins of concurrent lookups
      // stay), then join the winner's slot
      GORIO_SLOT_PAUSE(kPauseBeforeGiveBack);
      atomicSub(&c.slot_word[ns], (kLoading << kStateShift) | 1ull);
      continue;
    }
    publish_miss(c, page, ns);
    issued = true;
    slot_out = ns;
    return kAcqWait;
  }
  return kAcqNoSlot;
}

__device__ __forceinline__ void unpin(const CacheView &c, uint32_t s) { atomicSub(&c.slot_word[s], 1ull); }

__device__ __forceinline__ bool slot_ready(const CacheView &c, uint32_t s) {
  return sw_state(load_word(&c.slot_word[s])) == kReady;
}

// The fill of slot s is complete: LOADING -> READY.  The caller has made the
// page's bytes visible to every reader of the slot before this call.
__device__ __forceinline__ void mark_ready(const CacheView &c, uint32_t s) {
  atomicAdd(&c.slot_word[s], 1ull << kStateShift);
}

}  // namespace gorio
