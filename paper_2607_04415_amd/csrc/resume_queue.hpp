// The GPU resume queue's transitions (GORIO Sec. 3.1, Fig. 1: a ready table
// feeding a resume queue): which lanes wait on which cache slots, and the run
// queue the executor waves take lanes from.
//
// Like slot_state.hpp this header is written against the HIP atomic
// functions alone, with its fences, sleeps and pause points behind macros, so
// that the CPU harness under tests/ compiles the same code and runs it from
// many threads.
//
// A lane's state word:
//   RUNNING  an executor holds it (or it never ran)
//   PARKED   it waits for a page; its bit is set in the waiter set of each
//            cache slot it waits for (one 64-bit word per 64 lanes per slot)
//   QUEUED   it is in the run queue (at most once: only PARKED -> QUEUED by
//            CAS, or RUNNING -> QUEUED by its own executor, put it there)
// No wake is lost: the lane stores PARKED, then sets its bits, then (after a
// sequentially consistent fence) looks at its slots again and queues itself
// if one is READY; the side that fills a slot marks it READY, fences, and
// only then takes the slot's waiter set.  A wake that finds the lane's pages
// not ready after all costs one turn that parks it again.
// The run queue is a ring of lane + 1 entries (0 = free) of at least twice the
// lanes: a reserving tail counter and a claiming head counter.
#pragma once

#include <cstdint>

namespace gorio {

enum : uint32_t { kLsRunning = 0, kLsParked = 1, kLsQueued = 2 };
constexpr uint32_t kNoLane = 0xFFFFFFFFu;

#ifndef GORIO_QUEUE_PAUSE
#define GORIO_QUEUE_PAUSE(where)
#endif
enum : int { kPauseAfterParked = 0, kPauseBeforeRecheck = 1, kPauseBeforeTake = 2, kPauseAfterReserve = 3 };
#ifndef GORIO_QUEUE_FENCE_ACQ
#define GORIO_QUEUE_FENCE_ACQ() __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent")
#define GORIO_QUEUE_FENCE_REL() __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent")
#define GORIO_QUEUE_FENCE_SEQ() __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "agent")
#endif
#ifndef GORIO_QUEUE_SLEEP
#define GORIO_QUEUE_SLEEP() __builtin_amdgcn_s_sleep(1)
#endif

struct RunQueue {
  uint32_t lanes;
  uint32_t words;                 // 64-bit words of one waiter set (ceil(lanes / 64))
  unsigned long long *waiters;    // per cache slot: the lanes parked on its page (slots x words)
  uint32_t *lane_st;              // per lane: kLsRunning, kLsParked or kLsQueued
  unsigned long long *rq;         // run queue: lane + 1 per entry, 0 = free
  uint32_t rq_mask;               // capacity - 1 (capacity >= 2 x lanes, a power of two)
  unsigned long long *rq_head;    // entries taken
  unsigned long long *rq_tail;    // entries reserved
  unsigned int *next_lane;        // lanes handed their first query so far
};

// Append `lane`.  The entry's previous occupant was taken by the time the ring
// has come round to it, except by a reader that claimed it and has not cleared
// it yet: wait for that (or for stop()).
template <class Stop>
__device__ __forceinline__ void queue_push(const RunQueue &q, uint32_t lane, Stop stop) {
  const unsigned long long t = atomicAdd(q.rq_tail, 1ull);
  GORIO_QUEUE_PAUSE(kPauseAfterReserve);
  unsigned long long *e = &q.rq[t & q.rq_mask];
  while (__hip_atomic_load(e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0ull && !stop()) GORIO_QUEUE_SLEEP();
  __hip_atomic_store(e, (unsigned long long)lane + 1ull, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

// Take the next queued lane: kNoLane if none is queued, or stop() came
// first.  The caller then owns the lane (and acquires before reading its
// state).
template <class Stop>
__device__ __forceinline__ uint32_t queue_take(const RunQueue &q, Stop stop) {
  const unsigned long long h = __hip_atomic_load(q.rq_head, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const unsigned long long t = __hip_atomic_load(q.rq_tail, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (h >= t || atomicCAS(q.rq_head, h, h + 1) != h) return kNoLane;
  unsigned long long *e = &q.rq[h & q.rq_mask];
  unsigned long long v = 0;
  while ((v = __hip_atomic_load(e, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT)) == 0ull && !stop()) GORIO_QUEUE_SLEEP();
  if (v == 0ull) return kNoLane;
  __hip_atomic_store(e, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return (uint32_t)(v - 1ull);
}

// A lane that never ran, while there are any (kNoLane otherwise).
__device__ __forceinline__ uint32_t take_fresh_lane(const RunQueue &q) {
  if (__hip_atomic_load(q.next_lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= q.lanes) return kNoLane;
  const uint32_t nl = atomicAdd(q.next_lane, 1u);
  return nl < q.lanes ? nl : kNoLane;
}

__device__ __forceinline__ void lane_running(const RunQueue &q, uint32_t lane) {
  __hip_atomic_store(&q.lane_st[lane], (uint32_t)kLsRunning, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Its own executor queues a lane that can go on (the caller has released the
// lane's state first).
template <class Stop>
__device__ __forceinline__ void requeue_lane(const RunQueue &q, uint32_t lane, Stop stop) {
  __hip_atomic_store(&q.lane_st[lane], (uint32_t)kLsQueued, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  queue_push(q, lane, stop);
}

// Parking, in three steps with the caller's fences between them:
//   park_begin(lane); release fence; park_wait_on(lane, slot) for each slot;
//   sequentially consistent fence; if one of the slots is READY: park_recheck_wake.
// A lane taken from the queue first withdraws from the slots it parked on.
__device__ __forceinline__ void park_begin(const RunQueue &q, uint32_t lane) {
  __hip_atomic_store(&q.lane_st[lane], (uint32_t)kLsParked, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  GORIO_QUEUE_PAUSE(kPauseAfterParked);
}
__device__ __forceinline__ void park_wait_on(const RunQueue &q, uint32_t lane, uint32_t slot) {
  atomicOr(&q.waiters[(uint64_t)slot * q.words + (lane >> 6)], 1ull << (lane & 63u));
}
// A resumed lane withdraws from the waiter sets of the slots it parked on
// (the first of them to fill woke it; the others would wake it again for
// nothing).  It is RUNNING meanwhile, and parks afresh on what it still waits
// for, so no wake is lost.
__device__ __forceinline__ void park_withdraw(const RunQueue &q, uint32_t lane, uint32_t slot) {
  atomicAnd(&q.waiters[(uint64_t)slot * q.words + (lane >> 6)], ~(1ull << (lane & 63u)));
}
template <class Stop>
__device__ __forceinline__ bool park_recheck_wake(const RunQueue &q, uint32_t lane, Stop stop) {
  GORIO_QUEUE_PAUSE(kPauseBeforeRecheck);
  if (atomicCAS(&q.lane_st[lane], (uint32_t)kLsParked, (uint32_t)kLsQueued) != kLsParked) return false;
  queue_push(q, lane, stop);
  return true;
}

// The slot is READY and the caller has fenced (sequentially consistent)
// since: queue every lane parked on it.  Returns how many it queued.
template <class Stop>
__device__ __forceinline__ uint32_t wake_waiters(const RunQueue &q, uint32_t slot, Stop stop) {
  uint32_t woken = 0;
  GORIO_QUEUE_PAUSE(kPauseBeforeTake);
  for (uint32_t w = 0; w < q.words; ++w) {
    unsigned long long bits = atomicExch(&q.waiters[(uint64_t)slot * q.words + w], 0ull);
    GORIO_QUEUE_FENCE_ACQ();  // the lanes' PARKED states are seen
    while (bits) {
      const uint32_t lane = w * 64u + (uint32_t)__builtin_ctzll(bits);
      bits &= bits - 1;
      if (lane < q.lanes && atomicCAS(&q.lane_st[lane], (uint32_t)kLsParked, (uint32_t)kLsQueued) == kLsParked) {
        queue_push(q, lane, stop);
        ++woken;
      }
    }
  }
  return woken;
}

}  // namespace gorio
