// Paged beam search: a persistent kernel whose waves own query slots and
// overlap traversal with page service (GORIO Sec. 3.2 and Sec. 3.3).
//
// Each wave owns `oversub` query slots kept in its LDS (frontier, beam,
// candidate list, per-item wait state) plus a visited table in HBM.  The
// wave's scheduler loop
//   - admits a new query into a free slot (global atomic counter),
//   - resumes a parked query when a page it waits on is READY in the cache
//     (the per-slot ready test of Sec. 3.2) or when it can issue more requests,
// Page service runs beside it: by default a few fill waves (the lowest block
// indices) each consume a completion ring of their own, copy each page (4 KB
// from the pinned backing store into its HBM slot) and mark it READY.  With
// no fill waves, the query waves claim completions from one shared ring
// whenever their queries cannot run.
// A query runs its iteration (select -> expand -> evaluate -> merge) until a
// record it needs is not resident: the miss is published as a descriptor
// {page, slot}, the slot stays pinned, and the query is parked.  An
// iteration's next beam is selected only after every candidate of the
// current one is evaluated, so results equal the resident search's.
//
// blocking = 1 replaces split-phase service with wait-in-place: one query per
// wave and one outstanding page per lane (the blocking demand-paging path the
// paper compares against).
//
// paged_round (at the end of this file) runs the same per-query code for the
// host-scheduled mode: one workgroup per lane the host chose, the lane's
// state loaded from and saved to HBM around one turn; the fill waves then run
// as a kernel of their own (search_paged launched with only fill blocks).
#pragma once

#include "metric.hpp"
#include "resume_queue.hpp"

namespace gorio {

constexpr int kPagedMaxW = 64;
constexpr uint32_t kTodo = 0xFFFFFFFFu;  // item not requested yet
constexpr uint32_t kDone = 0xFFFFFFFEu;  // item handled; other values: waiting on that cache slot
constexpr int kPagedHtLog2 = 13;
constexpr uint32_t kFillBatch = 4;   // completions one wave claims and copies at a time

enum : uint32_t { kPhSelect = 0, kPhExpand = 1, kPhEval = 2 };

struct PagedParams {
  CacheView cache;
  PageGeom geom;  // where vectors and adjacency blocks sit inside a page
  uint32_t n, D, R;
  FastDiv Rdiv;
  uint32_t entry;
  uint32_t num_pages;
  const uint8_t *backing;                 // pinned host copy of every page
  const unsigned long long *cq;           // completion rings from the proxy (host memory), cq_mask + 1 entries each
  uint32_t cq_mask;
  const unsigned long long *cq_tail;      // proxy's publish index of each ring (host memory), tail_stride apart
  uint32_t tail_stride;
  uint32_t fill_waves;                    // blocks [0, fill_waves) only fill pages, wave k from ring k;
                                          // 0: one shared ring served by the query waves
  unsigned long long *cq_head;            // shared ring: next completion to claim (device)
  unsigned long long *tail_seen;          // shared ring: device mirror of its tail
  unsigned int *poll_lock;                // shared ring: try-lock for the one host read of the tail
  const unsigned int *abort_flag;         // host memory; nonzero ends the search
  unsigned int *abort_seen;               // device mirror of abort_flag
  const void *queries;                    // nq x D elements
  uint32_t nq, k, L, W;
  unsigned int *next_query;
  const uint32_t *order;                  // nullptr: queries in index order; else admission order
  unsigned int *done_queries;             // device: queries finished (fill waves stop at nq)
  unsigned long long *fill_head;          // host memory or nullptr: completions of ring k filled so far,
                                          // at fill_head[k * tail_stride] (host-scheduled lanes); a
                                          // fill wave starts from there
  unsigned long long fill_budget;         // nonzero: a fill wave leaves after this many wall-clock
                                          // ticks (a launch per round relaunches it)
  uint32_t *out_ids;
  uint32_t *out_dists;                    // distance bits (int32 or float32)
  uint32_t *ht_pool;                      // (grid * oversub) << kPagedHtLog2 entries
  uint32_t oversub, max_pending;
  uint32_t turn_passes;                   // host rounds: a query yields after this many passes over its
                                          // candidates that found pages ready (0 = no limit)
  int blocking;
  unsigned long long *stats;              // [eval, reeval, exp, iter, hit, miss, served, park, resume, -, bad]
};

template <int KPL>
struct QSlot {
  uint64_t F[KPL * kWave];
  uint32_t beam[kPagedMaxW];
  uint32_t bstate[kPagedMaxW];
  uint32_t cand[kCandCap];
  uint32_t cstate[kCandCap];
  uint32_t qi, active, phase, nbeam, b0, ncand, ht_used, forgot, parked, yielded;
};

struct PagedCounters {
  unsigned long long eval = 0, reeval = 0, exp = 0, iter = 0, hit = 0, miss = 0, served = 0,
                     park = 0, resume = 0;
};

__device__ __forceinline__ bool aborted(const PagedParams &p) {
  return __hip_atomic_load(p.abort_seen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
}

// GPU resume queue (Fig. 1's ready table feeding a resume queue, with nothing
// on the host): lanes keep their query state in HBM as in the host-scheduled
// mode, and the lane-state, waiter-set and run-queue transitions of
// resume_queue.hpp decide which lane runs next.  Its waits end when every
// query is done or on abort.
__device__ __forceinline__ bool queue_done(const PagedParams &p) {
  return aborted(p) || __hip_atomic_load(p.done_queries, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= p.nq;
}

// The fill of n slots (lane i < n: slot (uint32_t)e) is complete: queue the
// lanes parked on them.
__device__ __forceinline__ void wake_filled(const PagedParams &p, const RunQueue &q, unsigned long long e,
                                            uint32_t n) {
  GORIO_QUEUE_FENCE_SEQ();  // READY before the waiter sets are taken
  const uint32_t slot = (uint32_t)e;
  if ((uint32_t)lane_id() < n && slot < p.cache.slots) wake_waiters(q, slot, [&]() { return queue_done(p); });
}

// Byte offsets of node v's vector and adjacency block inside cache slot s.
template <bool N2S>
__device__ __forceinline__ uint32_t cached_vec(const PagedParams &p, uint32_t s, uint32_t v) {
  uint32_t page, pos;
  locate(p.geom, slot_ct<N2S>(p.geom, v), page, pos);
  return s * (uint32_t)p.cache.page_bytes + pos * p.geom.vec_stride;
}
template <bool N2S>
__device__ __forceinline__ uint32_t cached_adj(const PagedParams &p, uint32_t s, uint32_t v) {
  uint32_t page, pos;
  locate(p.geom, slot_ct<N2S>(p.geom, v), page, pos);
  return s * (uint32_t)p.cache.page_bytes + p.geom.adj_base + pos * p.geom.adj_stride;
}

template <bool N2S>
__device__ __forceinline__ uint32_t page_of(const PagedParams &p, uint32_t v) {
  return fastdiv(slot_ct<N2S>(p.geom, v), p.geom.rpp);
}

// Copy the 4 KB pages of completions i0 .. i0+3 (those below n; entry i in
// lane i of e) from the backing store into their cache slots: 16 loads in
// flight per lane, then the stores.  Kept out of line so the copy gets its
// own registers.
__device__ __attribute__((noinline)) void copy_pages4(const uint8_t *backing, __amdgpu_buffer_rsrc_t cache,
                                                      unsigned long long e, uint32_t i0, uint32_t n) {
  const int l = lane_id();
  const uint32_t i1 = min(i0 + 1, n - 1), i2 = min(i0 + 2, n - 1), i3 = min(i0 + 3, n - 1);
  const uint64_t e0 = readlane64(e, i0), e1 = readlane64(e, i1), e2 = readlane64(e, i2), e3 = readlane64(e, i3);
  const uint4 *s0 = reinterpret_cast<const uint4 *>(backing + (uint64_t)((uint32_t)(e0 >> 32) - 1u) * 4096u);
  const uint4 *s1 = reinterpret_cast<const uint4 *>(backing + (uint64_t)((uint32_t)(e1 >> 32) - 1u) * 4096u);
  const uint4 *s2 = reinterpret_cast<const uint4 *>(backing + (uint64_t)((uint32_t)(e2 >> 32) - 1u) * 4096u);
  const uint4 *s3 = reinterpret_cast<const uint4 *>(backing + (uint64_t)((uint32_t)(e3 >> 32) - 1u) * 4096u);
  const uint4 a0 = s0[l], a1 = s0[l + 64], a2 = s0[l + 128], a3 = s0[l + 192];
  const uint4 b0 = s1[l], b1 = s1[l + 64], b2 = s1[l + 128], b3 = s1[l + 192];
  const uint4 c0 = s2[l], c1 = s2[l + 64], c2 = s2[l + 128], c3 = s2[l + 192];
  const uint4 d0 = s3[l], d1 = s3[l + 64], d2 = s3[l + 128], d3 = s3[l + 192];
  const uint32_t lo = (uint32_t)l * 16u;
  uint32_t t = (uint32_t)e0 * 4096u + lo;
  coherent_store_u128(cache, t, a0); coherent_store_u128(cache, t + 1024, a1);
  coherent_store_u128(cache, t + 2048, a2); coherent_store_u128(cache, t + 3072, a3);
  if (i0 + 1 < n) {
    t = (uint32_t)e1 * 4096u + lo;
    coherent_store_u128(cache, t, b0); coherent_store_u128(cache, t + 1024, b1);
    coherent_store_u128(cache, t + 2048, b2); coherent_store_u128(cache, t + 3072, b3);
  }
  if (i0 + 2 < n) {
    t = (uint32_t)e2 * 4096u + lo;
    coherent_store_u128(cache, t, c0); coherent_store_u128(cache, t + 1024, c1);
    coherent_store_u128(cache, t + 2048, c2); coherent_store_u128(cache, t + 3072, c3);
  }
  if (i0 + 3 < n) {
    t = (uint32_t)e3 * 4096u + lo;
    coherent_store_u128(cache, t, d0); coherent_store_u128(cache, t + 1024, d1);
    coherent_store_u128(cache, t + 2048, d2); coherent_store_u128(cache, t + 3072, d3);
  }
}

// Mirror the host abort flag into HBM, where every wave polls it.
__device__ __forceinline__ void refresh_abort(const PagedParams &p) {
  if (__hip_atomic_load(p.abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != 0)
    atomicExch(p.abort_seen, 1u);
}

// Load completions [head, head + n) of a ring (entry i in lane i, n <= 64;
// entries are published before the tail that covers them).  Returns how many
// lead entries are well formed: a malformed one is never copied, so that the
// copy cannot leave the backing store or the cache; its waiter times out.
__device__ __forceinline__ uint32_t load_completions(const PagedParams &p, const unsigned long long *ring,
                                                     unsigned long long head, uint32_t n,
                                                     unsigned long long &e) {
  const int l = lane_id();
  e = 0;
  if ((uint32_t)l < n)
    e = __hip_atomic_load(&ring[(head + l) & p.cq_mask], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  const uint32_t pg = (uint32_t)(e >> 32) - 1u, sl = (uint32_t)e;
  const uint64_t mbad = ballot((uint32_t)l < n && (pg >= p.num_pages || sl >= p.cache.slots));
  if (mbad == 0) return n;
  if (l == 0) atomicAdd(&p.stats[10], (unsigned long long)__popcll(mbad));  // malformed completions
  return (uint32_t)__builtin_ctzll(mbad);
}

// Copy the pages of the completions in lanes [0, n) of e into their cache
// slots, kFillBatch at a time, and mark each batch READY once its bytes are
// performed device-wide.
__device__ __forceinline__ void fill_entries(const PagedParams &p, unsigned long long e, uint32_t n) {
  const int l = lane_id();
  const __amdgpu_buffer_rsrc_t crs = cache_rsrc(p.cache);
  for (uint32_t i0 = 0; i0 < n; i0 += kFillBatch) {
    if (p.cache.page_bytes == 4096) {
      copy_pages4(p.backing, crs, e, i0, n);
    } else {
      const uint32_t chunks = (uint32_t)(p.cache.page_bytes / 16);
      for (uint32_t i = i0; i < min(i0 + kFillBatch, n); ++i) {
        const uint64_t ei = readlane64(e, i);
        const uint4 *src = reinterpret_cast<const uint4 *>(p.backing + (uint64_t)((uint32_t)(ei >> 32) - 1u) *
                                                                           p.cache.page_bytes);
        const uint32_t base = (uint32_t)ei * (uint32_t)p.cache.page_bytes;
        for (uint32_t c = l; c < chunks; c += kWave) coherent_store_u128(crs, base + c * 16u, src[c]);
      }
    }
    wait_stores_performed();
    if ((uint32_t)l >= i0 && (uint32_t)l < min(i0 + kFillBatch, n))
      mark_ready(p.cache, (uint32_t)e);
  }
}

// Shared completion ring (no fill waves): claim up to kFillBatch completions
// and fill their pages.  Only the wave that wins the try-lock reads the
// proxy's tail from host memory; all others read its HBM mirror.
__device__ __forceinline__ uint32_t service_completions(const PagedParams &p) {
  const int l = lane_id();
  uint32_t n = 0;
  unsigned long long h = 0;
  if (l == 0) {
    h = __hip_atomic_load(p.cq_head, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    unsigned long long t = __hip_atomic_load(p.tail_seen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (h >= t && atomicCAS(p.poll_lock, 0u, 1u) == 0u) {
      t = __hip_atomic_load(p.cq_tail, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      atomicMax(p.tail_seen, t);
      refresh_abort(p);
      atomicExch(p.poll_lock, 0u);
    }
    if (h < t) {
      const unsigned long long want = min((unsigned long long)kFillBatch, t - h);
      if (atomicCAS(p.cq_head, h, h + want) == h) n = (uint32_t)want;
    }
  }
  n = first_lane_value(n);
  if (n == 0) return 0;
  h = readlane64(h, 0);
  unsigned long long e;
  n = load_completions(p, p.cq, h, n, e);  // a malformed entry stays claimed but unfilled
  fill_entries(p, e, n);
  return n;
}

// Frontier-to-LDS and back.
template <int KPL>
__device__ __forceinline__ void load_frontier(const QSlot<KPL> &S, uint64_t (&F)[KPL]) {
#pragma unroll
  for (int r = 0; r < KPL; ++r) F[r] = S.F[r * kWave + lane_id()];
}
template <int KPL>
__device__ __forceinline__ void store_frontier(QSlot<KPL> &S, const uint64_t (&F)[KPL]) {
#pragma unroll
  for (int r = 0; r < KPL; ++r) S.F[r * kWave + lane_id()] = F[r];
}

// Whether a parked query can make progress: a page it waits on is READY, or
// it has requests it may still issue.
template <int KPL>
__device__ __forceinline__ bool query_runnable(const PagedParams &p, const QSlot<KPL> &S) {
  const int l = lane_id();
  bool ready = false;
  uint32_t waiting = 0, todo = 0;
  if (S.phase == kPhExpand) {
    const uint32_t nb = min(S.nbeam - S.b0, min(kCandCap / p.R, (uint32_t)kPagedMaxW));
    if ((uint32_t)l < nb) {
      const uint32_t st = S.bstate[S.b0 + l];
      if (st < kDone) { ++waiting; ready = slot_ready(p.cache, st); }
      else if (st == kTodo) ++todo;
    }
  } else if (S.phase == kPhEval) {
    for (uint32_t c = l; c < S.ncand; c += kWave) {
      const uint32_t st = S.cstate[c];
      if (st < kDone) { ++waiting; ready |= slot_ready(p.cache, st); }
      else if (st == kTodo) ++todo;
    }
  } else {
    return true;
  }
  if (ballot(ready) != 0) return true;
  uint32_t nwait = 0, ntodo = 0;
  for (int m = 1; m < kWave; m <<= 1) {
    waiting += __shfl_xor(waiting, m);
    todo += __shfl_xor(todo, m);
  }
  nwait = waiting;
  ntodo = todo;
  if (p.blocking) return nwait == 0;
  return ntodo > 0 && nwait < p.max_pending;
}

// Start query qi in slot S: V = {entry}, and the entry is the first
// candidate to evaluate (the frontier is empty until it is).
template <int KPL>
__device__ __forceinline__ void admit_query(const PagedParams &p, QSlot<KPL> &S, uint32_t *ht, uint32_t qi) {
  const int l = lane_id();
  VisitedHbm<kPagedHtLog2>::clear(ht);
  if (l == 0) {
    S.qi = qi;
    S.active = 1;
    S.parked = 0;
    S.phase = kPhEval;
    S.nbeam = 0;
    S.b0 = 0;
    S.ncand = 1;
    S.cand[0] = p.entry;
    S.cstate[0] = kTodo;
    S.ht_used = 1;
    S.forgot = 0;
  }
#pragma unroll
  for (int r = 0; r < KPL; ++r) S.F[r * kWave + l] = kInfKey;
  __syncthreads();
  {
    uint32_t e1[1] = {p.entry};
    bool v1[1] = {l == 0}, n1[1], r1[1];
    VisitedHbm<kPagedHtLog2>::test_and_set_n<1>(ht, e1, v1, true, n1, r1);
  }
  __syncthreads();
}

// Runs one query until it finishes (returns true) or parks (false).
template <int KPL, class M, bool N2S>
__device__ bool run_query(const PagedParams &p, QSlot<KPL> &S, uint32_t *ht, uint32_t *qbuf, PagedCounters &ctr) {
  using HT = VisitedHbm<kPagedHtLog2>;
  const int l = lane_id();
  const uint32_t GB = min(kCandCap / p.R, (uint32_t)kPagedMaxW);
  constexpr int kIdsPerLane = kCandCap / kWave;
  const __amdgpu_buffer_rsrc_t crs = cache_rsrc(p.cache);

  M m;
  m.load_query(p.queries, S.qi, p.D, qbuf);
  if (l == 0) S.yielded = 0;
  __syncthreads();
  uint64_t F[KPL];
  load_frontier(S, F);
  uint32_t passes = 0;

  for (uint32_t guard = 0; guard < 4u * p.n + 16u; ++guard) {
    if (S.phase == kPhSelect) {
      uint32_t nbeam = 0;
#pragma unroll
      for (int r = 0; r < KPL; ++r) {
        const uint32_t e = r * kWave + l;
        bool unexp = e < p.L && F[r] != kInfKey && !(F[r] & 1ull);
        uint64_t m = ballot(unexp);
        uint32_t rank = nbeam + lanes_below(m);
        if (unexp && rank < p.W) {
          S.beam[rank] = key_id(F[r]);
          S.bstate[rank] = kTodo;
          F[r] |= 1ull;
        }
        nbeam += (uint32_t)__popcll(m);
      }
      nbeam = min(nbeam, p.W);
      if (nbeam == 0) {
#pragma unroll
        for (int r = 0; r < KPL; ++r) {
          const uint32_t e = r * kWave + l;
          if (e < p.k) {
            const bool ok = F[r] != kInfKey;
            p.out_ids[(uint64_t)S.qi * p.k + e] = ok ? key_id(F[r]) : kNoEdge;
            p.out_dists[(uint64_t)S.qi * p.k + e] = ok ? (uint32_t)(F[r] >> 32) : M::kPadDist;
          }
        }
        return true;
      }
      S.nbeam = nbeam;
      S.b0 = 0;
      S.ncand = 0;
      S.phase = kPhExpand;
      ctr.exp += nbeam;
      ++ctr.iter;
      __syncthreads();
    }

    if (S.phase == kPhExpand) {
      const uint32_t nb = min(S.nbeam - S.b0, GB);
      const bool mine = (uint32_t)l < nb;
      const uint32_t bi = S.b0 + min((uint32_t)l, nb - 1);
      uint32_t st = mine ? S.bstate[bi] : kDone;
      uint32_t slot = 0;
      bool ready = false;
      bool hit = false, miss = false;
      if (mine && st == kTodo) {
        bool issued;
        const uint32_t r = acquire_page(p.cache, page_of<N2S>(p, S.beam[bi]), true, slot, issued);
        if (r == kAcqReady) { ready = true; hit = true; }
        else if (r == kAcqWait) { st = slot; miss = true; }
      } else if (mine && st < kDone) {
        if (slot_ready(p.cache, st)) { ready = true; slot = st; }
      }
      ctr.hit += (uint32_t)__popcll(ballot(hit));
      ctr.miss += (uint32_t)__popcll(ballot(miss));
      if (mine && !ready) S.bstate[bi] = st;
      uint64_t rmask = ballot(ready);
      if (rmask) {
        order_after_ready();
        while (rmask) {
          const int b = __builtin_ctzll(rmask);
          rmask &= rmask - 1;
          const uint32_t s_b = readlane(slot, b);
          const uint32_t u = S.beam[S.b0 + b];
          const uint32_t adj = cached_adj<N2S>(p, s_b, u);
          const uint32_t deg = min(coherent_load_u32(crs, adj), p.R);
          for (uint32_t j0 = 0; j0 < p.R; j0 += kCandCap) {
            uint32_t ids[kIdsPerLane];
            bool valid[kIdsPerLane], isnew[kIdsPerLane], rec[kIdsPerLane];
#pragma unroll
            for (int t = 0; t < kIdsPerLane; ++t) {
              const uint32_t j = j0 + t * kWave + l;
              ids[t] = j < deg ? coherent_load_u32(crs, adj + 4u + 4u * j) : kNoEdge;
              valid[t] = ids[t] < p.n;
            }
            HT::template test_and_set_n<kIdsPerLane>(ht, ids, valid, S.ht_used < HT::kLimit, isnew, rec);
#pragma unroll
            for (int t = 0; t < kIdsPerLane; ++t) {
              const uint64_t mnew = ballot(isnew[t]);
              const uint64_t mrec = ballot(rec[t]);
              const uint32_t base = S.ncand;
              if (isnew[t]) {
                const uint32_t pos = base + lanes_below(mnew);
                S.cand[pos] = ids[t];
                S.cstate[pos] = kTodo;
              }
              S.ncand = base + (uint32_t)__popcll(mnew);
              S.ht_used += (uint32_t)__popcll(mrec);
              const uint32_t lost = (uint32_t)__popcll(mnew & ~mrec);
              ctr.reeval += lost;
              if (lost) S.forgot = 1;
            }
          }
          if (l == 0) {
            unpin(p.cache, s_b);
            S.bstate[S.b0 + b] = kDone;
          }
          __syncthreads();
        }
      }
      __syncthreads();
      const bool pending = mine && S.bstate[bi] != kDone;
      if (ballot(pending) != 0) break;  // park
      S.phase = kPhEval;
      __syncthreads();
    }

    if (S.phase == kPhEval) {
      // request or re-test every candidate; evaluate the resident ones
      uint32_t npend = 0;
      bool lane_waiting = false;
      for (uint32_t c = l; c < S.ncand; c += kWave) {
        const bool w = S.cstate[c] < kDone;
        npend += w ? 1u : 0u;
        lane_waiting |= w;
      }
      for (int m = 1; m < kWave; m <<= 1) npend += __shfl_xor(npend, m);
      uint32_t rslot[kIdsPerLane];
      bool rdy[kIdsPerLane];
#pragma unroll
      for (int t = 0; t < kIdsPerLane; ++t) {
        const uint32_t c = t * kWave + l;
        const bool mine = c < S.ncand;
        uint32_t st = mine ? S.cstate[c] : kDone;
        rdy[t] = false;
        rslot[t] = 0;
        // blocking: a lane keeps at most one page request outstanding
        const bool want = mine && st == kTodo && !(p.blocking && lane_waiting);
        const uint64_t mwant = ballot(want);
        const bool allowed = want && npend + lanes_below(mwant) < p.max_pending;
        bool waited = false, hit = false;
        if (allowed) {
          bool issued;
          uint32_t s;
          const uint32_t r = acquire_page(p.cache, page_of<N2S>(p, S.cand[c]), true, s, issued);
          if (r == kAcqReady) { rdy[t] = true; rslot[t] = s; hit = true; }
          else if (r == kAcqWait) { st = s; waited = true; }
        } else if (mine && st < kDone) {
          if (slot_ready(p.cache, st)) { rdy[t] = true; rslot[t] = st; }
        }
        if (mine && !rdy[t]) S.cstate[c] = st;
        lane_waiting |= waited;
        const uint32_t nw = (uint32_t)__popcll(ballot(waited));
        npend += nw;
        ctr.miss += nw;
        ctr.hit += (uint32_t)__popcll(ballot(hit));
      }
      // gather the ready candidates, 64 at a time
      bool any_ready = false;
#pragma unroll
      for (int t = 0; t < kIdsPerLane; ++t) any_ready |= ballot(rdy[t]) != 0;
      if (any_ready) {
        order_after_ready();
#pragma unroll
        for (int t = 0; t < kIdsPerLane; ++t) {
          const uint64_t mr = ballot(rdy[t]);
          if (mr == 0) continue;
          const uint32_t cnt = (uint32_t)__popcll(mr);
          uint64_t key = m.paged_keys([&](uint32_t si, uint32_t v) { return cached_vec<N2S>(p, si, v); }, crs,
                                      S.cand, t * kWave, rdy[t], rslot[t], mr);
          ctr.eval += cnt;
          merge_keys<KPL>(F, key, S.forgot != 0, p.L);
          if (rdy[t]) {
            unpin(p.cache, rslot[t]);
            S.cstate[t * kWave + l] = kDone;
          }
          __syncthreads();
        }
      }
      __syncthreads();
      bool left = false;
      for (uint32_t c = l; c < S.ncand; c += kWave) left |= S.cstate[c] != kDone;
      if (ballot(left) != 0) {
        // progress: pins were released, more requests may go out
        if (any_ready && (p.turn_passes == 0 || ++passes < p.turn_passes)) continue;
        if (any_ready && l == 0) S.yielded = 1;  // turn over, though it could go on
        break;                                   // park until a page arrives
      }
      // iteration group done
      S.b0 += min(S.nbeam - S.b0, GB);
      S.ncand = 0;
      S.phase = S.b0 < S.nbeam ? kPhExpand : kPhSelect;
      __syncthreads();
    }
  }
  store_frontier(S, F);
  __syncthreads();
  return false;
}

// Fill wave k: consumes completion ring k (its own: no atomics on the ring)
// and copies the pages until every query is done, or, with a budget, until
// the budget has passed (host-scheduled lanes run by a launch per round: the
// host launches the fill waves again, and they go on from the ring position
// they published, so no kernel of that mode ever waits for another stream's
// work).  Wave 0 also mirrors the host abort flag.
__device__ void fill_loop(const PagedParams &p, uint32_t k, const RunQueue *wake = nullptr) {
  const int l = lane_id();
  const unsigned long long *ring = p.cq + (uint64_t)k * (p.cq_mask + 1);
  const unsigned long long *tail = p.cq_tail + (uint64_t)k * p.tail_stride;
  unsigned long long *filled = p.fill_head ? p.fill_head + (uint64_t)k * p.tail_stride : nullptr;
  unsigned long long head = 0, served = 0;
  if (filled) {
    if (l == 0) head = __hip_atomic_load(filled, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    head = readlane64(head, 0);
  }
  const unsigned long long t_end = p.fill_budget ? (unsigned long long)wall_clock64() + p.fill_budget : ~0ull;
  uint32_t idle = 0;
  for (;;) {
    if (k == 0 && l == 0) refresh_abort(p);
    if (aborted(p)) break;
    if (__hip_atomic_load(p.done_queries, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= p.nq) break;
    if (p.fill_budget && (unsigned long long)wall_clock64() >= t_end) break;
    unsigned long long t = 0;
    if (l == 0) t = __hip_atomic_load(tail, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    t = readlane64(t, 0);
    if (t <= head) {
      if (++idle > 8) __builtin_amdgcn_s_sleep(2);
      continue;
    }
    idle = 0;
    while (head < t) {
      const uint32_t n = (uint32_t)min((unsigned long long)kWave, t - head);
      unsigned long long e;
      const uint32_t good = load_completions(p, ring, head, n, e);
      fill_entries(p, e, good);
      if (wake) wake_filled(p, *wake, e, good);
      served += good;
      head += good < n ? good + 1 : n;  // step over a malformed entry
    }
    // host-scheduled lanes: entries [0, head) of this ring are now READY
    if (filled && l == 0) __hip_atomic_store(filled, head, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
  }
  if (l == 0) atomicAdd(&p.stats[6], served);
}

template <int KPL, class M, bool N2S>
__global__ __launch_bounds__(kWave) void search_paged(PagedParams p) {
  // fill waves take the lowest block indices, so they are dispatched first
  if (blockIdx.x < p.fill_waves) {
    fill_loop(p, blockIdx.x);
    return;
  }
  const uint32_t qb = blockIdx.x - p.fill_waves;
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ __align__(16) uint32_t qbuf[M::kQueryWords];
  QSlot<KPL> *slots = reinterpret_cast<QSlot<KPL> *>(lds);
  const int l = lane_id();
  for (uint32_t j = 0; j < p.oversub; ++j) {
    if (l == 0) {
      slots[j].active = 0;
      slots[j].parked = 0;
    }
  }
  __syncthreads();
  PagedCounters ctr;
  bool admitting = true;
  uint32_t idle = 0;
  for (;;) {
    if (aborted(p)) break;
    bool any_active = false, progressed = false;
    for (uint32_t j = 0; j < p.oversub; ++j) {
      QSlot<KPL> &S = slots[j];
      uint32_t *ht = p.ht_pool + ((uint64_t)(qb * p.oversub + j) << kPagedHtLog2);
      if (!S.active) {
        if (!admitting) continue;
        uint32_t qi = 0;
        if (l == 0) qi = atomicAdd(p.next_query, 1u);
        qi = first_lane_value(qi);
        if (qi >= p.nq) {
          admitting = false;
          continue;
        }
        if (p.order) qi = first_lane_value(p.order[qi]);
        admit_query(p, S, ht, qi);
      } else if (S.parked) {
        any_active = true;
        if (!query_runnable(p, S)) continue;
        ++ctr.resume;
      }
      any_active = true;
      const bool done = run_query<KPL, M, N2S>(p, S, ht, qbuf, ctr);
      progressed = true;
      if (l == 0) {
        if (done) {
          S.active = 0;
          S.parked = 0;
          atomicAdd(p.done_queries, 1u);
        } else {
          S.parked = 1;
        }
      }
      if (!done) ++ctr.park;
      __syncthreads();
    }
    if (!any_active && !admitting) break;
    const uint32_t served = p.fill_waves ? 0u : service_completions(p);
    ctr.served += served;
    if (!progressed && served == 0) {
      if (++idle > 4) __builtin_amdgcn_s_sleep(2);
    } else {
      idle = 0;
    }
  }
  // A wave leaves only when none of its queries is active: every page any
  // query waits on has a waiting wave that keeps serving completions.
  if (l == 0) {
    atomicAdd(&p.stats[0], ctr.eval);
    atomicAdd(&p.stats[1], ctr.reeval);
    atomicAdd(&p.stats[2], ctr.exp);
    atomicAdd(&p.stats[3], ctr.iter);
    atomicAdd(&p.stats[4], ctr.hit);
    atomicAdd(&p.stats[5], ctr.miss);
    atomicAdd(&p.stats[6], ctr.served);
    atomicAdd(&p.stats[7], ctr.park);
    atomicAdd(&p.stats[8], ctr.resume);
  }
}


// ---------------------------------------------------------------------------
// Host-scheduled lanes (the host-scheduled comparison point of Sec. 5.1: a
// query scheduler on the host coordinates many query lanes, over the same GPU
// page cache, miss descriptors and proxy).  The host keeps the lanes' states
// in HBM and chooses which lane runs next; a turn runs the lane until its
// query finishes or parks (or yields) and reports what the lane now waits for.
// Turns are run by a persistent launch that takes them from a ring the host
// writes, or by one launch per round with a workgroup per chosen lane.  Fill
// waves (in the persistent launch, or in a kernel of their own beside the
// rounds) publish how far each completion ring has been filled, which is the
// completion state the host schedules from.
// ---------------------------------------------------------------------------
constexpr uint32_t kLaneWaitCap = 60;
enum : uint32_t { kLaneIdle = 0, kLaneParked = 1, kLaneDone = 2, kLaneYield = 3 };

// What a lane reported at the end of its turn (host memory, one per lane).
struct LaneOut {
  uint32_t code;                 // kLaneIdle (not runnable, not run), kLaneParked, kLaneDone, kLaneYield
                                 // (its turn ended while it could still proceed)
  uint32_t nwait;                // entries of wait[]
  uint32_t retry;                // 1: can proceed without one of wait[] arriving (requests it could
                                 // not issue for want of a free slot, or more waits than wait[] holds)
  uint32_t qi;                   // the lane's query
  uint32_t seq;                  // turns the lane has finished; written last, with a system-scope
                                 // release, so a new value means the report and the lane's state
                                 // in HBM are complete (the host need not wait for the launch)
  uint32_t wait[kLaneWaitCap];   // cache slots of the pages the lane waits for
};

struct RoundParams {
  const uint32_t *lanes;   // this launch's lanes, one per workgroup (host memory); nullptr: a
                           // persistent launch that takes its lanes from the run ring below
  const uint32_t *admit;   // per entry: query to start in the lane, or kNone to resume it
  uint32_t *state;         // per lane: its QSlot, state_words 32-bit words (HBM)
  uint32_t state_words;
  LaneOut *out;            // per lane (host memory)
  // persistent launch: blocks [0, fill_waves) fill pages, block fill_waves
  // mirrors the run ring's tail into device memory (so that idle waves poll
  // HBM, not the host link), the others run lane turns in the order the host
  // writes them to the run ring
  const unsigned long long *runq;       // host memory: (query + 1) << 32 | (lane + 1), query 0 = resume
  const unsigned long long *runq_tail;  // host memory: entries written
  unsigned long long *runq_tail_seen;   // device: its mirror
  unsigned long long *runq_head;        // device: entries taken
  uint32_t runq_mask;
  uint32_t out_lanes;                   // lanes (bounds the ring's lane ids)
};

// Record which cache slots a parked lane waits for.
template <int KPL>
__device__ __forceinline__ void report_waits(const PagedParams &p, const QSlot<KPL> &S, LaneOut &o, uint32_t code) {
  const int l = lane_id();
  const uint32_t *items = S.cstate;
  uint32_t n = 0;
  if (S.phase == kPhExpand) {
    items = S.bstate + S.b0;
    n = min(S.nbeam - S.b0, min(kCandCap / p.R, (uint32_t)kPagedMaxW));
  } else if (S.phase == kPhEval) {
    n = S.ncand;
  }
  uint32_t cnt = 0, todo = 0;
  for (uint32_t base = 0; base < n; base += kWave) {
    const uint32_t c = base + l;
    const uint32_t st = c < n ? items[c] : kDone;
    const bool w = st < kDone;
    const uint64_t mw = ballot(w);
    const uint32_t pos = cnt + lanes_below(mw);
    if (w && pos < kLaneWaitCap) o.wait[pos] = st;
    cnt += (uint32_t)__popcll(mw);
    todo += (uint32_t)__popcll(ballot(st == kTodo));
  }
  if (l == 0) {
    o.nwait = min(cnt, kLaneWaitCap);
    o.retry = (cnt > kLaneWaitCap || (todo > 0 && cnt < p.max_pending)) ? 1u : 0u;
    o.qi = S.qi;
    o.code = code;
  }
}

// One turn of lane `lane` (a new query qa, or kNone to go on with the one
// it holds): load its state, run until it parks, yields or finishes, store
// the state and report.
template <int KPL, class M, bool N2S>
__device__ void lane_turn(const PagedParams &p, const RoundParams &r, uint32_t lane, uint32_t qa,
                          unsigned char *lds, uint32_t *qbuf) {
  QSlot<KPL> &S = *reinterpret_cast<QSlot<KPL> *>(lds);
  uint32_t *sw = reinterpret_cast<uint32_t *>(lds);
  const int l = lane_id();
  uint32_t *ht = p.ht_pool + ((uint64_t)lane << kPagedHtLog2);
  uint32_t *st = r.state + (uint64_t)lane * r.state_words;
  LaneOut &o = r.out[lane];
  uint32_t seq0 = 0;
  if (l == 0) seq0 = __hip_atomic_load(&o.seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  // the turn is over: everything this wave wrote (the lane's state in HBM,
  // its report in host memory, the counters) is performed before the new
  // sequence number can be seen
  auto finish_turn = [&]() {
    if (l == 0) __hip_atomic_store(&o.seq, seq0 + 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
  };
  if (aborted(p)) {
    if (l == 0) {
      o.code = kLaneIdle;
      o.nwait = 0;
      o.retry = 1;
    }
    finish_turn();
    return;
  }
  PagedCounters ctr;
  if (qa != kNone) {
    admit_query(p, S, ht, qa);
  } else {
    for (uint32_t i = l; i < r.state_words; i += kWave) sw[i] = st[i];
    __syncthreads();
    if (!query_runnable(p, S)) {
      report_waits(p, S, o, kLaneIdle);
      finish_turn();
      return;
    }
    ++ctr.resume;
  }
  const bool done = run_query<KPL, M, N2S>(p, S, ht, qbuf, ctr);
  if (done) {
    if (l == 0) {
      atomicAdd(p.done_queries, 1u);
      o.nwait = 0;
      o.retry = 0;
      o.qi = S.qi;
      o.code = kLaneDone;
    }
  } else {
    ++ctr.park;
    __syncthreads();
    for (uint32_t i = l; i < r.state_words; i += kWave) st[i] = sw[i];
    report_waits(p, S, o, S.yielded ? kLaneYield : kLaneParked);
  }
  if (l == 0) {
    if (ctr.eval) atomicAdd(&p.stats[0], ctr.eval);
    if (ctr.reeval) atomicAdd(&p.stats[1], ctr.reeval);
    if (ctr.exp) atomicAdd(&p.stats[2], ctr.exp);
    if (ctr.iter) atomicAdd(&p.stats[3], ctr.iter);
    if (ctr.hit) atomicAdd(&p.stats[4], ctr.hit);
    if (ctr.miss) atomicAdd(&p.stats[5], ctr.miss);
    if (ctr.park) atomicAdd(&p.stats[7], ctr.park);
    if (ctr.resume) atomicAdd(&p.stats[8], ctr.resume);
  }
  finish_turn();
}

template <int KPL, class M, bool N2S>
__global__ __launch_bounds__(kWave) void paged_round(PagedParams p, RoundParams r) {
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ __align__(16) uint32_t qbuf[M::kQueryWords];
  if (r.lanes) {  // one lane per workgroup
    lane_turn<KPL, M, N2S>(p, r, r.lanes[blockIdx.x], r.admit[blockIdx.x], lds, qbuf);
    return;
  }
  if (blockIdx.x < p.fill_waves) {
    fill_loop(p, blockIdx.x);
    return;
  }
  const int l = lane_id();
  auto all_done = [&]() {
    return __hip_atomic_load(p.done_queries, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= p.nq;
  };
  uint32_t idle = 0;
  if (blockIdx.x == p.fill_waves) {  // the tail mirror
    unsigned long long seen = 0;
    while (!aborted(p) && !all_done()) {
      unsigned long long t = 0;
      if (l == 0) t = __hip_atomic_load(r.runq_tail, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM);
      t = readlane64(t, 0);
      if (t != seen) {
        if (l == 0) __hip_atomic_store(r.runq_tail_seen, t, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        seen = t;
        idle = 0;
      } else if (++idle > 8) {
        __builtin_amdgcn_s_sleep(1);
      }
    }
    return;
  }
  // executor: take the next entry of the run ring, run that lane's turn; leave
  // when every query is done (nothing more can be written) or on abort
  for (;;) {
    if (aborted(p)) break;
    int got = 0;
    unsigned long long idx = 0;
    if (l == 0) {
      const unsigned long long h = __hip_atomic_load(r.runq_head, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const unsigned long long t = __hip_atomic_load(r.runq_tail_seen, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
      if (h < t) {
        if (atomicCAS(r.runq_head, h, h + 1) == h) {
          got = 1;
          idx = h;
        }
      } else if (all_done()) {
        got = -1;
      }
    }
    got = __shfl(got, 0);
    if (got < 0) break;
    if (got == 0) {
      if (++idle > 8) __builtin_amdgcn_s_sleep(2);
      continue;
    }
    idle = 0;
    idx = readlane64(idx, 0);
    unsigned long long e = 0;
    if (l == 0) e = __hip_atomic_load(&r.runq[idx & r.runq_mask], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    e = readlane64(e, 0);
    const uint32_t lane = (uint32_t)e - 1u, q1 = (uint32_t)(e >> 32);
    if ((uint32_t)e == 0u || lane >= r.out_lanes) break;  // malformed: leave (the watchdog ends the search)
    // the lane's state and visited table were written by whichever wave ran
    // its last turn, which released them before its report
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    lane_turn<KPL, M, N2S>(p, r, lane, q1 ? q1 - 1u : kNone, lds, qbuf);
  }
}

// GPU resume queue: blocks [0, fill_waves) fill pages and queue the lanes
// parked on them; the others are executors.  An executor takes a queued lane
// (or, while there are lanes that never ran, hands the next lane the next
// query), runs its turn, and acts on the lane's report: a finished lane takes
// the next query at once, a lane that can go on is queued again, and a lane
// that waits for pages parks on their slots.  Every wait ends when every
// query is done or on abort.
template <int KPL, class M, bool N2S>
__global__ __launch_bounds__(kWave) void paged_queue(PagedParams p, RoundParams r, RunQueue q) {
  extern __shared__ __align__(16) unsigned char lds[];
  __shared__ __align__(16) uint32_t qbuf[M::kQueryWords];
  if (blockIdx.x < p.fill_waves) {
    fill_loop(p, blockIdx.x, &q);
    return;
  }
  const int l = lane_id();
  auto stop = [&]() { return queue_done(p); };
  uint32_t idle = 0;
  while (!queue_done(p)) {
    // a queued lane, else a lane that has not run yet
    uint32_t lane = kNoLane, qa = kNone;
    if (l == 0) {
      lane = queue_take(q, stop);
      if (lane == kNoLane) {
        const uint32_t nl = take_fresh_lane(q);
        if (nl != kNoLane) {
          const uint32_t qi = atomicAdd(p.next_query, 1u);
          if (qi < p.nq) {
            lane = nl;
            qa = p.order ? p.order[qi] : qi;
          }
        }
      }
    }
    lane = first_lane_value(lane);
    qa = first_lane_value(qa);
    if (lane >= q.lanes) {  // nothing to run (kNoLane), or not a lane
      if (++idle > 8) __builtin_amdgcn_s_sleep(2);
      continue;
    }
    idle = 0;
    if (l == 0) lane_running(q, lane);
    // the lane's state and visited table were written by the wave that ran
    // its last turn, released before the lane was queued
    GORIO_QUEUE_FENCE_ACQ();
    if (qa == kNone) {  // resumed: leave the waiter sets of the slots it parked on
      const LaneOut &o = r.out[lane];
      const uint32_t nw = min(o.nwait, kLaneWaitCap);
      const uint32_t sl = (uint32_t)l < nw ? o.wait[l] : kNone;
      if (sl < p.cache.slots) park_withdraw(q, lane, sl);
    }
    for (;;) {
      lane_turn<KPL, M, N2S>(p, r, lane, qa, lds, qbuf);
      // the report (written by several lanes of this wave) is complete and read from L2
      GORIO_QUEUE_FENCE_REL();
      __syncthreads();
      GORIO_QUEUE_FENCE_ACQ();
      const LaneOut &o = r.out[lane];
      const uint32_t code = o.code;
      if (code == kLaneDone) {
        uint32_t qi = 0;
        if (l == 0) qi = atomicAdd(p.next_query, 1u);
        qi = first_lane_value(qi);
        if (qi >= p.nq) break;  // the lane retires
        qa = p.order ? p.order[qi] : qi;
        continue;
      }
      if (aborted(p)) break;
      const uint32_t nw = min(o.nwait, kLaneWaitCap);
      if (code == kLaneYield || o.retry || nw == 0) {
        // it can go on without a page arriving (or could not report them all)
        GORIO_QUEUE_FENCE_REL();
        if (l == 0) requeue_lane(q, lane, stop);
        break;
      }
      // park: PARKED, then the bits, then a second look at the slots.  Each
      // lane of the wave takes its wait entry (at most one: the report holds
      // fewer waits than a wave has lanes) before the lane can be woken: from
      // then on another executor may run it and rewrite its report.
      static_assert(kLaneWaitCap <= kWave, "one wait entry per lane of the wave");
      const uint32_t sl = (uint32_t)l < nw ? o.wait[l] : kNone;
      const bool mine = sl < p.cache.slots;
      if (l == 0) park_begin(q, lane);
      GORIO_QUEUE_FENCE_REL();
      if (mine) park_wait_on(q, lane, sl);
      GORIO_QUEUE_FENCE_SEQ();
      const bool ready = mine && slot_ready(p.cache, sl);
      if (ballot(ready) != 0 && l == 0) park_recheck_wake(q, lane, stop);
      break;
    }
  }
}

}  // namespace gorio
