// Shared device-side definitions: record addressing, fast division and the
// per-wave visited filter.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wave.hpp"

namespace gorio {

constexpr uint32_t kNoEdge = 0xFFFFFFFFu;
constexpr uint32_t kHtEmpty = 0xFFFFFFFFu;
constexpr int kCandCap = 256;  // candidate ids gathered per beam group
constexpr int kMaxW = 256;

// floor(x / d) for x < 2^31 with one 64-bit multiply:  m = ceil(2^(31+s) / d),
// s = ceil(log2 d), q = (x * m) >> (31 + s)  (Granlund & Montgomery, PLDI 1994).
struct FastDiv {
  uint32_t d;
  uint32_t mul;
  uint32_t shift;  // 31 + s
};

inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t s = 0;
  while ((1ull << s) < d) ++s;
  FastDiv f;
  f.d = d;
  f.shift = 31 + s;
  f.mul = (uint32_t)(((1ull << (31 + s)) + d - 1) / d);
  return f;
}

__host__ __device__ __forceinline__ uint32_t fastdiv(uint32_t x, FastDiv f) {
  return (uint32_t)(((uint64_t)x * f.mul) >> f.shift);
}

// Where a node's vector and adjacency block (degree, ids) sit inside the
// packed page array.  Slot s is position i = s % rpp of page s / rpp:
//   vector    at page * page_bytes + i * vec_stride
//   adjacency at page * page_bytes + adj_base + i * adj_stride
// Contiguous records: vec_stride = adj_stride = record_bytes, adj_base =
// vec_bytes.  Vectors first: vec_stride = vec_bytes rounded up to 16,
// adj_base = rpp * vec_stride, adj_stride = record_bytes - vec_stride.
struct PageGeom {
  uint64_t page_bytes;
  uint32_t record_bytes;
  uint32_t vec_bytes;
  uint32_t vec_stride;
  uint32_t adj_base;
  uint32_t adj_stride;
  FastDiv rpp;             // records per page
  const uint32_t *node_to_slot;  // nullptr: slot = node id
  // 16-byte units: when every vector starts on a 16-byte boundary and the
  // index spans at most 4 GiB (units16 != 0: a buffer instruction's byte
  // offset, index x stride, is 32 bits), a vector is also named by its
  // locator page * page16 + i * vec16, the index of its first unit.
  uint32_t units16;
  FastDiv page16;          // page_bytes / 16
  FastDiv vec16;           // vec_stride / 16
};

__device__ __forceinline__ uint32_t slot_of(const PageGeom &g, uint32_t v) {
  return g.node_to_slot ? g.node_to_slot[v] : v;
}

// Page of slot s and its position inside the page.
__device__ __forceinline__ void locate(const PageGeom &g, uint32_t s, uint32_t &page, uint32_t &pos) {
  page = fastdiv(s, g.rpp);
  pos = s - page * g.rpp.d;
}

// Slot of node v when the caller knows at compile time whether a placement
// permutation exists (keeps the permutation load out of paths without one,
// so dependent record loads need not wait on it).
template <bool N2S>
__device__ __forceinline__ uint32_t slot_ct(const PageGeom &g, uint32_t v) {
  if constexpr (N2S) return g.node_to_slot[v];
  else return v;
}

// 16-byte load through a structured buffer resource: address = base +
// vindex * stride (the stride is part of the resource); an index at or past
// the resource's record count reads zeros instead of faulting.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ u32x4_t struct_buffer_load_b128(__amdgpu_buffer_rsrc_t rsrc, int vindex, int voffset, int soffset,
                                           int aux) __asm("llvm.amdgcn.struct.ptr.buffer.load.v4i32");

// The packed pages as 16-byte records (units16 != 0).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t units16_rsrc(const uint8_t *pages, const PageGeom &g) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(pages), (short)16, (int)g.units16, 0x00020000);
}

// Locator of slot s's vector (units16 != 0) and the slot a locator names.
__device__ __forceinline__ uint32_t vec_locator(const PageGeom &g, uint32_t s) {
  uint32_t page, pos;
  locate(g, s, page, pos);
  return page * g.page16.d + pos * g.vec16.d;
}
__device__ __forceinline__ uint32_t slot_of_locator(const PageGeom &g, uint32_t loc) {
  const uint32_t page = fastdiv(loc, g.page16);
  return page * g.rpp.d + fastdiv(loc - page * g.page16.d, g.vec16);
}

// Byte offsets of slot s's vector and adjacency block in the packed page array.
__device__ __forceinline__ uint64_t vec_offset(const PageGeom &g, uint32_t s) {
  uint32_t page, pos;
  locate(g, s, page, pos);
  return (uint64_t)page * g.page_bytes + (uint64_t)(pos * g.vec_stride);
}
__device__ __forceinline__ uint64_t adj_offset(const PageGeom &g, uint32_t s) {
  uint32_t page, pos;
  locate(g, s, page, pos);
  return (uint64_t)page * g.page_bytes + (uint64_t)(g.adj_base + pos * g.adj_stride);
}

// ---------------------------------------------------------------------------
// Visited filter in LDS, one table per wave: open addressing over buckets of
// four 32-bit slots (16 bytes, read with one ds_read_b128), linear probing
// from bucket to bucket.  An id is inserted into the first empty slot of the
// first bucket on its probe path that has one; slots are never freed, so a
// bucket seen with an empty slot and without the id proves the id absent.
// It may forget (a full table stops recording) but never invents a member, so
// a node is at worst evaluated twice; the frontier merge removes the copy.
// ---------------------------------------------------------------------------
template <int LOG2>
struct VisitedLds {
  static constexpr uint32_t kSize = 1u << LOG2;         // slots
  static constexpr uint32_t kWords = kSize;             // 32-bit LDS words
  static constexpr uint32_t kMaxId = 0xFFFFFFFFu;       // any id below kHtEmpty
  static constexpr uint32_t kBuckets = kSize / 4;
  static constexpr uint32_t kLimit = kSize - kSize / 4;  // stop recording at 75% load
  static constexpr int kMaxRounds = 64;

  __device__ __forceinline__ static uint32_t bucket(uint32_t id) {
    return (id * 0x9E3779B1u) >> (32 - (LOG2 - 2));
  }

  __device__ __forceinline__ static void clear(uint32_t *t) {
    uint4 *t4 = reinterpret_cast<uint4 *>(t);
    const uint4 e = make_uint4(kHtEmpty, kHtEmpty, kHtEmpty, kHtEmpty);
    for (uint32_t i = lane_id(); i < kBuckets; i += kWave) t4[i] = e;
  }

  // Bit j set: slot j of bucket v holds x.
  __device__ __forceinline__ static uint32_t match4(const uint4 &v, uint32_t x) {
    return (uint32_t)(v.x == x) | ((uint32_t)(v.y == x) << 1) | ((uint32_t)(v.z == x) << 2) |
           ((uint32_t)(v.w == x) << 3);
  }

  // One id (wave-uniform call, any lane mask): true when id was not recorded
  // before (evaluate it); `recorded` tells whether this call stored it.
  __device__ __forceinline__ static bool test_and_set(uint32_t *t, uint32_t id, bool may_store,
                                                       bool &recorded) {
    uint32_t ids[1] = {id};
    bool valid[1] = {true}, isnew[1], rec[1];
    test_and_set_n<1>(t, ids, valid, may_store, isnew, rec);
    recorded = rec[0];
    return isnew[0];
  }

  // N ids per lane at once: each round reads every pending id's bucket, then
  // claims the first empty slot with one LDS CAS.  isnew[i]: evaluate
  // ids[i]; recorded[i]: this call stored it.
  template <int N>
  __device__ __forceinline__ static void test_and_set_n(uint32_t *t, const uint32_t (&ids)[N],
                                                        const bool (&valid)[N], bool may_store,
                                                        bool (&isnew)[N], bool (&recorded)[N]) {
    const uint4 *t4 = reinterpret_cast<const uint4 *>(t);
    uint32_t b[N];
    bool pend[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
      b[i] = bucket(ids[i]);
      pend[i] = valid[i];
      isnew[i] = false;
      recorded[i] = false;
    }
    for (int round = 0; round < kMaxRounds; ++round) {
      bool any = false;
#pragma unroll
      for (int i = 0; i < N; ++i) any |= pend[i];
      if (ballot(any) == 0) break;
      uint4 v[N];
#pragma unroll
      for (int i = 0; i < N; ++i) {
        v[i] = make_uint4(kHtEmpty, kHtEmpty, kHtEmpty, kHtEmpty);
        if (pend[i]) v[i] = t4[b[i]];
      }
      // branch-free decision per id: recorded already / bucket full / absent
      bool cas[N];
      uint32_t slot[N];
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const uint32_t hitm = match4(v[i], ids[i]);
        const uint32_t emptym = match4(v[i], kHtEmpty);
        const bool absent = pend[i] && hitm == 0 && emptym != 0;
        const bool full = pend[i] && hitm == 0 && emptym == 0;
        cas[i] = absent && may_store;
        isnew[i] = isnew[i] || (absent && !may_store);
        slot[i] = b[i] * 4 + (uint32_t)__builtin_ctz(emptym | 16u);
        b[i] = full ? ((b[i] + 1) & (kBuckets - 1)) : b[i];
        pend[i] = full || cas[i];
      }
      uint32_t old[N];
#pragma unroll
      for (int i = 0; i < N; ++i) {
        old[i] = 0;
        if (cas[i]) old[i] = atomicCAS(&t[slot[i]], kHtEmpty, ids[i]);
      }
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const bool won = cas[i] && old[i] == kHtEmpty;
        const bool same = cas[i] && old[i] == ids[i];  // another lane recorded the same id
        isnew[i] = isnew[i] || won;
        recorded[i] = recorded[i] || won;
        pend[i] = pend[i] && !won && !same;           // lost the slot: read the bucket again
      }
    }
#pragma unroll
    for (int i = 0; i < N; ++i)
      if (pend[i]) isnew[i] = true;  // round limit: evaluate, unrecorded
  }
};

// Per-half unsigned minimum of two words (v_pk_min_u16), and a 24-bit
// multiply (v_mul_u32_u24: full rate, where a 32-bit multiply is not).
// Written as instructions so that the compiler keeps them as one operation
// instead of expanding them per half.
__device__ __forceinline__ uint32_t pk_min_u16(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_pk_min_u16 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ uint32_t mul_u24(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_mul_u32_u24 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// Compact visited filter in LDS: 16-bit entries, buckets of eight half-words
// (16 bytes, one ds_read_b128): seven id slots and, in the top half of the
// last word, a count of the claims made on the bucket.  Ids must be below
// 2^(LOG2 + 11) (2^23 for 4096 entries).  h = (id * odd) mod 2^(LOG2 + 11) is
// a bijection; its top LOG2 - 3 bits pick the home bucket, its low 14 bits r
// are stored as 1 + (d << 14 | r), where d in {0, 1} is the bucket's distance
// from home (0 marks an empty slot).  (bucket - d, r) gives back h, so an
// entry matches exactly one id: the filter never invents a member.
//
// An id lives in its home bucket unless that bucket was full when it was
// inserted, then in the next one; claims never decrease, so a home bucket
// with fewer than seven claims that lacks the id proves it absent.  Lanes
// that insert into the same bucket take distinct slots from one LDS atomic
// add on the claim count (no retries); lanes holding the same id then see,
// on reading the bucket back, whether a lower slot already holds it, and
// only the lowest keeps it.  Both buckets are read up front, so every call
// takes one round.  An id whose two buckets are full is not recorded (it may
// be evaluated again; the frontier merge drops the copy).
template <int LOG2>
struct VisitedLds16 {
  static constexpr uint32_t kSize = 1u << LOG2;          // 16-bit half-words
  static constexpr uint32_t kWords = kSize / 2;          // 32-bit LDS words
  static constexpr uint32_t kBuckets = kSize / 8;
  static constexpr uint32_t kSlots = 7;                  // id slots per bucket
  static constexpr uint32_t kLimit = kBuckets * kSlots;  // records at most this many ids
  static constexpr int kHomeBits = LOG2 - 3;
  // The hash h = id * odd constant mod 2^kHashBits is one-to-one, and
  // (home bucket, entry) = (h >> 14, 1 + (h & 0x3FFF)) names the id.  The
  // multiply reads the low 24 bits of the id, so ids must also be below 2^24.
  static constexpr int kHashBits = kHomeBits + 14;
  static constexpr uint32_t kMaxId = 1u << (kHashBits < 24 ? kHashBits : 24);  // ids must be below this

  __device__ __forceinline__ static void clear(uint32_t *t) {
    uint4 *t4 = reinterpret_cast<uint4 *>(t);
    for (uint32_t i = lane_id(); i < kBuckets; i += kWave) t4[i] = make_uint4(0u, 0u, 0u, 0u);
  }

  __device__ __forceinline__ static bool test_and_set(uint32_t *t, uint32_t id, bool may_store,
                                                       bool &recorded) {
    uint32_t ids[1] = {id};
    bool valid[1] = {true}, isnew[1], rec[1];
    test_and_set_n<1>(t, ids, valid, may_store, isnew, rec);
    recorded = rec[0];
    return isnew[0];
  }

  // Whether a bucket's id slots below `below` (0..7) hold entry e: a half
  // equals e iff that half of w ^ (e * 0x10001) is zero; halves at or above
  // `below`, and the claim count, are forced to 0xFFFF (never an entry).
  __device__ __forceinline__ static bool holds(const uint4 &v, uint32_t e, uint32_t below) {
    const uint32_t ee = e * 0x10001u;
    const uint64_t lo = ((uint64_t)v.y << 32) | v.x;                     // slots 0..3
    const uint64_t hi = ((uint64_t)(v.w | 0xFFFF0000u) << 32) | v.z;     // slots 4..6, count
    const uint32_t bl = below < 4u ? below : 4u, bh = below > 4u ? below - 4u : 0u;
    const uint64_t mlo = bl >= 4u ? 0ull : ~0ull << (16u * bl);
    const uint64_t mhi = ~0ull << (16u * bh);
    const uint64_t xlo = (lo | mlo) ^ (((uint64_t)ee << 32) | ee);
    const uint64_t xhi = (hi | mhi) ^ (((uint64_t)ee << 32) | ee);
    const uint32_t m = pk_min_u16(pk_min_u16((uint32_t)xlo, (uint32_t)(xlo >> 32)),
                                  pk_min_u16((uint32_t)xhi, (uint32_t)(xhi >> 32)));
    return (m & 0xFFFFu) == 0 || (m >> 16) == 0;
  }

  // Same contract as VisitedLds::test_and_set_n (ids below kMaxId).
  template <int N>
  __device__ __forceinline__ static void test_and_set_n(uint32_t *t, const uint32_t (&ids)[N],
                                                        const bool (&valid)[N], bool may_store,
                                                        bool (&isnew)[N], bool (&recorded)[N]) {
    const uint4 *t4 = reinterpret_cast<const uint4 *>(t);
    uint16_t *t16 = reinterpret_cast<uint16_t *>(t);
    uint32_t bk[N], e[N], slot[N];
    bool claim[N], won[N], over[N];
    uint4 v0[N], v1[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
      // v_mul_u32_u24 reads the low 24 bits of each operand: exact for ids
      // below 2^24; an invalid lane's id only picks some bucket to read
      const uint32_t h = mul_u24(ids[i], 0x9E3779B1u & 0xFFFFFFu) & ((1u << kHashBits) - 1);
      bk[i] = h >> 14;
      e[i] = 1u + (h & 0x3FFFu);
      v0[i] = t4[bk[i]];
      v1[i] = t4[(bk[i] + 1) & (kBuckets - 1)];
    }
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const bool hit0 = holds(v0[i], e[i], kSlots);
      const bool hit1 = holds(v1[i], e[i] + (1u << 14), kSlots);
      const bool full0 = (v0[i].w >> 16) >= kSlots, full1 = (v1[i].w >> 16) >= kSlots;
      // present: in home, or in the next bucket when home was full
      const bool present = hit0 || (full0 && hit1);
      const bool absent = valid[i] && !present;
      const bool lost = absent && full0 && full1;          // nowhere to record it
      claim[i] = absent && !lost && may_store;
      isnew[i] = absent && (lost || !may_store);
      recorded[i] = false;
      // claim in home when it had room, else in the next bucket
      const uint32_t d = full0 ? 1u : 0u;
      bk[i] = (bk[i] + d) & (kBuckets - 1);
      e[i] += d << 14;
    }
    asm volatile("" ::: "memory");  // the claims follow the bucket reads
    uint32_t old[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
      old[i] = 0;
      if (claim[i]) old[i] = atomicAdd(&t[bk[i] * 4 + 3], 0x10000u);
    }
#pragma unroll
    for (int i = 0; i < N; ++i) {
      slot[i] = old[i] >> 16;
      won[i] = claim[i] && slot[i] < kSlots;
      over[i] = claim[i] && slot[i] >= kSlots;              // lanes filled the bucket first
      if (won[i]) t16[bk[i] * 8 + slot[i]] = (uint16_t)e[i];
    }
    // LDS operations of one wave complete in order; keep the compiler from
    // moving the read-back above the 16-bit stores
    asm volatile("" ::: "memory");
    bool any = false;
#pragma unroll
    for (int i = 0; i < N; ++i) any |= claim[i];
    if (ballot(any) == 0) return;
#pragma unroll
    for (int i = 0; i < N; ++i) {
      if (ballot(claim[i]) == 0) continue;
      const uint4 v = t4[bk[i]];
      // a lower slot holding the same entry belongs to another lane with this
      // id; a lane that found the bucket full keeps its id only if no lane
      // recorded it there
      const bool dup = holds(v, e[i], won[i] ? slot[i] : kSlots);
      isnew[i] = isnew[i] || (claim[i] && !dup);
      recorded[i] = won[i] && !dup;
    }
  }
};

// Visited filter of a parked-capable query: the same open addressing in
// HBM.  Only its owning wave touches it; lookups use agent-scope atomic loads
// so that a line cached in the CU's L1 before an atomic update is never read.
template <int LOG2>
struct VisitedHbm {
  static constexpr uint32_t kSize = 1u << LOG2;
  static constexpr uint32_t kLimit = kSize - kSize / 4;
  static constexpr int kMaxProbe = 64;

  __device__ __forceinline__ static uint32_t hash(uint32_t id) {
    return (id * 0x9E3779B1u) >> (32 - LOG2);
  }

  // Plain stores, then an agent-scope fence so later atomics see them.
  __device__ __forceinline__ static void clear(uint32_t *t) {
    uint4 *t4 = reinterpret_cast<uint4 *>(t);
    const uint4 e = make_uint4(kHtEmpty, kHtEmpty, kHtEmpty, kHtEmpty);
    for (uint32_t i = lane_id(); i < kSize / 4; i += kWave) t4[i] = e;
    __threadfence();
  }

  template <int N>
  __device__ __forceinline__ static void test_and_set_n(uint32_t *t, const uint32_t (&ids)[N],
                                                        const bool (&valid)[N], bool may_store,
                                                        bool (&isnew)[N], bool (&recorded)[N]) {
    uint32_t h[N];
    bool pend[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
      h[i] = hash(ids[i]);
      pend[i] = valid[i];
      isnew[i] = false;
      recorded[i] = false;
    }
    for (int p = 0; p < kMaxProbe; ++p) {
      bool any = false;
#pragma unroll
      for (int i = 0; i < N; ++i) any |= pend[i];
      if (ballot(any) == 0) break;
      uint32_t old[N];
#pragma unroll
      for (int i = 0; i < N; ++i) {
        if (pend[i])
          old[i] = may_store ? atomicCAS(&t[h[i]], kHtEmpty, ids[i])
                             : __hip_atomic_load(&t[h[i]], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
#pragma unroll
      for (int i = 0; i < N; ++i) {
        if (!pend[i]) continue;
        if (old[i] == kHtEmpty) {
          isnew[i] = true;
          recorded[i] = may_store;
          pend[i] = false;
        } else if (old[i] == ids[i]) {
          pend[i] = false;
        } else {
          h[i] = (h[i] + 1) & (kSize - 1);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < N; ++i)
      if (pend[i]) isnew[i] = true;
  }
};

}  // namespace gorio
