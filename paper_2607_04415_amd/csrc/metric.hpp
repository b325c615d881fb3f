// Distance policies of the search kernels (squared L2, returned squared).
//
// A policy loads the query, evaluates the entry node, and turns a batch of
// candidate records into 64-bit frontier keys (distance bits << 32 |
// id << 1).  The kernels' traversal, filtering and merging do not depend on
// the element type: uint8 distances are non-negative int32 values and float32
// distances are >= +0, so both order correctly as unsigned 32-bit patterns.
//
//   MetricU8  - exact int32 distance: q.q + sum (x.x - 2 q.x) with
//               v_dot4_u32_u8 on coalesced reads, 8 lanes per vector.
//   MetricF32 - one lane per candidate (resident 96-d rows are gathered 8
//               lanes per vector by whole lines and handed to their lanes
//               through LDS);
//               t = q_d - x_d, acc = acc + t*t for d = 0 .. D-1 in order,
//               every operation rounded to nearest even with no fused
//               multiply-add, so the result is the same float as a plain
//               sequential loop.
#pragma once

#include "frontier.hpp"
#include "page_cache.hpp"

namespace gorio {

// ---------------------------------------------------------------------------
// uint8
// ---------------------------------------------------------------------------
// LOC16: the kernel keeps each candidate as its vector's 16-byte locator
// (identity placement, units16 != 0) instead of its id, stored so that the
// kRounds candidates of each group of 8 lanes are consecutive words: the
// batch's addresses arrive with kRounds / 4 LDS reads and no per-round
// address arithmetic, and ids are recovered from locators for the keys.
template <int VDW, bool EXACT, bool LOC16 = false>
struct MetricU8 {
  // vectors in flight per resident gather batch: 128 for up to 16 B per lane,
  // 64 for wider rows (kept small so that two waves fit each SIMD's registers)
  static constexpr int kRounds = VDW <= 4 ? 16 : 8;
  static constexpr int kBatch = kRounds * 8;
  static constexpr int kChunks = kBatch / kWave;
  static_assert(kRounds % 8 == 0, "rounds are reduced eight at a time");
  static constexpr int kQueryWords = 1;          // the query lives in registers
  // resident kernel: waves per SIMD and the 16-bit visited table that fits
  // them (4 waves: <= 128 registers, 4096 entries in 8 KB of LDS)
  static constexpr int kWavesPerSimd = VDW <= 4 ? 4 : 2;
  static constexpr int kHtLog2 = VDW <= 4 ? 12 : 13;
  // Waves per SIMD in the resident grid.  Two keep the gathers saturated
  // (a 100k-query batch on the 1M x 128-d index runs at the same rate with
  // two or four per SIMD); with two, each query finishes sooner and so does
  // a batch's tail, when the query counter has run dry and the chip empties
  // (10k queries: 0.79 ms against 0.85 ms with four).
  static constexpr int kGridWavesPerSimd = 2;
  static constexpr uint32_t kPadDist = 0x7FFFFFFFu;  // INT32_MAX
  static_assert(!LOC16 || (EXACT && VDW % 4 == 0), "locators address whole 16-byte units");
  static constexpr bool kLocators = LOC16;
  static constexpr bool kGathered = false;  // float32 line gather only

  // Where the kernel's compaction puts the i-th new candidate, and the word
  // it stores for node v (its id, or with LOC16 its vector's locator).
  __device__ __forceinline__ static uint32_t cand_pos(uint32_t i) {
    if constexpr (LOC16)
      return (i & ~(uint32_t)(kBatch - 1)) | ((i & 7u) * kRounds) | ((i >> 3) & (uint32_t)(kRounds - 1));
    else
      return i;
  }
  __device__ __forceinline__ static uint32_t cand_word(const PageGeom &geom, uint32_t v) {
    if constexpr (LOC16) return vec_locator(geom, v);
    else return v;
  }

  // After compaction of cnt candidates: give the rest of the last chunk of 64
  // the fallback node's word, so that every lane of every round of a chunk
  // loads a vector (the chunk's load count is then fixed).
  __device__ __forceinline__ static void pad_round(uint32_t *cand, uint32_t cnt, uint32_t fallback_word) {
    if constexpr (LOC16) {
      const uint32_t i = cnt + (uint32_t)lane_id();
      if (i < ((cnt + kWave - 1) & ~(uint32_t)(kWave - 1))) cand[cand_pos(i)] = fallback_word;
    }
  }

  U8Vec<VDW, EXACT> q;
  int qq;
  uint32_t dwords;

  __device__ __forceinline__ void load_query(const void *queries, uint32_t qi, uint32_t D, uint32_t *) {
    const int gl = lane_id() & 7;
    dwords = D >> 2;
    q.load(static_cast<const uint8_t *>(queries) + (uint64_t)qi * D, gl, dwords);
    int s = 0;
#pragma unroll
    for (int t = 0; t < VDW; ++t) s += (int)__builtin_amdgcn_udot4(q.w[t], q.w[t], 0u, false);
    qq = sum8(s);
  }

  // Distance bits of one record, computed by the whole wave (uniform result).
  __device__ __forceinline__ uint32_t dist_one(const uint8_t *rec) const {
    U8Vec<VDW, EXACT> x;
    x.load(rec, lane_id() & 7, dwords);
    return (uint32_t)(sum8(partial_u8(q, x)) + qq);
  }

  // Keys of candidates c0 .. c0 + kBatch - 1 of cand (kInfKey past cnt), from
  // the resident pages.  One round trip for the batch.
  template <bool N2S>
  __device__ __forceinline__ void resident_keys(const uint8_t *pages, const PageGeom &geom, const uint32_t *cand,
                                                uint32_t c0, uint32_t cnt, uint32_t fallback,
                                                uint64_t (&key)[kChunks]) const {
    static_assert(!LOC16, "with locators the kernel streams chunks (chunk_issue, chunk_key)");
    const int l = lane_id();
    const int g = l >> 3;
    const int gl = l & 7;
    // candidate node -> record; lanes past the count read the fallback record
    uint64_t rec[kRounds];
#pragma unroll
    for (int rr = 0; rr < kRounds; ++rr) {
      if (c0 + rr * 8 >= cnt) break;
      const uint32_t idx = c0 + rr * 8 + g;
      rec[rr] = vec_offset(geom, slot_ct<N2S>(geom, idx < cnt ? cand[idx] : fallback));
    }
    U8Vec<VDW, EXACT> x[kRounds];
#pragma unroll
    for (int rr = 0; rr < kRounds; ++rr) {
      if (c0 + rr * 8 >= cnt) break;
      x[rr].load(pages + rec[rr], gl, dwords);
    }
    // eight rounds at a time: lane gl of group g ends with round 8c + gl's distance
    int dist[kChunks];
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      dist[c] = 0;
      if (c0 + c * kWave >= cnt) break;
      int part[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) part[j] = c0 + (c * 8 + j) * 8 < cnt ? partial_u8(q, x[c * 8 + j]) : 0;
      dist[c] = transpose_sum8(part) + qq;
    }
    // lane l of chunk c holds candidate c0 + 64c + 8*(l%8) + l/8
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const uint32_t my_idx = c0 + c * kWave + gl * 8 + g;
      key[c] = my_idx < cnt ? (((uint64_t)(uint32_t)dist[c] << 32) | ((uint64_t)cand[my_idx] << 1)) : kInfKey;
    }
  }

  // Streaming gather (LOC16): the candidate list is evaluated in chunks of
  // 64, eight rounds of eight vectors; the kernel keeps two chunks in flight
  // (issues the next while reducing and merging the current one).  Group g's
  // eight locators of chunk c0 / 64 are consecutive words of the compacted
  // list (cand_pos).  Every chunk issues the same number of loads, so the
  // compiler's waits before a chunk's use leave the other chunk in flight.
  struct Chunk {
    U8Vec<VDW, EXACT> x[8];
  };
  __device__ __forceinline__ void chunk_issue(__amdgpu_buffer_rsrc_t rs, const uint32_t *cand, uint32_t c0,
                                              Chunk &ck) const {
    static_assert(LOC16 && kRounds == 16, "streaming needs locators and 16 rounds per 128 candidates");
    const int l = lane_id();
    const int g = l >> 3;
    const int gl = l & 7;
    const uint4 *src = reinterpret_cast<const uint4 *>(cand + (c0 & ~127u) + g * kRounds + ((c0 >> 6) & 1u) * 8u);
    const uint4 a = src[0], b = src[1];
    uint32_t loc[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int rr = 0; rr < 8; ++rr) asm volatile("" : "+v"(loc[rr]));
    // all eight rounds: positions past the count hold the fallback's locator
#pragma unroll
    for (int rr = 0; rr < 8; ++rr) {
      const uint32_t u = loc[rr] + (uint32_t)gl * (VDW / 4);
#pragma unroll
      for (int t = 0; t < VDW; t += 4) {
        const u32x4_t v = struct_buffer_load_b128(rs, (int)(u + t / 4), 0, 0, 0);
        ck.x[rr].w[t] = v.x; ck.x[rr].w[t + 1] = v.y; ck.x[rr].w[t + 2] = v.z; ck.x[rr].w[t + 3] = v.w;
      }
    }
  }
  // Key of this lane's candidate of the chunk (kInfKey past cnt): lane
  // (g, gl) ends with round gl of group g, candidate c0 + 8 gl + g.
  __device__ __forceinline__ uint64_t chunk_key(const PageGeom &geom, const uint32_t *cand, uint32_t c0,
                                                uint32_t cnt, const Chunk &ck) const {
    const int l = lane_id();
    const int g = l >> 3;
    const int gl = l & 7;
    int part[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) part[j] = partial_u8(q, ck.x[j]);
    const int dist = transpose_sum8(part) + qq;
    const bool ok = c0 + (uint32_t)gl * 8 + (uint32_t)g < cnt;
    const uint32_t pos = (c0 & ~127u) + g * kRounds + ((c0 >> 6) & 1u) * 8u + gl;
    const uint32_t v = ok ? slot_of_locator(geom, cand[pos]) : 0u;
    return ok ? (((uint64_t)(uint32_t)dist << 32) | ((uint64_t)v << 1)) : kInfKey;
  }

  // Paged: keys of the candidates whose pages are ready (rdy, slot per lane;
  // candidate index = base + lane).  off_of(slot, node) is the record's byte
  // offset in the cache.  The ready lanes are compacted and evaluated 8 per
  // round; the key of the i-th ready candidate ends up in some lane, the others
  // hold kInfKey.
  template <class OffOf>
  __device__ __forceinline__ uint64_t paged_keys(OffOf off_of, __amdgpu_buffer_rsrc_t crs, const uint32_t *cand,
                                                 uint32_t base, bool rdy, uint32_t slot, uint64_t mr) const {
    const int l = lane_id();
    const int g = l >> 3;
    const int gl = l & 7;
    const uint32_t cnt = (uint32_t)__popcll(mr);
    __shared__ uint32_t rc[kWave], rs[kWave];
    if (rdy) {
      const uint32_t my_rank = lanes_below(mr);
      rc[my_rank] = base + l;
      rs[my_rank] = slot;
    }
    __syncthreads();
    U8Vec<VDW, EXACT> x[8];
#pragma unroll
    for (int rr = 0; rr < 8; ++rr) {
      const uint32_t idx = rr * 8 + g;
      const uint32_t ci = idx < cnt ? rc[idx] : rc[0];
      const uint32_t si = idx < cnt ? rs[idx] : rs[0];
      load_cached_u8(x[rr], crs, off_of(si, cand[ci]), gl);
    }
    int part[8];
#pragma unroll
    for (int rr = 0; rr < 8; ++rr) part[rr] = partial_u8(q, x[rr]);
    const int mine_d = transpose_sum8(part) + qq;
    const uint32_t my_idx = gl * 8 + g;
    uint64_t key = kInfKey;
    if (my_idx < cnt) key = ((uint64_t)(uint32_t)mine_d << 32) | ((uint64_t)cand[rc[my_idx]] << 1);
    __syncthreads();
    return key;
  }

 private:
  // coherent read of a cached vector (see page_cache.hpp)
  __device__ __forceinline__ void load_cached_u8(U8Vec<VDW, EXACT> &x, __amdgpu_buffer_rsrc_t r, uint32_t rec,
                                                 int gl) const {
    const uint32_t b = rec + (uint32_t)gl * VDW * 4u;
    if constexpr (EXACT && VDW % 4 == 0) {
#pragma unroll
      for (int t = 0; t < VDW; t += 4) {
        const uint4 u = coherent_load_u128(r, b + t * 4u);
        x.w[t] = u.x; x.w[t + 1] = u.y; x.w[t + 2] = u.z; x.w[t + 3] = u.w;
      }
    } else {
#pragma unroll
      for (int t = 0; t < VDW; ++t)
        x.w[t] = (EXACT || (uint32_t)(gl * VDW + t) < dwords) ? coherent_load_u32(r, b + t * 4u) : 0u;
    }
  }
};

// ---------------------------------------------------------------------------
// float32
// ---------------------------------------------------------------------------
// NV4: the vector has at most 4 * NV4 floats.  EXACT: exactly 4 * NV4, read
// with 16-B loads all at once; otherwise dword loads of d < D, 16 at a time.
template <int NV4, bool EXACT>
struct MetricF32 {
  static constexpr int kBatch = kWave;  // one candidate per lane
  static constexpr int kChunks = 1;
  static constexpr int kQueryWords = 4 * NV4;
  static constexpr uint32_t kPadDist = 0x7F800000u;  // +inf
  // resident kernel: 96-d rows (gathered by lines, blocks staged through a
  // 4 KB LDS buffer) keep two batches of lines in registers, which fits one
  // wave per SIMD and leaves LDS for a 32 KB visited table; other widths run
  // two waves per SIMD with a 16 KB table
  static constexpr bool kGathered = EXACT && NV4 % 8 == 0;
  static constexpr int kWavesPerSimd = kGathered ? 1 : 2;
  static constexpr int kHtLog2 = kGathered ? 14 : 13;
  static constexpr int kGridWavesPerSimd = kWavesPerSimd;
  static constexpr int kStep = 16;                   // dwords per round trip (generic path)

  const float *qs;  // the query in LDS (wave-uniform reads)
  uint32_t D;

  static constexpr bool kLocators = false;
  __device__ __forceinline__ static void pad_round(uint32_t *, uint32_t, uint32_t) {}
  __device__ __forceinline__ static uint32_t cand_pos(uint32_t i) { return i; }
  __device__ __forceinline__ static uint32_t cand_word(const PageGeom &, uint32_t v) { return v; }

  // Copies the query into LDS; the caller synchronizes before use.
  __device__ __forceinline__ void load_query(const void *queries, uint32_t qi, uint32_t D_, uint32_t *qlds) {
    D = D_;
    const uint32_t *src = static_cast<const uint32_t *>(queries) + (uint64_t)qi * D_;
    for (uint32_t d = lane_id(); d < (uint32_t)kQueryWords; d += kWave) qlds[d] = d < D_ ? src[d] : 0u;
    qs = reinterpret_cast<const float *>(qlds);
  }

  // acc + (q_d - x_d)^2 for one element, each step rounded on its own
  __device__ __forceinline__ static float step(float acc, float qd, float xd) {
    const float t = __fsub_rn(qd, xd);
    return __fadd_rn(acc, __fmul_rn(t, t));
  }

  // Sequential distance of this lane's vector; ld4(i) returns bytes
  // [16i, 16i + 16) of the vector, ld1(d) the d-th float's bits.
  template <class Ld4, class Ld1>
  __device__ __forceinline__ float dist_lane(Ld4 ld4, Ld1 ld1) const {
    float acc = 0.0f;
    if constexpr (EXACT) {
      uint4 x[NV4];
#pragma unroll
      for (int i = 0; i < NV4; ++i) x[i] = ld4(i);
#pragma unroll
      for (int i = 0; i < NV4; ++i) {
        const float4 qv = *reinterpret_cast<const float4 *>(qs + 4 * i);
        acc = step(acc, qv.x, __uint_as_float(x[i].x));
        acc = step(acc, qv.y, __uint_as_float(x[i].y));
        acc = step(acc, qv.z, __uint_as_float(x[i].z));
        acc = step(acc, qv.w, __uint_as_float(x[i].w));
      }
    } else {
      for (uint32_t d0 = 0; d0 < D; d0 += kStep) {
        uint32_t x[kStep];
#pragma unroll
        for (int j = 0; j < kStep; ++j) x[j] = d0 + j < D ? ld1(d0 + j) : 0u;
#pragma unroll
        for (int j = 0; j < kStep; ++j)
          if (d0 + j < D) acc = step(acc, qs[d0 + j], __uint_as_float(x[j]));
      }
    }
    return acc;
  }

  __device__ __forceinline__ float dist_global(const uint8_t *rec) const {
    const uint32_t *w = reinterpret_cast<const uint32_t *>(rec);
    return dist_lane(
        [&](int i) {
          uint4 u;
          __builtin_memcpy(&u, __builtin_assume_aligned(w + 4 * i, 4), 16);
          return u;
        },
        [&](uint32_t d) { return w[d]; });
  }

  __device__ __forceinline__ float dist_cached(__amdgpu_buffer_rsrc_t r, uint32_t off) const {
    return dist_lane([&](int i) { return coherent_load_u128(r, off + 16u * (uint32_t)i); },
                     [&](uint32_t d) { return coherent_load_u32(r, off + 4u * d); });
  }

  // Distance bits of one record (lane 0 computes, the result is broadcast).
  __device__ __forceinline__ uint32_t dist_one(const uint8_t *rec) const {
    uint32_t b = 0;
    if (lane_id() == 0) b = __float_as_uint(dist_global(rec));
    return first_lane_value(b);
  }

  template <bool N2S>
  __device__ __forceinline__ void resident_keys(const uint8_t *pages, const PageGeom &geom, const uint32_t *cand,
                                                uint32_t c0, uint32_t cnt, uint32_t fallback,
                                                uint64_t (&key)[kChunks]) const {
    const uint32_t idx = c0 + lane_id();
    const uint32_t node = idx < cnt ? cand[idx] : fallback;
    const uint64_t off = vec_offset(geom, slot_ct<N2S>(geom, node));
    if constexpr (kGathered) {
      const uint32_t c = transposed_candidate();
      const float d = dist_gathered(pages, off);
      const uint32_t cn = (uint32_t)__shfl((int)node, (int)c);
      key[0] = c0 + c < cnt ? (((uint64_t)__float_as_uint(d) << 32) | ((uint64_t)cn << 1)) : kInfKey;
    } else {
      const float d = dist_global(pages + off);
      key[0] = idx < cnt ? (((uint64_t)__float_as_uint(d) << 32) | ((uint64_t)node << 1)) : kInfKey;
    }
  }

  // Resident gather of 64 vectors, lane i's vector at byte offset `off` of
  // lane i.  One lane reading a whole vector would make every 16-byte load
  // instruction touch 64 different cache lines; instead the 8 lanes of a
  // group read 8 vectors, one at a time, each lane 16 bytes of every 128
  // (so each load instruction covers whole lines).  The 16-byte blocks then
  // pass through LDS, half a batch at a time (32 vectors x 128 bytes = 4 KB),
  // so that each lane gets one 128-byte line of its own candidate's vector
  // for the sequential sum: no VALU work moves the blocks, and the LDS
  // traffic runs beside the arithmetic.  Lane i ends with candidate i.
  __device__ __forceinline__ static uint32_t transposed_candidate() { return lane_id(); }

  // Block k of LDS row t sits at 16-byte position k ^ ((t >> 1) & 7): the
  // writes of one round cover 1 KB contiguously and the reads (lane t, row
  // t) spread any 16 consecutive lanes over all 64 banks.
  __device__ __forceinline__ static uint32_t tpos(uint32_t row, uint32_t k) { return row * 8u + (k ^ ((row >> 1) & 7u)); }

  // Line j of the vectors of the group's 8 candidates: x[r][c] = float
  // 32 j + 4 gl + c of the vector of lane r * 8 + g.
  __device__ __forceinline__ static void load_line(const uint8_t *pages, uint64_t off, int j, uint32_t (&x)[8][4]) {
    const uint32_t l = lane_id(), g = l >> 3, gl = l & 7u;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const uint64_t o = __shfl(off, r * 8 + (int)g);
      const uint32_t *w = reinterpret_cast<const uint32_t *>(pages + o) + 32 * j + 4 * gl;
      uint4 u;
      __builtin_memcpy(&u, __builtin_assume_aligned(w, 4), 16);
      x[r][0] = u.x;
      x[r][1] = u.y;
      x[r][2] = u.z;
      x[r][3] = u.w;
    }
  }

  // acc over line j of this lane's vector.  x[r] holds block gl of line j of
  // the vector of lane r * 8 + g; through LDS, lane i receives y[k] = block k
  // of its own vector's line (floats 32 j + 4 k .. + 3), so k then the
  // component visits d in increasing order.
  __device__ __forceinline__ float sum_line(float acc, uint32_t (&x)[8][4], int j) const {
    __shared__ __align__(16) uint4 stage[32 * 8];
    const uint32_t l = lane_id(), g = l >> 3, gl = l & 7u, t = l & 31u;
    uint4 y[8];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const uint32_t row = (uint32_t)rr * 8u + g;
        stage[tpos(row, gl)] = make_uint4(x[4 * h + rr][0], x[4 * h + rr][1], x[4 * h + rr][2], x[4 * h + rr][3]);
      }
      if ((l >> 5) == (uint32_t)h) {
#pragma unroll
        for (int k = 0; k < 8; ++k) y[k] = stage[tpos(t, (uint32_t)k)];
      }
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float4 qv = *reinterpret_cast<const float4 *>(qs + 32 * j + 4 * k);
      acc = step(acc, qv.x, __uint_as_float(y[k].x));
      acc = step(acc, qv.y, __uint_as_float(y[k].y));
      acc = step(acc, qv.z, __uint_as_float(y[k].z));
      acc = step(acc, qv.w, __uint_as_float(y[k].w));
    }
    return acc;
  }

  // One batch of 64 candidates' vectors in flight (resident kernel, line
  // gather): the loads are issued by gather_issue and consumed by gather_key,
  // so that another batch's loads can be outstanding in between.
  struct Gathered {
    uint32_t x[NV4 / 8][8][4];
    uint32_t node;
  };

  template <bool N2S>
  __device__ __forceinline__ static void gather_issue(const uint8_t *pages, const PageGeom &geom, const uint32_t *cand,
                                                      uint32_t c0, uint32_t cnt, uint32_t fallback, Gathered &b) {
    const uint32_t idx = c0 + lane_id();
    b.node = idx < cnt ? cand[idx] : fallback;
    const uint64_t off = vec_offset(geom, slot_ct<N2S>(geom, b.node));
#pragma unroll
    for (int j = 0; j < NV4 / 8; ++j) load_line(pages, off, j, b.x[j]);
  }

  __device__ __forceinline__ uint64_t gather_key(Gathered &b, uint32_t c0, uint32_t cnt) const {
    float acc = 0.0f;
#pragma unroll
    for (int j = 0; j < NV4 / 8; ++j) acc = sum_line(acc, b.x[j], j);
    const uint32_t c = transposed_candidate();
    const uint32_t cn = (uint32_t)__shfl((int)b.node, (int)c);
    return c0 + c < cnt ? (((uint64_t)__float_as_uint(acc) << 32) | ((uint64_t)cn << 1)) : kInfKey;
  }

  __device__ __forceinline__ float dist_gathered(const uint8_t *pages, uint64_t off) const {
    static_assert(EXACT && NV4 % 8 == 0, "whole 128-byte lines per vector");
    constexpr int J = NV4 / 8;  // lines per vector, all in flight at once
    uint32_t x[J][8][4];
#pragma unroll
    for (int j = 0; j < J; ++j) load_line(pages, off, j, x[j]);
    float acc = 0.0f;
#pragma unroll
    for (int j = 0; j < J; ++j) acc = sum_line(acc, x[j], j);
    return acc;
  }

  template <class OffOf>
  __device__ __forceinline__ uint64_t paged_keys(OffOf off_of, __amdgpu_buffer_rsrc_t crs, const uint32_t *cand,
                                                 uint32_t base, bool rdy, uint32_t slot, uint64_t) const {
    uint64_t key = kInfKey;
    if (rdy) {
      const uint32_t node = cand[base + lane_id()];
      const float d = dist_cached(crs, off_of(slot, node));
      key = ((uint64_t)__float_as_uint(d) << 32) | ((uint64_t)node << 1);
    }
    return key;
  }
};

}  // namespace gorio
