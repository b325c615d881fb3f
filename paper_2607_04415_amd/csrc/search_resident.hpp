// HBM-resident beam search: one wavefront per query.
//
// Per query the wave keeps the frontier F (the L best keys of the evaluated
// set, ascending) in registers, 64 * KPL slots, slot e = r * 64 + lane, and its
// visited filter in LDS.  Key = (distance bits << 32) | (node id << 1) |
// expanded bit: ties order by id, and the flag rides along through the
// sorting networks.  One iteration (GORIO Sec. 1 / Sec. 2.2: expand nodes,
// compute distances, update the frontier):
//   select  - the first W unexpanded slots of F (ballot + prefix count);
//   expand  - one round trip reads the degree and id list of every chosen
//             node of a beam group (up to 256 ids, 4 per lane); with float32
//             line-gathered rows a beam of several groups reads the next
//             group's lists while the current one is filtered and evaluated;
//   filter  - ids already in the visited filter are dropped (LDS atomics),
//             the rest compacted into an LDS candidate list;
//   evaluate- one round trip gathers a batch of candidate vectors; the
//             distance policy (metric.hpp) turns them into keys: uint8 with
//             8 lanes per 128-B vector and v_dot4_u32_u8, float32 with one
//             lane per vector (96-d rows read 8 lanes per vector by lines,
//             then transposed in registers) and the sequential rounded sum;
//   merge   - only keys below F's L-th key can enter: a few are inserted by
//             rank (ballot + DPP shift), many are bitonic-sorted per 64-lane
//             chunk and bitonic-merged into F.
#pragma once

#include "metric.hpp"

namespace gorio {

struct ResidentParams {
  const uint8_t *pages;    // num_pages * page_bytes, HBM
  PageGeom geom;
  uint32_t n;
  uint32_t D;              // vector elements (uint8: a multiple of 4)
  uint32_t R;              // id slots per record
  FastDiv Rdiv;            // division by R
  uint32_t entry;
  const void *queries;     // nq x D elements
  uint32_t nq;
  uint32_t k, L, W;
  uint32_t *out_ids;       // nq x k
  uint32_t *out_dists;     // nq x k distance bits (int32 or float32)
  unsigned long long *stats;  // [evaluations, reevaluations, expansions, iterations]
  // Queries past the first grid are handed out by a counter that only grows:
  // every completed query takes one ticket, so a launch adds exactly nq, and
  // next_base is the counter's value when this launch starts (no reset between
  // launches).
  unsigned long long *next_query;
  unsigned long long next_base;
};

// Evaluates NCH chunks of 64 compacted candidates (locator metrics) and
// merges their keys into F, with two chunks in flight.
template <int NCH, int KPL, class M>
__device__ __forceinline__ void eval_chunks(const M &m, const ResidentParams &p, const uint32_t *cand, uint32_t cnt,
                                            uint64_t (&F)[KPL], bool forgot) {
  const __amdgpu_buffer_rsrc_t rs = units16_rsrc(p.pages, p.geom);
  typename M::Chunk A, B;
  m.chunk_issue(rs, cand, 0, A);
  if constexpr (NCH > 1) m.chunk_issue(rs, cand, kWave, B);
  uint64_t key = m.chunk_key(p.geom, cand, 0, cnt, A);
  if constexpr (NCH > 2) m.chunk_issue(rs, cand, 2 * kWave, A);
  merge_keys<KPL>(F, key, forgot, p.L);
  if constexpr (NCH > 1) {
    key = m.chunk_key(p.geom, cand, kWave, cnt, B);
    if constexpr (NCH > 3) m.chunk_issue(rs, cand, 3 * kWave, B);
    merge_keys<KPL>(F, key, forgot, p.L);
  }
  if constexpr (NCH > 2) merge_keys<KPL>(F, m.chunk_key(p.geom, cand, 2 * kWave, cnt, A), forgot, p.L);
  if constexpr (NCH > 3) merge_keys<KPL>(F, m.chunk_key(p.geom, cand, 3 * kWave, cnt, B), forgot, p.L);
}

// Evaluates NCH batches of 64 compacted candidates with the float32 line
// gather and merges their keys into F, two batches in flight (the same
// fixed schedule as eval_chunks).
template <int NCH, int KPL, bool N2S, class M>
__device__ __forceinline__ void eval_gathered(const M &m, const ResidentParams &p, const uint32_t *cand, uint32_t cnt,
                                              uint64_t (&F)[KPL], bool forgot) {
  typename M::Gathered A, B;
  M::template gather_issue<N2S>(p.pages, p.geom, cand, 0, cnt, p.entry, A);
  if constexpr (NCH > 1) M::template gather_issue<N2S>(p.pages, p.geom, cand, kWave, cnt, p.entry, B);
  uint64_t key = m.gather_key(A, 0, cnt);
  if constexpr (NCH > 2) M::template gather_issue<N2S>(p.pages, p.geom, cand, 2 * kWave, cnt, p.entry, A);
  merge_keys<KPL>(F, key, forgot, p.L);
  if constexpr (NCH > 1) {
    key = m.gather_key(B, kWave, cnt);
    if constexpr (NCH > 3) M::template gather_issue<N2S>(p.pages, p.geom, cand, 3 * kWave, cnt, p.entry, B);
    merge_keys<KPL>(F, key, forgot, p.L);
  }
  if constexpr (NCH > 2) merge_keys<KPL>(F, m.gather_key(A, 2 * kWave, cnt), forgot, p.L);
  if constexpr (NCH > 3) merge_keys<KPL>(F, m.gather_key(B, 3 * kWave, cnt), forgot, p.L);
}

// Waves per SIMD from the distance policy (M::kWavesPerSimd: 4 for uint8
// rows up to 128 bytes, with an 8 KB visited table; 1 for gathered 96-d
// float32 rows, which keep two batches of whole vectors in registers; 2
// otherwise): one wave's gathers overlap the others' filtering and merging.  The grid is as large as the chip holds at
// once; workgroup b starts with query b and then takes the next unclaimed
// query from a global counter, so the XCDs and CUs that finish early take
// more queries and the batch ends when the last queries end, wherever they
// run.
template <int KPL, class M, class HT, bool N2S>
__global__ __launch_bounds__(kWave, M::kWavesPerSimd) void search_resident(ResidentParams p) {
  constexpr int kChunks = M::kChunks;
  constexpr int kBatch = M::kBatch;
  constexpr int kIdsPerLane = kCandCap / kWave;

  __shared__ __align__(16) uint32_t ht[HT::kWords];
  __shared__ __align__(16) uint32_t cand[kCandCap];
  __shared__ uint32_t beam[kMaxW];
  __shared__ __align__(16) uint32_t qbuf[M::kQueryWords];

  const int l = lane_id();
  const uint32_t beams_per_group = min(kCandCap / p.R, (uint32_t)kWave);
  const uint32_t entry_word = M::cand_word(p.geom, p.entry);

  unsigned long long n_eval = 0, n_reeval = 0, n_exp = 0, n_iter = 0;

  for (uint32_t qi = blockIdx.x; qi < p.nq;) {
    HT::clear(ht);
    M m;
    m.load_query(p.queries, qi, p.D, qbuf);
    __syncthreads();

    uint32_t ht_used = 0;
    bool forgot = false;  // some node may have been evaluated twice

    // V = {entry}
    uint64_t F[KPL];
#pragma unroll
    for (int r = 0; r < KPL; ++r) F[r] = kInfKey;
    {
      const uint32_t d = m.dist_one(p.pages + vec_offset(p.geom, slot_ct<N2S>(p.geom, p.entry)));
      if (l == 0) {
        F[0] = ((uint64_t)d << 32) | ((uint64_t)p.entry << 1);
        bool rec;
        HT::test_and_set(ht, p.entry, true, rec);
      }
      ht_used = 1;
      ++n_eval;
    }
    __syncthreads();

    for (uint32_t guard = 0; guard <= p.n; ++guard) {
      // ---- select: first W unexpanded slots of F, in order -----------------
      uint32_t nbeam = 0;
#pragma unroll
      for (int r = 0; r < KPL; ++r) {
        const uint32_t e = r * kWave + l;
        bool unexp = e < p.L && F[r] != kInfKey && !(F[r] & 1ull);
        uint64_t m = ballot(unexp);
        uint32_t rank = nbeam + lanes_below(m);
        if (unexp && rank < p.W) {
          beam[rank] = key_id(F[r]);
          F[r] |= 1ull;
        }
        nbeam += (uint32_t)__popcll(m);
      }
      if (nbeam > p.W) nbeam = p.W;
      if (nbeam == 0) break;
      __syncthreads();
      n_exp += nbeam;
      ++n_iter;

      // ---- expand: degrees (lane b) and all id slots of a beam group at once.
      // Loads are unconditional (lanes past the group read the group's first
      // record) so that no branch separates them: one round trip per group.
      // Float32 line-gathered rows (W=8, R=64: two groups per beam) read the
      // next group's lists while this group is filtered and evaluated, so only
      // the first group's round trip is exposed.  Other metrics read a group's
      // lists when they reach it: a uint8 beam at W=4 fits one group, and a
      // second set of list registers would only constrain the allocator.
      constexpr bool kAhead = M::kGathered;
      struct AdjLoad {
        uint64_t off;  // lane b: adjacency block of the group's beam b
        uint32_t deg;  // lane b: its degree
        uint32_t ids[kIdsPerLane];
      };
      auto issue_adj = [&](uint32_t b0, AdjLoad &A) {
        const uint32_t nb = min(nbeam - b0, beams_per_group);
        const uint32_t nslots = nb * p.R;
        const uint32_t my_beam = beam[b0 + min((uint32_t)l, nb - 1)];
        A.off = adj_offset(p.geom, slot_ct<N2S>(p.geom, my_beam));
        A.deg = *reinterpret_cast<const uint32_t *>(p.pages + A.off);
#pragma unroll
        for (int t = 0; t < kIdsPerLane; ++t) {
          const uint32_t pos = min(t * kWave + (uint32_t)l, nslots - 1);
          const uint32_t b = fastdiv(pos, p.Rdiv);
          const uint64_t adj = __shfl(A.off, (int)b);
          A.ids[t] = reinterpret_cast<const uint32_t *>(p.pages + adj + 4)[pos - b * p.R];
        }
      };
      [[maybe_unused]] AdjLoad cur, nxt;
      if constexpr (kAhead) issue_adj(0, cur);
      for (uint32_t b0 = 0; b0 < nbeam; b0 += beams_per_group) {
        const uint32_t nb = min(nbeam - b0, beams_per_group);
        const uint32_t nslots = nb * p.R;
        uint32_t ids[kIdsPerLane];
        bool valid[kIdsPerLane];
        if constexpr (kAhead) {
          if (b0 + beams_per_group < nbeam) issue_adj(b0 + beams_per_group, nxt);
#pragma unroll
          for (int t = 0; t < kIdsPerLane; ++t) {
            const uint32_t pos = min(t * kWave + (uint32_t)l, nslots - 1);
            const uint32_t b = fastdiv(pos, p.Rdiv);
            const uint32_t deg = min((uint32_t)__shfl((int)cur.deg, (int)b), p.R);
            ids[t] = cur.ids[t];
            valid[t] = (uint32_t)(t * kWave + l) < nslots && pos - b * p.R < deg && ids[t] < p.n;
          }
        } else {
          const uint32_t my_beam = beam[b0 + min((uint32_t)l, nb - 1)];
          const uint64_t my_adj = adj_offset(p.geom, slot_ct<N2S>(p.geom, my_beam));
          const uint32_t my_deg = *reinterpret_cast<const uint32_t *>(p.pages + my_adj);
          uint32_t slot_beam[kIdsPerLane], slot_j[kIdsPerLane];
#pragma unroll
          for (int t = 0; t < kIdsPerLane; ++t) {
            const uint32_t pos = min(t * kWave + (uint32_t)l, nslots - 1);
            const uint32_t b = fastdiv(pos, p.Rdiv);
            slot_beam[t] = b;
            slot_j[t] = pos - b * p.R;
          }
#pragma unroll
          for (int t = 0; t < kIdsPerLane; ++t) {
            const uint64_t adj = __shfl(my_adj, (int)slot_beam[t]);
            ids[t] = reinterpret_cast<const uint32_t *>(p.pages + adj + 4)[slot_j[t]];
          }
#pragma unroll
          for (int t = 0; t < kIdsPerLane; ++t) {
            const uint32_t deg = min((uint32_t)__shfl((int)my_deg, (int)slot_beam[t]), p.R);
            valid[t] = (uint32_t)(t * kWave + l) < nslots && slot_j[t] < deg && ids[t] < p.n;
          }
        }
        // ---- filter through the visited table, compact the new ids ------------
        bool isnew[kIdsPerLane], recorded[kIdsPerLane];
        HT::template test_and_set_n<kIdsPerLane>(ht, ids, valid, ht_used < HT::kLimit, isnew, recorded);
        uint32_t cnt = 0;
#pragma unroll
        for (int t = 0; t < kIdsPerLane; ++t) {
          const uint64_t mnew = ballot(isnew[t]);
          const uint64_t mrec = ballot(recorded[t]);
          if (isnew[t]) cand[M::cand_pos(cnt + lanes_below(mnew))] = M::cand_word(p.geom, ids[t]);
          cnt += (uint32_t)__popcll(mnew);
          ht_used += (uint32_t)__popcll(mrec);
          const uint32_t lost = (uint32_t)__popcll(mnew & ~mrec);
          n_reeval += lost;
          forgot |= lost != 0;
        }
        M::pad_round(cand, cnt, entry_word);
        __syncthreads();
        n_eval += cnt;

        // ---- evaluate and merge -----------------------------------------------
        if constexpr (M::kLocators) {
          // chunks of 64 vectors, two in flight: the next chunk's gathers are
          // outstanding while this one is reduced and merged (a fixed schedule
          // per chunk count keeps every wait exact)
          static_assert(kCandCap == 4 * kWave, "at most four chunks");
          switch ((cnt + kWave - 1) / kWave) {
            case 1: eval_chunks<1, KPL>(m, p, cand, cnt, F, forgot); break;
            case 2: eval_chunks<2, KPL>(m, p, cand, cnt, F, forgot); break;
            case 3: eval_chunks<3, KPL>(m, p, cand, cnt, F, forgot); break;
            case 4: eval_chunks<4, KPL>(m, p, cand, cnt, F, forgot); break;
            default: break;
          }
        } else if constexpr (M::kGathered && !N2S) {
          // float32 line gather, two batches of 64 in flight (with a
          // placement permutation the next batch's slot loads would wait on
          // the older batch's loads, so that case takes the plain loop)
          switch ((cnt + kWave - 1) / kWave) {
            case 1: eval_gathered<1, KPL, N2S>(m, p, cand, cnt, F, forgot); break;
            case 2: eval_gathered<2, KPL, N2S>(m, p, cand, cnt, F, forgot); break;
            case 3: eval_gathered<3, KPL, N2S>(m, p, cand, cnt, F, forgot); break;
            case 4: eval_gathered<4, KPL, N2S>(m, p, cand, cnt, F, forgot); break;
            default: break;
          }
        } else {
          // batches of kBatch vectors, one round trip each
          for (uint32_t c0 = 0; c0 < cnt; c0 += kBatch) {
            uint64_t key[kChunks];
            m.template resident_keys<N2S>(p.pages, p.geom, cand, c0, cnt, p.entry, key);
#pragma unroll
            for (int c = 0; c < kChunks; ++c) merge_keys<KPL>(F, key[c], forgot, p.L);
          }
        }
        __syncthreads();
        if constexpr (kAhead) cur = nxt;
      }
    }

    // ---- result: first k slots of F -------------------------------------------
#pragma unroll
    for (int r = 0; r < KPL; ++r) {
      const uint32_t e = r * kWave + l;
      if (e < p.k) {
        const bool ok = F[r] != kInfKey;
        p.out_ids[(uint64_t)qi * p.k + e] = ok ? key_id(F[r]) : kNoEdge;
        p.out_dists[(uint64_t)qi * p.k + e] = ok ? (uint32_t)(F[r] >> 32) : M::kPadDist;
      }
    }
    uint32_t next = 0;
    if (l == 0) next = (uint32_t)(atomicAdd(p.next_query, 1ull) - p.next_base);
    qi = gridDim.x + first_lane_value(next);
  }

  if (l == 0) {
    atomicAdd(&p.stats[0], n_eval);
    atomicAdd(&p.stats[1], n_reeval);
    atomicAdd(&p.stats[2], n_exp);
    atomicAdd(&p.stats[3], n_iter);
  }
}

}  // namespace gorio
