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
//             node of a beam group (up to 256 ids, 4 per lane);
//   filter  - ids already in the visited filter are dropped (LDS atomics),
//             the rest compacted into an LDS candidate list;
//   evaluate- one round trip gathers a batch of candidate vectors; the
//             distance policy (metric.hpp) turns them into keys: uint8 with
//             8 lanes per 128-B vector and v_dot4_u32_u8, float32 with one
//             lane per vector and the sequential rounded sum;
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
  unsigned long long *next_query;  // zero at launch: queries handed out past the first grid
};

// Several waves per SIMD (M::kWavesPerSimd: 4 for uint8 rows up to 128 bytes,
// with an 8 KB visited table; 2 otherwise): one wave's gathers overlap the
// others' filtering and merging.  The grid is as large as the chip holds at
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

      for (uint32_t b0 = 0; b0 < nbeam; b0 += beams_per_group) {
        const uint32_t nb = min(nbeam - b0, beams_per_group);
        const uint32_t nslots = nb * p.R;
        // ---- expand: degrees (lane b) and all id slots of the group at once ---
        // Loads are unconditional (lanes past the group read the group's first
        // record) so that no branch separates them: one round trip in total.
        const uint32_t my_beam = beam[b0 + min((uint32_t)l, nb - 1)];
        const uint64_t my_adj = adj_offset(p.geom, slot_ct<N2S>(p.geom, my_beam));
        const uint32_t my_deg = *reinterpret_cast<const uint32_t *>(p.pages + my_adj);
        uint32_t ids[kIdsPerLane];
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
        bool valid[kIdsPerLane];
#pragma unroll
        for (int t = 0; t < kIdsPerLane; ++t) {
          const uint32_t deg = min((uint32_t)__shfl((int)my_deg, (int)slot_beam[t]), p.R);
          valid[t] = (uint32_t)(t * kWave + l) < nslots && slot_j[t] < deg && ids[t] < p.n;
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

        // ---- evaluate: gather a batch of vectors in one round trip -------------
        for (uint32_t c0 = 0; c0 < cnt; c0 += kBatch) {
          uint64_t key[kChunks];
          m.template resident_keys<N2S>(p.pages, p.geom, cand, c0, cnt, p.entry, key);
          const uint64_t thr = frontier_at<KPL>(F, p.L - 1);
          uint64_t pass_mask[kChunks];
          uint32_t survivors = 0;
#pragma unroll
          for (int c = 0; c < kChunks; ++c) {
            const bool pass = key[c] < thr;
            pass_mask[c] = ballot(pass);
            if (!pass) key[c] = kInfKey;
            survivors += (uint32_t)__popcll(pass_mask[c]);
          }
          if (survivors == 0) continue;
          // ---- merge into the frontier ----------------------------------------
          if (survivors <= kInsertMax) {
#pragma unroll
            for (int c = 0; c < kChunks; ++c) {
              uint64_t pm = pass_mask[c];
              while (pm) {
                const int lane = __builtin_ctzll(pm);
                pm &= pm - 1;
                insert_key<KPL>(F, readlane64(key[c], lane));
              }
            }
          } else {
#pragma unroll
            for (int c = 0; c < kChunks; ++c) {
              if (pass_mask[c] == 0) continue;
              uint64_t cc[1] = {key[c]};
              bitonic_sort<1, true>(cc);
              if (!forgot) {
                // no node can repeat: the P smallest of F and C are min(F, C reversed)
                F[KPL - 1] = min64(F[KPL - 1], cc[0]);
                bitonic_merge_up<KPL>(F);
              } else {
                merge_dedupe<KPL>(F, cc[0]);
              }
            }
          }
#pragma unroll
          for (int r = 0; r < KPL; ++r)
            if ((uint32_t)(r * kWave + l) >= p.L) F[r] = kInfKey;
        }
        __syncthreads();
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
    if (l == 0) next = (uint32_t)atomicAdd(p.next_query, 1ull);
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
