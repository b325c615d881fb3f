// HBM-resident beam search for uint8 vectors: one wavefront per query.
//
// Per query the wave keeps the frontier F (the L best keys of the evaluated
// set, ascending) in registers, 64 * KPL slots, slot e = r * 64 + lane, and its
// visited filter in LDS.  Key = (squared distance << 32) | (node id << 1) |
// expanded bit: ties order by id, and the flag rides along through the
// sorting networks.  One iteration (GORIO Sec. 1 / Sec. 2.2: expand nodes,
// compute distances, update the frontier):
//   select  - the first W unexpanded slots of F (ballot + prefix count);
//   expand  - one round trip reads the degree and id list of every chosen
//             node of a beam group (up to 256 ids, 4 per lane);
//   filter  - ids already in the visited filter are dropped (LDS atomics),
//             the rest compacted into an LDS candidate list;
//   evaluate- one round trip gathers up to 256 vectors: 8 lanes per 128-B
//             vector, 16 B per lane, v_dot4_u32_u8 on the coalesced reads,
//             sum (q - x)^2 = q.q + sum (x.x - 2 q.x) exact in int32;
//   merge   - only keys below F's L-th key can enter: a few are inserted by
//             rank (ballot + DPP shift), many are bitonic-sorted per 64-lane
//             chunk and bitonic-merged into F.
#pragma once

#include "common.hpp"

namespace gorio {

struct ResidentParams {
  const uint8_t *pages;    // num_pages * page_bytes, HBM
  PageGeom geom;
  uint32_t n;
  uint32_t D;              // uint8 dimensions (multiple of 4)
  uint32_t R;              // id slots per record
  FastDiv Rdiv;            // division by R
  uint32_t entry;
  const uint8_t *queries;  // nq x D
  uint32_t nq;
  uint32_t k, L, W;
  uint32_t *out_ids;       // nq x k
  int32_t *out_dists;      // nq x k
  unsigned long long *stats;  // [evaluations, reevaluations, expansions, iterations]
};

// Lane layout for distance evaluation: 8 groups of 8 lanes; group g handles
// one vector per round, lane gl of the group holds dwords [gl*VDW, gl*VDW+VDW).
// EXACT: the vector is exactly 8 * VDW dwords (no per-dword bound checks, and
// 16-B loads when VDW is a multiple of 4; records are 4-B aligned).
template <int VDW, bool EXACT>
struct U8Vec {
  uint32_t w[VDW];

  __device__ __forceinline__ void load(const uint8_t *rec, int gl, uint32_t dwords) {
    const uint32_t *p = reinterpret_cast<const uint32_t *>(rec) + gl * VDW;
    if constexpr (EXACT && VDW % 4 == 0) {
#pragma unroll
      for (int t = 0; t < VDW; t += 4) {
        uint4 u;
        __builtin_memcpy(&u, __builtin_assume_aligned(p + t, 4), 16);
        w[t] = u.x; w[t + 1] = u.y; w[t + 2] = u.z; w[t + 3] = u.w;
      }
    } else if constexpr (EXACT) {
#pragma unroll
      for (int t = 0; t < VDW; ++t) w[t] = p[t];
    } else {
#pragma unroll
      for (int t = 0; t < VDW; ++t) w[t] = (uint32_t)(gl * VDW + t) < dwords ? p[t] : 0u;
    }
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int t = 0; t < VDW; ++t) w[t] = 0u;
  }
};

// Partial of sum (x.x - 2 q.x) over this lane's dwords.
template <int VDW, bool EXACT>
__device__ __forceinline__ int partial_u8(const U8Vec<VDW, EXACT> &q, const U8Vec<VDW, EXACT> &x) {
  int s = 0;
#pragma unroll
  for (int t = 0; t < VDW; ++t) {
    uint32_t xx = __builtin_amdgcn_udot4(x.w[t], x.w[t], 0u, false);
    uint32_t qx = __builtin_amdgcn_udot4(q.w[t], x.w[t], 0u, false);
    s += (int)xx - 2 * (int)qx;
  }
  return s;
}

__device__ __forceinline__ uint32_t key_id(uint64_t key) { return (uint32_t)(key >> 1) & 0x7FFFFFFFu; }

// Key at frontier slot e (uniform e).
template <int KPL>
__device__ __forceinline__ uint64_t frontier_at(const uint64_t (&F)[KPL], uint32_t e) {
  uint64_t v = kInfKey;
#pragma unroll
  for (int r = 0; r < KPL; ++r)
    if ((uint32_t)r == e / kWave) v = readlane64(F[r], e % kWave);
  return v;
}

// Insert one key c (wave-uniform) by rank: slots at or above its rank move up
// by one, the last slot falls off.  A key whose node is already in F is
// dropped, so repeated evaluations never duplicate a frontier entry.
template <int KPL>
__device__ __forceinline__ void insert_key(uint64_t (&F)[KPL], uint64_t c) {
  uint32_t rank = 0;
  bool dup = false;
#pragma unroll
  for (int r = 0; r < KPL; ++r) {
    rank += (uint32_t)__popcll(ballot(F[r] < c));
    dup |= ballot(F[r] != kInfKey && (F[r] >> 1) == (c >> 1)) != 0;
  }
  if (dup || rank >= (uint32_t)(KPL * kWave)) return;
  uint64_t prev[KPL];
#pragma unroll
  for (int r = 0; r < KPL; ++r) {
    uint64_t fill = r == 0 ? kInfKey : readlane64(F[r == 0 ? 0 : r - 1], kWave - 1);
    prev[r] = wave_shr1_64(F[r], fill);
  }
  const uint32_t l = lane_id();
#pragma unroll
  for (int r = 0; r < KPL; ++r) {
    const uint32_t e = r * kWave + l;
    F[r] = e < rank ? F[r] : (e == rank ? c : prev[r]);
  }
}

// Slow path after the visited filter forgot a node: a candidate may repeat a
// frontier node or another candidate.  Merge without truncating (2P slots:
// F ascending then C descending is bitonic), drop all but the last copy of
// each node (the copy carrying the expanded bit sorts last), re-sort, keep P.
template <int KPL>
__device__ __forceinline__ void merge_dedupe(uint64_t (&F)[KPL], uint64_t c_desc) {
  uint64_t big[2 * KPL];
#pragma unroll
  for (int r = 0; r < KPL; ++r) {
    big[r] = F[r];
    big[KPL + r] = kInfKey;
  }
  big[2 * KPL - 1] = c_desc;
  bitonic_merge_up<2 * KPL>(big);
  uint64_t next[2 * KPL];
#pragma unroll
  for (int r = 0; r < 2 * KPL; ++r) {
    uint64_t fill = r + 1 < 2 * KPL ? readlane64(big[r + 1 < 2 * KPL ? r + 1 : r], 0) : kInfKey;
    next[r] = shfl_down1_64(big[r], fill);
  }
#pragma unroll
  for (int r = 0; r < 2 * KPL; ++r)
    if (big[r] != kInfKey && next[r] != kInfKey && (next[r] >> 1) == (big[r] >> 1)) big[r] = kInfKey;
  bitonic_sort<2 * KPL>(big, false);
#pragma unroll
  for (int r = 0; r < KPL; ++r) F[r] = big[r];
}

// Up to this many keys below the L-th frontier key are inserted one by one;
// more go through the sorting network.
constexpr uint32_t kInsertMax = 12;

template <int KPL, int VDW, bool EXACT, int HT_LOG2, bool N2S>
__global__ __launch_bounds__(kWave) void search_resident_u8(ResidentParams p) {
  using HT = VisitedLds<HT_LOG2>;
  // vectors in flight per gather batch: 256 for up to 16 B per lane, fewer for wider rows
  constexpr int kRounds = VDW <= 4 ? 32 : 128 / VDW;
  constexpr int kBatch = kRounds * 8;
  constexpr int kChunks = kBatch / kWave;
  constexpr int kIdsPerLane = kCandCap / kWave;

  __shared__ uint32_t ht[HT::kSize];
  __shared__ uint32_t cand[kCandCap];
  __shared__ uint32_t beam[kMaxW];

  const int l = lane_id();
  const int g = l >> 3;
  const int gl = l & 7;
  const uint32_t dwords = p.D >> 2;
  const uint32_t beams_per_group = min(kCandCap / p.R, (uint32_t)kWave);

  unsigned long long n_eval = 0, n_reeval = 0, n_exp = 0, n_iter = 0;

  for (uint32_t qi = blockIdx.x; qi < p.nq; qi += gridDim.x) {
    HT::clear(ht);
    U8Vec<VDW, EXACT> q;
    q.load(p.queries + (uint64_t)qi * p.D, gl, dwords);
    int qq = 0;
#pragma unroll
    for (int t = 0; t < VDW; ++t) qq += (int)__builtin_amdgcn_udot4(q.w[t], q.w[t], 0u, false);
    qq = sum8(qq);
    __syncthreads();

    uint32_t ht_used = 0;
    bool forgot = false;  // some node may have been evaluated twice

    // V = {entry}
    uint64_t F[KPL];
#pragma unroll
    for (int r = 0; r < KPL; ++r) F[r] = kInfKey;
    {
      U8Vec<VDW, EXACT> x;
      x.load(p.pages + record_offset(p.geom, slot_ct<N2S>(p.geom, p.entry)), gl, dwords);
      int d = sum8(partial_u8(q, x)) + qq;
      if (l == 0) {
        F[0] = ((uint64_t)(uint32_t)d << 32) | ((uint64_t)p.entry << 1);
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
        const uint64_t my_rec = record_offset(p.geom, slot_ct<N2S>(p.geom, my_beam));
        const uint32_t my_deg = *reinterpret_cast<const uint32_t *>(p.pages + my_rec + p.geom.vec_bytes);
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
          const uint64_t rec = __shfl(my_rec, (int)slot_beam[t]);
          ids[t] = reinterpret_cast<const uint32_t *>(p.pages + rec + p.geom.vec_bytes + 4)[slot_j[t]];
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
          if (isnew[t]) cand[cnt + lanes_below(mnew)] = ids[t];
          cnt += (uint32_t)__popcll(mnew);
          ht_used += (uint32_t)__popcll(mrec);
          const uint32_t lost = (uint32_t)__popcll(mnew & ~mrec);
          n_reeval += lost;
          forgot |= lost != 0;
        }
        __syncthreads();
        n_eval += cnt;

        // ---- evaluate: gather a batch of vectors in one round trip -------------
        for (uint32_t c0 = 0; c0 < cnt; c0 += kBatch) {
          // candidate node -> record; lanes past the count read the entry record
          uint64_t rec[kRounds];
#pragma unroll
          for (int rr = 0; rr < kRounds; ++rr) {
            if (c0 + rr * 8 >= cnt) break;
            const uint32_t idx = c0 + rr * 8 + g;
            const uint32_t node = idx < cnt ? cand[idx] : p.entry;
            rec[rr] = record_offset(p.geom, slot_ct<N2S>(p.geom, node));
          }
          U8Vec<VDW, EXACT> x[kRounds];
#pragma unroll
          for (int rr = 0; rr < kRounds; ++rr) {
            if (c0 + rr * 8 >= cnt) break;
            x[rr].load(p.pages + rec[rr], gl, dwords);
          }
          int dist[kChunks];
#pragma unroll
          for (int c = 0; c < kChunks; ++c) dist[c] = 0;
#pragma unroll
          for (int rr = 0; rr < kRounds; ++rr) {
            if (c0 + rr * 8 >= cnt) break;
            const int d = sum8(partial_u8(q, x[rr])) + qq;
            if (gl == (rr & 7)) dist[rr / 8] = d;
          }
          // lane l of chunk c holds candidate c0 + 64c + 8*(l%8) + l/8
          const uint64_t thr = frontier_at<KPL>(F, p.L - 1);
          uint64_t key[kChunks];
          uint64_t pass_mask[kChunks];
          uint32_t survivors = 0;
#pragma unroll
          for (int c = 0; c < kChunks; ++c) {
            const uint32_t my_idx = c0 + c * kWave + gl * 8 + g;
            key[c] = my_idx < cnt ? (((uint64_t)(uint32_t)dist[c] << 32) | ((uint64_t)cand[my_idx] << 1))
                                  : kInfKey;
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
              uint64_t m = pass_mask[c];
              while (m) {
                const int lane = __builtin_ctzll(m);
                m &= m - 1;
                insert_key<KPL>(F, readlane64(key[c], lane));
              }
            }
          } else {
#pragma unroll
            for (int c = 0; c < kChunks; ++c) {
              if (pass_mask[c] == 0) continue;
              uint64_t cc[1] = {key[c]};
              bitonic_sort<1>(cc, true);
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
        p.out_dists[(uint64_t)qi * p.k + e] = ok ? (int32_t)(F[r] >> 32) : INT32_MAX;
      }
    }
  }

  if (l == 0) {
    atomicAdd(&p.stats[0], n_eval);
    atomicAdd(&p.stats[1], n_reeval);
    atomicAdd(&p.stats[2], n_exp);
    atomicAdd(&p.stats[3], n_iter);
  }
}

}  // namespace gorio
