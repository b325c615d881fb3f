// HBM-resident beam search for uint8 vectors: one wavefront per query.
//
// Per query the wave keeps the frontier F (the L best keys of the evaluated
// set, ascending) in registers, 64 * KPL slots, slot e = r * 64 + lane, and its
// visited filter in LDS.  Key = (squared distance << 32) | (node id << 1) |
// expanded bit: ties order by id, and the flag rides along through the
// sorting networks.  One iteration (GORIO Sec. 1 / Sec. 2.2: expand nodes,
// compute distances, update the frontier):
//   select  - the first W unexpanded slots of F (ballot + prefix count);
//   expand  - read each chosen node's degree and neighbour ids;
//   filter  - drop ids already in the visited filter (LDS atomics), compact;
//   evaluate- 8 lanes per 128-B vector, v_dot4_u32_u8 on coalesced reads:
//             sum (q - x)^2 = q.q + sum (x.x - 2 q.x), exact in int32;
//   merge   - keys below F's L-th key are bitonic-sorted in a 64-lane chunk
//             and merged into F (bitonic merge), slots >= L cleared.
#pragma once

#include "common.hpp"

namespace gorio {

struct ResidentParams {
  const uint8_t *pages;    // num_pages * page_bytes, HBM
  PageGeom geom;
  uint32_t n;
  uint32_t D;              // uint8 dimensions (multiple of 4)
  uint32_t R;              // id slots per record
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
template <int VDW>
struct U8Vec {
  uint32_t w[VDW];

  __device__ __forceinline__ void load(const uint8_t *rec, int gl, uint32_t dwords) {
    const uint32_t *p = reinterpret_cast<const uint32_t *>(rec);
#pragma unroll
    for (int t = 0; t < VDW; ++t) {
      uint32_t di = gl * VDW + t;
      w[t] = di < dwords ? p[di] : 0u;
    }
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int t = 0; t < VDW; ++t) w[t] = 0u;
  }
};

// Partial of sum (x.x - 2 q.x) over this lane's dwords.
template <int VDW>
__device__ __forceinline__ int partial_u8(const U8Vec<VDW> &q, const U8Vec<VDW> &x) {
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

template <int KPL, int VDW, int HT_LOG2>
__global__ __launch_bounds__(kWave) void search_resident_u8(ResidentParams p) {
  using HT = VisitedLds<HT_LOG2>;
  __shared__ uint32_t ht[HT::kSize];
  __shared__ uint32_t cand[kCandCap];
  __shared__ uint32_t beam[kMaxW];

  const int l = lane_id();
  const int g = l >> 3;
  const int gl = l & 7;
  const uint32_t dwords = p.D >> 2;
  const uint32_t beams_per_group = kCandCap / p.R;

  unsigned long long n_eval = 0, n_reeval = 0, n_exp = 0, n_iter = 0;

  for (uint32_t qi = blockIdx.x; qi < p.nq; qi += gridDim.x) {
    HT::clear(ht);
    U8Vec<VDW> q;
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
      uint32_t page, off;
      locate(p.geom, p.entry, page, off);
      U8Vec<VDW> x;
      x.load(p.pages + page * p.geom.page_bytes + off, gl, dwords);
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
        const uint32_t b1 = min(nbeam, b0 + beams_per_group);
        // ---- expand + filter ------------------------------------------------
        uint32_t cnt = 0;
        for (uint32_t b = b0; b < b1; ++b) {
          const uint32_t u = first_lane_value(beam[b]);
          uint32_t page, off;
          locate(p.geom, u, page, off);
          const uint8_t *adj = p.pages + page * p.geom.page_bytes + off + p.geom.vec_bytes;
          const uint32_t deg = min(*reinterpret_cast<const uint32_t *>(adj), p.R);
          const uint32_t *ids = reinterpret_cast<const uint32_t *>(adj + 4);
          for (uint32_t j0 = 0; j0 < p.R; j0 += kWave) {
            const uint32_t j = j0 + l;
            uint32_t v = j < deg ? ids[j] : kNoEdge;
            bool valid = v < p.n;
            bool recorded = false;
            bool isnew = valid && HT::test_and_set(ht, v, ht_used < HT::kLimit, recorded);
            uint64_t mnew = ballot(isnew);
            uint64_t mrec = ballot(recorded);
            if (isnew) cand[cnt + lanes_below(mnew)] = v;
            cnt += (uint32_t)__popcll(mnew);
            ht_used += (uint32_t)__popcll(mrec);
            uint32_t lost = (uint32_t)__popcll(mnew & ~mrec);
            n_reeval += lost;
            forgot |= lost != 0;
          }
        }
        __syncthreads();
        n_eval += cnt;

        // ---- evaluate + merge, 64 candidates at a time -----------------------
        for (uint32_t c0 = 0; c0 < cnt; c0 += kWave) {
          U8Vec<VDW> x[8];
#pragma unroll
          for (int rr = 0; rr < 8; ++rr) {
            const uint32_t idx = c0 + rr * 8 + g;
            if (idx < cnt) {
              uint32_t page, off;
              locate(p.geom, cand[idx], page, off);
              x[rr].load(p.pages + page * p.geom.page_bytes + off, gl, dwords);
            } else {
              x[rr].zero();
            }
          }
          int mine = 0;
#pragma unroll
          for (int rr = 0; rr < 8; ++rr) {
            int d = sum8(partial_u8(q, x[rr])) + qq;
            if (gl == rr) mine = d;
          }
          const uint32_t my_idx = c0 + gl * 8 + g;
          uint64_t key = kInfKey;
          if (my_idx < cnt) key = ((uint64_t)(uint32_t)mine << 32) | ((uint64_t)cand[my_idx] << 1);

          // only keys below the current L-th frontier key can enter F
          const uint64_t thr = frontier_at<KPL>(F, p.L - 1);
          const bool pass = key < thr;
          if (ballot(pass) == 0) continue;
          uint64_t c[1] = {pass ? key : kInfKey};
          bitonic_sort<1>(c, true);
          if (!forgot) {
            // no node can repeat: the P smallest of F and C are min(F, C reversed)
            F[KPL - 1] = min64(F[KPL - 1], c[0]);
            bitonic_merge_up<KPL>(F);
          } else {
            merge_dedupe<KPL>(F, c[0]);
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
