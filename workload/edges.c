/*
 * Seeded synthetic graph edges for the benchmark workloads (input generation only).
 *
 * Each node i gets R_near + R_rand out-edges:
 *   - R_near "sampled-nearest" edges: draw a seeded sample of up to `sample` nodes
 *     of i's own cluster (without replacement, never i itself), rank them by exact
 *     squared L2 distance to i (ties by smaller id) and keep the R_near best in
 *     ascending order;
 *   - R_rand seeded uniform random edges over [0, n), distinct, never i and never
 *     a node already in the row.
 *
 * This builds the index graph that the search later walks; it is not part of the
 * search itself.  Each node draws from its own counter-based stream
 * (SplitMix64, Steele/Lea/Flood 2014, seeded by (seed, i)), so the output does
 * not depend on the number of threads.  Sampling without replacement uses
 * Floyd's algorithm (Bentley & Floyd, CACM 1987).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static inline uint64_t sm64_next(uint64_t *s)
{
    uint64_t z = (*s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* Uniform integer in [0, m) by rejection (no modulo bias). */
static inline uint64_t sm64_below(uint64_t *s, uint64_t m)
{
    uint64_t lim = UINT64_MAX - (UINT64_MAX % m);
    uint64_t x;
    do { x = sm64_next(s); } while (x >= lim);
    return x % m;
}

typedef struct { double d; uint32_t id; } near_t;

static inline int near_less(near_t a, near_t b)
{
    return a.d < b.d || (a.d == b.d && a.id < b.id);
}

static double pair_dist(int dtype, const void *x, uint32_t D, uint64_t a, uint64_t b)
{
    if (dtype == 0) {
        const uint8_t *pa = (const uint8_t *)x + a * D, *pb = (const uint8_t *)x + b * D;
        /* exact: D * 255^2 < 2^31 for D <= 33025 (checked by the caller) */
        int32_t s = 0;
        for (uint32_t d = 0; d < D; ++d) {
            int32_t t = (int32_t)pa[d] - (int32_t)pb[d];
            s += t * t;
        }
        return (double)s;
    } else {
        /* four interleaved float64 partial sums, combined in a fixed order: the
           same value on every machine, and the loop vectorizes */
        const float *pa = (const float *)x + a * D, *pb = (const float *)x + b * D;
        double s[4] = {0.0, 0.0, 0.0, 0.0};
        uint32_t d = 0;
        for (; d + 4 <= D; d += 4)
            for (int j = 0; j < 4; ++j) {
                double t = (double)pa[d + j] - (double)pb[d + j];
                s[j] += t * t;
            }
        for (; d < D; ++d) {
            double t = (double)pa[d] - (double)pb[d];
            s[0] += t * t;
        }
        return (s[0] + s[1]) + (s[2] + s[3]);
    }
}

/*
 * dtype: 0 = uint8, 1 = float32.
 * cluster_start[C+1] / members[n]: nodes of cluster c are
 *   members[cluster_start[c] .. cluster_start[c+1]) in ascending id order.
 * x: n x D row-major in members order (row t is the vector of node members[t]),
 *   so each cluster's vectors are contiguous.
 * graph: n x (r_near + r_rand) output.
 * Returns 0 on success, -1 on bad arguments, -2 on allocation failure.
 */
int gen_edges(int dtype, const void *x, uint64_t n, uint32_t D,
              const uint64_t *cluster_start, const uint32_t *members,
              const uint32_t *label, uint32_t C,
              uint32_t sample, uint32_t r_near, uint32_t r_rand,
              uint64_t seed, uint32_t *graph)
{
    const uint32_t R = r_near + r_rand;
    if (n < 2 || D == 0 || R == 0 || (uint64_t)r_rand + r_near >= n) return -1;
    if (dtype == 0 && D > 33025) return -1;
    uint64_t max_m = 0;
    for (uint32_t c = 0; c < C; ++c) {
        uint64_t m = cluster_start[c + 1] - cluster_start[c];
        if (m > max_m) max_m = m;
    }
    int err = 0;
#pragma omp parallel
    {
        uint32_t *pick = (uint32_t *)malloc(sizeof(uint32_t) * (sample + 1));
        uint8_t *mark = (uint8_t *)calloc(max_m + 1, 1);
        near_t *best = (near_t *)malloc(sizeof(near_t) * (r_near + 1));
        if (!pick || !mark || !best) {
#pragma omp atomic write
            err = -2;
        }
        /* nodes are visited cluster by cluster (members order), so the cluster a
           node samples from stays in cache; each node's output depends only on
           its own stream, not on the visiting order */
#pragma omp for schedule(dynamic, 256)
        for (int64_t ii = 0; ii < (int64_t)n; ++ii) {
            if (err) continue;
            const uint64_t i = members[ii];
            uint64_t st = seed * 0xD1B54A32D192ED03ull ^ ((i + 1) * 0x8CB92BA72F3D8DD7ull);
            const uint32_t c = label[i];
            const uint64_t base = cluster_start[c];
            const uint64_t m = cluster_start[c + 1] - base;
            /* position of i inside its (sorted) cluster list */
            uint64_t lo = 0, hi = m;
            while (lo < hi) {
                uint64_t mid = (lo + hi) / 2;
                if (members[base + mid] < i) lo = mid + 1; else hi = mid;
            }
            const uint64_t self_pos = lo;
            /* row of node i in x */
            const uint64_t xi = (uint64_t)ii;
            const uint64_t M = m - 1; /* cluster without i */
            uint64_t cnt = 0;
            if (M <= sample) {
                for (uint64_t t = 0; t < M; ++t) pick[cnt++] = (uint32_t)t;
            } else {
                for (uint64_t j = M - sample; j < M; ++j) {
                    uint64_t t = sm64_below(&st, j + 1);
                    if (mark[t]) t = j;
                    mark[t] = 1;
                    pick[cnt++] = (uint32_t)t;
                }
                for (uint64_t t = 0; t < cnt; ++t) mark[pick[t]] = 0;
            }
            /* keep the r_near best (dist, id), ascending */
            uint32_t nb = 0;
            for (uint64_t t = 0; t < cnt; ++t) {
                uint64_t p = pick[t];
                const uint64_t xv = base + (p < self_pos ? p : p + 1);
                uint32_t v = members[xv];
                near_t e = { pair_dist(dtype, x, D, xi, xv), v };
                if (nb == r_near && !near_less(e, best[nb - 1])) continue;
                uint32_t pos = (nb < r_near) ? nb++ : nb - 1;
                while (pos > 0 && near_less(e, best[pos - 1])) { best[pos] = best[pos - 1]; --pos; }
                best[pos] = e;
            }
            uint32_t *row = graph + i * R;
            uint32_t fill = 0;
            for (uint32_t t = 0; t < nb; ++t) row[fill++] = best[t].id;
            /* random edges: distinct, not self, not already present */
            while (fill < R) {
                uint32_t v = (uint32_t)sm64_below(&st, n);
                if (v == i) continue;
                int dup = 0;
                for (uint32_t t = 0; t < fill; ++t) if (row[t] == v) { dup = 1; break; }
                if (!dup) row[fill++] = v;
            }
        }
        free(pick); free(mark); free(best);
    }
    return err;
}
