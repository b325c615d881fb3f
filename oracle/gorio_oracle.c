/*
 * CPU oracle for paged graph beam search  --  TEST INFRASTRUCTURE ONLY.
 *
 * This file is the plain, slow, single-threaded reference that the GPU library
 * is checked against.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg load it; the GPU library never links, includes
 * or calls anything here, and nothing here is shared with it.
 *
 * What it computes (GORIO, Sec. 1 and Sec. 2.2: each query repeatedly expands
 * graph nodes, computes distances, updates a candidate frontier and discovers
 * the next pages to fetch; the search follows DiskANN's beam search, which the
 * paper's related-work section names as the graph-index family it targets):
 *
 *   key(v) = (dist(q, vec(v)), v)                  total order, smaller is better
 *   V = {entry}  (evaluated set),  X = {}  (expanded set)
 *   repeat:
 *     F = the min(L, |V|) smallest keys of V, ascending      (frontier)
 *     S = the first min(W, .) members of F, in F order, not in X   (beam)
 *     stop if S is empty
 *     X = X + S
 *     for u in S, for j < degree(u): v = id_j(u); skip v >= n;
 *         if v not in V: add v to V
 *   answer = first k of F, padded with (UINT32_MAX, INT32_MAX / +inf)
 *
 * The frontier is kept incrementally (sorted insertion, truncated to L).  This
 * equals the recomputed top-L of V because top-L(top-L(A) u B) = top-L(A u B);
 * debug mode recomputes F from V after every iteration and checks it.
 *
 * Records are read through this file's own page decoder from pages this file
 * packed itself:  node v lives at slot s = node_to_slot ? node_to_slot[v] : v,
 * position i = s % rpp of page s / rpp.  Its record is
 *   vector:          D bytes (uint8) or D little-endian float32
 *   adjacency block: [ uint32 degree ] [ R x uint32 neighbour ids, UINT32_MAX-padded ]
 * placed inside the page in one of two arrangements (the paper fixes the
 * block-granular 4 KB page as the unit, Sec. 3.1 and Fig. 1, and says nothing
 * about the bytes inside it):
 *   contiguous:    record i at byte i * record_bytes, vector then block;
 *   vectors first: vector i at byte i * V (V = vector bytes rounded up to 16),
 *                  block i at byte rpp * V + i * (record_bytes - V).
 * Every byte not written is zero.  Records never straddle pages.
 *
 * Distances are squared L2, returned squared:
 *   uint8:  exact integer sum of (q_d - x_d)^2;
 *   float32: t = q_d - x_d; acc = acc + t*t, each operation rounded to float32,
 *            d = 0 .. D-1 in order, no fused multiply-add (compile with
 *            -ffp-contract=off), no flush-to-zero.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_EINVAL 1
#define ORC_ENOMEM 2
#define ORC_EINVARIANT 3

#define ORC_U8 0
#define ORC_F32 1

#define ORC_NO_EDGE 0xFFFFFFFFu

typedef struct {
    const uint8_t *pages;
    uint64_t n;
    uint32_t D;
    uint32_t R;
    int32_t dtype;
    uint32_t page_bytes;
    uint32_t record_bytes;
    uint32_t records_per_page;
    const uint32_t *node_to_slot; /* NULL: slot = node id */
    uint32_t entry;
    int32_t vectors_first;        /* page arrangement, see above */
} orc_index;

typedef struct {
    uint64_t evaluations;  /* |V| at the end, the entry included */
    uint64_t expansions;   /* |X| at the end */
    uint64_t iterations;   /* beams expanded */
} orc_counts;

static uint32_t vec_bytes(int32_t dtype, uint32_t D)
{
    return dtype == ORC_U8 ? D : 4u * D;
}

/* vector slot width in a vectors-first page */
static uint32_t vec_slot(int32_t dtype, uint32_t D)
{
    return (vec_bytes(dtype, D) + 15u) / 16u * 16u;
}

/* smallest record for the arrangement */
uint32_t orc_record_bytes(int32_t dtype, uint32_t D, uint32_t R, int32_t vectors_first)
{
    return (vectors_first ? vec_slot(dtype, D) : vec_bytes(dtype, D)) + 4u + 4u * R;
}

/* ------------------------------------------------------------------------ */
/* distances                                                                 */
/* ------------------------------------------------------------------------ */
uint32_t orc_dist_u8(const uint8_t *a, const uint8_t *b, uint32_t D)
{
    uint64_t s = 0;
    for (uint32_t d = 0; d < D; ++d) {
        int64_t t = (int64_t)a[d] - (int64_t)b[d];
        s += (uint64_t)(t * t);
    }
    return (uint32_t)s;
}

float orc_dist_f32(const float *a, const float *b, uint32_t D)
{
    float acc = 0.0f;
    for (uint32_t d = 0; d < D; ++d) {
        float t = a[d] - b[d];
        float sq = t * t;
        acc = acc + sq;
    }
    return acc;
}

static uint32_t float_bits(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    return u;
}

/* ------------------------------------------------------------------------ */
/* page packing and decoding                                                 */
/* ------------------------------------------------------------------------ */
static const uint8_t *page_of(const orc_index *ix, uint64_t v, uint64_t *pos)
{
    uint64_t s = ix->node_to_slot ? ix->node_to_slot[v] : v;
    *pos = s % ix->records_per_page;
    return ix->pages + (s / ix->records_per_page) * ix->page_bytes;
}

/* node v's vector */
static const uint8_t *vector_of(const orc_index *ix, uint64_t v)
{
    uint64_t i;
    const uint8_t *page = page_of(ix, v, &i);
    if (ix->vectors_first) return page + i * vec_slot(ix->dtype, ix->D);
    return page + i * ix->record_bytes;
}

/* node v's adjacency block: degree, then R ids */
static const uint8_t *adjacency_of(const orc_index *ix, uint64_t v)
{
    uint64_t i;
    const uint8_t *page = page_of(ix, v, &i);
    if (ix->vectors_first) {
        const uint64_t V = vec_slot(ix->dtype, ix->D);
        return page + ix->records_per_page * V + i * (ix->record_bytes - V);
    }
    return page + i * ix->record_bytes + vec_bytes(ix->dtype, ix->D);
}

static uint32_t load_u32(const uint8_t *p)
{
    return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) | ((uint32_t)p[3] << 24);
}

static void store_u32(uint8_t *p, uint32_t v)
{
    p[0] = (uint8_t)v; p[1] = (uint8_t)(v >> 8); p[2] = (uint8_t)(v >> 16); p[3] = (uint8_t)(v >> 24);
}

uint64_t orc_num_pages(uint64_t n, uint32_t records_per_page)
{
    return (n + records_per_page - 1) / records_per_page;
}

/*
 * Checks the layout and graph, then writes num_pages * page_bytes bytes to
 * pages_out.  A graph row's UINT32_MAX entries mean "no edge"; the record
 * keeps the row's real edges in their given order, degree = their count, and
 * fills the rest of the id array with UINT32_MAX.  Any other id >= n, a
 * record that does not fit, or a node_to_slot that is not a permutation of
 * [0, n) is rejected with ORC_EINVAL.
 */
int orc_pack(int32_t dtype, const void *vectors, uint64_t n, uint32_t D,
             const uint32_t *graph, uint32_t R,
             uint32_t page_bytes, uint32_t record_bytes, uint32_t records_per_page,
             const uint32_t *node_to_slot, int32_t vectors_first, uint8_t *pages_out)
{
    if ((dtype != ORC_U8 && dtype != ORC_F32) || n == 0 || D == 0 || R == 0) return ORC_EINVAL;
    if (vectors_first != 0 && vectors_first != 1) return ORC_EINVAL;
    if (records_per_page == 0 || record_bytes < orc_record_bytes(dtype, D, R, vectors_first))
        return ORC_EINVAL;
    if ((uint64_t)record_bytes * records_per_page > page_bytes) return ORC_EINVAL;
    if (n >= 0x80000000ull) return ORC_EINVAL;
    for (uint64_t i = 0; i < n * R; ++i)
        if (graph[i] != ORC_NO_EDGE && graph[i] >= n) return ORC_EINVAL;
    if (node_to_slot) {
        uint8_t *seen = (uint8_t *)calloc(n, 1);
        if (!seen) return ORC_ENOMEM;
        for (uint64_t i = 0; i < n; ++i) {
            if (node_to_slot[i] >= n || seen[node_to_slot[i]]) { free(seen); return ORC_EINVAL; }
            seen[node_to_slot[i]] = 1;
        }
        free(seen);
    }
    orc_index ix = { pages_out, n, D, R, dtype, page_bytes, record_bytes, records_per_page,
                     node_to_slot, 0, vectors_first };
    memset(pages_out, 0, orc_num_pages(n, records_per_page) * (uint64_t)page_bytes);
    const uint32_t vb = vec_bytes(dtype, D);
    for (uint64_t v = 0; v < n; ++v) {
        memcpy((uint8_t *)vector_of(&ix, v), (const uint8_t *)vectors + v * vb, vb);
        uint8_t *adj = (uint8_t *)adjacency_of(&ix, v);
        uint32_t deg = 0;
        for (uint32_t j = 0; j < R; ++j) {
            uint32_t u = graph[v * R + j];
            if (u != ORC_NO_EDGE) store_u32(adj + 4 + 4 * deg++, u);
        }
        for (uint32_t j = deg; j < R; ++j) store_u32(adj + 4 + 4 * j, ORC_NO_EDGE);
        store_u32(adj, deg);
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* entry point: the medoid rule                                              */
/* ------------------------------------------------------------------------ */
/*
 * uint8:   c_d = floor((sum_i x_id + floor(n/2)) / n)  (integer arithmetic)
 * float32: c_d = (float)(sum_i (double)x_id / n), summed in i order
 * entry = the node minimising dist(c, x_i), ties to the smaller id.
 */
uint32_t orc_medoid(int32_t dtype, const void *vectors, uint64_t n, uint32_t D)
{
    uint32_t best = 0;
    if (dtype == ORC_U8) {
        const uint8_t *x = (const uint8_t *)vectors;
        uint8_t *c = (uint8_t *)malloc(D);
        for (uint32_t d = 0; d < D; ++d) {
            uint64_t s = 0;
            for (uint64_t i = 0; i < n; ++i) s += x[i * D + d];
            c[d] = (uint8_t)((s + n / 2) / n);
        }
        uint32_t bd = 0xFFFFFFFFu;
        for (uint64_t i = 0; i < n; ++i) {
            uint32_t dd = orc_dist_u8(c, x + i * D, D);
            if (dd < bd) { bd = dd; best = (uint32_t)i; }
        }
        free(c);
    } else {
        const float *x = (const float *)vectors;
        float *c = (float *)malloc(sizeof(float) * D);
        for (uint32_t d = 0; d < D; ++d) {
            double s = 0.0;
            for (uint64_t i = 0; i < n; ++i) s += (double)x[i * D + d];
            c[d] = (float)(s / (double)n);
        }
        uint32_t bd = 0xFFFFFFFFu;
        for (uint64_t i = 0; i < n; ++i) {
            uint32_t dd = float_bits(orc_dist_f32(c, x + i * D, D));
            if (dd < bd) { bd = dd; best = (uint32_t)i; }
        }
        free(c);
    }
    return best;
}

/* ------------------------------------------------------------------------ */
/* beam search                                                               */
/* ------------------------------------------------------------------------ */
typedef struct {
    uint64_t key;      /* (distance bits << 32) | node id */
    int expanded;
} fentry;

typedef struct {
    uint8_t *in_v;     /* n flags: node is in V */
    uint8_t *in_x;     /* n flags: node is in X */
    uint64_t *vkeys;   /* keys of V in evaluation order */
    uint64_t vcap;
    fentry *f;         /* frontier, ascending, at most L entries */
    uint64_t *scratch; /* debug: recomputed frontier */
} workspace;

static uint64_t key_of(const orc_index *ix, const void *q, uint32_t v)
{
    const uint8_t *rec = vector_of(ix, v);
    uint32_t dbits;
    if (ix->dtype == ORC_U8) {
        dbits = orc_dist_u8((const uint8_t *)q, rec, ix->D);
    } else {
        float xv[1024];
        const float *xp = xv;
        /* the record is little-endian float32; copy out to an aligned array */
        memcpy(xv, rec, 4u * ix->D);
        dbits = float_bits(orc_dist_f32((const float *)q, xp, ix->D));
    }
    return ((uint64_t)dbits << 32) | v;
}

/* Insert a key (not already present) into the sorted frontier of size *fs. */
static void frontier_insert(fentry *f, uint32_t *fs, uint32_t L, uint64_t key)
{
    uint32_t p = 0;
    while (p < *fs && f[p].key < key) ++p;
    if (p >= L) return;                       /* worse than all L kept keys */
    uint32_t last = (*fs < L) ? *fs : L - 1;  /* the L-th entry falls off when full */
    for (uint32_t i = last; i > p; --i) f[i] = f[i - 1];
    f[p].key = key;
    f[p].expanded = 0;
    if (*fs < L) ++*fs;
}

static int cmp_u64(const void *a, const void *b)
{
    uint64_t x = *(const uint64_t *)a, y = *(const uint64_t *)b;
    return x < y ? -1 : (x > y);
}

/* Debug check: F is strictly ascending and equals top-L(V) with X's flags. */
static int check_frontier(const workspace *w, uint64_t nv, const fentry *f, uint32_t fs, uint32_t L)
{
    for (uint32_t i = 1; i < fs; ++i)
        if (!(f[i - 1].key < f[i].key)) return ORC_EINVARIANT;
    uint64_t want = nv < L ? nv : L;
    if (fs != want) return ORC_EINVARIANT;
    memcpy(w->scratch, w->vkeys, nv * sizeof(uint64_t));
    qsort(w->scratch, nv, sizeof(uint64_t), cmp_u64);
    for (uint32_t i = 0; i < fs; ++i) {
        if (w->scratch[i] != f[i].key) return ORC_EINVARIANT;
        uint32_t id = (uint32_t)(f[i].key & 0xFFFFFFFFu);
        if ((w->in_x[id] != 0) != (f[i].expanded != 0)) return ORC_EINVARIANT;
    }
    return ORC_OK;
}

static int search_one(const orc_index *ix, workspace *w, const void *q,
                      uint32_t k, uint32_t L, uint32_t W,
                      uint32_t *ids, void *dists, orc_counts *cnt,
                      uint32_t *trace, uint64_t trace_cap, int debug)
{
    fentry *f = w->f;
    uint32_t fs = 0;
    uint64_t nv = 0, nx = 0, iters = 0, prev_nv = 0;
    uint32_t beam[256];
    int rc = ORC_OK;

    /* V = {entry} */
    w->in_v[ix->entry] = 1;
    w->vkeys[nv++] = key_of(ix, q, ix->entry);
    frontier_insert(f, &fs, L, w->vkeys[0]);

    for (uint64_t guard = 0; guard <= ix->n; ++guard) {
        /* beam: first W unexpanded frontier members, in frontier order */
        uint32_t nb = 0;
        for (uint32_t i = 0; i < fs && nb < W; ++i)
            if (!f[i].expanded) {
                f[i].expanded = 1;
                beam[nb++] = (uint32_t)(f[i].key & 0xFFFFFFFFu);
            }
        if (nb == 0) break;
        for (uint32_t b = 0; b < nb; ++b) {
            uint32_t u = beam[b];
            w->in_x[u] = 1;
            if (trace && nx < trace_cap) trace[nx] = u;
            ++nx;
            const uint8_t *adj = adjacency_of(ix, u);
            uint32_t deg = load_u32(adj);
            if (deg > ix->R) deg = ix->R;
            for (uint32_t j = 0; j < deg; ++j) {
                uint32_t v = load_u32(adj + 4 + 4 * j);
                if (v >= ix->n || w->in_v[v]) continue;
                w->in_v[v] = 1;
                uint64_t key = key_of(ix, q, v);
                if (nv == w->vcap) {
                    uint64_t ncap = w->vcap * 2;
                    uint64_t *nk = (uint64_t *)realloc(w->vkeys, ncap * sizeof(uint64_t));
                    uint64_t *ns = (uint64_t *)realloc(w->scratch, ncap * sizeof(uint64_t));
                    if (!nk || !ns) { if (nk) w->vkeys = nk; if (ns) w->scratch = ns; rc = ORC_ENOMEM; goto done; }
                    w->vkeys = nk; w->scratch = ns; w->vcap = ncap;
                }
                w->vkeys[nv++] = key;
                frontier_insert(f, &fs, L, key);
            }
        }
        ++iters;
        if (debug) {
            if (nv < prev_nv) { rc = ORC_EINVARIANT; goto done; }
            prev_nv = nv;
            rc = check_frontier(w, nv, f, fs, L);
            if (rc != ORC_OK) goto done;
        }
    }

    for (uint32_t i = 0; i < k; ++i) {
        if (i < fs) {
            ids[i] = (uint32_t)(f[i].key & 0xFFFFFFFFu);
            uint32_t db = (uint32_t)(f[i].key >> 32);
            if (ix->dtype == ORC_U8) ((int32_t *)dists)[i] = (int32_t)db;
            else memcpy((float *)dists + i, &db, 4);
        } else {
            ids[i] = ORC_NO_EDGE;
            if (ix->dtype == ORC_U8) ((int32_t *)dists)[i] = INT32_MAX;
            else { uint32_t inf = 0x7F800000u; memcpy((float *)dists + i, &inf, 4); }
        }
    }
    if (cnt) { cnt->evaluations = nv; cnt->expansions = nx; cnt->iterations = iters; }
done:
    /* reset the flags this query set, so the workspace is clean for the next one */
    for (uint64_t i = 0; i < nv; ++i) {
        uint32_t id = (uint32_t)(w->vkeys[i] & 0xFFFFFFFFu);
        w->in_v[id] = 0;
        w->in_x[id] = 0;
    }
    return rc;
}

/*
 * Searches queries [q_begin, q_end) of the nq x D query array one after the
 * other.  ids / dists are nq x k (int32 for uint8 data, float32 otherwise);
 * counts (nullable) is nq entries; trace (nullable) receives, per query, the
 * expanded nodes in expansion order (trace_cap entries per query).
 */
int orc_search(const orc_index *ix, const void *queries, uint64_t q_begin, uint64_t q_end,
               uint32_t k, uint32_t L, uint32_t W,
               uint32_t *ids, void *dists, orc_counts *counts,
               uint32_t *trace, uint64_t trace_cap, int debug)
{
    if (!ix || ix->entry >= ix->n || k == 0 || L == 0 || W == 0 || k > L || W > 256)
        return ORC_EINVAL;
    if (ix->dtype == ORC_F32 && ix->D > 1024) return ORC_EINVAL;
    workspace w;
    w.in_v = (uint8_t *)calloc(ix->n, 1);
    w.in_x = (uint8_t *)calloc(ix->n, 1);
    w.vcap = 4096;
    w.vkeys = (uint64_t *)malloc(w.vcap * sizeof(uint64_t));
    w.scratch = (uint64_t *)malloc(w.vcap * sizeof(uint64_t));
    w.f = (fentry *)malloc((uint64_t)L * sizeof(fentry));
    int rc = ORC_OK;
    if (!w.in_v || !w.in_x || !w.vkeys || !w.scratch || !w.f) rc = ORC_ENOMEM;
    const uint32_t qb = vec_bytes(ix->dtype, ix->D);
    for (uint64_t qi = q_begin; qi < q_end && rc == ORC_OK; ++qi) {
        const void *q = (const uint8_t *)queries + qi * qb;
        void *dq = ix->dtype == ORC_U8 ? (void *)((int32_t *)dists + qi * k)
                                       : (void *)((float *)dists + qi * k);
        rc = search_one(ix, &w, q, k, L, W, ids + qi * k, dq, counts ? counts + qi : NULL,
                        trace ? trace + qi * trace_cap : NULL, trace_cap, debug);
    }
    free(w.in_v); free(w.in_x); free(w.vkeys); free(w.scratch); free(w.f);
    return rc;
}
