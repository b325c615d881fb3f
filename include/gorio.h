/*
 * gorio.h -- C ABI of the MI355X (gfx950) paged graph beam-search library.
 *
 * The library implements the GPU side of GORIO ("GPU-Centered Remote I/O for
 * Graph ANNS over NVMe-oF"): batched DiskANN-style beam search whose node
 * records live in 4 KB pages.  Every search-side decision is taken on the GPU:
 * how each query advances, which pages it is missing, where a query waiting
 * for pages is kept and when it continues (Sec. 3.1, Fig. 1).  A host proxy
 * thread does nothing but read pages from the backing store and post their
 * completions where the GPU can see them (Sec. 3.3, Sec. 4 "CPU transport
 * proxy").  On one GPU a pinned host-memory backing store with an injected
 * per-request latency takes the place of the remote NVMe-oF namespace of
 * Sec. 4 ("Remote storage").
 *
 * Search semantics (Sec. 1 and Sec. 2.2 describe the search only as a loop
 * that grows a candidate frontier by visiting graph nodes and scoring their
 * neighbours, which in turn names the pages to read next):
 *   key(v) = (squared L2 distance(q, v), v)       -- ties broken by node id
 *   V = {entry};  X = {}
 *   repeat: F = the min(L, |V|) smallest keys of V;
 *           S = the first min(W, .) members of F not in X (in F order);
 *           stop if S is empty;  X += S;
 *           for u in S, for each of u's edges v: if v not in V, V += {v}
 *   result = the first k members of F.
 * Results do not depend on the cache size, the backing latency or the order
 * in which page requests complete.
 *
 * Page layout: node v is stored at slot s = node_to_slot ? node_to_slot[v] : v,
 * position i = s % records_per_page of page s / records_per_page.  Its record
 * is a vector (D x uint8 or D x float32) and an adjacency block ([uint32
 * degree][R x uint32 ids, padded with UINT32_MAX]).  A graph row's UINT32_MAX
 * entries mean "no edge"; the block keeps the row's other ids in order and
 * degree = their count.  Inside a page (bytes not covered below are zero):
 *   vectors first (the default): vector i at byte i * V, where V = vector
 *     bytes rounded up to 16, then adjacency block i at byte
 *     records_per_page * V + i * (record_bytes - V).  For 128-byte vectors
 *     every vector starts on a 128-byte line, so a distance evaluation reads
 *     one line instead of two;
 *   contiguous: record i at byte i * record_bytes, the adjacency block right
 *     after the vector (DiskANN's record order).
 * Both layouts put the same nodes in the same pages; only the bytes inside a
 * page move.
 *
 * Conventions for every call:
 *   - Status codes, never exceptions; gorio_last_error() returns a
 *     thread-local message for the last failing call on this thread.
 *   - The caller owns every array it passes; the library copies what it keeps.
 *   - One thread at a time per index; no call on an index may overlap a
 *     search on it from another thread.  Searches of one index issued on
 *     different streams run one after another: a search on another stream
 *     than the previous search of the index waits on the GPU for that search
 *     (an event the index records), because they share the index's counters;
 *     on the same stream, stream order does it where that stream is the null
 *     or the per-thread stream; on a created stream the search waits for the
 *     event all the same (a stream created after another was destroyed can
 *     get the same handle).  Different indexes may be
 *     used from different threads.
 *   - The device is the HIP device current when gorio_build_index is called;
 *     later calls switch to it and restore the caller's device.
 *
 * Environment (read by each paged search; tuning and test hooks, none needed
 * for normal use):
 *   GORIO_FILL_WAVES       waves that only copy arriving pages (default 32, at most 64)
 *   GORIO_MAX_PENDING      page requests per query, overriding gorio_set_scheduler's
 *   GORIO_HOST_EXECUTOR    host-scheduled lanes: 1 (default) = one persistent launch runs
 *                          the turns the host writes to a ring; 0 = a launch per round
 *   GORIO_TURN_PASSES      host-scheduled lanes: passes that found pages ready before a lane
 *                          yields (default: none with the executor, 2 with a launch per round)
 *   GORIO_FILL_BUDGET_US   launch per round: the fill kernel leaves after this long and is
 *                          launched again (default 2000)
 *   GORIO_ROUND_FLIGHTS    launch per round: round kernels in flight, each on a stream of
 *                          its own (default 2, at most 8)
 *   GORIO_ROUNDS_STATS     1: print the host scheduler's counters to stderr
 *   GORIO_WATCHDOG_S       a paged search still running after this many seconds is
 *                          aborted with GORIO_ETIMEOUT (default 120)
 *   GORIO_PROXY_JITTER_US  extra random delay per page request (completions reorder)
 *   GORIO_PROXY_HOLD       1: the proxy completes nothing (exercises the watchdog)
 *   GORIO_CTRL_STRIDE      spacing of the paged search's control words, in 8-byte words
 *                          (default 32, read when the cache is set)
 */
#ifndef GORIO_H
#define GORIO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct gorio_index gorio_index;

typedef enum {
    GORIO_OK = 0,
    GORIO_EINVAL = 1,        /* an argument is out of range or inconsistent */
    GORIO_ENOMEM = 2,        /* device or pinned host allocation failed */
    GORIO_EDEVICE = 3,       /* a HIP runtime call or a kernel failed */
    GORIO_ETIMEOUT = 4,      /* paged search did not finish within the watchdog limit */
    GORIO_EUNSUPPORTED = 5   /* valid request the library does not implement */
} gorio_status;

typedef enum { GORIO_U8 = 0, GORIO_F32 = 1 } gorio_dtype;

/* Arrangement of the bytes inside a page (see the top of this file). */
typedef enum {
    GORIO_LAYOUT_DEFAULT = 0,        /* vectors first */
    GORIO_LAYOUT_VECTORS_FIRST = 1,
    GORIO_LAYOUT_CONTIGUOUS = 2
} gorio_arrangement;

/* Node-record placement in pages.  Zero fields take the default. */
typedef struct {
    uint32_t page_bytes;          /* page size; default 4096; multiple of 16 */
    uint32_t record_bytes;        /* bytes per node; default V + 4 + 4R with V = vec_bytes
                                     (contiguous) or vec_bytes rounded up to 16 (vectors
                                     first); >= that default's minimum, multiple of 4 */
    uint32_t records_per_page;    /* default page_bytes / record_bytes */
    uint32_t arrangement;         /* gorio_arrangement; 0 = default (vectors first) */
    const uint32_t *node_to_slot; /* host array of n entries, a permutation of [0, n); NULL = identity */
} gorio_page_layout;

/* Per-search counters (filled when gorio_search gets a non-NULL stats). */
typedef struct {
    double kernel_ms;          /* GPU time of the search launch(es), HIP events on the search stream */
    double wall_ms;            /* host wall time inside gorio_search */
    uint64_t evaluations;      /* distance evaluations, including re-evaluations */
    uint64_t reevaluations;    /* evaluations whose node could not be recorded in the visited filter
                                  (may repeat an earlier one of the same query) */
    uint64_t expansions;       /* nodes expanded (adjacency lists read) */
    uint64_t iterations;       /* beams expanded, summed over queries */
    uint64_t hits;             /* paged mode: record accesses served by a resident page */
    uint64_t misses;           /* paged mode: record accesses that had to wait for a page */
    uint64_t pages_served;     /* paged mode: pages moved from the backing store into the cache */
    uint64_t bytes_served;     /* paged mode: pages_served * page_bytes */
    uint64_t parks;            /* paged mode: times a query was set aside waiting for pages */
    uint64_t resumes;          /* paged mode: times a parked query was picked up again */
    uint64_t proxy_peak;       /* paged mode: most page requests the proxy held at once */
} gorio_stats;

/* Read-only facts about a built index. */
typedef struct {
    gorio_dtype dtype;
    uint64_t n;
    uint32_t D, R;
    uint32_t page_bytes, record_bytes, records_per_page;
    int vectors_first;         /* 1: vectors-first pages, 0: contiguous records */
    uint64_t num_pages;
    uint64_t index_bytes;      /* num_pages * page_bytes */
    uint32_t entry;            /* entry node used by every search */
    int resident;              /* 1: all pages in HBM; 0: paged through the HBM cache */
    uint64_t cache_slots;      /* paged mode: number of page slots in the HBM cache */
    int device;                /* HIP device ordinal */
} gorio_index_info;

/*
 * Build an index: pack records into pages and choose the entry node.  The
 * index is a DiskANN-style graph (Sec. 5.1) stored as fixed-size graph pages
 * that are the unit of every read (Sec. 3.1, Fig. 1: graph pages on the remote
 * namespace; Sec. 4 "Remote storage": the page-cache path fetches whole
 * pages).  Record and page layout as described at the top of this file.
 *   vectors: host, n x D row-major (uint8 or float32 per dtype).
 *   graph:   host, n x R row-major uint32; UINT32_MAX = no edge; any other id must be < n.
 *   layout:  NULL = all defaults.
 *   entry:   UINT32_MAX = medoid rule: the node nearest (squared L2, ties to the
 *            smaller id) to the centroid c, where for uint8 c_d = floor((sum_i x_id
 *            + floor(n/2)) / n) and for float32 c_d = (float)(sum_i (double)x_id / n)
 *            summed in i order; otherwise the given node (< n).
 * Limits: 1 <= n < 2^31; uint8: D % 4 == 0, D <= 512; float32: D <= 256; 1 <= R <= 256.
 * The packed index is placed in HBM (resident mode).  *out is set only on GORIO_OK.
 */
gorio_status gorio_build_index(gorio_dtype dtype, const void *vectors, uint64_t n, uint32_t D,
                               const uint32_t *graph, uint32_t R,
                               const gorio_page_layout *layout, uint32_t entry,
                               gorio_index **out);

/*
 * Size the HBM page cache (GORIO Sec. 3.2: GPU page cache with a per-slot ready
 * table; Sec. 4: BaM-derived page-cache path).
 * bytes >= index_bytes: resident mode, every page in HBM, no misses.
 * otherwise: paged mode with floor(bytes / page_bytes) slots; the pages move
 * to a pinned host backing store and the cache starts cold.  Too few slots for
 * the configured query slots to make progress -> GORIO_EINVAL.
 */
gorio_status gorio_set_cache(gorio_index *ix, uint64_t bytes);

/*
 * Configure the backing-store proxy for paged mode (Sec. 3.3 / Sec. 4: the
 * proxy batches submissions and completions and caps outstanding remote I/O).
 *   latency_us:      injected delay from a page request's publication to its completion (>= 0).
 *   max_outstanding: cap on requests the proxy holds in flight (0 = default 4096).
 *   oversub:         query slots per resident wavefront of the persistent kernel (1..16).
 *   blocking:        scheduling mode.
 *                    0 = split-phase: the persistent GPU scheduler parks a query
 *                        on a missing page and runs other ready queries (Sec. 3.3);
 *                    1 = wait in place for each missing page, one query per wave
 *                        (the blocking demand-paging path the paper compares
 *                        against, Sec. 5.1, Table 2);
 *                    2 = host-scheduled lanes: a host thread (the caller's)
 *                        keeps the query lanes and decides which runs next, as
 *                        their pages are filled; a persistent GPU launch runs the
 *                        turns it hands over through a ring in host memory (or,
 *                        with GORIO_HOST_EXECUTOR=0, a launch per round), using
 *                        the same page cache, descriptors and proxy (the
 *                        GustANN-style scheduler over GORIO's backend that the
 *                        paper compares against, Sec. 5.1, Table 2).  oversub is
 *                        ignored; the lanes are min(query_waves or 8 per compute
 *                        unit, slots / (2 * max_pending), nq, 8192).
 *                    3 = GPU resume queue (Sec. 3.1, Fig. 1: a ready table
 *                        feeding a resume queue): the same lanes, with their
 *                        state in HBM, but nothing on the host except the proxy
 *                        and the watchdog; a lane that parks joins the waiter
 *                        set of each cache slot it waits for, the fill wave
 *                        that makes a slot READY queues those lanes in a run
 *                        queue in HBM, and executor waves of one persistent
 *                        launch run the queued lanes' turns.  oversub is
 *                        ignored; the lanes are counted as in mode 2.
 *                    Results are the same in every mode.
 * Takes effect at the next search.  Ignored in resident mode.
 * Errors: GORIO_EINVAL for a NULL index or an argument out of range.
 */
gorio_status gorio_set_backing(gorio_index *ix, double latency_us, uint32_t max_outstanding,
                               uint32_t oversub, int blocking);

/*
 * Shape of the paged scheduler (Sec. 3.3: the persistent scheduler runs many
 * queries per wave and caps the page requests in flight).
 *   query_waves: most waves that run queries (0 = 8 per compute unit).
 *   max_pending: page requests one query keeps outstanding (1..256; 0 = 32).
 * A search runs min(query_waves * oversub, slots / (2 * max_pending), nq)
 * queries at once, in ceil(that / oversub) waves (one query per wave when
 * blocking): every query may pin max_pending slots, and half of the cache is
 * kept free for the clock to evict.  With equal query_waves, the blocking
 * mode therefore holds oversub times fewer queries than the split-phase mode,
 * which is the comparison of Sec. 5.2 (waits in place vs. yields and runs
 * other queries).  Takes effect at the next search; ignored in resident mode.
 * Errors: GORIO_EINVAL for a NULL index, query_waves > 65536 or
 * max_pending > 256.
 */
gorio_status gorio_set_scheduler(gorio_index *ix, uint32_t query_waves, uint32_t max_pending);

/*
 * Batched search (GORIO Sec. 3.3: persistent scheduler; each query is finished
 * or parked on a missing page and later resumed).
 *   queries: nq x D (uint8 or float32), host or device pointer.
 *   ids:     nq x k uint32 out; dists: nq x k out, int32 (uint8 data) or float32.
 *            Both host or device pointers (detected per pointer).  Host
 *            buffers are staged through a device buffer the index keeps
 *            (grown when a batch needs more) and the call returns once the
 *            answers are back in them.
 *   Slots past the reachable set are padded with UINT32_MAX and INT32_MAX / +inf.
 *   stats:   NULL or a struct to fill; non-NULL makes the call wait for the search.
 *   stream:  hipStream_t to launch on (NULL = the null stream).  With device
 *            pointers and stats == NULL a resident search returns without
 *            waiting; a paged search always returns when it is done (the
 *            calling thread runs its watchdog, and in mode 2 its scheduler).
 * Requires 1 <= k <= L <= 256 and 1 <= W <= L (paged: W <= 64).  nq == 0 is a
 * no-op.  Errors: GORIO_EINVAL for arguments out of range, GORIO_EUNSUPPORTED
 * for a paged W above 64, GORIO_ENOMEM / GORIO_EDEVICE from the device,
 * GORIO_ETIMEOUT when a paged search did not finish within the watchdog
 * limit (the counters so far are filled; the cache is reset), and
 * GORIO_EUNSUPPORTED on a stream under graph capture (each search takes its
 * query tickets from a base the host advances, so a replay would be wrong;
 * gorio_search_noalloc is the entry point to capture).
 */
gorio_status gorio_search(gorio_index *ix, const void *queries, uint64_t nq,
                          uint32_t k, uint32_t L, uint32_t W,
                          uint32_t *ids, void *dists, gorio_stats *stats, void *stream);

/*
 * gorio_search for callers that cannot allocate memory: code running under
 * HIP graph capture, serving loops and harnesses that forbid hipMalloc.  It
 * allocates nothing and stages nothing; the caller passes device buffers.
 * Resident indexes only (a paged index -> GORIO_EUNSUPPORTED).
 *   queries, ids, dists: device pointers, as for gorio_search (host pointers
 *            -> GORIO_EINVAL).  k, L, W and nq: as for gorio_search.
 *   stats:   NULL, or filled with kernel_ms, evaluations, reevaluations,
 *            expansions and iterations (the call then waits for the search).
 *   stream:  hipStream_t (NULL = the null stream).
 * Under graph capture on `stream` the call records and waits for no event
 * (the caller orders the graph's replays with other work on the index) and
 * takes no statistics (stats != NULL -> GORIO_EINVAL); every replay clears
 * the scratch and runs the whole search again.
 * Scratch: the search's counters live in a fixed 128-byte device array of
 * the library, one per GPU, kept until the process ends; no batch size needs
 * more.  Each call clears it first.  Calls that overlap on one GPU (different
 * indexes, streams or threads) share that array and race; serialise them.
 * Results are the same as gorio_search's.
 */
gorio_status gorio_search_noalloc(gorio_index *ix, const void *queries, uint64_t nq,
                                  uint32_t k, uint32_t L, uint32_t W,
                                  uint32_t *ids, void *dists, gorio_stats *stats, void *stream);

/* Facts about the index (entry node, page counts, mode). */
gorio_status gorio_index_info_get(const gorio_index *ix, gorio_index_info *info);

/*
 * Copy `count` packed pages starting at page `first` to host memory `dst`
 * (count * page_bytes bytes), from HBM or the backing store.
 */
gorio_status gorio_copy_pages(const gorio_index *ix, uint64_t first, uint64_t count, void *dst);

/*
 * Locality-aware node placement (host only; no device is touched): fills
 * node_to_slot (n entries, a permutation of [0, n)) so that graph neighbours
 * share pages, for use as gorio_page_layout.node_to_slot.  Graph pages are the
 * unit of I/O (Sec. 3.1); the disk-resident ANNS work the paper builds on
 * places neighbours together for this reason (Sec. 6).  Rule: visit nodes
 * breadth-first from `entry`, neighbours in adjacency order; a visited node
 * without a slot takes the next slot and then fills the rest of its page
 * (records_per_page slots) with its own slot-less neighbours, in adjacency
 * order; unreached nodes follow in id order.  Deterministic.
 *   graph: host, n x R row-major; UINT32_MAX = no edge; other ids must be < n.
 * Errors: GORIO_EINVAL for NULL pointers, n, R or records_per_page out of range,
 * entry >= n or a bad id.
 */
gorio_status gorio_locality_order(const uint32_t *graph, uint64_t n, uint32_t R, uint32_t entry,
                                  uint32_t records_per_page, uint32_t *node_to_slot);

/*
 * Cluster placement (host call; runs on the current HIP device): k-means on
 * the vectors, then node_to_slot places the nodes cluster by cluster (id order
 * inside a cluster), for use as gorio_page_layout.node_to_slot.  Graph pages
 * are the unit of I/O (Sec. 3.1) and page layout and graph locality decide how
 * much of a fetched page a search uses (Sec. 6, DiskANN and Starling); a paged
 * cache holds a few clusters' pages at once, so placing nodes by cluster and
 * admitting queries by cluster (gorio_set_query_order) lets queries in flight
 * reuse each other's pages.
 *   vectors:    host, n x D row-major, uint8 or float32 per dtype.
 *   clusters:   K centroids, 1 <= K <= min(n, 65536).  Initial centroids are the
 *               vectors of nodes floor(i n / K); then `iterations` (<= 64) Lloyd
 *               steps (nearest centroid by squared L2 in float32 on the GPU, ties to
 *               the smaller index; each centroid becomes the mean of its members,
 *               an empty one stays).
 *   node_to_slot: host out, n entries, a permutation of [0, n).
 *   centroids:  host out, K x D float32 (the final centroids).
 * Deterministic.  Results of a search never depend on the placement.
 * Errors: GORIO_EINVAL for NULL pointers or n, D (1..1024), K, iterations out of
 * range; GORIO_ENOMEM / GORIO_EDEVICE from the device.
 */
gorio_status gorio_cluster_order(gorio_dtype dtype, const void *vectors, uint64_t n, uint32_t D,
                                 uint32_t clusters, uint32_t iterations, uint32_t *node_to_slot,
                                 float *centroids);

/*
 * Admission order of paged searches (the persistent scheduler of Sec. 3.3
 * decides which query a free slot takes next): with K > 0 centroids each paged
 * search first assigns every query to its nearest centroid (squared L2 in
 * float32, ties to the smaller index) and admits the queries cluster by
 * cluster, in index order inside a cluster, so the queries in flight share
 * pages (the cross-query reuse that Sec. 7.2 names as miss coalescing).  Each
 * query's answer is unchanged and is written to its own row.  Resident
 * searches ignore the order.
 *   centroids: host, K x D float32 (e.g. from gorio_cluster_order); copied.
 *   clusters:  K, 0 <= K <= 65536; 0 restores index order.
 * Errors: GORIO_EINVAL for a NULL index, K > 65536, or NULL centroids with K > 0.
 */
gorio_status gorio_set_query_order(gorio_index *ix, const float *centroids, uint32_t clusters);

/*
 * Release everything the index owns: its HBM pages or cache, the ready-table
 * words and rings of Sec. 3.2, the pinned backing store and the proxy thread
 * of Sec. 3.3 / Sec. 4 ("CPU transport proxy"), which is stopped first.  Must
 * not overlap a search on the index.  NULL is a no-op.
 */
void gorio_free_index(gorio_index *ix);

/*
 * Message for the last failing call on this thread ("" if none).  Errors are
 * returned as status codes so that no failure of the transport path (Sec. 4)
 * or of a search crosses the ABI as an exception; the text says which check
 * or which HIP call failed.  The pointer stays valid until the next failing
 * call on the same thread.
 */
const char *gorio_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GORIO_H */
