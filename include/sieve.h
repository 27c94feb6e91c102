/*
 * sieve.h -- C ABI of the MI355X (gfx950) threshold-aware IVF search library.
 *
 * The operation (SieveIVF, arXiv 2608.03199):
 *   Given an IVF index over a corpus X and a query batch Q, each query q ranks
 *   the IVF centroids by inner product (Sec. 2.3, Sec. 4.1) and probes the
 *   partitions in that order.  A probe is a hit when the partition holds a
 *   candidate x with <q, x> >= tau (the threshold candidate set R(q, tau),
 *   Sec. 2.2); the query stops after W consecutive threshold-empty probes or
 *   after nprobe_max probes (Sec. 3.5, Sec. 4.1, Algorithm 1).  The result is
 *   the top-k of all qualifying candidates met on the way (the final MergeTopK
 *   of Algorithm 1).  Lookahead (Sec. 4.3, Algorithm 2) dispatches, ahead of
 *   time, every probe that the stop rule has already committed; it changes no
 *   output (the equivalence argument of Sec. 4.3).  sieve_search_fixed is the
 *   fixed-probe IVF baseline (Sec. 2.3): every query probes min(nprobe, nlist)
 *   partitions.
 *
 * Conventions shared by every entry point:
 *   - Return value: SIEVE_OK (0) or a negative sieve_status.  On error no
 *     output buffer is written and sieve_last_error() describes the cause.
 *     Argument checks run before any HIP call.
 *   - Residency: every array argument is a DEVICE pointer on the current HIP
 *     device (for example torch.Tensor.data_ptr() of a CUDA tensor), laid out
 *     row-major and contiguous.  "stream" is a hipStream_t (NULL = the null
 *     stream); all work is ordered on it.
 *   - Similarity is the raw inner product of the stored values; the library
 *     never renormalises.  With unit-normalised data it is the cosine.
 *   - Centroid order: score descending, ties to the lower centroid index,
 *     decided in double precision (an fp32 screen whose near-ties are
 *     re-scored in fp64, so the order is that of exact-product fp64 sums).
 *   - Result order: score descending, ties to the lower id.  Fewer than k
 *     qualifying candidates are padded with id -1 and score -INFINITY.
 *   - Thread safety: one search at a time per index handle (the handle caches
 *     its device workspace).  Different handles are independent.
 */
#ifndef SIEVE_H
#define SIEVE_H

#include <stdint.h>

#if defined(__GNUC__)
#define SIEVE_API __attribute__((visibility("default")))
#else
#define SIEVE_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sieve_status {
  SIEVE_OK = 0,
  SIEVE_EINVAL = -1,       /* a null required pointer, an out-of-range size or flag, bad offsets */
  SIEVE_ENOMEM = -2,       /* device memory could not be allocated                               */
  SIEVE_EDEVICE = -3,      /* a HIP runtime call failed (the message names it)                   */
  SIEVE_EUNSUPPORTED = -4, /* valid, but outside this build's limits (see each function)         */
  SIEVE_EINTERNAL = -5     /* an internal consistency check failed                               */
} sieve_status;

typedef enum sieve_dtype {
  SIEVE_F32 = 0, /* IEEE binary32 storage, fp32 MFMA accumulate                 */
  SIEVE_F16 = 1  /* IEEE binary16 storage, exact products, fp32 MFMA accumulate */
} sieve_dtype;

/* Any W >= min(nprobe_max, nlist) disables early stopping; this value is the
 * conventional "infinite window". */
#define SIEVE_W_INF 0x7fffffff
/* Largest k accepted (the paper's k sweep reaches 50, Sec. 6.4). */
#define SIEVE_K_MAX 64

/* Values of the lookahead argument of sieve_search and sieve_search_multi.
 * They change only how the (query, partition) searches are grouped into
 * rounds; the outputs are identical for all four (Sec. 4.3).
 *   OFF          Algorithm 1: one rank per query per round (next / stale).
 *   COMMITTED    Algorithm 2: every rank up to the stop line is issued as soon
 *                as it is committed, and no rank past it is ever searched.
 *   SERIAL       the serial-traversal ablation of Sec. 6.3: Algorithm 1's
 *                rounds, and no partition scan is shared by two queries.
 *   SPECULATIVE  Algorithm 2 plus speculative issue, an addition of this
 *                library: when a stop line moves far, ranks past it are issued
 *                too (at most 3 W); the stop rule is then replayed over the
 *                recorded per-rank outcomes, and what ranks past the final line
 *                found is discarded.  It can search more (query, partition)
 *                pairs than Algorithm 2 (stats.items) and take fewer rounds.
 *                Batches of more than 2^20 queries issue committed ranks only. */
#define SIEVE_LOOKAHEAD_OFF 0
#define SIEVE_LOOKAHEAD_COMMITTED 1
#define SIEVE_LOOKAHEAD_SERIAL 2
#define SIEVE_LOOKAHEAD_SPECULATIVE 3

typedef struct sieve_index sieve_index; /* opaque, owned by the library */

/* Counters of one search call (filled when a non-NULL pointer is passed). */
typedef struct sieve_stats {
  int32_t rounds;           /* bulk-synchronous scheduling rounds                          */
  int32_t nprobe_eff;       /* min(nprobe_max, nlist)                                      */
  int32_t scan_launches;    /* partition-scan kernel launches                              */
  int32_t pool_retries;     /* re-runs after the candidate pool overflowed (results equal) */
  int64_t items;            /* (query, rank) searches executed; with speculative issue
                               this may exceed probes_total: ranks past a stop line can
                               be searched early, and what they find is discarded        */
  int64_t probes_total;     /* sum over queries of out_probes                              */
  int64_t vectors_scanned;  /* sum over items of the probed list's length                  */
  int64_t list_loads;       /* sum over rounds of distinct non-empty lists probed          */
  int64_t hits;             /* qualifying (query, row) pairs found (searched ranks past the
                               final stop line included)                                  */
  double scan_bytes;        /* algorithmic bytes of the scan: list rows + per-item query
                               rows and item records + candidate records written          */
  double scan_flops;        /* 2 * d * vectors_scanned                                     */
  double rank_flops;        /* 2 * d * nq * nlist (the centroid screen)                    */
  float ms_rank, ms_sched, ms_scan, ms_update, ms_finalize, ms_total; /* device time, ms */
  int64_t pool_entries;     /* candidate records written for the final merge: at most k per
                               (query, scan tile), at most hits                           */
  int64_t heavy_records;    /* groups of up to 16 (query, tile) pairs whose qualifying rows
                               outnumbered the scan's per-tile slots and went through the
                               exact top-k pass                                           */
} sieve_stats;

/*
 * sieve_load_index -- copy an IVF index (Sec. 2.3) into a library-owned
 * device layout.
 *   vectors      [n * d] of dtype, partition-major: the rows of list l are
 *                rows list_offsets[l] .. list_offsets[l+1]-1.
 *   dtype        SIEVE_F32 or SIEVE_F16 (queries and centroids share it).
 *   n            number of rows (>= 0); d: dimension, a multiple of 8 with
 *                8 <= d <= 4096 for fp16 and <= 2048 for fp32 (else
 *                SIEVE_EUNSUPPORTED).
 *   list_offsets [nlist + 1] int64: non-decreasing, list_offsets[0] == 0,
 *                list_offsets[nlist] == n (checked on a host copy; else
 *                SIEVE_EINVAL).  Empty lists are allowed.
 *   nlist        1 <= nlist <= 16384 (else SIEVE_EUNSUPPORTED).
 *   ids          [n] int64 row ids (the ids returned by searches; each id is
 *                expected once).
 *   centroids    [nlist * d] of dtype.
 *   out          receives the handle; the caller's buffers may be freed on
 *                return.  Free with sieve_free_index.
 * Device memory: the row-major copy of the vectors, and for the dimensions the
 * scan handles at compile time (fp16 64/128/768, fp32 64/128) a second copy in
 * MFMA fragment order (each list padded to whole 16-row blocks), about twice
 * the vectors' bytes in all; the centroids get a fragment-order copy too for
 * the ranking kernels' compile-time dimensions (fp16 128/768, fp32 64/128).
 * An allocation failure returns SIEVE_ENOMEM.
 * Synchronous: returns once the copies are complete.
 */
SIEVE_API int sieve_load_index(const void* vectors, int32_t dtype, int64_t n, int32_t d,
                               const int64_t* list_offsets, int32_t nlist, const int64_t* ids,
                               const void* centroids, void* stream, sieve_index** out);

/*
 * sieve_search -- threshold-aware search with the consecutive-empty stop rule
 * (Sec. 4.1), partition-major continuous batching (Sec. 4.2, Algorithm 1) and,
 * with lookahead, committed-prefix lookahead (Sec. 4.3, Algorithm 2).
 *   queries      [nq * d] of the index dtype; nq >= 0 (0 returns at once).
 *   exclude_ids  [nq] int64 or NULL: row id to skip for each query (a
 *                self-join passes each query's own id); the skipped row is
 *                neither a hit nor a result.
 *   k            1 <= k <= SIEVE_K_MAX.
 *   tau          similarity threshold, a candidate qualifies when its fp32
 *                score >= tau; NaN is SIEVE_EINVAL.
 *   W            consecutive-empty window, W >= 1 (SIEVE_W_INF: never stop).
 *   nprobe_max   >= 1; clamped to nlist; the clamped value must be <= 2048
 *                (else SIEVE_EUNSUPPORTED).
 *   lookahead    one of the SIEVE_LOOKAHEAD_* values above (else
 *                SIEVE_EINVAL); outputs are identical for all of them.
 *   out_ids      [nq * k] int64, out_scores [nq * k] float: per query the
 *                top-k qualifying candidates, score descending then id
 *                ascending, padded with (-1, -INFINITY).
 *   out_probes   [nq] int32: partitions searched, including the W trailing
 *                empty ones (min(L + W, n) with L the last hit rank).
 *   stats        NULL or a struct to fill.
 * Synchronous: returns once the outputs are complete on the stream.
 */
SIEVE_API int sieve_search(const sieve_index* idx, const void* queries, int64_t nq,
                           const int64_t* exclude_ids, int32_t k, float tau, int32_t W,
                           int32_t nprobe_max, int32_t lookahead, int64_t* out_ids,
                           float* out_scores, int32_t* out_probes, sieve_stats* stats,
                           void* stream);

/*
 * sieve_search_fixed -- fixed-probe IVF baseline (Sec. 2.3): every query
 * probes its first min(nprobe, nlist) ranked partitions and returns the top-k
 * of the qualifying candidates found there.  Arguments as for sieve_search;
 * out_probes[i] = min(nprobe, nlist).  Queries are processed in chunks so
 * that the materialised (query, rank) items fit the workspace.
 */
SIEVE_API int sieve_search_fixed(const sieve_index* idx, const void* queries, int64_t nq,
                                 const int64_t* exclude_ids, int32_t k, float tau, int32_t nprobe,
                                 int64_t* out_ids, float* out_scores, int32_t* out_probes,
                                 sieve_stats* stats, void* stream);

/*
 * sieve_search_calibrated -- threshold search whose window W is chosen inside
 * the call (Appendix A, Algorithm 3).  The sampled queries are searched with
 * full probing (nprobe = min(nprobe_max, nlist)) and keep that result; the
 * stop rule is replayed over their recorded per-partition outcomes: each
 * neighbour of a sampled fixed-probe result has a required window, the
 * smallest W whose stop-rule prefix reaches the partition where it was found,
 * and the chosen W is the smallest W < n whose sample-relative loss
 * 1 - (neighbours with required window <= W) / (all neighbours) is < eps,
 * else n (full probing).  Every other query is then searched with Algorithm 2
 * lookahead (SIEVE_LOOKAHEAD_COMMITTED) and the chosen W.  A sample without any neighbour (or ns = 0) uses
 * W_fallback.
 *   sample       [ns] int32 distinct query indices in [0, nq) (device); the
 *                caller draws them (uniformly without replacement in the
 *                paper).  ns <= 2^20.  Checked on a host copy (SIEVE_EINVAL).
 *   eps          sample-relative loss target, 0 < eps <= 1 (e.g. 0.005).
 *   W_fallback   >= 1, used when the sample has no neighbour.
 *   out_W        HOST pointer: receives the window used for the rest.
 * Other arguments and outputs as for sieve_search (out_probes of a sampled
 * query is min(nprobe_max, nlist)).  stats (if given) are the sums over the
 * two searches, the fixed-probe sample and the lookahead rest (nprobe_eff:
 * min(nprobe_max, nlist)).  Calls that overlap on one index race, as for
 * every search.
 */
SIEVE_API int sieve_search_calibrated(const sieve_index* idx, const void* queries, int64_t nq,
                                      const int64_t* exclude_ids, int32_t k, float tau,
                                      int32_t nprobe_max, const int32_t* sample, int64_t ns,
                                      float eps, int32_t W_fallback, int64_t* out_ids,
                                      float* out_scores, int32_t* out_probes, int32_t* out_W,
                                      sieve_stats* stats, void* stream);

/*
 * sieve_search_multi -- threshold search over several independently built
 * indexes of one corpus (the coarse shards of the paper's 100M layout,
 * Sec. 6.1): each index runs sieve_search with its own stop rule, and the
 * per-query results are merged into one top-k in the result order (score
 * descending, id ascending).
 *   idxs         HOST array of nidx (1 .. SIEVE_MULTI_MAX) handles on one
 *                device, with the same dtype and d; row ids must be unique
 *                across the indexes (the merge does not deduplicate).
 *   out_probes   [nq] the sum over the indexes of the partitions searched.
 * Other arguments as for sieve_search (exclude_ids apply to every index).
 * Workspace for the per-index results lives in idxs[0].  stats (if given)
 * are sums over the indexes.
 */
#define SIEVE_MULTI_MAX 256
SIEVE_API int sieve_search_multi(const sieve_index* const* idxs, int32_t nidx,
                                 const void* queries, int64_t nq, const int64_t* exclude_ids,
                                 int32_t k, float tau, int32_t W, int32_t nprobe_max,
                                 int32_t lookahead, int64_t* out_ids, float* out_scores,
                                 int32_t* out_probes, sieve_stats* stats, void* stream);

/*
 * sieve_search_multi_calibrated -- sieve_search_multi with the in-call window
 * calibration of Appendix A done per index: every index runs
 * sieve_search_calibrated on the same sampled query indices (its own sample
 * outcomes choose its own W, its sampled queries keep its fixed-probe
 * result, the rest use its W with Algorithm 2 lookahead), and the per-query
 * results are merged as in sieve_search_multi.
 *   out_W        HOST array of nidx: the window each index used.
 * Other arguments as for sieve_search_calibrated and sieve_search_multi.
 */
SIEVE_API int sieve_search_multi_calibrated(const sieve_index* const* idxs, int32_t nidx,
                                            const void* queries, int64_t nq,
                                            const int64_t* exclude_ids, int32_t k, float tau,
                                            int32_t nprobe_max, const int32_t* sample, int64_t ns,
                                            float eps, int32_t W_fallback, int64_t* out_ids,
                                            float* out_scores, int32_t* out_probes,
                                            int32_t* out_W, sieve_stats* stats, void* stream);

/*
 * sieve_rank -- the probe order alone (Sec. 4.1): for each query, the first
 * min(nprobe, nlist) centroid indices by inner product, descending, ties to
 * the lower index, decided in fp64 (see the conventions above).
 *   out_order    [nq * min(nprobe, nlist)] int32, row-major.
 * Other arguments and limits as for sieve_search.
 */
SIEVE_API int sieve_rank(const sieve_index* idx, const void* queries, int64_t nq, int32_t nprobe,
                         int32_t* out_order, void* stream);

/*
 * sieve_rank_noalloc -- sieve_rank for callers that cannot allocate memory
 * (code under stream capture, serving loops, harnesses that forbid device
 * allocation): the same outputs, bit for bit, with no device or host
 * allocation in the call.  Its workspace is a fixed 64 MiB device array of
 * the library, one per GPU, kept until the process ends; queries are ranked
 * in chunks that fit it.  Calls on one GPU share that array: calls that
 * overlap in time on one GPU (on other streams or threads) race on it and
 * must be serialised by the caller.  The call synchronises its stream once
 * per attempt (as sieve_rank does) to read the tie-overflow flag.
 *   Returns SIEVE_EUNSUPPORTED when one query's workspace (nlist * 4 bytes
 *   on the screen path, about (min(nprobe, nlist) + 128) * 8 bytes on the
 *   prefix path) does not fit the array, or on devices above 63; other
 *   arguments, limits and errors as for sieve_rank.
 */
SIEVE_API int sieve_rank_noalloc(const sieve_index* idx, const void* queries, int64_t nq,
                                 int32_t nprobe, int32_t* out_order, void* stream);

/*
 * sieve_round_log -- per-round record of the last search call on this handle
 * that was given a stats pointer (for fixed probing, one record per query
 * chunk).  Diagnostics for the roofline of the partition scan: each record
 * holds the round's algorithmic scan work and the scan launch's device time.
 *   out          HOST array of max records (may be NULL when max = 0).
 *   n_rounds     HOST pointer: receives the number of rounds of that search
 *                (records past max, or past the 256 kept, are not written).
 * Returns SIEVE_EINVAL for a NULL handle or n_rounds, or max < 0.
 */
typedef struct sieve_round {
  int64_t items;       /* (query, rank) searches dispatched in the round                */
  int64_t list_rows;   /* rows of the distinct non-empty lists touched (read once each) */
  int64_t item_rows;   /* sum over the items of their list's rows (rows scored)         */
  int64_t list_loads;  /* distinct non-empty lists touched                              */
  int64_t candidates;  /* candidate records the scan wrote                              */
  double scan_bytes;   /* list rows + per-item query rows and records + candidates, B   */
  double scan_flops;   /* 2 * d * item_rows                                             */
  float ms_scan;       /* device time of the round's scan launch (HIP events)           */
  int32_t kind;        /* 0: threshold-search round, 1: fixed-probe chunk               */
} sieve_round;
SIEVE_API int sieve_round_log(const sieve_index* idx, sieve_round* out, int32_t max,
                              int32_t* n_rounds);

/* Release an index and its cached workspace.  NULL is a no-op. */
SIEVE_API void sieve_free_index(sieve_index* idx);

/* Message of the last failed call on this thread ("" if none).  Valid until
 * the next call on the same thread. */
SIEVE_API const char* sieve_last_error(void);

/* Library version string. */
SIEVE_API const char* sieve_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SIEVE_H */
