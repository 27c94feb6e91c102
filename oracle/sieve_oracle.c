/*
 * sieve_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, sequential, obviously-correct CPU oracle for threshold-aware IVF
 * search (SieveIVF).  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg load this code; the GPU library never links, includes or
 * calls it, and it shares no header, helper, table or constant with it.
 *
 * Every score is a double-precision dot product summed over the dimension
 * index in ascending order; fp16 inputs are widened to double exactly by a
 * decoder written from the IEEE 754 binary16 definition.  There is no
 * blocking, no SIMD intrinsic and no reordering beyond what the paper's
 * definitions state.  Threads (if asked for) only split the query batch into
 * disjoint contiguous blocks; each thread runs the same per-query code.
 *
 * What each routine follows:
 *   - R(q, tau) = { x : sim(q, x) >= tau }, inclusive            (Sec. 2.2)
 *   - partitions are probed in centroid-ranked order P_i         (Sec. 4.1)
 *   - a probe is "empty" when no candidate reaches tau; a hit
 *     resets the consecutive-empty counter, W empties stop      (Sec. 3.5, 4.1, Table 2)
 *   - mode A: the stop rule walked sequentially, one probe
 *     at a time (Algorithm 1's per-query rule)                  (Sec. 3.5, 4.1, 4.2)
 *   - mode B: lookahead over the committed prefix (stop line),
 *     newest committed rank searched first on purpose            (Sec. 4.3, Algorithm 2)
 *   - flags: queries whose result may legitimately differ in a
 *     lower-precision implementation (a score within 1e-4 of tau,
 *     of the k-th/(k+1)-th boundary, or of a returned neighbour)
 *   - final MergeTopK over all accumulated local results        (Algorithm 1, final merge)
 *   - fixed probing = the same traversal with no stop rule      (Sec. 2.3)
 *   - exhaustive filtered top-k over the whole corpus           (Sec. 6.1 ground truth)
 *   - in-call W calibration by replay of recorded outcomes     (Appendix A, Algorithm 3)
 *
 * Readings where the paper is silent (each one is also listed in the design notes):
 *   - similarity is the raw inner product of the stored vectors (the data are
 *     unit-normalised, so this is the cosine of Sec. 6.1);
 *   - centroid order: score descending, ties to the lower centroid index;
 *   - result order: score descending, ties to the lower id;
 *   - fewer than k qualifying candidates: pad with id -1, score -inf;
 *   - a query's own row (by id, exclude_ids) is neither a hit nor a result;
 *   - a list with no rows is a threshold-empty probe;
 *   - nprobe_max above nlist is clamped to nlist (|P_i| in Algorithm 1);
 *   - W >= n never stops early (W = 0x7fffffff encodes "infinity").
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_F32 0
#define OR_F16 1

#define OR_FLAG_TAU_EDGE 1      /* some scanned score lies within 1e-4 of tau      */
#define OR_FLAG_KTH_TIE 2       /* the k-th and (k+1)-th candidates within 1e-4    */
#define OR_FLAG_ORDER_TIE 4     /* two adjacent returned scores within 1e-4        */
#define OR_FLAG_CENTROID_TIE 8  /* two adjacent ranked centroid scores within 1e-12 */

#define OR_EDGE_BAND 1e-4
#define OR_CENTROID_BAND 1e-12

#define OR_MODE_A 0  /* sequential walk of the stop rule (Algorithm 1)   */
#define OR_MODE_B 1  /* committed prefix under a stop line (Algorithm 2) */

/* ---------------------------------------------------------------------- */
/* IEEE 754 binary16 -> double, from the format definition:               */
/*   sign(1) exponent(5, bias 15) fraction(10);                           */
/*   exponent 0: subnormal, value = fraction * 2^-24;                     */
/*   exponent 31: infinity (fraction 0) or NaN.                           */
/* ---------------------------------------------------------------------- */
double oracle_half_to_double(uint16_t h) {
  int sign = (h >> 15) & 1;
  int expo = (h >> 10) & 31;
  int frac = h & 1023;
  double v;
  if (expo == 0) {
    v = ldexp((double)frac, -24);
  } else if (expo == 31) {
    v = frac ? NAN : INFINITY;
  } else {
    v = ldexp((double)(1024 + frac), expo - 25);
  }
  return sign ? -v : v;
}

static double elem(const void* base, int dtype, int64_t i) {
  if (dtype == OR_F32) return (double)((const float*)base)[i];
  return oracle_half_to_double(((const uint16_t*)base)[i]);
}

/* <q, row r of base>, q already widened to double; sum in dimension order. */
static double dot_row(const double* q, const void* base, int dtype, int64_t r, int d) {
  double s = 0.0;
  for (int t = 0; t < d; ++t) s += q[t] * elem(base, dtype, r * (int64_t)d + t);
  return s;
}

typedef struct {
  const void* vectors;
  int dtype;
  int64_t n;
  int d;
  const int64_t* list_offsets;
  int nlist;
  const int64_t* ids;
  const void* centroids;
} or_index;

/* ---------------------------------------------------------------------- */
/* Centroid ranking (Sec. 4.1): order all centroids by (score desc, index */
/* asc) and keep the first n.  The comparator is a total order, so the    */
/* library sort's result is unique.                                       */
/* ---------------------------------------------------------------------- */
typedef struct {
  double s;
  int c;
} cscore_t;

static int centroid_cmp(const void* pa, const void* pb) {
  const cscore_t* a = (const cscore_t*)pa;
  const cscore_t* b = (const cscore_t*)pb;
  if (a->s > b->s) return -1;
  if (a->s < b->s) return 1;
  return (a->c > b->c) - (a->c < b->c);
}

static void rank_centroids(const or_index* ix, const double* q, int n, int* order, double* cscore,
                           cscore_t* work) {
  for (int c = 0; c < ix->nlist; ++c) {
    work[c].s = dot_row(q, ix->centroids, ix->dtype, c, ix->d);
    work[c].c = c;
  }
  qsort(work, (size_t)ix->nlist, sizeof(cscore_t), centroid_cmp);
  for (int j = 0; j < n; ++j) {
    order[j] = work[j].c;
    cscore[j] = work[j].s;
  }
}

/* ---------------------------------------------------------------------- */
/* Candidate list (the query's accumulated local results).                */
/* ---------------------------------------------------------------------- */
typedef struct {
  double s;
  int64_t id;
  int rank; /* 1-based probe rank of the list the candidate was found in */
} cand;

typedef struct {
  cand* v;
  int64_t len, cap;
} cand_vec;

static int cv_push(cand_vec* cv, double s, int64_t id, int rank) {
  if (cv->len == cv->cap) {
    int64_t nc = cv->cap ? 2 * cv->cap : 64;
    cand* nv = (cand*)realloc(cv->v, (size_t)nc * sizeof(cand));
    if (!nv) return -1;
    cv->v = nv;
    cv->cap = nc;
  }
  cv->v[cv->len].s = s;
  cv->v[cv->len].id = id;
  cv->v[cv->len].rank = rank;
  cv->len++;
  return 0;
}

/* total order of results: score descending, then id ascending */
static int cand_cmp(const void* pa, const void* pb) {
  const cand* a = (const cand*)pa;
  const cand* b = (const cand*)pb;
  if (a->s > b->s) return -1;
  if (a->s < b->s) return 1;
  if (a->id < b->id) return -1;
  if (a->id > b->id) return 1;
  return 0;
}

/* Local search of one partition for one query (Sec. 5: the local output is */
/* filtered by tau; the probe is a hit iff that output is non-empty).      */
static int search_list(const or_index* ix, const double* q, int list, int rank, int64_t excl,
                       int has_excl, double tau, cand_vec* out, int* flags, int64_t* scanned) {
  int hit = 0;
  for (int64_t r = ix->list_offsets[list]; r < ix->list_offsets[list + 1]; ++r) {
    if (has_excl && ix->ids[r] == excl) continue;
    double v = dot_row(q, ix->vectors, ix->dtype, r, ix->d);
    (*scanned)++;
    /* a score this close to tau may be decided either way in lower precision */
    if (fabs(v - tau) < OR_EDGE_BAND) *flags |= OR_FLAG_TAU_EDGE;
    if (v >= tau) {
      hit = 1;
      if (cv_push(out, v, ix->ids[r], rank)) return -1;
    }
  }
  return hit;
}

typedef struct {
  /* inputs */
  const or_index* ix;
  const void* queries;
  const int64_t* exclude_ids;
  int k;
  double tau;
  int W;
  int n;  /* effective nprobe = min(nprobe_max, nlist) */
  int mode;
  /* outputs */
  int64_t* out_ids;
  double* out_scores;
  int32_t* out_probes;
  int32_t* out_flags;
  int32_t* out_last_hit;
  uint8_t* out_hitseq; /* [nq*n] 1 hit, 0 empty, 2 not visited; or NULL */
  int32_t* out_order;  /* [nq*n] ranked list ids; or NULL */
  int64_t* out_scanned; /* [nq] vectors scored; or NULL */
  int64_t* out_ncand;   /* [nq] qualifying candidates found; or NULL */
  int32_t* out_rank;    /* [nq*k] probe rank each returned result was found at (0 pad); or NULL */
  /* work range */
  int64_t q0, q1;
  int status;
} or_job;

/* One query, start to finish. */
static int one_query(const or_job* jb, int64_t qi, double* qd, int* order, double* cscore,
                     cscore_t* work, int* stack, uint8_t* hit_at, cand_vec* cv) {
  const or_index* ix = jb->ix;
  const int n = jb->n, d = ix->d, W = jb->W;
  int flags = 0;
  int64_t scanned = 0;
  for (int t = 0; t < d; ++t) qd[t] = elem(jb->queries, ix->dtype, qi * (int64_t)d + t);
  int has_excl = jb->exclude_ids != NULL;
  int64_t excl = has_excl ? jb->exclude_ids[qi] : 0;

  rank_centroids(ix, qd, n, order, cscore, work);
  for (int j = 0; j + 1 < n; ++j)
    if (cscore[j] - cscore[j + 1] < OR_CENTROID_BAND) flags |= OR_FLAG_CENTROID_TIE;

  for (int j = 0; j < n; ++j) hit_at[j] = 2;
  cv->len = 0;
  int probes = 0, last_hit = 0;

  if (jb->mode == OR_MODE_A) {
    /* The stop rule as a sequential walk (Sec. 3.5, Sec. 4.1): ranks are
     * probed one at a time in order; a hit clears the run of consecutive
     * empty probes, an empty probe lengthens it, and the query is done when
     * the run reaches W or all n ranks are probed.  Algorithm 1 applies the
     * same rule per query, one completed probe at a time. */
    int run = 0;
    for (int j = 1; j <= n; ++j) {
      int h = search_list(ix, qd, order[j - 1], j, excl, has_excl, jb->tau, cv, &flags, &scanned);
      if (h < 0) return -1;
      hit_at[j - 1] = (uint8_t)h;
      probes = j;
      if (h) {
        run = 0;
        last_hit = j;
      } else if (++run >= W) {
        break;
      }
    }
  } else {
    /* Lookahead (Sec. 4.3, Algorithm 2): the ranks up to the stop line s are
     * committed; s starts at min(W, n), and a hit found at rank j commits
     * every rank up to min(j + W, n).  Each committed rank is searched once.
     * Here the most recently committed rank is searched first, so outcomes
     * arrive out of rank order on purpose; the query is done when nothing
     * committed is left unsearched, and its probe count is s. */
    int s = W < n ? W : n;
    int committed = 0, top = 0; /* stack holds at most n ranks */
    for (;;) {
      while (committed < s) stack[top++] = ++committed;
      if (top == 0) break;
      int j = stack[--top];
      int h = search_list(ix, qd, order[j - 1], j, excl, has_excl, jb->tau, cv, &flags, &scanned);
      if (h < 0) return -1;
      hit_at[j - 1] = (uint8_t)h;
      if (h) {
        int line = (W > n - j) ? n : j + W; /* min(j + W, n) without overflow */
        if (line > s) s = line;
        if (j > last_hit) last_hit = j;
      }
    }
    probes = s;
  }

  /* MergeTopK over all accumulated local results (no call for an empty
   * vector: its storage may be NULL, which qsort must not be given). */
  if (cv->len > 1) qsort(cv->v, (size_t)cv->len, sizeof(cand), cand_cmp);
  int k = jb->k;
  /* the last returned slot may go either way: the best candidate left out
   * scores within the band of it */
  if (cv->len > k && cv->v[k - 1].s - cv->v[k].s < OR_EDGE_BAND) flags |= OR_FLAG_KTH_TIE;
  int kept = cv->len < k ? (int)cv->len : k;
  /* two returned neighbours whose relative order may go either way */
  for (int r = 0; r + 1 < kept; ++r)
    if (cv->v[r].s - cv->v[r + 1].s < OR_EDGE_BAND) flags |= OR_FLAG_ORDER_TIE;
  for (int r = 0; r < k; ++r) {
    jb->out_ids[qi * k + r] = r < kept ? cv->v[r].id : -1;
    jb->out_scores[qi * k + r] = r < kept ? cv->v[r].s : -INFINITY;
    if (jb->out_rank) jb->out_rank[qi * k + r] = r < kept ? cv->v[r].rank : 0;
  }
  jb->out_probes[qi] = probes;
  if (jb->out_flags) jb->out_flags[qi] = flags;
  if (jb->out_last_hit) jb->out_last_hit[qi] = last_hit;
  if (jb->out_hitseq) memcpy(jb->out_hitseq + qi * n, hit_at, (size_t)n);
  if (jb->out_order)
    for (int j = 0; j < n; ++j) jb->out_order[qi * n + j] = order[j];
  if (jb->out_scanned) jb->out_scanned[qi] = scanned;
  if (jb->out_ncand) jb->out_ncand[qi] = cv->len;
  return 0;
}

static void* run_job(void* arg) {
  or_job* jb = (or_job*)arg;
  const or_index* ix = jb->ix;
  double* qd = (double*)malloc(sizeof(double) * (size_t)ix->d);
  int* order = (int*)malloc(sizeof(int) * (size_t)ix->nlist);
  double* cscore = (double*)malloc(sizeof(double) * (size_t)ix->nlist);
  cscore_t* work = (cscore_t*)malloc(sizeof(cscore_t) * (size_t)ix->nlist);
  int* stack = (int*)malloc(sizeof(int) * (size_t)ix->nlist);
  uint8_t* hit_at = (uint8_t*)malloc((size_t)ix->nlist);
  cand_vec cv = {0, 0, 0};
  jb->status = 0;
  if (!qd || !order || !cscore || !work || !stack || !hit_at) jb->status = -2;
  for (int64_t qi = jb->q0; qi < jb->q1 && jb->status == 0; ++qi)
    if (one_query(jb, qi, qd, order, cscore, work, stack, hit_at, &cv)) jb->status = -2;
  free(qd);
  free(order);
  free(cscore);
  free(work);
  free(stack);
  free(hit_at);
  free(cv.v);
  return NULL;
}

static int check_index(const void* vectors, int dtype, int64_t n, int d, const int64_t* offs,
                       int nlist, const int64_t* ids, const void* cents) {
  if (!vectors && n > 0) return -1;
  if (!offs || !cents || (!ids && n > 0)) return -1;
  if (dtype != OR_F32 && dtype != OR_F16) return -1;
  if (d < 1 || nlist < 1 || n < 0) return -1;
  if (offs[0] != 0 || offs[nlist] != n) return -1;
  for (int c = 0; c < nlist; ++c)
    if (offs[c + 1] < offs[c]) return -1;
  return 0;
}

/*
 * oracle_search: per query, rank centroids, probe in order, scan each probed
 * list exhaustively in fp64 and apply the consecutive-empty stop rule.
 * W >= n (e.g. 0x7fffffff) gives fixed probing at n = min(nprobe_max, nlist).
 * Returns 0, -1 on invalid arguments, -2 on allocation failure.
 */
int oracle_search(const void* vectors, int dtype, int64_t n_vec, int d, const int64_t* list_offsets,
                  int nlist, const int64_t* ids, const void* centroids, const void* queries,
                  int64_t nq, const int64_t* exclude_ids, int k, float tau, int W, int nprobe_max,
                  int mode, int nthreads, int64_t* out_ids, double* out_scores, int32_t* out_probes,
                  int32_t* out_flags, int32_t* out_last_hit, uint8_t* out_hitseq,
                  int32_t* out_order, int64_t* out_scanned, int64_t* out_ncand,
                  int32_t* out_rank) {
  if (check_index(vectors, dtype, n_vec, d, list_offsets, nlist, ids, centroids)) return -1;
  if (nq < 0 || (nq > 0 && !queries) || k < 1 || W < 1 || nprobe_max < 1) return -1;
  if (mode != OR_MODE_A && mode != OR_MODE_B) return -1;
  if (isnan(tau)) return -1;
  if (nq > 0 && (!out_ids || !out_scores || !out_probes)) return -1;
  or_index ix = {vectors, dtype, n_vec, d, list_offsets, nlist, ids, centroids};
  int n = nprobe_max < nlist ? nprobe_max : nlist;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if ((int64_t)nthreads > nq) nthreads = nq > 0 ? (int)nq : 1;
  or_job jobs[256];
  pthread_t th[256];
  for (int t = 0; t < nthreads; ++t) {
    or_job jb = {&ix, queries, exclude_ids, k, (double)tau, W, n, mode, out_ids, out_scores,
                 out_probes, out_flags, out_last_hit, out_hitseq, out_order, out_scanned,
                 out_ncand, out_rank, nq * t / nthreads, nq * (t + 1) / nthreads, 0};
    jobs[t] = jb;
  }
  if (nthreads == 1) {
    run_job(&jobs[0]);
    return jobs[0].status;
  }
  for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, run_job, &jobs[t]);
  int st = 0;
  for (int t = 0; t < nthreads; ++t) {
    pthread_join(th[t], NULL);
    if (jobs[t].status) st = jobs[t].status;
  }
  return st;
}

/* ---------------------------------------------------------------------- */
/* Exhaustive filtered top-k over the whole corpus, in row order, with no */
/* IVF at all: the ground truth G_{tau,k}(q) of the pooled recall metric  */
/* (Sec. 6.1).                                                            */
/* ---------------------------------------------------------------------- */
typedef struct {
  const void* vectors;
  int dtype;
  int64_t n;
  int d;
  const int64_t* ids;
  const void* queries;
  const int64_t* exclude_ids;
  int k;
  double tau;
  int64_t* out_ids;
  double* out_scores;
  int64_t* out_count;
  int64_t q0, q1;
  int status;
} bf_job;

static void* run_bf(void* arg) {
  bf_job* jb = (bf_job*)arg;
  double* qd = (double*)malloc(sizeof(double) * (size_t)jb->d);
  cand_vec cv = {0, 0, 0};
  jb->status = qd ? 0 : -2;
  for (int64_t qi = jb->q0; qi < jb->q1 && jb->status == 0; ++qi) {
    for (int t = 0; t < jb->d; ++t) qd[t] = elem(jb->queries, jb->dtype, qi * (int64_t)jb->d + t);
    cv.len = 0;
    for (int64_t r = 0; r < jb->n; ++r) {
      if (jb->exclude_ids && jb->ids[r] == jb->exclude_ids[qi]) continue;
      double v = dot_row(qd, jb->vectors, jb->dtype, r, jb->d);
      if (v >= jb->tau && cv_push(&cv, v, jb->ids[r], 0)) {
        jb->status = -2;
        break;
      }
    }
    if (cv.len > 1) qsort(cv.v, (size_t)cv.len, sizeof(cand), cand_cmp);
    for (int r = 0; r < jb->k; ++r) {
      jb->out_ids[qi * jb->k + r] = r < cv.len ? cv.v[r].id : -1;
      jb->out_scores[qi * jb->k + r] = r < cv.len ? cv.v[r].s : -INFINITY;
    }
    if (jb->out_count) jb->out_count[qi] = cv.len;
  }
  free(qd);
  free(cv.v);
  return NULL;
}

int oracle_bruteforce(const void* vectors, int dtype, int64_t n_vec, int d, const int64_t* ids,
                      const void* queries, int64_t nq, const int64_t* exclude_ids, int k,
                      float tau, int nthreads, int64_t* out_ids, double* out_scores,
                      int64_t* out_count) {
  if ((n_vec > 0 && (!vectors || !ids)) || d < 1 || n_vec < 0) return -1;
  if (dtype != OR_F32 && dtype != OR_F16) return -1;
  if (nq < 0 || (nq > 0 && (!queries || !out_ids || !out_scores)) || k < 1 || isnan(tau)) return -1;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if ((int64_t)nthreads > nq) nthreads = nq > 0 ? (int)nq : 1;
  bf_job jobs[256];
  pthread_t th[256];
  for (int t = 0; t < nthreads; ++t) {
    bf_job jb = {vectors, dtype, n_vec, d, ids, queries, exclude_ids, k, (double)tau,
                 out_ids, out_scores, out_count, nq * t / nthreads, nq * (t + 1) / nthreads, 0};
    jobs[t] = jb;
  }
  if (nthreads == 1) {
    run_bf(&jobs[0]);
    return jobs[0].status;
  }
  for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, run_bf, &jobs[t]);
  int st = 0;
  for (int t = 0; t < nthreads; ++t) {
    pthread_join(th[t], NULL);
    if (jobs[t].status) st = jobs[t].status;
  }
  return st;
}

/* ---------------------------------------------------------------------- */
/* In-call window calibration (Appendix A, Algorithm 3), replay part.     */
/*                                                                        */
/* Input: for each sampled query, its fixed-probe result A_fixed(q) (the  */
/* ids of its top-k at full probing, -1 padded), the rank at which each   */
/* of those neighbours was found, and the full hit sequence h[1..n] of    */
/* its fixed-probe run.  For each neighbour the required window is the    */
/* smallest W whose stop-rule prefix reaches the rank where it was found; */
/* H[W] counts neighbours by required window; loss(W) = 1 - (prefix sum  */
/* of H up to W) / Z; the chosen window is the smallest W < n with       */
/* loss(W) < eps, else n (full probing).                                  */
/*                                                                        */
/* The prefix a window W reaches is computed by running the stop rule on  */
/* the recorded hit sequence, exactly as the sequential traversal would:  */
/* walk ranks 1.., reset on a hit, stop after W consecutive empties.      */
/* ---------------------------------------------------------------------- */
static int replay_reach(const uint8_t* h, int n, int W) {
  int stale = 0;
  for (int j = 1; j <= n; ++j) {
    if (h[j - 1] == 1)
      stale = 0;
    else
      stale++;
    if (stale >= W) return j;
  }
  return n;
}

/* out_hist has n+1 entries; entry W (1..n) counts neighbours whose required
 * window is exactly W.  Returns the chosen window, or -1 on bad arguments. */
int oracle_calibrate(int64_t ns, int n, int k, const uint8_t* hitseq, const int32_t* found_rank,
                     double eps, int64_t* out_hist, int64_t* out_z) {
  if (ns < 0 || n < 1 || k < 1 || (ns > 0 && (!hitseq || !found_rank)) || !out_hist) return -1;
  for (int w = 0; w <= n; ++w) out_hist[w] = 0;
  int64_t z = 0;
  for (int64_t q = 0; q < ns; ++q) {
    const uint8_t* h = hitseq + q * n;
    for (int r = 0; r < k; ++r) {
      int fr = found_rank[q * k + r];
      if (fr < 1) continue; /* padding */
      z++;
      int req = n;
      for (int w = 1; w <= n; ++w)
        if (replay_reach(h, n, w) >= fr) {
          req = w;
          break;
        }
      out_hist[req]++;
    }
  }
  if (out_z) *out_z = z;
  if (z == 0) return -2; /* no neighbour in the sample: caller applies its fallback */
  int64_t retained = 0;
  for (int w = 1; w <= n - 1; ++w) {
    retained += out_hist[w];
    double loss = 1.0 - (double)retained / (double)z;
    if (loss < eps) return w;
  }
  return n;
}
