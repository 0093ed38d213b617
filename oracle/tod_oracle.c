/*
 * Oracle for the kNN / LOF outlier-detection hot path (TOD, arXiv 2110.14007).
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, the smoke check and the CPU-baseline
 * leg of the benchmark may load this library.  The product path (libtod.so)
 * never calls, links or includes anything from here, and this file shares no
 * code, header or table with it.
 *
 * What it computes, and from which passage of the paper:
 *
 *   kNN  The paper's kNN functional operator is cdist followed by topk
 *        (Section 4.2; Section 6.1 "Simple concatenation").  The pairwise
 *        quantity is the squared Euclidean distance of Eq. (dist-decomp).
 *        The oracle evaluates it in the *direct-difference* form
 *            D2(i,j) = sum_t (x_it - y_jt)^2
 *        in fp64 (every fp32 input is exactly representable in fp64), summed
 *        sequentially over t, then keeps the k smallest under the
 *        lexicographic key (D2, j): ties go to the lower reference index.
 *        Reported distances are sqrt(D2) (Euclidean, not squared).
 *
 *   kNN score  The kNN detector of Table 1 (kNNOD) scores a point by the
 *        distance to its k-th nearest neighbour (higher = more outlying,
 *        Section 3.1's output convention).
 *
 *   LOF  Table 1 lists LOF (Breunig et al. 2000), which the paper cites but
 *        does not define.  The oracle takes the standard definition with
 *        exactly k neighbours per point:
 *            kdist(o)    = distance from o to its k-th neighbour
 *            reach(p,o)  = max(kdist(o), D(p,o))          for o in N_k(p)
 *            lrd(p)      = 1 / (mean_{o in N_k(p)} reach(p,o) + 1e-10)
 *            LOF(p)      = mean_{o in N_k(p)} lrd(o) / lrd(p)
 *        The 1e-10 guard keeps duplicate points finite; it is this project's
 *        stated convention.
 *
 * Everything is plain loops in fp64; the only concession to speed is a
 * bounded insertion list per query row (so memory stays O(k)) and threading
 * over independent query rows.  Build with -ffp-contract=off so that no
 * multiply-add is fused: every operation above is a separately rounded IEEE
 * fp64 operation.
 */
#include <math.h>
#include <pthread.h>
#include <sched.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL 1
#define ORACLE_ENOMEM 2

/* -------------------------------------------------------------------------- */
/* Threading helper: split [0, count) across workers.                          */
/* -------------------------------------------------------------------------- */

typedef void (*range_fn)(void* ctx, int64_t begin, int64_t end);

typedef struct {
  range_fn fn;
  void* ctx;
  int64_t begin, end;
} worker_arg;

static void* worker_main(void* p) {
  worker_arg* w = (worker_arg*)p;
  w->fn(w->ctx, w->begin, w->end);
  return NULL;
}

int oracle_default_threads(void) {
  cpu_set_t set;
  if (sched_getaffinity(0, sizeof(set), &set) == 0) {
    int c = CPU_COUNT(&set);
    if (c > 0) return c;
  }
  long c = sysconf(_SC_NPROCESSORS_ONLN);
  return c > 0 ? (int)c : 1;
}

static void parallel_for(int64_t count, int nthreads, range_fn fn, void* ctx) {
  if (nthreads <= 0) nthreads = oracle_default_threads();
  if (nthreads > count) nthreads = (int)(count > 0 ? count : 1);
  if (nthreads <= 1) {
    fn(ctx, 0, count);
    return;
  }
  pthread_t* tid = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nthreads);
  worker_arg* args = (worker_arg*)malloc(sizeof(worker_arg) * (size_t)nthreads);
  int started = 0;
  for (int t = 0; t < nthreads; ++t) {
    args[t].fn = fn;
    args[t].ctx = ctx;
    args[t].begin = count * t / nthreads;
    args[t].end = count * (t + 1) / nthreads;
    if (pthread_create(&tid[t], NULL, worker_main, &args[t]) == 0) {
      started = t + 1;
    } else {
      /* Could not start a thread: do this share inline. */
      fn(ctx, args[t].begin, args[t].end);
      tid[t] = 0;
    }
  }
  for (int t = 0; t < started; ++t)
    if (tid[t]) pthread_join(tid[t], NULL);
  free(tid);
  free(args);
}

/* -------------------------------------------------------------------------- */
/* kNN by brute force.                                                         */
/* -------------------------------------------------------------------------- */

/* Squared Euclidean distance, direct-difference form, sequential fp64 sum. */
static double sq_dist(const float* a, const float* b, int64_t d) {
  double s = 0.0;
  for (int64_t t = 0; t < d; ++t) {
    double diff = (double)a[t] - (double)b[t];
    double sq = diff * diff;
    s = s + sq;
  }
  return s;
}

typedef struct {
  const float* xq;
  const float* xr;
  int64_t nr, d;
  int32_t k, exclude_self;
  const int64_t* rows; /* query row ids, or NULL for 0..count-1 */
  int64_t* idx_out;    /* count x k */
  double* dist_out;    /* count x k (Euclidean) */
} knn_ctx;

/*
 * Keep the k smallest (D2, j) seen so far in ascending order.  References
 * are visited in increasing j, so a newcomer with the same D2 as a kept
 * entry always has the larger index and belongs after it: the insertion
 * point is the first kept entry whose D2 is strictly larger.
 */
static void knn_rows(void* p, int64_t begin, int64_t end) {
  knn_ctx* c = (knn_ctx*)p;
  const int32_t k = c->k;
  double* best_d2 = (double*)malloc(sizeof(double) * (size_t)k);
  int64_t* best_j = (int64_t*)malloc(sizeof(int64_t) * (size_t)k);
  for (int64_t r = begin; r < end; ++r) {
    const int64_t qi = c->rows ? c->rows[r] : r;
    const float* q = c->xq + qi * c->d;
    int32_t filled = 0;
    for (int32_t s = 0; s < k; ++s) {
      best_d2[s] = INFINITY;
      best_j[s] = -1;
    }
    for (int64_t j = 0; j < c->nr; ++j) {
      if (c->exclude_self && j == qi) continue;
      double d2 = sq_dist(q, c->xr + j * c->d, c->d);
      if (filled == k && !(d2 < best_d2[k - 1])) continue;
      int32_t pos = filled < k ? filled : k - 1;
      while (pos > 0 && best_d2[pos - 1] > d2) {
        best_d2[pos] = best_d2[pos - 1];
        best_j[pos] = best_j[pos - 1];
        --pos;
      }
      best_d2[pos] = d2;
      best_j[pos] = j;
      if (filled < k) ++filled;
    }
    for (int32_t s = 0; s < k; ++s) {
      c->idx_out[r * k + s] = best_j[s];
      c->dist_out[r * k + s] = sqrt(best_d2[s]);
    }
  }
  free(best_d2);
  free(best_j);
}

/*
 * kNN of query rows against a reference set.
 *   xq[nq x d], xr[nr x d]  fp32, row-major (host memory)
 *   rows      optional list of nrows query ids; NULL means all nq rows
 *   exclude_self  skip reference j == query id (requires xq == xr)
 *   idx_out[nrows x k]  neighbour ids sorted by (D, j)
 *   dist_out[nrows x k] Euclidean distances (fp64)
 */
int oracle_knn(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d, int32_t k,
               int32_t exclude_self, const int64_t* rows, int64_t nrows, int32_t nthreads,
               int64_t* idx_out, double* dist_out) {
  if (!xq || !xr || !idx_out || !dist_out || nq <= 0 || nr <= 0 || d <= 0 || k <= 0)
    return ORACLE_EINVAL;
  if (k > nr - (exclude_self ? 1 : 0)) return ORACLE_EINVAL;
  int64_t count = rows ? nrows : nq;
  if (rows)
    for (int64_t r = 0; r < nrows; ++r)
      if (rows[r] < 0 || rows[r] >= nq) return ORACLE_EINVAL;
  knn_ctx c = {xq, xr, nr, d, k, exclude_self, rows, idx_out, dist_out};
  parallel_for(count, nthreads, knn_rows, &c);
  return ORACLE_OK;
}

/* -------------------------------------------------------------------------- */
/* LOF from complete neighbour lists.                                          */
/* -------------------------------------------------------------------------- */

/*
 * Full-set LOF.  idx[n x k], dist[n x k] are every point's k nearest
 * neighbours (self excluded) in (D, j) order.  Outputs (each nullable):
 * kdist[n], lrd[n], lof[n].
 */
int oracle_lof(int64_t n, int32_t k, const int64_t* idx, const double* dist, double* kdist_out,
               double* lrd_out, double* lof_out) {
  if (n <= 0 || k <= 0 || !idx || !dist) return ORACLE_EINVAL;
  double* kdist = (double*)malloc(sizeof(double) * (size_t)n);
  double* lrd = (double*)malloc(sizeof(double) * (size_t)n);
  if (!kdist || !lrd) {
    free(kdist);
    free(lrd);
    return ORACLE_ENOMEM;
  }
  for (int64_t p = 0; p < n; ++p) kdist[p] = dist[p * k + (k - 1)];
  for (int64_t p = 0; p < n; ++p) {
    double sum = 0.0;
    for (int32_t s = 0; s < k; ++s) {
      int64_t o = idx[p * k + s];
      double dpo = dist[p * k + s];
      double reach = kdist[o] > dpo ? kdist[o] : dpo;
      sum = sum + reach;
    }
    lrd[p] = 1.0 / (sum / (double)k + 1e-10);
  }
  for (int64_t p = 0; p < n; ++p) {
    double sum = 0.0;
    for (int32_t s = 0; s < k; ++s) sum = sum + lrd[idx[p * k + s]];
    if (lof_out) lof_out[p] = (sum / (double)k) / lrd[p];
  }
  if (kdist_out) memcpy(kdist_out, kdist, sizeof(double) * (size_t)n);
  if (lrd_out) memcpy(lrd_out, lrd, sizeof(double) * (size_t)n);
  free(kdist);
  free(lrd);
  return ORACLE_OK;
}

/* -------------------------------------------------------------------------- */
/* LOF of a few rows of a large set.                                           */
/* -------------------------------------------------------------------------- */

/* Sorted, de-duplicated copy of v[0..m).  Returns the new length. */
static int cmp_i64(const void* a, const void* b) {
  int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
  return x < y ? -1 : (x > y ? 1 : 0);
}
static int64_t sort_unique(int64_t* v, int64_t m) {
  if (m == 0) return 0;
  qsort(v, (size_t)m, sizeof(int64_t), cmp_i64);
  int64_t w = 1;
  for (int64_t r = 1; r < m; ++r)
    if (v[r] != v[w - 1]) v[w++] = v[r];
  return w;
}

/*
 * LOF(p) for the listed rows p of X (self excluded), computed from first
 * principles without the full n x k lists: LOF(p) needs lrd of p and of each
 * o in N_k(p); lrd(o) needs kdist of each u in N_k(o).  So the kNN lists of
 * A = rows, B = N(A) and C = N(B) are computed (C only for its k-distance),
 * and the definitions above are applied to them.  Outputs per listed row:
 * lof_out[nrows], lrd_out[nrows] and kdist_out[nrows] (the latter two
 * nullable).
 */
int oracle_lof_rows(const float* x, int64_t n, int64_t d, int32_t k, const int64_t* rows,
                    int64_t nrows, int32_t nthreads, double* lof_out, double* lrd_out,
                    double* kdist_out) {
  if (!x || !rows || !lof_out || n <= 1 || d <= 0 || k <= 0 || k > n - 1 || k > 256 ||
      nrows <= 0)
    return ORACLE_EINVAL;
  int status = ORACLE_ENOMEM;
  /* Per-point tables over the whole set; NaN/-1 marks "not computed". */
  double* kdist = (double*)malloc(sizeof(double) * (size_t)n);
  double* lrd = (double*)malloc(sizeof(double) * (size_t)n);
  int64_t* where = (int64_t*)malloc(sizeof(int64_t) * (size_t)n); /* row in lists */
  int64_t* set = NULL;
  int64_t* lidx = NULL;
  double* ldist = NULL;
  if (!kdist || !lrd || !where) goto done;
  for (int64_t i = 0; i < n; ++i) {
    kdist[i] = NAN;
    lrd[i] = NAN;
    where[i] = -1;
  }

  /* Grow the set A, A+N(A), A+N(A)+N(N(A)) level by level. */
  int64_t cap = nrows;
  set = (int64_t*)malloc(sizeof(int64_t) * (size_t)cap);
  if (!set) goto done;
  memcpy(set, rows, sizeof(int64_t) * (size_t)nrows);
  int64_t m = sort_unique(set, nrows);
  for (int64_t r = 0; r < m; ++r)
    if (set[r] < 0 || set[r] >= n) {
      status = ORACLE_EINVAL;
      goto done;
    }
  int64_t have = 0; /* lists computed for set[0..have) */
  for (int level = 0; level < 3; ++level) {
    /* Lists for the members not yet listed. */
    int64_t todo = 0;
    for (int64_t r = 0; r < m; ++r)
      if (where[set[r]] < 0) ++todo;
    if (todo > 0) {
      int64_t* q = (int64_t*)malloc(sizeof(int64_t) * (size_t)todo);
      int64_t* nidx = (int64_t*)realloc(lidx, sizeof(int64_t) * (size_t)(have + todo) * (size_t)k);
      if (nidx) lidx = nidx;
      double* ndist = (double*)realloc(ldist, sizeof(double) * (size_t)(have + todo) * (size_t)k);
      if (ndist) ldist = ndist;
      if (!q || !nidx || !ndist) {
        free(q);
        goto done;
      }
      int64_t t = 0;
      for (int64_t r = 0; r < m; ++r)
        if (where[set[r]] < 0) q[t++] = set[r];
      int rc = oracle_knn(x, n, x, n, d, k, 1, q, todo, nthreads, lidx + have * k,
                          ldist + have * k);
      if (rc != ORACLE_OK) {
        free(q);
        status = rc;
        goto done;
      }
      for (int64_t r = 0; r < todo; ++r) {
        where[q[r]] = have + r;
        kdist[q[r]] = ldist[(have + r) * k + (k - 1)];
      }
      have += todo;
      free(q);
    }
    if (level == 2) break;
    /* Next level: add the neighbours of every listed member. */
    int64_t ncap = m + m * (int64_t)k;
    int64_t* nset = (int64_t*)malloc(sizeof(int64_t) * (size_t)ncap);
    if (!nset) goto done;
    memcpy(nset, set, sizeof(int64_t) * (size_t)m);
    int64_t w = m;
    for (int64_t r = 0; r < m; ++r) {
      int64_t at = where[set[r]];
      for (int32_t s = 0; s < k; ++s) nset[w++] = lidx[at * k + s];
    }
    free(set);
    set = nset;
    m = sort_unique(set, w);
  }

  /* lrd for A and N(A): every neighbour's kdist is known by construction. */
  for (int64_t r = 0; r < nrows; ++r) {
    int64_t p = rows[r];
    int64_t members[1 + 256];
    int32_t nm = 0;
    members[nm++] = p;
    for (int32_t s = 0; s < k; ++s) members[nm++] = lidx[where[p] * k + s];
    for (int32_t t = 0; t < nm; ++t) {
      int64_t o = members[t];
      if (!isnan(lrd[o])) continue;
      int64_t at = where[o];
      double sum = 0.0;
      for (int32_t s = 0; s < k; ++s) {
        int64_t u = lidx[at * k + s];
        double dou = ldist[at * k + s];
        double reach = kdist[u] > dou ? kdist[u] : dou;
        sum = sum + reach;
      }
      lrd[o] = 1.0 / (sum / (double)k + 1e-10);
    }
    double sum = 0.0;
    for (int32_t s = 0; s < k; ++s) sum = sum + lrd[lidx[where[p] * k + s]];
    lof_out[r] = (sum / (double)k) / lrd[p];
    if (lrd_out) lrd_out[r] = lrd[p];
    if (kdist_out) kdist_out[r] = kdist[p];
  }
  status = ORACLE_OK;
done:
  free(kdist);
  free(lrd);
  free(where);
  free(set);
  free(lidx);
  free(ldist);
  return status;
}

/* -------------------------------------------------------------------------- */
/* Neighbours within range.                                                    */
/* -------------------------------------------------------------------------- */

/*
 * NWR (Section 5.3): for a query row i, every reference row j whose distance
 * is at most the threshold phi.  phi is a radius; a pair is in range iff the
 * squared distance D2 (the same sequential fp64 direct-difference sum as the
 * kNN above) satisfies D2 <= phi * phi, both sides in fp64.  References are
 * listed in increasing j.
 */
typedef struct {
  const float* xq;
  const float* xr;
  int64_t nr, d;
  double phi2;
  int32_t exclude_self;
  const int64_t* rows;
  int64_t* counts;       /* count pass: pairs per row */
  const int64_t* start;  /* fill pass: first output slot per row, or NULL */
  int64_t* idx_out;
  double* dist_out;
} nwr_ctx;

static void nwr_rows(void* p, int64_t begin, int64_t end) {
  nwr_ctx* c = (nwr_ctx*)p;
  for (int64_t r = begin; r < end; ++r) {
    const int64_t qi = c->rows ? c->rows[r] : r;
    const float* q = c->xq + qi * c->d;
    int64_t m = 0;
    for (int64_t j = 0; j < c->nr; ++j) {
      if (c->exclude_self && j == qi) continue;
      double d2 = sq_dist(q, c->xr + j * c->d, c->d);
      if (!(d2 <= c->phi2)) continue;
      if (c->start) {
        c->idx_out[c->start[r] + m] = j;
        c->dist_out[c->start[r] + m] = sqrt(d2);
      }
      ++m;
    }
    if (!c->start) c->counts[r] = m;
  }
}

/*
 * Count pass: counts_out[nrows] = pairs in range per query row.
 * Fill pass (start != NULL): row r's pairs go to idx_out / dist_out from
 * start[r] on (Euclidean distances, fp64).
 */
int oracle_nwr(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d, double phi,
               int32_t exclude_self, const int64_t* rows, int64_t nrows, int32_t nthreads,
               int64_t* counts_out, const int64_t* start, int64_t* idx_out, double* dist_out) {
  if (!xq || !xr || nq <= 0 || nr <= 0 || d <= 0 || !(phi >= 0.0)) return ORACLE_EINVAL;
  if (start ? (!idx_out || !dist_out) : !counts_out) return ORACLE_EINVAL;
  int64_t count = rows ? nrows : nq;
  if (rows)
    for (int64_t r = 0; r < nrows; ++r)
      if (rows[r] < 0 || rows[r] >= nq) return ORACLE_EINVAL;
  nwr_ctx c = {xq, xr, nr, d, phi * phi, exclude_self, rows, counts_out, start, idx_out, dist_out};
  parallel_for(count, nthreads, nwr_rows, &c);
  return ORACLE_OK;
}
