/*
 * tod.h - C ABI of libtod, an MI355X (gfx950) implementation of the exact
 * kNN / LOF outlier-detection hot path of TOD (Zhao, Chen, Jia; arXiv
 * 2110.14007).
 *
 * The library computes, for query rows X_q and reference rows X_r:
 *   - the k nearest references of every query (the paper's kNN functional
 *     operator = cdist fused with topk, Sections 4.2 and 6.1), exact under
 *     the lexicographic key (distance, reference index), so ties go to the
 *     lower index;
 *   - the kNN-OD outlier score (distance to the k-th neighbour, Table 1);
 *   - the LOF outlier score (Table 1; Breunig et al. 2000, with exactly k
 *     neighbours and lrd = 1 / (mean reach-distance + 1e-10)), or, through
 *     tod_lof_ties, on Breunig's tie-inclusive k-distance neighbourhoods.
 *
 * It follows the paper's provable quantization (Section 5.2): inputs are
 * quantised (fp32 / fp16 / bf16 after centring and power-of-two scaling),
 * distances are evaluated in that precision to shortlist K' candidates per
 * query, a certificate checks that no excluded reference can reach the
 * exact k-th distance, and rows that fail it are recomputed exactly
 * (Section 5.2, step iii).  Distances are fused with selection so the n x n
 * matrix never exists (Section 6.1, operator fusion); queries stream through
 * in blocks and references in splits (Section 6, automatic batching).
 *
 * Conventions shared by every entry point:
 *   - Every data pointer is a DEVICE pointer (HIP), owned by the caller.
 *     Inputs are fp32, row-major, contiguous, 16-byte aligned.
 *   - The library allocates no device memory: the caller passes a workspace
 *     (256-byte aligned).  tod_workspace_size() bytes run the queries in as
 *     few blocks as the planner likes; a smaller workspace makes the kNN
 *     entry points plan smaller query blocks (tod_plan_workspace).
 *   - Distances are Euclidean (not squared).  Index outputs are 0-based rows
 *     of the reference set.  Output rows are sorted by (distance, index).
 *   - Arguments are validated on the host before any HIP call; on an
 *     argument error nothing is launched and outputs are untouched.
 *   - Calls are blocking: they return after the work queued on `stream`
 *     (a hipStream_t, or NULL for the default stream) has finished, so the
 *     returned status is final.  The library keeps no state between calls;
 *     calls on different streams with different workspaces may overlap.
 *   - On any error other than TOD_OK, output contents are unspecified.
 */
#ifndef TOD_H
#define TOD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TOD_OK = 0,
  TOD_ERR_INVALID_ARG = 1, /* null pointer, non-positive size, k out of range, bad struct_size */
  TOD_ERR_NONFINITE = 2,   /* NaN or Inf in the input (the rounding analysis needs finite data) */
  TOD_ERR_WORKSPACE = 3,   /* workspace misaligned, or too small for one 32-row query block */
  TOD_ERR_UNSUPPORTED = 4, /* k > 256, d > 4096, or more than 2^31 - 1 rows */
  TOD_ERR_HIP = 5,         /* a HIP launch or runtime call failed; see tod_last_error() */
  TOD_ERR_INTERNAL = 6,
  TOD_ERR_CAPACITY = 7     /* tod_nwr, tod_loci, tod_lof_ties: more pairs in range than the
                            * output capacity (tod_nwr still writes the row offsets and the
                            * total) */
} tod_status;

/* Precision of the shortlist filter (the exact recheck always works from the
 * original fp32 rows with fp64 accumulation). */
typedef enum {
  TOD_PREC_AUTO = 0,
  TOD_PREC_FP32 = 1, /* fp32 FMA distance tile: the reference filter (shortest shortlist,
                      * fewest fallbacks), not the fast path.  Its vector FMA work has a
                      * floor of 2d flop per pair at the non-packed fp32 rate, 8.1 ms at
                      * n = 100,000, d = 32 against the fp16 tile's 2.2 ms, and it runs at
                      * about 10x the fp16 tile's time. */
  TOD_PREC_FP16 = 2, /* fp16 MFMA distance tile, fp32 accumulate */
  TOD_PREC_BF16 = 3  /* bf16 MFMA distance tile, fp32 accumulate */
} tod_precision;

/* Outlier score from the k exact neighbour distances of a point (the kNN
 * detector of Table 1: the distance to the k-th neighbour, or an aggregate of
 * the k distances such as Angiulli and Pizzuti's weight, their sum). */
typedef enum {
  TOD_SCORE_KTH = 0,    /* distance to the k-th nearest neighbour (default) */
  TOD_SCORE_MEAN = 1,   /* mean of the k distances */
  TOD_SCORE_MEDIAN = 2, /* median of the k distances (mean of the two middle ones for even k) */
  TOD_SCORE_SUM = 3     /* sum of the k distances */
} tod_score;

typedef struct {
  uint32_t struct_size;  /* must be sizeof(tod_options) */
  int32_t precision;     /* tod_precision; AUTO picks by d */
  int32_t exclude_self;  /* tod_knn only: drop reference j == query i (requires xq == xr, nq == nr) */
  int32_t shortlist;     /* K' (candidates per query kept by the filter); 0 = planner */
  int64_t query_block;   /* query rows per block (rounded up to 32); 0 = planner */
  int32_t ref_splits;    /* reference splits processed in parallel; 0 = planner */
  float margin_scale;    /* >= 1: multiplies every error term of the certificate; 1 = default */
  int32_t force_fallback;/* debug: treat every row as uncertified (exact recomputation) */
  int32_t no_recheck;    /* debug: return the filter's shortlist order without verification */
  int32_t reorder;       /* scan order of an X-against-X call (tod_knn with xq == xr, tod_knn_score,
                          * tod_lof): 0 = planner, 1 = on, -1 = off.  On: the rows are grouped by
                          * their nearest of G evenly spaced rows (G = 16, or for rows of at most
                          * 16 elements one per 8192 rows, up to 1024) and every query block
                          * first scans the references of its own group, so the filter's
                          * thresholds tighten early.  Results are identical either way. */
  int32_t score;         /* tod_score: the kNN outlier score of tod_knn_score, tod_knn_decision
                          * and tod_lof's knn_score_out */
  int32_t tail_parts;    /* fp16 / bf16 filter with one reference split: the workgroups of a
                          * query block's last, partly filled round of the GPU scan the
                          * references in this many parts on separate workgroups (their lists
                          * are merged before the recheck); 0 = planner, 1 = off, at most 8.
                          * Results are identical either way. */
} tod_options;

/* Plan and per-phase timings of one call (filled when a non-NULL pointer is
 * passed; timings are measured with HIP events on the call's stream). */
/* (The recheck's candidate count m is not reported per call: it grows per
 * row, k + 8 first and then 16 more at a time up to K', so rows_certified and
 * rows_fallback carry what a single maximum would summarise.) */
typedef struct {
  uint32_t struct_size;   /* must be sizeof(tod_stats) */
  int32_t precision;      /* resolved tod_precision */
  int32_t kprime;         /* shortlist length K' */
  int32_t ref_splits;     /* S */
  int64_t query_block;    /* B_q */
  int64_t blocks;         /* number of query blocks */
  int64_t rows_certified; /* rows whose shortlist passed the certificate */
  int64_t rows_fallback;  /* rows recomputed exactly */
  int64_t tile_launches;  /* launches of the fused distance + selection kernel (a block with a
                           * tail split takes two) */
  float ms_prep, ms_tile, ms_recheck, ms_fallback, ms_score, ms_total;
                          /* ms_recheck includes the merge of the split lists, which runs
                           * inside the recheck kernel (there is no separate ms_merge) */
  int32_t reordered;      /* 1 if the scan used the grouped row order (see tod_options.reorder) */
  int64_t pairs_candidate; /* range queries (tod_nwr, tod_loci, tod_lof_ties): pairs the filter
                            * could not rule out of range */
  int64_t pairs_uncertain; /* range queries: candidates whose test needed the exact distance */
  int64_t pairs_in_range;  /* range queries: pairs within the threshold */
  int32_t tail_parts;      /* parts the last partly filled round was scanned in (1: none) */
  int64_t tail_rows;       /* query rows scanned in parts, summed over the blocks */
  int32_t list_runs;       /* 2 if each shortlist was built as two runs of K'/2 entries (the
                            * register-list tile over two pieces of the scan order: K' = 128
                            * on rows of 129..512 elements), else 1 */
} tod_stats;

/* Fill *opts with defaults: AUTO precision (the fp16 filter of Section 5.2's
 * provable quantization), planner-chosen K', query block and splits
 * (Section 6), self pair kept, margin_scale 1. */
void tod_default_options(tod_options* opts);

/*
 * Workspace bytes with which the call runs its queries in as few blocks as
 * the planner likes (Section 6: the batches are sized to the GPU memory at
 * hand; a smaller workspace gives smaller query blocks, see
 * tod_plan_workspace).  One function serves every entry point through
 *   mode 0: tod_knn, tod_knn_score, tod_knn_decision (any query and reference sets);
 *   mode 1: tod_lof, tod_abod, tod_cof (X against itself, nq == nr: these
 *           keep the neighbour lists and the LOF buffers as well);
 *   mode 2: tod_knn_classify (neighbour lists for the vote).
 * (mode is an addition to the interface the kNN/LOF calls alone would need:
 * the detectors built on the same lists need more room.)
 * Returns 0 if the arguments are invalid or unsupported.
 */
size_t tod_workspace_size(int64_t nq, int64_t nr, int64_t d, int32_t k, int32_t mode,
                          const tod_options* opts);

/*
 * kNN: for each of the nq query rows xq[nq x d], the k nearest rows of
 * xr[nr x d] (Section 4.2, kNN = cdist + topk; exact as in Section 7's
 * exactness claim).
 *   idx_out[nq x k]  int64, reference row ids sorted by (distance, id)
 *   dist_out[nq x k] fp32, Euclidean distances (rounded from fp64)
 * opts may be NULL (defaults).  stats may be NULL.
 * Requires 1 <= k <= nr - exclude_self, k <= 256, d <= 4096.
 */
tod_status tod_knn(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d,
                   int32_t k, const tod_options* opts, void* workspace, size_t ws_bytes,
                   void* stream, int64_t* idx_out, float* dist_out, tod_stats* stats);

/*
 * tod_knn for callers that cannot allocate device memory (serving loops that
 * keep allocation off their path, harnesses that forbid hipMalloc): the same
 * computation and outputs as tod_knn, with no workspace argument.  Its
 * workspace is a static device array of TOD_NOALLOC_SCRATCH_BYTES inside the
 * library, one per GPU (the loaded code object holds it until the process
 * ends); the call makes no hipMalloc, hipFree, HIP event or other allocating
 * call.  The planner fits the query blocks and reference splits into that
 * array as it does for a small caller workspace (tod_plan_workspace with
 * ws_bytes = TOD_NOALLOC_SCRATCH_BYTES gives the plan).
 *   TOD_ERR_WORKSPACE  the problem does not fit the array (not even one
 *                      32-row query block beside the fixed buffers, or
 *                      opts fixes query_block / ref_splits beyond it): use
 *                      tod_knn with a workspace of its own.
 * Every call on a GPU shares that GPU's array, and the array keeps the last
 * call's contents (each call initialises what it reads).  Calls that overlap
 * on one GPU (other threads, other streams) race on it: the caller
 * serialises them.  The call still synchronises `stream` before it returns,
 * so it cannot be captured into a HIP graph.  stats, if given, carries the
 * plan and row counts; its timings are 0 (no events are created).
 */
#define TOD_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
tod_status tod_knn_noalloc(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d,
                           int32_t k, const tod_options* opts, void* stream, int64_t* idx_out,
                           float* dist_out, tod_stats* stats);

/*
 * kNN-OD scores of X against itself (each point's own row excluded), the
 * detector's fit (Appendix D's fit / decision_scores_):
 *   score_out[n] = opts->score of the k neighbour distances (default: the
 *                  distance to the k-th nearest neighbour, Table 1's kNN).
 * idx_out[n x k] and dist_out[n x k] are optional (NULL to skip).
 */
tod_status tod_knn_score(const float* x, int64_t n, int64_t d, int32_t k,
                         const tod_options* opts, void* workspace, size_t ws_bytes,
                         void* stream, float* score_out, int64_t* idx_out, float* dist_out,
                         tod_stats* stats);

/*
 * LOF of X against itself (Table 1; Breunig et al. 2000, exactly k
 * neighbours, self excluded):
 *   lof_out[n]       fp32 LOF scores (computed in fp64)
 *   knn_score_out[n] optional: kNN-OD score from the same neighbour lists
 *   idx_out, dist_out optional neighbour lists as in tod_knn
 * (The optional outputs cost no extra pass: LOF needs the exact lists and
 * k-distances anyway, so a caller that wants both detectors makes one call.)
 */
tod_status tod_lof(const float* x, int64_t n, int64_t d, int32_t k, const tod_options* opts,
                   void* workspace, size_t ws_bytes, void* stream, float* lof_out,
                   float* knn_score_out, int64_t* idx_out, float* dist_out, tod_stats* stats);

/*
 * LOF on Breunig et al.'s k-distance neighbourhoods (Table 1's LOF; a user
 * of neighbours within range, Section 5.3): every point tied at the
 * k-distance belongs, so a neighbourhood can hold more than k points.  For
 * every row p of X (its own row excluded):
 *   kd2(p)   = the k-th smallest D2(p, o), o != p
 *   N_k(p)   = {o != p : D2(p, o) <= kd2(p)}
 *   reach(p, o) = max(sqrt(kd2(o)), sqrt(D2(p, o)))
 *   lrd(p)   = 1 / (mean over N_k(p) of reach(p, o) + 1e-10)
 *   LOF(p)   = mean over N_k(p) of lrd(o), divided by lrd(p)
 * D2 is the fp64 squared distance summed over the columns in order without
 * fused multiply-adds; membership is decided exactly in it (as tod_nwr
 * decides range membership).  Where no distance ties the k-distance, N_k(p)
 * is the k nearest and the result is tod_lof's.
 * Steps: the exact kNN lists with k + 1 entries (as tod_knn, self excluded;
 * k entries when k = n - 1), kd2 from the first k; if every row's (k+1)-th
 * neighbour is farther than kd2 (by more than the summation orders can
 * differ), no point ties and the neighbourhoods are the k-lists; otherwise
 * they come from the range query at each row's own radius (tod_nwr's
 * fp16 / bf16 range filter with exact verification).  Then lrd and LOF.
 *   capacity         pairs (p, o) the workspace holds, summed over p; at
 *                    least n k (no ties)
 *   lof_out[n]       fp32 LOF scores (computed in fp64)
 *   count_out[n]     optional: |N_k(p)| (int32)
 * Workspace: tod_lof_ties_workspace_size(n, d, k, capacity, opts) bytes (0:
 * invalid sizes or options).  Requires d <= 512 and an fp16 / bf16 / AUTO
 * precision (TOD_ERR_UNSUPPORTED otherwise); opts->exclude_self is ignored
 * (always on).  TOD_ERR_CAPACITY if the neighbourhoods hold more than
 * capacity pairs: stats->pairs_in_range (when stats is given) then holds the
 * number needed, and lof_out is unspecified.
 */
size_t tod_lof_ties_workspace_size(int64_t n, int64_t d, int32_t k, int64_t capacity,
                                   const tod_options* opts);
tod_status tod_lof_ties(const float* x, int64_t n, int64_t d, int32_t k, int64_t capacity,
                        const tod_options* opts, void* workspace, size_t ws_bytes, void* stream,
                        float* lof_out, int32_t* count_out, tod_stats* stats);

/*
 * kNN-OD scores of new points xq[nq x d] against the fitted set xr[nr x d]
 * (Appendix D's decision_function, the inductive setting): the same score as
 * tod_knn_score, from the k nearest rows of xr, nothing excluded (a row of xr
 * passed again as a query is its own neighbour at distance 0).
 *   score_out[nq] fp32; idx_out, dist_out optional as in tod_knn.
 * opts->exclude_self must be 0.
 */
tod_status tod_knn_decision(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d,
                            int32_t k, const tod_options* opts, void* workspace, size_t ws_bytes,
                            void* stream, float* score_out, int64_t* idx_out, float* dist_out,
                            tod_stats* stats);

/*
 * kNN classifier (Appendix B's kNN_CLF: cdist, topk, then a majority vote):
 * the predicted class of every row of xq is the most frequent label among
 * its k nearest rows of xr, ties going to the smallest label.
 *   labels_r[nr]  int32 (device), classes 0 .. n_classes - 1
 *   pred_out[nq]  int32 (device)
 * Requires 1 <= n_classes <= 65536 and opts->exclude_self == 0 (unless
 * xq == xr: then each point votes without itself).  A label outside
 * [0, n_classes) makes the call fail with TOD_ERR_INVALID_ARG (after the
 * kernels ran; pred_out is then unspecified).  Workspace: mode 2.
 */
tod_status tod_knn_classify(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d,
                            int32_t k, const int32_t* labels_r, int32_t n_classes,
                            const tod_options* opts, void* workspace, size_t ws_bytes,
                            void* stream, int32_t* pred_out, tod_stats* stats);

/*
 * ABOD as Section 4.3 builds it from the kNN and cosine-similarity operators:
 * for every point of X (its own row excluded), the mean over the unordered
 * pairs {b, c} of its k nearest neighbours of the cosine of the angle between
 * x_b - x_i and x_c - x_i (fp64, rounded to fp32).  Pairs with a
 * zero-length difference (a duplicate of x_i) are left out; a point without
 * any pair left scores 0.  Higher means more outlying (the neighbours lie in
 * one direction).
 *   score_out[n] fp32; idx_out, dist_out optional lists as in tod_knn.
 * Requires 2 <= k <= 64 (TOD_ERR_INVALID_ARG below, TOD_ERR_UNSUPPORTED above).
 * Workspace: mode 1 of tod_workspace_size.
 */
tod_status tod_abod(const float* x, int64_t n, int64_t d, int32_t k, const tod_options* opts,
                    void* workspace, size_t ws_bytes, void* stream, float* score_out,
                    int64_t* idx_out, float* dist_out, tod_stats* stats);

/*
 * COF, the connectivity-based outlier factor (Tang et al.; Table 1), of
 * every point of X (its own row excluded).  For point p and G = {p} plus its
 * k nearest neighbours, the set-based nearest path starts from {p} and adds,
 * k times, the point of G nearest to the points added so far (distance to a
 * set = smallest distance to a member; ties to the lower row index); step i
 * costs that distance c_i.  The average chaining distance is
 *   ac(p) = sum_i 2 (k + 1 - i) / (k (k + 1)) c_i
 * and COF(p) = (ac(p) + 1e-10) / (mean over the neighbours o of ac(o) + 1e-10)
 * (fp64, rounded to fp32; the 1e-10 keeps duplicates finite, as LOF's does).
 *   cof_out[n] fp32; knn_score_out, idx_out, dist_out optional as in tod_lof.
 * Requires 1 <= k <= 63 (TOD_ERR_UNSUPPORTED above).  Workspace: mode 1.
 */
tod_status tod_cof(const float* x, int64_t n, int64_t d, int32_t k, const tod_options* opts,
                   void* workspace, size_t ws_bytes, void* stream, float* cof_out,
                   float* knn_score_out, int64_t* idx_out, float* dist_out, tod_stats* stats);

/*
 * Host-only planner (Section 6 automatic batching): fills *plan with the
 * precision, K', query block, reference splits and block count that tod_knn
 * would use, without touching the GPU.  Only the plan fields of tod_stats
 * are written; tile_launches counts one launch per block (the tail split is
 * decided at run time from the GPU's occupancy).
 */
tod_status tod_plan(int64_t nq, int64_t nr, int64_t d, int32_t k, const tod_options* opts,
                    tod_stats* plan);

/*
 * The plan a call would use with a workspace of ws_bytes (Section 6:
 * automatic batching sized to the memory at hand; the paper batches so that
 * large inputs fit a GPU's memory).  A workspace smaller than
 * tod_workspace_size() is not an error by itself: the query block shrinks to
 * what the room beside the fixed buffers (quantised copies, norms, radii,
 * worklist, neighbour lists) holds, at S x K' x 8 bytes per query row, the
 * reference splits S follow the smaller block, and the rows run in more
 * blocks with identical results.  TOD_ERR_WORKSPACE if not even one 32-row
 * block fits, or if opts fixes query_block or ref_splits and the plan does
 * not fit.  mode as in tod_workspace_size; the plan is for X against itself
 * when mode == 1 or opts->exclude_self is set, else for separate sets.
 * Host only, like tod_plan.
 */
tod_status tod_plan_workspace(int64_t nq, int64_t nr, int64_t d, int32_t k, int32_t mode,
                              const tod_options* opts, size_t ws_bytes, tod_stats* plan);

/*
 * Neighbours within range (NWR, Section 5.3: the case study of provable
 * quantization).  For every query row i, the reference rows j whose
 * Euclidean distance is at most phi.  The decision is exact: a pair is in
 * range iff its squared distance, summed in fp64 over the columns in order
 * from the fp32 rows ((double)x - (double)y, squared, added), is at most
 * phi * phi rounded to fp64.  The filter evaluates every pair in fp16 / bf16
 * (MFMA, fp32 accumulation); pairs it can place on neither side of phi with
 * certainty (Eq. (nwr-check)'s test |D - phi| > Err, with this library's
 * error bound) are recomputed exactly, the others are decided by the filter.
 *   row_ptr_out[nq + 1] int64 (device): CSR offsets, row i's pairs occupy
 *                       [row_ptr_out[i], row_ptr_out[i + 1]).  Always written.
 *   idx_out[capacity]   int64 (device), nullable: reference ids, ascending
 *                       within a row.  NULL = count only.
 *   dist_out[capacity]  fp32 (device), nullable: their Euclidean distances
 *                       (fp64 rounded to fp32).
 *   total_out           HOST pointer, nullable: the number of pairs in range.
 * opts: precision AUTO (= FP16) or FP16 / BF16 (FP32 is TOD_ERR_UNSUPPORTED:
 * the range filter is an MFMA tile), exclude_self (drops j == i; requires
 * xq == xr and nq == nr), ref_splits, margin_scale, force_fallback (no pair
 * is ruled in by the filter: every candidate is recomputed).  shortlist,
 * query_block, no_recheck and reorder do not apply.
 * Workspace: a fixed part plus room for candidate pairs (8 bytes each);
 * tod_nwr_workspace_size() gives the fixed part plus room for 64 candidates
 * per query row and 2^20 more.  Any extra bytes are used as candidate room.
 * Query rows are processed in as many batches (of multiples of 32 rows) as
 * that room needs: automatic batching sized to memory (Section 6).
 * TOD_ERR_WORKSPACE if 32 consecutive query rows have more candidates than
 * the room holds (tod_last_error() names the bytes needed).
 * TOD_ERR_CAPACITY if idx_out is given and the total exceeds capacity; then
 * row_ptr_out and *total_out are valid and idx_out / dist_out unspecified.
 * Requires phi finite and >= 0, d <= 512.
 */
size_t tod_nwr_workspace_size(int64_t nq, int64_t nr, int64_t d, const tod_options* opts);
tod_status tod_nwr(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d,
                   double phi, const tod_options* opts, void* workspace, size_t ws_bytes,
                   void* stream, int64_t* row_ptr_out, int64_t capacity, int64_t* idx_out,
                   float* dist_out, int64_t* total_out, tod_stats* stats);

/*
 * LOCI, the multi-granularity deviation factor of Papadimitriou et al.
 * (one of Table 1's proximity-based detectors; like LOF it is built on
 * neighbours within range, Section 5.3), at a ladder of sampling radii
 * r_0 < r_1 < ... < r_{L-1}.  For every row p of X and every radius r_l:
 *   n_alpha[p][l] = |{q : d(p, q) <= alpha r_l}|  (counting neighbourhood)
 *   n_r[p][l]     = |{q : d(p, q) <= r_l}|        (sampling neighbourhood)
 * (p itself belongs to both); n_hat and sigma are the mean and the population
 * standard deviation of n_alpha[q][l] over q in the sampling neighbourhood,
 *   MDEF = 1 - n_alpha[p][l] / n_hat,   sigma_MDEF = sigma / n_hat.
 * Membership is exact, as in tod_nwr: d(p, q) <= r iff the fp64 squared
 * distance summed over the columns in order is <= fl(r * r), and
 * d(p, q) <= alpha r iff it is <= fl(fl(alpha * r)^2).  The neighbourhood
 * sums S1 = sum n_alpha[q][l] and S2 = sum n_alpha[q][l]^2 are exact 64-bit
 * integers; then, in fp64 and in this order, n_hat = S1 / n_r,
 * var = S2 / n_r - n_hat * n_hat (negative values become 0),
 * sigma = sqrt(var), MDEF, sigma_MDEF.  A radius counts for p when
 * n_r[p][l] >= n_min.  flag_out[p] = 1 when MDEF > k_sigma * sigma_MDEF at a
 * counted radius; score_out[p] = the largest MDEF / sigma_MDEF over the
 * counted radii, where a radius with sigma_MDEF = 0 (all samples equal, so
 * MDEF = 0) contributes 0, and 0 when no radius counts.
 *   radii               HOST array [n_radii] fp64, strictly increasing, >= 0,
 *                       finite; 1 <= n_radii <= 32.
 *   alpha               in (0, 1]; n_min >= 1; k_sigma finite, >= 0.
 *   capacity            pairs (p, q) with d(p, q) <= r_{L-1}, self pairs
 *                       included, that the workspace holds.  If more are in
 *                       range the call returns TOD_ERR_CAPACITY and, when
 *                       stats is given, stats->pairs_in_range = the number
 *                       needed (size the workspace for it and call again).
 *   score_out[n]        fp64 (device).
 *   flag_out[n]         int32 (device), nullable.
 *   n_alpha_out, n_r_out [n * n_radii] int32 (device), nullable, row-major
 *                       (radius fastest).
 *   mdef_out, sigma_mdef_out [n * n_radii] fp64 (device), nullable.
 * opts as tod_nwr (precision AUTO / FP16 / BF16, ref_splits, margin_scale,
 * force_fallback); exclude_self must be 0 (p samples itself).  Requires
 * n <= 2^20, which keeps S2 below 2^63 (TOD_ERR_UNSUPPORTED above).
 * Workspace: tod_loci_workspace_size(n, d, n_radii, capacity, opts) bytes,
 * 256-byte aligned; stats: the neighbours-within-range pass's fields, with
 * ms_score the time of the two LOCI kernels.
 */
size_t tod_loci_workspace_size(int64_t n, int64_t d, int32_t n_radii, int64_t capacity,
                               const tod_options* opts);
tod_status tod_loci(const float* x, int64_t n, int64_t d, const double* radii, int32_t n_radii,
                    double alpha, int32_t n_min, double k_sigma, int64_t capacity,
                    const tod_options* opts, void* workspace, size_t ws_bytes, void* stream,
                    double* score_out, int32_t* flag_out, int32_t* n_alpha_out,
                    int32_t* n_r_out, double* mdef_out, double* sigma_mdef_out,
                    tod_stats* stats);

/* Static string naming a status code. */
const char* tod_status_string(tod_status status);

/* Detail of the last error on the calling thread ("" if none). */
const char* tod_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TOD_H */
