// Internal declarations shared by the host driver (api.cpp) and the HIP
// kernels of libtod.  Not part of the public ABI.
#pragma once

#include <string>

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/tod.h"

namespace tod {

// ---------------------------------------------------------------------------
// Plan (automatic batching, Section 6): every size the kernels depend on.
// ---------------------------------------------------------------------------
struct Plan {
  int64_t nq, nr, d;
  int32_t k;
  int32_t precision;   // resolved tod_precision (never AUTO)
  int32_t kprime;      // K' (16, 32, 64, 128 or 256)
  int32_t splits;      // S: reference splits
  int64_t split_len;   // references per split (multiple of 32)
  int64_t query_block; // B_q (multiple of 32)
  int64_t blocks;      // ceil(nq / B_q)
  int32_t dpad;        // row stride of the quantised copies (elements)
  int32_t dpad_t;      // tile kernel specialisation: dpad if the query operand fits in
                       // registers (fp32: 8..64, fp16/bf16: 16..128), else 0
  int32_t esize;       // bytes per quantised element (4 or 2)
  int64_t nq_pad, nr_pad; // row counts padded to 32
  int32_t waves_per_group; // waves per workgroup of the tile kernel
  int32_t tile_kind;   // 0: LDS-list tile kernel (tile.h); 1: register-list MFMA kernel (mtile.h)
  int32_t fold;        // 1: rows carry the accumulator seed as extra columns (mtile.h layout)
  int32_t seedprod;    // 1: the register-list tile forms the seed -N_j/2 by one MFMA of four
                       // filter-precision parts of -N_j/(2c) against c (hn_r holds the parts)
  int32_t dmain;       // fold layout: columns [0, dmain) hold the row, [dmain, dmain + 4) the seed
  int32_t scale_exp;   // E: the scaled, centred rows satisfy max |s (x - mu)| < 2^E
  int32_t self;        // query set == reference set (one quantised copy)
  int32_t exclude_self;
  int32_t lof;         // LOF buffers needed
  int32_t lists;       // int32 / fp64 neighbour lists kept in the workspace (LOF, score
                       // aggregates, classifier)
  int32_t order;       // 1: grouped scan order (order.hip), X against X only
  int32_t groups;      // seed groups of the grouped order (order_groups)
  int32_t runs = 1;    // 2: the register-list tile scans the references in 2 S pieces of the
                       // scan order with lists of K' / 2; each query's K' slots per split
                       // then hold two ascending runs (rows of 256+ elements, K' = 128)
  int32_t tail_parts = 1;  // most parts a tail workgroup's scan is cut into (1: no tail split)
  int32_t tail_auto = 0;   // 1: pick the parts by the model in tail_pieces; 0: use tail_parts
  int64_t tail_lists = 0;  // K' lists the tail region holds (query rows x parts)
};

// Pieces for the tail split of a launch whose last round holds tw of the
// `slots` workgroups the GPU runs at once (tw = 0: no partial round) on `cus`
// compute units.  P pieces make tw P work items of 1/P of a scan each, which
// take ceil(tw P / slots) rounds of 1/P.  Every extra piece costs its rows a
// list filled from nothing and one more list to merge, charged at 2% of a
// round.  The planner splits only a tail that leaves some compute unit idle
// (tw < cus): a tail with a workgroup on every unit runs each of them faster
// than a full round does, and splitting it was measured slower.  At most
// pmax pieces, at least 4 stages per piece, and the tail rows' lists must fit
// the tail region.  Without the planner (automatic = false) the most pieces
// these limits allow, up to pmax.
inline int tail_pieces(int64_t tw, int64_t slots, int64_t cus, int pmax, bool automatic,
                       int64_t nst, int64_t cap_lists, int64_t tail_rows) {
  if (tw <= 0 || slots <= 0 || tail_rows <= 0) return 1;
  if (automatic && tw >= cus) return 1;
  int best = 1;
  double best_cost = 1.0;
  for (int P = 2; P <= pmax; ++P) {
    if (nst < 4 * P || tail_rows * P > cap_lists) break;
    if (!automatic) {
      best = P;
      continue;
    }
    const double rounds = (double)((tw * P + slots - 1) / slots);
    const double cost = rounds / P + 0.02 * (P - 1);
    if (cost < best_cost - 1e-9) {
      best = P;
      best_cost = cost;
    }
  }
  return best;
}

// Workspace regions (byte offsets from the workspace base, 256-aligned).
struct Layout {
  size_t ctrl, mu64, mu32, colpart, xq_r, xq_q, hn_r, n64_q, rho_q, partial, ptail, worklist,
      fbtau, fbpart, fbidx, idx32, d64, lrd, kdist, perm, lab, oseed, cstart, bcnt, boff,
      total;
  int32_t colpart_blocks;
};

constexpr int kUncParts = 32, kUncStride = 16;

// Control block at the start of the workspace (device side).  (Certified rows
// are not counted here: every query row is either certified or on the
// worklist.)
struct Ctrl {
  uint32_t nonfinite;       // set to 1 if any input value is NaN/Inf
  uint32_t maxabs_bits;     // max |x - mu| over both sets, fp32 bits (non-negative)
  uint64_t nmax_bits;       // max ||xhat_j||^2 over references, fp64 bits
  uint64_t pmax_bits;       // max rho_j over references, fp64 bits
  uint32_t worklist_count;  // rows appended for exact recomputation
  uint32_t internal;        // set when a kernel finds an inconsistency it cannot recover from
  uint64_t fold_max_bits;   // max over references of the folded seed's error, fp64 bits
  uint32_t bad_label;       // classifier: a reference label outside [0, n_classes)
  uint32_t pad0;
  // NWR: candidate pairs recomputed exactly, as kUncParts partial counts
  // 128 bytes apart (the total is their sum).  Atomics on one address from
  // every wave serialise: at 3 x 10^4 rows they took as long as the rest of
  // the verification.
  uint64_t uncertain[kUncParts * kUncStride];
};

// Everything a kernel needs to know about the problem.
struct Args {
  const float* xq;  // original fp32 queries [nq x d]
  const float* xr;  // original fp32 references [nr x d]
  int64_t nq, nr;
  int32_t d, dpad, k, kprime;
  int32_t splits;
  int64_t split_len;
  int32_t exclude_self;
  int32_t precision;
  float margin_scale;
  int32_t force_fallback, no_recheck;
  int32_t fold, dmain, scale_exp;
  int32_t seedprod;  // see Plan::seedprod
  // workspace views
  Ctrl* ctrl;
  double* mu64;
  float* mu32;
  double* colpart;
  void* xq_r;       // quantised references [nr_pad x dpad]
  void* xq_q;       // quantised queries [nq_pad x dpad] (== xq_r when self)
  float* hn_r;      // -0.5 * fl32(||xhat_j||^2) per reference [nr_pad]; with seedprod the
                    // four seed parts of reference j (filter precision, 8 bytes) instead
  double* n64_q;    // ||xhat_i||^2 per query (fp64) [nq_pad]
  double* rho_q;    // quantisation radius per query, rounded up [nq_pad]
  double* rho_r;    // quantisation radius per reference when the sets differ (NWR), else null
  uint64_t* partial;   // per (query in block, split) sorted K' lists
  // Tail split (register-list tile, one reference split): a tile launch with
  // parts > 1 scans the references in `parts` pieces of the scan order, piece
  // blockIdx.y, and writes list (query, piece) at partial + (query * parts +
  // piece) * K'.  The recheck takes the rows of its block from tail_q0 on
  // from ptail, tail_parts lists each.
  int32_t parts;
  // runs > 1: each K' list the recheck reads holds `runs` ascending runs of
  // K' / runs entries (pieces of the scan order); they are merged there, and
  // every reference a run left out has a key >= that run's last entry.
  int32_t runs;
  int32_t tail_parts;
  int64_t tail_q0;
  uint64_t* ptail;
  int32_t* worklist;   // global query ids that failed the certificate
  double* fbtau;       // per worklist entry: the k-th smallest exact D^2 the recheck measured
  uint2* fbpart;       // fallback chunk lists: (D^2 bits hi, lo) [kFbGrid x k]
  uint32_t* fbidx;     // fallback chunk lists: reference ids [kFbGrid x k]
  // grouped scan order (all null when the input order is kept)
  int32_t* perm;       // position -> input row [nr]
  int32_t* lab;        // input row -> group [nr]
  int32_t groups;      // seed groups of the grouped order
  float* oseed;        // the seed rows of rows of at most 16 elements [groups x 16]
  int32_t* cstart;     // first position of each group [groups + 1]
  int32_t* bcnt;       // rows per group in each block of kOrdRows rows
  int32_t* boff;       // first position of each block's rows of each group
  int32_t* idx32;      // [nq x k] neighbour ids (LOF)
  double* d64;         // [nq x k] exact distances (LOF)
  double* lrd;         // [nq] LOF scratch
  double* kdist;       // [nq] exact k-distance of every row (LOF), beside the lists so that
                       // the neighbours' k-distances are gathered from a dense array
  // outputs (nullable)
  int64_t* idx_out;
  float* dist_out;
  float* score_out;
  float* lof_out;
  int32_t score;            // tod_score of score_out
  int32_t n_classes;        // classifier
  const int32_t* labels_r;  // classifier: reference labels [nr]
  int32_t* pred_out;        // classifier: predicted classes [nq]
  // neighbours within range (rtile.h, nwr.hip)
  double phi;          // the range threshold (a distance)
  const double* phi2_row;  // null, or a squared radius per query row [nq]: the range test of
                           // row q is then D2 <= phi2_row[q] (exact fp64), phi unused
  int32_t* ccount;     // count pass: candidates per (query, split) [nq_pad x S]
  int64_t* coff;       // their exclusive prefix sums [nq x S + 1]
  int64_t cbase;       // candidate offset of the first row of the current query batch
  uint32_t* cand;      // candidate reference ids of the batch; bit 31: not ruled in by the filter
  float* cand_d;       // fill pass: the candidate's accumulator; after verification: its
                       // distance if kept (0 if not measured), -1 if not
  int64_t ccap;        // candidate room
  int32_t* incnt;      // pairs in range per query row [nq]
  int64_t* row_ptr;    // CSR offsets [nq + 1] (the caller's output)
  int64_t out_cap;     // entries idx_out / dist_out can hold
};

// Power-of-two scale s with s * maxabs < 2^E (exact scaling of the centred
// rows; the fp16 range then holds every quantised value, product and folded
// seed part).
__device__ __forceinline__ double scale_from_maxabs(uint32_t bits, int scale_exp) {
  const float m = __uint_as_float(bits);
  if (!(m > 0.0f)) return 1.0;
  const int e = isinf(m) ? 128 : ilogbf(m);  // m < 2^(e+1)
  return ldexp(1.0, scale_exp - 1 - e);
}

// Constant the queries carry in the seed columns of the fold layout: the
// seed -N_j/2 is stored as parts of -N_j/(2c) so that fp16 parts stay in range.
__host__ __device__ constexpr double fold_const(int precision) {
  return precision == TOD_PREC_FP16 ? 32768.0 : 1.0;
}

// Grouped scan order: the most seed groups (their count, a power of two, is
// order_groups'), rows per counting block, and the smallest reference set the
// planner groups by default.
constexpr int kOrdMaxC = 1024;
constexpr int kOrdRows = 1024;
constexpr int64_t kOrderMinRows = 4096;
int32_t order_groups(int64_t nr, int64_t d);
int32_t order_blocks(int64_t nr);
hipError_t launch_order(const Plan& p, const Args& a, hipStream_t s);

// Exact squared distance of two fp32 rows, as the definition states it: fp64,
// columns in order, ((double)x - (double)y)^2 added one at a time with no
// fused multiply-add.  Rows of a multiple of four elements are read as float4
// (16-byte aligned rows).
__device__ __forceinline__ double exact_d2(const float* __restrict__ q,
                                           const float* __restrict__ r, int d) {
#pragma clang fp contract(off)
  double s = 0.0;
  if ((d & 3) == 0) {
    for (int t = 0; t < d; t += 4) {
      const float4 x = *reinterpret_cast<const float4*>(q + t);
      const float4 y = *reinterpret_cast<const float4*>(r + t);
      double e = (double)x.x - (double)y.x;
      s = s + e * e;
      e = (double)x.y - (double)y.y;
      s = s + e * e;
      e = (double)x.z - (double)y.z;
      s = s + e * e;
      e = (double)x.w - (double)y.w;
      s = s + e * e;
    }
  } else {
    for (int t = 0; t < d; ++t) {
      const double e = (double)q[t] - (double)r[t];
      s = s + e * e;
    }
  }
  return s;
}

// LOCI (Papadimitriou et al.): arguments of the two passes over the
// neighbours within the largest radius (tod_nwr's CSR, self pairs included).
constexpr int kLociMaxRadii = 32;
struct LociArgs {
  const float* x;
  int64_t n;
  int32_t d;
  int32_t nl;   // radii
  int32_t nls;  // row stride of na / nr (8, 16 or 32 >= nl)
  int32_t n_min;
  double k_sigma;
  const int64_t* row_ptr;
  const int64_t* idx;
  uint8_t* bins;  // per pair: index of the first sampling radius that holds it
  int32_t* na;    // [n x nls] counting-neighbourhood sizes n(p, alpha r_l)
  int32_t* nr;    // [n x nls] sampling-neighbourhood sizes n(p, r_l)
  double r2[kLociMaxRadii];  // fl(r_l * r_l)
  double a2[kLociMaxRadii];  // fl(fl(alpha * r_l)^2)
  double* score;
  int32_t* flag;
  int32_t* na_out;
  int32_t* nr_out;
  double* mdef_out;
  double* smdef_out;
};
hipError_t launch_loci(const LociArgs& a, hipStream_t s);

// Fallback scan grid and the most chunks one failing row is cut into.
constexpr int kFbGrid = 1024;
constexpr int kFbMaxChunks = 64;

// Number of blocks of the column-mean reduction (also sizes its workspace).
int32_t colsum_blocks(int64_t nr);

// Kernel launchers (return hipSuccess or the launch error).
hipError_t launch_prep(const Plan& p, const Args& a, hipStream_t s);
// Query rows of a block from q0 on scanned in `parts` pieces (the tail split).
struct TileTail {
  int64_t q0;
  int32_t parts;
};
// The register-list tile fills *tail (no tail split: q0 = q_rows, parts = 1);
// the other tile kernels leave it untouched.
hipError_t launch_tile(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                       hipStream_t s, TileTail* tail);
hipError_t launch_tile_f32(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                           hipStream_t s);
hipError_t launch_tile_f16(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                           hipStream_t s);
hipError_t launch_tile_bf16(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                            hipStream_t s);
hipError_t launch_mtile_f16(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                            hipStream_t s, TileTail* tail);
hipError_t launch_mtile_bf16(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                             hipStream_t s, TileTail* tail);
hipError_t launch_recheck(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                          hipStream_t s);
hipError_t launch_fallback(const Plan& p, const Args& a, hipStream_t s);
hipError_t launch_lof(const Plan& p, const Args& a, hipStream_t s);
// LOF on tie-inclusive neighbourhoods (lof.hip): each row's squared
// k-distance from its exact kNN list (k1 = k + 1 entries, the last one to
// rule ties out; *tie set where one is possible), the neighbourhoods as the
// k-lists when no row has a possible tie, then lrd and LOF over the CSR
// neighbourhoods (else those of the range query at each row's radius).
hipError_t launch_ties_radius(const float* x, int64_t n, int d, int k, int k1,
                              const int64_t* lists, double* kd2, int32_t* tie, hipStream_t s);
hipError_t launch_ties_lists(int64_t n, int k, int k1, const int64_t* lists, int64_t* row_ptr,
                             int64_t* nbr, hipStream_t s);
hipError_t launch_lof_ties(const float* x, int64_t n, int d, const int64_t* row_ptr,
                           const int64_t* nbr, const double* kd2, double* lrd, float* lof,
                           int32_t* count, hipStream_t s);
// kNN score aggregates (mean, median, sum) and the classifier's majority vote
// from the exact lists.
hipError_t launch_score(const Plan& p, const Args& a, hipStream_t s);
hipError_t launch_vote(const Plan& p, const Args& a, hipStream_t s);
hipError_t launch_abod(const Plan& p, const Args& a, hipStream_t s);
// COF: average chaining distances into lrd (fp64 [n]), COF into lof_out.
hipError_t launch_cof(const Plan& p, const Args& a, hipStream_t s);

// Neighbours within range: fused MFMA tile with the range test (count pass:
// candidates per (query, split); fill pass: their ids, in increasing j per
// row), exact verification, CSR assembly.
hipError_t launch_range_tile_f16(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                                 bool fill, hipStream_t s);
hipError_t launch_range_tile_bf16(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                                  bool fill, hipStream_t s);
// Exclusive prefix sums of n int32 values into out[0..n] (out[n] = total),
// plus *base when base is not null.  part holds scan_parts(n) int64.
int64_t scan_parts(int64_t n);
hipError_t launch_scan(const int32_t* in, int64_t n, int64_t* out, const int64_t* base,
                       int64_t* part, hipStream_t s);
// goff[g] = coff[min(32 g, nq) * S] for g = 0..groups.
hipError_t launch_group_offsets(const Args& a, int64_t groups, int64_t* goff, hipStream_t s);
hipError_t launch_range_verify(const Args& a, int64_t b0, int64_t rows, int32_t want_dist,
                               hipStream_t s);
hipError_t launch_range_emit(const Args& a, int64_t b0, int64_t rows, hipStream_t s);

// Planner and layout (host only, no HIP calls).
tod_status make_plan(int64_t nq, int64_t nr, int64_t d, int32_t k, int32_t lof, int32_t self,
                     const tod_options& o, Plan* plan, const char** why);
Layout make_layout(const Plan& p);

tod_status make_plan_nwr(int64_t nq, int64_t nr, int64_t d, int32_t self, const tod_options& o,
                         Plan* plan, const char** why);
// NWR workspace regions; cand is the first byte of the candidate room.
struct NwrLayout {
  size_t ctrl, mu64, mu32, colpart, xq_r, xq_q, hn_r, n64_q, rho_q, rho_r, ccount, coff, part,
      goff, incnt, cand;
  int64_t groups;  // 32-row query groups
  int32_t colpart_blocks;
};
NwrLayout make_layout_nwr(const Plan& p);
// Candidate pairs a workspace of ws_bytes holds (0 if it is smaller than the fixed part).
int64_t nwr_candidate_room(const NwrLayout& L, size_t ws_bytes);

}  // namespace tod
