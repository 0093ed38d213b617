// Fused distance tiles + per-row top-K' selection, certificate with exact
// recheck, and exact fallback (the kNN functional operator of Section 4.2
// evaluated with provable quantization, Section 5.2, and operator fusion,
// Section 6.1).
//
// Distance tile.  For query i and reference j the filter ranks
//     key_ij = fl32(N_j) - 2 <xhat_i, xhat_j>
// (the right-hand expansion of Eq. (dist-decomp) without the row constant
// ||xhat_i||^2).  A wave owns 32 queries and walks its reference split in
// 32-row tiles; each lane ends a tile holding 16 accumulators for one query:
//     acc = -N_j/2 + <xhat_i, xhat_j>,    key = -2 * acc   (exact scaling).
// fp16/bf16 use v_mfma_f32_32x32x16_{f16,bf16} (rows = references,
// columns = queries, fp32 accumulate); fp32 uses VALU FMA chains.
//
// Selection.  Each query keeps a sorted list of its K' best (key, index)
// entries in LDS and a per-lane threshold in acc space.  A tile costs one
// max-reduction and one compare per lane unless some lane beats its
// threshold; survivors go to a per-(query, half-wave) LDS queue, and full
// queues are merged into the lists with wave64 bitonic networks.  The n x n
// matrix never exists (Section 6.1's fused cdist + topk).
//
// Certificate (step iii of Section 5.2, re-derived for top-k).  After the
// reference splits are merged, the K'-th key h bounds every excluded
// reference: key_ij >= h.  With the fp32 accumulation bound
//     |key_ij - (N_j - 2<xhat_i, xhat_j>)| <= gamma_{d+2} (N_i + 2 Nmax) + 2^-23 Nmax
// and the quantisation radii, every excluded j satisfies
//     s ||x_i - x_j|| >= sqrt(N_i + h - e) - rho_i - Pmax = LB.
// The K' candidates are re-measured in fp64 from the original fp32 rows:
// the definition's terms ((double)x - (double)y)^2, each rounded exactly as
// the definition rounds it (no fused multiply-add), but summed in another
// order (each lane of a group adds its strided column chunks in order, then
// the lanes' partial sums are added as a tree).  Two orders of summing d
// non-negative fp64 terms differ by at most 2 (d - 1) 2^-53 of the sum,
// below 2^-40 for d <= 4096; only candidates whose squared distances are that
// close can be ranked differently from the definition, i.e. only exact
// near-ties (within 2^-40 of each other).  The candidates are sorted
// by (D^2, j); if LB > s * D_(k) no excluded reference can enter the top k and
// the row is final.  Otherwise the row goes to the exact fallback scan.
#include <math.h>

#include "tod_internal.h"
#include "wave.h"

namespace tod {

namespace {



// Make this wave's LDS writes visible to its other lanes.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Row-independent inputs of the certificate (see file header).
struct CertConst {
  double nmax, pmax, s, gam, seedw, fold_err, ms, derr;
};

__device__ CertConst cert_const(const Args& a) {
  CertConst c;
  c.nmax = __longlong_as_double((long long)a.ctrl->nmax_bits);
  c.pmax = __longlong_as_double((long long)a.ctrl->pmax_bits);
  c.s = scale_from_maxabs(a.ctrl->maxabs_bits, a.scale_exp);
  const double u = 0x1p-23;  // per-addition allowance (2x the fp32 unit roundoff)
  // The seed as four parts against a constant: folded into the rows, or the
  // product of the register-list tile's seed MFMA; same terms either way.
  const bool parts = a.fold || a.seedprod;
  // d products, the seed (one term, or four parts) and one spare.
  const double t = (double)a.d + (parts ? 6.0 : 2.0);
  c.gam = t * u / (1.0 - t * u);
  c.ms = (double)a.margin_scale;
  // Seed weight in the sum of |terms|: N_j/2 for an fp32 seed; the parts'
  // magnitudes sum to at most (N_j/2)(1 + 2^-7) (bf16 parts; fp16 less).
  c.seedw = parts ? 2.0 + 0x1p-6 : 2.0;
  c.fold_err = parts ? 2.0 * __longlong_as_double((long long)a.ctrl->fold_max_bits) : 0.0;
  // Terms that do not depend on the row: u Nmax, the folded seed error and
  // the subnormal allowance.
  c.derr = u * c.nmax + c.fold_err + (double)a.d * 0x1p-120;
  return c;
}

// Lower bound test of the certificate for a row with squared norm ni and
// radius rho_i.  Returns true when no reference outside the shortlist can be
// among the k nearest.
__device__ bool certified(const CertConst& c, double ni, double rho_i, uint64_t hent,
                          double tau2) {
  if (hent == kEmpty) return true;  // the shortlist holds every reference
  const double h = (double)key_of(hent);
  const double err = c.ms * (c.gam * (ni + c.seedw * c.nmax) * (1.0 + 1e-6) + c.derr) +
                     1e-12 * (ni + fabs(h));
  const double arg = ni + h - err;
  const double lb = (arg > 0.0 ? sqrt(arg) : 0.0) - c.ms * (rho_i + c.pmax);
  return lb * (1.0 - 1e-9) > c.s * sqrt(tau2) * (1.0 + 1e-9);
}

// Write one neighbour (rank < k) of query qi to every requested output.
__device__ __forceinline__ void emit(const Args& a, int64_t qi, int rank, uint32_t j, double d2) {
  const int64_t pos = qi * a.k + rank;
  const double dd = sqrt(d2);
  if (a.idx_out) a.idx_out[pos] = (int64_t)j;
  if (a.dist_out) a.dist_out[pos] = (float)dd;
  if (a.idx32) {
    a.idx32[pos] = (int32_t)j;
    a.d64[pos] = dd;
  }
  if (rank == a.k - 1) {
    if (a.score_out) a.score_out[qi] = (float)dd;
    if (a.kdist) a.kdist[qi] = dd;
  }
}

__device__ __forceinline__ double shfl_xor_f64(double v, int mask) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  return __longlong_as_double((long long)shfl_xor64(b, mask));
}

// (q - r)^2 of four consecutive elements added to part in element order.
__device__ __forceinline__ double add_sq4(double part, float4 q, float4 r) {
#pragma clang fp contract(off)
  double df = (double)q.x - (double)r.x;
  part = part + df * df;
  df = (double)q.y - (double)r.y;
  part = part + df * df;
  df = (double)q.z - (double)r.z;
  part = part + df * df;
  df = (double)q.w - (double)r.w;
  part = part + df * df;
  return part;
}

__device__ __forceinline__ double add_sq1(double part, float q, float r) {
#pragma clang fp contract(off)
  const double df = (double)q - (double)r;
  return part + df * df;
}

// One pass of measure: candidate c (if below c1) by the lpc lanes of this group.
__device__ __forceinline__ void measure_pass(const Args& a, const float* __restrict__ qrow,
                                             const uint64_t* sl, double* sd2, int c, int c1,
                                             int lpc, int sub) {
  const uint64_t e = c < c1 ? sl[c] : kEmpty;
  const int d = a.d;
  double part = 0.0;
  if (e != kEmpty) {
    const float* rrow = a.xr + (int64_t)index_of(e) * d;
    if ((d & 3) == 0) {
      const float4* r4 = reinterpret_cast<const float4*>(rrow);
      const float4* q4 = reinterpret_cast<const float4*>(qrow);
      const int nch = d >> 2;
      int ch = sub;
      for (; ch + 3 * lpc < nch; ch += 4 * lpc) {
        const float4 r0 = r4[ch], r1 = r4[ch + lpc], r2 = r4[ch + 2 * lpc], r3 = r4[ch + 3 * lpc];
        const float4 q0 = q4[ch], q1 = q4[ch + lpc], q2 = q4[ch + 2 * lpc], q3 = q4[ch + 3 * lpc];
        part = add_sq4(part, q0, r0);
        part = add_sq4(part, q1, r1);
        part = add_sq4(part, q2, r2);
        part = add_sq4(part, q3, r3);
      }
      for (; ch < nch; ch += lpc) part = add_sq4(part, q4[ch], r4[ch]);
    } else {
      int t = sub;
      for (; t + 3 * lpc < d; t += 4 * lpc) {
        const float r0 = rrow[t], r1 = rrow[t + lpc], r2 = rrow[t + 2 * lpc], r3 = rrow[t + 3 * lpc];
        const float q0 = qrow[t], q1 = qrow[t + lpc], q2 = qrow[t + 2 * lpc], q3 = qrow[t + 3 * lpc];
        part = add_sq1(part, q0, r0);
        part = add_sq1(part, q1, r1);
        part = add_sq1(part, q2, r2);
        part = add_sq1(part, q3, r3);
      }
      for (; t < d; t += lpc) part = add_sq1(part, qrow[t], rrow[t]);
    }
  }
  for (int off = lpc >> 1; off > 0; off >>= 1) part = part + shfl_xor_f64(part, off);
  if (sub == 0 && c < c1) sd2[c] = e != kEmpty ? part : (double)INFINITY;
}

// Exact D^2 (the definition's direct differences, fp64) of the shortlist
// entries [c0, c1), c1 - c0 <= 64, into sd2.  Groups of lpc lanes take one
// candidate each: lpc = 64 / next_pow2(c1 - c0), but at least d / 64 (a power
// of two, at most 16) so that a load instruction of a long row covers few
// rows; the candidates then take several passes.  Lane `sub` of a group sums
// the chunks sub, sub + lpc, ... of the row in order (4 elements per chunk
// when rows are 16-byte aligned, else 1), four chunks' loads in flight at a
// time, and the group's partial sums are tree-reduced.
__device__ __forceinline__ void measure(const Args& a, const float* __restrict__ qrow,
                                        const uint64_t* sl, double* sd2, int c0, int c1,
                                        int lane) {
  int G = 1;
  while (G < c1 - c0) G <<= 1;
  int lpc = 64 / G;
  while (lpc < 16 && lpc * 64 < a.d) lpc <<= 1;
  const int grp = lane / lpc, sub = lane & (lpc - 1), per = 64 / lpc;
  for (int cb = c0; cb < c1; cb += per) measure_pass(a, qrow, sl, sd2, cb + grp, c1, lpc, sub);
}

// Merge of the per-split lists, then the progressive exact recheck: the
// candidates are measured exactly in key order, m at a time, until the
// certificate holds with h = the key of the first unmeasured candidate (every
// reference outside the first m has a key >= h) or the list is exhausted.
// One wave per query on a persistent grid; each measuring pass has all of its
// candidates' loads in flight at once.
template <int KP, int W>
__global__ void __launch_bounds__(W * 64)
recheck_kernel(Args a, int64_t q_begin, int64_t q_rows) {
#pragma clang fp contract(off)
  constexpr int EL = KP >= 64 ? KP / 64 : 1;
  __shared__ uint64_t sl[W][KP];
  __shared__ double sd2[W][KP];
  __shared__ double stau[W];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (a.ctrl->nonfinite) return;
  const CertConst cc = cert_const(a);
  // Each wave walks the block's queries with a grid stride.  (Every row is
  // either certified or put on the worklist, so the host derives the number
  // of certified rows from the worklist count: no counter of their own, whose
  // same-address atomics, one per wave, cost as much as the rest of the
  // kernel at 10^5 rows.)
  for (int64_t ql = (int64_t)blockIdx.x * W + wave; ql < q_rows; ql += (int64_t)gridDim.x * W) {
    // With the grouped scan order the filter worked on positions: the query's
    // input row is perm[position], and so is every candidate's (mapped below,
    // before anything is measured, ranked or written).
    const int64_t qpos = q_begin + ql;
    const int64_t qi = a.perm ? (int64_t)a.perm[qpos] : qpos;
    const double ni = a.n64_q[qpos], rho_i = a.rho_q[qpos];
    // Final aggregation of the per-split candidate lists (Section 6.1).
    // Rows of the tail split have one list per scanned piece.
    const bool tl = ql >= a.tail_q0;
    const int nlists = tl ? a.tail_parts : a.splits;
    const uint64_t* src =
        tl ? a.ptail + (ql - a.tail_q0) * a.tail_parts * KP : a.partial + ql * a.splits * KP;
    // With runs (a.runs == 2, K' = 128) a list holds two ascending runs of
    // 64, each the best of one piece of the scan order: they are merged into
    // one ascending list, and `cap`, the smaller of the run ends, bounds every
    // reference a run left out (a run that is not full left none out).
    uint64_t cap = kEmpty;
    auto sort_runs = [&](uint64_t(&v)[EL]) __attribute__((always_inline)) {
      if constexpr (EL == 2) {
        if (a.runs == 2) {
          cap = umin64(cap, umin64(shfl64(v[0], 63), shfl64(v[1], 63)));
          v[1] = shfl_xor64(v[1], 63);  // run 1 descending: the pair is bitonic
          bitonic_merge<2>(v, lane);
        }
      }
    };
    uint64_t list[EL];
#pragma unroll
    for (int r = 0; r < EL; ++r) {
      const int e = r * 64 + lane;
      list[r] = e < KP ? src[e] : kEmpty;
    }
    sort_runs(list);
    for (int s = 1; s < nlists; ++s) {
      uint64_t other[EL];
#pragma unroll
      for (int r = 0; r < EL; ++r) {
        const int e = r * 64 + lane;
        other[r] = e < KP ? src[(int64_t)s * KP + e] : kEmpty;
      }
      sort_runs(other);
      merge_lists<EL>(list, other, lane);
    }
#pragma unroll
    for (int r = 0; r < EL; ++r) {
      const int e = r * 64 + lane;
      uint64_t v = list[r];
      if (a.perm && v != kEmpty)
        v = (v & 0xffffffff00000000ull) | (uint32_t)a.perm[index_of(v)];
      if (e < KP) sl[wave][e] = v;
    }
    wave_lds_sync();

    const int k = a.k;
    const float* qrow = a.xq + qi * a.d;
    int done = 0;
    int m = a.no_recheck ? k : (k + 8 < KP ? k + 8 : KP);
    bool ok = false;
    int rank[EL];
    while (true) {
      for (int c0 = done; c0 < m; c0 += 64)
        measure(a, qrow, sl[wave], sd2[wave], c0, c0 + 64 < m ? c0 + 64 : m, lane);
      done = m;
      wave_lds_sync();
      // Rank of each measured candidate under (D^2, j); tau = rank k-1.
#pragma unroll
      for (int r = 0; r < EL; ++r) {
        const int c = r * 64 + lane;
        int cr = -1;
        if (c < m) {
          if (a.no_recheck) {
            cr = c;  // debug: keep the filter's order
          } else {
            const double mine = sd2[wave][c];
            const uint32_t mj = index_of(sl[wave][c]);
            cr = 0;
            for (int c2 = 0; c2 < m; ++c2) {
              const double o = sd2[wave][c2];
              cr += (o < mine || (o == mine && index_of(sl[wave][c2]) < mj)) ? 1 : 0;
            }
          }
          if (cr == k - 1) stau[wave] = sd2[wave][c];
        }
        rank[r] = cr;
      }
      wave_lds_sync();
      if (a.no_recheck) {
        ok = true;
        break;
      }
      // Every reference outside the first m candidates has a key >= h.
      const uint64_t hent = umin64(m < KP ? sl[wave][m] : sl[wave][KP - 1], cap);
      ok = certified(cc, ni, rho_i, hent, stau[wave]);
      if (ok || m >= KP) break;
      m = m + 16 < KP ? m + 16 : KP;
    }
    if (a.force_fallback && !a.no_recheck) ok = false;
    if (ok) {
#pragma unroll
      for (int r = 0; r < EL; ++r) {
        const int c = r * 64 + lane;
        if (c < m && rank[r] >= 0 && rank[r] < k)
          emit(a, qi, rank[r], index_of(sl[wave][c]), sd2[wave][c]);
      }
    } else if (lane == 0) {
      const uint32_t w = atomicAdd(&a.ctrl->worklist_count, 1u);
      a.worklist[w] = (int32_t)qi;
      a.fbtau[w] = stau[wave];
    }
    wave_lds_sync();  // the next query reuses this wave's LDS rows
  }
}

// Recheck of short lists over short rows: one lane per candidate.
//
// With K' <= 32 entries and rows of at most 64 elements (a multiple of four),
// a wave takes 64 / K' queries at once, K' lanes each, and lane g of a
// query's group measures the query's g-th candidate alone.  Its exact D^2 is
// then the definition's own sum: fp64, columns in order, no fused
// multiply-add.  All K' candidates are measured at once, so the certificate
// takes h = the K'-th key, the largest bound the list gives.  (The general
// kernel above stops at the first m whose h certifies; a row it certifies is
// certified here too, and the exact k nearest are the same.)  The group's
// (D^2, j) pairs are sorted by a bitonic network across its lanes, after
// which lane r of the group holds rank r.
// Value of v in lane (lane ^ m) for m in {1, 2, 4, 8, 16}: DPP quad
// permutations for 1 and 2, a bit-mask swizzle (within 32 lanes) otherwise;
// neither goes through LDS memory.
__device__ __forceinline__ uint32_t lane_xor(uint32_t v, int m) {
  switch (m) {
    case 1: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);
    case 2: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);
    case 4: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x1F | (4 << 10));
    case 8: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x1F | (8 << 10));
    default: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x1F | (16 << 10));
  }
}
__device__ __forceinline__ uint64_t lane_xor64(uint64_t v, int m) {
  return ((uint64_t)lane_xor((uint32_t)(v >> 32), m) << 32) | lane_xor((uint32_t)v, m);
}

// DC: the most 16-byte chunks of a row (d <= 4 DC).
template <int KP, int W, int DC>
__global__ void __launch_bounds__(W * 64)
    __attribute__((amdgpu_waves_per_eu(DC <= 4 ? 4 : (DC == 8 ? 3 : 2))))
recheck_lanes_kernel(Args a, int64_t q_begin, int64_t q_rows) {
#pragma clang fp contract(off)
  static_assert(KP == 16 || KP == 32, "groups of 16 or 32 lanes");
  constexpr int G = 64 / KP;  // queries per wave
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = lane & (KP - 1), grp = lane / KP, g0 = lane - g;
  if (a.ctrl->nonfinite) return;
  const CertConst cc = cert_const(a);
  const int d = a.d, k = a.k, nch = d >> 2;
  const int64_t step = (int64_t)gridDim.x * W * G;
  // A group past the block's rows repeats the wave's first query and writes
  // nothing.
  auto row_of = [&](int64_t qb) { return qb + grp < q_rows ? qb + grp : qb; };
  // Lists of the row's splits (or of the pieces of a tail-split row).
  auto lists_of = [&](int64_t ql, int& nlists) -> const uint64_t* {
    const bool tl = ql >= a.tail_q0;
    nlists = tl ? a.tail_parts : a.splits;
    return tl ? a.ptail + (ql - a.tail_q0) * a.tail_parts * KP : a.partial + ql * a.splits * KP;
  };
  // A trip's first loads (its list entry, input row, squared norm and radius)
  // are issued one trip ahead; its outputs are written one trip late, after
  // the next trip's loads.  Stores count against the same in-order wait
  // counter as loads, so a store ahead of a load would be waited for with it.
  struct Ahead {
    uint64_t v;
    int64_t qi;
    double ni, rho;
  };
  auto fetch = [&](int64_t qb) __attribute__((always_inline)) {
    const int64_t ql = row_of(qb), qpos = q_begin + ql;
    int nl;
    Ahead x;
    x.v = lists_of(ql, nl)[g];
    x.qi = a.perm ? (int64_t)a.perm[qpos] : qpos;
    x.ni = a.n64_q[qpos];
    x.rho = a.rho_q[qpos];
    return x;
  };
  bool plive = false, pok = false;
  int64_t pqi = 0;
  uint32_t pj = 0;
  uint64_t pdb = 0;
  double ptau = 0.0;
  auto put = [&]() __attribute__((always_inline)) {
    if (!plive) return;
    if (pok) {
      if (g < k) emit(a, pqi, g, pj, __longlong_as_double((long long)pdb));
    } else if (g == 0) {
      const uint32_t w = atomicAdd(&a.ctrl->worklist_count, 1u);
      a.worklist[w] = (int32_t)pqi;
      a.fbtau[w] = ptau;
    }
  };
  int64_t qb = ((int64_t)blockIdx.x * W + wave) * G;
  Ahead cur = {kEmpty, 0, 0.0, 0.0};
  if (qb < q_rows) cur = fetch(qb);
  for (; qb < q_rows; qb += step) {
    Ahead nxt = cur;
    if (qb + step < q_rows) nxt = fetch(qb + step);
    const bool live = qb + grp < q_rows;
    const int64_t qi = cur.qi;
    // Final aggregation of the per-split (or per-piece) lists: lane g holds
    // entry g of the running list; the next list is read reversed, so that
    // the elementwise minimum holds the K' smallest of both as a bitonic
    // sequence, which a bitonic merge sorts.  Groups with fewer lists than
    // the wave's most merge empty ones.
    int nlists;
    const uint64_t* src = lists_of(row_of(qb), nlists);
    uint64_t v = cur.v;
    int nlw = nlists;
#pragma unroll
    for (int off = KP; off < 64; off <<= 1) nlw = max(nlw, __shfl_xor(nlw, off, 64));
    for (int s = 1; s < nlw; ++s) {
      v = umin64(v, s < nlists ? src[(int64_t)s * KP + (KP - 1 - g)] : kEmpty);
#pragma unroll
      for (int st = KP / 2; st > 0; st >>= 1) {
        const uint64_t o = lane_xor64(v, st);
        v = (g & st) ? umax64(v, o) : umin64(v, o);
      }
    }
    // Every reference outside the list has a key >= the K'-th key.
    const uint64_t hent = shfl64(v, g0 + KP - 1);
    // With the grouped scan order the list holds positions: map to rows.
    // (An empty slot measures row 0 and is then set to +inf: the loads stay
    // outside divergent code, and the chunk tests on nch are uniform.)
    const bool empty = v == kEmpty;
    uint32_t j = empty ? 0u : index_of(v);
    if (a.perm) j = (uint32_t)a.perm[j];
    const float4* q4 = reinterpret_cast<const float4*>(a.xq + qi * d);
    const float4* r4 = reinterpret_cast<const float4*>(a.xr + (int64_t)j * d);
    float4 qv[DC], rv[DC];
#pragma unroll
    for (int c = 0; c < DC; ++c)
      if (c < nch) {
        qv[c] = q4[c];
        rv[c] = r4[c];
      }
    put();  // the previous trip's outputs
    double sum = 0.0;
#pragma unroll
    for (int c = 0; c < DC; ++c)
      if (c < nch) sum = add_sq4(sum, qv[c], rv[c]);
    const double d2 = empty ? (double)INFINITY : sum;
    if (empty) j = index_of(kEmpty);
    // Non-negative doubles order as their bit patterns.
    uint64_t db = (uint64_t)__double_as_longlong(d2);
    if (!a.no_recheck) {
#pragma unroll
      for (int size = 2; size <= KP; size <<= 1)
#pragma unroll
        for (int st = size >> 1; st > 0; st >>= 1) {
          const uint64_t pd = lane_xor64(db, st);
          const uint32_t pjx = lane_xor(j, st);
          const bool keep_small = ((g & size) == 0) == ((g & st) == 0);
          const bool mine_less = db < pd || (db == pd && j < pjx);
          if (keep_small != mine_less) {
            db = pd;
            j = pjx;
          }
        }
    }
    // (no_recheck, a debugging switch, keeps the filter's order.)
    const double tau2 = __longlong_as_double((long long)shfl64(db, g0 + k - 1));
    bool ok = a.no_recheck ? true : certified(cc, cur.ni, cur.rho, hent, tau2);
    if (a.force_fallback && !a.no_recheck) ok = false;
    plive = live;
    pok = ok;
    pqi = qi;
    pj = j;
    pdb = db;
    ptau = tau2;
    cur = nxt;
  }
  put();
}

// ---------------------------------------------------------------------------
// Exact fallback (Section 5.2: the rows the verification cannot certify are
// computed again at full precision): a brute-force fp64 scan of every
// reference for the rows in the worklist.  The scan is spread over (row,
// reference chunk) pairs so that a handful of failing rows still fills the
// GPU: with c failing rows each row is cut into P = clamp(kFbGrid / c, 1,
// kFbMaxChunks) chunks.  A chunk keeps its k smallest (D^2, j) in LDS; with
// P == 1 it is the answer, otherwise the P sorted chunk lists go to the
// workspace and fallback_merge_kernel picks the k smallest of them per row.
// ---------------------------------------------------------------------------
constexpr int kFbThreads = 256;
constexpr int kFbSize = 1024;  // sorted best k in [0, k), candidates appended after them
constexpr int kFbSlab = 32;    // columns of the reference rows staged per pass

__device__ __forceinline__ bool lex_less(uint64_t d1, uint32_t j1, uint64_t d2, uint32_t j2) {
  return d1 < d2 || (d1 == d2 && j1 < j2);
}

__device__ __forceinline__ int fb_chunks(uint32_t count) {
  if (count == 0) return 1;
  const uint32_t p = kFbGrid / count;
  return p < 1 ? 1 : (p > (uint32_t)kFbMaxChunks ? kFbMaxChunks : (int)p);
}

// Sort the first n entries (n a power of two, at most kFbSize).
__device__ void fb_sort(uint64_t* kd, uint32_t* kj, int n) {
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < n / 2; i += kFbThreads) {
        const int lo = 2 * stride * (i / stride) + (i % stride);
        const int hi = lo + stride;
        const bool asc = (lo & size) == 0;
        const bool swap = asc ? lex_less(kd[hi], kj[hi], kd[lo], kj[lo])
                              : lex_less(kd[lo], kj[lo], kd[hi], kj[hi]);
        if (swap) {
          const uint64_t td = kd[lo];
          kd[lo] = kd[hi];
          kd[hi] = td;
          const uint32_t tj = kj[lo];
          kj[lo] = kj[hi];
          kj[hi] = tj;
        }
      }
      __syncthreads();
    }
  }
}

__global__ void __launch_bounds__(kFbThreads) fallback_scan_kernel(Args a) {
#pragma clang fp contract(off)
  __shared__ uint64_t kd[kFbSize];
  __shared__ uint32_t kj[kFbSize];
  __shared__ float rows[kFbThreads][kFbSlab + 1];
  __shared__ float qs[kFbSlab];
  __shared__ int bufcnt;
  if (a.ctrl->nonfinite) return;
  const uint32_t count = a.ctrl->worklist_count;
  const int P = fb_chunks(count);
  const int64_t clen = (a.nr + P - 1) / P;
  const int tid = threadIdx.x;
  const int k = a.k, d = a.d;
  for (int64_t pair = blockIdx.x; pair < (int64_t)count * P; pair += gridDim.x) {
    const int64_t w = pair / P;
    const int c = (int)(pair % P);
    const int64_t qi = a.worklist[w];
    const int64_t j0 = (int64_t)c * clen;
    const int64_t j1 = j0 + clen < a.nr ? j0 + clen : a.nr;
    for (int i = tid; i < kFbSize; i += kFbThreads) {
      kd[i] = kEmpty;
      kj[i] = 0xffffffffu;
    }
    if (tid == 0) bufcnt = 0;
    __syncthreads();
    // Only references with D^2 <= tau' can be among the row's k nearest.
    // tau, the k-th smallest of the D^2 the recheck measured for this row,
    // bounds the k-th smallest D^2 over all references; the recheck sums in
    // another order than this scan, and over at most 4096 non-negative terms
    // the two sums differ by less than 2^-40 relative, so tau' = the next
    // double above fl(tau (1 + 2^-30)), more than tau (1 + 2^-31), keeps
    // every one of them.
    const double tau = a.fbtau[w];
    uint64_t thr_d = kEmpty;
    uint32_t thr_j = 0xffffffffu;
    if (tau < INFINITY) {
      const double tp = nextafter(tau * (1.0 + 0x1p-30), INFINITY);
      thr_d = (uint64_t)__double_as_longlong(tp);
    }
    const float* qrow = a.xq + qi * d;
    for (int64_t base = j0; base < j1; base += kFbThreads) {
      // Thread tid measures reference base + tid.  The block's rows are read
      // kFbSlab columns at a time with coalesced loads (lane -> column) and
      // staged in LDS; each thread then adds its row's squared differences in
      // column order, so D^2 is the sequential sum of the definition.
      const int nrow = j1 - base < kFbThreads ? (int)(j1 - base) : kFbThreads;
      const int col = tid & (kFbSlab - 1), row0 = tid / kFbSlab;
      constexpr int kRowStep = kFbThreads / kFbSlab;
      double d2 = 0.0;
      for (int c0 = 0; c0 < d; c0 += kFbSlab) {
        const int wcols = d - c0 < kFbSlab ? d - c0 : kFbSlab;
        // Uniform slab origin plus 32-bit per-lane offsets (< 2^31: at most
        // kFbThreads rows of at most 4096 columns).  Rows past the chunk and
        // columns past the slab are clamped to valid ones; nothing reads them.
        const float* slab = a.xr + base * d + c0;
        const int cc = col < wcols ? col : wcols - 1;
        float v[kFbSlab];
#pragma unroll
        for (int i = 0; i < kFbSlab; ++i) {
          const int r = row0 + i * kRowStep;
          v[i] = slab[(r < nrow ? r : nrow - 1) * d + cc];
        }
        const float qv = (tid < wcols) ? qrow[c0 + tid] : 0.0f;
        __syncthreads();  // the previous slab has been consumed
#pragma unroll
        for (int i = 0; i < kFbSlab; ++i) rows[row0 + i * kRowStep][col] = v[i];
        if (tid < kFbSlab) qs[tid] = qv;
        __syncthreads();
#pragma unroll 8
        for (int t = 0; t < wcols; ++t) {
          const double df = (double)qs[t] - (double)rows[tid][t];
          d2 = d2 + df * df;
        }
      }
      const int64_t j = base + tid;
      if (tid < nrow && !(a.exclude_self && j == qi)) {
        const uint64_t db = (uint64_t)__double_as_longlong(d2);
        if (lex_less(db, (uint32_t)j, thr_d, thr_j)) {
          const int slot = atomicAdd(&bufcnt, 1);
          kd[k + slot] = db;
          kj[k + slot] = (uint32_t)j;
        }
      }
      __syncthreads();
      const bool last = base + kFbThreads >= j1;
      // Merge when another pass could overflow the buffer, and at the end;
      // only the first next_pow2(k + appended) entries are sorted (the rest
      // are empty).
      if (bufcnt > kFbSize - k - kFbThreads || (last && bufcnt > 0)) {
        int n = 2;
        while (n < k + bufcnt) n <<= 1;
        fb_sort(kd, kj, n);
        for (int i = k + tid; i < kFbSize; i += kFbThreads) {
          kd[i] = kEmpty;
          kj[i] = 0xffffffffu;
        }
        if (lex_less(kd[k - 1], kj[k - 1], thr_d, thr_j)) {
          thr_d = kd[k - 1];
          thr_j = kj[k - 1];
        }
        __syncthreads();
        if (tid == 0) bufcnt = 0;
      }
      __syncthreads();
    }
    if (P == 1) {
      if (tid < k) emit(a, qi, tid, kj[tid], __longlong_as_double((long long)kd[tid]));
    } else if (tid < k) {
      uint2* dst = a.fbpart + pair * k + tid;
      const uint64_t e = kd[tid];
      // (D^2 bits, index); an unfilled slot keeps the all-ones sentinel
      dst[0] = make_uint2((uint32_t)(e >> 32), (uint32_t)e);
      a.fbidx[pair * k + tid] = kj[tid];
    }
    __syncthreads();
  }
}

// One wave per worklist row: the k smallest of its P sorted chunk lists, by
// repeatedly taking the smallest list head (ties to the lower index).
__global__ void __launch_bounds__(64) fallback_merge_kernel(Args a) {
  if (a.ctrl->nonfinite) return;
  const uint32_t count = a.ctrl->worklist_count;
  const int P = fb_chunks(count);
  if (P == 1) return;
  const int lane = threadIdx.x;
  const int k = a.k;
  for (int64_t w = blockIdx.x; w < (int64_t)count; w += gridDim.x) {
    const int64_t qi = a.worklist[w];
    int pos = 0;  // next unread entry of this lane's list (lanes >= P hold none)
    auto head = [&](uint64_t& d, uint32_t& j) {
      if (lane < P && pos < k) {
        const int64_t at = (w * P + lane) * k + pos;
        const uint2 v = a.fbpart[at];
        d = ((uint64_t)v.x << 32) | v.y;
        j = a.fbidx[at];
      } else {
        d = kEmpty;
        j = 0xffffffffu;
      }
    };
    uint64_t hd;
    uint32_t hj;
    head(hd, hj);
    for (int r = 0; r < k; ++r) {
      uint64_t bd = hd;
      uint32_t bj = hj;
      int bl = lane;
      for (int off = 32; off > 0; off >>= 1) {
        const uint64_t od = shfl_xor64(bd, off);
        const uint32_t oj = __shfl_xor(bj, off, 64);
        const int ol = __shfl_xor(bl, off, 64);
        if (lex_less(od, oj, bd, bj)) {
          bd = od;
          bj = oj;
          bl = ol;
        }
      }
      if (lane == 0) emit(a, qi, r, bj, __longlong_as_double((long long)bd));
      if (lane == bl) {
        ++pos;
        head(hd, hj);
      }
    }
  }
}

template <int KP>
hipError_t launch_recheck_t(const Args& a, int64_t q_begin, int64_t q_rows, hipStream_t st) {
  constexpr int W = 4;
  if constexpr (KP <= 32) {
    if (a.d <= 64 && (a.d & 3) == 0) {
      constexpr int G = 64 / KP;
      int64_t g = (q_rows + W * G - 1) / (W * G);
      if (g > 4096) g = 4096;
      const auto kern = a.d <= 8    ? recheck_lanes_kernel<KP, W, 2>
                        : a.d <= 16 ? recheck_lanes_kernel<KP, W, 4>
                        : a.d <= 32 ? recheck_lanes_kernel<KP, W, 8>
                                    : recheck_lanes_kernel<KP, W, 16>;
      hipLaunchKernelGGL(kern, dim3((unsigned)g), dim3(W * 64), 0, st, a, q_begin, q_rows);
      return hipGetLastError();
    }
  }
  int64_t g = (q_rows + W - 1) / W;
  if (g > 4096) g = 4096;
  hipLaunchKernelGGL((recheck_kernel<KP, W>), dim3((unsigned)g), dim3(W * 64), 0, st, a, q_begin,
                     q_rows);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tile(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                       hipStream_t st, TileTail* tail) {
  if (p.tile_kind == 1) {
    if (p.precision == TOD_PREC_FP16) return launch_mtile_f16(p, a, q_begin, q_rows, st, tail);
    if (p.precision == TOD_PREC_BF16) return launch_mtile_bf16(p, a, q_begin, q_rows, st, tail);
    return hipErrorInvalidValue;
  }
  switch (p.precision) {
    case TOD_PREC_FP32: return launch_tile_f32(p, a, q_begin, q_rows, st);
    case TOD_PREC_FP16: return launch_tile_f16(p, a, q_begin, q_rows, st);
    case TOD_PREC_BF16: return launch_tile_bf16(p, a, q_begin, q_rows, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_recheck(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                          hipStream_t st) {
  switch (p.kprime) {
    case 16: return launch_recheck_t<16>(a, q_begin, q_rows, st);
    case 32: return launch_recheck_t<32>(a, q_begin, q_rows, st);
    case 64: return launch_recheck_t<64>(a, q_begin, q_rows, st);
    case 128: return launch_recheck_t<128>(a, q_begin, q_rows, st);
    case 256: return launch_recheck_t<256>(a, q_begin, q_rows, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_fallback(const Plan& p, const Args& a, hipStream_t st) {
  hipLaunchKernelGGL(fallback_scan_kernel, dim3(kFbGrid), dim3(kFbThreads), 0, st, a);
  hipLaunchKernelGGL(fallback_merge_kernel, dim3(kFbGrid), dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace tod
