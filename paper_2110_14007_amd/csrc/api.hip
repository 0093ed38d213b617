// Host side of libtod: argument validation, the batching planner, the
// workspace layout and the launch sequence of one call.
//
// One call runs, in stream order:
//   prep       centre, scale, quantise, norms and radii          (Section 5.2 step i)
//   per query block (automatic batching, Section 6):
//     tile     fused distance tile + top-K' per reference split   (Sections 5.2 ii, 6.1)
//     recheck  merge splits, exact recheck, certificate           (Section 5.2 iii)
//   fallback   exact scan of rows that failed the certificate     (Section 5.2 iii)
//   lof        LOF from the exact lists (tod_lof only)            (Table 1)
// then one stream synchronisation to read the status flags back.
#include <math.h>
#include <string.h>

#include <mutex>
#include <string>
#include <vector>

#include "tod_internal.h"

namespace {

thread_local std::string g_last_error;

tod_status fail(tod_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

int64_t next_pow2(int64_t v) {
  int64_t p = 1;
  while (p < v) p <<= 1;
  return p;
}

constexpr int64_t kMaxRows = 0x7fffffffLL;
constexpr int64_t kMaxD = 4096;
constexpr int32_t kMaxK = 256;
constexpr int32_t kMaxKPrime = 256;
// Tail split: at most 8 pieces, and a tail region of at most 2^18 lists.
constexpr int32_t kMaxTailParts = 8;
constexpr int64_t kTailLists = 1 << 18;

tod_status resolve_options(const tod_options* in, tod_options* out) {
  tod_default_options(out);
  if (!in) return TOD_OK;
  if (in->struct_size != sizeof(tod_options))
    return fail(TOD_ERR_INVALID_ARG, "tod_options.struct_size does not match this library");
  *out = *in;
  if (out->precision < TOD_PREC_AUTO || out->precision > TOD_PREC_BF16)
    return fail(TOD_ERR_INVALID_ARG, "unknown precision");
  if (out->shortlist < 0 || out->shortlist > kMaxKPrime)
    return fail(TOD_ERR_INVALID_ARG, "shortlist must be in [0, 256]");
  if (out->query_block < 0) return fail(TOD_ERR_INVALID_ARG, "query_block must be >= 0");
  if (out->ref_splits < 0 || out->ref_splits > 64)
    return fail(TOD_ERR_INVALID_ARG, "ref_splits must be in [0, 64]");
  if (out->margin_scale == 0.0f) out->margin_scale = 1.0f;
  if (!(out->margin_scale >= 1.0f) || isinf(out->margin_scale))
    return fail(TOD_ERR_INVALID_ARG, "margin_scale must be a finite value >= 1");
  if (out->reorder < -1 || out->reorder > 1)
    return fail(TOD_ERR_INVALID_ARG, "reorder must be -1, 0 or 1");
  if (out->score < TOD_SCORE_KTH || out->score > TOD_SCORE_SUM)
    return fail(TOD_ERR_INVALID_ARG, "unknown score");
  if (out->tail_parts < 0 || out->tail_parts > kMaxTailParts)
    return fail(TOD_ERR_INVALID_ARG, "tail_parts must be in [0, 8]");
  return TOD_OK;
}

tod_status check_sizes(int64_t nq, int64_t nr, int64_t d, int32_t k, int32_t excl) {
  if (nq <= 0 || nr <= 0) return fail(TOD_ERR_INVALID_ARG, "row counts must be positive");
  if (d <= 0) return fail(TOD_ERR_INVALID_ARG, "d must be positive");
  if (k <= 0) return fail(TOD_ERR_INVALID_ARG, "k must be positive");
  if (nq > kMaxRows || nr > kMaxRows)
    return fail(TOD_ERR_UNSUPPORTED, "more than 2^31 - 1 rows");
  if (d > kMaxD) return fail(TOD_ERR_UNSUPPORTED, "d > 4096");
  if (k > kMaxK) return fail(TOD_ERR_UNSUPPORTED, "k > 256");
  if ((int64_t)k > nr - (excl ? 1 : 0))
    return fail(TOD_ERR_INVALID_ARG, "k exceeds the number of candidate references");
  return TOD_OK;
}

}  // namespace

namespace tod {

// Reference splits for a query block of qb rows (Section 6 customised cdist
// batching): enough waves for two per SIMD on 256 CUs x 4 SIMDs, but at
// least 2048 references per split (every split keeps its own K' list per
// query, so splits cost selection work), and at most 16.
int64_t auto_splits(int64_t qb, int64_t nr) {
  const int64_t waves = (qb + 31) / 32;
  int64_t s = (2048 + waves - 1) / waves;
  const int64_t cap = nr / 2048 > 1 ? nr / 2048 : 1;
  if (s > cap) s = cap;
  if (s > 16) s = 16;
  return s < 1 ? 1 : s;
}

// S splits of 32-row multiples (fewer if the rounding leaves some empty).
void set_splits(Plan* p, int64_t s) {
  if (s < 1) s = 1;
  const int64_t len = round_up((p->nr + s - 1) / s, 32);
  p->splits = (int32_t)((p->nr + len - 1) / len);
  p->split_len = len;
}

tod_status make_plan(int64_t nq, int64_t nr, int64_t d, int32_t k, int32_t lof, int32_t self,
                     const tod_options& o, Plan* p, const char** why) {
  *why = "";
  memset(p, 0, sizeof(*p));
  p->nq = nq;
  p->nr = nr;
  p->d = d;
  p->k = k;
  p->lof = lof;
  p->lists = (lof || o.score != TOD_SCORE_KTH) ? 1 : 0;
  p->self = self;
  p->exclude_self = o.exclude_self ? 1 : 0;
  // Filter precision (provable quantization, Section 5.2 step ii).  The fp16
  // MFMA filter: with power-of-two scaling its 11-bit mantissa gives the
  // certificate the smallest margin of the MFMA types, hence the shortest
  // shortlist (bf16 needs about twice as many candidates at the same speed).
  int32_t prec = o.precision;
  if (prec == TOD_PREC_AUTO) prec = TOD_PREC_FP16;
  p->precision = prec;
  // Shortlist length K': a power of two >= k with room for the certificate's
  // margin.  The margin a row needs grows with the filter's rounding error:
  // k + 4 at fp32, k + max(8, k/4) at fp16, k + max(24, k) at bf16 (bf16's
  // 8-bit significand leaves about one row in ten uncertified at 2k when k is
  // small).
  int64_t kp;
  if (o.shortlist > 0) {
    kp = o.shortlist;
  } else if (prec == TOD_PREC_FP32) {
    kp = k + 4;
  } else if (prec == TOD_PREC_FP16) {
    kp = k + (k / 4 > 8 ? (k + 3) / 4 : 8);
  } else {
    kp = k + (k > 24 ? k : 24);
  }
  if (kp < k) kp = k;
  kp = next_pow2(kp < 16 ? 16 : kp);
  if (kp > kMaxKPrime) kp = kMaxKPrime;
  p->kprime = (int32_t)kp;
  // Row stride of the quantised copies.  Small rows are padded to a power of
  // two so that the tile kernel can keep the query operand in registers.
  if (prec == TOD_PREC_FP32) {
    const int64_t dp = round_up(d, 4);
    p->dpad_t = dp <= 64 ? (int32_t)next_pow2(dp < 8 ? 8 : dp) : 0;
    p->dpad = p->dpad_t ? p->dpad_t : (int32_t)dp;
  } else {
    const int64_t dp = round_up(d, 16);
    p->dpad_t = dp <= 512 ? (int32_t)next_pow2(dp) : 0;
    p->dpad = p->dpad_t ? p->dpad_t : (int32_t)dp;
  }
  p->scale_exp = 14;
  p->esize = prec == TOD_PREC_FP32 ? 4 : 2;
  p->nq_pad = round_up(nq, 32);
  p->nr_pad = round_up(nr, 32);
  // Query blocks (Section 6 direct batching along samples).
  int64_t qb = o.query_block > 0 ? round_up(o.query_block, 32) : p->nq_pad;
  if (qb > p->nq_pad) qb = p->nq_pad;
  p->query_block = qb;
  p->blocks = (nq + qb - 1) / qb;
  set_splits(p, o.ref_splits > 0 ? o.ref_splits : auto_splits(qb, nr));
  p->waves_per_group = kp <= 32 ? 4 : (kp == 64 ? 2 : 1);
  // The register-list MFMA kernel covers fp16 / bf16 filters whose query
  // operand fits in registers and whose shortlist is 16, 32 or 64 long.  Rows
  // of at most 8 elements carry the accumulator seed -N_j/2 in their padding
  // (columns 8..11 of a 16-wide row); longer rows get it from LDS.
  p->tile_kind = (prec != TOD_PREC_FP32 && d <= 512 && kp <= 64) ? 1 : 0;
  // K' = 128 on rows of 256 or more elements (bf16 at k of 33..64): the
  // register-list kernel with 64-entry lists over two pieces of the scan
  // order.  Every reference a piece left out has a key >= that piece's 64th,
  // so the recheck bounds the excluded references by the smaller of the two
  // run ends.  (A 128-entry register list beside the 128-register query
  // operand leaves the compiler too few registers: it spills the operand to
  // scratch memory.)
  p->runs = 1;
  if (prec != TOD_PREC_FP32 && d <= 512 && kp == 128 && p->dpad_t >= 256) {
    p->tile_kind = 1;
    p->runs = 2;
  }
  if (p->tile_kind == 1) {
    p->waves_per_group = 4;
    if (d <= 8) {
      p->fold = 1;
      p->dmain = 8;
      p->dpad = p->dpad_t = 16;
      // fp16: |seed part| <= 8 2^(2E) / 2 / 2^15 must stay below 2^15.
      if (prec == TOD_PREC_FP16) p->scale_exp = 14;
    } else {
      // Longer rows: the seed -N_j/2 is the product of four parts of
      // -N_j/(2c) (staged beside the rows, 8 bytes a row) with c, one MFMA
      // per sub-tile, instead of 16 fp32 seeds read from LDS by every lane.
      // fp16 parts: N_j / 2^16 <= d 2^(2E - 16) must stay below 2^15, i.e.
      // d 2^(2E) <= 2^31.
      p->seedprod = 1;
      if (prec == TOD_PREC_FP16) {
        int lg = 0;
        while ((int64_t)1 << lg < d) ++lg;
        const int e = (31 - lg) / 2;
        p->scale_exp = e < 14 ? e : 14;
      }
    }
  }
  // Grouped scan order: X against X through the register-list kernel with one
  // reference split (each workgroup then scans the whole set from its own
  // group on); by default from kOrderMinRows references on.
  const bool want = o.reorder > 0 || (o.reorder == 0 && nr >= kOrderMinRows);
  // (With runs, the tile scans the whole set in pieces whatever S is.)
  p->order = (self && p->tile_kind == 1 && (p->splits == 1 || p->runs > 1) && want) ? 1 : 0;
  p->groups = order_groups(nr, d);
  // Tail split of the register-list tile with one reference split (not with
  // runs: their pieces already halve every workgroup's scan).
  p->tail_parts = 1;
  p->tail_auto = 0;
  p->tail_lists = 0;
  if (p->tile_kind == 1 && p->splits == 1 && p->runs == 1 && o.tail_parts != 1) {
    p->tail_parts = o.tail_parts == 0 ? kMaxTailParts : o.tail_parts;
    p->tail_auto = o.tail_parts == 0 ? 1 : 0;
    const int64_t want_lists = p->query_block * p->tail_parts;
    p->tail_lists = want_lists < kTailLists ? want_lists : kTailLists;
  }
  return TOD_OK;
}

Layout make_layout(const Plan& p) {
  Layout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += (bytes + 255) / 256 * 256;
    return at;
  };
  L.colpart_blocks = colsum_blocks(p.nr);
  L.ctrl = take(sizeof(Ctrl));
  L.mu64 = take(sizeof(double) * p.d);
  L.mu32 = take(sizeof(float) * p.d);
  L.colpart = take(sizeof(double) * p.d * L.colpart_blocks);
  L.xq_r = take((size_t)p.nr_pad * p.dpad * p.esize);
  L.xq_q = p.self ? L.xq_r : take((size_t)p.nq_pad * p.dpad * p.esize);
  L.hn_r = take((p.seedprod ? 8 : sizeof(float)) * p.nr_pad);
  L.n64_q = take(sizeof(double) * (p.self ? p.nr_pad : p.nq_pad));
  L.rho_q = take(sizeof(double) * (p.self ? p.nr_pad : p.nq_pad));
  L.partial = take(sizeof(uint64_t) * p.query_block * p.splits * p.kprime);
  L.ptail = take(sizeof(uint64_t) * p.tail_lists * p.kprime);
  L.worklist = take(sizeof(int32_t) * p.nq);
  L.fbtau = take(sizeof(double) * p.nq);
  // Chunk lists exist only when fewer than kFbGrid rows fail, so kFbGrid
  // lists of k entries always suffice.
  L.fbpart = take(sizeof(uint2) * (size_t)tod::kFbGrid * p.k);
  L.fbidx = take(sizeof(uint32_t) * (size_t)tod::kFbGrid * p.k);
  if (p.order) {
    const int32_t nb = order_blocks(p.nr);
    L.perm = take(sizeof(int32_t) * p.nr_pad);
    L.lab = take(sizeof(int32_t) * p.nr);
    L.oseed = take(sizeof(float) * 16 * (size_t)p.groups);
    L.cstart = take(sizeof(int32_t) * (size_t)(p.groups + 1));
    L.bcnt = take(sizeof(int32_t) * (size_t)nb * p.groups);
    L.boff = take(sizeof(int32_t) * (size_t)nb * p.groups);
  } else {
    L.perm = L.lab = L.oseed = L.cstart = L.bcnt = L.boff = 0;
  }
  if (p.lists) {
    L.idx32 = take(sizeof(int32_t) * p.nq * p.k);
    L.d64 = take(sizeof(double) * p.nq * p.k);
  } else {
    L.idx32 = L.d64 = 0;
  }
  L.lrd = p.lof ? take(sizeof(double) * p.nq) : 0;
  L.kdist = p.lof ? take(sizeof(double) * p.nq) : 0;
  L.total = off;
  return L;
}

// Automatic batching sized to the caller's memory (Section 6): when the
// workspace is smaller than the plan's layout, the tail split's region is
// dropped first; if that is not enough, the query block shrinks to
// what the room left beside the fixed buffers holds (partial lists of
// S x K' entries per query row), the reference splits follow the smaller
// block (and shrink too if the room demands it).  Fails only when not even
// one 32-row block fits, or when the caller fixed the query block or the
// splits.
tod_status fit_plan(Plan* p, size_t ws_bytes, const tod_options& o, std::string* why) {
  if (o.query_block > 0 || o.ref_splits > 0) {
    *why = "the query block or the reference splits were fixed by the caller";
    return TOD_ERR_WORKSPACE;
  }
  // The tail split's lists go first: the same blocks without it.
  Plan q = *p;
  q.tail_parts = 1;
  q.tail_auto = 0;
  q.tail_lists = 0;
  if (make_layout(q).total <= ws_bytes) {
    *p = q;
    return TOD_OK;
  }
  // The grouped scan order needs buffers of its own and applies only with one
  // split; a shrunken plan may end up with one split where the one-block plan
  // had several.  The order's buffers are therefore reserved first (where the
  // order could apply), and left out only when the block does not fit beside
  // them: the order is an optimisation, the block is not.
  const size_t per = (size_t)q.kprime * sizeof(uint64_t);  // partial-list bytes per row and split
  const bool want = o.reorder > 0 || (o.reorder == 0 && q.nr >= kOrderMinRows);
  const bool may_order = q.self && q.tile_kind == 1 && want;
  size_t need = 0;
  for (int with_order = may_order ? 1 : 0; with_order >= 0; --with_order) {
    Plan f = q;
    f.query_block = 0;  // no partial lists: the fixed part of the layout
    f.order = with_order;
    const size_t fixed = make_layout(f).total;
    need = fixed + 32 * per + 256;
    if (ws_bytes < need) continue;
    const size_t room = ws_bytes - fixed - 256;  // the partial region's alignment slack
    int64_t qb = (int64_t)(room / per) / 32 * 32;
    if (qb > f.nq_pad) qb = f.nq_pad;
    int64_t s = auto_splits(qb, f.nr);
    const int64_t smax = (int64_t)(room / ((size_t)qb * per));
    if (s > smax) s = smax;
    f.query_block = qb;
    f.blocks = (f.nq + qb - 1) / qb;
    set_splits(&f, s);
    f.order = (with_order && (f.splits == 1 || f.runs > 1)) ? 1 : 0;
    if (make_layout(f).total > ws_bytes) {
      *why = "internal: the fitted plan does not fit";
      return TOD_ERR_INTERNAL;
    }
    *p = f;
    return TOD_OK;
  }
  *why = "not even one 32-row query block fits: need at least " + std::to_string(need) + " bytes";
  return TOD_ERR_WORKSPACE;
}

// Neighbours within range: the fp16 / bf16 MFMA range tile (rtile.h) over
// rows padded to a power of two of at least 16 elements, reference splits by
// the kNN rule, no query blocks of its own (the batches follow from the
// candidate counts and the workspace, see tod_nwr).
tod_status make_plan_nwr(int64_t nq, int64_t nr, int64_t d, int32_t self, const tod_options& o,
                         Plan* p, const char** why) {
  *why = "";
  memset(p, 0, sizeof(*p));
  p->nq = nq;
  p->nr = nr;
  p->d = d;
  p->self = self;
  p->exclude_self = o.exclude_self ? 1 : 0;
  int32_t prec = o.precision == TOD_PREC_AUTO ? TOD_PREC_FP16 : o.precision;
  if (prec == TOD_PREC_FP32) {
    *why = "tod_nwr filters in fp16 or bf16 (MFMA); fp32 is not offered";
    return TOD_ERR_UNSUPPORTED;
  }
  if (d > 512) {
    *why = "tod_nwr supports rows of at most 512 elements";
    return TOD_ERR_UNSUPPORTED;
  }
  p->precision = prec;
  p->dpad = p->dpad_t = (int32_t)next_pow2(round_up(d, 16));
  p->esize = 2;
  p->scale_exp = 14;
  p->nq_pad = round_up(nq, 32);
  p->nr_pad = round_up(nr, 32);
  p->query_block = p->nq_pad;
  p->blocks = 1;
  set_splits(p, o.ref_splits > 0 ? o.ref_splits : auto_splits(p->nq_pad, nr));
  p->waves_per_group = 4;
  p->tile_kind = 2;
  return TOD_OK;
}

NwrLayout make_layout_nwr(const Plan& p) {
  NwrLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += (bytes + 255) / 256 * 256;
    return at;
  };
  L.colpart_blocks = colsum_blocks(p.nr);
  L.groups = p.nq_pad / 32;
  const int64_t nc = p.nq * p.splits;
  L.ctrl = take(sizeof(Ctrl));
  L.mu64 = take(sizeof(double) * p.d);
  L.mu32 = take(sizeof(float) * p.d);
  L.colpart = take(sizeof(double) * p.d * L.colpart_blocks);
  L.xq_r = take((size_t)p.nr_pad * p.dpad * p.esize);
  L.xq_q = p.self ? L.xq_r : take((size_t)p.nq_pad * p.dpad * p.esize);
  L.hn_r = take(sizeof(float) * p.nr_pad);
  L.n64_q = take(sizeof(double) * (p.self ? p.nr_pad : p.nq_pad));
  L.rho_q = take(sizeof(double) * (p.self ? p.nr_pad : p.nq_pad));
  L.rho_r = p.self ? L.rho_q : take(sizeof(double) * p.nr_pad);
  L.ccount = take(sizeof(int32_t) * p.nq_pad * p.splits);
  L.coff = take(sizeof(int64_t) * (nc + 1));
  const int64_t parts = scan_parts(nc > p.nq ? nc : p.nq);
  L.part = take(sizeof(int64_t) * parts);
  L.goff = take(sizeof(int64_t) * (L.groups + 1));
  L.incnt = take(sizeof(int32_t) * p.nq);
  L.cand = off;
  return L;
}

int64_t nwr_candidate_room(const NwrLayout& L, size_t ws_bytes) {
  if (ws_bytes < L.cand + 512) return 0;
  // ids (4 B) and distances (4 B), each region 256-aligned
  return (int64_t)((ws_bytes - L.cand - 512) / 8);
}

}  // namespace tod

namespace {

using tod::Args;
using tod::Layout;
using tod::Plan;

struct Timers {
  bool on = false;
  std::vector<hipEvent_t> ev;
  hipEvent_t mark(hipStream_t st) {
    if (!on) return nullptr;
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    (void)hipEventRecord(e, st);
    ev.push_back(e);
    return e;
  }
  static float ms(hipEvent_t a, hipEvent_t b) {
    float t = 0.0f;
    if (a && b && hipEventElapsedTime(&t, a, b) == hipSuccess) return t;
    return 0.0f;
  }
  ~Timers() {
    for (hipEvent_t e : ev) (void)hipEventDestroy(e);
  }
};

tod_status hip_fail(hipError_t e, const char* where) {
  return fail(TOD_ERR_HIP, std::string(where) + ": " + hipGetErrorString(e));
}

// mode: 0 kNN lists / scores, 1 LOF, 2 classifier, 3 ABOD, 4 COF.
tod_status run(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d, int32_t k,
               const tod_options* opts_in, int32_t force_excl, int32_t mode, void* ws,
               size_t ws_bytes, void* stream, int64_t* idx_out, float* dist_out,
               float* score_out, float* lof_out, const int32_t* labels_r, int32_t n_classes,
               int32_t* pred_out, tod_stats* stats, bool events = true) {
  g_last_error.clear();
  const int32_t lof = (mode == 1 || mode == 4) ? 1 : 0;  // COF uses LOF's buffers
  tod_options o;
  tod_status st = resolve_options(opts_in, &o);
  if (st != TOD_OK) return st;
  if (force_excl) o.exclude_self = 1;
  if (stats && stats->struct_size != sizeof(tod_stats))
    return fail(TOD_ERR_INVALID_ARG, "tod_stats.struct_size does not match this library");
  if (!xq || !xr) return fail(TOD_ERR_INVALID_ARG, "null input pointer");
  if (!ws) return fail(TOD_ERR_INVALID_ARG, "null workspace");
  st = check_sizes(nq, nr, d, k, o.exclude_self);
  if (st != TOD_OK) return st;
  const int32_t self = (xq == xr && nq == nr) ? 1 : 0;
  if (o.exclude_self && !self)
    return fail(TOD_ERR_INVALID_ARG, "exclude_self requires the query set to be the reference set");
  if (((uintptr_t)xq | (uintptr_t)xr) & 15)
    return fail(TOD_ERR_INVALID_ARG, "input pointers must be 16-byte aligned");
  if ((uintptr_t)ws & 255) return fail(TOD_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  Plan p;
  const char* why = "";
  st = tod::make_plan(nq, nr, d, k, lof, self, o, &p, &why);
  if (st != TOD_OK) return fail(st, why);
  if (mode >= 2) p.lists = 1;
  Layout L = tod::make_layout(p);
  if (ws_bytes < L.total) {
    std::string w;
    st = tod::fit_plan(&p, ws_bytes, o, &w);
    if (st != TOD_OK)
      return fail(st, "workspace of " + std::to_string(ws_bytes) + " bytes too small (" + w +
                          "; the one-block plan needs " + std::to_string(L.total) + ")");
    L = tod::make_layout(p);
  }
  char* base = (char*)ws;
  Args a;
  memset(&a, 0, sizeof(a));
  a.xq = xq;
  a.xr = xr;
  a.nq = nq;
  a.nr = nr;
  a.d = (int32_t)d;
  a.dpad = p.dpad;
  a.k = k;
  a.kprime = p.kprime;
  a.splits = p.splits;
  a.split_len = p.split_len;
  a.exclude_self = p.exclude_self;
  a.precision = p.precision;
  a.margin_scale = o.margin_scale;
  a.force_fallback = o.force_fallback ? 1 : 0;
  a.fold = p.fold;
  a.seedprod = p.seedprod;
  a.dmain = p.dmain;
  a.scale_exp = p.scale_exp;
  a.no_recheck = o.no_recheck ? 1 : 0;
  a.ctrl = (tod::Ctrl*)(base + L.ctrl);
  a.mu64 = (double*)(base + L.mu64);
  a.mu32 = (float*)(base + L.mu32);
  a.colpart = (double*)(base + L.colpart);
  a.xq_r = base + L.xq_r;
  a.xq_q = base + L.xq_q;
  a.hn_r = (float*)(base + L.hn_r);
  a.n64_q = (double*)(base + L.n64_q);
  a.rho_q = (double*)(base + L.rho_q);
  a.partial = (uint64_t*)(base + L.partial);
  a.parts = 1;
  a.runs = p.runs;
  a.tail_parts = 1;
  a.tail_q0 = p.nq;
  a.ptail = p.tail_lists ? (uint64_t*)(base + L.ptail) : nullptr;
  a.worklist = (int32_t*)(base + L.worklist);
  a.fbtau = (double*)(base + L.fbtau);
  a.fbpart = (uint2*)(base + L.fbpart);
  a.fbidx = (uint32_t*)(base + L.fbidx);
  a.perm = p.order ? (int32_t*)(base + L.perm) : nullptr;
  a.lab = p.order ? (int32_t*)(base + L.lab) : nullptr;
  a.groups = p.groups;
  a.oseed = p.order ? (float*)(base + L.oseed) : nullptr;
  a.cstart = p.order ? (int32_t*)(base + L.cstart) : nullptr;
  a.bcnt = p.order ? (int32_t*)(base + L.bcnt) : nullptr;
  a.boff = p.order ? (int32_t*)(base + L.boff) : nullptr;
  a.idx32 = p.lists ? (int32_t*)(base + L.idx32) : nullptr;
  a.d64 = p.lists ? (double*)(base + L.d64) : nullptr;
  a.lrd = lof ? (double*)(base + L.lrd) : nullptr;
  a.kdist = lof ? (double*)(base + L.kdist) : nullptr;
  a.score = o.score;
  a.labels_r = labels_r;
  a.n_classes = n_classes;
  a.pred_out = pred_out;
  a.idx_out = idx_out;
  a.dist_out = dist_out;
  a.score_out = score_out;
  a.lof_out = lof_out;

  hipStream_t s = (hipStream_t)stream;
  Timers tm;
  tm.on = stats != nullptr && events;
  hipEvent_t e0 = tm.mark(s);
  hipError_t he = tod::launch_prep(p, a, s);
  if (he != hipSuccess) return hip_fail(he, "prep launch");
  hipEvent_t e_prep = tm.mark(s);
  std::vector<std::pair<hipEvent_t, hipEvent_t>> tile_ev;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> rc_ev;
  int32_t tail_parts = 1;
  int64_t tail_rows = 0, launches = 0;
  for (int64_t b = 0; b < p.blocks; ++b) {
    const int64_t q0 = b * p.query_block;
    const int64_t rows = nq - q0 < p.query_block ? nq - q0 : p.query_block;
    hipEvent_t ts = tm.mark(s);
    tod::TileTail tt{rows, 1};
    he = tod::launch_tile(p, a, q0, rows, s, &tt);
    if (he != hipSuccess) return hip_fail(he, "tile launch");
    hipEvent_t te = tm.mark(s);
    tod::Args ar = a;
    ar.tail_q0 = tt.q0;
    ar.tail_parts = tt.parts;
    launches += (tt.q0 > 0 ? 1 : 0) + (tt.parts > 1 ? 1 : 0);
    if (tt.parts > 1) {
      tail_parts = tt.parts > tail_parts ? tt.parts : tail_parts;
      tail_rows += rows - tt.q0;
    }
    he = tod::launch_recheck(p, ar, q0, rows, s);
    if (he != hipSuccess) return hip_fail(he, "recheck launch");
    hipEvent_t re = tm.mark(s);
    if (tm.on) {
      tile_ev.emplace_back(ts, te);
      rc_ev.emplace_back(te, re);
    }
  }
  hipEvent_t e_rc = tm.mark(s);
  he = tod::launch_fallback(p, a, s);
  if (he != hipSuccess) return hip_fail(he, "fallback launch");
  hipEvent_t e_fb = tm.mark(s);
  if (mode == 1) {
    he = tod::launch_lof(p, a, s);
    if (he != hipSuccess) return hip_fail(he, "lof launch");
  }
  if (mode == 4) {
    he = tod::launch_cof(p, a, s);
    if (he != hipSuccess) return hip_fail(he, "cof launch");
  }
  if (score_out && o.score != TOD_SCORE_KTH && mode != 3) {
    he = tod::launch_score(p, a, s);
    if (he != hipSuccess) return hip_fail(he, "score launch");
  }
  if (mode == 2) {
    he = tod::launch_vote(p, a, s);
    if (he != hipSuccess) return hip_fail(he, "vote launch");
  }
  if (mode == 3) {
    he = tod::launch_abod(p, a, s);
    if (he != hipSuccess) return hip_fail(he, "abod launch");
  }
  hipEvent_t e_end = tm.mark(s);
  tod::Ctrl host;
  he = hipMemcpyAsync(&host, a.ctrl, sizeof(host), hipMemcpyDeviceToHost, s);
  if (he != hipSuccess) return hip_fail(he, "status readback");
  he = hipStreamSynchronize(s);
  if (he != hipSuccess) return hip_fail(he, "stream synchronize");
  if (stats) {
    stats->precision = p.precision;
    stats->kprime = p.kprime;
    stats->ref_splits = p.splits;
    stats->query_block = p.query_block;
    stats->blocks = p.blocks;
    // Every query row is either certified or on the worklist.
    stats->rows_certified = p.nq - (int64_t)host.worklist_count;
    stats->rows_fallback = (int64_t)host.worklist_count;
    stats->tile_launches = launches;
    stats->reordered = p.order;
    stats->pairs_candidate = stats->pairs_uncertain = stats->pairs_in_range = 0;
    stats->tail_parts = tail_parts;
    stats->tail_rows = tail_rows;
    stats->list_runs = p.runs;
    stats->ms_prep = Timers::ms(e0, e_prep);
    float t = 0.0f, r = 0.0f;
    for (auto& pr : tile_ev) t += Timers::ms(pr.first, pr.second);
    for (auto& pr : rc_ev) r += Timers::ms(pr.first, pr.second);
    stats->ms_tile = t;
    stats->ms_recheck = r;
    stats->ms_fallback = Timers::ms(e_rc, e_fb);
    stats->ms_score = Timers::ms(e_fb, e_end);
    stats->ms_total = Timers::ms(e0, e_end);
  }
  if (host.nonfinite) return fail(TOD_ERR_NONFINITE, "input contains NaN or Inf");
  if (host.bad_label) return fail(TOD_ERR_INVALID_ARG, "a reference label is outside [0, n_classes)");
  return TOD_OK;
}

tod_status run_nwr(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d,
                   double phi, const tod_options* opts_in, void* ws, size_t ws_bytes,
                   void* stream, int64_t* row_ptr_out, int64_t capacity, int64_t* idx_out,
                   float* dist_out, int64_t* total_out, tod_stats* stats,
                   const double* phi2_row = nullptr) {
  // phi2_row: a squared radius per query row (device, finite, >= 0) in place
  // of phi (LOF on tie-inclusive neighbourhoods).
  g_last_error.clear();
  tod_options o;
  tod_status st = resolve_options(opts_in, &o);
  if (st != TOD_OK) return st;
  if (stats && stats->struct_size != sizeof(tod_stats))
    return fail(TOD_ERR_INVALID_ARG, "tod_stats.struct_size does not match this library");
  if (!xq || !xr) return fail(TOD_ERR_INVALID_ARG, "null input pointer");
  if (!row_ptr_out) return fail(TOD_ERR_INVALID_ARG, "null row_ptr output");
  if (!ws) return fail(TOD_ERR_INVALID_ARG, "null workspace");
  if (phi2_row) phi = 0.0;
  if (!(phi >= 0.0) || isinf(phi)) return fail(TOD_ERR_INVALID_ARG, "phi must be finite and >= 0");
  if (idx_out && capacity < 0) return fail(TOD_ERR_INVALID_ARG, "capacity must be >= 0");
  if (dist_out && !idx_out) return fail(TOD_ERR_INVALID_ARG, "dist_out needs idx_out");
  if (nq <= 0 || nr <= 0) return fail(TOD_ERR_INVALID_ARG, "row counts must be positive");
  if (d <= 0) return fail(TOD_ERR_INVALID_ARG, "d must be positive");
  if (nq > kMaxRows || nr > kMaxRows) return fail(TOD_ERR_UNSUPPORTED, "more than 2^31 - 1 rows");
  const int32_t self = (xq == xr && nq == nr) ? 1 : 0;
  if (o.exclude_self && !self)
    return fail(TOD_ERR_INVALID_ARG, "exclude_self requires the query set to be the reference set");
  if (((uintptr_t)xq | (uintptr_t)xr) & 15)
    return fail(TOD_ERR_INVALID_ARG, "input pointers must be 16-byte aligned");
  if ((uintptr_t)ws & 255) return fail(TOD_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  Plan p;
  const char* why = "";
  st = tod::make_plan_nwr(nq, nr, d, self, o, &p, &why);
  if (st != TOD_OK) return fail(st, why);
  const tod::NwrLayout L = tod::make_layout_nwr(p);
  const int64_t room = tod::nwr_candidate_room(L, ws_bytes);
  if (room < 1)
    return fail(TOD_ERR_WORKSPACE, "workspace too small: need more than " +
                                       std::to_string(L.cand + 512) + " bytes, got " +
                                       std::to_string(ws_bytes));
  char* base = (char*)ws;
  Args a;
  memset(&a, 0, sizeof(a));
  a.xq = xq;
  a.xr = xr;
  a.nq = nq;
  a.nr = nr;
  a.d = (int32_t)d;
  a.dpad = p.dpad;
  a.splits = p.splits;
  a.split_len = p.split_len;
  a.exclude_self = p.exclude_self;
  a.precision = p.precision;
  a.margin_scale = o.margin_scale;
  a.force_fallback = o.force_fallback ? 1 : 0;
  a.scale_exp = p.scale_exp;
  a.ctrl = (tod::Ctrl*)(base + L.ctrl);
  a.mu64 = (double*)(base + L.mu64);
  a.mu32 = (float*)(base + L.mu32);
  a.colpart = (double*)(base + L.colpart);
  a.xq_r = base + L.xq_r;
  a.xq_q = base + L.xq_q;
  a.hn_r = (float*)(base + L.hn_r);
  a.n64_q = (double*)(base + L.n64_q);
  a.rho_q = (double*)(base + L.rho_q);
  a.rho_r = (double*)(base + L.rho_r);
  a.phi = phi;
  a.phi2_row = phi2_row;
  a.ccount = (int32_t*)(base + L.ccount);
  a.coff = (int64_t*)(base + L.coff);
  a.incnt = (int32_t*)(base + L.incnt);
  a.cand = (uint32_t*)(base + L.cand);
  a.cand_d = (float*)(base + L.cand + ((size_t)room * 4 + 255) / 256 * 256);
  a.ccap = room;
  a.row_ptr = row_ptr_out;
  a.idx_out = idx_out;
  a.dist_out = dist_out;
  a.out_cap = idx_out ? capacity : 0;
  int64_t* part = (int64_t*)(base + L.part);
  int64_t* goff = (int64_t*)(base + L.goff);
  const auto tile = p.precision == TOD_PREC_FP16 ? tod::launch_range_tile_f16
                                                 : tod::launch_range_tile_bf16;

  hipStream_t s = (hipStream_t)stream;
  Timers tm;
  tm.on = stats != nullptr;
  hipEvent_t e0 = tm.mark(s);
  hipError_t he = tod::launch_prep(p, a, s);
  if (he != hipSuccess) return hip_fail(he, "prep launch");
  hipEvent_t e_prep = tm.mark(s);
  he = tile(p, a, 0, nq, false, s);
  if (he != hipSuccess) return hip_fail(he, "range tile launch (count)");
  hipEvent_t e_count = tm.mark(s);
  he = tod::launch_scan(a.ccount, nq * p.splits, a.coff, nullptr, part, s);
  if (he == hipSuccess) he = tod::launch_group_offsets(a, L.groups, goff, s);
  if (he != hipSuccess) return hip_fail(he, "candidate offsets launch");
  hipEvent_t e_scan = tm.mark(s);
  // Candidate offsets at 32-row group boundaries decide the batches.
  std::vector<int64_t> g(L.groups + 1);
  tod::Ctrl host;
  he = hipMemcpyAsync(g.data(), goff, sizeof(int64_t) * g.size(), hipMemcpyDeviceToHost, s);
  if (he == hipSuccess) he = hipMemcpyAsync(&host, a.ctrl, sizeof(host), hipMemcpyDeviceToHost, s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);
  if (he != hipSuccess) return hip_fail(he, "candidate count readback");
  if (host.nonfinite) return fail(TOD_ERR_NONFINITE, "input contains NaN or Inf");
  std::vector<std::pair<int64_t, int64_t>> batches;  // [group begin, group end)
  for (int64_t g0 = 0; g0 < L.groups;) {
    int64_t g1 = g0 + 1;
    if (g[g1] - g[g0] > room) {
      const size_t need = L.cand + 512 + (size_t)(g[g1] - g[g0]) * 8;
      return fail(TOD_ERR_WORKSPACE,
                  "workspace too small: 32 query rows have " + std::to_string(g[g1] - g[g0]) +
                      " candidate pairs; need at least " + std::to_string(need) + " bytes");
    }
    while (g1 < L.groups && g[g1 + 1] - g[g0] <= room) ++g1;
    batches.emplace_back(g0, g1);
    g0 = g1;
  }
  std::vector<std::pair<hipEvent_t, hipEvent_t>> tile_ev, rc_ev;
  int64_t largest = 0;
  for (const auto& bt : batches) {
    const int64_t b0 = 32 * bt.first;
    const int64_t b1 = 32 * bt.second < nq ? 32 * bt.second : nq;
    const int64_t rows = b1 - b0;
    largest = rows > largest ? rows : largest;
    a.cbase = g[bt.first];
    hipEvent_t ts = tm.mark(s);
    he = tile(p, a, b0, rows, true, s);
    if (he != hipSuccess) return hip_fail(he, "range tile launch (fill)");
    hipEvent_t te = tm.mark(s);
    he = tod::launch_range_verify(a, b0, rows, dist_out ? 1 : 0, s);
    if (he == hipSuccess)
      he = tod::launch_scan(a.incnt + b0, rows, row_ptr_out + b0, b0 ? row_ptr_out + b0 : nullptr,
                            part, s);
    if (he == hipSuccess && idx_out) he = tod::launch_range_emit(a, b0, rows, s);
    if (he != hipSuccess) return hip_fail(he, "range verify / emit launch");
    hipEvent_t re = tm.mark(s);
    if (tm.on) {
      tile_ev.emplace_back(ts, te);
      rc_ev.emplace_back(te, re);
    }
  }
  hipEvent_t e_end = tm.mark(s);
  int64_t total = 0;
  he = hipMemcpyAsync(&total, row_ptr_out + nq, sizeof(total), hipMemcpyDeviceToHost, s);
  if (he == hipSuccess) he = hipMemcpyAsync(&host, a.ctrl, sizeof(host), hipMemcpyDeviceToHost, s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);
  if (he != hipSuccess) return hip_fail(he, "status readback");
  if (total_out) *total_out = total;
  if (stats) {
    stats->precision = p.precision;
    stats->kprime = 0;
    stats->ref_splits = p.splits;
    stats->query_block = largest;
    stats->blocks = (int64_t)batches.size();
    stats->rows_certified = 0;
    stats->rows_fallback = 0;
    stats->tile_launches = 1 + (int64_t)batches.size();
    stats->reordered = 0;
    stats->ms_prep = Timers::ms(e0, e_prep);
    float t = Timers::ms(e_prep, e_count), r = Timers::ms(e_count, e_scan);
    for (auto& pr : tile_ev) t += Timers::ms(pr.first, pr.second);
    for (auto& pr : rc_ev) r += Timers::ms(pr.first, pr.second);
    stats->ms_tile = t;
    stats->ms_recheck = r;
    stats->ms_fallback = 0.0f;
    stats->ms_score = 0.0f;
    stats->ms_total = Timers::ms(e0, e_end);
    stats->pairs_candidate = g[L.groups];
    int64_t unc = 0;
    for (int i = 0; i < tod::kUncParts; ++i) unc += (int64_t)host.uncertain[i * tod::kUncStride];
    stats->pairs_uncertain = unc;
    stats->pairs_in_range = total;
    stats->tail_parts = 1;
    stats->tail_rows = 0;
    stats->list_runs = 1;
  }
  if (host.internal) return fail(TOD_ERR_INTERNAL, "range tile passes disagree");
  if (idx_out && total > capacity)
    return fail(TOD_ERR_CAPACITY, "pairs in range: " + std::to_string(total) + ", capacity " +
                                      std::to_string(capacity));
  return TOD_OK;
}

// Bytes of a neighbours-within-range workspace whose candidate buffer holds
// `room` pairs (-1: 64 per padded query row and 2^20 more); 0 if the sizes
// or options are invalid.
size_t nwr_ws_bytes(int64_t nq, int64_t nr, int64_t d, const tod_options& o, int32_t self,
                    int64_t room) {
  if (nq <= 0 || nr <= 0 || d <= 0 || nq > kMaxRows || nr > kMaxRows) return 0;
  Plan p;
  const char* why;
  if (tod::make_plan_nwr(nq, nr, d, self, o, &p, &why) != TOD_OK) return 0;
  const tod::NwrLayout L = tod::make_layout_nwr(p);
  const size_t r = room >= 0 ? (size_t)room : (size_t)64 * p.nq_pad + ((size_t)1 << 20);
  return L.cand + 512 + r * 8;
}

// LOCI workspace: the neighbour lists at the largest radius (CSR offsets,
// ids, one radius index byte per pair), the per-radius neighbourhood sizes,
// then the neighbours-within-range pass's own workspace.
struct LociLayout {
  size_t row_ptr, idx, bins, na, nr, nwr;
};

int32_t loci_stride(int32_t nl) { return nl <= 8 ? 8 : (nl <= 16 ? 16 : 32); }

LociLayout loci_layout(int64_t n, int32_t nl, int64_t capacity) {
  LociLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += (bytes + 255) / 256 * 256;
    return at;
  };
  const size_t cells = (size_t)n * (size_t)loci_stride(nl);
  L.row_ptr = take(sizeof(int64_t) * (size_t)(n + 1));
  L.idx = take(sizeof(int64_t) * (size_t)capacity);
  L.bins = take((size_t)capacity);
  L.na = take(sizeof(int32_t) * cells);
  L.nr = take(sizeof(int32_t) * cells);
  L.nwr = off;
  return L;
}

constexpr int64_t kLociMaxRows = (int64_t)1 << 20;

tod_status check_loci(int64_t n, int64_t d, const double* radii, int32_t nl, double alpha,
                      int32_t n_min, double k_sigma, int64_t capacity) {
  if (n <= 0 || d <= 0) return fail(TOD_ERR_INVALID_ARG, "row count and d must be positive");
  if (n > kLociMaxRows) return fail(TOD_ERR_UNSUPPORTED, "LOCI supports at most 2^20 rows");
  if (d > 4096) return fail(TOD_ERR_UNSUPPORTED, "d > 4096");
  if (!radii) return fail(TOD_ERR_INVALID_ARG, "null radii");
  if (nl < 1 || nl > tod::kLociMaxRadii)
    return fail(TOD_ERR_INVALID_ARG, "n_radii must be in [1, 32]");
  for (int32_t l = 0; l < nl; ++l) {
    if (!(radii[l] >= 0.0) || isinf(radii[l]))
      return fail(TOD_ERR_INVALID_ARG, "radii must be finite and >= 0");
    if (l > 0 && !(radii[l] > radii[l - 1]))
      return fail(TOD_ERR_INVALID_ARG, "radii must be strictly increasing");
  }
  if (!(alpha > 0.0 && alpha <= 1.0)) return fail(TOD_ERR_INVALID_ARG, "alpha must be in (0, 1]");
  if (n_min < 1) return fail(TOD_ERR_INVALID_ARG, "n_min must be >= 1");
  if (!(k_sigma >= 0.0) || isinf(k_sigma))
    return fail(TOD_ERR_INVALID_ARG, "k_sigma must be finite and >= 0");
  if (capacity < n) return fail(TOD_ERR_INVALID_ARG, "capacity must be >= n (every point is its own neighbour)");
  return TOD_OK;
}

tod_status run_loci(const float* x, int64_t n, int64_t d, const double* radii, int32_t nl,
                    double alpha, int32_t n_min, double k_sigma, int64_t capacity,
                    const tod_options* opts_in, void* ws, size_t ws_bytes, void* stream,
                    double* score_out, int32_t* flag_out, int32_t* na_out, int32_t* nr_out,
                    double* mdef_out, double* smdef_out, tod_stats* stats) {
  g_last_error.clear();
  tod_options o;
  tod_status st = resolve_options(opts_in, &o);
  if (st != TOD_OK) return st;
  if (o.exclude_self)
    return fail(TOD_ERR_INVALID_ARG, "LOCI samples every point itself: exclude_self must be 0");
  if (!x) return fail(TOD_ERR_INVALID_ARG, "null input pointer");
  if (!score_out) return fail(TOD_ERR_INVALID_ARG, "null score output");
  st = check_loci(n, d, radii, nl, alpha, n_min, k_sigma, capacity);
  if (st != TOD_OK) return st;
  if (!ws) return fail(TOD_ERR_INVALID_ARG, "null workspace");
  if ((uintptr_t)ws & 255) return fail(TOD_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  const LociLayout L = loci_layout(n, nl, capacity);
  if (ws_bytes <= L.nwr)
    return fail(TOD_ERR_WORKSPACE, "workspace too small for " + std::to_string(capacity) +
                                       " pairs: need " +
                                       std::to_string(tod_loci_workspace_size(n, d, nl, capacity,
                                                                              opts_in)) +
                                       " bytes");
  char* base = (char*)ws;
  int64_t* row_ptr = (int64_t*)(base + L.row_ptr);
  int64_t* idx = (int64_t*)(base + L.idx);
  int64_t total = 0;
  // The neighbour lists at the largest radius: exact membership, every
  // point its own neighbour, ids ascending within a row.
  st = run_nwr(x, n, x, n, d, radii[nl - 1], &o, base + L.nwr, ws_bytes - L.nwr, stream, row_ptr,
               capacity, idx, nullptr, &total, stats);
  if (st != TOD_OK) return st;

  tod::LociArgs a;
  memset(&a, 0, sizeof(a));
  a.x = x;
  a.n = n;
  a.d = (int32_t)d;
  a.nl = nl;
  a.nls = loci_stride(nl);
  a.n_min = n_min;
  a.k_sigma = k_sigma;
  a.row_ptr = row_ptr;
  a.idx = idx;
  a.bins = (uint8_t*)(base + L.bins);
  a.na = (int32_t*)(base + L.na);
  a.nr = (int32_t*)(base + L.nr);
  for (int32_t l = 0; l < nl; ++l) {
    a.r2[l] = radii[l] * radii[l];
    const double ar = alpha * radii[l];
    a.a2[l] = ar * ar;
  }
  a.score = score_out;
  a.flag = flag_out;
  a.na_out = na_out;
  a.nr_out = nr_out;
  a.mdef_out = mdef_out;
  a.smdef_out = smdef_out;
  hipStream_t s = (hipStream_t)stream;
  Timers tm;
  tm.on = stats != nullptr;
  hipEvent_t e0 = tm.mark(s);
  hipError_t he = tod::launch_loci(a, s);
  if (he != hipSuccess) return hip_fail(he, "LOCI launch");
  hipEvent_t e1 = tm.mark(s);
  if (stats) {
    he = hipStreamSynchronize(s);
    if (he != hipSuccess) return hip_fail(he, "LOCI synchronize");
    const float ms = Timers::ms(e0, e1);
    stats->ms_score = ms;
    stats->ms_total += ms;
  }
  return TOD_OK;
}

// LOF on tie-inclusive neighbourhoods: the exact kNN lists with one entry
// more than k (when another point exists), each row's squared k-distance and
// whether a point can tie with it, the neighbourhoods as CSR (the k-lists if
// no row can have a tie, else a range query per row at its radius), lrd and
// LOF.  Workspace: the CSR offsets and ids, the lists, the squared
// k-distances and lrd, the tie flag, then a region the kNN call and the
// range query use in turn.
struct LofTiesLayout {
  size_t row_ptr, nbr, lists, kd2, lrd, tie, inner;
};

// Neighbours per list: k + 1 when another point exists (it rules ties out).
int32_t lof_ties_k1(int64_t n, int32_t k) { return (int64_t)k < n - 1 ? k + 1 : k; }

LofTiesLayout lof_ties_layout(int64_t n, int32_t k, int64_t capacity) {
  LofTiesLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += (bytes + 255) / 256 * 256;
    return at;
  };
  L.row_ptr = take(sizeof(int64_t) * (size_t)(n + 1));
  L.nbr = take(sizeof(int64_t) * (size_t)capacity);
  L.lists = take(sizeof(int64_t) * (size_t)n * (size_t)lof_ties_k1(n, k));
  L.kd2 = take(sizeof(double) * (size_t)n);
  L.lrd = take(sizeof(double) * (size_t)n);
  L.tie = take(sizeof(int32_t));
  L.inner = off;
  return L;
}

// Bytes of the shared region: the kNN call's workspace (X against itself)
// or the range query's with candidate room for every pair of the
// neighbourhoods, a quarter more for the filter's uncertain ones and 2^20
// (one fill pass for all rows), whichever is larger; 0 if invalid.
size_t lof_ties_inner_bytes(int64_t n, int64_t d, int32_t k, int64_t capacity,
                            const tod_options& o) {
  Plan p;
  const char* why;
  if (tod::make_plan(n, n, d, lof_ties_k1(n, k), 0, 1, o, &p, &why) != TOD_OK) return 0;
  const size_t knn = tod::make_layout(p).total;
  const size_t nwr = nwr_ws_bytes(n, n, d, o, 1, capacity + capacity / 4 + ((int64_t)1 << 20));
  if (nwr == 0) return 0;
  return knn > nwr ? knn : nwr;
}

tod_status check_lof_ties(int64_t n, int64_t d, int32_t k, int64_t capacity,
                          const tod_options& o) {
  tod_status st = check_sizes(n, n, d, k, 1);
  if (st != TOD_OK) return st;
  if (d > 512)
    return fail(TOD_ERR_UNSUPPORTED, "tod_lof_ties supports rows of at most 512 elements");
  if (o.precision == TOD_PREC_FP32)
    return fail(TOD_ERR_UNSUPPORTED,
                "tod_lof_ties filters in fp16 or bf16 (its range query is MFMA only)");
  if (capacity < n * (int64_t)k)
    return fail(TOD_ERR_INVALID_ARG, "capacity must be >= n k (every neighbourhood holds k points)");
  return TOD_OK;
}

tod_status run_lof_ties(const float* x, int64_t n, int64_t d, int32_t k, int64_t capacity,
                        const tod_options* opts_in, void* ws, size_t ws_bytes, void* stream,
                        float* lof_out, int32_t* count_out, tod_stats* stats) {
  g_last_error.clear();
  tod_options o;
  tod_status st = resolve_options(opts_in, &o);
  if (st != TOD_OK) return st;
  o.exclude_self = 1;
  if (stats && stats->struct_size != sizeof(tod_stats))
    return fail(TOD_ERR_INVALID_ARG, "tod_stats.struct_size does not match this library");
  if (!x) return fail(TOD_ERR_INVALID_ARG, "null input pointer");
  if (!lof_out) return fail(TOD_ERR_INVALID_ARG, "null LOF output");
  if (!ws) return fail(TOD_ERR_INVALID_ARG, "null workspace");
  if ((uintptr_t)ws & 255) return fail(TOD_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  st = check_lof_ties(n, d, k, capacity, o);
  if (st != TOD_OK) return st;
  const LofTiesLayout L = lof_ties_layout(n, k, capacity);
  const size_t inner = lof_ties_inner_bytes(n, d, k, capacity, o);
  if (inner == 0) return fail(TOD_ERR_INVALID_ARG, "sizes or options the planner rejects");
  if (ws_bytes < L.inner + inner)
    return fail(TOD_ERR_WORKSPACE, "workspace too small for " + std::to_string(capacity) +
                                       " pairs: need " + std::to_string(L.inner + inner) +
                                       " bytes, got " + std::to_string(ws_bytes));
  char* base = (char*)ws;
  int64_t* row_ptr = (int64_t*)(base + L.row_ptr);
  int64_t* nbr = (int64_t*)(base + L.nbr);
  int64_t* lists = (int64_t*)(base + L.lists);
  double* kd2 = (double*)(base + L.kd2);
  double* lrd = (double*)(base + L.lrd);
  int32_t* tie = (int32_t*)(base + L.tie);
  const int32_t k1 = lof_ties_k1(n, k);
  hipStream_t s = (hipStream_t)stream;
  // 1. Exact kNN lists (X against itself, self excluded), k1 entries.
  st = run(x, n, x, n, d, k1, &o, 1, 0, base + L.inner, ws_bytes - L.inner, stream, lists,
           nullptr, nullptr, nullptr, nullptr, 0, nullptr, stats);
  if (st != TOD_OK) return st;
  Timers tm;
  tm.on = stats != nullptr;
  hipEvent_t e0 = tm.mark(s);
  // 2. Each row's squared k-distance in the range query's exact arithmetic,
  //    and whether any row can have a point tied with it.
  hipError_t he = tod::launch_ties_radius(x, n, (int)d, k, k1, lists, kd2, tie, s);
  int32_t any_tie = 0;
  if (he == hipSuccess)
    he = hipMemcpyAsync(&any_tie, tie, sizeof(any_tie), hipMemcpyDeviceToHost, s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);
  if (he != hipSuccess) return hip_fail(he, "k-distance launch");
  hipEvent_t e1 = tm.mark(s);
  // 3. The neighbourhoods: the k-lists where no tie is possible, else the
  //    range query at each row's own radius.
  tod_stats rs;
  memset(&rs, 0, sizeof(rs));
  rs.struct_size = sizeof(tod_stats);
  int64_t total = 0;
  if (!any_tie) {
    he = tod::launch_ties_lists(n, k, k1, lists, row_ptr, nbr, s);
    if (he != hipSuccess) return hip_fail(he, "neighbourhood launch");
    total = n * (int64_t)k;
    st = TOD_OK;
  } else {
    st = run_nwr(x, n, x, n, d, 0.0, &o, base + L.inner, ws_bytes - L.inner, stream, row_ptr,
                 capacity, nbr, nullptr, &total, stats ? &rs : nullptr, kd2);
  }
  if (stats) {
    stats->pairs_candidate = rs.pairs_candidate;
    stats->pairs_uncertain = rs.pairs_uncertain;
    stats->pairs_in_range = total;
  }
  if (st != TOD_OK) return st;
  // 4. lrd and LOF over the neighbourhoods.
  hipEvent_t e2 = tm.mark(s);
  he = tod::launch_lof_ties(x, n, (int)d, row_ptr, nbr, kd2, lrd, lof_out, count_out, s);
  if (he != hipSuccess) return hip_fail(he, "LOF launch");
  hipEvent_t e3 = tm.mark(s);
  if (stats) {
    he = hipStreamSynchronize(s);
    if (he != hipSuccess) return hip_fail(he, "LOF synchronize");
    const float t_rad = Timers::ms(e0, e1), t_lof = Timers::ms(e2, e3);
    stats->ms_prep += rs.ms_prep;
    stats->ms_tile += rs.ms_tile;
    stats->ms_recheck += rs.ms_recheck + t_rad;
    stats->ms_score = t_lof;
    stats->ms_total += t_rad + rs.ms_total + t_lof;
    stats->tile_launches += rs.tile_launches;
  }
  return TOD_OK;
}

}  // namespace

extern "C" {

void tod_default_options(tod_options* o) {
  if (!o) return;
  memset(o, 0, sizeof(*o));
  o->struct_size = sizeof(tod_options);
  o->precision = TOD_PREC_AUTO;
  o->margin_scale = 1.0f;
}

size_t tod_workspace_size(int64_t nq, int64_t nr, int64_t d, int32_t k, int32_t mode,
                          const tod_options* opts) {
  tod_options o;
  if (resolve_options(opts, &o) != TOD_OK) return 0;
  if (mode < 0 || mode > 2) return 0;
  const int32_t lof = mode == 1 ? 1 : 0;
  if (lof) o.exclude_self = 1;
  if (check_sizes(nq, nr, d, k, o.exclude_self) != TOD_OK) return 0;
  if (lof && nq != nr) return 0;
  Plan p;
  const char* why;
  // Mode 1 sizes for X against itself.  Modes 0 and 2 serve separate query
  // and reference sets and X against itself (tod_knn_score, or tod_knn with
  // xq == xr), so they take the larger of the two layouts.
  if (tod::make_plan(nq, nr, d, k, lof, lof, o, &p, &why) != TOD_OK) return 0;
  if (mode == 2) p.lists = 1;
  size_t total = tod::make_layout(p).total;
  if (!lof && nq == nr) {
    Plan ps;
    if (tod::make_plan(nq, nr, d, k, 0, 1, o, &ps, &why) != TOD_OK) return 0;
    if (mode == 2) ps.lists = 1;
    const size_t t2 = tod::make_layout(ps).total;
    total = t2 > total ? t2 : total;
  }
  return total;
}

tod_status tod_knn(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d,
                   int32_t k, const tod_options* opts, void* workspace, size_t ws_bytes,
                   void* stream, int64_t* idx_out, float* dist_out, tod_stats* stats) {
  if (!idx_out || !dist_out) return fail(TOD_ERR_INVALID_ARG, "null output pointer");
  return run(xq, nq, xr, nr, d, k, opts, 0, 0, workspace, ws_bytes, stream, idx_out, dist_out,
             nullptr, nullptr, nullptr, 0, nullptr, stats);
}

// Workspace of tod_knn_noalloc: one copy per GPU, held by the loaded code
// object from load until the process ends.  Host code never uses this name
// as an address (on the host it is only a stand-in for the symbol): the
// device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[TOD_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_at[kMaxDevices] = {};

// Device address of the current device's scratch array (looked up on the
// first call on that device, with that device current).
tod_status scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t he = hipGetDevice(&dev);
  if (he != hipSuccess) return hip_fail(he, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(TOD_ERR_UNSUPPORTED, "tod_knn_noalloc: device ordinal " + std::to_string(dev) +
                                         " beyond the " + std::to_string(kMaxDevices) +
                                         " devices it keeps a scratch address for");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_at[dev]) {
    void* ptr = nullptr;
    he = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (he != hipSuccess) return hip_fail(he, "hipGetSymbolAddress(scratch)");
    if (!ptr || ((uintptr_t)ptr & 255))
      return fail(TOD_ERR_INTERNAL, "tod_knn_noalloc: scratch address null or misaligned");
    g_scratch_at[dev] = ptr;
  }
  *out = g_scratch_at[dev];
  return TOD_OK;
}
}  // namespace

tod_status tod_knn_noalloc(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d,
                           int32_t k, const tod_options* opts, void* stream, int64_t* idx_out,
                           float* dist_out, tod_stats* stats) {
  g_last_error.clear();
  if (!idx_out || !dist_out) return fail(TOD_ERR_INVALID_ARG, "null output pointer");
  void* ws = nullptr;
  tod_status st = scratch_of_current_device(&ws);
  if (st != TOD_OK) return st;
  // No HIP events (their creation may allocate): stats carries the plan and
  // the row counts, with zero timings.
  st = run(xq, nq, xr, nr, d, k, opts, 0, 0, ws, TOD_NOALLOC_SCRATCH_BYTES, stream, idx_out,
           dist_out, nullptr, nullptr, nullptr, 0, nullptr, stats, /*events=*/false);
  if (st == TOD_ERR_WORKSPACE)
    return fail(st, "tod_knn_noalloc: the problem does not fit the library's static scratch of " +
                        std::to_string(TOD_NOALLOC_SCRATCH_BYTES) + " bytes (" + g_last_error +
                        "); use tod_knn with a workspace of its own");
  return st;
}

tod_status tod_knn_score(const float* x, int64_t n, int64_t d, int32_t k,
                         const tod_options* opts, void* workspace, size_t ws_bytes,
                         void* stream, float* score_out, int64_t* idx_out, float* dist_out,
                         tod_stats* stats) {
  if (!score_out) return fail(TOD_ERR_INVALID_ARG, "null score output");
  return run(x, n, x, n, d, k, opts, 1, 0, workspace, ws_bytes, stream, idx_out, dist_out,
             score_out, nullptr, nullptr, 0, nullptr, stats);
}

tod_status tod_lof(const float* x, int64_t n, int64_t d, int32_t k, const tod_options* opts,
                   void* workspace, size_t ws_bytes, void* stream, float* lof_out,
                   float* knn_score_out, int64_t* idx_out, float* dist_out, tod_stats* stats) {
  if (!lof_out) return fail(TOD_ERR_INVALID_ARG, "null LOF output");
  return run(x, n, x, n, d, k, opts, 1, 1, workspace, ws_bytes, stream, idx_out, dist_out,
             knn_score_out, lof_out, nullptr, 0, nullptr, stats);
}

tod_status tod_knn_decision(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d,
                            int32_t k, const tod_options* opts, void* workspace, size_t ws_bytes,
                            void* stream, float* score_out, int64_t* idx_out, float* dist_out,
                            tod_stats* stats) {
  g_last_error.clear();
  if (!score_out) return fail(TOD_ERR_INVALID_ARG, "null score output");
  if (opts && opts->struct_size == sizeof(tod_options) && opts->exclude_self)
    return fail(TOD_ERR_INVALID_ARG, "tod_knn_decision scores new points: exclude_self must be 0");
  return run(xq, nq, xr, nr, d, k, opts, 0, 0, workspace, ws_bytes, stream, idx_out, dist_out,
             score_out, nullptr, nullptr, 0, nullptr, stats);
}

tod_status tod_knn_classify(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d,
                            int32_t k, const int32_t* labels_r, int32_t n_classes,
                            const tod_options* opts, void* workspace, size_t ws_bytes,
                            void* stream, int32_t* pred_out, tod_stats* stats) {
  g_last_error.clear();
  if (!labels_r || !pred_out) return fail(TOD_ERR_INVALID_ARG, "null labels or prediction output");
  if (n_classes < 1 || n_classes > 65536)
    return fail(TOD_ERR_INVALID_ARG, "n_classes must be in [1, 65536]");
  return run(xq, nq, xr, nr, d, k, opts, 0, 2, workspace, ws_bytes, stream, nullptr, nullptr,
             nullptr, nullptr, labels_r, n_classes, pred_out, stats);
}

tod_status tod_abod(const float* x, int64_t n, int64_t d, int32_t k, const tod_options* opts,
                    void* workspace, size_t ws_bytes, void* stream, float* score_out,
                    int64_t* idx_out, float* dist_out, tod_stats* stats) {
  g_last_error.clear();
  if (!score_out) return fail(TOD_ERR_INVALID_ARG, "null score output");
  if (k < 2) return fail(TOD_ERR_INVALID_ARG, "ABOD needs k >= 2 (pairs of neighbours)");
  if (k > 64) return fail(TOD_ERR_UNSUPPORTED, "ABOD supports k <= 64");
  return run(x, n, x, n, d, k, opts, 1, 3, workspace, ws_bytes, stream, idx_out, dist_out,
             score_out, nullptr, nullptr, 0, nullptr, stats);
}

tod_status tod_cof(const float* x, int64_t n, int64_t d, int32_t k, const tod_options* opts,
                   void* workspace, size_t ws_bytes, void* stream, float* cof_out,
                   float* knn_score_out, int64_t* idx_out, float* dist_out, tod_stats* stats) {
  g_last_error.clear();
  if (!cof_out) return fail(TOD_ERR_INVALID_ARG, "null COF output");
  if (k > 63) return fail(TOD_ERR_UNSUPPORTED, "COF supports k <= 63");
  return run(x, n, x, n, d, k, opts, 1, 4, workspace, ws_bytes, stream, idx_out, dist_out,
             knn_score_out, cof_out, nullptr, 0, nullptr, stats);
}

size_t tod_nwr_workspace_size(int64_t nq, int64_t nr, int64_t d, const tod_options* opts) {
  tod_options o;
  if (resolve_options(opts, &o) != TOD_OK) return 0;
  // Sized for separate query and reference sets (enough for any call), with
  // room for 64 candidates per query row and 2^20 more.
  return nwr_ws_bytes(nq, nr, d, o, 0, -1);
}

tod_status tod_nwr(const float* xq, int64_t nq, const float* xr, int64_t nr, int64_t d,
                   double phi, const tod_options* opts, void* workspace, size_t ws_bytes,
                   void* stream, int64_t* row_ptr_out, int64_t capacity, int64_t* idx_out,
                   float* dist_out, int64_t* total_out, tod_stats* stats) {
  return run_nwr(xq, nq, xr, nr, d, phi, opts, workspace, ws_bytes, stream, row_ptr_out,
                 capacity, idx_out, dist_out, total_out, stats);
}

size_t tod_loci_workspace_size(int64_t n, int64_t d, int32_t n_radii, int64_t capacity,
                               const tod_options* opts) {
  tod_options o;
  if (resolve_options(opts, &o) != TOD_OK) return 0;
  if (n <= 0 || d <= 0 || n > kLociMaxRows || n_radii < 1 || n_radii > tod::kLociMaxRadii ||
      capacity < n)
    return 0;
  o.exclude_self = 0;
  // The neighbours-within-range pass gets candidate room for every pair in
  // range and a quarter more for the filter's uncertain ones, so that one
  // fill pass covers all rows (a batch per few hundred rows would leave
  // the GPU mostly idle).
  const size_t nwr = nwr_ws_bytes(n, n, d, o, 1, capacity + capacity / 4 + ((int64_t)1 << 20));
  if (nwr == 0) return 0;
  return loci_layout(n, n_radii, capacity).nwr + nwr;
}

tod_status tod_loci(const float* x, int64_t n, int64_t d, const double* radii, int32_t n_radii,
                    double alpha, int32_t n_min, double k_sigma, int64_t capacity,
                    const tod_options* opts, void* workspace, size_t ws_bytes, void* stream,
                    double* score_out, int32_t* flag_out, int32_t* n_alpha_out,
                    int32_t* n_r_out, double* mdef_out, double* sigma_mdef_out,
                    tod_stats* stats) {
  return run_loci(x, n, d, radii, n_radii, alpha, n_min, k_sigma, capacity, opts, workspace,
                  ws_bytes, stream, score_out, flag_out, n_alpha_out, n_r_out, mdef_out,
                  sigma_mdef_out, stats);
}

size_t tod_lof_ties_workspace_size(int64_t n, int64_t d, int32_t k, int64_t capacity,
                                   const tod_options* opts) {
  tod_options o;
  if (resolve_options(opts, &o) != TOD_OK) return 0;
  o.exclude_self = 1;
  if (check_lof_ties(n, d, k, capacity, o) != TOD_OK) return 0;
  const size_t inner = lof_ties_inner_bytes(n, d, k, capacity, o);
  if (inner == 0) return 0;
  return lof_ties_layout(n, k, capacity).inner + inner;
}

tod_status tod_lof_ties(const float* x, int64_t n, int64_t d, int32_t k, int64_t capacity,
                        const tod_options* opts, void* workspace, size_t ws_bytes, void* stream,
                        float* lof_out, int32_t* count_out, tod_stats* stats) {
  return run_lof_ties(x, n, d, k, capacity, opts, workspace, ws_bytes, stream, lof_out,
                      count_out, stats);
}

tod_status tod_plan(int64_t nq, int64_t nr, int64_t d, int32_t k, const tod_options* opts,
                    tod_stats* plan) {
  g_last_error.clear();
  if (!plan || plan->struct_size != sizeof(tod_stats))
    return fail(TOD_ERR_INVALID_ARG, "plan must point to a tod_stats with struct_size set");
  tod_options o;
  tod_status st = resolve_options(opts, &o);
  if (st != TOD_OK) return st;
  st = check_sizes(nq, nr, d, k, o.exclude_self);
  if (st != TOD_OK) return st;
  Plan p;
  const char* why;
  st = tod::make_plan(nq, nr, d, k, 0, o.exclude_self ? 1 : 0, o, &p, &why);
  if (st != TOD_OK) return fail(st, why);
  plan->precision = p.precision;
  plan->kprime = p.kprime;
  plan->ref_splits = p.splits;
  plan->query_block = p.query_block;
  plan->blocks = p.blocks;
  plan->tile_launches = p.blocks;
  plan->reordered = p.order;
  plan->list_runs = p.runs;
  return TOD_OK;
}

tod_status tod_plan_workspace(int64_t nq, int64_t nr, int64_t d, int32_t k, int32_t mode,
                              const tod_options* opts, size_t ws_bytes, tod_stats* plan) {
  g_last_error.clear();
  if (!plan || plan->struct_size != sizeof(tod_stats))
    return fail(TOD_ERR_INVALID_ARG, "plan must point to a tod_stats with struct_size set");
  if (mode < 0 || mode > 2) return fail(TOD_ERR_INVALID_ARG, "mode must be 0, 1 or 2");
  tod_options o;
  tod_status st = resolve_options(opts, &o);
  if (st != TOD_OK) return st;
  const int32_t lof = mode == 1 ? 1 : 0;
  if (lof) o.exclude_self = 1;
  if (lof && nq != nr) return fail(TOD_ERR_INVALID_ARG, "mode 1 is X against itself: nq == nr");
  st = check_sizes(nq, nr, d, k, o.exclude_self);
  if (st != TOD_OK) return st;
  Plan p;
  const char* why;
  const int32_t self = o.exclude_self ? 1 : 0;
  st = tod::make_plan(nq, nr, d, k, lof, self, o, &p, &why);
  if (st != TOD_OK) return fail(st, why);
  if (mode == 2) p.lists = 1;
  const size_t need = tod::make_layout(p).total;
  if (ws_bytes < need) {
    std::string w;
    st = tod::fit_plan(&p, ws_bytes, o, &w);
    if (st != TOD_OK)
      return fail(st, "workspace of " + std::to_string(ws_bytes) + " bytes too small (" + w +
                          "; the one-block plan needs " + std::to_string(need) + ")");
  }
  plan->precision = p.precision;
  plan->kprime = p.kprime;
  plan->ref_splits = p.splits;
  plan->query_block = p.query_block;
  plan->blocks = p.blocks;
  plan->tile_launches = p.blocks;
  plan->reordered = p.order;
  plan->list_runs = p.runs;
  return TOD_OK;
}

const char* tod_status_string(tod_status s) {
  switch (s) {
    case TOD_OK: return "TOD_OK";
    case TOD_ERR_INVALID_ARG: return "TOD_ERR_INVALID_ARG";
    case TOD_ERR_NONFINITE: return "TOD_ERR_NONFINITE";
    case TOD_ERR_WORKSPACE: return "TOD_ERR_WORKSPACE";
    case TOD_ERR_UNSUPPORTED: return "TOD_ERR_UNSUPPORTED";
    case TOD_ERR_HIP: return "TOD_ERR_HIP";
    case TOD_ERR_INTERNAL: return "TOD_ERR_INTERNAL";
    case TOD_ERR_CAPACITY: return "TOD_ERR_CAPACITY";
  }
  return "TOD_ERR_UNKNOWN";
}

const char* tod_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
