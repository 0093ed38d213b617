// Fused MFMA distance tile + top-K' selection with the shortlist in registers
// (Section 6.1's fusion of cdist and topk, evaluated in the filter precision
// of Section 5.2 step ii).
//
// Work decomposition.  A workgroup of W waves owns W x 32 queries and walks one
// reference split in stages of 32*NS rows.  A stage of quantised reference
// rows (and their accumulator seeds -N_j/2) is staged once per workgroup in
// LDS, double-buffered: the next stage's global loads are in flight while the
// current one is consumed.  Each wave keeps its 32 queries' operand in
// registers for the whole kernel.  v_mfma_f32_32x32x16_{f16,bf16} takes the
// references as A (rows) and the queries as B (columns); lane l ends a
// 32-row sub-tile holding 16 accumulators of query l % 32:
//     acc = -N_j/2 + <xhat_i, xhat_j>,    key = -2 acc = fl(N_j) - 2 <xhat_i, xhat_j>.
//
// Selection.  Query q is owned by the lane pair (q, q + 32).  Its K' = 2R best
// entries form one ascending list split over the pair: lane q holds entries
// 0..R-1, lane q + 32 entries R..2R-1, all in registers.  An entry is 64 bits:
// the accumulator mapped to an unsigned key that ascends as acc descends, and
// the reference index below it.  Both lanes keep the acc of entry K'-1 as a
// threshold; a sub-tile costs a max3 reduction and one compare per lane unless
// some accumulator beats it.  Survivors are appended to an LDS queue (16 or 28
// slots) of their lane.  When a queue could overflow, the whole wave merges: every lane
// sorts its queue, each pair merges its two queues and then the merged queue
// with its list by bitonic stages whose cross-lane step is v_permlane32_swap.
// No LDS round trip is needed for the lists, so LDS holds only the staged
// references and the queues.
//
// Exactness does not depend on how ties between equal keys are broken inside
// the filter: every reference left out of the final shortlist has a key no
// smaller than the K'-th key h, which is all the certificate uses.
#pragma once

#include <type_traits>

#include "tod_internal.h"
#include "wave.h"

namespace tod {
namespace mt {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

template <typename ET>
struct Frag;
template <>
struct Frag<_Float16> {
  using V = f16x8;
};
template <>
struct Frag<__bf16> {
  using V = bf16x8;
};

template <typename ET>
__device__ __forceinline__ f32x16 mfma(typename Frag<ET>::V a, typename Frag<ET>::V b, f32x16 c) {
  if constexpr (std::is_same<ET, _Float16>::value)
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

constexpr int kMerge = 16;  // queue entries one merge takes per lane

// Queue slots per lane.  16-entry lists see few insertions: a 16-slot queue
// filled half a sub-tile at a time keeps LDS small enough for three
// workgroups per CU.  Longer lists insert often: a 28-slot queue takes a whole
// sub-tile after at most one merge (which leaves at most 12 entries), and
// merges wait until some lane holds 13 entries.  28 slots is the most that
// keeps two workgroups per CU at rows of 32 and 64 elements; 24 slots merged
// more often (C2's tile 8% slower), 32 slots left one workgroup per CU.
template <int R>
constexpr int queue_cap() { return R <= 8 ? 16 : 28; }

// Workgroup barrier of the two-stage staging pipeline: this wave's LDS writes
// are complete before it, and global loads still in flight stay in flight (a
// release fence would wait for them).  The asm also keeps the compiler from
// moving memory accesses across it.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// LDS byte address of a pointer into the workgroup's shared memory.
__device__ __forceinline__ uint32_t lds_off(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Direct staging: each active lane moves 16 bytes from global memory to LDS
// address lds + 16 * lane (global_load_lds_dwordx4; lds must be wave-uniform).
// Issued from asm so that the compiler, which cannot tell the LDS buffers
// apart, does not wait for every staging load before each LDS read; the
// caller orders them with dl_barrier().  M0 is set right before the load,
// with the one wait state an LDS DMA needs after an SALU write of M0 (the
// compiler inserts it for its own code, never inside asm).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g),
               "s"(__builtin_amdgcn_readfirstlane(lds))
               : "memory", "m0");
}
#pragma clang diagnostic pop

// Barrier of the direct-staging pipeline: this wave's staging loads except
// the newest N are complete (so is every LDS access), then all waves meet.
template <int N>
__device__ __forceinline__ void dl_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// f(std::integral_constant<int, 0>{}), ..., f(<N - 1>): a loop whose index is
// a constant in every iteration, so that arrays indexed by it stay in
// registers.
template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// Value of v in the partner lane (lane ^ 32).
__device__ __forceinline__ uint32_t xchg32(uint32_t v, int h) {
  const auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return h ? p[0] : p[1];
}
__device__ __forceinline__ uint64_t xchg64(uint64_t v, int h) {
  return ((uint64_t)xchg32((uint32_t)(v >> 32), h) << 32) | xchg32((uint32_t)v, h);
}

// Entries are ordered by their key (the high word) alone: a 32-bit compare.
// The order of equal keys does not matter to the filter (see the file header).
__device__ __forceinline__ bool key_lt(uint64_t a, uint64_t b) {
  return (uint32_t)(a >> 32) < (uint32_t)(b >> 32);
}

// Ascending compare-exchange.
__device__ __forceinline__ void ce(uint64_t& x, uint64_t& y) {
  const bool sw = key_lt(y, x);
  const uint64_t lo = sw ? y : x;
  const uint64_t hi = sw ? x : y;
  x = lo;
  y = hi;
}

// Keep min (h == 0) or max (h == 1) of x and the partner's value p.
__device__ __forceinline__ uint64_t keep(uint64_t x, uint64_t p, int h) {
  const bool take = h ? key_lt(x, p) : key_lt(p, x);
  return take ? p : x;
}

// Bitonic sort of N registers, ascending.
template <int N>
__device__ __forceinline__ void sort_asc(uint64_t (&v)[N]) {
#pragma unroll
  for (int size = 2; size <= N; size <<= 1)
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1)
#pragma unroll
      for (int i = 0; i < N; ++i) {
        if (i & stride) continue;
        const int j = i | stride;
        if ((i & size) == 0 || size == N)
          ce(v[i], v[j]);
        else
          ce(v[j], v[i]);
      }
}

// Sort a bitonic sequence of N registers ascending.
template <int N>
__device__ __forceinline__ void clean_asc(uint64_t (&v)[N]) {
#pragma unroll
  for (int stride = N >> 1; stride > 0; stride >>= 1)
#pragma unroll
    for (int i = 0; i < N; ++i)
      if (!(i & stride)) ce(v[i], v[i | stride]);
}

// Accumulator bits -> entry key that ascends as the accumulator descends.
__device__ __forceinline__ uint64_t entry_of(uint32_t accbits, uint32_t idx) {
  const uint32_t hi = accbits ^ ((uint32_t)((int32_t)~accbits >> 31) & 0x7fffffffu);
  return ((uint64_t)hi << 32) | idx;
}

__device__ __forceinline__ float acc_of(uint64_t e) {
  const uint32_t hi = (uint32_t)(e >> 32);
  const uint32_t u = (hi & 0x80000000u) ? hi : (hi ^ 0x7fffffffu);
  return __uint_as_float(u);
}

// Threshold in accumulator space from the K'-th entry (none yet: -inf).
__device__ __forceinline__ float thr_of(uint64_t e) {
  return e == kEmpty ? -INFINITY : acc_of(e);
}

// Maximum of three (v_max3_f32, formed by the compiler).  It must stay
// visible to the compiler: the hardware does not interlock a VALU read of an
// MFMA result, and the compiler inserts the wait states such a read needs
// (12 after v_mfma_f32_32x32x16_{f16,bf16} on gfx950) only for instructions
// it generates itself, not for inline asm.  An asm v_max3_f32 here could read
// an accumulator the MFMA had not yet written and skip a sub-tile that holds
// a survivor.  The operands are never NaN, so fmax is the plain maximum.
__device__ __forceinline__ float max3f(float a, float b, float c) {
  return __builtin_fmaxf(__builtin_fmaxf(a, b), c);
}

// Reference row (0..31 within the sub-tile) of accumulator r in this lane
// (32x32 MFMA output layout: column = lane % 32).
__device__ __forceinline__ int out_row(int r, int h) { return 8 * (r >> 2) + 4 * h + (r & 3); }
// The part of out_row that does not depend on the lane.  Paths that form row
// ids take the lane's part 4h through an opaque copy and add this constant:
// otherwise the compiler keeps the 16 values out_row(r, h) in registers for
// the whole kernel.
__host__ __device__ constexpr int out_row_c(int r) { return 8 * (r >> 2) + (r & 3); }

// Merge the first kMerge entries of every lane's queue (fewer where cnt is
// smaller) into its pair's list; all 64 lanes take part.
// list: this lane's R entries of the pair's ascending K' = 2R list.
template <int R>
__device__ __forceinline__ void merge_queues(uint64_t (&L)[R], const uint2* myq, int cnt, int h) {
  constexpr int M = kMerge;
  uint64_t Q[M];
#pragma unroll
  for (int i = 0; i < M; ++i) {
    const uint2 v = myq[i * 64];
    Q[i] = i < cnt ? entry_of(v.x, v.y) : kEmpty;
  }
  sort_asc<M>(Q);
  // Merge the pair's two sorted queues: lane q keeps the M smallest, lane
  // q + 32 the M largest (each a bitonic sequence), then sort each.  Element
  // i meets the partner's element M-1-i; both ends of a pair are exchanged
  // before either is overwritten.
#pragma unroll
  for (int i = 0; i < M / 2; ++i) {
    const uint64_t pa = xchg64(Q[M - 1 - i], h);
    const uint64_t pb = xchg64(Q[i], h);
    Q[i] = keep(Q[i], pa, h);
    Q[M - 1 - i] = keep(Q[M - 1 - i], pb, h);
  }
  clean_asc<M>(Q);
  // Now the pair's queue is ascending: lane q holds Q[0..M), lane q + 32
  // Q[M..2M).  The 2R smallest of list and queue are min(L[e], Q[2R-1-e]).
  if constexpr (R == M) {
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const uint64_t o = xchg64(Q[R - 1 - i], h);
      L[i] = key_lt(o, L[i]) ? o : L[i];
    }
  } else if constexpr (R < M) {
    // Q[2R-1-e] lies in lane q: for lane q itself at index 2R-1-i, for lane
    // q + 32 (e = R + i) at index R-1-i of the partner.
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const uint64_t p = xchg64(Q[R - 1 - i], h);
      const uint64_t o = h ? p : Q[2 * R - 1 - i];
      L[i] = key_lt(o, L[i]) ? o : L[i];
    }
  } else {
    static_assert(R == 2 * M, "list length per lane must be 8, 16 or 32");
    // The queue has 2M = R entries, so only lane q + 32's entries can change:
    // e = R + i pairs with Q[2M-1-i], which for i < M is this lane's Q[M-1-i]
    // and for i >= M the partner's Q[2M-1-i].
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const uint64_t o = i < M ? Q[M - 1 - i] : xchg64(Q[2 * M - 1 - i], h);
      const uint64_t m = key_lt(o, L[i]) ? o : L[i];
      L[i] = h ? m : L[i];
    }
  }
  // The 2R entries now form a bitonic sequence over the pair: one cross-lane
  // stage, then sort each half.
#pragma unroll
  for (int i = 0; i < R; ++i) L[i] = keep(L[i], xchg64(L[i], h), h);
  clean_asc<R>(L);
}

// Row layouts.  The accumulator seed -N_j/2 is formed by the MFMA from parts
// p_1..p_4 of -N_j/(2c) in the filter precision against the constant c:
//     acc = sum_t xhat_it xhat_jt + c sum_p p_p = <xhat_i, xhat_j> - N_j/2.
// Plain (FOLD = false): the row padded to DPAD (16 ... 512); the parts (8
// bytes a row) are staged in LDS beside the rows, and a sub-tile starts with
// one seed MFMA: A row j = (p_1..p_4, 0 ...), B = c in its first four k rows.
// That replaces 16 fp32 seeds per lane (four 16-byte LDS reads by every
// lane, most of the LDS traffic at rows of 32 elements) with one 8-byte read
// and one MFMA.  Fold (FOLD = true, rows of at most 8 elements, DPAD = 16):
// the parts sit in columns 8..11 of the row and the queries carry c there,
// so the single 16-wide MFMA step, which would otherwise multiply zero
// padding, forms the seed too.
template <int DPAD, bool FOLD>
struct Layout {
  static constexpr int k16 = DPAD / 16;  // 16-wide k-steps
  // LDS row stride: 32-byte rows are stored unpadded with their halves
  // swizzled (swz); longer rows get 16 bytes of padding so the rows of a read
  // group hit distinct banks.
  static constexpr int rowb = DPAD == 16 ? 32 : DPAD * 2 + 16;
  static constexpr int cpr = DPAD / 8;  // 16-byte chunks per row
  // Sub-tiles per stage: the stage pair, seeds and four queues stay under
  // 80 KiB so that at least two workgroups share a CU.  (Folded rows with
  // 16-entry lists take stages of four: see launch_mtile.)
  static constexpr int ns = DPAD == 16 ? 8 : (DPAD == 32 ? 4 : (DPAD == 64 ? 2 : 1));
  // Rows of 256 or more elements keep a 32-query operand of DPAD/2 VGPRs
  // per lane: such kernels run one wave per SIMD.
  static constexpr bool wide = DPAD >= 256;
  static_assert(!FOLD || DPAD == 16, "the folded seed uses the padding of 8-wide rows");
};

// Half swap of 32-byte staged rows: rows 4..7 and 8..11 of every 16 keep
// their halves swapped, which spreads the first halves of any 8 or 16
// consecutive rows over distinct LDS banks.
__device__ __forceinline__ int swz(int r) { return ((r >> 2) ^ (r >> 3)) & 1; }

// Stage buffers: rows of 512 elements are staged directly into LDS, two
// stages ahead (three buffers) for waves of 32 queries and one stage ahead
// (two buffers, stages twice as long) for waves of 64; other rows through
// registers (two buffers).
__host__ __device__ constexpr int stage_buffers(int dpad, bool fold, int nq) {
  return dpad >= 512 && !fold && nq == 1 ? 3 : 2;
}

// Query columns per wave: 64 (two 32-query groups sharing every A fragment)
// for rows of 512 elements with lists of up to 32 entries, whose 32-step MFMA
// chains otherwise need one LDS fragment per MFMA; 32 otherwise.  The two
// groups' operands take all 256 AGPRs; 64-entry lists for two groups (128
// VGPRs) then leave the compiler too few registers, and it spills part of
// the operand to scratch memory.
__host__ __device__ constexpr int query_groups(int dpad, bool fold, int r) {
  return dpad >= 512 && !fold && r <= 16 ? 2 : 1;
}

// Queue slots per lane and query group (two groups: 16 slots, the LDS of two
// 28-slot queues per wave does not fit beside the stages).
template <int R, int NQ>
constexpr int queue_slots() { return NQ == 1 ? queue_cap<R>() : 16; }

// Stage buffers, their seeds and the queues.
__host__ __device__ constexpr size_t lds_bytes(int dpad, bool fold, int w, int ns, int qcap,
                                               int nq) {
  return (size_t)stage_buffers(dpad, fold, nq) * 32 * ns * (dpad == 16 ? 32 : dpad * 2 + 16) +
         (fold ? 0 : (size_t)stage_buffers(dpad, fold, nq) * 32 * ns * sizeof(uint2)) +
         (size_t)w * nq * qcap * 64 * sizeof(uint2);
}

// At least two waves per SIMD for lists of up to 32 entries and rows of up to
// 128 elements: the register budget then stays within 256 per lane, which
// lets the compiler keep the MFMA accumulators in VGPRs (no AGPR copies
// around every sub-tile).  16-entry lists on 16-element rows fit three waves
// (at most 168 registers; their 48 KiB of LDS also admits three workgroups
// per CU), and four on folded rows (at most 128 registers; 16-wave
// workgroups, see launch_mtile; the unfolded row's seed MFMA and parts would
// spill there).  64-entry lists and wider rows need more
// registers and run one wave per SIMD.
template <int DPAD, bool FOLD, int R>
__host__ __device__ constexpr int min_waves() {
  return R >= 32 || DPAD >= 256 ? 1 : (DPAD == 16 && R <= 8 ? (FOLD ? 4 : 3) : 2);
}

template <typename ET, int DPAD, bool FOLD, int R, int W, int NS, int NG, int NQ>
__global__ void __launch_bounds__(W * 64)
    __attribute__((amdgpu_waves_per_eu(min_waves<DPAD, FOLD, R>())))
mtile_kernel(Args a, int64_t q_begin, int64_t q_rows) {
  using V = typename Frag<ET>::V;
  using LY = Layout<DPAD, FOLD>;
  static_assert(NQ == 1 || (NG == 1 && LY::wide), "two query groups: wide rows, one sub-tile");
  static_assert(NG <= NS && NS % NG == 0, "fast-path groups tile the stage");
  constexpr int kQCap = queue_slots<R, NQ>();
  constexpr int KC = LY::k16;
  constexpr bool kInterleave = NG == 1 && KC >= 16;
  constexpr int kAhead = NQ > 1 ? 2 : 4;  // A fragments in flight ahead of the MFMA chain
  constexpr int ROWB = LY::rowb;
  constexpr bool SWZ = ROWB == 32;
  constexpr int TR = 32 * NS;  // reference rows per stage
  constexpr int STAGE = TR * ROWB;
  constexpr int CPR = LY::cpr;
  constexpr int CHUNKS = TR * CPR;
  constexpr int NT = W * 64;
  constexpr int NL = (CHUNKS + NT - 1) / NT;
  static_assert(NL <= 16, "staged chunks per thread");
  constexpr bool DL = DPAD >= 512 && !FOLD;  // direct staging
  constexpr int NBUF = stage_buffers(DPAD, FOLD, NQ);
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* stage = smem;
  uint2* hnb = (uint2*)(smem + NBUF * STAGE);  // plain layout: seed parts of the staged rows
  uint2* qbase = (uint2*)(smem + NBUF * STAGE + (FOLD ? 0 : NBUF * TR * sizeof(uint2)));

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, col = lane & 31;
  if (a.ctrl->nonfinite) return;  // uniform over the grid
  // This lane's queue of query group u: qbase + ((wave NQ + u) kQCap + i) 64 + lane.
  uint2* const myq0 = qbase + wave * NQ * kQCap * 64 + lane;

  // The wave's queries: NQ groups of 32 from q0 on (group u: q0 + 32 u ..).
  const int64_t group = (int64_t)blockIdx.x * W + wave;
  const bool active = group * 32 * NQ < q_rows;  // uniform per wave
  const int64_t q0 = q_begin + group * 32 * NQ;
  // blockIdx.y: the reference split, or with the tail split (a.parts > 1,
  // one split) the piece of the scan order this workgroup takes.
  const int split = blockIdx.y;
  const bool pieces = a.parts > 1;
  const int64_t r_begin = pieces ? 0 : (int64_t)split * a.split_len;
  const int64_t r_end = r_begin + a.split_len < a.nr ? r_begin + a.split_len : a.nr;
  const int64_t r_end32 = (r_end + 31) & ~(int64_t)31;  // rows < r_end32 exist (padded copy)
  const bool selfq = a.exclude_self != 0;

  // Query operand: NQ groups of 32 queries, lane holds column col, k-half h;
  // in the fold layout the seed columns carry the constant c.  A group past
  // the block's rows loads the first group's rows (its lists are never written).
  V bq[NQ][KC];
  {
#pragma unroll
    for (int u = 0; u < NQ; ++u) {
      const bool live = active && group * 32 * NQ + 32 * u < q_rows;
      const ET* qrow = (const ET*)a.xq_q + (live ? q0 + 32 * u + col : active ? q0 + col : 0) *
                                               (int64_t)DPAD;
#pragma unroll
      for (int c = 0; c < KC; ++c)
        bq[u][c] = *reinterpret_cast<const V*>(qrow + 16 * c + 8 * h);
    }
    if constexpr (LY::wide) {
      // One wave per SIMD: the operand lives in AGPRs, which the MFMA reads
      // as its B operand directly.  Left to itself the compiler keeps it in
      // VGPRs, spills it to AGPRs under the lists' register pressure and
      // copies it back before every MFMA (about 110 copies per sub-tile at
      // rows of 512 elements).
#pragma unroll
      for (int u = 0; u < NQ; ++u)
#pragma unroll
        for (int c = 0; c < KC; ++c) asm volatile("" : "+a"(bq[u][c]));
    }
    if constexpr (FOLD) {
      const ET cf = (ET)(float)fold_const(std::is_same<ET, _Float16>::value ? TOD_PREC_FP16
                                                                           : TOD_PREC_BF16);
      if (h) {
        V v;
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = e < 4 ? cf : (ET)0.0f;
        bq[0][0] = v;
      }
    }
  }

  // Per query group u: the list, the threshold (a pair survives iff acc >
  // thr[u]) and the entries in this lane's queue.
  uint64_t L[NQ][R];
  float thr[NQ];
  int cnt[NQ];
#pragma unroll
  for (int u = 0; u < NQ; ++u) {
#pragma unroll
    for (int i = 0; i < R; ++i) L[u][i] = kEmpty;
    thr[u] = -INFINITY;
    cnt[u] = 0;
  }

  // Stage staging: every thread moves up to NL 16-byte chunks.  Rows past the
  // split's padded end are clamped to its last row: they are loaded but never
  // read back.  Rows of 256 or more elements (one 32-row sub-tile per stage,
  // one wave per SIMD, registers to spare) are loaded two stages ahead into
  // two register sets with fixed roles; shorter rows one stage ahead.
  constexpr bool PF2 = DPAD >= 256 && !DL;
  const unsigned char* xr_bytes = (const unsigned char*)a.xq_r;
  uint4 st[DL ? 1 : NL], su[PF2 ? NL : 1];
#pragma unroll
  for (int i = 0; i < (DL ? 1 : NL); ++i) st[i] = make_uint4(0, 0, 0, 0);
#pragma unroll
  for (int i = 0; i < (PF2 ? NL : 1); ++i) su[i] = make_uint4(0, 0, 0, 0);
  static_assert(TR / 2 <= NT, "the seed parts of two rows per thread");
  uint4 sth = make_uint4(0, 0, 0, 0), suh = sth;

  // A fragment of sub-tile s, 16-wide k-step c: row col, elements 16c + 8h..+7.
  // 32-byte rows store the two halves of row r swapped where bits 2 and 3 of
  // r differ (swz), so that the 8 or 16 lanes served together by a 16-byte
  // LDS read fall into distinct banks; the swap depends on col only.
  const int ahalf = SWZ ? 16 * (h ^ swz(col)) : 16 * h;
  auto afrag = [&](const unsigned char* buf, int s, int c) {
    return *reinterpret_cast<const V*>(buf + (32 * s + col) * ROWB + 32 * c + ahalf);
  };
  // Seed MFMA operand B (plain layout): c in k rows 0..3, which lanes of
  // half 0 hold; zero elsewhere.
  V bseed;
  {
    const ET cf = (ET)(float)fold_const(std::is_same<ET, _Float16>::value ? TOD_PREC_FP16
                                                                         : TOD_PREC_BF16);
#pragma unroll
    for (int e = 0; e < 8; ++e) bseed[e] = (h == 0 && e < 4) ? cf : (ET)0.0f;
  }
  // Accumulator seeds of sub-tile s: -N_j/2 of rows 8g + 4h + 0..3.  Plain
  // layout: the seed MFMA on row col's parts (lanes of half 1 read them too;
  // their B is zero); zero in the fold layout, where the data MFMA adds them.
  auto seed = [&](const uint2* hn, int s) {
    f32x16 v;
#pragma unroll
    for (int r = 0; r < 16; ++r) v[r] = 0.0f;
    if constexpr (!FOLD) {
      const uint2 raw = hn[32 * s + col];
      const V ps = __builtin_bit_cast(V, make_uint4(raw.x, raw.y, 0u, 0u));
      v = mfma<ET>(ps, bseed, v);
    }
    return v;
  };
  // Rows past the split and the query's own row (self exclusion) never survive.
  // Row indices fit in 32 bits (at most 2^31 - 1 rows), so the tests are
  // 32-bit scalar compares; the row limit is one value per sub-tile (rows >=
  // lim are past the split).
  const uint32_t q0u = (uint32_t)q0, endu = (uint32_t)r_end;
  // qu: first query of the accumulator's query group.
  auto mask = [&](f32x16& v, uint32_t ts, uint32_t qu) {
    const bool diag = selfq && ts == qu;
    const uint32_t rem = ts < endu ? endu - ts : 0u;
    if (diag || rem < 32u) {
      const int lim = rem < 32u ? (int)rem : 32;
      int hb = 4 * h;
      asm volatile("" : "+v"(hb));
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = hb + out_row_c(r);
        if (row >= lim || (diag && row == col)) v[r] = -INFINITY;
      }
    }
  };
  // Maximum of the 16 accumulators as two partial maxima (7 max3 each): a
  // group of sub-tiles then combines 2 NG values, which costs fewer
  // instructions than combining NG finished maxima.
  struct Max2 {
    float f, g;
  };
  auto max16p = [](const f32x16& v) {
    const float a = max3f(v[0], v[1], v[2]), b = max3f(v[3], v[4], v[5]);
    const float c = max3f(v[6], v[7], v[8]), d = max3f(v[9], v[10], v[11]);
    const float e = max3f(v[12], v[13], v[14]);
    return Max2{max3f(a, b, c), max3f(d, e, v[15])};
  };
  auto max16 = [&](const f32x16& v) {
    const Max2 p = max16p(v);
    return max3f(p.f, p.g, p.g);
  };
  // Merge the first kMerge queue entries of every lane into the lists, move
  // the rest (at most kQCap - kMerge) to the front and tighten the threshold.
  // (U: std::integral_constant of the query group.)
  auto flush = [&](auto U) __attribute__((always_inline)) {
    constexpr int u = decltype(U)::value;
    uint2* const myq = myq0 + u * kQCap * 64;
    merge_queues<R>(L[u], myq, cnt[u], h);
#pragma unroll
    for (int i = kMerge; i < kQCap; ++i)
      if (i < cnt[u]) myq[(i - kMerge) * 64] = myq[i * 64];
    cnt[u] = cnt[u] > kMerge ? cnt[u] - kMerge : 0;
    const uint64_t last = L[u][R - 1];
    const uint64_t t = xchg64(last, h);
    thr[u] = thr_of(h ? last : t);
  };
  // Append this lane's survivors of a sub-tile to its queue.
  //   16-slot queue: half a sub-tile at a time, merging whenever the half
  //   could overflow it (one merge site: the halves are a loop).
  //   28-slot queue: room for the whole sub-tile is made first; then each
  //   quarter costs a max, a compare and a uniform branch unless some lane's
  //   value beats its threshold.
  // An append writes the next free slot unconditionally and advances the
  // count only for a survivor (no exec-mask branch per value); the room made
  // beforehand keeps every written slot inside the queue.
  // (v by value, halves as whole vectors: a per-element choice between
  // v[r] and v[8 + r] on a loop counter can become a dynamic index, which
  // puts the accumulators in scratch memory.)
  auto insert = [&](auto U, const f32x16 v, uint32_t ts) __attribute__((always_inline)) {
    constexpr int u = decltype(U)::value;
    uint2* const myq = myq0 + u * kQCap * 64;
    uint32_t tb = ts + 4u * (uint32_t)h;  // row id of accumulator r: tb + out_row_c(r)
    asm volatile("" : "+v"(tb));
    if constexpr (kQCap == 16) {
      typedef float f32x8 __attribute__((ext_vector_type(8)));
      const f32x8 lo = __builtin_shufflevector(v, v, 0, 1, 2, 3, 4, 5, 6, 7);
      const f32x8 hi = __builtin_shufflevector(v, v, 8, 9, 10, 11, 12, 13, 14, 15);
#pragma unroll 1
      for (int hf = 0; hf < 2; ++hf) {
        const f32x8 cur = hf ? hi : lo;
        const float mh = max3f(max3f(cur[0], cur[1], cur[2]), max3f(cur[3], cur[4], cur[5]),
                               max3f(cur[6], cur[7], cur[7]));
        if (!__ballot(mh > thr[u])) continue;
        if (__ballot(cnt[u] > kQCap - 8)) flush(U);
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          myq[cnt[u] * 64] = make_uint2(__float_as_uint(cur[r]),
                                        tb + 16u * (uint32_t)hf + (uint32_t)out_row_c(r));
          cnt[u] += cur[r] > thr[u] ? 1 : 0;
        }
      }
    } else {
      if (__ballot(cnt[u] > kQCap - 16)) flush(U);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float mq = max3f(max3f(v[4 * q], v[4 * q + 1], v[4 * q + 2]), v[4 * q + 3], v[4 * q + 3]);
        if (__ballot(mq > thr[u])) {
#pragma unroll
          for (int r = 4 * q; r < 4 * q + 4; ++r) {
            myq[cnt[u] * 64] = make_uint2(__float_as_uint(v[r]), tb + (uint32_t)out_row_c(r));
            cnt[u] += v[r] > thr[u] ? 1 : 0;
          }
        }
      }
    }
  };

#define TOD_MT_FETCH(T0, REG, REGH)                                                          \
  _Pragma("unroll") for (int i = 0; i < NL; ++i) {                                          \
    const int c = tid + i * NT;                                                             \
    if (CHUNKS % NT == 0 || c < CHUNKS) {                                                   \
      const int row = c / CPR, cc = c % CPR;                                                \
      const int64_t gr = (T0) + row < r_end32 ? (T0) + row : r_end32 - 1;                   \
      REG[i] = *reinterpret_cast<const uint4*>(xr_bytes + gr * (int64_t)(DPAD * 2) + cc * 16); \
    }                                                                                       \
  }                                                                                         \
  if (!FOLD && tid < TR / 2) {                                                              \
    const int64_t gr = (T0) + 2 * tid < r_end32 ? (T0) + 2 * tid : r_end32 - 2;             \
    REGH = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint2*>(a.hn_r) + gr);     \
  }
#define TOD_MT_PUT(B, REG, REGH)                                                             \
  _Pragma("unroll") for (int i = 0; i < NL; ++i) {                                          \
    const int c = tid + i * NT;                                                             \
    if (CHUNKS % NT == 0 || c < CHUNKS)                                                     \
      *reinterpret_cast<uint4*>(stage + (B) * STAGE + (c / CPR) * ROWB +                      \
                                ((c % CPR) ^ (SWZ ? swz(c / CPR) : 0)) * 16) = REG[i];      \
  }                                                                                         \
  if (!FOLD && tid < TR / 2) *reinterpret_cast<uint4*>(hnb + (B) * TR + 2 * tid) = REGH;

  // Direct staging (rows of 512 elements): each wave moves 8 whole rows (one
  // 1 KiB row per instruction) and the seed parts of 8 rows of a stage
  // straight into LDS.
  // The rows a wave stages depend on the wave only, so their addresses are
  // formed in scalar registers (one wave index read through readfirstlane,
  // used by the staging alone); only the lane's 16-byte offset is a vector
  // value.  A stage starts at a multiple of 32 below the split's end, so all
  // its 32 rows exist in the padded copy.  dl_row(i) issues row i (i < 8) or
  // the seeds (i = 8) of the stage set by dl_t0 / dl_b.
  const uint32_t lbase = lds_off(smem);
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  int64_t dl_t0 = 0;
  int dl_b = 0;
  auto dl_row = [&](int i) __attribute__((always_inline)) {
    if (i < TR / W) {
      const int r = wv + W * i;
      dma16(xr_bytes + (dl_t0 + r) * (int64_t)(DPAD * 2) + lane * 16,
            lbase + dl_b * STAGE + r * ROWB);
    } else if (lane < 4) {  // the seed parts of 8 rows: 64 bytes
      dma16((const unsigned char*)(reinterpret_cast<const uint2*>(a.hn_r) + dl_t0 + 8 * wv) +
                lane * 16,
            lbase + NBUF * STAGE + (dl_b * TR + 8 * wv) * (int)sizeof(uint2));
    }
  };
  constexpr int kDlRows = TR / W + 1;  // staging loads per wave and stage

  // One stage: its sub-tiles from LDS buffer b.  With direct staging the
  // loads of the stage set by dl_t0 / dl_b are issued between the MFMAs of
  // the chain (one after every third k-step), where the wave would otherwise
  // wait for its own MFMAs.
  auto stage_body = [&](int64_t t0, int b) __attribute__((always_inline)) {
    const unsigned char* buf = stage + b * STAGE;
    const uint2* hn = hnb + b * TR;
    if (!active) return;
    const uint32_t t0u = (uint32_t)t0;
    const uint32_t avail = endu - t0u;  // every scanned stage starts below r_end
    const int live = avail < (uint32_t)TR ? (int)((avail + 31) >> 5) : NS;
    // Only a stage holding the diagonal sub-tile or the split's end needs the
    // masking code; the test is made once per stage, on scalars.
    // (Query group u's diagonal sub-tile starts at row q0 + 32 u.)
    bool diag_here = false;
#pragma unroll
    for (int u = 0; u < NQ; ++u) diag_here = diag_here || q0u + 32u * u - t0u < (uint32_t)TR;
    const bool smask = (selfq && diag_here) || avail < (uint32_t)TR;
    // Fast path over NG sub-tiles (independent MFMA chains, one reduction),
    // with no insertion code.  All A fragments and seeds of the group are read
    // before the first MFMA, so that one LDS round trip covers the group's
    // MFMA chains.  Long rows (one wave per SIMD, nothing else to overlap
    // with) keep kAhead fragments in flight ahead of the MFMA chain instead:
    // the LDS reads of later k-steps then run under the MFMAs of earlier ones.
    auto group = [&](int g0) __attribute__((always_inline)) {
      constexpr std::integral_constant<int, 0> Z{};
      f32x16 acc[NG][NQ];
      if constexpr (DL) {
        // One sub-tile.  The staging loads are ordered against the LDS reads
        // (asm with side effects), so the reads ahead of the chain are
        // written out in the order they are to run: fragment c + kAhead is
        // read as fragment c enters the chain, and after every third k-step
        // one staging row is issued.
        static_assert(NG == 1, "one sub-tile per stage");
        acc[0][0] = seed(hn, g0);  // its parts are read first
        V w[kAhead];
#pragma unroll
        for (int c = 0; c < kAhead; ++c) w[c] = afrag(buf, g0, c);
#pragma unroll
        for (int u = 1; u < NQ; ++u) acc[0][u] = acc[0][0];
#pragma unroll
        for (int c = 0; c < KC; ++c) {
          const V cur = w[c % kAhead];
          if (c + kAhead < KC) w[c % kAhead] = afrag(buf, g0, c + kAhead);
#pragma unroll
          for (int u = 0; u < NQ; ++u) acc[0][u] = mfma<ET>(cur, bq[u][c], acc[0][u]);
          if (c % 3 == 1 && c / 3 < TR / W) dl_row(c / 3);
        }
      } else {
        // (Addresses from the group's first row: the sub-tile offsets are
        // then immediate offsets of the LDS reads.)
        const unsigned char* gbuf = buf + g0 * (32 * ROWB);
        const uint2* ghn = hn + 32 * g0;
        V af[NG][KC];
#pragma unroll
        for (int s = 0; s < NG; ++s) {
#pragma unroll
          for (int c = 0; c < KC; ++c) af[s][c] = afrag(gbuf, s, c);
          acc[s][0] = seed(ghn, s);
#pragma unroll
          for (int u = 1; u < NQ; ++u) acc[s][u] = acc[s][0];
        }
        // Every A fragment feeds the MFMAs of all NQ query groups.
#pragma unroll
        for (int c = 0; c < KC; ++c)
#pragma unroll
          for (int s = 0; s < NG; ++s)
#pragma unroll
            for (int u = 0; u < NQ; ++u) acc[s][u] = mfma<ET>(af[s][c], bq[u][c], acc[s][u]);
      }
      // (Plain layout: one LDS read and one MFMA more per sub-tile, the seed's.)
      constexpr int kSeed = FOLD ? 0 : 1;
      if constexpr (kInterleave) {
        __builtin_amdgcn_sched_group_barrier(0x100, kAhead + kSeed, 0);
        if constexpr (kSeed) __builtin_amdgcn_sched_group_barrier(0x008, kSeed, 0);
#pragma unroll
        for (int c = 0; c < KC - kAhead; ++c) {
          __builtin_amdgcn_sched_group_barrier(0x008, NQ, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NQ * kAhead, 0);
      } else {
        __builtin_amdgcn_sched_group_barrier(0x100, NG * (KC + kSeed), 0);
        __builtin_amdgcn_sched_group_barrier(0x008, NG * (NQ * KC + kSeed), 0);
      }
      // Masks first (one branch per group), then the NG x NQ independent max
      // trees, which the scheduler interleaves.
      if (smask) {
#pragma unroll
        for (int s = 0; s < NG; ++s)
#pragma unroll
          for (int u = 0; u < NQ; ++u)
            mask(acc[s][u], t0u + 32u * (uint32_t)(g0 + s), q0u + 32u * (uint32_t)u);
      }
      // (Sub-tiles past the split are fully masked.)
      Max2 mp[NG][NQ];
#pragma unroll
      for (int s = 0; s < NG; ++s)
#pragma unroll
        for (int u = 0; u < NQ; ++u) mp[s][u] = max16p(acc[s][u]);
      float ms[NG][NQ];
#pragma unroll
      for (int s = 0; s < NG; ++s)
#pragma unroll
        for (int u = 0; u < NQ; ++u) ms[s][u] = max3f(mp[s][u].f, mp[s][u].g, mp[s][u].g);
      if constexpr (NQ > 1) {
        // One sub-tile, NQ query groups: insert each group's survivors from
        // its accumulators.
        bool any = false;
#pragma unroll
        for (int u = 0; u < NQ; ++u) any = any || ms[0][u] > thr[u];
        if (!__ballot(any)) return;
        uint32_t ts = t0u + 32u * (uint32_t)g0;
        asm volatile("" : "+s"(ts));  // ids formed here (see below)
        static_assert(NQ == 2, "two query groups");
        constexpr std::integral_constant<int, 1> One{};
        if (__ballot(ms[0][0] > thr[0])) insert(Z, acc[0][0], ts);
        if (__ballot(ms[0][1] > thr[1])) insert(One, acc[0][1], ts);
        return;
      }
      // Group maximum from the 2 NG partial maxima (the per-sub-tile maxima
      // above are formed only where the slow path reads them).
      float pv[2 * NG];
#pragma unroll
      for (int s = 0; s < NG; ++s) {
        pv[2 * s] = mp[s][0].f;
        pv[2 * s + 1] = mp[s][0].g;
      }
      float m = pv[0];
#pragma unroll
      for (int i = 1; i < 2 * NG; i += 2) m = max3f(m, pv[i], pv[i + 1 < 2 * NG ? i + 1 : i]);
      if (!__ballot(m > thr[0])) return;
      // Slow path: sub-tile by sub-tile.  Rows of several k-steps reuse the
      // group's accumulators, one copy of the insertion code per sub-tile (a
      // recomputation would put its LDS reads and MFMA chain on the latency
      // of every slow entry, which the workgroup's other waves wait out at the
      // next stage barrier).  Rows of one k-step recompute the sub-tile (one
      // MFMA, bit-identical), which keeps the fast path's accumulators dead
      // after their reduction and the kernel at three waves per SIMD.
      const int gl = live - g0 < NG ? live - g0 : NG;
      if constexpr (NG > 1 && KC >= 2) {
#pragma unroll
        for (int s = 0; s < NG; ++s) {
          if (s >= gl || !__ballot(ms[s][0] > thr[0])) continue;
          uint32_t ts = t0u + 32u * (uint32_t)(g0 + s);
          asm volatile("" : "+s"(ts));  // ids formed here (see below)
          insert(Z, acc[s][0], ts);
        }
        return;
      }
#pragma unroll 1
      for (int s = 0; s < gl; ++s) {
        float msel = ms[0][0];
#pragma unroll
        for (int u = 1; u < NG; ++u) msel = s == u ? ms[u][0] : msel;
        if (!__ballot(msel > thr[0])) continue;
        uint32_t ts = t0u + 32u * (uint32_t)(g0 + s);
        // Opaque to the optimizer: otherwise it carries the 16 row ids
        // ts + out_row(r, h) through the fast path as per-lane induction
        // variables (16 additions per sub-tile) instead of forming them here.
        asm volatile("" : "+s"(ts));
        if constexpr (NG == 1) {
          insert(Z, acc[0][0], ts);
        } else {
          f32x16 a1 = seed(hn, g0 + s);
#pragma unroll
          for (int c = 0; c < KC; ++c) a1 = mfma<ET>(afrag(buf, g0 + s, c), bq[0][c], a1);
          if (smask) mask(a1, ts, q0u);
          insert(Z, a1, ts);
        }
      }
    };
    if constexpr (NG == NS) {
      group(0);
    } else {
#pragma unroll 1
      for (int g0 = 0; g0 < live; g0 += NG) group(g0);
    }
  };

  // Stage order.  With the grouped scan order (X against X, one split) the
  // workgroup starts at the stage holding the first row of the group of its
  // first query and wraps around; concurrent workgroups mostly share a group,
  // and so the stream they read.  Otherwise the split is scanned in order.
  const int nst = (int)((r_end - r_begin + TR - 1) / TR);
  int st0 = 0;
  if (a.cstart) {
    // The last group starting at or before p0 (starts ascend; an empty group
    // shares its start with the next one).
    const int p0 = (int)(q_begin + (int64_t)blockIdx.x * (W * 32 * NQ));
    int lo = 0, hi = a.groups;  // cstart[lo] <= p0 < cstart[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (a.cstart[mid] <= p0) lo = mid;
      else hi = mid;
    }
    st0 = (int)((a.cstart[lo] - r_begin) / TR);
  }
  // Tail split: piece `split` of `parts` takes the stages [ib, ib + nscan) of
  // the scan order.
  int nscan = nst;
  if (pieces) {
    // (64-bit products: up to 128 pieces with two runs of 64 splits.)
    const int ib = (int)((int64_t)split * nst / a.parts);
    nscan = (int)((int64_t)(split + 1) * nst / a.parts) - ib;
    st0 += ib;
    st0 = st0 >= nst ? st0 - nst : st0;
  }
  // First row of the i-th stage scanned (i < nscan + 2 <= nst + 2; stages past
  // the last one wrap round and are loaded but never read).
  auto t_of = [&](int i) -> int64_t {
    int s = st0 + i;
    s = s >= nst ? s - nst : s;
    s = s >= nst ? s - nst : s;
    return r_begin + (int64_t)s * TR;
  };

  if constexpr (DL) {
    // Rows of 512 elements: two stages ahead with three buffers, one stage
    // ahead with two.  The compiler-visible wait first retires the query
    // operand's loads, so that the compiler, which does not see the staging
    // loads, has no load of its own left to wait for.
    static_assert(TR == 8 * W && W == 4, "direct staging: 8 rows and their seed parts per wave");
    static_assert(KC >= 3 * (TR / W), "staging loads spread over the MFMA chain");
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    auto dl_issue = [&](int64_t t0, int b) __attribute__((always_inline)) {
      dl_t0 = t0;
      dl_b = b;
#pragma unroll
      for (int i = 0; i < kDlRows; ++i) dl_row(i);
    };
    // The seeds of stage (tn, bn) are loaded first (two lanes: a branch, kept
    // out of the chain); a stage body issues the rows inside its chain, and a
    // wave with no queries has no chain and issues them itself.
    auto dl_body = [&](int64_t t0, int b, int64_t tn, int bn) __attribute__((always_inline)) {
      dl_t0 = tn;
      dl_b = bn;
      dl_row(TR / W);
      if (active) stage_body(t0, b);
      else
#pragma unroll
        for (int i = 0; i < TR / W; ++i) dl_row(i);
    };
    if constexpr (NBUF == 3) {
      dl_issue(t_of(0), 0);
      dl_issue(t_of(1), 1);
      dl_barrier<kDlRows>();
      for (int it = 0; it < nscan; ++it) {
        // Buffer (it + 2) % 3 was last read in trip it - 1, before its barrier.
        dl_body(t_of(it), it % 3, t_of(it + 2), (it + 2) % 3);
        dl_barrier<kDlRows>();
      }
    } else {
      dl_issue(t_of(0), 0);
      dl_barrier<0>();
      for (int it = 0; it < nscan; ++it) {
        // Buffer (it + 1) & 1 was last read in trip it - 1, before its barrier.
        dl_body(t_of(it), it & 1, t_of(it + 1), (it + 1) & 1);
        dl_barrier<0>();
      }
    }
    // No staging write may outlive the workgroup's LDS allocation.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  } else {
  TOD_MT_FETCH(t_of(0), st, sth)
  TOD_MT_PUT(0, st, sth)
  if constexpr (PF2) {
    // Two stages per trip: each register set has a fixed role in straight-line
    // code, so every wait is for the older set only, and the stage barrier
    // (no release fence) leaves the newer set's loads in flight.
    TOD_MT_FETCH(t_of(1), su, suh)
    stage_barrier();
    for (int it = 0;;) {
      TOD_MT_FETCH(t_of(it + 2), st, sth)
      stage_body(t_of(it), 0);
      TOD_MT_PUT(1, su, suh)
      stage_barrier();
      if (++it >= nscan) break;
      TOD_MT_FETCH(t_of(it + 2), su, suh)
      stage_body(t_of(it), 1);
      TOD_MT_PUT(0, st, sth)
      stage_barrier();
      if (++it >= nscan) break;
    }
  } else {
    __syncthreads();
    for (int it = 0; it < nscan; ++it) {
      TOD_MT_FETCH(t_of(it + 1), st, sth)
      stage_body(t_of(it), it & 1);
      TOD_MT_PUT((it + 1) & 1, st, sth)
      __syncthreads();
    }
  }
  }
#undef TOD_MT_FETCH
#undef TOD_MT_PUT
  if (active) {
    static_for<0, NQ>([&](auto U) __attribute__((always_inline)) {
      constexpr int u = decltype(U)::value;
      while (__ballot(cnt[u] > 0)) flush(U);
      const int64_t ql = group * 32 * NQ + 32 * u + col;
      if (ql < q_rows) {
        uint64_t* dst =
            a.partial + (ql * (pieces ? a.parts : a.splits) + split) * (2 * R) + h * R;
#pragma unroll
        for (int i = 0; i < R; ++i) {
          const uint64_t e = L[u][i];
          dst[i] = e == kEmpty ? kEmpty : make_entry(-2.0f * acc_of(e), (uint32_t)e);
        }
      }
    });
  }
}

// Sub-tiles per fast-path group: four for rows of up to 32 elements (one
// k-step or two), two (the whole stage) for rows of 64, one otherwise.  Two
// independent MFMA chains at 64 took the C3 tile from 198 to 184 ms.
//
// Folded rows with 16-entry lists run four waves per SIMD (min_waves) in one
// workgroup of 16 waves per CU, 512 queries, with stages of 16 sub-tiles:
// the stage pair (32 KiB) and the 16 queues (128 KiB) fill the CU's 160 KiB,
// and every staged row serves 512 queries.  At 4 x 10^6 rows: 666 ms with
// three waves per SIMD (4 waves a workgroup, stages of eight), 647 ms with
// four (stages of four, four workgroups per CU), 591 ms with 8-wave
// workgroups and stages of eight, 580 ms in this form (622 ms with stages
// of eight).  Rows of 64 elements with 32-entry lists (28-slot queues) take
// 8-wave workgroups, one per CU, with stages of four sub-tiles (150 KiB of
// LDS): at 10^6 rows 180 -> 163 ms.  Rows of 32 elements keep 4-wave
// workgroups: 8 waves took that tile from 2.17 to 3.1-3.6 ms.
//
// Tail split: a block of G workgroups on a GPU that runs S of them at once
// ends with a round of G mod S workgroups that leaves most of the GPU idle.
// With one reference split, those workgroups' scans are cut into P pieces on
// P times as many workgroups (tail_pieces picks P), in a second launch whose
// lists go to the tail region.
template <typename ET, int DPAD, bool FOLD, int R,
          int W = (FOLD && R <= 8 ? 16 : (DPAD == 64 && !FOLD && R == 16) ? 8 : 4),
          int NS = (FOLD && R <= 8 ? 16 : (DPAD == 64 && !FOLD && R == 16) ? 4 : Layout<DPAD, FOLD>::ns),
          int NG = (DPAD <= 32 ? 4 : (DPAD == 64 ? 2 : 1)), int NQ = query_groups(DPAD, FOLD, R)>
hipError_t launch_mtile(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                        hipStream_t st, TileTail* tail) {
  const size_t lds = lds_bytes(DPAD, FOLD, W, NS, queue_slots<R, NQ>(), NQ);
  static_assert(lds_bytes(DPAD, FOLD, W, NS, queue_slots<R, NQ>(), NQ) <= 160 * 1024,
                "LDS per workgroup");
  const auto kern = mtile_kernel<ET, DPAD, FOLD, R, W, NS, NG, NQ>;
  constexpr int QW = W * 32 * NQ;  // queries per workgroup
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const int64_t wgs = (q_rows + QW - 1) / QW;
  if (p.runs > 1) {
    // Runs: every workgroup's scan in runs x S pieces of the scan order, each
    // piece's list at partial + (query (runs S) + piece) K'/runs, i.e. the
    // recheck's S lists of K' entries, `runs` ascending runs each.
    Args b = a;
    b.parts = p.runs * p.splits;
    b.splits = 1;
    b.split_len = a.nr;
    hipLaunchKernelGGL(kern, dim3((unsigned)wgs, (unsigned)b.parts), dim3(W * 64), lds, st, b,
                       q_begin, q_rows);
    if (tail) {
      tail->q0 = q_rows;
      tail->parts = 1;
    }
    return hipGetLastError();
  }
  int64_t main_wgs = wgs;
  int parts = 1;
  if (p.splits == 1 && p.tail_parts > 1 && a.ptail) {
    int dev = 0, cus = 0, per = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, (const void*)kern, W * 64, lds) ==
            hipSuccess &&
        cus > 0 && per > 0) {
      const int64_t slots = (int64_t)cus * per;
      const int64_t tw = wgs % slots;
      const int64_t trows = q_rows - (wgs - tw) * QW;
      const int64_t nst = (a.nr + 32 * NS - 1) / (32 * NS);
      parts = tail_pieces(tw, slots, cus, p.tail_parts, p.tail_auto != 0, nst, p.tail_lists,
                          trows);
      if (parts > 1) main_wgs = wgs - tw;
    } else {
      (void)hipGetLastError();  // no occupancy figures: no tail split
    }
  }
  const int64_t main_rows = main_wgs * QW < q_rows ? main_wgs * QW : q_rows;
  if (main_wgs > 0) {
    hipLaunchKernelGGL(kern, dim3((unsigned)main_wgs, (unsigned)p.splits), dim3(W * 64), lds, st,
                       a, q_begin, main_rows);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (tail) {
    tail->q0 = parts > 1 ? main_rows : q_rows;
    tail->parts = parts;
  }
  if (parts == 1) return hipSuccess;
  Args b = a;
  b.partial = a.ptail;
  b.parts = parts;
  hipLaunchKernelGGL(kern, dim3((unsigned)(wgs - main_wgs), (unsigned)parts), dim3(W * 64), lds,
                     st, b, q_begin + main_rows, q_rows - main_rows);
  return hipGetLastError();
}

template <typename ET, int DPAD, bool FOLD>
hipError_t launch_mtile_r(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                          hipStream_t st, TileTail* tail) {
  switch (p.kprime) {
    case 16: return launch_mtile<ET, DPAD, FOLD, 8>(p, a, q_begin, q_rows, st, tail);
    case 32: return launch_mtile<ET, DPAD, FOLD, 16>(p, a, q_begin, q_rows, st, tail);
    case 64: return launch_mtile<ET, DPAD, FOLD, 32>(p, a, q_begin, q_rows, st, tail);
    case 128:  // two runs of 64 (rows of 256 or more elements)
      if constexpr (DPAD >= 256 && !FOLD)
        return p.runs == 2 ? launch_mtile<ET, DPAD, FOLD, 32>(p, a, q_begin, q_rows, st, tail)
                           : hipErrorInvalidValue;
      else
        return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

template <typename ET>
hipError_t launch_mtile_any(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                            hipStream_t st, TileTail* tail) {
  if (p.fold) return p.dpad_t == 16 ? launch_mtile_r<ET, 16, true>(p, a, q_begin, q_rows, st, tail)
                                    : hipErrorInvalidValue;
  switch (p.dpad_t) {
    case 16: return launch_mtile_r<ET, 16, false>(p, a, q_begin, q_rows, st, tail);
    case 32: return launch_mtile_r<ET, 32, false>(p, a, q_begin, q_rows, st, tail);
    case 64: return launch_mtile_r<ET, 64, false>(p, a, q_begin, q_rows, st, tail);
    case 128: return launch_mtile_r<ET, 128, false>(p, a, q_begin, q_rows, st, tail);
    case 256: return launch_mtile_r<ET, 256, false>(p, a, q_begin, q_rows, st, tail);
    case 512: return launch_mtile_r<ET, 512, false>(p, a, q_begin, q_rows, st, tail);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mt
}  // namespace tod
