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
// some accumulator beats it.  Survivors are appended to a 16-slot LDS queue of
// their lane.  When a queue could overflow, the whole wave merges: every lane
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

constexpr int kQCap = 16;  // queue slots per lane
constexpr int kHalf = 8;   // accumulators appended between capacity checks

// Value of v in the partner lane (lane ^ 32).
__device__ __forceinline__ uint32_t xchg32(uint32_t v, int h) {
  const auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return h ? p[0] : p[1];
}
__device__ __forceinline__ uint64_t xchg64(uint64_t v, int h) {
  return ((uint64_t)xchg32((uint32_t)(v >> 32), h) << 32) | xchg32((uint32_t)v, h);
}

// Ascending compare-exchange.
__device__ __forceinline__ void ce(uint64_t& x, uint64_t& y) {
  const bool sw = y < x;
  const uint64_t lo = sw ? y : x;
  const uint64_t hi = sw ? x : y;
  x = lo;
  y = hi;
}

// Keep min (h == 0) or max (h == 1) of x and the partner's value p.
__device__ __forceinline__ uint64_t keep(uint64_t x, uint64_t p, int h) {
  const bool take = h ? (x < p) : (p < x);
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

__device__ __forceinline__ float max3f(float a, float b, float c) {
  float d;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "v"(c));
  return d;
}

// Reference row (0..31 within the sub-tile) of accumulator r in this lane
// (32x32 MFMA output layout: column = lane % 32).
__device__ __forceinline__ int out_row(int r, int h) { return 8 * (r >> 2) + 4 * h + (r & 3); }

// Merge every lane's queue into its pair's list (all 64 lanes take part).
// list: this lane's R entries of the pair's ascending K' = 2R list.
template <int R>
__device__ __forceinline__ void merge_queues(uint64_t (&L)[R], const uint2* myq, int cnt, int h) {
  constexpr int M = kQCap;
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
      L[i] = o < L[i] ? o : L[i];
    }
  } else if constexpr (R < M) {
    // Q[2R-1-e] lies in lane q: for lane q itself at index 2R-1-i, for lane
    // q + 32 (e = R + i) at index R-1-i of the partner.
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const uint64_t p = xchg64(Q[R - 1 - i], h);
      const uint64_t o = h ? p : Q[2 * R - 1 - i];
      L[i] = o < L[i] ? o : L[i];
    }
  } else {
    static_assert(R == 2 * M, "list length per lane must be 8, 16 or 32");
    // The queue has 2M = R entries, so only lane q + 32's entries can change:
    // e = R + i pairs with Q[2M-1-i], which for i < M is this lane's Q[M-1-i]
    // and for i >= M the partner's Q[2M-1-i].
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const uint64_t o = i < M ? Q[M - 1 - i] : xchg64(Q[2 * M - 1 - i], h);
      const uint64_t m = o < L[i] ? o : L[i];
      L[i] = h ? m : L[i];
    }
  }
  // The 2R entries now form a bitonic sequence over the pair: one cross-lane
  // stage, then sort each half.
#pragma unroll
  for (int i = 0; i < R; ++i) L[i] = keep(L[i], xchg64(L[i], h), h);
  clean_asc<R>(L);
}

// LDS row stride of a staged reference row.  Rows of 32 bytes are read
// conflict-free as they are; longer rows get 16 bytes of padding so that the
// eight rows read by one group of lanes fall in different banks.
__host__ __device__ constexpr int row_bytes(int dpad) { return dpad == 16 ? 32 : dpad * 2 + 16; }

__host__ __device__ constexpr size_t lds_bytes(int dpad, int w, int ns) {
  return (size_t)2 * 32 * ns * row_bytes(dpad) + (size_t)2 * 32 * ns * sizeof(float) +
         (size_t)w * kQCap * 64 * sizeof(uint2);
}

// Two waves per SIMD: the register budget stays within 256 per lane, which
// lets the compiler keep the MFMA accumulators in VGPRs (no AGPR copies
// around every sub-tile).
template <typename ET, int DPAD, int R, int W, int NS, int NG>
__global__ void __launch_bounds__(W * 64) __attribute__((amdgpu_waves_per_eu(2)))
mtile_kernel(Args a, int64_t q_begin, int64_t q_rows) {
  using V = typename Frag<ET>::V;
  constexpr int KC = DPAD / 16;  // MFMA k-steps
  constexpr int ROWB = row_bytes(DPAD);
  constexpr int TR = 32 * NS;  // reference rows per stage
  constexpr int STAGE = TR * ROWB;
  constexpr int CPR = DPAD * 2 / 16;  // 16-byte chunks per row
  constexpr int CHUNKS = TR * CPR;
  constexpr int NL = (CHUNKS + W * 64 - 1) / (W * 64);
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* stage = smem;
  float* hnb = (float*)(smem + 2 * STAGE);
  uint2* qbase = (uint2*)(smem + 2 * STAGE + 2 * TR * sizeof(float));

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, col = lane & 31;
  if (a.ctrl->nonfinite) return;  // uniform over the grid
  const uint2* myq_r = qbase + wave * kQCap * 64 + lane;
  uint2* myq = qbase + wave * kQCap * 64 + lane;

  const int64_t group = (int64_t)blockIdx.x * W + wave;
  const bool active = group * 32 < q_rows;  // uniform per wave
  const int64_t q0 = q_begin + group * 32;
  const int split = blockIdx.y;
  const int64_t r_begin = (int64_t)split * a.split_len;
  const int64_t r_end = r_begin + a.split_len < a.nr ? r_begin + a.split_len : a.nr;
  const int64_t r_end32 = (r_end + 31) & ~(int64_t)31;  // rows < r_end32 exist (padded copy)
  const bool selfq = a.exclude_self != 0;

  // Query operand: 32 queries x DPAD, lane holds column col, k-half h.
  V bq[KC];
  {
    const ET* qrow = (const ET*)a.xq_q + (active ? q0 + col : 0) * (int64_t)DPAD;
#pragma unroll
    for (int c = 0; c < KC; ++c) bq[c] = *reinterpret_cast<const V*>(qrow + 16 * c + 8 * h);
  }

  uint64_t L[R];
#pragma unroll
  for (int i = 0; i < R; ++i) L[i] = kEmpty;
  float thr = -INFINITY;  // a pair survives iff acc > thr
  int cnt = 0;            // entries in this lane's queue

  // Stage staging: every thread moves NL 16-byte chunks.  Rows past the
  // split's padded end are clamped to its last row: they are loaded but never
  // read back, so every load and LDS write is unconditional.
  static_assert(CHUNKS % (W * 64) == 0, "stage chunks must divide evenly over the threads");
  static_assert(TR / 4 <= W * 64, "one float4 of seeds per thread");
  const unsigned char* xr_bytes = (const unsigned char*)a.xq_r;
  static_assert(NL >= 1 && NL <= 4, "one to four staged chunks per thread");
  uint4 st0 = make_uint4(0, 0, 0, 0), st1 = st0, st2 = st0, st3 = st0;
  float4 sth = make_float4(0.f, 0.f, 0.f, 0.f);
  auto chunk_src = [&](int64_t t0, int c) {
    const int row = c / CPR, cc = c % CPR;
    const int64_t gr = t0 + row < r_end32 ? t0 + row : r_end32 - 1;
    return reinterpret_cast<const uint4*>(xr_bytes + gr * (int64_t)(DPAD * 2) + cc * 16);
  };
  auto chunk_dst = [&](unsigned char* buf, int c) {
    return reinterpret_cast<uint4*>(buf + (c / CPR) * ROWB + (c % CPR) * 16);
  };
  auto fetch = [&](int64_t t0) {
    st0 = *chunk_src(t0, tid);
    if constexpr (NL > 1) st1 = *chunk_src(t0, tid + W * 64);
    if constexpr (NL > 2) st2 = *chunk_src(t0, tid + 2 * W * 64);
    if constexpr (NL > 3) st3 = *chunk_src(t0, tid + 3 * W * 64);
    if (tid < TR / 4) {
      const int64_t gr = t0 + 4 * tid < r_end32 ? t0 + 4 * tid : r_end32 - 4;
      sth = *reinterpret_cast<const float4*>(a.hn_r + gr);
    }
  };
  auto put = [&](int b) {
    unsigned char* buf = stage + b * STAGE;
    *chunk_dst(buf, tid) = st0;
    if constexpr (NL > 1) *chunk_dst(buf, tid + W * 64) = st1;
    if constexpr (NL > 2) *chunk_dst(buf, tid + 2 * W * 64) = st2;
    if constexpr (NL > 3) *chunk_dst(buf, tid + 3 * W * 64) = st3;
    if (tid < TR / 4) *reinterpret_cast<float4*>(hnb + b * TR + 4 * tid) = sth;
  };

  // Accumulator seeds -N_j/2 of sub-tile s (rows 8g + 4h + 0..3 of lane's half).
  auto seed = [&](const float* hn, int s) {
    f32x16 v;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 t = *reinterpret_cast<const float4*>(hn + 32 * s + 8 * g + 4 * h);
      v[4 * g + 0] = t.x;
      v[4 * g + 1] = t.y;
      v[4 * g + 2] = t.z;
      v[4 * g + 3] = t.w;
    }
    return v;
  };
  // A fragment of sub-tile s, k-step c: row col, elements 16c + 8h .. + 7.
  auto afrag = [&](const unsigned char* buf, int s, int c) {
    return *reinterpret_cast<const V*>(buf + (32 * s + col) * ROWB + 32 * c + 16 * h);
  };
  // Rows past the split and the query's own row (self exclusion) never survive.
  auto mask = [&](f32x16& v, int64_t ts) {
    const bool diag = selfq && ts == q0;
    if (diag || ts + 32 > r_end) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = out_row(r, h);
        if (ts + row >= r_end || (diag && row == col)) v[r] = -INFINITY;
      }
    }
  };
  auto max16 = [](const f32x16& v) {
    const float a = max3f(v[0], v[1], v[2]), b = max3f(v[3], v[4], v[5]);
    const float c = max3f(v[6], v[7], v[8]), d = max3f(v[9], v[10], v[11]);
    const float e = max3f(v[12], v[13], v[14]);
    return fmaxf(max3f(a, b, c), max3f(d, e, v[15]));
  };
  // Append this lane's survivors of a sub-tile to its queue, merging first
  // whenever a half could overflow it.
  auto insert = [&](const f32x16& v, int64_t ts) {
#pragma unroll 1
    for (int hf = 0; hf < 2; ++hf) {
      float cur[kHalf];
#pragma unroll
      for (int r = 0; r < kHalf; ++r) cur[r] = hf ? v[kHalf + r] : v[r];
      float mh = cur[0];
#pragma unroll
      for (int r = 1; r < kHalf; ++r) mh = fmaxf(mh, cur[r]);
      if (!__ballot(mh > thr)) continue;
      if (__ballot(cnt > kQCap - kHalf)) {
        merge_queues<R>(L, myq_r, cnt, h);
        cnt = 0;
        const uint64_t last = L[R - 1];
        const uint64_t t = xchg64(last, h);
        thr = thr_of(h ? last : t);
      }
#pragma unroll
      for (int r = 0; r < kHalf; ++r) {
        if (cur[r] > thr) {
          myq[cnt * 64] =
              make_uint2(__float_as_uint(cur[r]), (uint32_t)(ts + out_row(kHalf * hf + r, h)));
          ++cnt;
        }
      }
    }
  };

  fetch(r_begin);
  put(0);
  __syncthreads();
  int it = 0;
  for (int64_t t0 = r_begin; t0 < r_end; t0 += TR, ++it) {
    fetch(t0 + TR);  // past the end this reloads clamped rows nobody reads
    const int b = it & 1;
    const unsigned char* buf = stage + b * STAGE;
    const float* hn = hnb + b * TR;
    if (active) {
      const int live = r_end - t0 < TR ? (int)((r_end - t0 + 31) >> 5) : NS;
#pragma unroll 1
      for (int g0 = 0; g0 < live; g0 += NG) {
        // Fast path: NG sub-tiles at once (independent MFMA chains, one
        // reduction), with no insertion code.
        f32x16 acc[NG];
#pragma unroll
        for (int s = 0; s < NG; ++s) acc[s] = seed(hn, g0 + s);
#pragma unroll
        for (int c = 0; c < KC; ++c)
#pragma unroll
          for (int s = 0; s < NG; ++s) acc[s] = mfma<ET>(afrag(buf, g0 + s, c), bq[c], acc[s]);
        float ms[NG];
#pragma unroll
        for (int s = 0; s < NG; ++s) {
          mask(acc[s], t0 + 32 * (g0 + s));
          ms[s] = max16(acc[s]);  // sub-tiles past the split are fully masked
        }
        float m = ms[0];
#pragma unroll
        for (int s = 1; s < NG; ++s) m = fmaxf(m, ms[s]);
        if (__ballot(m > thr)) {
          // Slow path: sub-tile by sub-tile (one copy of the insertion and
          // merge code), recomputing the accumulators of each sub-tile that
          // holds a survivor.
          const int gl = live - g0 < NG ? live - g0 : NG;
#pragma unroll 1
          for (int s = 0; s < gl; ++s) {
            float msel = ms[0];
#pragma unroll
            for (int u = 1; u < NG; ++u) msel = s == u ? ms[u] : msel;
            if (!__ballot(msel > thr)) continue;
            const int64_t ts = t0 + 32 * (g0 + s);
            f32x16 a1 = seed(hn, g0 + s);
#pragma unroll
            for (int c = 0; c < KC; ++c) a1 = mfma<ET>(afrag(buf, g0 + s, c), bq[c], a1);
            mask(a1, ts);
            insert(a1, ts);
          }
        }
      }
    }
    put((it + 1) & 1);
    __syncthreads();
  }
  if (active) {
    if (__ballot(cnt > 0)) merge_queues<R>(L, myq_r, cnt, h);
    const int64_t ql = group * 32 + col;
    if (ql < q_rows) {
      uint64_t* dst = a.partial + (ql * a.splits + split) * (2 * R) + h * R;
#pragma unroll
      for (int i = 0; i < R; ++i) {
        const uint64_t e = L[i];
        dst[i] = e == kEmpty ? kEmpty : make_entry(-2.0f * acc_of(e), (uint32_t)e);
      }
    }
  }
}

template <typename ET, int DPAD, int R, int W = 4, int NS = (DPAD <= 32 ? 8 : (DPAD == 64 ? 4 : 2)),
          int NG = 2>
hipError_t launch_mtile(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                        hipStream_t st) {
  const size_t lds = lds_bytes(DPAD, W, NS);
  const auto kern = mtile_kernel<ET, DPAD, R, W, NS, NG>;
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const int64_t groups = (q_rows + 31) / 32;
  const dim3 grid((unsigned)((groups + W - 1) / W), (unsigned)p.splits);
  hipLaunchKernelGGL(kern, grid, dim3(W * 64), lds, st, a, q_begin, q_rows);
  return hipGetLastError();
}

template <typename ET, int DPAD>
hipError_t launch_mtile_r(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                          hipStream_t st) {
  switch (p.kprime) {
    case 16: return launch_mtile<ET, DPAD, 8>(p, a, q_begin, q_rows, st);
    case 32: return launch_mtile<ET, DPAD, 16>(p, a, q_begin, q_rows, st);
    case 64: return launch_mtile<ET, DPAD, 32>(p, a, q_begin, q_rows, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename ET>
hipError_t launch_mtile_any(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                            hipStream_t st) {
  switch (p.dpad_t) {
    case 16: return launch_mtile_r<ET, 16>(p, a, q_begin, q_rows, st);
    case 32: return launch_mtile_r<ET, 32>(p, a, q_begin, q_rows, st);
    case 64: return launch_mtile_r<ET, 64>(p, a, q_begin, q_rows, st);
    case 128: return launch_mtile_r<ET, 128>(p, a, q_begin, q_rows, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mt
}  // namespace tod
