// Fused MFMA distance tile + range test for neighbours within range (NWR,
// Section 5.3), the low-precision evaluation of provable quantization
// (Section 5.2 step ii) with cdist fused into the comparison (Section 6.1),
// so the n x n distance matrix never exists.
//
// A workgroup of 4 waves owns 128 queries and walks one reference split in
// stages of 32 NS rows staged in LDS (double-buffered), exactly as the kNN
// tile does; each wave keeps its 32 queries' operand in registers and
// v_mfma_f32_32x32x16_{f16,bf16} leaves lane l with 16 accumulators of query
// l % 32:
//     acc = <xhat_i, xhat_j> - fl(N_j)/2,    key t = -2 acc.
//
// Range test.  Eq. (nwr-check) decides a pair from the low-precision value
// when |D - phi| exceeds the rounding error.  Here the error bound is the
// kNN certificate's (fp32 accumulation bound with the row norms, plus the
// quantisation radii rho), applied per query row with the reference maxima
// Nmax and Pmax, and turned into two accumulator thresholds per row:
//     acc <  aout  =>  s ||x_i - x_j|| > s phi (1 + 4e-9)     out of range for certain
//     acc >  ain   =>  s ||x_i - x_j|| < s phi (1 - 4e-9)     in range for certain
// Everything else (aout <= acc <= ain) is uncertain.  The slack 4e-9 makes
// the certain decisions agree with the exact fp64 test D2 <= phi^2 as well.
//
// Count pass: each (query, split) counts its candidates (acc >= aout).
// Fill pass: each writes its candidates' reference ids, in increasing j, to
// its slot range of the candidate buffer (offsets from the count pass), with
// bit 31 set for the uncertain ones.  A sub-tile costs a max3 reduction and
// one compare per lane unless some lane has a candidate.
#pragma once

#include "mtile.h"
#include "tod_internal.h"

namespace tod {
namespace rt {

using mt::Frag;
using mt::f32x16;

__device__ __forceinline__ float round_down_f32(double x) {
  float f = (float)x;
  if ((double)f > x) f = nextafterf(f, -INFINITY);
  return f;
}

__device__ __forceinline__ float round_up_f32(double x) {
  float f = (float)x;
  if ((double)f < x) f = nextafterf(f, INFINITY);
  return f;
}

// Accumulator thresholds of query row q (file header).  With N_i the row's
// squared norm, E the accumulation bound of any pair of the row and
// r = rho_i + Pmax (both times margin_scale):
//   acc < aout  =>  t > (s phi (1 + 4e-9) + r)^2 + E - N_i  =>  s D > s phi (1 + 4e-9)
//   acc > ain   =>  t < (s phi (1 - 4e-9) - r)^2 - E - N_i  =>  s D < s phi (1 - 4e-9)
// using |t - (N_j - 2<xhat_i, xhat_j>)| <= E and | s D - ||xhat_i - xhat_j|| | <= r.
// Each fp64 threshold is widened by 1e-12 of its terms (fp64 rounding of the
// thresholds and of N_i) and rounded outward to fp32.
__device__ __forceinline__ void range_thresholds(const Args& a, int64_t q, float& aout,
                                                 float& ain) {
  const double nmax = __longlong_as_double((long long)a.ctrl->nmax_bits);
  const double pmax = __longlong_as_double((long long)a.ctrl->pmax_bits);
  const double s = scale_from_maxabs(a.ctrl->maxabs_bits, a.scale_exp);
  const double u = 0x1p-23;  // per-addition allowance (2x the fp32 unit roundoff)
  const double tt = (double)a.d + 2.0;
  const double gam = tt * u / (1.0 - tt * u);
  const double ms = (double)a.margin_scale;
  const double ni = a.n64_q[q];
  const double err = ms * (gam * (ni + 2.0 * nmax) * (1.0 + 1e-6) + u * nmax +
                           (double)a.d * 0x1p-120);
  const double r = ms * (a.rho_q[q] + pmax);
  // A per-row squared radius enters through its fp64 square root; the 4e-9
  // slack below covers that rounding many times over.
  const double ps = s * (a.phi2_row ? sqrt(a.phi2_row[q]) : a.phi);
  const double bo = ps * (1.0 + 4e-9) + r;
  const double tout = bo * bo + err - ni + 1e-12 * (bo * bo + ni + err);
  aout = round_down_f32(-0.5 * tout);
  if (aout < -3.4028234663852886e38f) aout = -3.4028234663852886e38f;  // never -inf
  ain = INFINITY;
  const double bi = ps * (1.0 - 4e-9) - r;
  if (bi > 0.0 && !a.force_fallback) {
    const double tin = bi * bi - err - ni - 1e-12 * (bi * bi + ni + err);
    ain = round_up_f32(-0.5 * tin);
  }
}

template <typename ET, int DPAD, bool FILL>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(DPAD >= 512 ? 1 : 2)))
range_tile_kernel(Args a, int64_t q_begin, int64_t q_rows) {
  using V = typename Frag<ET>::V;
  using LY = mt::Layout<DPAD, false>;
  constexpr int W = 4, NT = 256;
  constexpr int KC = LY::k16;
  constexpr int ROWB = LY::rowb;
  constexpr int NS = LY::ns;
  constexpr int TR = 32 * NS;  // reference rows per stage
  constexpr int STAGE = TR * ROWB;
  constexpr int CPR = LY::cpr;
  constexpr int CHUNKS = TR * CPR;
  constexpr int NL = (CHUNKS + NT - 1) / NT;
  static_assert(TR / 4 <= NT, "one float4 of seeds per thread");
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* stage = smem;
  float* hnb = (float*)(smem + 2 * STAGE);

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, col = lane & 31;
  if (a.ctrl->nonfinite) return;  // uniform over the grid
  const int64_t group = (int64_t)blockIdx.x * W + wave;
  const bool active = group * 32 < q_rows;  // uniform per wave
  const int64_t q0 = q_begin + group * 32;
  const int64_t q = q0 + col;
  const bool qvalid = active && group * 32 + col < q_rows;
  const int split = blockIdx.y;
  const int64_t r_begin = (int64_t)split * a.split_len;
  const int64_t r_end = r_begin + a.split_len < a.nr ? r_begin + a.split_len : a.nr;
  const int64_t r_end32 = (r_end + 31) & ~(int64_t)31;  // rows < r_end32 exist (padded copy)
  const bool selfq = a.exclude_self != 0;

  // Lanes without a query (past the batch) never see a candidate.
  float aout = INFINITY, ain = INFINITY;
  if (qvalid) range_thresholds(a, q, aout, ain);

  V bq[KC];
  {
    const ET* qrow = (const ET*)a.xq_q + (active ? q0 + col : 0) * (int64_t)DPAD;
#pragma unroll
    for (int c = 0; c < KC; ++c) bq[c] = *reinterpret_cast<const V*>(qrow + 16 * c + 8 * h);
  }

  // Count pass: this lane's candidates.  Fill pass: candidates of the lane
  // pair written so far (the same in both lanes).
  int run = 0;
  uint32_t* dst = nullptr;
  float* fdst = nullptr;  // the candidates' accumulators (for the per-pair test)
  int64_t room = 0;
  if constexpr (FILL) {
    if (qvalid) {
      const int64_t o = a.coff[q * a.splits + split];
      dst = a.cand + (o - a.cbase);
      fdst = a.cand_d + (o - a.cbase);
      room = a.coff[q * a.splits + split + 1] - o;
    }
  }

  // Staging: every thread moves up to NL 16-byte chunks of a stage (rows past
  // the split's padded end are clamped to its last row: loaded, never read).
  // The staging registers start zeroed: left undefined, the compiler keeps
  // them as a stack object in scratch memory.
  const unsigned char* xr_bytes = (const unsigned char*)a.xq_r;
  uint4 st[NL];
#pragma unroll
  for (int i = 0; i < NL; ++i) st[i] = make_uint4(0, 0, 0, 0);
  float4 sth = make_float4(0.f, 0.f, 0.f, 0.f);
#define TOD_RT_FETCH(T0)                                                                     \
  _Pragma("unroll") for (int i = 0; i < NL; ++i) {                                          \
    const int c = tid + i * NT;                                                             \
    if (CHUNKS % NT == 0 || c < CHUNKS) {                                                   \
      const int row = c / CPR, cc = c % CPR;                                                \
      const int64_t gr = (T0) + row < r_end32 ? (T0) + row : r_end32 - 1;                   \
      st[i] = *reinterpret_cast<const uint4*>(xr_bytes + gr * (int64_t)(DPAD * 2) + cc * 16); \
    }                                                                                       \
  }                                                                                         \
  if (tid < TR / 4) {                                                                       \
    const int64_t gr = (T0) + 4 * tid < r_end32 ? (T0) + 4 * tid : r_end32 - 4;             \
    sth = *reinterpret_cast<const float4*>(a.hn_r + gr);                                    \
  }
#define TOD_RT_PUT(B)                                                                        \
  _Pragma("unroll") for (int i = 0; i < NL; ++i) {                                          \
    const int c = tid + i * NT;                                                             \
    if (CHUNKS % NT == 0 || c < CHUNKS)                                                     \
      *reinterpret_cast<uint4*>(stage + (B) * STAGE + (c / CPR) * ROWB + (c % CPR) * 16) =    \
          st[i];                                                                            \
  }                                                                                         \
  if (tid < TR / 4) *reinterpret_cast<float4*>(hnb + (B) * TR + 4 * tid) = sth;

  auto body = [&](int64_t t0, int b) __attribute__((always_inline)) {
    if (!active) return;
    const unsigned char* buf = stage + b * STAGE;
    const float* hn = hnb + b * TR;
    const int live = r_end - t0 < TR ? (int)((r_end - t0 + 31) >> 5) : NS;
#pragma unroll 1
    for (int s = 0; s < live; ++s) {
      const int64_t ts = t0 + 32 * s;
      V af[KC];
#pragma unroll
      for (int c = 0; c < KC; ++c)
        af[c] = *reinterpret_cast<const V*>(buf + (32 * s + col) * ROWB + 32 * c + 16 * h);
      f32x16 acc;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float4 t = *reinterpret_cast<const float4*>(hn + 32 * s + 8 * g + 4 * h);
        acc[4 * g + 0] = t.x;
        acc[4 * g + 1] = t.y;
        acc[4 * g + 2] = t.z;
        acc[4 * g + 3] = t.w;
      }
#pragma unroll
      for (int c = 0; c < KC; ++c) acc = mt::mfma<ET>(af[c], bq[c], acc);
      // Rows past the split and the query's own row (self exclusion) are never candidates.
      const bool diag = selfq && ts == q0;
      if (diag || ts + 32 > r_end) {
        const int lim = ts + 32 > r_end ? (int)(r_end - ts) : 32;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = mt::out_row(r, h);
          if (row >= lim || (diag && row == col)) acc[r] = -INFINITY;
        }
      }
      const float m0 = mt::max3f(acc[0], acc[1], acc[2]), m1 = mt::max3f(acc[3], acc[4], acc[5]);
      const float m2 = mt::max3f(acc[6], acc[7], acc[8]), m3 = mt::max3f(acc[9], acc[10], acc[11]);
      const float m4 = mt::max3f(acc[12], acc[13], acc[14]);
      const float m = mt::max3f(mt::max3f(m0, m1, m2), mt::max3f(m3, m4, acc[15]), m0);
      if (!__ballot(m >= aout)) continue;
      uint32_t cm = 0, um = 0;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        cm |= (acc[r] >= aout ? 1u : 0u) << r;
        um |= (acc[r] <= ain ? 1u : 0u) << r;
      }
      um &= cm;
      if constexpr (!FILL) {
        run += __builtin_popcount(cm);
      } else {
        // The pair's candidates of this sub-tile in row order: accumulator r
        // of lane half hh holds row 8 (r / 4) + 4 hh + r % 4.
        const uint32_t pm = mt::xchg32(cm, h);
        const uint32_t m_lo = h ? pm : cm, m_hi = h ? cm : pm;
        uint32_t rows = 0;
#pragma unroll
        for (int g = 0; g < 4; ++g)
          rows |= (((m_lo >> (4 * g)) & 15u) << (8 * g)) | (((m_hi >> (4 * g)) & 15u) << (8 * g + 4));
        // One trip per candidate of this lane (usually one or two).
        auto accv = [&](int r) {
          float v = acc[0];
#pragma unroll
          for (int e = 1; e < 16; ++e) v = r == e ? acc[e] : v;
          return v;
        };
        for (uint32_t m = cm; m; m &= m - 1u) {
          const int r = __builtin_ctz(m);
          const int row = mt::out_row(r, h);
          const int pos = run + __builtin_popcount(rows & ((1u << row) - 1u));
          if (pos < room) {
            dst[pos] = (uint32_t)(ts + row) | (((um >> r) & 1u) << 31);
            fdst[pos] = accv(r);
          } else
            atomicOr(&a.ctrl->internal, 1u);  // the passes disagree: report, never overrun
        }
        run += __builtin_popcount(rows);
      }
    }
  };

  const int nst = (int)((r_end - r_begin + TR - 1) / TR);
  auto t_of = [&](int i) -> int64_t { return r_begin + (int64_t)(i < nst ? i : 0) * TR; };
  TOD_RT_FETCH(t_of(0))
  TOD_RT_PUT(0)
  __syncthreads();
  for (int it = 0; it < nst; ++it) {
    TOD_RT_FETCH(t_of(it + 1))  // the stage after the last is a reload of the first, never read
    body(t_of(it), it & 1);
    TOD_RT_PUT((it + 1) & 1)
    __syncthreads();
  }
#undef TOD_RT_FETCH
#undef TOD_RT_PUT
  if constexpr (!FILL) {
    const int tot = run + (int)mt::xchg32((uint32_t)run, h);
    if (qvalid && h == 0) a.ccount[q * a.splits + split] = tot;
  } else {
    if (qvalid && h == 0 && run != room) atomicOr(&a.ctrl->internal, 1u);
  }
}

template <typename ET, int DPAD>
hipError_t launch_range(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows, bool fill,
                        hipStream_t st) {
  using LY = mt::Layout<DPAD, false>;
  const size_t lds = (size_t)2 * 32 * LY::ns * LY::rowb + (size_t)2 * 32 * LY::ns * sizeof(float);
  const auto kern = fill ? range_tile_kernel<ET, DPAD, true> : range_tile_kernel<ET, DPAD, false>;
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const int64_t groups = (q_rows + 31) / 32;
  const dim3 grid((unsigned)((groups + 3) / 4), (unsigned)p.splits);
  hipLaunchKernelGGL(kern, grid, dim3(256), lds, st, a, q_begin, q_rows);
  return hipGetLastError();
}

template <typename ET>
hipError_t launch_range_any(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                            bool fill, hipStream_t st) {
  switch (p.dpad) {
    case 16: return launch_range<ET, 16>(p, a, q_begin, q_rows, fill, st);
    case 32: return launch_range<ET, 32>(p, a, q_begin, q_rows, fill, st);
    case 64: return launch_range<ET, 64>(p, a, q_begin, q_rows, fill, st);
    case 128: return launch_range<ET, 128>(p, a, q_begin, q_rows, fill, st);
    case 256: return launch_range<ET, 256>(p, a, q_begin, q_rows, fill, st);
    case 512: return launch_range<ET, 512>(p, a, q_begin, q_rows, fill, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace rt
}  // namespace tod
