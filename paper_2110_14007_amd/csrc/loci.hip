// LOCI (Papadimitriou et al., ICDE 2003; one of Table 1's proximity-based
// detectors, built like LOF on neighbours within range, Section 5.3): the
// multi-granularity deviation factor of every point at a ladder of sampling
// radii r_0 < ... < r_{L-1}, from tod_nwr's CSR of the pairs within r_{L-1}
// (self pairs included, membership exact).
//
//   count  one wave per point p, one pair (p, q) per lane: the pair's exact
//          squared distance (the definition's fp64 sum, as in the range
//          verification), the index of the first sampling radius and of the
//          first counting radius (alpha r_l) that hold it.  The sampling
//          index is kept (one byte per pair) for the next pass; lane-private
//          cumulative counts over the radii are summed over the wave into
//          n(p, r_l) and n(p, alpha r_l).
//   sums   one wave per point p: S1[l] and S2[l], the sums of n(q, alpha r_l)
//          and of its square over the pairs (p, q) whose sampling index is
//          at most l, in 64-bit integers (exact: n <= 2^20 keeps S2 below
//          2^63), lane-private and then summed over the wave.  Lane l then
//          takes radius l: n_hat = S1 / n_r, var = S2 / n_r - n_hat^2 (0 if
//          negative), sigma = sqrt(var), MDEF = 1 - n_alpha / n_hat,
//          sigma_MDEF = sigma / n_hat, in that order in fp64 (correctly
//          rounded division and square root); the wave takes the largest
//          MDEF / sigma_MDEF over the radii with n_r >= n_min as the score
//          and flags the point when MDEF > k_sigma * sigma_MDEF at one of them.
#include <math.h>

#include "tod_internal.h"
#include "wave.h"

namespace tod {

namespace {

constexpr int kW = 4;  // waves per workgroup, one point per wave at a time
constexpr int kU = 16;  // pairs per lane in flight

template <int NLM>
__global__ void __launch_bounds__(kW * 64) loci_count_kernel(LociArgs a) {
#pragma clang fp contract(off)
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nl = a.nl;
  for (int64_t p = (int64_t)blockIdx.x * kW + wave; p < a.n; p += (int64_t)gridDim.x * kW) {
    const float* xp = a.x + p * a.d;
    const int64_t e1 = a.row_ptr[p + 1];
    int cr[NLM], ca[NLM];  // pairs within r_l / alpha r_l seen by this lane
#pragma unroll
    for (int l = 0; l < NLM; ++l) cr[l] = ca[l] = 0;
    // kU pairs per lane per trip: their ids, then their rows' loads, are in
    // flight together (one pair at a time leaves the wave waiting on each
    // dependent gather).
    for (int64_t e0 = a.row_ptr[p]; e0 < e1; e0 += 64 * kU) {
      int64_t q[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int64_t e = e0 + 64 * u + lane;
        q[u] = e < e1 ? a.idx[e] : -1;
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        if (q[u] < 0) continue;
        const double d2 = exact_d2(xp, a.x + q[u] * a.d, a.d);
        int br = 0, ba = 0;  // first radius index holding the pair (nl: none)
#pragma unroll
        for (int l = 0; l < NLM; ++l) {
          if (l < nl) {
            br += a.r2[l] < d2 ? 1 : 0;
            ba += a.a2[l] < d2 ? 1 : 0;
          }
        }
        a.bins[e0 + 64 * u + lane] = (uint8_t)br;
#pragma unroll
        for (int l = 0; l < NLM; ++l) {
          cr[l] += l >= br ? 1 : 0;
          ca[l] += l >= ba ? 1 : 0;
        }
      }
    }
    int32_t* nrp = a.nr + p * a.nls;
    int32_t* nap = a.na + p * a.nls;
#pragma unroll
    for (int l = 0; l < NLM; ++l) {
      if (l < nl) {  // uniform
        int tr = cr[l], ta = ca[l];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
          tr += __shfl_xor(tr, off, 64);
          ta += __shfl_xor(ta, off, 64);
        }
        if (lane == 0) {
          nrp[l] = tr;
          nap[l] = ta;
        }
      }
    }
  }
}

template <int NLM>
__global__ void __launch_bounds__(kW * 64) loci_sum_kernel(LociArgs a) {
#pragma clang fp contract(off)
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nl = a.nl, nls = a.nls;
  for (int64_t p = (int64_t)blockIdx.x * kW + wave; p < a.n; p += (int64_t)gridDim.x * kW) {
    uint64_t s1[NLM], s2[NLM];
#pragma unroll
    for (int l = 0; l < NLM; ++l) s1[l] = s2[l] = 0;
    const int64_t e1 = a.row_ptr[p + 1];
    for (int64_t e0 = a.row_ptr[p]; e0 < e1; e0 += 64 * kU) {
      // kU pairs per lane per trip, their loads in flight together.
      int64_t q[kU];
      int b[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int64_t e = e0 + 64 * u + lane;
        const bool live = e < e1;
        q[u] = live ? a.idx[e] : 0;
        b[u] = live ? (int)a.bins[e] : NLM;  // past the row: contributes to no radius
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        // n(q, alpha r_l) for every l: the row of q, 16-byte chunks (the row
        // stride nls is a multiple of 8).
        const int4* nq4 = reinterpret_cast<const int4*>(a.na + q[u] * nls);
#pragma unroll
        for (int c = 0; c < NLM / 4; ++c) {
          if (4 * c < nl) {
            const int4 v = nq4[c];
            const int vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int l = 4 * c + t;
              if (l < nl && l >= b[u]) {
                const uint64_t w = (uint32_t)vv[t];
                s1[l] += w;
                s2[l] += w * w;
              }
            }
          }
        }
      }
    }
    // Wave sums; lane l keeps radius l's.
    uint64_t m1 = 0, m2 = 0;
#pragma unroll
    for (int l = 0; l < NLM; ++l) {
      if (l < nl) {  // uniform
        uint64_t t1 = s1[l], t2 = s2[l];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
          t1 += shfl_xor64(t1, off);
          t2 += shfl_xor64(t2, off);
        }
        if (lane == l) {
          m1 = t1;
          m2 = t2;
        }
      }
    }
    double ratio = -INFINITY;
    bool counted = false, flagged = false;
    if (lane < nl) {
      const int32_t nrv = a.nr[p * nls + lane], nav = a.na[p * nls + lane];
      const double nrd = (double)nrv;
      const double nhat = (double)m1 / nrd;
      double var = (double)m2 / nrd - nhat * nhat;
      if (var < 0.0) var = 0.0;
      const double sigma = sqrt(var);
      const double mdef = 1.0 - (double)nav / nhat;
      const double smdef = sigma / nhat;
      counted = nrv >= a.n_min;
      if (counted) {
        ratio = smdef > 0.0 ? mdef / smdef : 0.0;
        flagged = mdef > a.k_sigma * smdef;
      }
      const int64_t at = p * nl + lane;
      if (a.na_out) a.na_out[at] = nav;
      if (a.nr_out) a.nr_out[at] = nrv;
      if (a.mdef_out) a.mdef_out[at] = mdef;
      if (a.smdef_out) a.smdef_out[at] = smdef;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const double o = __longlong_as_double(
          (long long)shfl_xor64((uint64_t)__double_as_longlong(ratio), off));
      ratio = o > ratio ? o : ratio;
    }
    const bool any = __ballot(counted) != 0;
    const bool flag = __ballot(flagged) != 0;
    if (lane == 0) {
      a.score[p] = any ? ratio : 0.0;
      if (a.flag) a.flag[p] = flag ? 1 : 0;
    }
  }
}

template <int NLM>
hipError_t launch_loci_t(const LociArgs& a, hipStream_t s) {
  int64_t g = (a.n + kW - 1) / kW;
  if (g > 8192) g = 8192;
  hipLaunchKernelGGL(loci_count_kernel<NLM>, dim3((unsigned)g), dim3(kW * 64), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(loci_sum_kernel<NLM>, dim3((unsigned)g), dim3(kW * 64), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_loci(const LociArgs& a, hipStream_t s) {
  if (a.nl < 1 || a.nl > kLociMaxRadii || a.nls < a.nl) return hipErrorInvalidValue;
  switch (a.nls) {
    case 8: return launch_loci_t<8>(a, s);
    case 16: return launch_loci_t<16>(a, s);
    case 32: return launch_loci_t<32>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tod
