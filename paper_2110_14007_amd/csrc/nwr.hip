// Neighbours within range (Section 5.3): exact verification of the filter's
// uncertain pairs (Section 5.2 step iii: exact recomputation only for the
// pairs the low-precision check cannot decide) and assembly of the CSR output.
//
// After the fill pass (rtile.h) the candidate buffer holds, for each query
// row of the batch, its candidates in increasing reference index; bit 31
// marks the ones the filter could not rule in.
//   verify  one wave per row.  An uncertain candidate first gets the
//           tile's test again with its own reference norm and radius in
//           place of the maxima (pair_test); the ones still undecided (and
//           every kept candidate when distances are requested) are gathered
//           in an LDS list and then get, 64 at a time, the exact squared
//           distance, computed as in the definition: fp64, columns in order,
//           ((double)x - (double)y)^2 added one at a time with no fused
//           multiply-add, so the in-range decision D2 <= phi^2 is the same
//           bit for bit as a plain fp64 evaluation (against phi^2, or the
//           row's own squared radius when one is given per row).  Kept
//           candidates get their distance (or 0), dropped ones -1; the row's
//           count is stored.
//   scan    row offsets = exclusive prefix sums of the counts (continuing
//           from the previous batch's last offset).
//   emit    one wave per row: kept candidates are compacted in order (ballot
//           ranks) into idx_out / dist_out at the row's offset, within the
//           caller's capacity.
#include <math.h>

#include "tod_internal.h"

namespace tod {

namespace {

constexpr int kScanT = 256;
constexpr int kScanPer = 16;
constexpr int kScanChunk = kScanT * kScanPer;

// Range test of one pair with the pair's own reference norm and radius
// (the tile's per-row thresholds use the reference maxima): +1 in range for
// certain, -1 out of range for certain, 0 undecided.  acc is the pair's fp32
// accumulator from the fill pass, t = -2 acc its key; the bounds are the
// tile's (rtile.h) with N_j <= -2 hn_r[j] (1 + 2^-22) and rho_j in place of
// Nmax and Pmax.
__device__ __forceinline__ int pair_test(const Args& a, double s, double gam, double ni,
                                         double rho_i, double phi, uint32_t j, float acc) {
  const double ms = (double)a.margin_scale;
  const double u = 0x1p-23;
  const double nj = -2.0 * (double)a.hn_r[j] * (1.0 + 0x1p-22);
  const double e = ms * (gam * (ni + 2.0 * nj) * (1.0 + 1e-6) + u * nj + (double)a.d * 0x1p-120);
  const double r = ms * (rho_i + a.rho_r[j]);
  const double t = -2.0 * (double)acc;
  const double slack = 1e-12 * (ni + fabs(t) + e);
  const double ps = s * phi;
  const double hi = ni + t + e + slack;
  if (hi >= 0.0 && sqrt(hi) + r < ps * (1.0 - 4e-9)) return 1;
  const double lo = ni + t - e - slack;
  if (lo > 0.0 && sqrt(lo) - r > ps * (1.0 + 4e-9)) return -1;
  return 0;
}

// Candidates of one row that need their exact distance, gathered per wave
// so that a row's pairs share one 64-lane pass of the exact sums (a pass
// costs one sequential chain of d fp64 additions whatever the number of
// active lanes).
constexpr int kExactList = 256;

// LDS writes of this wave are visible to its other lanes.
__device__ __forceinline__ void wave_lds_fence() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_wave_barrier();
}

__global__ void __launch_bounds__(256)
range_verify_kernel(Args a, int64_t b0, int64_t rows, int32_t want_dist) {
  __shared__ uint32_t xlist[4][kExactList];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = b0 + (int64_t)blockIdx.x * 4 + wave;
  if (row >= b0 + rows) return;  // uniform per wave
  const int64_t beg = a.coff[row * a.splits] - a.cbase;
  const int64_t end = a.coff[(row + 1) * a.splits] - a.cbase;
  const float* qrow = a.xq + row * (int64_t)a.d;
  // The row's radius: one for all rows, or the row's own squared radius (its
  // root only feeds the filter's margins, never the exact test).
  const double phi2 = a.phi2_row ? a.phi2_row[row] : a.phi * a.phi;
  const double phi = a.phi2_row ? sqrt(phi2) : a.phi;
  const double s = scale_from_maxabs(a.ctrl->maxabs_bits, a.scale_exp);
  const double tt = (double)a.d + 2.0;
  const double gam = tt * 0x1p-23 / (1.0 - tt * 0x1p-23);
  const double ni = a.n64_q[row], rho_i = a.rho_q[row];
  const uint64_t lt = (1ull << lane) - 1;  // lanes below this one
  int kept = 0, unc = 0, nx = 0;
  // Exact pass over the gathered list: entry = (p - beg) << 1 | uncertain.
  auto exact_pass = [&]() {
    wave_lds_fence();  // the list's entries are visible to every lane
    for (int i0 = 0; i0 < nx; i0 += 64) {
      const bool live = i0 + lane < nx;
      const uint32_t e = live ? xlist[wave][i0 + lane] : 0u;
      const int64_t p = beg + (e >> 1);
      const bool u = (e & 1u) != 0;
      double d2 = 0.0;
      if (live) d2 = exact_d2(qrow, a.xr + (int64_t)(a.cand[p] & 0x7fffffffu) * a.d, a.d);
      const bool keep = live && (!u || d2 <= phi2);
      if (live) a.cand_d[p] = keep ? (float)sqrt(d2) : -1.0f;
      kept += __popcll(__ballot(keep));
    }
    nx = 0;
    wave_lds_fence();  // the list is refilled after every lane has read it
  };
  for (int64_t p0 = beg; p0 < end; p0 += 64) {
    const int64_t p = p0 + lane;
    const bool live = p < end;
    const uint32_t c = live ? a.cand[p] : 0u;
    const uint32_t j = c & 0x7fffffffu;
    // Uncertain for the tile: first the per-pair test (not under
    // force_fallback, which recomputes every candidate).
    int pt = 0;
    if (live && (c >> 31) && !a.force_fallback)
      pt = pair_test(a, s, gam, ni, rho_i, phi, j, a.cand_d[p]);
    const bool u = live && (c >> 31) && pt == 0;
    const bool need = live && (u || (want_dist && pt >= 0));
    // Decided without the exact distance: in range for certain (distance
    // not asked for) or out of range.
    const bool keep_now = live && !need && pt >= 0;
    if (live && !need) a.cand_d[p] = keep_now ? 0.0f : -1.0f;
    kept += __popcll(__ballot(keep_now));
    unc += __popcll(__ballot(u));
    const uint64_t nb = __ballot(need);
    if (nx + __popcll(nb) > kExactList) exact_pass();
    if (need) xlist[wave][nx + __popcll(nb & lt)] = (uint32_t)((p - beg) << 1) | (u ? 1u : 0u);
    nx += __popcll(nb);
  }
  if (nx) exact_pass();
  if (lane == 0) {
    a.incnt[row] = kept;
    if (unc)
      atomicAdd((unsigned long long*)&a.ctrl->uncertain[(blockIdx.x % kUncParts) * kUncStride],
                (unsigned long long)unc);
  }
}

__global__ void __launch_bounds__(256)
range_emit_kernel(Args a, int64_t b0, int64_t rows) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = b0 + (int64_t)blockIdx.x * 4 + wave;
  if (row >= b0 + rows) return;  // uniform per wave
  const int64_t beg = a.coff[row * a.splits] - a.cbase;
  const int64_t end = a.coff[(row + 1) * a.splits] - a.cbase;
  int64_t out = a.row_ptr[row];
  const uint64_t below = (1ull << lane) - 1ull;
  for (int64_t p0 = beg; p0 < end; p0 += 64) {
    const int64_t p = p0 + lane;
    const bool live = p < end;
    const float dd = live ? a.cand_d[p] : -1.0f;
    const bool keep = dd >= 0.0f;
    const uint64_t m = __ballot(keep);
    const int64_t pos = out + __popcll(m & below);
    if (keep && pos < a.out_cap) {
      a.idx_out[pos] = (int64_t)(a.cand[p] & 0x7fffffffu);
      if (a.dist_out) a.dist_out[pos] = dd;
    }
    out += __popcll(m);
  }
}

// Block sums of kScanChunk-element chunks.
__global__ void __launch_bounds__(kScanT)
scan_sum_kernel(const int32_t* __restrict__ in, int64_t n, int64_t* __restrict__ part) {
  __shared__ int64_t red[kScanT / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanChunk;
  int64_t s = 0;
  for (int i = threadIdx.x; i < kScanChunk; i += kScanT) {
    const int64_t k = base + i;
    if (k < n) s += in[k];
  }
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t t = 0;
    for (int w = 0; w < kScanT / 64; ++w) t += red[w];
    part[blockIdx.x] = t;
  }
}

// Exclusive scan of the np block sums in place (one workgroup), plus *base.
__global__ void __launch_bounds__(kScanT)
scan_top_kernel(int64_t* __restrict__ part, int64_t np, const int64_t* __restrict__ base) {
  __shared__ int64_t sh[kScanT];
  int64_t carry = base ? *base : 0;
  for (int64_t c0 = 0; c0 < np; c0 += kScanT) {
    const int64_t k = c0 + threadIdx.x;
    const int64_t v = k < np ? part[k] : 0;
    sh[threadIdx.x] = v;
    __syncthreads();
    for (int o = 1; o < kScanT; o <<= 1) {
      const int64_t t = threadIdx.x >= o ? sh[threadIdx.x - o] : 0;
      __syncthreads();
      sh[threadIdx.x] += t;
      __syncthreads();
    }
    if (k < np) part[k] = carry + sh[threadIdx.x] - v;
    carry += sh[kScanT - 1];
    __syncthreads();
  }
}

// out[i] = part[block] + prefix of the block's chunk up to i; out[n] = total.
__global__ void __launch_bounds__(kScanT)
scan_final_kernel(const int32_t* __restrict__ in, int64_t n, const int64_t* __restrict__ part,
                  int64_t* __restrict__ out) {
  __shared__ int64_t sh[kScanT];
  const int64_t base = (int64_t)blockIdx.x * kScanChunk + (int64_t)threadIdx.x * kScanPer;
  int32_t v[kScanPer];
  int64_t s = 0;
#pragma unroll
  for (int i = 0; i < kScanPer; ++i) {
    v[i] = base + i < n ? in[base + i] : 0;
    s += v[i];
  }
  sh[threadIdx.x] = s;
  __syncthreads();
  for (int o = 1; o < kScanT; o <<= 1) {
    const int64_t t = threadIdx.x >= o ? sh[threadIdx.x - o] : 0;
    __syncthreads();
    sh[threadIdx.x] += t;
    __syncthreads();
  }
  int64_t acc = part[blockIdx.x] + sh[threadIdx.x] - s;
#pragma unroll
  for (int i = 0; i < kScanPer; ++i) {
    if (base + i < n) out[base + i] = acc;
    acc += v[i];
    if (base + i == n - 1) out[n] = acc;
  }
}

__global__ void group_offsets_kernel(const int64_t* __restrict__ coff, int64_t nq, int32_t splits,
                                     int64_t groups, int64_t* __restrict__ goff) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g > groups) return;
  const int64_t row = 32 * g < nq ? 32 * g : nq;
  goff[g] = coff[row * splits];
}

unsigned blocks_for_rows(int64_t rows) { return (unsigned)((rows + 3) / 4); }

}  // namespace

int64_t scan_parts(int64_t n) { return (n + kScanChunk - 1) / kScanChunk; }

hipError_t launch_scan(const int32_t* in, int64_t n, int64_t* out, const int64_t* base,
                       int64_t* part, hipStream_t s) {
  const int64_t np = scan_parts(n);
  hipLaunchKernelGGL(scan_sum_kernel, dim3((unsigned)np), dim3(kScanT), 0, s, in, n, part);
  hipLaunchKernelGGL(scan_top_kernel, dim3(1), dim3(kScanT), 0, s, part, np, base);
  hipLaunchKernelGGL(scan_final_kernel, dim3((unsigned)np), dim3(kScanT), 0, s, in, n,
                     (const int64_t*)part, out);
  return hipGetLastError();
}

hipError_t launch_group_offsets(const Args& a, int64_t groups, int64_t* goff, hipStream_t s) {
  hipLaunchKernelGGL(group_offsets_kernel, dim3((unsigned)((groups + 1 + 255) / 256)), dim3(256),
                     0, s, (const int64_t*)a.coff, a.nq, a.splits, groups, goff);
  return hipGetLastError();
}

hipError_t launch_range_verify(const Args& a, int64_t b0, int64_t rows, int32_t want_dist,
                               hipStream_t s) {
  hipLaunchKernelGGL(range_verify_kernel, dim3(blocks_for_rows(rows)), dim3(256), 0, s, a, b0,
                     rows, want_dist);
  return hipGetLastError();
}

hipError_t launch_range_emit(const Args& a, int64_t b0, int64_t rows, hipStream_t s) {
  hipLaunchKernelGGL(range_emit_kernel, dim3(blocks_for_rows(rows)), dim3(256), 0, s, a, b0,
                     rows);
  return hipGetLastError();
}

}  // namespace tod
