// Grouped scan order for X against X.
//
// The rows are partitioned by their nearest of kOrdC seed rows (the rows at
// positions floor(c n / kOrdC), squared distance in fp32, ties to the lower
// seed) and laid out group by group, each group in input order (a stable
// counting sort).  The quantised copy, its norms and radii are written in
// that order; a tile workgroup starts its scan at the first row of the group
// holding its first query, so near references come first and the filter's
// thresholds tighten early.  The exact kNN set of every row does not depend on
// the order: the recheck maps positions back to input rows before it ranks and
// writes anything.
#include "tod_internal.h"

namespace tod {

namespace {

constexpr int kAssignThreads = 256;

// lab[row] = nearest seed (one thread per row; the seeds sit in LDS).
__global__ void __launch_bounds__(kAssignThreads)
assign_kernel(const float* __restrict__ x, int64_t n, int d, int32_t* __restrict__ lab) {
  extern __shared__ float seeds[];  // [kOrdC][d]
  for (int i = threadIdx.x; i < kOrdC * d; i += blockDim.x) {
    const int c = i / d, t = i - c * d;
    const int64_t srow = (int64_t)c * n / kOrdC;
    seeds[i] = x[srow * d + t];
  }
  __syncthreads();
  const int64_t row = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= n) return;
  float acc[kOrdC];
#pragma unroll
  for (int c = 0; c < kOrdC; ++c) acc[c] = 0.0f;
  const float* in = x + row * d;
  for (int t = 0; t < d; ++t) {
    const float v = in[t];
#pragma unroll
    for (int c = 0; c < kOrdC; ++c) {
      const float df = v - seeds[c * d + t];
      acc[c] = fmaf(df, df, acc[c]);
    }
  }
  int best = 0;
#pragma unroll
  for (int c = 1; c < kOrdC; ++c) best = acc[c] < acc[best] ? c : best;
  lab[row] = best;
}

// Rows per group in each block of kOrdRows rows.
__global__ void __launch_bounds__(256)
count_kernel(const int32_t* __restrict__ lab, int64_t n, int32_t* __restrict__ bcnt) {
  __shared__ int32_t cnt[kOrdC];
  if (threadIdx.x < kOrdC) cnt[threadIdx.x] = 0;
  __syncthreads();
  const int64_t r0 = (int64_t)blockIdx.x * kOrdRows;
  const int64_t r1 = r0 + kOrdRows < n ? r0 + kOrdRows : n;
  for (int64_t r = r0 + threadIdx.x; r < r1; r += blockDim.x) atomicAdd(&cnt[lab[r]], 1);
  __syncthreads();
  if (threadIdx.x < kOrdC) bcnt[(int64_t)blockIdx.x * kOrdC + threadIdx.x] = cnt[threadIdx.x];
}

// Group starts and each block's first position in its group: one wave per
// group sums the group's counts over the blocks, then (every total known)
// forms the blocks' exclusive prefix sums 64 blocks at a time.
__global__ void __launch_bounds__(kOrdC * 64)
scan_kernel(const int32_t* __restrict__ bcnt, int nb, int32_t* __restrict__ boff,
            int32_t* __restrict__ cstart) {
  __shared__ int32_t tot[kOrdC];
  const int c = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int32_t t = 0;
  for (int b = lane; b < nb; b += 64) t += bcnt[(int64_t)b * kOrdC + c];
  for (int off = 32; off > 0; off >>= 1) t += __shfl_xor(t, off, 64);
  if (lane == 0) tot[c] = t;
  __syncthreads();
  int32_t start = 0;
  for (int i = 0; i < c; ++i) start += tot[i];
  if (lane == 0) {
    cstart[c] = start;
    if (c == kOrdC - 1) cstart[kOrdC] = start + tot[c];
  }
  int32_t at = start;
  for (int b0 = 0; b0 < nb; b0 += 64) {
    const int b = b0 + lane;
    const int32_t v = b < nb ? bcnt[(int64_t)b * kOrdC + c] : 0;
    int32_t incl = v;  // inclusive prefix sum over the wave
    for (int off = 1; off < 64; off <<= 1) {
      const int32_t o = __shfl_up(incl, off, 64);
      if (lane >= off) incl += o;
    }
    if (b < nb) boff[(int64_t)b * kOrdC + c] = at + incl - v;
    at += __shfl(incl, 63, 64);
  }
}

// perm[position] = row, stable within each group: one wave per block walks
// its rows 64 at a time and ranks each group's members by ballot.
__global__ void __launch_bounds__(64)
scatter_kernel(const int32_t* __restrict__ lab, int64_t n, const int32_t* __restrict__ boff,
               int32_t* __restrict__ perm) {
  const int lane = threadIdx.x;
  int32_t base[kOrdC];
#pragma unroll
  for (int c = 0; c < kOrdC; ++c) base[c] = boff[(int64_t)blockIdx.x * kOrdC + c];
  const int64_t r0 = (int64_t)blockIdx.x * kOrdRows;
  const int64_t r1 = r0 + kOrdRows < n ? r0 + kOrdRows : n;
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  for (int64_t r = r0; r < r1; r += 64) {
    const int64_t row = r + lane;
    const int l = row < r1 ? lab[row] : -1;
#pragma unroll
    for (int c = 0; c < kOrdC; ++c) {
      const uint64_t m = __ballot(l == c);
      if (l == c) perm[base[c] + __popcll(m & below)] = (int32_t)row;
      base[c] += __popcll(m);
    }
  }
}

}  // namespace

int32_t order_blocks(int64_t nr) { return (int32_t)((nr + kOrdRows - 1) / kOrdRows); }

hipError_t launch_order(const Plan& p, const Args& a, hipStream_t st) {
  const int64_t n = p.nr;
  const int nb = order_blocks(n);
  const size_t lds = sizeof(float) * kOrdC * (size_t)p.d;
  hipLaunchKernelGGL(assign_kernel, dim3((unsigned)((n + kAssignThreads - 1) / kAssignThreads)),
                     dim3(kAssignThreads), lds, st, a.xr, n, (int)p.d, a.lab);
  hipLaunchKernelGGL(count_kernel, dim3((unsigned)nb), dim3(256), 0, st, a.lab, n, a.bcnt);
  hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(kOrdC * 64), 0, st, a.bcnt, nb, a.boff, a.cstart);
  hipLaunchKernelGGL(scatter_kernel, dim3((unsigned)nb), dim3(64), 0, st, a.lab, n, a.boff,
                     a.perm);
  return hipGetLastError();
}

}  // namespace tod
