// Grouped scan order for X against X.
//
// The rows are partitioned by their nearest of G seed rows (the rows at
// positions floor(c n / G), squared distance in fp32, ties to the lower
// seed; G from order_groups) and laid out group by group, each group in input
// order (a stable counting sort).  The quantised copy, its norms and radii
// are written in that order; a tile workgroup starts its scan at the first
// row of the group holding its first query, so near references come first
// and the filter's thresholds tighten early.  The exact kNN set of every row
// does not depend on the order: the recheck maps positions back to input rows
// before it ranks and writes anything.
#include "tod_internal.h"

namespace tod {

namespace {

constexpr int kAssignThreads = 256;
constexpr int kSmallD = 16;       // rows this short keep the row in registers
constexpr int kWideGroups = 16;   // seed groups for longer rows

// The G seed rows of short rows, zero-padded to DT columns, gathered once.
__global__ void __launch_bounds__(256)
seeds_kernel(const float* __restrict__ x, int64_t n, int d, int G, int DT,
             float* __restrict__ seeds) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= G * DT) return;
  const int c = i / DT, t = i - c * DT;
  const int64_t srow = (int64_t)c * n / G;
  seeds[i] = t < d ? x[srow * d + t] : 0.0f;
}

// Rows of at most kSmallD elements: lab[row] = nearest of G seeds (the row in
// registers, zero-padded to DT = d rounded up to 4 columns; every lane reads
// the same seed, so the seeds come through the scalar cache as wave-uniform
// loads).
template <int DT>
__global__ void __launch_bounds__(kAssignThreads)
assign_small_kernel(const float* __restrict__ x, int64_t n, int d, int G,
                    const float4* __restrict__ gseeds, int32_t* __restrict__ lab) {
  const int64_t row = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= n) return;
  float v[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) v[t] = t < d ? x[row * d + t] : 0.0f;
  float best_d = INFINITY;
  int best = 0;
  // (Unrolled so that the scalar loads of several seeds are in flight at once.)
#pragma unroll 8
  for (int c = 0; c < G; ++c) {
    float acc = 0.0f;
#pragma unroll
    for (int q = 0; q < DT / 4; ++q) {
      const float4 s4 = gseeds[c * (DT / 4) + q];
      const float sv[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float df = v[4 * q + t] - sv[t];
        acc = fmaf(df, df, acc);
      }
    }
    if (acc < best_d) {
      best_d = acc;
      best = c;
    }
  }
  lab[row] = best;
}

// Longer rows, kWideGroups seeds: lab[row] = nearest seed (one thread per
// row; the seeds sit in LDS).
__global__ void __launch_bounds__(kAssignThreads)
assign_kernel(const float* __restrict__ x, int64_t n, int d, int32_t* __restrict__ lab) {
  extern __shared__ float seeds[];  // [kWideGroups][d]
  for (int i = threadIdx.x; i < kWideGroups * d; i += blockDim.x) {
    const int c = i / d, t = i - c * d;
    const int64_t srow = (int64_t)c * n / kWideGroups;
    seeds[i] = x[srow * d + t];
  }
  __syncthreads();
  const int64_t row = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= n) return;
  float acc[kWideGroups];
#pragma unroll
  for (int c = 0; c < kWideGroups; ++c) acc[c] = 0.0f;
  const float* in = x + row * d;
  for (int t = 0; t < d; ++t) {
    const float v = in[t];
#pragma unroll
    for (int c = 0; c < kWideGroups; ++c) {
      const float df = v - seeds[c * d + t];
      acc[c] = fmaf(df, df, acc[c]);
    }
  }
  int best = 0;
#pragma unroll
  for (int c = 1; c < kWideGroups; ++c) best = acc[c] < acc[best] ? c : best;
  lab[row] = best;
}

// Rows per group in each block of kOrdRows rows.
__global__ void __launch_bounds__(256)
count_kernel(const int32_t* __restrict__ lab, int64_t n, int G, int32_t* __restrict__ bcnt) {
  __shared__ int32_t cnt[kOrdMaxC];
  for (int c = threadIdx.x; c < G; c += blockDim.x) cnt[c] = 0;
  __syncthreads();
  const int64_t r0 = (int64_t)blockIdx.x * kOrdRows;
  const int64_t r1 = r0 + kOrdRows < n ? r0 + kOrdRows : n;
  for (int64_t r = r0 + threadIdx.x; r < r1; r += blockDim.x) atomicAdd(&cnt[lab[r]], 1);
  __syncthreads();
  for (int c = threadIdx.x; c < G; c += blockDim.x) bcnt[(int64_t)blockIdx.x * G + c] = cnt[c];
}

// Inclusive prefix sum over the wave.
__device__ __forceinline__ int32_t wave_incl_sum(int32_t v, int lane) {
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t o = __shfl_up(v, off, 64);
    if (lane >= off) v += o;
  }
  return v;
}

// Each block's first position within its group: one wave per group walks
// the blocks' counts 64 at a time (exclusive prefix sums), and leaves the
// group's total in cstart[c + 1].
__global__ void __launch_bounds__(256)
block_offsets_kernel(const int32_t* __restrict__ bcnt, int nb, int G,
                     int32_t* __restrict__ boff, int32_t* __restrict__ cstart) {
  const int lane = threadIdx.x & 63;
  const int c = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (c >= G) return;  // uniform per wave
  int32_t at = 0;
  for (int b0 = 0; b0 < nb; b0 += 64) {
    const int b = b0 + lane;
    const int32_t v = b < nb ? bcnt[(int64_t)b * G + c] : 0;
    const int32_t incl = wave_incl_sum(v, lane);
    if (b < nb) boff[(int64_t)b * G + c] = at + incl - v;
    at += __shfl(incl, 63, 64);
  }
  if (lane == 0) cstart[c + 1] = at;
}

// Group starts: cstart[0..G] becomes the exclusive prefix sums of the group
// totals (one workgroup, 64 groups per step).
__global__ void __launch_bounds__(64)
group_starts_kernel(int G, int32_t* __restrict__ cstart) {
  const int lane = threadIdx.x;
  int32_t at = 0;
  for (int c0 = 0; c0 < G; c0 += 64) {
    const int c = c0 + lane;
    const int32_t v = c < G ? cstart[c + 1] : 0;
    const int32_t incl = wave_incl_sum(v, lane);
    if (c < G) cstart[c + 1] = at + incl;
    at += __shfl(incl, 63, 64);
  }
  if (lane == 0) cstart[0] = 0;
}

// perm[position] = row, stable within each group: one wave per block walks
// its rows 64 at a time; each lane counts the lanes of the same group below
// it (its rank) and in all (the group's count in these 64 rows), writes its
// row at the group's next position plus its rank, and the group's first lane
// advances the group's next position.  (A group's next position starts at
// the group's start plus the block's offset within the group.)
__global__ void __launch_bounds__(64)
scatter_kernel(const int32_t* __restrict__ lab, int64_t n, int G,
               const int32_t* __restrict__ boff, const int32_t* __restrict__ cstart,
               int32_t* __restrict__ perm) {
  __shared__ int32_t next[kOrdMaxC];
  const int lane = threadIdx.x;
  for (int c = lane; c < G; c += 64) next[c] = cstart[c] + boff[(int64_t)blockIdx.x * G + c];
  __syncthreads();
  const int64_t r0 = (int64_t)blockIdx.x * kOrdRows;
  const int64_t r1 = r0 + kOrdRows < n ? r0 + kOrdRows : n;
  for (int64_t r = r0; r < r1; r += 64) {
    const int64_t row = r + lane;
    const int l = row < r1 ? lab[row] : -1;
    int rank = 0, cnt = 0;
    for (int j = 0; j < 64; ++j) {
      const bool eq = __shfl(l, j, 64) == l;
      cnt += eq ? 1 : 0;
      rank += (eq && j < lane) ? 1 : 0;
    }
    if (l >= 0) perm[next[l] + rank] = (int32_t)row;
    __syncthreads();  // every lane has read next[] before it moves
    if (l >= 0 && rank == 0) next[l] += cnt;
    __syncthreads();
  }
}

}  // namespace

// Seed groups: kWideGroups for rows of more than kSmallD elements; for
// shorter rows the most powers of two up to kOrdMaxC that leave each group
// at least kOrdRowsPerGroup rows.  Fine groups pay where neighbours are near
// in few dimensions: at 4 10^6 uniform rows of 8 elements, 256 groups against
// 16 cut the tile's time by 8% (577 -> 530 ms; 512 and 1024 groups measured
// the same within the spread and cost more in the assignment); rows of 32 and
// 64 elements (Gaussian mixtures, 10^5 and 10^6 rows) were slower with 64 or
// 256 groups, whose workgroups share fewer reference streams.
constexpr int64_t kOrdRowsPerGroup = 8192;

int32_t order_groups(int64_t nr, int64_t d) {
  if (d > kSmallD) return kWideGroups;
  int64_t g = kWideGroups;
  while (g * 2 <= kOrdMaxC && g * 2 * kOrdRowsPerGroup <= nr) g *= 2;
  return (int32_t)g;
}

int32_t order_blocks(int64_t nr) { return (int32_t)((nr + kOrdRows - 1) / kOrdRows); }

hipError_t launch_order(const Plan& p, const Args& a, hipStream_t st) {
  const int64_t n = p.nr;
  const int nb = order_blocks(n);
  const int G = p.groups;
  const unsigned ga = (unsigned)((n + kAssignThreads - 1) / kAssignThreads);
  if (p.d <= kSmallD) {
    const int DT = (int)((p.d + 3) & ~3);
    hipLaunchKernelGGL(seeds_kernel, dim3((unsigned)((G * DT + 255) / 256)), dim3(256), 0, st,
                       a.xr, n, (int)p.d, G, DT, a.oseed);
    const auto kern = DT == 4   ? assign_small_kernel<4>
                      : DT == 8 ? assign_small_kernel<8>
                      : DT == 12 ? assign_small_kernel<12>
                                 : assign_small_kernel<16>;
    hipLaunchKernelGGL(kern, dim3(ga), dim3(kAssignThreads), 0, st, a.xr, n, (int)p.d, G,
                       reinterpret_cast<const float4*>(a.oseed), a.lab);
  } else {
    if (G != kWideGroups) return hipErrorInvalidValue;
    hipLaunchKernelGGL(assign_kernel, dim3(ga), dim3(kAssignThreads),
                       sizeof(float) * kWideGroups * (size_t)p.d, st, a.xr, n, (int)p.d, a.lab);
  }
  hipLaunchKernelGGL(count_kernel, dim3((unsigned)nb), dim3(256), 0, st, a.lab, n, G, a.bcnt);
  hipLaunchKernelGGL(block_offsets_kernel, dim3((unsigned)((G + 3) / 4)), dim3(256), 0, st,
                     a.bcnt, nb, G, a.boff, a.cstart);
  hipLaunchKernelGGL(group_starts_kernel, dim3(1), dim3(64), 0, st, G, a.cstart);
  hipLaunchKernelGGL(scatter_kernel, dim3((unsigned)nb), dim3(64), 0, st, a.lab, n, G, a.boff,
                     a.cstart, a.perm);
  return hipGetLastError();
}

}  // namespace tod
