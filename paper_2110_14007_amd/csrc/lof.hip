// LOF from the exact kNN lists (Table 1's LOF; Breunig et al. 2000, with
// exactly k neighbours per point, self excluded):
//   kdist(o)   = D(o, k-th neighbour of o)
//   reach(p,o) = max(kdist(o), D(p,o))
//   lrd(p)     = 1 / (mean_o reach(p,o) + 1e-10)
//   LOF(p)     = mean_o lrd(o) / lrd(p)
// All arithmetic is fp64 in neighbour order, without fused multiply-add; two
// gather passes over the n x k lists (HBM / L2 bound).
//
// Access pattern.  A workgroup takes P <= kFlat / k consecutive points.  Its
// threads first walk the P k (point, neighbour) entries flat, so that the
// list reads are coalesced, gather the neighbour's value from a dense n-array
// (kdist for lrd, lrd for LOF; the recheck writes kdist beside the lists) and
// park the entry's term in LDS; then one thread per point adds its k terms in
// neighbour order.
#include "tod_internal.h"

namespace tod {

namespace {

constexpr int kThreads = 256;
constexpr int kFlat = 4096;  // (point, neighbour) terms a workgroup parks in LDS (32 KiB)

__global__ void __launch_bounds__(kThreads)
lrd_kernel(int64_t n, int k, int P, const int32_t* __restrict__ idx,
           const double* __restrict__ d64, const double* __restrict__ kdist,
           double* __restrict__ lrd, const Ctrl* ctrl) {
#pragma clang fp contract(off)
  __shared__ double term[kFlat];
  if (ctrl->nonfinite) return;
  const int64_t p0 = (int64_t)blockIdx.x * P;
  const int64_t pend = p0 + P < n ? p0 + P : n;
  const int64_t f0 = p0 * k, f1 = pend * k;
  for (int64_t f = f0 + threadIdx.x; f < f1; f += kThreads) {
    const int64_t o = idx[f];
    const double dpo = d64[f];
    const double ko = (o >= 0 && o < n) ? kdist[o] : dpo;
    term[f - f0] = ko > dpo ? ko : dpo;  // reach(p, o)
  }
  __syncthreads();
  const int64_t p = p0 + threadIdx.x;
  if (threadIdx.x < P && p < n) {
    const double* t = term + (int64_t)threadIdx.x * k;
    double sum = 0.0;
    for (int s = 0; s < k; ++s) sum = sum + t[s];
    lrd[p] = 1.0 / (sum / (double)k + 1e-10);
  }
}

__global__ void __launch_bounds__(kThreads)
lof_kernel(int64_t n, int k, int P, const int32_t* __restrict__ idx,
           const double* __restrict__ lrd, float* __restrict__ lof, const Ctrl* ctrl) {
#pragma clang fp contract(off)
  __shared__ double term[kFlat];
  if (ctrl->nonfinite) return;
  const int64_t p0 = (int64_t)blockIdx.x * P;
  const int64_t pend = p0 + P < n ? p0 + P : n;
  const int64_t f0 = p0 * k, f1 = pend * k;
  for (int64_t f = f0 + threadIdx.x; f < f1; f += kThreads) {
    const int64_t o = idx[f];
    term[f - f0] = (o >= 0 && o < n) ? lrd[o] : lrd[f / k];
  }
  __syncthreads();
  const int64_t p = p0 + threadIdx.x;
  if (threadIdx.x < P && p < n) {
    const double* t = term + (int64_t)threadIdx.x * k;
    double sum = 0.0;
    for (int s = 0; s < k; ++s) sum = sum + t[s];
    lof[p] = (float)((sum / (double)k) / lrd[p]);
  }
}

// ---------------------------------------------------------------------------
// LOF on tie-inclusive k-distance neighbourhoods (tod_lof_ties; Breunig et
// al.'s N_k(p), which keeps every point tied at the k-distance, so that it can
// hold more than k points; Section 5.3's range operator finds it):
//   kd2(p)   = the k-th smallest D2(p, o), o != p
//   N_k(p)   = {o != p : D2(p, o) <= kd2(p)}     (a range query per row)
//   reach(p, o) = max(sqrt(kd2(o)), sqrt(D2(p, o)))
//   lrd(p)   = 1 / (sum_N reach / |N_k(p)| + 1e-10)
//   LOF(p)   = (sum_N lrd(o) / |N_k(p)|) / lrd(p)
// D2 is the definition's fp64 sum over the columns in order (exact_d2), the
// same arithmetic as the range query's exact test, so that a point tied with
// the k-th neighbour in that arithmetic lands in N_k(p) and no list entry
// falls out of it.  One wave per point; the per-lane partial sums are added
// in a fixed butterfly (run-to-run identical).
// ---------------------------------------------------------------------------

__device__ __forceinline__ double wave_sum(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// kd2[p] = the largest D2(p, o) over p's k exact neighbours, i.e. the k-th
// smallest (the largest, should the list order disagree with the column-order
// sum in the last bit).  The lists hold k1 = k + 1 neighbours when another
// point exists: a row whose (k+1)-th neighbour is farther than kd2 by more
// than the two summation orders can differ (relative 1e-11, against at most
// (d + 2) 2^-52 for d <= 4096) has no point tied at its k-distance, so its
// neighbourhood is its k-list; any other row sets *tie.
__global__ void __launch_bounds__(256)
ties_radius_kernel(const float* __restrict__ x, int64_t n, int d, int k, int k1,
                   const int64_t* __restrict__ lists, double* __restrict__ kd2,
                   int32_t* __restrict__ tie) {
#pragma clang fp contract(off)
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t p = (int64_t)blockIdx.x * 4 + wave;
  if (p >= n) return;  // uniform per wave
  const float* xp = x + p * (int64_t)d;
  double m = 0.0, nxt = INFINITY;
  for (int i = lane; i < k1; i += 64) {
    const int64_t o = lists[p * k1 + i];
    const double v = exact_d2(xp, x + o * (int64_t)d, d);
    if (i < k) m = v > m ? v : m;
    else nxt = v;
  }
  for (int o = 32; o > 0; o >>= 1) {
    const double t = __shfl_xor(m, o, 64);
    m = t > m ? t : m;
    const double u = __shfl_xor(nxt, o, 64);
    nxt = u < nxt ? u : nxt;
  }
  if (lane == 0) {
    kd2[p] = m;
    if (k1 > k && !(nxt * (1.0 - 1e-11) > m)) *tie = 1;
  }
}

__global__ void tie_clear_kernel(int32_t* tie) {
  if (threadIdx.x == 0) *tie = 0;
}

// Neighbourhoods of a set with no ties at the k-distance: the first k entries
// of every (k1-entry) list, as CSR.
__global__ void __launch_bounds__(256)
ties_lists_kernel(int64_t n, int k, int k1, const int64_t* __restrict__ lists,
                  int64_t* __restrict__ row_ptr, int64_t* __restrict__ nbr) {
  const int64_t f = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (f < n * k) nbr[f] = lists[(f / k) * k1 + f % k];
  if (f <= n) row_ptr[f] = f * k;
}

__global__ void __launch_bounds__(256)
lrd_ties_kernel(const float* __restrict__ x, int64_t n, int d, const int64_t* __restrict__ row_ptr,
                const int64_t* __restrict__ nbr, const double* __restrict__ kd2,
                double* __restrict__ lrd) {
#pragma clang fp contract(off)
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t p = (int64_t)blockIdx.x * 4 + wave;
  if (p >= n) return;  // uniform per wave
  const float* xp = x + p * (int64_t)d;
  const int64_t beg = row_ptr[p], end = row_ptr[p + 1];
  double sum = 0.0;
  for (int64_t e = beg + lane; e < end; e += 64) {
    const int64_t o = nbr[e];
    const double dpo = sqrt(exact_d2(xp, x + o * (int64_t)d, d));
    const double ko = sqrt(kd2[o]);
    sum = sum + (ko > dpo ? ko : dpo);  // reach(p, o)
  }
  sum = wave_sum(sum);
  if (lane == 0) lrd[p] = 1.0 / (sum / (double)(end - beg) + 1e-10);
}

__global__ void __launch_bounds__(256)
lof_ties_kernel(int64_t n, const int64_t* __restrict__ row_ptr, const int64_t* __restrict__ nbr,
                const double* __restrict__ lrd, float* __restrict__ lof,
                int32_t* __restrict__ count) {
#pragma clang fp contract(off)
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t p = (int64_t)blockIdx.x * 4 + wave;
  if (p >= n) return;  // uniform per wave
  const int64_t beg = row_ptr[p], end = row_ptr[p + 1];
  double sum = 0.0;
  for (int64_t e = beg + lane; e < end; e += 64) sum = sum + lrd[nbr[e]];
  sum = wave_sum(sum);
  if (lane == 0) {
    lof[p] = (float)((sum / (double)(end - beg)) / lrd[p]);
    if (count) count[p] = (int32_t)(end - beg);
  }
}

}  // namespace

hipError_t launch_ties_radius(const float* x, int64_t n, int d, int k, int k1,
                              const int64_t* lists, double* kd2, int32_t* tie, hipStream_t st) {
  hipLaunchKernelGGL(tie_clear_kernel, dim3(1), dim3(64), 0, st, tie);
  hipLaunchKernelGGL(ties_radius_kernel, dim3((unsigned)((n + 3) / 4)), dim3(256), 0, st, x, n, d,
                     k, k1, lists, kd2, tie);
  return hipGetLastError();
}

hipError_t launch_ties_lists(int64_t n, int k, int k1, const int64_t* lists, int64_t* row_ptr,
                             int64_t* nbr, hipStream_t st) {
  const int64_t cnt = n * k > n + 1 ? n * k : n + 1;
  hipLaunchKernelGGL(ties_lists_kernel, dim3((unsigned)((cnt + 255) / 256)), dim3(256), 0, st, n,
                     k, k1, lists, row_ptr, nbr);
  return hipGetLastError();
}

hipError_t launch_lof_ties(const float* x, int64_t n, int d, const int64_t* row_ptr,
                           const int64_t* nbr, const double* kd2, double* lrd, float* lof,
                           int32_t* count, hipStream_t st) {
  const unsigned g = (unsigned)((n + 3) / 4);
  hipLaunchKernelGGL(lrd_ties_kernel, dim3(g), dim3(256), 0, st, x, n, d, row_ptr, nbr, kd2, lrd);
  hipLaunchKernelGGL(lof_ties_kernel, dim3(g), dim3(256), 0, st, n, row_ptr, nbr,
                     (const double*)lrd, lof, count);
  return hipGetLastError();
}

hipError_t launch_lof(const Plan& p, const Args& a, hipStream_t st) {
  // Points per workgroup: P k <= kFlat terms fit in LDS and P <= kThreads
  // points are summed one per thread (k <= 256 gives P >= 16).
  const int P = kFlat / p.k < kThreads ? kFlat / p.k : kThreads;
  const unsigned g = (unsigned)((p.nq + P - 1) / P);
  hipLaunchKernelGGL(lrd_kernel, dim3(g), dim3(kThreads), 0, st, p.nq, p.k, P, a.idx32, a.d64,
                     a.kdist, a.lrd, a.ctrl);
  hipLaunchKernelGGL(lof_kernel, dim3(g), dim3(kThreads), 0, st, p.nq, p.k, P, a.idx32, a.lrd,
                     a.lof_out, a.ctrl);
  return hipGetLastError();
}

}  // namespace tod
