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

}  // namespace

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
