// LOF from the exact kNN lists (Table 1's LOF; Breunig et al. 2000, with
// exactly k neighbours per point, self excluded):
//   kdist(o)   = D(o, k-th neighbour of o)
//   reach(p,o) = max(kdist(o), D(p,o))
//   lrd(p)     = 1 / (mean_o reach(p,o) + 1e-10)
//   LOF(p)     = mean_o lrd(o) / lrd(p)
// All arithmetic is fp64 in neighbour order, without fused multiply-add; two
// gather passes over the n x k lists (HBM / L2 bound).
#include "tod_internal.h"

namespace tod {

namespace {

constexpr int kThreads = 256;

__global__ void __launch_bounds__(kThreads)
lrd_kernel(int64_t n, int k, const int32_t* __restrict__ idx, const double* __restrict__ d64,
           double* __restrict__ lrd, const Ctrl* ctrl) {
#pragma clang fp contract(off)
  if (ctrl->nonfinite) return;
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  double sum = 0.0;
  for (int s = 0; s < k; ++s) {
    const int64_t o = idx[p * k + s];
    const double dpo = d64[p * k + s];
    const double ko = (o >= 0 && o < n) ? d64[o * k + (k - 1)] : dpo;
    const double reach = ko > dpo ? ko : dpo;
    sum = sum + reach;
  }
  lrd[p] = 1.0 / (sum / (double)k + 1e-10);
}

__global__ void __launch_bounds__(kThreads)
lof_kernel(int64_t n, int k, const int32_t* __restrict__ idx, const double* __restrict__ lrd,
           float* __restrict__ lof, const Ctrl* ctrl) {
#pragma clang fp contract(off)
  if (ctrl->nonfinite) return;
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  double sum = 0.0;
  for (int s = 0; s < k; ++s) {
    const int64_t o = idx[p * k + s];
    sum = sum + ((o >= 0 && o < n) ? lrd[o] : lrd[p]);
  }
  lof[p] = (float)((sum / (double)k) / lrd[p]);
}

}  // namespace

hipError_t launch_lof(const Plan& p, const Args& a, hipStream_t st) {
  const unsigned g = (unsigned)((p.nq + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(lrd_kernel, dim3(g), dim3(kThreads), 0, st, p.nq, p.k, a.idx32, a.d64, a.lrd,
                     a.ctrl);
  hipLaunchKernelGGL(lof_kernel, dim3(g), dim3(kThreads), 0, st, p.nq, p.k, a.idx32, a.lrd,
                     a.lof_out, a.ctrl);
  return hipGetLastError();
}

}  // namespace tod
