// kNN outlier-score aggregates and the kNN classifier's vote, both from the
// exact neighbour lists (int32 ids, fp64 distances, sorted by (distance, id))
// that the recheck and the fallback leave in the workspace.
//
//   score  Table 1's kNN detector scores a point by its neighbour distances:
//          the k-th one (written by the recheck itself), or their mean,
//          median (mean of the two middle ones for even k) or sum (the
//          weight of Angiulli and Pizzuti, whose detector the paper cites).
//          fp64 in neighbour order, rounded once to fp32.
//   vote   Appendix B's kNN classifier: the most frequent label among the k
//          neighbours, ties going to the smallest label.  A label outside
//          [0, n_classes) sets a flag the host turns into an error.
// One thread per query row: O(k) and O(k^2) work per row on lists the
// previous kernels just wrote (L2-resident).
#include "tod_internal.h"

namespace tod {

namespace {

constexpr int kThreads = 256;

__global__ void __launch_bounds__(kThreads)
score_kernel(int64_t n, int k, int score, const double* __restrict__ d64,
             float* __restrict__ out, const Ctrl* ctrl) {
#pragma clang fp contract(off)
  if (ctrl->nonfinite) return;
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  const double* d = d64 + p * k;
  double v;
  if (score == TOD_SCORE_MEDIAN) {
    v = (k & 1) ? d[k / 2] : 0.5 * (d[k / 2 - 1] + d[k / 2]);
  } else {
    double s = 0.0;
    for (int r = 0; r < k; ++r) s = s + d[r];
    v = score == TOD_SCORE_MEAN ? s / (double)k : s;
  }
  out[p] = (float)v;
}

__global__ void __launch_bounds__(kThreads)
vote_kernel(int64_t n, int k, int64_t nr, const int32_t* __restrict__ idx,
            const int32_t* __restrict__ labels, int32_t n_classes, int32_t* __restrict__ pred,
            Ctrl* ctrl) {
  if (ctrl->nonfinite) return;
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  const int32_t* nb = idx + p * k;
  auto label = [&](int r) {
    const int32_t j = nb[r];
    return (j >= 0 && j < nr) ? labels[j] : -1;
  };
  int32_t best = -1, best_n = 0;
  bool bad = false;
  for (int r = 0; r < k; ++r) {
    const int32_t c = label(r);
    if (c < 0 || c >= n_classes) {
      bad = true;
      continue;
    }
    // Count label c once, at its first occurrence in the list.
    bool seen = false;
    for (int s = 0; s < r && !seen; ++s) seen = label(s) == c;
    if (seen) continue;
    int cnt = 1;
    for (int s = r + 1; s < k; ++s) cnt += label(s) == c ? 1 : 0;
    if (cnt > best_n || (cnt == best_n && c < best)) {
      best = c;
      best_n = cnt;
    }
  }
  if (bad) atomicOr(&ctrl->bad_label, 1u);
  pred[p] = best;
}

}  // namespace

hipError_t launch_score(const Plan& p, const Args& a, hipStream_t st) {
  const unsigned g = (unsigned)((p.nq + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(score_kernel, dim3(g), dim3(kThreads), 0, st, p.nq, p.k, a.score,
                     (const double*)a.d64, a.score_out, (const Ctrl*)a.ctrl);
  return hipGetLastError();
}

hipError_t launch_vote(const Plan& p, const Args& a, hipStream_t st) {
  const unsigned g = (unsigned)((p.nq + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(vote_kernel, dim3(g), dim3(kThreads), 0, st, p.nq, p.k, p.nr,
                     (const int32_t*)a.idx32, a.labels_r, a.n_classes, a.pred_out, a.ctrl);
  return hipGetLastError();
}

}  // namespace tod
