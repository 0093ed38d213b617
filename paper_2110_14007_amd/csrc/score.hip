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
//   abod   Section 4.3's ABOD: the mean cosine over pairs of neighbours of
//          the differences to them (abod_kernel below).
//   cof    Table 1's COF: average chaining distance of the set-based nearest
//          path over the point and its neighbours, relative to the
//          neighbours' (cof_ac_kernel, cof_kernel below).
// Scores and votes take one thread per query row: O(k) and O(k^2) work per
// row on lists the previous kernels just wrote (L2-resident).
#include <math.h>

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

// ABOD as Section 4.3 builds it from the kNN and cosine-similarity operators:
// for point i with neighbours b, c the cosine of the angle between
// x_b - x_i and x_c - x_i, averaged over the unordered pairs of distinct
// neighbours.  One wave per point: the Gram matrix of the k difference
// vectors (k <= 64, b <= c: at most 2080 entries, 33 per lane) is summed in
// fp64 over the columns in order, 16 columns at a time staged through LDS
// as exact fp64 differences; then each lane turns its off-diagonal entries
// into cosines (pairs with a zero-length difference are left out) and the
// wave averages them.  A point without any pair left scores 0.
constexpr int kAbodMaxK = 64;
constexpr int kAbodCols = 16;
constexpr int kAbodPer = (kAbodMaxK * (kAbodMaxK + 1) / 2 + 63) / 64;

__global__ void __launch_bounds__(256)
abod_kernel(int64_t n, int k, int d, const float* __restrict__ x, const int32_t* __restrict__ idx,
            float* __restrict__ out, const Ctrl* ctrl) {
#pragma clang fp contract(off)
  __shared__ double diff[4][kAbodMaxK][kAbodCols];
  __shared__ double norm[4][kAbodMaxK];
  __shared__ uint32_t pairs[kAbodMaxK * (kAbodMaxK + 1) / 2];
  if (ctrl->nonfinite) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int T = k * (k + 1) / 2;
  // (b, c) of entry e, b <= c, row-major over the upper triangle.
  for (int b = 0, e = 0; b < k; ++b)
    for (int c = b; c < k; ++c, ++e)
      if (e % 256 == (int)threadIdx.x % 256 && e < T) pairs[e] = ((uint32_t)b << 16) | (uint32_t)c;
  __syncthreads();
  const int64_t row = (int64_t)blockIdx.x * 4 + wave;
  if (row >= n) return;  // uniform per wave; no block barrier follows
  const int32_t* nb = idx + row * k;
  const float* xi = x + row * (int64_t)d;
  double acc[kAbodPer];
#pragma unroll
  for (int m = 0; m < kAbodPer; ++m) acc[m] = 0.0;
  for (int t0 = 0; t0 < d; t0 += kAbodCols) {
    for (int q = lane; q < k * kAbodCols; q += 64) {
      const int b = q / kAbodCols, t = q % kAbodCols;
      const int64_t j = nb[b];
      diff[wave][b][t] = t0 + t < d ? (double)x[j * d + t0 + t] - (double)xi[t0 + t] : 0.0;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
#pragma unroll
    for (int m = 0; m < kAbodPer; ++m) {
      const int e = lane + 64 * m;
      if (e < T) {
        const int b = (int)(pairs[e] >> 16), c = (int)(pairs[e] & 0xffff);
        double s = acc[m];
        for (int t = 0; t < kAbodCols; ++t) s = s + diff[wave][b][t] * diff[wave][c][t];
        acc[m] = s;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  }
#pragma unroll
  for (int m = 0; m < kAbodPer; ++m) {
    const int e = lane + 64 * m;
    if (e < T && (pairs[e] >> 16) == (pairs[e] & 0xffff)) norm[wave][pairs[e] & 0xffff] = acc[m];
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  double sum = 0.0;
  int cnt = 0;
#pragma unroll
  for (int m = 0; m < kAbodPer; ++m) {
    const int e = lane + 64 * m;
    if (e < T) {
      const int b = (int)(pairs[e] >> 16), c = (int)(pairs[e] & 0xffff);
      const double nbb = norm[wave][b], ncc = norm[wave][c];
      if (b != c && nbb > 0.0 && ncc > 0.0) {
        sum = sum + acc[m] / sqrt(nbb * ncc);
        ++cnt;
      }
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    sum = sum + __shfl_xor(sum, o, 64);
    cnt += __shfl_xor(cnt, o, 64);
  }
  if (lane == 0) out[row] = (float)(cnt ? sum / (double)cnt : 0.0);
}

// COF (Tang et al., Table 1): for point p and the point set G = {p} +
// N_k(p), the set-based nearest path starts from S = {p} and adds, k times,
// the point of G outside S nearest to S (ties to the lower row index); the
// i-th step costs that distance c_i and the average chaining distance is
// ac(p) = sum_i 2 (k + 1 - i) / (k (k + 1)) c_i.  One wave per point (lane l
// stands for the l-th point of G): the squared distances of all pairs of G
// (the fp64 column-ordered sums of the definition, at most 2016 pairs, 32 per
// lane), then k steps of a wave-wide argmin over the points outside S.
constexpr int kCofMaxK = 63;
constexpr int kCofPer = ((kCofMaxK + 1) * kCofMaxK / 2 + 63) / 64;

__global__ void __launch_bounds__(64)
cof_ac_kernel(int64_t n, int k, int d, const float* __restrict__ x,
              const int32_t* __restrict__ idx, double* __restrict__ ac, const Ctrl* ctrl) {
#pragma clang fp contract(off)
  __shared__ double rows[kCofMaxK + 1][kAbodCols];
  __shared__ double d2m[kCofMaxK + 1][kCofMaxK + 2];
  __shared__ uint32_t pairs[(kCofMaxK + 1) * kCofMaxK / 2];
  if (ctrl->nonfinite) return;
  const int lane = threadIdx.x;
  const int64_t p = blockIdx.x;
  const int m = k + 1;
  const int T = m * (m - 1) / 2;
  for (int b = 0, e = 0; b < m; ++b)
    for (int c = b + 1; c < m; ++c, ++e)
      if ((e & 63) == lane) pairs[e] = ((uint32_t)b << 16) | (uint32_t)c;
  auto gid = [&](int l) -> int64_t { return l == 0 ? p : (int64_t)idx[p * k + l - 1]; };
  double acc[kCofPer];
#pragma unroll
  for (int q = 0; q < kCofPer; ++q) acc[q] = 0.0;
  for (int t0 = 0; t0 < d; t0 += kAbodCols) {
    for (int q = lane; q < m * kAbodCols; q += 64) {
      const int l = q / kAbodCols, t = q % kAbodCols;
      rows[l][t] = t0 + t < d ? (double)x[gid(l) * d + t0 + t] : 0.0;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
#pragma unroll
    for (int q = 0; q < kCofPer; ++q) {
      const int e = lane + 64 * q;
      if (e < T) {
        const int b = (int)(pairs[e] >> 16), c = (int)(pairs[e] & 0xffff);
        double s = acc[q];
        for (int t = 0; t < kAbodCols; ++t) {
          const double df = rows[b][t] - rows[c][t];
          s = s + df * df;
        }
        acc[q] = s;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  }
#pragma unroll
  for (int q = 0; q < kCofPer; ++q) {
    const int e = lane + 64 * q;
    if (e < T) {
      const int b = (int)(pairs[e] >> 16), c = (int)(pairs[e] & 0xffff);
      d2m[b][c] = acc[q];
      d2m[c][b] = acc[q];
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  const bool live = lane < m;
  bool in_s = lane == 0;
  double best = live && lane > 0 ? d2m[0][lane] : INFINITY;
  const uint32_t gl = live ? (uint32_t)gid(lane) : 0xffffffffu;
  double total = 0.0;
  for (int i = 1; i <= k; ++i) {
    double kb = (live && !in_s) ? best : INFINITY;
    uint32_t kg = (live && !in_s) ? gl : 0xffffffffu;
    int kl = lane;
    for (int o = 32; o > 0; o >>= 1) {
      const double ob = __shfl_xor(kb, o, 64);
      const uint32_t og = __shfl_xor(kg, o, 64);
      const int ol = __shfl_xor(kl, o, 64);
      if (ob < kb || (ob == kb && og < kg)) {
        kb = ob;
        kg = og;
        kl = ol;
      }
    }
    total = total + 2.0 * (double)(k + 1 - i) / (double)(k * (k + 1)) * sqrt(kb);
    if (lane == kl) in_s = true;
    if (live && !in_s && d2m[kl][lane] < best) best = d2m[kl][lane];
  }
  if (lane == 0) ac[p] = total;
}

__global__ void __launch_bounds__(kThreads)
cof_kernel(int64_t n, int k, const int32_t* __restrict__ idx, const double* __restrict__ ac,
           float* __restrict__ out, const Ctrl* ctrl) {
#pragma clang fp contract(off)
  if (ctrl->nonfinite) return;
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  double s = 0.0;
  for (int r = 0; r < k; ++r) s = s + ac[idx[p * k + r]];
  out[p] = (float)((ac[p] + 1e-10) / (s / (double)k + 1e-10));
}

}  // namespace

hipError_t launch_cof(const Plan& p, const Args& a, hipStream_t st) {
  hipLaunchKernelGGL(cof_ac_kernel, dim3((unsigned)p.nq), dim3(64), 0, st, p.nq, p.k, (int)p.d,
                     a.xq, (const int32_t*)a.idx32, a.lrd, (const Ctrl*)a.ctrl);
  hipLaunchKernelGGL(cof_kernel, dim3((unsigned)((p.nq + kThreads - 1) / kThreads)),
                     dim3(kThreads), 0, st, p.nq, p.k, (const int32_t*)a.idx32,
                     (const double*)a.lrd, a.lof_out, (const Ctrl*)a.ctrl);
  return hipGetLastError();
}

hipError_t launch_abod(const Plan& p, const Args& a, hipStream_t st) {
  hipLaunchKernelGGL(abod_kernel, dim3((unsigned)((p.nq + 3) / 4)), dim3(256), 0, st, p.nq, p.k,
                     (int)p.d, a.xq, (const int32_t*)a.idx32, a.score_out, (const Ctrl*)a.ctrl);
  return hipGetLastError();
}

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
