// Input quantisation: step (i) of provable quantization (Section 5.2).
//
// Every row x is replaced for the filter by xhat = Q(s * (x - mu)), where mu
// is the fp32-rounded column mean of the references (centring shrinks the
// norms that enter the rounding bound), s is a power of two that puts
// max |s (x - mu)| just below 2^14 (exact scaling; Section 5.3 scales the
// input for the same reason), and Q rounds to the filter precision with
// values below the smallest normal flushed to zero.  Distances are invariant
// under the translation and s is exact, so ||x_i - x_j|| * s is exactly the
// distance between the real vectors c = s (x - mu).
//
// Per row the kernel also records, in fp64:
//   N    = ||xhat||^2                          (query rows: for the certificate)
//   hn   = -0.5 * fl32(N)                      (reference rows: accumulator seed)
//   rho  >= ||c - xhat||                       (quantisation radius, rounded up)
// and over the references the maxima Nmax = max N and Pmax = max rho.
// With the grouped scan order (order.hip) the reference rows are written in
// that order: position p holds input row perm[p].
#include <math.h>

#include "tod_internal.h"

namespace tod {

namespace {

constexpr int kThreads = 256;
constexpr int kFinalCols = 8;  // columns per block of the column-mean final sum

__global__ void init_ctrl_kernel(Ctrl* ctrl) {
  uint32_t* w = reinterpret_cast<uint32_t*>(ctrl);
  for (int i = threadIdx.x; i < (int)(sizeof(Ctrl) / 4); i += blockDim.x) w[i] = 0;
}

// Column partial sums of the references over contiguous row ranges
// (deterministic: fixed ranges, fixed reduction order).
__global__ void __launch_bounds__(kThreads)
colsum_partial_kernel(const float* __restrict__ x, int64_t n, int d, int64_t rows_per_block,
                      double* __restrict__ part) {
  __shared__ double red[kThreads];
  const int cpp = d < kThreads ? d : kThreads;  // columns per pass
  const int rsub = kThreads / cpp;              // row lanes per column
  const int tid = threadIdx.x;
  const int c_off = tid % cpp, r_off = tid / cpp;
  const int64_t r0 = (int64_t)blockIdx.x * rows_per_block;
  const int64_t r1 = r0 + rows_per_block < n ? r0 + rows_per_block : n;
  for (int cbase = 0; cbase < d; cbase += cpp) {
    const int c = cbase + c_off;
    double s = 0.0;
    if (r_off < rsub && c < d)
      for (int64_t r = r0 + r_off; r < r1; r += rsub) s += (double)x[r * d + c];
    red[tid] = s;
    __syncthreads();
    if (tid < cpp && cbase + tid < d) {
      double t = 0.0;
      for (int i = 0; i < rsub; ++i) t += red[i * cpp + tid];
      part[(int64_t)blockIdx.x * d + cbase + tid] = t;
    }
    __syncthreads();
  }
}

// One block per group of columns: kThreads / cpb threads per column sum
// fixed, strided subsets of the partial sums, then a fixed-order tree
// (deterministic).
__global__ void __launch_bounds__(kThreads)
colsum_final_kernel(const double* __restrict__ part, int nb, int d, int64_t n,
                    double* __restrict__ mu64, float* __restrict__ mu32) {
  __shared__ double red[kThreads];
  const int cpb = d < kFinalCols ? d : kFinalCols;  // columns per block
  const int tpc = kThreads / cpb;                   // threads per column
  const int tid = threadIdx.x, cl = tid % cpb, sub = tid / cpb;
  const int c = blockIdx.x * cpb + cl;
  double t = 0.0;
  if (sub < tpc && c < d)
    for (int b = sub; b < nb; b += tpc) t += part[(int64_t)b * d + c];
  red[tid] = t;
  __syncthreads();
  if (sub == 0 && c < d) {
    double s = 0.0;
    for (int i = 0; i < tpc; ++i) s += red[i * cpb + cl];
    const double m = s / (double)n;
    mu64[c] = m;
    mu32[c] = (float)m;
  }
}

// max |x - mu| (fp32 bits, rounded up) and the non-finite flag.
__global__ void __launch_bounds__(kThreads)
maxabs_kernel(const float* __restrict__ x, int64_t rows, int d, const float* __restrict__ mu32,
              Ctrl* ctrl) {
  __shared__ float red[kThreads];
  float m = 0.0f;
  bool bad = false;
  const int64_t total = rows * d;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  // The column index is tracked incrementally (no division per element).
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int cstep = (int)(stride % d);
  int col = (int)(i0 % d);
  for (int64_t i = i0; i < total; i += stride) {
    const float v = x[i];
    const int cc = col;
    col += cstep;
    col = col >= d ? col - d : col;
    if (!isfinite(v)) {
      bad = true;
    } else {
      const double diff = fabs((double)v - (double)mu32[cc]);
      float f = (float)diff;
      if ((double)f < diff) f = nextafterf(f, INFINITY);
      m = fmaxf(m, f);
    }
  }
  if (bad) atomicOr(&ctrl->nonfinite, 1u);
  red[threadIdx.x] = m;
  __syncthreads();
  for (int w = kThreads / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + w]);
    __syncthreads();
  }
  if (threadIdx.x == 0) atomicMax(&ctrl->maxabs_bits, __float_as_uint(red[0]));
}

template <typename T>
__device__ __forceinline__ T quantise(double c);

template <>
__device__ __forceinline__ float quantise<float>(double c) {
  float f = (float)c;
  return fabsf(f) < 1.17549435e-38f ? 0.0f : f;
}

template <>
__device__ __forceinline__ _Float16 quantise<_Float16>(double c) {
  _Float16 h = (_Float16)(float)c;
  return fabsf((float)h) < 6.103515625e-05f ? (_Float16)0.0f : h;
}

template <>
__device__ __forceinline__ __bf16 quantise<__bf16>(double c) {
  __bf16 b = (__bf16)(float)c;
  return fabsf((float)b) < 1.17549435e-38f ? (__bf16)0.0f : b;
}

// Largest value over the wave (non-negative doubles compare as their bits).
__device__ __forceinline__ double wave_max(double v) {
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = __shfl_xor((uint32_t)b, off, 64);
    const uint32_t hi = __shfl_xor((uint32_t)(b >> 32), off, 64);
    const double o = __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
    v = o > v ? o : v;
  }
  return v;
}

// Largest value over the workgroup of kThreads threads, for every thread
// (every lane of a wave may hold its own value).  All threads must call it.
__device__ __forceinline__ double block_max(double v, double* red) {
  v = wave_max(v);
  __syncthreads();  // red may still be in use by a previous call
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double m = red[0];
  for (int w = 1; w < kThreads / 64; ++w) m = red[w] > m ? red[w] : m;
  return m;
}

__device__ __forceinline__ void atomic_max_nonneg(uint64_t* addr, double v) {
  atomicMax((unsigned long long*)addr, (unsigned long long)__double_as_longlong(v));
}

// The seed -N/2 as four parts of v = -N/(2c) in the filter precision, split
// greedily (p_1 = Q(v), p_2 = Q(v - p_1), ...; every residual is exact in
// fp64, so the sum of the parts stays exact too); returns err >=
// |c sum p + N/2|, rounded up.  The certificate adds the largest err over the
// references.
template <typename T>
__device__ __forceinline__ double seed_parts(double nsq, double cfold, T (&q)[4]) {
  double v = -0.5 * nsq / cfold, sum = 0.0;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    q[t] = (T)(float)v;
    const double qd = (double)(float)q[t];
    sum += qd;
    v -= qd;
  }
  const double e = fabs(cfold * sum + 0.5 * nsq);
  return e * (1.0 + 0x1p-40) + 0x1p-60 * nsq;
}

// One thread per row, rows walked with a grid stride.  Rows in [n, n_pad)
// are zero-filled so that the tile kernels may read whole 32-row tiles.  The
// reference maxima are kept per thread and reduced over the workgroup at the
// end: one atomic per maximum per workgroup, and at most 1024 workgroups
// (same-address atomics serialise: one per 256 rows cost about half of this
// kernel's time at 4 x 10^6 rows).  Rows of 8-element chunks are written 16
// bytes at a time.
//
// Fold layout (fold != 0): columns [0, d) hold xhat, [d, dmain) zeros,
// [dmain, dmain + 4) the seed parts p_1..p_4 in the filter precision and the
// rest zeros.  The parts split v = -N/(2c) greedily (p_1 = Q(v), p_2 =
// Q(v - p_1), ...), every residual exact in fp64, so that c * sum p = -N/2 up
// to err = |c sum p + N/2|, computed exactly and rounded up; the certificate
// adds the largest err over the references.
template <typename T>
__global__ void __launch_bounds__(kThreads)
quantise_kernel(const float* __restrict__ x, int64_t n, int64_t n_pad, int d, int dpad,
                const float* __restrict__ mu32, Ctrl* ctrl, T* __restrict__ xq,
                float* __restrict__ hn, double* __restrict__ n64, double* __restrict__ rho,
                int is_ref, int fold, int dmain, int scale_exp, double cfold,
                const int32_t* __restrict__ perm, int seedprod) {
  const double s = scale_from_maxabs(ctrl->maxabs_bits, scale_exp);
  const bool vec = (dpad & 7) == 0 && sizeof(T) * 8 % 16 == 0;
  double mn = 0.0, mp = 0.0, mf = 0.0;  // this thread's maxima
  for (int64_t row = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; row < n_pad;
       row += (int64_t)gridDim.x * blockDim.x) {
    T* out = xq + row * dpad;
    if (row >= n) {
      for (int t = 0; t < dpad; ++t) out[t] = (T)0.0f;
      if (hn && seedprod) reinterpret_cast<uint2*>(hn)[row] = make_uint2(0u, 0u);
      else if (hn) hn[row] = 0.0f;
      if (n64) n64[row] = 0.0;
      if (rho) rho[row] = 0.0;
      continue;
    }
    const float* in = x + (perm ? (int64_t)perm[row] : row) * d;
    double nsq = 0.0, r2 = 0.0, c2 = 0.0, ferr = 0.0;
    // Element t of the padded row (the sums advance in column order).
    double v = 0.0, fsum = 0.0;
    auto elem = [&](int t) -> T {
      if (t < d) {
        const double c = s * ((double)in[t] - (double)mu32[t]);
        const T q = quantise<T>(c);
        const double qd = (double)(float)q;
        nsq += qd * qd;
        r2 += (c - qd) * (c - qd);
        c2 += c * c;
        return q;
      }
      if (fold && t >= dmain && t < dmain + 4) {
        if (t == dmain) v = -0.5 * nsq / cfold;
        const T q = (T)(float)v;
        const double qd = (double)(float)q;
        fsum += qd;  // parts of decreasing magnitude: the sum stays exact
        v -= qd;     // exact: qd is v rounded to fewer bits
        return q;
      }
      return (T)0.0f;
    };
    if (vec) {
      for (int t0 = 0; t0 < dpad; t0 += 8) {
        T buf[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) buf[e] = elem(t0 + e);
#pragma unroll
        for (int h = 0; h < (int)(sizeof(T) * 8 / 16); ++h)
          reinterpret_cast<uint4*>(out + t0)[h] = reinterpret_cast<const uint4*>(buf)[h];
      }
    } else {
      for (int t = 0; t < dpad; ++t) out[t] = elem(t);
    }
    if (fold) {
      const double e = fabs(cfold * fsum + 0.5 * nsq);
      ferr = e * (1.0 + 0x1p-40) + 0x1p-60 * nsq;
    }
    // Round the radius up: covers the fp64 rounding of c and of the sums.
    const double rho_up = sqrt(r2) * (1.0 + 0x1p-40) + 0x1p-50 * sqrt(c2);
    if (is_ref && seedprod) {
      T q[4];
      ferr = seed_parts<T>(nsq, cfold, q);
      reinterpret_cast<uint2*>(hn)[row] = *reinterpret_cast<const uint2*>(q);
    } else if (is_ref) {
      hn[row] = -0.5f * (float)nsq;
    }
    if (n64) n64[row] = nsq;
    if (rho) rho[row] = rho_up;
    mn = nsq > mn ? nsq : mn;
    mp = rho_up > mp ? rho_up : mp;
    mf = ferr > mf ? ferr : mf;
  }
  if (is_ref) {  // uniform: one atomic per maximum per workgroup
    __shared__ double red[kThreads / 64];
    const double bn = block_max(mn, red), bp = block_max(mp, red);
    const double bf = block_max(mf, red);
    if (threadIdx.x == 0) {
      atomic_max_nonneg(&ctrl->nmax_bits, bn);
      atomic_max_nonneg(&ctrl->pmax_bits, bp);
      atomic_max_nonneg(&ctrl->fold_max_bits, bf);
    }
  }
}

// Sum over the wave (butterfly: every lane ends with the same value).
__device__ __forceinline__ double wave_sum(double v) {
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = __shfl_xor((uint32_t)b, off, 64);
    const uint32_t hi = __shfl_xor((uint32_t)(b >> 32), off, 64);
    v = v + __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
  }
  return v;
}

// One wave per row for rows without the fold layout: the row is read and the
// quantised row written with the lanes over the columns (coalesced), and the
// three sums are reduced over the wave.  Same outputs as quantise_kernel; the
// sums are added in another order, which the certificate's allowances for the
// fp64 rounding of N and rho cover.  Each wave walks rows with a grid stride
// and issues one atomic per maximum at the end.
template <typename T>
__global__ void __launch_bounds__(kThreads)
quantise_rows_kernel(const float* __restrict__ x, int64_t n, int64_t n_pad, int d, int dpad,
                     const float* __restrict__ mu32, Ctrl* ctrl, T* __restrict__ xq,
                     float* __restrict__ hn, double* __restrict__ n64,
                     double* __restrict__ rho, int is_ref, int scale_exp,
                     const int32_t* __restrict__ perm, int seedprod, double cfold) {
  const int lane = threadIdx.x & 63;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  const double s = scale_from_maxabs(ctrl->maxabs_bits, scale_exp);
  double wn = 0.0, wp = 0.0;  // this wave's maxima (the same in every lane)
  double wf = 0.0;            // largest seed-part error (lane 0)
  for (int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6; row < n_pad;
       row += nwaves) {
    T* out = xq + row * dpad;
    if (row >= n) {
      for (int t = lane; t < dpad; t += 64) out[t] = (T)0.0f;
      if (lane == 0) {
        if (hn && seedprod) reinterpret_cast<uint2*>(hn)[row] = make_uint2(0u, 0u);
        else if (hn) hn[row] = 0.0f;
        if (n64) n64[row] = 0.0;
        if (rho) rho[row] = 0.0;
      }
      continue;
    }
    const float* in = x + (perm ? (int64_t)perm[row] : row) * d;
    double nsq = 0.0, r2 = 0.0, c2 = 0.0;
    for (int t = lane; t < dpad; t += 64) {
      T q = (T)0.0f;
      if (t < d) {
        const double c = s * ((double)in[t] - (double)mu32[t]);
        q = quantise<T>(c);
        const double qd = (double)(float)q;
        nsq += qd * qd;
        r2 += (c - qd) * (c - qd);
        c2 += c * c;
      }
      out[t] = q;
    }
    nsq = wave_sum(nsq);
    r2 = wave_sum(r2);
    c2 = wave_sum(c2);
    // Round the radius up: covers the fp64 rounding of c and of the sums.
    const double rho_up = sqrt(r2) * (1.0 + 0x1p-40) + 0x1p-50 * sqrt(c2);
    if (lane == 0) {
      if (is_ref && seedprod) {
        T q[4];
        const double ferr = seed_parts<T>(nsq, cfold, q);
        reinterpret_cast<uint2*>(hn)[row] = *reinterpret_cast<const uint2*>(q);
        wf = ferr > wf ? ferr : wf;
      } else if (is_ref) {
        hn[row] = -0.5f * (float)nsq;
      }
      if (n64) n64[row] = nsq;
      if (rho) rho[row] = rho_up;
    }
    wn = nsq > wn ? nsq : wn;
    wp = rho_up > wp ? rho_up : wp;
  }
  if (is_ref) {  // uniform: one atomic per maximum per workgroup
    __shared__ double red[kThreads / 64];
    const double bn = block_max(wn, red), bp = block_max(wp, red);
    const double bf = block_max(wf, red);
    if (threadIdx.x == 0) {
      atomic_max_nonneg(&ctrl->nmax_bits, bn);
      atomic_max_nonneg(&ctrl->pmax_bits, bp);
      if (seedprod) atomic_max_nonneg(&ctrl->fold_max_bits, bf);
    }
  }
}

template <typename T>
hipError_t launch_quantise(const Plan& p, const Args& a, hipStream_t st) {
  const double cf = fold_const(p.precision);
  if (!p.fold && p.d >= 64) {
    // 4 waves per block; at most 1024 blocks (one atomic per maximum each).
    const auto grid_rows = [](int64_t rows) {
      int64_t g = (rows + 3) / 4;
      return (unsigned)(g < 1 ? 1 : (g > 1024 ? 1024 : g));
    };
    hipLaunchKernelGGL(quantise_rows_kernel<T>, dim3(grid_rows(p.nr_pad)), dim3(kThreads), 0, st,
                       a.xr, p.nr, p.nr_pad, (int)p.d, p.dpad, a.mu32, a.ctrl, (T*)a.xq_r,
                       a.hn_r, p.self ? a.n64_q : (double*)nullptr,
                       p.self ? a.rho_q : a.rho_r, 1, p.scale_exp, a.perm, p.seedprod, cf);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.self) return e;
    hipLaunchKernelGGL(quantise_rows_kernel<T>, dim3(grid_rows(p.nq_pad)), dim3(kThreads), 0, st,
                       a.xq, p.nq, p.nq_pad, (int)p.d, p.dpad, a.mu32, a.ctrl, (T*)a.xq_q,
                       (float*)nullptr, a.n64_q, a.rho_q, 0, p.scale_exp,
                       (const int32_t*)nullptr, 0, cf);
    return hipGetLastError();
  }
  const auto grid_threads = [](int64_t rows) {
    const int64_t g = (rows + kThreads - 1) / kThreads;
    return (unsigned)(g < 1 ? 1 : (g > 1024 ? 1024 : g));
  };
  const unsigned blocks_r = grid_threads(p.nr_pad);
  hipLaunchKernelGGL(quantise_kernel<T>, dim3(blocks_r), dim3(kThreads), 0, st, a.xr,
                     p.nr, p.nr_pad, (int)p.d, p.dpad, a.mu32, a.ctrl, (T*)a.xq_r, a.hn_r,
                     p.self ? a.n64_q : (double*)nullptr, p.self ? a.rho_q : a.rho_r, 1,
                     p.fold, p.dmain, p.scale_exp, cf, a.perm, p.seedprod);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.self) return e;
  const unsigned blocks_q = grid_threads(p.nq_pad);
  hipLaunchKernelGGL(quantise_kernel<T>, dim3(blocks_q), dim3(kThreads), 0, st, a.xq,
                     p.nq, p.nq_pad, (int)p.d, p.dpad, a.mu32, a.ctrl, (T*)a.xq_q, (float*)nullptr,
                     a.n64_q, a.rho_q, 0, p.fold, p.dmain, p.scale_exp, cf,
                     (const int32_t*)nullptr, 0);
  return hipGetLastError();
}

}  // namespace

// About 1024 blocks of consecutive rows for the column partial sums (enough
// to fill the GPU when n is small and d large, few enough partials per
// column for the final sum).
int32_t colsum_blocks(int64_t nr) {
  const int64_t rpb = (nr + 1023) / 1024;
  return (int32_t)((nr + rpb - 1) / rpb);
}

hipError_t launch_prep(const Plan& p, const Args& a, hipStream_t st) {
  hipLaunchKernelGGL(init_ctrl_kernel, dim3(1), dim3(64), 0, st, a.ctrl);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int32_t nb = colsum_blocks(p.nr);
  const int64_t rpb = (p.nr + nb - 1) / nb;
  hipLaunchKernelGGL(colsum_partial_kernel, dim3(nb), dim3(kThreads), 0, st, a.xr, p.nr,
                     (int)p.d, rpb, a.colpart);
  const int cpb = p.d < kFinalCols ? (int)p.d : kFinalCols;
  hipLaunchKernelGGL(colsum_final_kernel, dim3((unsigned)((p.d + cpb - 1) / cpb)),
                     dim3(kThreads), 0, st, a.colpart, nb, (int)p.d, p.nr, a.mu64, a.mu32);
  // At most 1024 blocks: each ends with one atomic on the same word, and
  // same-address atomics serialise.
  const auto grid_for = [](int64_t total) {
    int64_t g = (total + kThreads * 4 - 1) / (kThreads * 4);
    return (unsigned)(g < 1 ? 1 : (g > 1024 ? 1024 : g));
  };
  hipLaunchKernelGGL(maxabs_kernel, dim3(grid_for(p.nr * p.d)), dim3(kThreads), 0, st, a.xr,
                     p.nr, (int)p.d, a.mu32, a.ctrl);
  if (!p.self)
    hipLaunchKernelGGL(maxabs_kernel, dim3(grid_for(p.nq * p.d)), dim3(kThreads), 0, st, a.xq,
                       p.nq, (int)p.d, a.mu32, a.ctrl);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.order) {
    e = launch_order(p, a, st);
    if (e != hipSuccess) return e;
  }
  switch (p.precision) {
    case TOD_PREC_FP32: return launch_quantise<float>(p, a, st);
    case TOD_PREC_FP16: return launch_quantise<_Float16>(p, a, st);
    default: return launch_quantise<__bf16>(p, a, st);
  }
}

}  // namespace tod
