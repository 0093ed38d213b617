// Fused distance tile + top-K' selection (Section 6.1's cdist + topk fusion,
// evaluated in the filter precision of Section 5.2 step ii).
//
// Work decomposition.  A workgroup of W waves owns W x 32 queries and walks
// one reference split in tiles of 32 rows.  The quantised reference tile is
// staged once per workgroup in LDS (double-buffered: the next tile's global
// loads are in flight while the current tile is consumed) and read by every
// wave; each wave keeps its 32 queries' operand in registers.  A wave's
// 32 x 32 tile of keys lands as 16 accumulators per lane, lane = query
// (lane % 32), accumulator r = reference tile_row(r, lane).
//
//   fp16 / bf16: v_mfma_f32_32x32x16_{f16,bf16}, A = reference rows from
//                LDS, B = query rows from registers, C seeded with -N_j/2.
//   fp32:        v_fma_f32 chains, reference rows broadcast from LDS.
//
// acc = -N_j/2 + <xhat_i, xhat_j>; key = -2 acc = fl(N_j) - 2 <xhat_i, xhat_j>.
//
// Selection.  Per query: a sorted list of its K' best (key, index) entries
// and a queue of fresh survivors (16 slots per query and half-wave) in LDS,
// plus an acc-space threshold per lane.  A tile costs a max3 reduction and
// one compare per lane unless a lane beats its threshold.  Survivors are
// appended; a query whose queue half would overflow is merged into its list
// by a bitonic network inside a 32-lane half (two queries per network), which
// also lowers that query's threshold.
#pragma once

#include <type_traits>

#include "halfwave.h"
#include "tod_internal.h"
#include "wave.h"

namespace tod {
namespace tile {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kQH = 16;       // queue slots per (query, half-wave)
constexpr int kQ = 2 * kQH;   // queue slots per query

template <int PREC>
struct Elem;
template <>
struct Elem<TOD_PREC_FP32> {
  using T = float;
  static constexpr int size = 4;
};
template <>
struct Elem<TOD_PREC_FP16> {
  using T = _Float16;
  using V = half8_t;
  static constexpr int size = 2;
};
template <>
struct Elem<TOD_PREC_BF16> {
  using T = __bf16;
  using V = bf16x8_t;
  static constexpr int size = 2;
};

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Maximum of three (v_max3_f32, formed by the compiler).  Not inline asm: the
// compiler inserts the wait states a VALU read of an MFMA result needs only
// for instructions it generates itself.  The operands are never NaN.
__device__ __forceinline__ float max3(float a, float b, float c) {
  return __builtin_fmaxf(__builtin_fmaxf(a, b), c);
}

// Reference row (0..31 within the tile) held by accumulator r of `lane`.
template <int PREC>
__device__ __forceinline__ int tile_row(int r, int lane) {
  if constexpr (PREC == TOD_PREC_FP32) {
    return 16 * (lane >> 5) + r;
  } else {
    // 32x32 MFMA accumulator layout: column = lane % 32, rows as below.
    return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  }
}

__host__ __device__ constexpr int row_bytes(int dpad, int es) { return dpad * es + 16; }

// Rows longer than the register-operand shapes are staged in column slabs of
// kSlabBytes per row (32 rows per slab), so LDS use does not grow with d:
// at most 33 KiB of slab plus the lists (K' = 256: 72 KiB) per workgroup.
constexpr int kSlabBytes = 1024;

// LDS bytes of the tile kernel for these parameters (host and device agree).
// dbuf: the double-buffered whole-row staging of the register-operand shapes.
__host__ __device__ constexpr size_t lds_bytes(int dpad, int es, int kp, int w, bool dbuf) {
  return (dbuf ? (size_t)2 * 32 * row_bytes(dpad, es) : (size_t)32 * (kSlabBytes + 16)) + 256 +
         (size_t)w * 32 * (kp + kQ) * sizeof(uint64_t);
}

// Merge the queues of the queries in `qmask` (bit q = query q of this wave)
// into their lists; two queries per half-wave network.
template <int KP>
__device__ void flush_queries(uint64_t* lbuf, const uint64_t* qbuf, uint32_t qmask, int& cnt,
                              float& thr, int lane) {
  constexpr int R = KP <= 32 ? 1 : KP / 32;
  constexpr int TR = (KP - 1) >> 5, TL = (KP - 1) & 31;
  wave_lds_sync();
  const int h = lane >> 5, j = lane & 31;
  while (qmask) {
    const int qa = __builtin_ctz(qmask);
    qmask &= qmask - 1;
    int qb = -1;
    if (qmask) {
      qb = __builtin_ctz(qmask);
      qmask &= qmask - 1;
    }
    const int q = h ? qb : qa;
    const int ca0 = __builtin_amdgcn_readlane(cnt, qa);
    const int ca1 = __builtin_amdgcn_readlane(cnt, qa + 32);
    const int cb0 = qb >= 0 ? __builtin_amdgcn_readlane(cnt, qb) : 0;
    const int cb1 = qb >= 0 ? __builtin_amdgcn_readlane(cnt, qb + 32) : 0;
    const int pos = j & (kQH - 1), sh = j >> 4;
    const int c = h ? (sh ? cb1 : cb0) : (sh ? ca1 : ca0);
    uint64_t e = kEmpty;
    if (q >= 0 && pos < c) e = qbuf[q * kQ + sh * kQH + pos];
    half_sort32(e, lane);
    uint64_t list[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int idx = r * 32 + j;
      list[r] = (q >= 0 && idx < KP) ? lbuf[q * KP + idx] : kEmpty;
    }
    half_merge<R>(list, e, lane);
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int idx = r * 32 + j;
      if (q >= 0 && idx < KP) lbuf[q * KP + idx] = list[r];
    }
    const uint32_t lo = (uint32_t)list[TR], hi = (uint32_t)(list[TR] >> 32);
    const uint64_t ta = ((uint64_t)__builtin_amdgcn_readlane(hi, TL) << 32) |
                        __builtin_amdgcn_readlane(lo, TL);
    const uint64_t tb = ((uint64_t)__builtin_amdgcn_readlane(hi, 32 + TL) << 32) |
                        __builtin_amdgcn_readlane(lo, 32 + TL);
    if (j == qa) {
      thr = ta == kEmpty ? -INFINITY : -0.5f * key_of(ta);
      cnt = 0;
    }
    if (j == qb) {
      thr = tb == kEmpty ? -INFINITY : -0.5f * key_of(tb);
      cnt = 0;
    }
  }
  wave_lds_sync();
}

template <int PREC, int KP, int W, int DPAD>
__global__ void __launch_bounds__(W * 64)
tile_kernel(Args a, int64_t q_begin, int64_t q_rows) {
  using T = typename Elem<PREC>::T;
  constexpr int ES = Elem<PREC>::size;
  constexpr bool QREG = DPAD > 0;  // query operand held in registers
  const int dpad = QREG ? DPAD : a.dpad;
  // Staged row stride: whole rows (register-operand shapes) or one slab.
  const int rowb = QREG ? row_bytes(dpad, ES) : kSlabBytes + 16;
  const int tile_bytes = 32 * rowb;
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* tiles = smem;
  float* hnbuf = (float*)(smem + (QREG ? 2 : 1) * tile_bytes);
  uint64_t* wbase = (uint64_t*)(smem + (QREG ? 2 : 1) * tile_bytes + 256);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  uint64_t* lbuf = wbase + (size_t)wave * 32 * (KP + kQ);
  uint64_t* qbuf = lbuf + 32 * KP;
  if (a.ctrl->nonfinite) return;  // uniform: every thread reads the same flag

  const int64_t group = (int64_t)blockIdx.x * W + wave;
  const bool active = group * 32 < q_rows;
  const int64_t q0 = q_begin + group * 32;
  const int split = blockIdx.y;
  const int64_t r_begin = (int64_t)split * a.split_len;
  const int64_t r_end = r_begin + a.split_len < a.nr ? r_begin + a.split_len : a.nr;
  const int myq = lane & 31;
  const bool selfq = a.exclude_self != 0;
  const T* xqq = (const T*)a.xq_q;
  const unsigned char* xr_bytes = (const unsigned char*)a.xq_r;

  // Query operand.
  constexpr int KC = QREG ? (PREC == TOD_PREC_FP32 ? DPAD / 4 : DPAD / 16) : 1;
  using QV = typename std::conditional<PREC == TOD_PREC_FP32, float4,
                                       typename Elem<PREC == TOD_PREC_FP32 ? TOD_PREC_FP16
                                                                           : PREC>::V>::type;
  QV qv[KC];
  const T* qrow = xqq + (active ? q0 + myq : 0) * (int64_t)dpad;
  if constexpr (QREG) {
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      if constexpr (PREC == TOD_PREC_FP32)
        qv[c] = *reinterpret_cast<const float4*>(qrow + 4 * c);
      else
        qv[c] = *reinterpret_cast<const QV*>(qrow + 16 * c + 8 * (lane >> 5));
    }
  }

  for (int i = lane; i < 32 * (KP + kQ); i += 64) lbuf[i] = kEmpty;
  wave_lds_sync();
  float thr = -INFINITY;  // a pair survives iff acc > thr
  int cnt = 0;            // entries in this lane's queue half
  uint64_t* myqueue = qbuf + myq * kQ + (lane >> 5) * kQH;

  // Tile staging: chunks of 16 bytes, row-major.
  const int cpr = dpad * ES / 16;  // chunks per row
  const int n16 = 32 * cpr;
  constexpr int NL = QREG ? (32 * DPAD * ES / 16 + W * 64 - 1) / (W * 64) : 1;
  uint4 st[NL];
  float4 sth = make_float4(0.f, 0.f, 0.f, 0.f);
  auto fetch = [&](int64_t t0) {
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int c = tid + i * W * 64;
      if (c < n16) {
        const int row = c / cpr, cc = c % cpr;
        st[i] = *reinterpret_cast<const uint4*>(xr_bytes + (t0 + row) * (int64_t)dpad * ES +
                                                cc * 16);
      }
    }
    if (tid < 8) sth = *reinterpret_cast<const float4*>(a.hn_r + t0 + 4 * tid);
  };
  auto put = [&](int b) {
    unsigned char* buf = tiles + b * tile_bytes;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int c = tid + i * W * 64;
      if (c < n16) {
        const int row = c / cpr, cc = c % cpr;
        *reinterpret_cast<uint4*>(buf + row * rowb + cc * 16) = st[i];
      }
    }
    if (tid < 8) *reinterpret_cast<float4*>(hnbuf + b * 32 + 4 * tid) = sth;
  };
  // Long rows: columns [c0, c0 + w) of the tile's 32 rows (one slab, w * ES
  // <= kSlabBytes), single-buffered; the seeds come with the first slab.
  auto copy_slab = [&](int64_t t0, int c0, int w) {
    const int scpr = w * ES / 16;
    for (int c = tid; c < 32 * scpr; c += W * 64) {
      const int row = c / scpr, cc = c % scpr;
      *reinterpret_cast<uint4*>(tiles + row * rowb + cc * 16) = *reinterpret_cast<const uint4*>(
          xr_bytes + ((t0 + row) * (int64_t)dpad + c0) * ES + cc * 16);
    }
    if (c0 == 0 && tid < 8)
      *reinterpret_cast<float4*>(hnbuf + 4 * tid) =
          *reinterpret_cast<const float4*>(a.hn_r + t0 + 4 * tid);
  };
  constexpr int kSlabE = kSlabBytes / ES;  // elements per slab row

  if constexpr (QREG) {
    fetch(r_begin);
    put(0);
  }
  __syncthreads();
  // Seeds of the tile's accumulators: -N_j/2 of the rows this lane holds.
  auto seed_fp32 = [&](const float* hn, float (&acc)[16]) {
    const float* hnp = hn + 16 * (lane >> 5);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 v = *reinterpret_cast<const float4*>(hnp + 4 * g);
      acc[4 * g + 0] = v.x;
      acc[4 * g + 1] = v.y;
      acc[4 * g + 2] = v.z;
      acc[4 * g + 3] = v.w;
    }
  };
  auto seed_mfma = [&](const float* hn, floatx16& cacc) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 v = *reinterpret_cast<const float4*>(hn + 8 * g + 4 * (lane >> 5));
      cacc[4 * g + 0] = v.x;
      cacc[4 * g + 1] = v.y;
      cacc[4 * g + 2] = v.z;
      cacc[4 * g + 3] = v.w;
    }
  };
  // Add the products of columns [c0, c0 + w) (staged rows in buf, whose
  // column 0 is column c0) to the accumulators.
  // Chunk c (4 columns) of the FMA chain: query values q4, staged rows at rbase.
  auto fma_chunk = [&](const unsigned char* rbase, int c, float4 q4, float (&acc)[16]) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float4 rv = *reinterpret_cast<const float4*>(rbase + r * rowb + 16 * c);
      acc[r] = fmaf(q4.x, rv.x, acc[r]);
      acc[r] = fmaf(q4.y, rv.y, acc[r]);
      acc[r] = fmaf(q4.z, rv.z, acc[r]);
      acc[r] = fmaf(q4.w, rv.w, acc[r]);
    }
  };
  auto accum_fp32 = [&](const unsigned char* buf, int c0, int w, float (&acc)[16]) {
    const unsigned char* rbase = buf + 16 * (lane >> 5) * rowb;
    if constexpr (QREG && PREC == TOD_PREC_FP32) {
#pragma unroll
      for (int c = 0; c < KC; ++c) fma_chunk(rbase, c, qv[c], acc);
    } else {
#pragma nounroll
      for (int c = 0; c < w / 4; ++c)
        fma_chunk(rbase, c, *reinterpret_cast<const float4*>(qrow + c0 + 4 * c), acc);
    }
  };
  auto accum_mfma = [&](const unsigned char* buf, int c0, int w, floatx16& cacc) {
    if constexpr (PREC != TOD_PREC_FP32) {
      using V = typename Elem<PREC>::V;
      const unsigned char* arow = buf + myq * rowb + (lane >> 5) * 16;
      auto step = [&](int c, V bv) {
        const V av = *reinterpret_cast<const V*>(arow + 32 * c);
        if constexpr (PREC == TOD_PREC_FP16)
          cacc = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, bv, cacc, 0, 0, 0);
        else
          cacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, cacc, 0, 0, 0);
      };
      if constexpr (QREG) {
#pragma unroll
        for (int c = 0; c < KC; ++c) step(c, qv[c]);
      } else {
#pragma nounroll
        for (int c = 0; c < w / 16; ++c)
          step(c, *reinterpret_cast<const V*>(qrow + c0 + 16 * c + 8 * (lane >> 5)));
      }
    }
  };
  int it = 0;
  for (int64_t t0 = r_begin; t0 < r_end; t0 += 32, ++it) {
    const bool nxt = t0 + 32 < r_end;
    float acc[16];
    if constexpr (QREG) {
      if (nxt) fetch(t0 + 32);
      const int b = it & 1;
      const unsigned char* buf = tiles + b * tile_bytes;
      const float* hn = hnbuf + b * 32;
      if (active) {
        if constexpr (PREC == TOD_PREC_FP32) {
          seed_fp32(hn, acc);
          accum_fp32(buf, 0, dpad, acc);
        } else {
          floatx16 cacc;
          seed_mfma(hn, cacc);
          accum_mfma(buf, 0, dpad, cacc);
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[r] = cacc[r];
        }
      }
    } else {
      // Slab by slab: every wave takes part in the staging and barriers.
      floatx16 cacc;
      for (int c0 = 0; c0 < dpad; c0 += kSlabE) {
        const int w = dpad - c0 < kSlabE ? dpad - c0 : kSlabE;
        if (c0) __syncthreads();  // the previous slab has been consumed
        copy_slab(t0, c0, w);
        __syncthreads();
        if (active) {
          if constexpr (PREC == TOD_PREC_FP32) {
            if (c0 == 0) seed_fp32(hnbuf, acc);
            accum_fp32(tiles, c0, w, acc);
          } else {
            if (c0 == 0) seed_mfma(hnbuf, cacc);
            accum_mfma(tiles, c0, w, cacc);
          }
        }
      }
      if constexpr (PREC != TOD_PREC_FP32) {
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] = cacc[r];
      }
    }
    if (active) {
      const bool diag = selfq && t0 == q0;
      if (diag || t0 + 32 > r_end) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = tile_row<PREC>(r, lane);
          if (t0 + row >= r_end || (diag && row == myq)) acc[r] = -INFINITY;
        }
      }
      float m = max3(acc[0], acc[1], acc[2]);
#pragma unroll
      for (int r = 3; r < 15; r += 2) m = max3(m, acc[r], acc[r + 1]);
      m = fmaxf(m, acc[15]);
      if (__ballot(m > thr)) {
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const uint64_t need = __ballot(cnt > kQH - 4);
          if (need)
            flush_queries<KP>(lbuf, qbuf, (uint32_t)need | (uint32_t)(need >> 32), cnt, thr,
                              lane);
#pragma unroll
          for (int r = 4 * rg; r < 4 * rg + 4; ++r) {
            if (acc[r] > thr) {
              myqueue[cnt] = make_entry(-2.0f * acc[r], (uint32_t)(t0 + tile_row<PREC>(r, lane)));
              ++cnt;
            }
          }
        }
      }
    }
    if constexpr (QREG) {
      if (nxt) put((it + 1) & 1);
    }
    __syncthreads();
  }
  if (active) {
    const uint64_t need = __ballot(cnt > 0);
    if (need) flush_queries<KP>(lbuf, qbuf, (uint32_t)need | (uint32_t)(need >> 32), cnt, thr,
                                lane);
    for (int q = 0; q < 32; ++q) {
      const int64_t ql = group * 32 + q;
      if (ql >= q_rows) break;
      uint64_t* dst = a.partial + (ql * a.splits + split) * KP;
      for (int e = lane; e < KP; e += 64) dst[e] = lbuf[q * KP + e];
    }
  }
}

template <int PREC, int KP, int W, int DPAD>
hipError_t launch_one(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                      hipStream_t st) {
  constexpr int ES = Elem<PREC>::size;
  const size_t lds = lds_bytes(DPAD > 0 ? DPAD : p.dpad, ES, KP, W, DPAD > 0);
  const auto kern = tile_kernel<PREC, KP, W, DPAD>;
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const int64_t groups = (q_rows + 31) / 32;
  const dim3 grid((unsigned)((groups + W - 1) / W), (unsigned)p.splits);
  hipLaunchKernelGGL(kern, grid, dim3(W * 64), lds, st, a, q_begin, q_rows);
  return hipGetLastError();
}

template <int PREC, int KP, int W>
hipError_t launch_kp(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                     hipStream_t st) {
  if constexpr (PREC == TOD_PREC_FP32) {
    switch (p.dpad_t) {
      case 8: return launch_one<PREC, KP, W, 8>(p, a, q_begin, q_rows, st);
      case 16: return launch_one<PREC, KP, W, 16>(p, a, q_begin, q_rows, st);
      case 32: return launch_one<PREC, KP, W, 32>(p, a, q_begin, q_rows, st);
      case 64: return launch_one<PREC, KP, W, 64>(p, a, q_begin, q_rows, st);
      default: return launch_one<PREC, KP, W, 0>(p, a, q_begin, q_rows, st);
    }
  } else {
    switch (p.dpad_t) {
      case 16: return launch_one<PREC, KP, W, 16>(p, a, q_begin, q_rows, st);
      case 32: return launch_one<PREC, KP, W, 32>(p, a, q_begin, q_rows, st);
      case 64: return launch_one<PREC, KP, W, 64>(p, a, q_begin, q_rows, st);
      case 128: return launch_one<PREC, KP, W, 128>(p, a, q_begin, q_rows, st);
      default: return launch_one<PREC, KP, W, 0>(p, a, q_begin, q_rows, st);
    }
  }
}

template <int PREC>
hipError_t launch_prec(const Plan& p, const Args& a, int64_t q_begin, int64_t q_rows,
                       hipStream_t st) {
  switch (p.kprime) {
    case 16: return launch_kp<PREC, 16, 4>(p, a, q_begin, q_rows, st);
    case 32: return launch_kp<PREC, 32, 4>(p, a, q_begin, q_rows, st);
    case 64: return launch_kp<PREC, 64, 2>(p, a, q_begin, q_rows, st);
    case 128: return launch_kp<PREC, 128, 1>(p, a, q_begin, q_rows, st);
    case 256: return launch_kp<PREC, 256, 1>(p, a, q_begin, q_rows, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tile
}  // namespace tod
