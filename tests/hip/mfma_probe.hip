// Test-only probe of the MFMA arithmetic the distance tile relies on: one
// wave runs the chain  acc = C0;  acc = v_mfma_f32_32x32x16_{f16,bf16}(A_c, B_c, acc)
// for c = 0 .. kc-1, i.e. C = C0 + A B with A: 32 x 16kc, B: 16kc x 32, and
// writes C (fp32, row-major 32 x 32).  Operand layout of the instruction:
// lane l holds row (A) / column (B) l % 32, elements 16c + 8 (l / 32) .. +7;
// accumulator r of lane l is C[8 (r / 4) + 4 (l / 32) + r % 4][l % 32].
// The host side compares C with the exact sums (the certificate's model of
// the fp32 accumulation error).  Not part of the library.
#include <hip/hip_runtime.h>

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

template <typename V, bool BF>
__global__ void __launch_bounds__(64) chain(const unsigned short* A, const unsigned short* B,
                                            const float* C0, float* C, int kc) {
  const int l = threadIdx.x, col = l & 31, h = l >> 5;
  const int K = 16 * kc;
  f32x16 acc;
  for (int r = 0; r < 16; ++r) acc[r] = C0[(8 * (r >> 2) + 4 * h + (r & 3)) * 32 + col];
  for (int c = 0; c < kc; ++c) {
    V a, b;
    for (int e = 0; e < 8; ++e) {
      const unsigned short ua = A[col * K + 16 * c + 8 * h + e];
      const unsigned short ub = B[(16 * c + 8 * h + e) * 32 + col];
      a[e] = __builtin_bit_cast(typename std::remove_reference<decltype(a[0])>::type, ua);
      b[e] = __builtin_bit_cast(typename std::remove_reference<decltype(b[0])>::type, ub);
    }
    if constexpr (BF)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
    else
      acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc, 0, 0, 0);
  }
  for (int r = 0; r < 16; ++r) C[(8 * (r >> 2) + 4 * h + (r & 3)) * 32 + col] = acc[r];
}

extern "C" int probe_mfma_chain(int bf16, const void* A, const void* B, const void* C0, void* C,
                                int kc, void* stream) {
  if (kc < 1 || !A || !B || !C0 || !C) return 1;
  if (bf16)
    hipLaunchKernelGGL((chain<bf16x8, true>), dim3(1), dim3(64), 0, (hipStream_t)stream,
                       (const unsigned short*)A, (const unsigned short*)B, (const float*)C0,
                       (float*)C, kc);
  else
    hipLaunchKernelGGL((chain<f16x8, false>), dim3(1), dim3(64), 0, (hipStream_t)stream,
                       (const unsigned short*)A, (const unsigned short*)B, (const float*)C0,
                       (float*)C, kc);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
