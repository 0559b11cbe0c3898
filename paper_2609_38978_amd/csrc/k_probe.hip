// Hardware probes behind the certified fast paths.
//
// The k-means assignment and the PAMA retrieval accept a fast bf16-MFMA
// result only when it is provably the float64 one, under two error models of
// the hardware: every addition of a v_mfma_f32_32x32x16_bf16 accumulation
// chain errs by at most 2^-23 of the magnitudes involved, and v_exp_f32 has a
// small relative error.  These kernels run exactly those instructions on
// caller-chosen operands so that tests can measure both against float64.
#include "common.h"
#include "kernels.h"

namespace park {

typedef __bf16 pb_bf16x8_t __attribute__((ext_vector_type(8)));
typedef float pb_f32x16_t __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256) void k_probe_exp2(const float* __restrict__ x,
                                                    float* __restrict__ y, long n) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i < n) y[i] = __builtin_amdgcn_exp2f(x[i]);
}

// One wavefront per problem p: C[p] = C0[p] + A[p] Bt[p]^T as a chain of
// K / 16 MFMAs in k order (the shape of the k-means and PAMA score chains).
// A [32][K] and Bt [32][K] bf16 (row i of A, column j of B), C0, C [32][32].
// Lane l supplies row l % 32 of A and column l % 32 of B, k = 16 s + 8 (l / 32)
// .. + 8; accumulator element q of lane l is C[8 (q / 4) + 4 (l / 32) + q % 4][l % 32].
__global__ __launch_bounds__(64) void k_probe_mfma(const bf16_t* __restrict__ A,
                                                   const bf16_t* __restrict__ Bt,
                                                   const float* __restrict__ C0,
                                                   float* __restrict__ Cout, int K) {
  const int p = blockIdx.x, l = threadIdx.x, c32 = l & 31, hf = l >> 5;
  const bf16_t* Ap = A + (size_t)p * 32 * K + (size_t)c32 * K + 8 * hf;
  const bf16_t* Bp = Bt + (size_t)p * 32 * K + (size_t)c32 * K + 8 * hf;
  const float* c0 = C0 + (size_t)p * 1024;
  pb_f32x16_t acc;
#pragma unroll
  for (int q = 0; q < 16; ++q) acc[q] = c0[(8 * (q >> 2) + 4 * hf + (q & 3)) * 32 + c32];
  for (int s = 0; s < K / 16; ++s) {
    const pb_bf16x8_t a = __builtin_bit_cast(pb_bf16x8_t, *(const uint4*)(Ap + 16 * s));
    const pb_bf16x8_t b = __builtin_bit_cast(pb_bf16x8_t, *(const uint4*)(Bp + 16 * s));
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
  }
  float* co = Cout + (size_t)p * 1024;
#pragma unroll
  for (int q = 0; q < 16; ++q) co[(8 * (q >> 2) + 4 * hf + (q & 3)) * 32 + c32] = acc[q];
}

park_status launch_probe_exp2(const float* x, float* y, long n, hipStream_t st) {
  if (n == 0) return PARK_OK;
  PARK_LAUNCH("probe_exp2", k_probe_exp2, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, x,
              y, n);
  return PARK_OK;
}

park_status launch_probe_mfma(const bf16_t* A, const bf16_t* Bt, const float* C0, float* C,
                              int nprob, int K, hipStream_t st) {
  if (nprob == 0) return PARK_OK;
  PARK_LAUNCH("probe_mfma", k_probe_mfma, dim3(nprob), dim3(64), 0, st, A, Bt, C0, C, K);
  return PARK_OK;
}

}  // namespace park
