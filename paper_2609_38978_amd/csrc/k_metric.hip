// QRKC query metric (Sec. 5.2, App. D.2 "Numerically stable Cholesky
// factorization", Alg. 3 first five steps):
//   G = Q^T Q / L, symmetrised;  s = max(tr G / d, s_min);
//   Gbar = (1 - alpha) G + alpha s I + eps s I;  Gbar = R R^T (R lower).
// Products of bf16/fp32 inputs are exact in float64, so the Gram matrix is
// accumulated with float64 FMAs; partial sums over row chunks are reduced in a
// fixed order (deterministic).
#include "common.h"
#include "kernels.h"

namespace park {

// Partial Gram matrix of one row chunk: part[h][chunk] = sum_r x_r x_r^T.
// 256 threads on a 16x16 grid; each owns a (D/16)x(D/16) tile of G.
template <typename T, int D>
__global__ __launch_bounds__(256) void k_gram_partial(const T* __restrict__ X, int N, int rows_per,
                                                      double* __restrict__ part) {
  constexpr int TS = D / 16;
  constexpr int RB = 32;  // rows staged per LDS round
  __shared__ float xs[RB][D + 4];
  const int h = blockIdx.y, ch = blockIdx.x, nch = gridDim.x;
  const int r0 = ch * rows_per, r1 = min(N, r0 + rows_per);
  const int ti = threadIdx.x >> 4, tj = threadIdx.x & 15;
  const T* Xh = X + (size_t)h * N * D;
  double acc[TS][TS];
#pragma unroll
  for (int a = 0; a < TS; ++a)
#pragma unroll
    for (int b = 0; b < TS; ++b) acc[a][b] = 0.0;

  for (int rb = r0; rb < r1; rb += RB) {
    const int nr = min(RB, r1 - rb);
    for (int e = threadIdx.x; e < RB * D; e += 256) {
      const int r = e / D, c = e % D;
      xs[r][c] = (r < nr) ? to_f(Xh[(size_t)(rb + r) * D + c]) : 0.0f;
    }
    __syncthreads();
    for (int r = 0; r < nr; ++r) {
      double xa[TS], xb[TS];
#pragma unroll
      for (int a = 0; a < TS; ++a) xa[a] = (double)xs[r][ti * TS + a];
#pragma unroll
      for (int b = 0; b < TS; ++b) xb[b] = (double)xs[r][tj * TS + b];
#pragma unroll
      for (int a = 0; a < TS; ++a)
#pragma unroll
        for (int b = 0; b < TS; ++b) acc[a][b] = fma(xa[a], xb[b], acc[a][b]);
    }
    __syncthreads();
  }
  double* out = part + ((size_t)h * nch + ch) * D * D;
#pragma unroll
  for (int a = 0; a < TS; ++a)
#pragma unroll
    for (int b = 0; b < TS; ++b) out[(ti * TS + a) * D + tj * TS + b] = acc[a][b];
}

// G[h] = (sum over chunks, in chunk order) / N
__global__ __launch_bounds__(256) void k_gram_reduce(const double* __restrict__ part, int nch, int DD,
                                                     double invN, double* __restrict__ G) {
  const int h = blockIdx.y;
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= DD) return;
  const double* p = part + (size_t)h * nch * DD + e;
  double s = 0.0;
  for (int c = 0; c < nch; ++c) s += p[(size_t)c * DD];
  G[(size_t)h * DD + e] = s * invN;
}

// Symmetrise, scale, stabilise and factorise; one workgroup per head, the
// matrix held in LDS.  Right-looking Cholesky in float64.
template <int D>
__global__ __launch_bounds__(256) void k_metric_chol(const double* __restrict__ G, double alpha,
                                                     double eps, double s_min,
                                                     double* __restrict__ Gbar_out,
                                                     double* __restrict__ R_out, int* status) {
  extern __shared__ double A[];  // D*D
  __shared__ double red[256];
  __shared__ double piv;
  __shared__ int bad;
  const int h = blockIdx.x, tid = threadIdx.x;
  const double* Gh = G + (size_t)h * D * D;
  for (int e = tid; e < D * D; e += 256) A[e] = Gh[e];
  if (tid == 0) bad = 0;
  __syncthreads();
  // symmetrise: (G + G^T) / 2
  for (int e = tid; e < D * D; e += 256) {
    const int i = e / D, j = e % D;
    if (i < j) {
      const double v = (A[i * D + j] + A[j * D + i]) / 2.0;
      A[i * D + j] = v;
      A[j * D + i] = v;
    }
  }
  __syncthreads();
  // s = max(tr G / d, s_min)
  double t = 0.0;
  if (tid == 0)
    for (int i = 0; i < D; ++i) t += A[i * D + i];
  if (tid == 0) red[0] = fmax(t / (double)D, s_min);
  __syncthreads();
  const double s = red[0];
  const double as = alpha * s, es = eps * s;
  for (int e = tid; e < D * D; e += 256) {
    const int i = e / D, j = e % D;
    double v = (1.0 - alpha) * A[e];
    if (i == j) v = (v + as) + es;
    if (!isfinite(v)) bad = 1;
    A[e] = v;
  }
  __syncthreads();
  double* Gb = Gbar_out + (size_t)h * D * D;
  for (int e = tid; e < D * D; e += 256) Gb[e] = A[e];
  // Cholesky, lower triangle in place
  for (int k = 0; k < D; ++k) {
    if (tid == 0) {
      const double p = A[k * D + k];
      if (!(p > 0.0) || !isfinite(p)) bad = 1;
      piv = sqrt(fmax(p, 0.0));
      A[k * D + k] = piv;
    }
    __syncthreads();
    const double lkk = piv;
    for (int i = k + 1 + tid; i < D; i += 256) A[i * D + k] = A[i * D + k] / lkk;
    __syncthreads();
    // trailing update of the lower triangle, 16 x 16 thread grid
    for (int i = k + 1 + (tid >> 4); i < D; i += 16) {
      const double lik = A[i * D + k];
      for (int j = k + 1 + (tid & 15); j <= i; j += 16)
        A[i * D + j] = fma(-lik, A[j * D + k], A[i * D + j]);
    }
    __syncthreads();
  }
  double* R = R_out + (size_t)h * D * D;
  for (int e = tid; e < D * D; e += 256) {
    const int i = e / D, j = e % D;
    R[e] = (j <= i) ? A[e] : 0.0;
  }
  if (tid == 0 && bad) raise_status(status, ST_NOT_SPD);
}

// Transformed points Xt = X R (row form of x~ = R^T x), float64 sums,
// float output.  Diagnostic only (the k-means uses the factored metric).
template <typename T, int D>
__global__ __launch_bounds__(D) void k_transform(const T* __restrict__ X, const double* __restrict__ R,
                                                 int N, float* __restrict__ Xt) {
  __shared__ double xr[D];
  const int h = blockIdx.y, j = threadIdx.x;
  const double* Rh = R + (size_t)h * D * D;
  for (int r = blockIdx.x; r < N; r += gridDim.x) {
    xr[j] = (double)to_f(X[((size_t)h * N + r) * D + j]);
    __syncthreads();
    double s = 0.0;
    for (int a = 0; a < D; ++a) s = fma(xr[a], Rh[a * D + j], s);
    Xt[((size_t)h * N + r) * D + j] = (float)s;
    __syncthreads();
  }
}

// ---------------------------------------------------------------- launchers
size_t gram_chunks(int H, int N) {
  // enough workgroups to fill the chip, at least 256 rows each
  int nch = (512 + H - 1) / H;
  nch = nch < 1 ? 1 : nch;
  const int max_by_rows = (N + 255) / 256;
  if (nch > max_by_rows) nch = max_by_rows;
  if (nch > 64) nch = 64;
  return (size_t)(nch < 1 ? 1 : nch);
}

park_status launch_metric(const void* Q, int H, int N, int D, int dtype, double alpha, double eps,
                          double s_min, double* part, double* G, double* Gbar, double* R,
                          int* status, hipStream_t st) {
  const int nch = (int)gram_chunks(H, N);
  const int rows_per = (N + nch - 1) / nch;
  dim3 g1(nch, H);
  if (D == 128) {
    if (dtype == PARK_BF16)
      PARK_LAUNCH("gram_partial", (k_gram_partial<bf16_t, 128>), g1, dim3(256), 0, st,
                  (const bf16_t*)Q, N, rows_per, part);
    else
      PARK_LAUNCH("gram_partial", (k_gram_partial<float, 128>), g1, dim3(256), 0, st,
                  (const float*)Q, N, rows_per, part);
  } else {
    if (dtype == PARK_BF16)
      PARK_LAUNCH("gram_partial", (k_gram_partial<bf16_t, 64>), g1, dim3(256), 0, st,
                  (const bf16_t*)Q, N, rows_per, part);
    else
      PARK_LAUNCH("gram_partial", (k_gram_partial<float, 64>), g1, dim3(256), 0, st,
                  (const float*)Q, N, rows_per, part);
  }
  const int DD = D * D;
  PARK_LAUNCH("gram_reduce", k_gram_reduce, dim3((DD + 255) / 256, H), dim3(256), 0, st, part, nch,
              DD, 1.0 / (double)N, G);
  const size_t lds = (size_t)DD * sizeof(double);
  if (D == 128) {
    // set once, outside any stream capture that may follow
    static const hipError_t attr = hipFuncSetAttribute(
        (const void*)k_metric_chol<128>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (attr != hipSuccess) return fail(PARK_ERR_HIP, "metric: cannot reserve %zu bytes of LDS", lds);
    PARK_LAUNCH("metric_chol", k_metric_chol<128>, dim3(H), dim3(256), lds, st, G, alpha, eps,
                s_min, Gbar, R, status);
  } else {
    PARK_LAUNCH("metric_chol", k_metric_chol<64>, dim3(H), dim3(256), lds, st, G, alpha, eps,
                s_min, Gbar, R, status);
  }
  return PARK_OK;
}

park_status launch_transform(const void* X, const double* R, int H, int N, int D, int dtype,
                             float* Xt, hipStream_t st) {
  const int gx = N < 4096 ? N : 4096;
  dim3 g(gx, H);
  if (D == 128) {
    if (dtype == PARK_BF16)
      PARK_LAUNCH("transform", (k_transform<bf16_t, 128>), g, dim3(128), 0, st, (const bf16_t*)X,
                  R, N, Xt);
    else
      PARK_LAUNCH("transform", (k_transform<float, 128>), g, dim3(128), 0, st, (const float*)X, R,
                  N, Xt);
  } else {
    if (dtype == PARK_BF16)
      PARK_LAUNCH("transform", (k_transform<bf16_t, 64>), g, dim3(64), 0, st, (const bf16_t*)X, R,
                  N, Xt);
    else
      PARK_LAUNCH("transform", (k_transform<float, 64>), g, dim3(64), 0, st, (const float*)X, R,
                  N, Xt);
  }
  return PARK_OK;
}

}  // namespace park
