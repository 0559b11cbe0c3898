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

// Symmetrise, scale, stabilise and factorise; one workgroup per head.
// The 256 threads form a 16 x 16 grid; thread (ti, tj) holds the entries
// (ti + 16 r, tj + 16 c), r, c < D/16, of the matrix in registers for the
// whole right-looking Cholesky.  Step k reads column k from a double-buffered
// LDS vector, applies M[i][j] -= M[i][k] M[j][k] / M[k][k] to the trailing
// block, and the owners of column k+1 publish it: one barrier per column.
// Column j keeps its value from step j; L[i][j] = that / sqrt(M[j][j]).
template <int D>
__global__ __launch_bounds__(256) void k_metric_chol(const double* __restrict__ G, double alpha,
                                                     double eps, double s_min,
                                                     double* __restrict__ Gbar_out,
                                                     double* __restrict__ R_out, int* status) {
  static_assert(D % 16 == 0 && D <= 128, "16 x 16 thread grid");
  constexpr int NB = D / 16;
  __shared__ double col[2][D];
  __shared__ double pv[D];
  __shared__ double sc;
  __shared__ int bad;
  const int h = blockIdx.x, tid = threadIdx.x;
  const int ti = tid >> 4, tj = tid & 15;
  const double* Gh = G + (size_t)h * D * D;
  if (tid == 0) bad = 0;
  if (tid < D) pv[tid] = Gh[tid * D + tid];
  double a[NB][NB];
  // symmetrise: (G + G^T) / 2
#pragma unroll
  for (int r = 0; r < NB; ++r)
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      const int i = ti + 16 * r, j = tj + 16 * c;
      a[r][c] = (i == j) ? Gh[i * D + j] : (Gh[i * D + j] + Gh[j * D + i]) / 2.0;
    }
  __syncthreads();
  // s = max(tr G / d, s_min), summed in index order
  if (tid == 0) {
    double t = 0.0;
    for (int i = 0; i < D; ++i) t += pv[i];
    sc = fmax(t / (double)D, s_min);
  }
  __syncthreads();
  const double s = sc;
  const double as = alpha * s, es = eps * s;
  double* Gb = Gbar_out + (size_t)h * D * D;
  bool nf = false;
#pragma unroll
  for (int r = 0; r < NB; ++r)
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      const int i = ti + 16 * r, j = tj + 16 * c;
      double v = (1.0 - alpha) * a[r][c];
      if (i == j) v = (v + as) + es;
      nf |= !isfinite(v);
      a[r][c] = v;
      Gb[i * D + j] = v;
    }
  if (nf) bad = 1;
  if (tj == 0)
#pragma unroll
    for (int r = 0; r < NB; ++r) col[0][ti + 16 * r] = a[r][0];
  __syncthreads();
#pragma unroll
  for (int kc = 0; kc < NB; ++kc) {
#pragma unroll 1
    for (int kt = 0; kt < 16; ++kt) {
      const int k = 16 * kc + kt, cur = k & 1;
      const double p = col[cur][k];
      if (tid == 0) {
        if (!(p > 0.0) || !isfinite(p)) bad = 1;
        pv[k] = sqrt(fmax(p, 0.0));
      }
      const double ip = 1.0 / p;
      double vi[NB], vj[NB];
#pragma unroll
      for (int r = kc; r < NB; ++r) {
        const int i = ti + 16 * r;
        vi[r] = (i > k) ? col[cur][i] * ip : 0.0;
      }
#pragma unroll
      for (int c = kc; c < NB; ++c) {
        const int j = tj + 16 * c;
        vj[c] = (j > k) ? col[cur][j] : 0.0;
      }
#pragma unroll
      for (int r = kc; r < NB; ++r)
#pragma unroll
        for (int c = kc; c < NB; ++c) a[r][c] = fma(-vi[r], vj[c], a[r][c]);
      // publish column k + 1 (rows from its own block on)
      if (kt < 15) {
        if (tj == kt + 1)
#pragma unroll
          for (int r = kc; r < NB; ++r) col[cur ^ 1][ti + 16 * r] = a[r][kc];
      } else if (kc + 1 < NB) {
        if (tj == 0)
#pragma unroll
          for (int r = kc + 1; r < NB; ++r) col[cur ^ 1][ti + 16 * r] = a[r][kc + 1];
      }
      __syncthreads();
    }
  }
  double* R = R_out + (size_t)h * D * D;
#pragma unroll
  for (int r = 0; r < NB; ++r)
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      const int i = ti + 16 * r, j = tj + 16 * c;
      R[i * D + j] = (j < i) ? a[r][c] / pv[j] : (j == i ? pv[j] : 0.0);
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
  if (D == 128)
    PARK_LAUNCH("metric_chol", k_metric_chol<128>, dim3(H), dim3(256), 0, st, G, alpha, eps,
                s_min, Gbar, R, status);
  else
    PARK_LAUNCH("metric_chol", k_metric_chol<64>, dim3(H), dim3(256), 0, st, G, alpha, eps,
                s_min, Gbar, R, status);
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
