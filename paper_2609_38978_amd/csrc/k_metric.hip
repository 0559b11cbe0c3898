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

// Partial Gram matrix of one row chunk, part[h][chunk] = sum_r x_r x_r^T, on
// fp64 MFMA (products of the bf16 / fp32
// inputs are exact in fp64, accumulation in fp64).  Lane l takes row
// r + l/16 of a 4-row step and the E = D/16 consecutive elements
// E c .. E c + E - 1 (c = l % 16) with one load; value e of the lane is then
// entry c of the 16-wide column block e, so the block product (a, b) is
// G[E m + a][E n + b] = sum_r x[r][E m + a] x[r][E n + b] (m, n < 16).  Of
// the E (E + 1) / 2 blocks with a <= b, wavefront w owns those with index
// p = w (mod 4); the lower triangle is written by transposition.  Register i
// of lane l holds output entry (l/16 + 4 i, l % 16).
typedef double gram_f64x4_t __attribute__((ext_vector_type(4)));

template <typename T, int D>
__global__ __launch_bounds__(256) void k_gram_mfma(const T* __restrict__ X, int N, int rows_per,
                                                   double* __restrict__ part) {
  constexpr int E = D / 16, NPAIR = E * (E + 1) / 2, PW = (NPAIR + 3) / 4;  // PW: pairs per wavefront
  const int h = blockIdx.y, ch = blockIdx.x, nch = gridDim.x;
  const int r0 = ch * rows_per, r1 = min(N, r0 + rows_per);
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l = threadIdx.x & 63, c = l & 15, rq = l >> 4;
  const T* Xh = X + (size_t)h * N * D;
  gram_f64x4_t acc[PW];
#pragma unroll
  for (int k = 0; k < PW; ++k) acc[k] = gram_f64x4_t{0.0, 0.0, 0.0, 0.0};
  auto load = [&](int r, double (&x)[E]) {
    if (r < r1) {
      if constexpr (sizeof(T) == 2) {
        const bf16_t* src = (const bf16_t*)Xh + (size_t)r * D + E * c;
        if constexpr (E == 8) {
          const uint4 u = *(const uint4*)src;
          const uint32_t wv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int e = 0; e < 8; ++e)
            x[e] = (double)__uint_as_float((e & 1) ? (wv[e >> 1] & 0xffff0000u) : (wv[e >> 1] << 16));
        } else {
          const uint2 u = *(const uint2*)src;
          const uint32_t wv[2] = {u.x, u.y};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            x[e] = (double)__uint_as_float((e & 1) ? (wv[e >> 1] & 0xffff0000u) : (wv[e >> 1] << 16));
        }
      } else {
        const float* src = (const float*)Xh + (size_t)r * D + E * c;
#pragma unroll
        for (int e = 0; e < E; e += 4) {
          const float4 f = *(const float4*)(src + e);
          x[e] = f.x;
          x[e + 1] = f.y;
          x[e + 2] = f.z;
          x[e + 3] = f.w;
        }
      }
    } else {
#pragma unroll
      for (int e = 0; e < E; ++e) x[e] = 0.0;
    }
  };
  double x[E], xn[E];
  load(r0 + rq, x);
  for (int rb = r0; rb < r1; rb += 4) {
    load(rb + 4 + rq, xn);  // next step in flight
    // block pair p = (a, b), a <= b, in row-major order of the upper triangle
#pragma unroll
    for (int a = 0, p = 0; a < E; ++a)
#pragma unroll
      for (int b = a; b < E; ++b, ++p)
        if ((p & 3) == w) acc[p >> 2] = __builtin_amdgcn_mfma_f64_16x16x4f64(x[a], x[b], acc[p >> 2], 0, 0, 0);
#pragma unroll
    for (int e = 0; e < E; ++e) x[e] = xn[e];
  }
  double* out = part + ((size_t)h * nch + ch) * D * D;
#pragma unroll
  for (int a = 0, p = 0; a < E; ++a)
#pragma unroll
    for (int b = a; b < E; ++b, ++p) {
      if ((p & 3) != w) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // lane (c, rq) register i holds entry (rq + 4 i, c) of the 16 x 16 block
        const int gi = E * (rq + 4 * i) + a, gj = E * c + b;
        out[(size_t)gi * D + gj] = acc[p >> 2][i];
        if (a != b) out[(size_t)gj * D + gi] = acc[p >> 2][i];
      }
    }
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

// Symmetrise, scale and stabilise (Eq. (11)):
//   Gbar = (1 - alpha) (G + G^T) / 2 + (alpha s + eps s) I,
//   s = max(tr G / d, s_min) (trace summed in index order);
// one workgroup per head.  A non-finite entry (non-finite queries) raises
// ST_NONFINITE.
template <int D>
__global__ __launch_bounds__(256) void k_metric_gbar(const double* __restrict__ G, double alpha,
                                                     double eps, double s_min,
                                                     double* __restrict__ Gbar_out, int* status) {
  __shared__ double pv[D];
  __shared__ double sc;
  __shared__ int bad;
  const int h = blockIdx.x, tid = threadIdx.x;
  const double* Gh = G + (size_t)h * D * D;
  if (tid == 0) bad = 0;
  if (tid < D) pv[tid] = Gh[tid * D + tid];
  __syncthreads();
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
  for (int e = tid; e < D * D; e += 256) {
    const int i = e / D, j = e - i * D;
    double v = (i == j) ? Gh[i * D + j] : (Gh[i * D + j] + Gh[j * D + i]) / 2.0;
    v = (1.0 - alpha) * v;
    if (i == j) v = (v + as) + es;
    nf |= !isfinite(v);
    Gb[e] = v;
  }
  if (nf) bad = 1;
  __syncthreads();
  if (tid == 0 && bad) raise_status(status, ST_NONFINITE);
}

// Cholesky factor of Gbar = L L^T (R = L; x~ = R^T x); one workgroup per
// head.  The 256 threads form a 16 x 16 grid; thread (ti, tj) holds the
// entries (ti + 16 r, tj + 16 c), r, c < D/16, of the matrix in registers for
// the whole right-looking Cholesky.  Step k reads column k from a
// double-buffered LDS vector, applies M[i][j] -= M[i][k] M[j][k] / M[k][k] to
// the trailing block, and the owners of column k+1 publish it: one barrier
// per column.  Column j keeps its value from step j; L[i][j] = that /
// sqrt(M[j][j]).  A pivot that is not positive raises ST_NOT_SPD.
template <int D>
__global__ __launch_bounds__(256) void k_metric_chol(const double* __restrict__ Gbar,
                                                     double* __restrict__ R_out, int* status) {
  static_assert(D % 16 == 0 && D <= 128, "16 x 16 thread grid");
  constexpr int NB = D / 16;
  __shared__ double col[2][D];
  __shared__ double pv[D];
  __shared__ int bad;
  const int h = blockIdx.x, tid = threadIdx.x;
  const int ti = tid >> 4, tj = tid & 15;
  const double* Gb = Gbar + (size_t)h * D * D;
  if (tid == 0) bad = 0;
  double a[NB][NB];
#pragma unroll
  for (int r = 0; r < NB; ++r)
#pragma unroll
    for (int c = 0; c < NB; ++c) a[r][c] = Gb[(ti + 16 * r) * D + tj + 16 * c];
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
                          double s_min, double* part, double* G, double* Gbar, int* status,
                          hipStream_t st) {
  const int nch = (int)gram_chunks(H, N);
  const int rows_per = (N + nch - 1) / nch;
  dim3 g1(nch, H);
  if (D == 128) {
    if (dtype == PARK_BF16)
      PARK_LAUNCH("gram_partial", (k_gram_mfma<bf16_t, 128>), g1, dim3(256), 0, st,
                  (const bf16_t*)Q, N, rows_per, part);
    else
      PARK_LAUNCH("gram_partial", (k_gram_mfma<float, 128>), g1, dim3(256), 0, st,
                  (const float*)Q, N, rows_per, part);
  } else {
    if (dtype == PARK_BF16)
      PARK_LAUNCH("gram_partial", (k_gram_mfma<bf16_t, 64>), g1, dim3(256), 0, st,
                  (const bf16_t*)Q, N, rows_per, part);
    else
      PARK_LAUNCH("gram_partial", (k_gram_mfma<float, 64>), g1, dim3(256), 0, st,
                  (const float*)Q, N, rows_per, part);
  }
  const int DD = D * D;
  PARK_LAUNCH("gram_reduce", k_gram_reduce, dim3((DD + 255) / 256, H), dim3(256), 0, st, part, nch,
              DD, 1.0 / (double)N, G);
  if (D == 128)
    PARK_LAUNCH("metric_gbar", k_metric_gbar<128>, dim3(H), dim3(256), 0, st, G, alpha, eps,
                s_min, Gbar, status);
  else
    PARK_LAUNCH("metric_gbar", k_metric_gbar<64>, dim3(H), dim3(256), 0, st, G, alpha, eps,
                s_min, Gbar, status);
  return PARK_OK;
}

park_status launch_metric_factor(const double* Gbar, int H, int D, double* R, int* status,
                                 hipStream_t st) {
  if (D == 128)
    PARK_LAUNCH("metric_chol", k_metric_chol<128>, dim3(H), dim3(256), 0, st, Gbar, R, status);
  else
    PARK_LAUNCH("metric_chol", k_metric_chol<64>, dim3(H), dim3(256), 0, st, Gbar, R, status);
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
