// k-means of one side (Sec. 5.2, Alg. 3): seeded init, T x (assign, update),
// then the stable permutation.
//
// The QRKC side clusters x~ = R^T x under the Euclidean distance.  Because
// |R^T (x - mu)|^2 = (x - mu)^T Gbar (x - mu) (Eq. (11), App. D.2), the
// assignment only needs, per centroid mu_v kept in the input space,
//   w_v = Gbar mu_v  and  b_v = mu_v^T Gbar mu_v,
// since argmin_v |x~ - mu~_v|^2 = argmin_v (b_v - 2 x . w_v).  The Euclidean
// side uses w_v = mu_v.  Centroids are means of the input-space points, the
// image under R^T of the transformed-space means (linearity).
#include "common.h"
#include "kernels.h"

namespace park {

// ------------------------------------------------------------------ init
__device__ __forceinline__ uint64_t splitmix64_at(uint64_t seed, uint64_t i) {
  // output number i (0-based) of SplitMix64 seeded with `seed`
  uint64_t z = seed + (i + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// First C entries of the Fisher-Yates shuffle of 0..N-1 whose step i swaps
// positions i and j_i = i + (r_i mod (N - i)).  Evaluated in parallel: the
// value at position p before step i is the value that the last earlier step
// m with j_m = p moved there (the value position m held before step m), or p
// itself; these "last writer" links form a forest resolved by pointer jumping.
__global__ __launch_bounds__(1024) void k_init_idx(int N, int C, uint64_t seed, int side,
                                                   int* __restrict__ init) {
  __shared__ int jj[2048];
  __shared__ int root[2048];
  __shared__ int prevt[2048];
  const int h = blockIdx.x, tid = threadIdx.x;
  const uint64_t sh = seed ^ (0x9E3779B97F4A7C15ull * (uint64_t)(2 * h + side + 1));
  for (int i = tid; i < C; i += 1024)
    jj[i] = i + (int)(splitmix64_at(sh, (uint64_t)i) % (uint64_t)(N - i));
  __syncthreads();
  for (int k = tid; k < C; k += 1024) {
    int lw = k;  // last m < k with j_m == k (self if none)
    for (int m = k - 1; m >= 0; --m)
      if (jj[m] == k) {
        lw = m;
        break;
      }
    root[k] = lw;
    int pt = -1;  // last m < k with j_m == j_k
    const int jk = jj[k];
    if (jk != k)
      for (int m = k - 1; m >= 0; --m)
        if (jj[m] == jk) {
          pt = m;
          break;
        }
    prevt[k] = pt;
  }
  __syncthreads();
  // pointer jumping to the roots: value entering position k at step k
  for (int it = 0; (1 << it) < 2 * C; ++it) {
    int nv[2];
    for (int q = 0; q < 2; ++q) {
      const int k = tid + q * 1024;
      nv[q] = k < C ? root[root[k]] : 0;
    }
    __syncthreads();
    for (int q = 0; q < 2; ++q) {
      const int k = tid + q * 1024;
      if (k < C) root[k] = nv[q];
    }
    __syncthreads();
  }
  for (int i = tid; i < C; i += 1024) {
    const int j = jj[i];
    const int val = (j == i) ? root[i] : (prevt[i] >= 0 ? root[prevt[i]] : j);
    init[(size_t)h * C + i] = val;
  }
}

template <typename T>
__global__ void k_seed_centroids(const T* __restrict__ X, const int* __restrict__ init, int N, int D,
                                 int C, double* __restrict__ mu) {
  const int h = blockIdx.y, v = blockIdx.x, a = threadIdx.x;
  const int idx = init[(size_t)h * C + v];
  mu[((size_t)h * C + v) * D + a] = (double)to_f(X[((size_t)h * N + idx) * D + a]);
}

// w_v = Gbar mu_v (or mu_v), b_v = mu_v . w_v;  16 centroids per workgroup.
// Gbar is symmetric, so thread (a, group) reads column a of it coalesced and
// applies each element to 16 / (256 / D) centroids.
template <int D>
__global__ __launch_bounds__(256) void k_prep(const double* __restrict__ mu,
                                              const double* __restrict__ Gbar, int C,
                                              double* __restrict__ w, double* __restrict__ b) {
  constexpr int CB = 16, NG = 256 / D, PER = CB / NG;
  __shared__ double ms[CB][D];
  __shared__ double ws[CB][D + 1];
  const int h = blockIdx.y, v0 = blockIdx.x * CB, tid = threadIdx.x;
  for (int e = tid; e < CB * D; e += 256) {
    const int r = e / D, a = e % D;
    ms[r][a] = (v0 + r < C) ? mu[((size_t)h * C + v0 + r) * D + a] : 0.0;
  }
  __syncthreads();
  const int a = tid % D, grp = tid / D;
  double acc[PER];
  if (Gbar) {
    const double* G = Gbar + (size_t)h * D * D;
#pragma unroll
    for (int k = 0; k < PER; ++k) acc[k] = 0.0;
    for (int c = 0; c < D; ++c) {
      const double g = G[(size_t)c * D + a];
#pragma unroll
      for (int k = 0; k < PER; ++k) acc[k] = fma(g, ms[grp + NG * k][c], acc[k]);
    }
  } else {
#pragma unroll
    for (int k = 0; k < PER; ++k) acc[k] = ms[grp + NG * k][a];
  }
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int r = grp + NG * k;
    ws[r][a] = acc[k];
    if (v0 + r < C) w[((size_t)h * C + v0 + r) * D + a] = acc[k];
  }
  __syncthreads();
  if (tid < CB && v0 + tid < C) {
    double s = 0.0;
    for (int c = 0; c < D; ++c) s = fma(ms[tid][c], ws[tid][c], s);
    b[(size_t)h * C + v0 + tid] = s;
  }
}

// Exact float64 assignment: labels[j] = argmin_v (b_v - 2 x_j . w_v), ties to
// the lowest v.  64 tokens x 64 centroids per step, 4x4 per thread.
template <typename T, int D>
__global__ __launch_bounds__(256) void k_assign64(const T* __restrict__ X, const double* __restrict__ w,
                                                  const double* __restrict__ b, int N, int C,
                                                  int* __restrict__ labels, int* status) {
  constexpr int TM = 64, TC = 64, DC = 32;
  __shared__ float xs[TM][D + 1];
  __shared__ double wsm[TC][DC + 1];
  __shared__ double bs[TC];
  __shared__ double rs[16][TM];
  __shared__ int ri[16][TM];
  const int h = blockIdx.y, t0 = blockIdx.x * TM, tid = threadIdx.x;
  const T* Xh = X + (size_t)h * N * D;
  for (int e = tid; e < TM * D; e += 256) {
    const int r = e / D, c = e % D;
    xs[r][c] = (t0 + r < N) ? to_f(Xh[(size_t)(t0 + r) * D + c]) : 0.0f;
  }
  const int tg = tid & 15, cg = tid >> 4;
  double best[4];
  int bidx[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    best[i] = INFINITY;
    bidx[i] = 0x7fffffff;
  }
  const double* wh = w + (size_t)h * C * D;
  for (int c0 = 0; c0 < C; c0 += TC) {
    double acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
    for (int a0 = 0; a0 < D; a0 += DC) {
      __syncthreads();
      for (int e = tid; e < TC * DC; e += 256) {
        const int r = e / DC, c = e % DC;
        wsm[r][c] = (c0 + r < C) ? wh[(size_t)(c0 + r) * D + a0 + c] : 0.0;
      }
      if (a0 == 0 && tid < TC) bs[tid] = (c0 + tid < C) ? b[(size_t)h * C + c0 + tid] : 0.0;
      __syncthreads();
#pragma unroll 4
      for (int a = 0; a < DC; ++a) {
        double xv[4], wv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) xv[i] = (double)xs[tg + 16 * i][a0 + a];
#pragma unroll
        for (int j = 0; j < 4; ++j) wv[j] = wsm[cg + 16 * j][a];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = fma(xv[i], wv[j], acc[i][j]);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int v = c0 + cg + 16 * j;
      if (v < C) {
        const double bv = bs[cg + 16 * j];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const double s = fma(-2.0, acc[i][j], bv);
          if (s < best[i] || (s == best[i] && v < bidx[i])) {
            best[i] = s;
            bidx[i] = v;
          }
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    rs[cg][tg + 16 * i] = best[i];
    ri[cg][tg + 16 * i] = bidx[i];
  }
  __syncthreads();
  if (tid < TM && t0 + tid < N) {
    double bb = rs[0][tid];
    int bi = ri[0][tid];
    for (int g = 1; g < 16; ++g) {
      const double s = rs[g][tid];
      const int v = ri[g][tid];
      if (s < bb || (s == bb && v < bi)) {
        bb = s;
        bi = v;
      }
    }
    if (!isfinite(bb) || bi >= C) {
      raise_status(status, ST_NONFINITE);
      bi = 0;
    }
    labels[(size_t)h * N + t0 + tid] = bi;
  }
}

// Segmented mean over permuted rows: block v of head h averages
// X[perm[i]] (X[i] when perm is null) for offsets[v] <= i < offsets[v+1],
// summing in float64 in increasing position order.  Empty blocks keep mu64
// and give c32 = 0.
template <typename T>
__global__ void k_segment_mean(const T* __restrict__ X, const int* __restrict__ perm,
                               const int* __restrict__ offsets, int N, int D, int C,
                               double* __restrict__ mu64, float* __restrict__ c32,
                               int* __restrict__ sizes) {
  const int h = blockIdx.y, v = blockIdx.x, a = threadIdx.x;
  const int* off = offsets + (size_t)h * (C + 1);
  const int o0 = min(max(off[v], 0), N), o1 = min(max(off[v + 1], o0), N);
  const int n = o1 - o0;
  if (sizes && a == 0) sizes[(size_t)h * C + v] = n;
  const size_t dst = ((size_t)h * C + v) * D + a;
  if (n <= 0) {
    if (c32) c32[dst] = 0.0f;
    return;
  }
  const int* p = perm ? perm + (size_t)h * N : nullptr;
  const T* Xh = X + (size_t)h * N * D;
  double s = 0.0;
  for (int r = o0; r < o1; ++r) {
    const int idx = p ? p[r] : r;
    if ((unsigned)idx < (unsigned)N) s += (double)to_f(Xh[(size_t)idx * D + a]);
  }
  const double m = s / (double)n;
  if (mu64) mu64[dst] = m;
  if (c32) c32[dst] = (float)m;
}

// ---------------------------------------------------------------- launchers
park_status launch_segment_mean(const void* X, const int* perm, const int* offsets, int H, int N,
                                int D, int dtype, int C, double* mu64, float* c32, int* sizes,
                                hipStream_t st) {
  dim3 g(C, H);
  if (dtype == PARK_BF16)
    PARK_LAUNCH("segment_mean", k_segment_mean<bf16_t>, g, dim3(D), 0, st, (const bf16_t*)X, perm,
                offsets, N, D, C, mu64, c32, sizes);
  else
    PARK_LAUNCH("segment_mean", k_segment_mean<float>, g, dim3(D), 0, st, (const float*)X, perm,
                offsets, N, D, C, mu64, c32, sizes);
  return PARK_OK;
}

template <typename T, int D>
static park_status kmeans_impl(const T* X, const double* Gbar, int H, int N, int C, int T_,
                               uint64_t seed, int side, const KmeansBufs& kb, int* status,
                               hipStream_t st) {
  PARK_LAUNCH("kmeans_init", k_init_idx, dim3(H), dim3(1024), 0, st, N, C, seed, side, kb.init);
  PARK_LAUNCH("kmeans_seed", k_seed_centroids<T>, dim3(C, H), dim3(D), 0, st, X,
              (const int*)kb.init, N, D, C, kb.mu);
  for (int t = 0; t < T_; ++t) {
    PARK_LAUNCH("kmeans_prep", k_prep<D>, dim3((C + 15) / 16, H), dim3(256), 0, st,
                (const double*)kb.mu, Gbar, C, kb.w, kb.b);
    PARK_LAUNCH("kmeans_assign64", (k_assign64<T, D>), dim3((N + 63) / 64, H), dim3(256), 0, st, X,
                (const double*)kb.w, (const double*)kb.b, N, C, kb.labels, status);
    if (t + 1 < T_) {
      PARK_TRY(launch_count_sort(kb.labels, H, N, C, kb.thist, kb.perm, kb.offsets, st));
      PARK_LAUNCH("segment_mean", k_segment_mean<T>, dim3(C, H), dim3(D), 0, st, X,
                  (const int*)kb.perm, (const int*)kb.offsets, N, D, C, kb.mu, (float*)nullptr,
                  (int*)nullptr);
    }
  }
  return launch_count_sort(kb.labels, H, N, C, kb.thist, kb.perm, kb.offsets, st);
}

park_status launch_kmeans(const void* X, const double* Gbar, int H, int N, int D, int dtype, int C,
                          int T, uint64_t seed, int side, const KmeansBufs& kb, hipStream_t st) {
  int* status = kb.status;
  if (D == 128) {
    if (dtype == PARK_BF16)
      return kmeans_impl<bf16_t, 128>((const bf16_t*)X, Gbar, H, N, C, T, seed, side, kb, status, st);
    return kmeans_impl<float, 128>((const float*)X, Gbar, H, N, C, T, seed, side, kb, status, st);
  }
  if (dtype == PARK_BF16)
    return kmeans_impl<bf16_t, 64>((const bf16_t*)X, Gbar, H, N, C, T, seed, side, kb, status, st);
  return kmeans_impl<float, 64>((const float*)X, Gbar, H, N, C, T, seed, side, kb, status, st);
}

}  // namespace park
