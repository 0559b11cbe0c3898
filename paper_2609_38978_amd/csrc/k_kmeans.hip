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
#include <stdlib.h>

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
  __shared__ unsigned long long key[2048];
  const int h = blockIdx.x, tid = threadIdx.x;
  const uint64_t sh = seed ^ (0x9E3779B97F4A7C15ull * (uint64_t)(2 * h + side + 1));
  int SZ = 2;  // power of two the sort below runs over
  while (SZ < C) SZ <<= 1;
  for (int i = tid; i < SZ; i += 1024) {
    if (i < C) {
      const int j = i + (int)(splitmix64_at(sh, (uint64_t)i) % (uint64_t)(N - i));
      jj[i] = j;
      key[i] = ((unsigned long long)j << 11) | (unsigned)i;
      root[i] = -1;
    } else {
      key[i] = ~0ull;
    }
  }
  __syncthreads();
  // root[k] = the last step m < k with j_m = k (j_m >= m, so every m with
  // j_m = k != m qualifies), else k
  for (int m = tid; m < C; m += 1024) {
    const int t = jj[m];
    if (t < C && t != m) atomicMax(&root[t], m);
  }
  // prevt[k] = the last step m < k with j_m = j_k: the predecessor of (j_k, k)
  // in the sorted list of pairs (j, step)
  for (int len = 2; len <= SZ; len <<= 1)
    for (int j = len >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < SZ; i += 1024) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const unsigned long long x = key[i], y = key[ixj];
          const bool up = (i & len) == 0;
          if ((x > y) == up) {
            key[i] = y;
            key[ixj] = x;
          }
        }
      }
      __syncthreads();
    }
  for (int s = tid; s < C; s += 1024) {
    const unsigned long long x = key[s];
    const int k = (int)(x & 2047ull);
    const bool same = s > 0 && (key[s - 1] >> 11) == (x >> 11);
    prevt[k] = (same && jj[k] != k) ? (int)(key[s - 1] & 2047ull) : -1;
    if (root[k] < 0) root[k] = k;
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

// plain float64 copy (warm-start centroids in, final means out)
__global__ __launch_bounds__(256) void k_copy64(const double* __restrict__ src,
                                                double* __restrict__ dst, long n) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i < n) dst[i] = src[i];
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
// applies each element to 16 / (256 / D) centroids.  When `w3` is given the
// fast-path operands are written too: w_v split into three bf16 parts (three
// planes of H*C*D), b_v in float, |w_v| rounded up and the |b_v| term of the
// error bound (see k_assign_fast); `m2`/`mn` give the candidate filter the
// centroids in two bf16 parts and |mu_v|.
//
// Cluster radii for the candidate filter (rmode 2): the previous assignment
// left in dmax[a] an upper bound of max D(x, mu_a^old)^2 over the tokens it
// labelled a, and by the triangle inequality every such token has
// D(x, mu_a) <= sqrt(dmax[a]) + D(mu_a^old, mu_a).  The move is
// D(mu_old, mu)^2 = b - 2 mu . w_old + b_old (w_old, b_old: this buffer's
// values before the update), rounded up by a margin of 1e-9 of the
// magnitudes involved; r2[a] = (sqrt(dmax) + move)^2, rounded up, or -1 for
// a cluster the sort left empty.  rmode >= 1 then clears dmax for the
// coming assignment.
template <int D, int NT>
__global__ __launch_bounds__(NT) void k_prep(const double* __restrict__ mu,
                                              const double* __restrict__ Gbar, int C,
                                              double* __restrict__ w, double* __restrict__ b,
                                              bf16_t* __restrict__ w3,
                                              size_t plane, float* __restrict__ b32, int Cpad,
                                              float* __restrict__ wn, float* __restrict__ eb,
                                              float* __restrict__ bmax, bf16_t* __restrict__ m2,
                                              float* __restrict__ mn,
                                              const int* __restrict__ offsets,
                                              double* __restrict__ r2,
                                              unsigned long long* __restrict__ dmax, int rmode) {
  // NT threads: D lanes per centroid group, 16 / (NT / D) centroids per
  // thread.  1024 threads shorten each thread's float64 chain over the D
  // columns (small grids); 256 read the metric rows fewer times (large grids)
  constexpr int CB = 16, NG = NT / D, PER = CB / NG;
  static_assert(PER >= 1 && CB % NG == 0, "centroid groups");
  __shared__ double ms[CB][D];
  __shared__ double ws[CB][D + 1];
  __shared__ float fnl[CB], fel[CB];
  const int h = blockIdx.y, v0 = blockIdx.x * CB, tid = threadIdx.x;
  for (int e = tid; e < CB * D; e += NT) {
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
    // sixteen metric rows' loads issued together, then their products (the
    // same fma order over the columns)
    for (int c0 = 0; c0 < D; c0 += 16) {
      double g[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) g[j] = G[(size_t)(c0 + j) * D + a];
#pragma unroll
      for (int j = 0; j < 16; ++j)
#pragma unroll
        for (int k = 0; k < PER; ++k) acc[k] = fma(g[j], ms[grp + NG * k][c0 + j], acc[k]);
    }
  } else {
#pragma unroll
    for (int k = 0; k < PER; ++k) acc[k] = ms[grp + NG * k][a];
  }
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int r = grp + NG * k;
    ws[r][a] = acc[k];
    if (v0 + r < C) {
      const size_t o = ((size_t)h * C + v0 + r) * D + a;
      // (w itself is written at the end: the radius bound reads the old w)
      if (w3) {
        // w = w1 + w2 + w3 + r with bf16 parts and |r| <= 2^-24 |w| (1 + 2^-7)
        const bf16_t p1 = f2bf((float)acc[k]);
        const double r1 = acc[k] - (double)bf2f(p1);
        const bf16_t p2 = f2bf((float)r1);
        const double r2 = r1 - (double)bf2f(p2);
        w3[o] = p1;
        w3[o + plane] = p2;
        w3[o + 2 * plane] = f2bf((float)r2);
      }
      if (m2) {  // the centroid itself in two bf16 parts (candidate filter)
        const double mv = ms[r][a];
        const bf16_t q1 = f2bf((float)mv);
        m2[o] = q1;
        m2[o + plane] = f2bf((float)(mv - (double)bf2f(q1)));
      }
    }
  }
  __syncthreads();
  // b_v and |w_v|^2: 16 lanes per centroid (the first four wavefronts),
  // partial sums added in a fixed tree
  if (tid < 256) {
    constexpr int LPC = 256 / CB;
    const int r = tid / LPC, sub = tid % LPC;
    double s = 0.0, n2 = 0.0, m2s = 0.0, dso = 0.0, dsa = 0.0;
    const double* wold = w + ((size_t)h * C + min(v0 + r, C - 1)) * D;
    double wo[D / LPC];  // the old w of this lane's columns, loaded together
#pragma unroll
    for (int j = 0; j < D / LPC; ++j) wo[j] = rmode == 2 ? wold[sub + LPC * j] : 0.0;
#pragma unroll
    for (int j = 0; j < D / LPC; ++j) {
      const int c = sub + LPC * j;
      s = fma(ms[r][c], ws[r][c], s);
      n2 = fma(ws[r][c], ws[r][c], n2);
      m2s = fma(ms[r][c], ms[r][c], m2s);
      if (rmode == 2) {
        dso = fma(ms[r][c], wo[j], dso);
        dsa += fabs(ms[r][c] * wo[j]);
      }
    }
#pragma unroll
    for (int o = LPC / 2; o > 0; o >>= 1) {
      s += __shfl_xor(s, o, 64);
      n2 += __shfl_xor(n2, o, 64);
      m2s += __shfl_xor(m2s, o, 64);
      if (rmode == 2) {
        dso += __shfl_xor(dso, o, 64);
        dsa += __shfl_xor(dsa, o, 64);
      }
    }
    if (rmode >= 1 && sub == 0 && v0 + r < C) {
      const size_t cidx = (size_t)h * C + v0 + r;
      if (rmode == 2) {
        const int* off = offsets + (size_t)h * (C + 1);
        const int n = off[v0 + r + 1] - off[v0 + r];
        double rr = -1.0;
        if (n > 0) {
          const double bo = b[cidx];  // b before the update (this thread writes it below)
          const double mv2 = s - 2.0 * dso + bo + 1e-9 * (fabs(s) + fabs(bo) + 2.0 * dsa);
          const double mv = sqrt(fmax(mv2, 0.0)) * (1.0 + 1e-12);
          const double dm = fmax(__longlong_as_double((long long)dmax[cidx]), 0.0);
          const double R = sqrt(dm) * (1.0 + 1e-12) + mv;
          rr = R * R * (1.0 + 1e-12);
        }
        r2[cidx] = rr;
      }
      dmax[cidx] = 0ull;
    }
    if (mn && sub == 0 && v0 + r < C) mn[(size_t)h * C + v0 + r] = (float)(sqrt(m2s) * (1.0 + 1e-6));
    float fnr = 0.0f, fer = 0.0f;
    if (sub == 0 && v0 + r < C) {
      b[(size_t)h * C + v0 + r] = s;
      if (b32) {
        fnr = (float)(sqrt(n2) * (1.0 + 1e-6));
        fer = (float)(fabs(s) * (2.0 * 1.1 * 5.9604644775390625e-08) * (1.0 + 1e-6));
        b32[(size_t)h * Cpad + v0 + r] = (float)s;
        wn[(size_t)h * Cpad + v0 + r] = fnr;
        eb[(size_t)h * Cpad + v0 + r] = fer;
      }
    }
    if (sub == 0) {
      fnl[r] = fnr;
      fel[r] = fer;
    }
  }
  __syncthreads();
  // w itself (the reduction above has read the old values)
  for (int e = tid; e < CB * D; e += NT) {
    const int r = e / D, a = e % D;
    if (v0 + r < C) w[((size_t)h * C + v0 + r) * D + a] = ws[r][a];
  }
  float fn = tid < CB ? fnl[tid] : 0.0f, fe = tid < CB ? fel[tid] : 0.0f;
  if (b32 && blockIdx.x == gridDim.x - 1)  // padding centroids: score +inf, no error term
    for (int v = C + tid; v < Cpad; v += NT) {
      b32[(size_t)h * Cpad + v] = INFINITY;
      wn[(size_t)h * Cpad + v] = 0.0f;
      eb[(size_t)h * Cpad + v] = 0.0f;
    }
  if (b32 && tid < 64) {
    // this block's maxima of |w_v| and eb_v (reduced by the assignment)
    for (int o = 8; o > 0; o >>= 1) {
      fn = fmaxf(fn, __shfl_xor(fn, o, 64));
      fe = fmaxf(fe, __shfl_xor(fe, o, 64));
    }
    if (tid == 0) {
      bmax[((size_t)h * gridDim.x + blockIdx.x) * 2] = fn;
      bmax[((size_t)h * gridDim.x + blockIdx.x) * 2 + 1] = fe;
    }
  }
}

// ---------------------------------------------------------------------------
// Fast assignment on bf16 MFMA with certification.
//
// For a bf16 point x the score s_v = b_v - 2 x.w_v is evaluated with w_v
// split into NP bf16 parts, w = w1 + w2 (+ w3) + r, with |r| <= 2^-16 (1.01)
// |w| for two parts and 2^-24 (1 + 2^-7)|w| for three.  All products are
// bf16 x bf16, exact in float.  With delta = 2^-23 per addition inside an
// MFMA (any faithful rounding) and 2^-24 for a VALU rounding, the forward
// error of t^ = x.w is at most
//   et sum_a |x_a w_a|,  et = er 1.01 + (D+1) delta (1 + 2^-7)
//                            + 2^-8 1.01 ((NP-1) D + 1) delta + 2^-24 1.01,
// er the residual bound above.  This covers two orders of evaluation: x.w1
// and the smaller parts (terms 2^-8 smaller) in two chains of
// v_mfma_f32_32x32x16_bf16 added once, and (the fast path) the smaller parts'
// chain continued by the D products of x.w1, whose partial sums are then at
// most (1 + 2^-8 1.01)(1 + 2^-7) sum_a |x_a w_a|, i.e. D delta (1.012) in
// place of (D+1) delta (1 + 2^-7) + 2^-24 1.01.  Two parts take 2/3 of the MFMA work and
// double the bound; they pay off when the centroid count makes the pass
// MFMA-bound (C >= 512), three parts otherwise.
// and with sum_a |x_a w_a| <= |x| |w_v|, the float roundings of b_v and of
// the score, and |s^_v| <= |b_v| + 2.01 |x| |w_v|:
//   |s^_v - s_v| <= E_v = Kx |w_v| + eb_v,
//   Kx = 1.1 (2 et + 2.01 2^-24) |x|,  eb_v = 1.1 * 2 * 2^-24 |b_v|
// (the factor 1.1 covers the rounding of |x| and of the bound itself).
//
// Certification: with v1 the fast argmin and L the smallest fast score of
// every other centroid, v1 is the exact argmin when
//   L - Emax > s^_v1 + E_v1,   Emax = Kx max_v |w_v| + max_v eb_v >= E_v.
// Otherwise (near-ties, exact ties) the token is listed for the float64
// refinement.
//
// Bookkeeping per lane and token (the lane sees half of the centroids): the
// two smallest fast scores (best <= L) and the id of the smallest, three VALU
// operations per score: best = min(best, s), L = med3(best, L, s), and the
// id taken when s < best, so ties keep the lower id and an equal score later
// in the sweep lands in L (exact ties are never certified).
//
// Workgroup = kmeans_tile tokens (4 wavefronts x TB blocks of 32).  Centroid tiles of
// 32 rows of the NP parts go from HBM to an NS-slot LDS ring by LDS DMA (rows
// swizzled in 16-byte chunks, see the reads), later tiles in flight while
// this one is scored.  MFMA orientation (32x32x16, the shape with twice the
// throughput of 16x16x32 here): A = 32 centroids x 16 dims, B = 16 dims x 32
// tokens, so lane l holds centroids 8b + 4(l/32) + r (b, r < 4) of token l%32.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// One wave-wide LDS DMA (lane l's 16 bytes at g land at LDS byte lds + 16 l),
// as inline assembly so that the compiler does not drain every DMA in flight
// before each LDS read; completion is waited for explicitly.
__device__ __forceinline__ void km_dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ uint32_t km_lds_addr(const void* p) {
  return (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)p;
}
template <int D>
__device__ __forceinline__ int km_swz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
// waits until at most N vector-memory operations of this wavefront are outstanding
template <int N>
__device__ __forceinline__ void km_wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
#ifndef PARK_KM_NS
#define PARK_KM_NS 3
#endif

template <int D, int NP>
__global__ __launch_bounds__(256, 2) void k_assign_fast(const bf16_t* __restrict__ X,
                                                     const bf16_t* __restrict__ w3, size_t plane,
                                                     const float* __restrict__ b32, int Cpad,
                                                     const float* __restrict__ wn,
                                                     const float* __restrict__ eb,
                                                     const float* __restrict__ bmax, int nbm,
                                                     int N, int C,
                                                     int* __restrict__ labels,
                                                     int* __restrict__ flags,
                                                     float* __restrict__ flagu,
                                                     int* __restrict__ nflag) {
  constexpr int TB = PARK_KM_TB, CT = 32, KS = D / 16, CPR = D / 8, RPI = 64 / CPR;
  constexpr int NI = NP * CT / (4 * RPI);  // DMAs per wavefront and tile
  static_assert(NI * 4 * RPI == NP * CT && (NP == 2 || NP == 3), "tile shape");
  static_assert(kmeans_tile == 128 * TB, "tile tokens");
  constexpr float U24 = 5.9604645e-08f, DEL = 1.1920929e-07f;
  // residual of the split: 2^-16 (two parts) or 2^-24 (three parts), relative
  constexpr float ER = NP == 2 ? 1.52587891e-05f : U24;
  constexpr float ET = ER * 1.01f + (D + 1) * DEL * 1.0079f +
                       0.00390625f * 1.01f * ((NP - 1) * D + 1) * DEL + U24 * 1.01f;
  constexpr float KXC = 1.1f * (2.0f * ET + 2.01f * U24) * 1.0001f;
  constexpr int NS = PARK_KM_NS;  // LDS ring slots: NS - 1 tiles in flight
  __shared__ __attribute__((aligned(16))) bf16_t Wt[NS][NP * CT * D];  // [slot][part][row][D]
  // b values by tile (tile % (NS + 1)): a tile's stay until its deferred ranking
  __shared__ __attribute__((aligned(16))) float Bt[NS + 1][CT];
  __shared__ float mx_s[2];
  __shared__ int wcnt[4];
  const int h = blockIdx.y, tid = threadIdx.x, l = tid & 63, hf = l >> 5, c32 = l & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int t0 = blockIdx.x * kmeans_tile + w * 32 * TB;
  const bf16_t* Xh = X + (size_t)h * N * D;
  const bf16_t* P1 = w3 + (size_t)h * C * D;
  const float* bh = b32 + (size_t)h * Cpad;
  // LDS DMA lanes: row of the tile's NP*CT part-rows, chunk pch
  const int pch = l % CPR;
  const int ntiles = (C + CT - 1) / CT;
  auto issue = [&](int tile, int slot) {
    const int c0 = tile * CT;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int row = (w * NI + i) * RPI + l / CPR;
      const int part = row / CT, r = row % CT;
      const int v = min(c0 + r, C - 1);
      const bf16_t* src = P1 + part * plane + (size_t)v * D + 8 * (pch ^ km_swz<D>(r));
      km_dma16(src, km_lds_addr(&Wt[slot][0] + (w * NI + i) * 512));
    }
    if (w == 0 && l < CT / 4) km_dma16(bh + c0 + 4 * l, km_lds_addr(&Bt[tile % (NS + 1)][0]));
  };
  // the first tiles travel while the points are loaded
#pragma unroll
  for (int p = 0; p < NS - 1; ++p)
    if (p < ntiles) issue(p, p);
  // B operand: lane l holds dims 16 s + 8 (l/32) .. + 8 of token t0 + 32 tb + l%32
  bf16x8_t xf[TB][KS];
  float xsq[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    xsq[tb] = 0.0f;
    const int tok = t0 + 32 * tb + c32;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      uint4 raw = make_uint4(0u, 0u, 0u, 0u);
      if (tok < N) raw = *(const uint4*)(Xh + (size_t)tok * D + 16 * s + 8 * hf);
      xf[tb][s] = __builtin_bit_cast(bf16x8_t, raw);
      const uint32_t q[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bf16x2_t p2 = __builtin_bit_cast(bf16x2_t, q[e]);
        xsq[tb] = __builtin_amdgcn_fdot2_f32_bf16(p2, p2, xsq[tb], false);
      }
    }
  }
  if (tid < 64) {
    float a = 0.0f, c = 0.0f;
    for (int i = tid; i < nbm; i += 64) {
      a = fmaxf(a, bmax[((size_t)h * nbm + i) * 2]);
      c = fmaxf(c, bmax[((size_t)h * nbm + i) * 2 + 1]);
    }
    for (int o = 32; o > 0; o >>= 1) {
      a = fmaxf(a, __shfl_xor(a, o, 64));
      c = fmaxf(c, __shfl_xor(c, o, 64));
    }
    if (tid == 0) {
      mx_s[0] = a;
      mx_s[1] = c;
    }
  }
  float kx[TB], best[TB], L[TB];
  // id of the best centroid minus (first centroid of the current tile + 4 hf),
  // so that the per-score select takes a constant
  int brel[TB], bidx[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    const float xs = xsq[tb] + __shfl_xor(xsq[tb], 32, 64);
    // |x|^2 below 2^-100 may have lost its square terms to underflow: such a
    // token gets an infinite bound and is listed for the float64 path
    kx[tb] = xs >= 7.88860905e-31f ? KXC * sqrtf(xs) : INFINITY;
    best[tb] = INFINITY;
    L[tb] = INFINITY;
    brel[tb] = -(1 << 30);  // no centroid yet
  }
  // all global loads done before the tile loop (its waits are explicit)
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
#pragma unroll
    for (int s = 0; s < KS; ++s) asm volatile("" ::"v"(xf[tb][s]));
    asm volatile("" ::"v"(kx[tb]));
  }

  const int swk = km_swz<D>(c32);
  const int rowo = c32 * D;
  // tile t: its DMAs done, barrier, the next tile's DMAs issued; its scores
  // (-2 x.w without b) into a
  auto scores = [&](int t, f32x16_t (&a)[TB]) {
    // own DMAs of tile t done (wavefront 0 also fetches the b tile)
    if (NS > 2 && t + 1 < ntiles) {
      if (w == 0) km_wait_vmcnt<NI + 1>();
      else km_wait_vmcnt<NI>();
    } else {
      km_wait_vmcnt<0>();
    }
    __syncthreads();  // tile t landed; tile t-1 consumed by every wavefront
    if (t + NS - 1 < ntiles) issue(t + NS - 1, (t + NS - 1) % NS);
    const int slot = t % NS;
    const bf16_t* W1 = &Wt[slot][0];
    const bf16_t* W2 = W1 + CT * D;
    const bf16_t* W3 = W2 + CT * D;  // third part (NP == 3)
    // the small parts first, then the leading part on top of them (one
    // accumulator, no separate addition of the two sums)
#pragma unroll
    for (int tb = 0; tb < TB; ++tb)
#pragma unroll
      for (int q = 0; q < 16; ++q) a[tb][q] = 0.0f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int co = rowo + 8 * ((2 * s + hf) ^ swk);
      const bf16x8_t a2 = *(const bf16x8_t*)(W2 + co);
      bf16x8_t a3;
      if constexpr (NP == 3) a3 = *(const bf16x8_t*)(W3 + co);
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        a[tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, xf[tb][s], a[tb], 0, 0, 0);
        if constexpr (NP == 3)
          a[tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, xf[tb][s], a[tb], 0, 0, 0);
      }
    }
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int co = rowo + 8 * ((2 * s + hf) ^ swk);
      const bf16x8_t a1 = *(const bf16x8_t*)(W1 + co);
#pragma unroll
      for (int tb = 0; tb < TB; ++tb)
        a[tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, xf[tb][s], a[tb], 0, 0, 0);
    }
  };
  // ranking of tile t's scores, tiles in order
  auto rank = [&](const f32x16_t (&a)[TB], int t) {
    float bvt[16];
#pragma unroll
    for (int bq = 0; bq < 4; ++bq) {
      const float4 b4 = *(const float4*)(&Bt[t % (NS + 1)][8 * bq + 4 * hf]);
      bvt[4 * bq] = b4.x;
      bvt[4 * bq + 1] = b4.y;
      bvt[4 * bq + 2] = b4.z;
      bvt[4 * bq + 3] = b4.w;
    }
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const float sc = fmaf(-2.0f, a[tb][q], bvt[q]);
        const bool nb = sc < best[tb];
        L[tb] = __builtin_amdgcn_fmed3f(best[tb], L[tb], sc);
        best[tb] = fminf(best[tb], sc);
        brel[tb] = nb ? 8 * (q >> 2) + (q & 3) : brel[tb];
      }
      brel[tb] -= CT;  // relative to the next tile
      // done before the next step's wait (not sunk past it, where its
      // scores would have to outlive the next tile's)
      asm volatile("" ::"v"(best[tb]), "v"(L[tb]), "v"(brel[tb]));
    }
  };
  // software pipeline: the MFMAs of tile t and the ranking of tile t-1 in
  // the same step (two score sets, alternating), so that the VALU ranking
  // runs while the matrix unit works
  f32x16_t A0[TB], A1[TB];
  if (ntiles > 0) {
    scores(0, A0);
    int t = 1;
    for (; t + 1 < ntiles; t += 2) {
      scores(t, A1);
      rank(A0, t - 1);
      scores(t + 1, A0);
      rank(A1, t);
    }
    if (t < ntiles) {
      scores(t, A1);
      rank(A0, t - 1);
      rank(A1, t);
    } else {
      rank(A0, t - 1);
    }
  }
#pragma unroll
  for (int tb = 0; tb < TB; ++tb)
    bidx[tb] = brel[tb] >= -(1 << 29) ? brel[tb] + ntiles * CT + 4 * hf : -1;
  const float nmax = mx_s[0], ebmax = mx_s[1];
  bool fl[TB];
  float ubv[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    // merge the two halves holding this token (ties: lowest id)
    {
      const float ob = __shfl_xor(best[tb], 32, 64), oL = __shfl_xor(L[tb], 32, 64);
      const int oi = __shfl_xor(bidx[tb], 32, 64);
      const bool mine_valid = bidx[tb] >= 0, other_valid = oi >= 0;
      const bool take = other_valid && (!mine_valid || ob < best[tb] ||
                                        (ob == best[tb] && oi < bidx[tb]));
      const float loser = take ? (mine_valid ? best[tb] : INFINITY)
                               : (other_valid ? ob : INFINITY);
      L[tb] = fminf(fminf(L[tb], oL), loser);
      best[tb] = take ? ob : best[tb];
      bidx[tb] = take ? oi : bidx[tb];
    }
    const int tok = t0 + 32 * tb + c32;
    fl[tb] = false;
    ubv[tb] = INFINITY;  // an upper bound of the smallest exact score
    if (hf == 0 && tok < N) {
      bool ok = false;
      if (bidx[tb] >= 0 && isfinite(best[tb])) {
        const int v = bidx[tb];
        const float e1 = fmaf(kx[tb], wn[(size_t)h * Cpad + v], eb[(size_t)h * Cpad + v]);
        const float emax = fmaf(kx[tb], nmax, ebmax) * 1.0001f;
        ubv[tb] = best[tb] + e1;
        ok = (L[tb] - emax) > ubv[tb];
      }
      if (ok) labels[(size_t)h * N + tok] = bidx[tb];
      fl[tb] = !ok;
    }
  }
  // listed tokens: this tile's list at flags[h][kmeans_tile * tile ...] in lane
  // order, its length in nflag[h][tile]; no atomics
  uint64_t bal[TB];
  int tot = 0;
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    bal[tb] = __ballot(fl[tb]);
    tot += __popcll(bal[tb]);
  }
  if (l == 0) wcnt[w] = tot;
  __syncthreads();
  int base = blockIdx.x * kmeans_tile;
  for (int q = 0; q < w; ++q) base += wcnt[q];
  if (tid == 0) nflag[(size_t)h * gridDim.x + blockIdx.x] = wcnt[0] + wcnt[1] + wcnt[2] + wcnt[3];
  if (tot > 0) {
    const uint64_t below = (1ull << l) - 1ull;
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      if (fl[tb]) {
        const int slot = base + __popcll(bal[tb] & below);
        flags[(size_t)h * N + slot] = t0 + 32 * tb + c32;
        flagu[(size_t)h * N + slot] = ubv[tb];
      }
      base += __popcll(bal[tb]);
    }
  }
}

// Float64 assignment of the tokens the fast path could not certify.
//
// Every exact score lies in [s^_v - E_v, s^_v + E_v], here with fast scores on
// the three-part split (w = w1 + w2 + w3 + r, |r| <= 2^-24 (1+2^-7)|w|, error
// constant as in the fast path with the two small parts in the second chain),
// so with U the listed upper bound of the smallest exact score (from the fast
// path's own scores and bounds), the exact argmin lies in the candidate set
// {v : s^_v - E_v <= U}.  One sweep over the centroids (MFMA, as in the fast
// path, centroid tiles through an NS-slot LDS DMA ring) collects each token's
// candidates in LDS; they are then scored in float64 (b_v - 2 x.w_v, partial
// sums over PL lanes added in a fixed tree) and the minimum, ties to the
// lowest id, is the label.  Near-ties leave two or three candidates; a token
// with more than KMAX (exact duplicates, degenerate data) is scored against
// every centroid.
// Workgroups take chunks of 64 listed tokens (16 per wavefront), so that the
// sweep of one chunk is short and the listed tokens spread over many CUs.
template <int D>
__global__ __launch_bounds__(256) void k_refine_cand(const bf16_t* __restrict__ X,
                                                     const bf16_t* __restrict__ w3, size_t plane,
                                                     const float* __restrict__ b32,
                                                     const float* __restrict__ wn,
                                                     const float* __restrict__ eb, int Cpad,
                                                     const double* __restrict__ w64,
                                                     const double* __restrict__ b64, int H, int N,
                                                     int C, int rg,
                                                     const int* __restrict__ flags,
                                                     const float* __restrict__ flagu,
                                                     const int* __restrict__ nflag,
                                                     int* __restrict__ labels, int* status,
                                                     const double* __restrict__ xn,
                                                     unsigned long long* __restrict__ dmax) {
  constexpr int CT = 32, KS = D / 32, CPR = D / 8, RPI = 64 / CPR;
  constexpr int NI = 3 * CT / (4 * RPI);  // DMAs per wavefront and tile
  constexpr int NS = PARK_KM_NS;
  constexpr int TC = 64;                  // listed tokens per chunk
  constexpr int KMAX = 4;                 // candidates kept per token
  constexpr int PL = 16, PE = D / PL;     // lanes per scored pair, elements per lane
  constexpr int KP = 4;                   // pairs per lane group and pass
  constexpr float U24 = 5.9604645e-08f, DEL = 1.1920929e-07f;
  constexpr float ET = U24 * 1.01f + (D + 1) * DEL * 1.0079f + 0.00390625f * 1.01f * (2 * D + 1) * DEL +
                       U24 * 1.01f;
  constexpr float KXC = 1.1f * (2.0f * ET + 2.01f * U24) * 1.0001f;
  __shared__ __attribute__((aligned(16))) bf16_t Wt[NS][3 * CT * D];
  __shared__ __attribute__((aligned(16))) float Bt[NS][CT];
  __shared__ __attribute__((aligned(16))) float Nt[NS][CT];
  __shared__ __attribute__((aligned(16))) float Et[NS][CT];
  __shared__ int ccount[TC];
  __shared__ int ctok[TC];
  __shared__ int cv[TC * KMAX];  // candidates by token slot
  __shared__ int poff[TC];
  __shared__ int npairs;
  __shared__ int nover;
  __shared__ int over[TC];
  __shared__ double rbest[4];
  __shared__ int ridx[4];
  __shared__ int wsc[4];
  __shared__ int spos[TC];  // list position of each slot of the chunk (-1: none)
  __shared__ float cx2[TC];  // |x|^2 of each slot's token
  // after the sweep the ring holds the pair lists and float64 scores
  double* const cs = (double*)&Wt[0][0];  // [TC * KMAX] scores of the packed pairs
  int* const ptl = (int*)(cs + TC * KMAX);  // [TC * KMAX] token slot of each pair
  int* const pv = ptl + TC * KMAX;          // [TC * KMAX] centroid of each pair
  double* const xrow = (double*)(pv + TC * KMAX);  // [D]
  double* const obest = xrow + D;                  // [TC]
  int* const oidx = (int*)(obest + TC);            // [TC]
  static_assert((3 * TC * KMAX + 2 * D + 3 * TC) * 8 <= (int)sizeof(Wt), "aliases fit the ring");
  // XCD-aware: the workgroups of a head run on one XCD (its L2 holds the head's centroids)
  const int nitems = H * rg, per = (nitems + 7) >> 3;
  const int item = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (item >= nitems) return;
  const int h = item / rg, wg = item - h * rg;
  const int tid = threadIdx.x, l = tid & 63, g = l >> 4, c16 = l & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  // listed tokens of head h: per-tile lists of the fast pass
  const int NT = (N + kmeans_tile - 1) / kmeans_tile;
  const int* nf = nflag + (size_t)h * NT;
  int cnt = 0;
  for (int t = tid; t < NT; t += 256) cnt += min(max(nf[t], 0), kmeans_tile);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
  if (l == 0) wsc[w] = cnt;
  __syncthreads();
  cnt = wsc[0] + wsc[1] + wsc[2] + wsc[3];
  const int nchunks = (cnt + TC - 1) / TC;
  if (wg >= nchunks) return;
  const bf16_t* Xh = X + (size_t)h * N * D;
  const bf16_t* P1 = w3 + (size_t)h * C * D;
  const float* bh = b32 + (size_t)h * Cpad;
  const float* nh = wn + (size_t)h * Cpad;
  const float* eh = eb + (size_t)h * Cpad;
  const double* wh = w64 + (size_t)h * C * D;
  const double* b64h = b64 + (size_t)h * C;
  const int pch = l % CPR;
  const int nt = (C + CT - 1) / CT;
  auto issue = [&](int tile, int slot) {
    const int c0 = tile * CT;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int row = (w * NI + i) * RPI + l / CPR;
      const int part = row / CT, r = row % CT;
      const int v = min(c0 + r, C - 1);
      const bf16_t* src = P1 + part * plane + (size_t)v * D + 8 * (pch ^ km_swz<D>(r));
      km_dma16(src, km_lds_addr(&Wt[slot][0] + (w * NI + i) * 512));
    }
    if (w == 0 && l < CT / 4) {
      km_dma16(bh + c0 + 4 * l, km_lds_addr(&Bt[slot][0]));
      km_dma16(nh + c0 + 4 * l, km_lds_addr(&Nt[slot][0]));
      km_dma16(eh + c0 + 4 * l, km_lds_addr(&Et[slot][0]));
    }
  };
  const int swk = km_swz<D>(c16);
  const int tl = 16 * w + c16;  // this lane's token slot in the chunk
  for (int chunk = wg; chunk < nchunks; chunk += rg) {
    // list positions of this chunk's slots: scan of the tile list lengths
    __syncthreads();  // wsc and spos of the previous chunk consumed
    if (tid < TC) spos[tid] = -1;
    {
      const int lo = chunk * TC;
      int carry = 0;
      for (int p0 = 0; p0 < NT && carry < lo + TC; p0 += 256) {
        const int t = p0 + tid;
        const int c = t < NT ? min(max(nf[t], 0), kmeans_tile) : 0;
        int inc = c;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(inc, o, 64);
          if (l >= o) inc += y;
        }
        __syncthreads();  // previous piece's wsc read; spos cleared
        if (l == 63) wsc[w] = inc;
        __syncthreads();
        int pre = carry, tot = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          pre += q < w ? wsc[q] : 0;
          tot += wsc[q];
        }
        pre += inc - c;
        const int a0 = max(pre, lo), a1 = min(pre + c, lo + TC);
        for (int i = a0; i < a1; ++i) spos[i - lo] = t * kmeans_tile + (i - pre);
        carry += tot;
      }
    }
    __syncthreads();
    bf16x8_t xf[KS];
    float kx, U;
    {
      const int sp = spos[tl];
      int tok = sp >= 0 ? flags[(size_t)h * N + sp] : -1;
      tok = (unsigned)tok < (unsigned)N ? tok : -1;
      U = tok >= 0 ? flagu[(size_t)h * N + sp] : -INFINITY;
      if (U != U) U = INFINITY;  // NaN: every centroid is a candidate
      float xsq = 0.0f;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        uint4 raw = make_uint4(0u, 0u, 0u, 0u);
        if (tok >= 0) raw = *(const uint4*)(Xh + (size_t)tok * D + 32 * s + 8 * g);
        xf[s] = __builtin_bit_cast(bf16x8_t, raw);
        asm volatile("" ::"v"(xf[s]));  // loads complete here, not inside the tile loop
        const uint32_t q[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = __uint_as_float(q[e] << 16), hi = __uint_as_float(q[e] & 0xffff0000u);
          xsq = fmaf(lo, lo, fmaf(hi, hi, xsq));
        }
      }
      xsq += __shfl_xor(xsq, 16, 64);
      xsq += __shfl_xor(xsq, 32, 64);
      kx = KXC * sqrtf(xsq);
      asm volatile("" ::"v"(U));
      if (g == 0) {
        ccount[tl] = 0;
        ctok[tl] = tok;
        cx2[tl] = xsq;
      }
    }
    if (tid == 0) nover = 0;
#pragma unroll
    for (int p = 0; p < NS - 1; ++p)
      if (p < nt) issue(p, p);
    for (int t = 0; t < nt; ++t) {
      // own DMAs of tile t done (wavefront 0 also fetches the b, |w|, eb tiles)
      if (NS > 2 && t + 1 < nt) {
        if (w == 0) km_wait_vmcnt<NI + 3>();
        else km_wait_vmcnt<NI>();
      } else {
        km_wait_vmcnt<0>();
      }
      __syncthreads();  // tile t landed everywhere; tile t-1 consumed
      if (t + NS - 1 < nt) issue(t + NS - 1, (t + NS - 1) % NS);
      const int slot = t % NS;
      const bf16_t* W1 = &Wt[slot][0];
      const bf16_t* W2 = W1 + CT * D;
      const bf16_t* W3 = W2 + CT * D;
#pragma unroll
      for (int cb = 0; cb < CT / 16; ++cb) {
        f32x4_t ahi = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f}, arest = ahi;
        const int rowo = (16 * cb + c16) * D;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const int co = rowo + 8 * ((4 * s + g) ^ swk);
          const bf16x8_t a1 = *(const bf16x8_t*)(W1 + co);
          const bf16x8_t a2 = *(const bf16x8_t*)(W2 + co);
          const bf16x8_t a3 = *(const bf16x8_t*)(W3 + co);
          ahi = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, xf[s], ahi, 0, 0, 0);
          arest = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, xf[s], arest, 0, 0, 0);
          arest = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a3, xf[s], arest, 0, 0, 0);
        }
        const int cl = 16 * cb + 4 * g;
        const float4 b4 = *(const float4*)(&Bt[slot][cl]);
        const float4 n4 = *(const float4*)(&Nt[slot][cl]);
        const float4 e4 = *(const float4*)(&Et[slot][cl]);
        const float bv[4] = {b4.x, b4.y, b4.z, b4.w}, nv[4] = {n4.x, n4.y, n4.z, n4.w},
                    ev[4] = {e4.x, e4.y, e4.z, e4.w};
        const int vb = t * CT + cl;
        bool cand[4], anyc = false;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float sc = fmaf(-2.0f, ahi[r] + arest[r], bv[r]);
          const float er = fmaf(kx, nv[r], ev[r]);
          cand[r] = vb + r < C && !(sc - er > U);
          anyc |= cand[r];
        }
        if (__any(anyc)) {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (cand[r]) {
              const int pos = atomicAdd(&ccount[tl], 1);
              if (pos < KMAX) cv[tl * KMAX + pos] = vb + r;
            }
        }
      }
    }
    __syncthreads();
    // pack the pairs (token, candidate) of tokens with 1..KMAX candidates;
    // list the others (more candidates) for the all-centroid pass
    if (w == 0) {
      const int nc = ccount[l];
      const bool packed = ctok[l] >= 0 && nc >= 1 && nc <= KMAX;
      const int np = packed ? nc : 0;
      int inc = np;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(inc, o, 64);
        if (l >= o) inc += y;
      }
      const int start = inc - np;
      poff[l] = start;
      for (int j = 0; j < np; ++j) {
        ptl[start + j] = l;
        pv[start + j] = cv[l * KMAX + j];
      }
      if (ctok[l] >= 0 && !packed) over[atomicAdd(&nover, 1)] = l;
      if (l == 63) npairs = inc;
    }
    __syncthreads();
    // float64 scores of the packed pairs, PL lanes per pair (PE dimensions each)
    {
      const int lp = tid / PL, sub = tid % PL, np = npairs;
      for (int base = 0; base < np; base += KP * (256 / PL)) {
        double a[KP];
        int pp[KP];
#pragma unroll
        for (int k = 0; k < KP; ++k) {
          const int p = base + (256 / PL) * k + lp;
          pp[k] = p < np ? p : -1;
          a[k] = 0.0;
          if (p < np) {
            const int tok = ctok[ptl[p]];
            uint32_t q[PE / 2];  // this lane's PE dimensions, two bf16 per word
            if constexpr (PE == 8) {
              const uint4 xu = *(const uint4*)(Xh + (size_t)tok * D + sub * PE);
              q[0] = xu.x;
              q[1] = xu.y;
              q[2] = xu.z;
              q[3] = xu.w;
            } else {
              const uint2 xu = *(const uint2*)(Xh + (size_t)tok * D + sub * PE);
              q[0] = xu.x;
              q[1] = xu.y;
            }
            const double* wr = wh + (size_t)pv[p] * D + sub * PE;
#pragma unroll
            for (int e = 0; e < PE / 2; ++e) {
              a[k] = fma((double)__uint_as_float(q[e] << 16), wr[2 * e], a[k]);
              a[k] = fma((double)__uint_as_float(q[e] & 0xffff0000u), wr[2 * e + 1], a[k]);
            }
          }
        }
#pragma unroll
        for (int k = 0; k < KP; ++k) {
          double t = a[k];
#pragma unroll
          for (int o = PL / 2; o > 0; o >>= 1) t += __shfl_xor(t, o, 64);
          if (sub == 0 && pp[k] >= 0) cs[pp[k]] = fma(-2.0, t, b64h[pv[pp[k]]]);
        }
      }
    }
    __syncthreads();
    // tokens with too many candidates: float64 scores of every centroid
    for (int i = 0; i < nover; ++i) {
      const int ot = over[i], tok = ctok[ot];
      for (int a0 = tid; a0 < D; a0 += 256) xrow[a0] = (double)to_f(Xh[(size_t)tok * D + a0]);
      __syncthreads();
      double bb = INFINITY;
      int bi = 0x7fffffff;
      for (int v = tid; v < C; v += 256) {
        const double* wr = wh + (size_t)v * D;
        double acc = 0.0;
        for (int a0 = 0; a0 < D; ++a0) acc = fma(xrow[a0], wr[a0], acc);
        const double sc = fma(-2.0, acc, b64h[v]);
        if (sc < bb) {
          bb = sc;
          bi = v;
        }
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const double ob = __shfl_xor(bb, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (ob < bb || (ob == bb && oi < bi)) {
          bb = ob;
          bi = oi;
        }
      }
      if (l == 0) {
        rbest[w] = bb;
        ridx[w] = bi;
      }
      __syncthreads();
      if (tid == 0) {
        for (int q = 1; q < 4; ++q)
          if (rbest[q] < rbest[0] || (rbest[q] == rbest[0] && ridx[q] < ridx[0])) {
            rbest[0] = rbest[q];
            ridx[0] = ridx[q];
          }
        obest[ot] = rbest[0];
        oidx[ot] = ridx[0];
      }
      __syncthreads();
    }
    // labels: the smallest float64 score, ties to the lowest id
    if (tid < TC) {
      const int tok = ctok[tid], nc = ccount[tid];
      if (tok >= 0) {
        double bb;
        int bi;
        if (nc >= 1 && nc <= KMAX) {
          bb = INFINITY;
          bi = 0x7fffffff;
          for (int j = 0; j < nc; ++j) {
            const int p = poff[tid] + j;
            const double sc = cs[p];
            const int v = pv[p];
            if (sc < bb || (sc == bb && v < bi)) {
              bb = sc;
              bi = v;
            }
          }
        } else {
          bb = obest[tid];
          bi = oidx[tid];
        }
        if (!isfinite(bb) || (unsigned)bi >= (unsigned)C) {
          raise_status(status, ST_NONFINITE);
          bi = 0;
        } else if (dmax) {
          // radius bound of the next filtered round (see k_prep)
          const double d2 = fmax(xn[(size_t)h * N + tok] + bb +
                                     1e-12 * (fabs(b64h[bi]) +
                                              2.0 * sqrt((double)cx2[tid]) * (double)nh[bi]),
                                 0.0);
          atomicMax(&dmax[(size_t)h * C + bi], (unsigned long long)__double_as_longlong(d2));
        }
        labels[(size_t)h * N + tok] = bi;
      }
    }
    __syncthreads();
  }
}

// Exact float64 assignment: labels[j] = argmin_v (b_v - 2 x_j . w_v), ties to
// the lowest v.  TM tokens x 64 centroids per step (centroids staged in LDS
// in 32-dim slices), 4 tokens x (64 / (256 / (TM / 4))) centroids per
// thread.  With a token list (list != null) it assigns only the first
// count[h] listed tokens (the ones the fast path left uncertified);
// workgroups loop over tiles.
template <typename T, int D, int TM>
__global__ __launch_bounds__(256) void k_assign64(const T* __restrict__ X, const double* __restrict__ w,
                                                  const double* __restrict__ b, int N, int C,
                                                  const int* __restrict__ list,
                                                  const int* __restrict__ count,
                                                  int* __restrict__ labels, int* status) {
  constexpr int TC = 64, DC = 32;
  constexpr int TGN = TM / 4;        // token groups (4 tokens each, strided by TGN)
  constexpr int CGN = 256 / TGN;     // centroid groups
  constexpr int CPT = TC / CGN;      // centroids per thread and tile (strided by CGN)
  __shared__ float xs[TM][D + 1];
  __shared__ double wsm[TC][DC + 1];
  __shared__ double bs[TC];
  __shared__ double rs[CGN][TM];
  __shared__ int ri[CGN][TM];
  __shared__ int tok_s[TM];
  const int h = blockIdx.y, tid = threadIdx.x;
  const int ntok = list ? min(count[h], N) : N;
  const T* Xh = X + (size_t)h * N * D;
  const double* wh = w + (size_t)h * C * D;
  const int tg = tid % TGN, cg = tid / TGN;
  for (int t0 = blockIdx.x * TM; t0 < ntok; t0 += gridDim.x * TM) {
    __syncthreads();
    if (tid < TM) {
      int tok = -1;
      if (t0 + tid < ntok) tok = list ? list[(size_t)h * N + t0 + tid] : t0 + tid;
      tok_s[tid] = ((unsigned)tok < (unsigned)N) ? tok : -1;
    }
    __syncthreads();
    for (int e = tid; e < TM * D; e += 256) {
      const int r = e / D, c = e % D;
      const int tok = tok_s[r];
      xs[r][c] = tok >= 0 ? to_f(Xh[(size_t)tok * D + c]) : 0.0f;
    }
    double best[4];
    int bidx[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      best[i] = INFINITY;
      bidx[i] = 0x7fffffff;
    }
    for (int c0 = 0; c0 < C; c0 += TC) {
      double acc[4][CPT];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < CPT; ++j) acc[i][j] = 0.0;
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
          double xv[4], wv[CPT];
#pragma unroll
          for (int i = 0; i < 4; ++i) xv[i] = (double)xs[tg + TGN * i][a0 + a];
#pragma unroll
          for (int j = 0; j < CPT; ++j) wv[j] = wsm[cg + CGN * j][a];
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < CPT; ++j) acc[i][j] = fma(xv[i], wv[j], acc[i][j]);
        }
      }
#pragma unroll
      for (int j = 0; j < CPT; ++j) {
        const int v = c0 + cg + CGN * j;
        if (v < C) {
          const double bv = bs[cg + CGN * j];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const double sc = fma(-2.0, acc[i][j], bv);
            if (sc < best[i] || (sc == best[i] && v < bidx[i])) {
              best[i] = sc;
              bidx[i] = v;
            }
          }
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      rs[cg][tg + TGN * i] = best[i];
      ri[cg][tg + TGN * i] = bidx[i];
    }
    __syncthreads();
    if (tid < TM && tok_s[tid] >= 0) {
      double bb = rs[0][tid];
      int bi = ri[0][tid];
      for (int q = 1; q < CGN; ++q) {
        const double sc = rs[q][tid];
        const int v = ri[q][tid];
        if (sc < bb || (sc == bb && v < bi)) {
          bb = sc;
          bi = v;
        }
      }
      if (!isfinite(bb) || bi >= C) {
        raise_status(status, ST_NONFINITE);
        bi = 0;
      }
      labels[(size_t)h * N + tok_s[tid]] = bi;
    }
  }
}

// Segmented mean over permuted rows: block v of head h averages
// X[perm[i]] (X[i] when perm is null) for offsets[v] <= i < offsets[v+1] in
// float64.  256 threads = 16 row lanes x 16 column chunks (D/16 columns
// each); row lane j sums rows j, j+16, ... and the 16 partial sums are added
// in lane order, so the result is deterministic.  Empty blocks keep mu64 and
// give c32 = 0.
template <typename T, int D>
__global__ __launch_bounds__(256) void k_segment_mean(const T* __restrict__ X,
                                                      const int* __restrict__ perm,
                                                      const int* __restrict__ offsets, int N,
                                                      int C, double* __restrict__ mu64,
                                                      float* __restrict__ c32,
                                                      int* __restrict__ sizes) {
  constexpr int RL = 16, CW = D / 16;  // row lanes, columns per thread
  __shared__ double part[RL][D + 1];
  const int h = blockIdx.y, v = blockIdx.x, tid = threadIdx.x;
  const int* off = offsets + (size_t)h * (C + 1);
  const int o0 = min(max(off[v], 0), N), o1 = min(max(off[v + 1], o0), N);
  const int n = o1 - o0;
  if (sizes && tid == 0) sizes[(size_t)h * C + v] = n;
  const size_t dst = ((size_t)h * C + v) * D;
  if (n <= 0) {
    if (c32)
      for (int a = tid; a < D; a += 256) c32[dst + a] = 0.0f;
    return;
  }
  const int* p = perm ? perm + (size_t)h * N : nullptr;
  const T* Xh = X + (size_t)h * N * D;
  const int j = tid / 16, c0 = (tid % 16) * CW;
  double acc[CW];
#pragma unroll
  for (int c = 0; c < CW; ++c) acc[c] = 0.0;
  // rows j, j + RL, ... in order; four rows' loads in flight at a time,
  // each row segment (CW elements) read as 8- or 16-byte vectors
  constexpr int UR = 4, NW = (int)sizeof(T) * CW / 4;
  static_assert(NW == 2 || NW % 4 == 0, "row segment of 8 or 16k bytes");
  for (int r0 = o0 + j; r0 < o1; r0 += UR * RL) {
    int idx[UR];
#pragma unroll
    for (int u = 0; u < UR; ++u) {
      const int r = r0 + u * RL;
      idx[u] = r < o1 ? (p ? p[r] : r) : -1;
    }
    uint32_t xw[UR][NW];
#pragma unroll
    for (int u = 0; u < UR; ++u) {
      const bool ok = (unsigned)idx[u] < (unsigned)N;
      const T* xr = Xh + (size_t)(ok ? idx[u] : 0) * D + c0;
      if constexpr (NW == 2) {
        uint2 q = ok ? *(const uint2*)xr : make_uint2(0u, 0u);
        xw[u][0] = q.x;
        xw[u][1] = q.y;
      } else {
#pragma unroll
        for (int k = 0; k < NW / 4; ++k) {
          const uint4 q = ok ? ((const uint4*)xr)[k] : make_uint4(0u, 0u, 0u, 0u);
          xw[u][4 * k] = q.x;
          xw[u][4 * k + 1] = q.y;
          xw[u][4 * k + 2] = q.z;
          xw[u][4 * k + 3] = q.w;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < UR; ++u)
#pragma unroll
      for (int c = 0; c < CW; ++c) {
        float f;
        if constexpr (sizeof(T) == 2)
          f = __uint_as_float((c & 1) ? (xw[u][c >> 1] & 0xffff0000u) : (xw[u][c >> 1] << 16));
        else
          f = __uint_as_float(xw[u][c]);
        acc[c] += (double)f;
      }
  }
#pragma unroll
  for (int c = 0; c < CW; ++c) part[j][c0 + c] = acc[c];
  __syncthreads();
  for (int a = tid; a < D; a += 256) {
    double sum = 0.0;
    for (int q = 0; q < RL; ++q) sum += part[q][a];
    const double m = sum / (double)n;
    if (mu64) mu64[dst + a] = m;
    if (c32) c32[dst + a] = (float)m;
  }
}

// ---------------------------------------------------------------- launchers
park_status launch_segment_mean(const void* X, const int* perm, const int* offsets, int H, int N,
                                int D, int dtype, int C, double* mu64, float* c32, int* sizes,
                                hipStream_t st) {
  dim3 g(C, H);
  if (D == 128) {
    if (dtype == PARK_BF16)
      PARK_LAUNCH("segment_mean", (k_segment_mean<bf16_t, 128>), g, dim3(256), 0, st,
                  (const bf16_t*)X, perm, offsets, N, C, mu64, c32, sizes);
    else
      PARK_LAUNCH("segment_mean", (k_segment_mean<float, 128>), g, dim3(256), 0, st,
                  (const float*)X, perm, offsets, N, C, mu64, c32, sizes);
  } else {
    if (dtype == PARK_BF16)
      PARK_LAUNCH("segment_mean", (k_segment_mean<bf16_t, 64>), g, dim3(256), 0, st,
                  (const bf16_t*)X, perm, offsets, N, C, mu64, c32, sizes);
    else
      PARK_LAUNCH("segment_mean", (k_segment_mean<float, 64>), g, dim3(256), 0, st,
                  (const float*)X, perm, offsets, N, C, mu64, c32, sizes);
  }
  return PARK_OK;
}

// PARK_KMEANS_FILTER=0 runs every assignment round dense (the same labels;
// for timing the filter against the dense sweep)
static bool kmeans_filter_enabled() {
  const char* e = getenv("PARK_KMEANS_FILTER");
  return !(e && e[0] == '0');
}

// PARK_KFILTER_EXACT_RADIUS=1 measures every round's radii with k_radius
// instead of bounding them from the previous assignment (the same labels)
static bool kfilter_exact_radius() {
  const char* e = getenv("PARK_KFILTER_EXACT_RADIUS");
  return e && e[0] == '1';
}

template <typename T, int D>
static park_status kmeans_impl(const T* X, const double* Gbar, int H, int N, int C, int T_,
                               uint64_t seed, int side, const KmeansBufs& kb, int* status,
                               hipStream_t st) {
  constexpr bool fast = sizeof(T) == 2;  // bf16 points: MFMA fast path + float64 refine
  const size_t plane = (size_t)H * C * D;
  const long ncen = (long)H * C * D;
  if (kb.mu_init) {  // warm start: the caller's centroids (the previous recompute's means)
    PARK_LAUNCH("kmeans_warm", k_copy64, dim3((unsigned)((ncen + 255) / 256)), dim3(256), 0, st,
                kb.mu_init, kb.mu, ncen);
  } else {
    PARK_LAUNCH("kmeans_init", k_init_idx, dim3(H), dim3(1024), 0, st, N, C, seed, side, kb.init);
    PARK_LAUNCH("kmeans_seed", k_seed_centroids<T>, dim3(C, H), dim3(D), 0, st, X,
                (const int*)kb.init, N, D, C, kb.mu);
  }
  // refine grid: persistent workgroups per head looping over 64-token chunks
  int rg = (2048 + H - 1) / H;
  const int max_tiles = (N + 63) / 64;
  rg = rg < 2 ? 2 : rg;
  rg = rg > max_tiles ? max_tiles : rg;
  // the exact candidate filter for the rounds after the first (bf16 points),
  // where the dense sweep is MFMA-bound (C >= 512); below that the dense
  // round is a few tens of microseconds and the filter's passes cost more
  const bool filt = fast && kb.kf != nullptr && C >= 512 && kmeans_filter_enabled();
  const bool exact_radius = kfilter_exact_radius();
  if constexpr (fast)
    if (filt) PARK_TRY(launch_kfilter_setup((const bf16_t*)X, Gbar, H, N, D, *kb.kf, st));
  bf16_t* m2 = filt ? kb.kf->m2 : nullptr;
  float* mn = filt ? kb.kf->mn : nullptr;
  for (int t = 0; t < T_; ++t) {
    const int nbm = (C + 15) / 16;
    // radii: round 1 measures them (k_radius); later rounds bound them from
    // the previous assignment's distances and the centroids' moves
    const int rmode = !filt || t == 0 ? 0 : (t == 1 || exact_radius ? 1 : 2);
    double* r2 = filt ? kb.kf->r2 : nullptr;
    unsigned long long* dmax = filt ? kb.kf->dmax : nullptr;
    if ((long)nbm * H < 512)
      PARK_LAUNCH("kmeans_prep", (k_prep<D, 1024>), dim3(nbm, H), dim3(1024), 0, st,
                  (const double*)kb.mu, Gbar, C, kb.w, kb.b, fast ? kb.w3 : nullptr, plane,
                  fast ? kb.b32 : nullptr, kmeans_cpad(C), fast ? kb.wn : nullptr,
                  fast ? kb.eb : nullptr, kb.hmax, m2, mn, (const int*)kb.offsets, r2, dmax,
                  rmode);
    else
      PARK_LAUNCH("kmeans_prep", (k_prep<D, 256>), dim3(nbm, H), dim3(256), 0, st,
                  (const double*)kb.mu, Gbar, C, kb.w, kb.b, fast ? kb.w3 : nullptr, plane,
                  fast ? kb.b32 : nullptr, kmeans_cpad(C), fast ? kb.wn : nullptr,
                  fast ? kb.eb : nullptr, kb.hmax, m2, mn, (const int*)kb.offsets, r2, dmax,
                  rmode);
    if constexpr (fast) {
      if (filt && t > 0)
        PARK_TRY(launch_kfilter_round((const bf16_t*)X, H, N, D, C, kb, *kb.kf, rmode == 1, st));
      else if (C >= 512)
        PARK_LAUNCH("kmeans_assign_fast", (k_assign_fast<D, 2>), dim3((N + kmeans_tile - 1) / kmeans_tile, H),
                    dim3(256), 0, st, (const bf16_t*)X, (const bf16_t*)kb.w3, plane,
                    (const float*)kb.b32, kmeans_cpad(C), (const float*)kb.wn, (const float*)kb.eb,
                    (const float*)kb.hmax, nbm, N, C, kb.labels, kb.flags, kb.flagu, kb.nflag);
      else
        PARK_LAUNCH("kmeans_assign_fast", (k_assign_fast<D, 3>), dim3((N + kmeans_tile - 1) / kmeans_tile, H),
                    dim3(256), 0, st, (const bf16_t*)X, (const bf16_t*)kb.w3, plane,
                    (const float*)kb.b32, kmeans_cpad(C), (const float*)kb.wn, (const float*)kb.eb,
                    (const float*)kb.hmax, nbm, N, C, kb.labels, kb.flags, kb.flagu, kb.nflag);
      PARK_LAUNCH("kmeans_refine64", k_refine_cand<D>, dim3(8 * ((rg * H + 7) / 8)),
                  dim3(256), 0, st, (const bf16_t*)X, (const bf16_t*)kb.w3, plane,
                  (const float*)kb.b32, (const float*)kb.wn, (const float*)kb.eb, kmeans_cpad(C),
                  (const double*)kb.w, (const double*)kb.b, H, N, C, rg, (const int*)kb.flags,
                  (const float*)kb.flagu, (const int*)kb.nflag, kb.labels, status,
                  filt && t > 0 ? (const double*)kb.kf->xn : nullptr,
                  filt && t > 0 ? kb.kf->dmax : nullptr);
    } else {
      PARK_LAUNCH("kmeans_assign64", (k_assign64<T, D, 64>), dim3((N + 63) / 64, H), dim3(256), 0, st,
                  X, (const double*)kb.w, (const double*)kb.b, N, C, (const int*)nullptr,
                  (const int*)nullptr, kb.labels, status);
    }
    if (t + 1 < T_) {
      PARK_TRY(launch_count_sort(kb.labels, H, N, C, kb.thist, kb.perm, kb.offsets, st));
      PARK_LAUNCH("segment_mean", (k_segment_mean<T, D>), dim3(C, H), dim3(256), 0, st, X,
                  (const int*)kb.perm, (const int*)kb.offsets, N, C, kb.mu, (float*)nullptr,
                  (int*)nullptr);
    }
  }
  PARK_TRY(launch_count_sort(kb.labels, H, N, C, kb.thist, kb.perm, kb.offsets, st));
  if (kb.mu_out) {
    // the means of the final clusters (an empty cluster keeps the centroid
    // of the last assignment): the next recompute's warm start
    PARK_LAUNCH("kmeans_warm", k_copy64, dim3((unsigned)((ncen + 255) / 256)), dim3(256), 0, st,
                (const double*)kb.mu, kb.mu_out, ncen);
    PARK_LAUNCH("segment_mean", (k_segment_mean<T, D>), dim3(C, H), dim3(256), 0, st, X,
                (const int*)kb.perm, (const int*)kb.offsets, N, C, kb.mu_out, (float*)nullptr,
                (int*)nullptr);
  }
  return PARK_OK;
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
