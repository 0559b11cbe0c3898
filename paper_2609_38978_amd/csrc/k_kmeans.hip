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
// applies each element to 16 / (256 / D) centroids.  `wT` (optional) receives
// w transposed, [D][C] per head, for the float64 refinement.  When `w3` is
// given the fast-path operands are written too: w_v split into three bf16
// parts (three planes of H*C*D), b_v in float, |w_v| rounded up and the
// |b_v| term of the error bound (see k_assign_fast).
template <int D>
__global__ __launch_bounds__(256) void k_prep(const double* __restrict__ mu,
                                              const double* __restrict__ Gbar, int C,
                                              double* __restrict__ w, double* __restrict__ b,
                                              bf16_t* __restrict__ w3,
                                              size_t plane, float* __restrict__ b32, int Cpad,
                                              float* __restrict__ wn, float* __restrict__ eb,
                                              float* __restrict__ bmax, int* __restrict__ nflag) {
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
    if (v0 + r < C) {
      const size_t o = ((size_t)h * C + v0 + r) * D + a;
      w[o] = acc[k];
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
    }
  }
  __syncthreads();
  float fn = 0.0f, fe = 0.0f;
  if (tid < CB && v0 + tid < C) {
    double s = 0.0, n2 = 0.0;
    for (int c = 0; c < D; ++c) {
      s = fma(ms[tid][c], ws[tid][c], s);
      n2 = fma(ws[tid][c], ws[tid][c], n2);
    }
    b[(size_t)h * C + v0 + tid] = s;
    if (b32) {
      fn = (float)(sqrt(n2) * (1.0 + 1e-6));
      fe = (float)(fabs(s) * (2.0 * 1.1 * 5.9604644775390625e-08) * (1.0 + 1e-6));
      b32[(size_t)h * Cpad + v0 + tid] = (float)s;
      wn[(size_t)h * Cpad + v0 + tid] = fn;
      eb[(size_t)h * Cpad + v0 + tid] = fe;
    }
  }
  if (b32 && blockIdx.x == gridDim.x - 1)  // padding centroids: score +inf, no error term
    for (int v = C + tid; v < Cpad; v += 256) {
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
      if (blockIdx.x == 0) nflag[h] = 0;  // the previous refinement has completed
    }
  }
}

// ---------------------------------------------------------------------------
// Fast assignment on bf16 MFMA with certification.
//
// For a bf16 point x the score s_v = b_v - 2 x.w_v is evaluated with w_v
// split into NP bf16 parts, w = w1 + w2 (+ w3) + r, with |r| <= 2^-16 (1.01)
// |w| for two parts and 2^-24 (1 + 2^-7)|w| for three.  All products are
// bf16 x bf16, exact in float.  x.w1 is accumulated over the D dimensions in
// one chain of v_mfma_f32_16x16x32_bf16, the smaller parts (terms 2^-8
// smaller) in a second chain, and the two are added once.  With delta =
// 2^-23 per addition inside an MFMA (any faithful rounding) and 2^-24 for
// the VALU rounding, the forward error of t^ = x.w is at most
//   et sum_a |x_a w_a|,  et = er 1.01 + (D+1) delta (1 + 2^-7)
//                            + 2^-8 1.01 ((NP-1) D + 1) delta + 2^-24 1.01,
// er the residual bound above.  Two parts take 2/3 of the MFMA work and
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
// Bookkeeping per lane and token (the lane sees a quarter of the centroids):
// best (score and id) and L.  Each 16-centroid step gives the lane 4 scores;
// their minimum m either stays above best (the common case: L = min(L, m))
// or some lane of the wavefront takes the per-score path.  The running best
// starts at an estimate of the score of the token's previous label (plus a
// margin) with no id, so after the first iterations almost no score beats
// it; the estimate never enters L, and a token whose best is still that
// estimate at the end is listed for refinement.  Correctness does not depend
// on the estimate, only the number of listed tokens does.
//
// Workgroup = 256 tokens (4 wavefronts x 4 blocks of 16).  Centroid tiles of
// 32 rows of the three parts go from HBM to a two-slot LDS ring by LDS DMA
// (rows swizzled in 16-byte chunks, see the reads), the next tile in flight
// while this one is scored.  MFMA orientation: A = 16 centroids x 32 dims,
// B = 32 dims x 16 tokens, so lane l holds centroids 4(l/16)+r of token l%16.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

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
__global__ __launch_bounds__(256) void k_assign_fast(const bf16_t* __restrict__ X,
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
  constexpr int TB = 4, CT = 32, KS = D / 32, CPR = D / 8, RPI = 64 / CPR;
  constexpr int NI = NP * CT / (4 * RPI);  // DMAs per wavefront and tile
  static_assert(NI * 4 * RPI == NP * CT && (NP == 2 || NP == 3), "tile shape");
  constexpr float U24 = 5.9604645e-08f, DEL = 1.1920929e-07f;
  // residual of the split: 2^-16 (two parts) or 2^-24 (three parts), relative
  constexpr float ER = NP == 2 ? 1.52587891e-05f : U24;
  constexpr float ET = ER * 1.01f + (D + 1) * DEL * 1.0079f +
                       0.00390625f * 1.01f * ((NP - 1) * D + 1) * DEL + U24 * 1.01f;
  constexpr float KXC = 1.1f * (2.0f * ET + 2.01f * U24) * 1.0001f;
  constexpr int NS = PARK_KM_NS;  // LDS ring slots: NS - 1 tiles in flight
  __shared__ __attribute__((aligned(16))) bf16_t Wt[NS][NP * CT * D];  // [slot][part][row][D]
  __shared__ __attribute__((aligned(16))) float Bt[NS][CT];
  __shared__ float mx_s[2];
  const int h = blockIdx.y, tid = threadIdx.x, l = tid & 63, g = l >> 4, c16 = l & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int t0 = blockIdx.x * 256 + w * 64;
  const bf16_t* Xh = X + (size_t)h * N * D;
  const bf16_t* P1 = w3 + (size_t)h * C * D;
  const float* bh = b32 + (size_t)h * Cpad;
  bf16x8_t xf[TB][KS];
  float xsq[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    xsq[tb] = 0.0f;
    const int tok = t0 + 16 * tb + c16;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      uint4 raw = make_uint4(0u, 0u, 0u, 0u);
      if (tok < N) raw = *(const uint4*)(Xh + (size_t)tok * D + 32 * s + 8 * g);
      xf[tb][s] = __builtin_bit_cast(bf16x8_t, raw);
      const uint32_t q[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float lo = __uint_as_float(q[e] << 16), hi = __uint_as_float(q[e] & 0xffff0000u);
        xsq[tb] = fmaf(lo, lo, fmaf(hi, hi, xsq[tb]));
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
  // running best: an estimate of the previous label's score plus a margin
  float kx[TB], best[TB], L[TB];
  int bidx[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    float xs = xsq[tb] + __shfl_xor(xsq[tb], 16, 64);
    xs += __shfl_xor(xs, 32, 64);
    kx[tb] = KXC * sqrtf(xs);
    const int tok = t0 + 16 * tb + c16;
    int prev = tok < N ? labels[(size_t)h * N + tok] : -1;
    prev = (unsigned)prev < (unsigned)C ? prev : -1;
    float dot = 0.0f;
    if (prev >= 0) {
      const bf16_t* wp = P1 + (size_t)prev * D + 8 * g;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const uint4 u1 = *(const uint4*)(wp + 32 * s);
        const uint4 u2 = *(const uint4*)(wp + plane + 32 * s);
        const uint4 u3 = *(const uint4*)(wp + 2 * plane + 32 * s);
        const uint4 ux = __builtin_bit_cast(uint4, xf[tb][s]);
        const uint32_t a1[4] = {u1.x, u1.y, u1.z, u1.w}, a2[4] = {u2.x, u2.y, u2.z, u2.w},
                       a3[4] = {u3.x, u3.y, u3.z, u3.w}, ax[4] = {ux.x, ux.y, ux.z, ux.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float wl = (__uint_as_float(a1[e] << 16) + __uint_as_float(a2[e] << 16)) +
                           __uint_as_float(a3[e] << 16);
          const float wh = (__uint_as_float(a1[e] & 0xffff0000u) +
                            __uint_as_float(a2[e] & 0xffff0000u)) +
                           __uint_as_float(a3[e] & 0xffff0000u);
          dot = fmaf(__uint_as_float(ax[e] << 16), wl, dot);
          dot = fmaf(__uint_as_float(ax[e] & 0xffff0000u), wh, dot);
        }
      }
    }
    dot += __shfl_xor(dot, 16, 64);
    dot += __shfl_xor(dot, 32, 64);
    best[tb] = INFINITY;
    if (prev >= 0) {
      // the fast score of prev is within e of its exact score, and the float
      // estimate (three parts, 32-term lane sums) within 2^-17 |x| |w| of it
      const float wnp = wn[(size_t)h * Cpad + prev];
      const float e = fmaf(kx[tb], wnp, eb[(size_t)h * Cpad + prev]);
      const float est = fmaf(-2.0f, dot, bh[prev]);
      best[tb] = est + 1.05f * e + (7.62939453e-06f / KXC) * kx[tb] * wnp + 1e-7f * fabsf(est);
    }
    L[tb] = INFINITY;
    bidx[tb] = -1;
  }
  // all global loads done before the tile loop (its waits are explicit)
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
#pragma unroll
    for (int s = 0; s < KS; ++s) asm volatile("" ::"v"(xf[tb][s]));
    asm volatile("" ::"v"(best[tb]), "v"(kx[tb]));
  }

  // LDS DMA lanes: row rr[i] of the tile's 3*CT part-rows, chunk pch
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
    if (w == 0 && l < CT / 4) km_dma16(bh + c0 + 4 * l, km_lds_addr(&Bt[slot][0]));
  };
#pragma unroll
  for (int p = 0; p < NS - 1; ++p)
    if (p < ntiles) issue(p, p);
  const int swk = km_swz<D>(c16);
  for (int t = 0; t < ntiles; ++t) {
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
#pragma unroll
    for (int cb = 0; cb < CT / 16; ++cb) {
      f32x4_t ahi[TB], arest[TB];
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        ahi[tb] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        arest[tb] = ahi[tb];
      }
      const int rowo = (16 * cb + c16) * D;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const int co = rowo + 8 * ((4 * s + g) ^ swk);
        const bf16x8_t a1 = *(const bf16x8_t*)(W1 + co);
        const bf16x8_t a2 = *(const bf16x8_t*)(W2 + co);
        bf16x8_t a3;
        if constexpr (NP == 3) a3 = *(const bf16x8_t*)(W3 + co);
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
          ahi[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, xf[tb][s], ahi[tb], 0, 0, 0);
          arest[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, xf[tb][s], arest[tb], 0, 0, 0);
          if constexpr (NP == 3)
            arest[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a3, xf[tb][s], arest[tb], 0, 0, 0);
        }
      }
      const float4 b4 = *(const float4*)(&Bt[slot][16 * cb + 4 * g]);
      const float bv[4] = {b4.x, b4.y, b4.z, b4.w};
      const int vbase = t * CT + 16 * cb + 4 * g;
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        float sc[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) sc[r] = fmaf(-2.0f, ahi[tb][r] + arest[tb][r], bv[r]);
        const float m = fminf(fminf(sc[0], sc[1]), fminf(sc[2], sc[3]));
        const bool c = m < best[tb];
        if (__any(c)) {
          if (c) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const bool nb = sc[r] < best[tb];
              const float out = nb ? (bidx[tb] >= 0 ? best[tb] : INFINITY) : sc[r];
              L[tb] = fminf(L[tb], out);
              best[tb] = nb ? sc[r] : best[tb];
              bidx[tb] = nb ? vbase + r : bidx[tb];
            }
          } else {
            L[tb] = fminf(L[tb], m);
          }
        } else {
          L[tb] = fminf(L[tb], m);
        }
      }
    }
  }
  const float nmax = mx_s[0], ebmax = mx_s[1];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    // merge over the four lane groups holding this token (ties: lowest id)
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float ob = __shfl_xor(best[tb], o, 64), oL = __shfl_xor(L[tb], o, 64);
      const int oi = __shfl_xor(bidx[tb], o, 64);
      const bool mine_valid = bidx[tb] >= 0, other_valid = oi >= 0;
      const bool take = other_valid && (!mine_valid || ob < best[tb] ||
                                        (ob == best[tb] && oi < bidx[tb]));
      const float loser = take ? (mine_valid ? best[tb] : INFINITY)
                               : (other_valid ? ob : INFINITY);
      L[tb] = fminf(fminf(L[tb], oL), loser);
      best[tb] = take ? ob : best[tb];
      bidx[tb] = take ? oi : bidx[tb];
    }
    const int tok = t0 + 16 * tb + c16;
    if (g == 0 && tok < N) {
      bool ok = false;
      float ub = INFINITY;  // an upper bound of the smallest exact score
      if (bidx[tb] >= 0 && isfinite(best[tb])) {
        const int v = bidx[tb];
        const float e1 = fmaf(kx[tb], wn[(size_t)h * Cpad + v], eb[(size_t)h * Cpad + v]);
        const float emax = fmaf(kx[tb], nmax, ebmax) * 1.0001f;
        ub = best[tb] + e1;
        ok = (L[tb] - emax) > ub;
      }
      if (ok) {
        labels[(size_t)h * N + tok] = bidx[tb];
      } else {
        const int slot = atomicAdd(nflag + h, 1);
        flags[(size_t)h * N + slot] = tok;
        flagu[(size_t)h * N + slot] = ub;
      }
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
// path) collects each token's candidates in LDS; they are then scored in
// float64 (b_v - 2 x.w_v, partial sums over 8 lanes added in a fixed tree)
// and the minimum, ties to the lowest id, is the label.
// Near-ties leave two or three candidates; a token with more than KMAX
// (exact duplicates, degenerate data) is scored against every centroid.
// Workgroups take chunks of 256 listed tokens (4 wavefronts x 4 x 16).
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
                                                     int* __restrict__ labels, int* status) {
  constexpr int TB = 4, CT = 32, KS = D / 32, CPR = D / 8, RPI = 64 / CPR;
  constexpr int NI = 3 * CT / (4 * RPI);
  constexpr int KMAX = 4;            // candidates kept per token
  constexpr int PL = 8, PE = D / PL;  // lanes per scored pair, elements per lane
  constexpr float U24 = 5.9604645e-08f, DEL = 1.1920929e-07f;
  constexpr float ET = U24 * 1.01f + (D + 1) * DEL * 1.0079f + 0.00390625f * 1.01f * (2 * D + 1) * DEL +
                       U24 * 1.01f;
  constexpr float KXC = 1.1f * (2.0f * ET + 2.01f * U24) * 1.0001f;
  __shared__ __attribute__((aligned(16))) bf16_t Wt[2][3 * CT * D];
  __shared__ __attribute__((aligned(16))) float Bt[2][CT];
  __shared__ __attribute__((aligned(16))) float Nt[2][CT];
  __shared__ __attribute__((aligned(16))) float Et[2][CT];
  __shared__ int ccount[256];
  __shared__ int ctok[256];
  __shared__ int cv[256 * KMAX];    // candidates by token slot
  __shared__ double cs[256 * KMAX];  // float64 scores of the packed pairs
  __shared__ int nover;
  __shared__ int over[256];
  __shared__ double xrow[D];
  __shared__ double rbest[4];
  __shared__ int ridx[4];
  __shared__ int wsum[4];
  __shared__ int poff[256];
  __shared__ int ptl[256 * KMAX];
  __shared__ int pv[256 * KMAX];
  __shared__ int npairs;
  __shared__ double obest[256];
  __shared__ int oidx[256];
  // XCD-aware: the workgroups of a head run on one XCD (its L2 holds the head's centroids)
  const int nitems = H * rg, per = (nitems + 7) >> 3;
  const int item = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (item >= nitems) return;
  const int h = item / rg, wg = item - h * rg;
  const int tid = threadIdx.x, l = tid & 63, g = l >> 4, c16 = l & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int cnt = min(nflag[h], N);
  const int nchunks = (cnt + 255) / 256;
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
  for (int chunk = wg; chunk < nchunks; chunk += rg) {
    // this chunk's tokens: wavefront w, block tb, column c16 -> local id 64w + 16tb + c16
    bf16x8_t xf[TB][KS];
    float kx[TB], U[TB];
    int tk[TB];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      const int idx = chunk * 256 + 64 * w + 16 * tb + c16;
      int tok = idx < cnt ? flags[(size_t)h * N + idx] : -1;
      tok = (unsigned)tok < (unsigned)N ? tok : -1;
      tk[tb] = tok;
      U[tb] = tok >= 0 ? flagu[(size_t)h * N + idx] : -INFINITY;
      if (U[tb] != U[tb]) U[tb] = INFINITY;  // NaN: every centroid is a candidate
      float xsq = 0.0f;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        uint4 raw = make_uint4(0u, 0u, 0u, 0u);
        if (tok >= 0) raw = *(const uint4*)(Xh + (size_t)tok * D + 32 * s + 8 * g);
        xf[tb][s] = __builtin_bit_cast(bf16x8_t, raw);
        asm volatile("" ::"v"(xf[tb][s]));  // loads complete here, not inside the tile loop
        const uint32_t q[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = __uint_as_float(q[e] << 16), hi = __uint_as_float(q[e] & 0xffff0000u);
          xsq = fmaf(lo, lo, fmaf(hi, hi, xsq));
        }
      }
      xsq += __shfl_xor(xsq, 16, 64);
      xsq += __shfl_xor(xsq, 32, 64);
      kx[tb] = KXC * sqrtf(xsq);
      asm volatile("" ::"v"(U[tb]));
      if (g == 0) {
        ccount[64 * w + 16 * tb + c16] = 0;
        ctok[64 * w + 16 * tb + c16] = tok;
      }
    }
    if (tid == 0) nover = 0;
    issue(0, 0);
    for (int t = 0; t < nt; ++t) {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();  // tile t landed everywhere; tile t-1 consumed
      if (t + 1 < nt) issue(t + 1, (t + 1) & 1);
      const int slot = t & 1;
      const bf16_t* W1 = &Wt[slot][0];
      const bf16_t* W2 = W1 + CT * D;
      const bf16_t* W3 = W2 + CT * D;
#pragma unroll
      for (int cb = 0; cb < CT / 16; ++cb) {
        f32x4_t ahi[TB], arest[TB];
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
          ahi[tb] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
          arest[tb] = ahi[tb];
        }
        const int rowo = (16 * cb + c16) * D;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const int co = rowo + 8 * ((4 * s + g) ^ swk);
          const bf16x8_t a1 = *(const bf16x8_t*)(W1 + co);
          const bf16x8_t a2 = *(const bf16x8_t*)(W2 + co);
          const bf16x8_t a3 = *(const bf16x8_t*)(W3 + co);
#pragma unroll
          for (int tb = 0; tb < TB; ++tb) {
            ahi[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, xf[tb][s], ahi[tb], 0, 0, 0);
            arest[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, xf[tb][s], arest[tb], 0, 0, 0);
            arest[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a3, xf[tb][s], arest[tb], 0, 0, 0);
          }
        }
        const int cl = 16 * cb + 4 * g;
        const float4 b4 = *(const float4*)(&Bt[slot][cl]);
        const float4 n4 = *(const float4*)(&Nt[slot][cl]);
        const float4 e4 = *(const float4*)(&Et[slot][cl]);
        const float bv[4] = {b4.x, b4.y, b4.z, b4.w}, nv[4] = {n4.x, n4.y, n4.z, n4.w},
                    ev[4] = {e4.x, e4.y, e4.z, e4.w};
        const int vb = t * CT + cl;
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
          bool cand[4], anyc = false;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float sc = fmaf(-2.0f, ahi[tb][r] + arest[tb][r], bv[r]);
            const float er = fmaf(kx[tb], nv[r], ev[r]);
            cand[r] = vb + r < C && !(sc - er > U[tb]);
            anyc |= cand[r];
          }
          if (__any(anyc)) {
            const int tl = 64 * w + 16 * tb + c16;
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (cand[r]) {
                const int pos = atomicAdd(&ccount[tl], 1);
                if (pos < KMAX) cv[tl * KMAX + pos] = vb + r;
              }
          }
        }
      }
    }
    __syncthreads();
    // pack the pairs (token, candidate) of tokens with 1..KMAX candidates;
    // list the others (more candidates) for the all-centroid pass
    {
      const int tl = tid;
      const int nc = ccount[tl];
      const bool packed = ctok[tl] >= 0 && nc >= 1 && nc <= KMAX;
      const int np = packed ? nc : 0;
      int inc = np;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(inc, o, 64);
        if (l >= o) inc += y;
      }
      if (l == 63) wsum[w] = inc;
      if (ctok[tl] >= 0 && !packed) over[atomicAdd(&nover, 1)] = tl;
      __syncthreads();
      int pre = 0;
      for (int q = 0; q < w; ++q) pre += wsum[q];
      const int start = pre + inc - np;
      poff[tl] = start;
      for (int j = 0; j < np; ++j) {
        ptl[start + j] = tl;
        pv[start + j] = cv[tl * KMAX + j];
      }
      if (tid == 255) npairs = start + np;
    }
    __syncthreads();
    // float64 scores of the packed pairs, PL lanes per pair (PE dimensions each)
    {
      const int lp = l / PL, sub = l % PL, np = npairs;
      for (int base = 0; base < np; base += 64) {
        double a[2];
        int pp[2];
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const int p = base + 32 * k + 8 * w + lp;
          pp[k] = p < np ? p : -1;
          a[k] = 0.0;
          if (p < np) {
            const int tok = ctok[ptl[p]];
            const bf16_t* xr = Xh + (size_t)tok * D + sub * PE;
            const double* wr = wh + (size_t)pv[p] * D + sub * PE;
#pragma unroll
            for (int e0 = 0; e0 < PE; e0 += 8) {
              const uint4 xu = *(const uint4*)(xr + e0);
              const uint32_t q[4] = {xu.x, xu.y, xu.z, xu.w};
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                a[k] = fma((double)__uint_as_float(q[e] << 16), wr[e0 + 2 * e], a[k]);
                a[k] = fma((double)__uint_as_float(q[e] & 0xffff0000u), wr[e0 + 2 * e + 1], a[k]);
              }
            }
          }
        }
#pragma unroll
        for (int k = 0; k < 2; ++k) {
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
      const int tl = over[i], tok = ctok[tl];
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
        obest[tl] = rbest[0];
        oidx[tl] = ridx[0];
      }
      __syncthreads();
    }
    // labels: the smallest float64 score, ties to the lowest id
    {
      const int tl = tid, tok = ctok[tl], nc = ccount[tl];
      if (tok >= 0) {
        double bb;
        int bi;
        if (nc >= 1 && nc <= KMAX) {
          bb = INFINITY;
          bi = 0x7fffffff;
          for (int j = 0; j < nc; ++j) {
            const int p = poff[tl] + j;
            const double sc = cs[p];
            const int v = pv[p];
            if (sc < bb || (sc == bb && v < bi)) {
              bb = sc;
              bi = v;
            }
          }
        } else {
          bb = obest[tl];
          bi = oidx[tl];
        }
        if (!isfinite(bb) || (unsigned)bi >= (unsigned)C) {
          raise_status(status, ST_NONFINITE);
          bi = 0;
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
  for (int r = o0 + j; r < o1; r += RL) {
    const int idx = p ? p[r] : r;
    if ((unsigned)idx < (unsigned)N) {
      const T* xr = Xh + (size_t)idx * D + c0;
#pragma unroll
      for (int c = 0; c < CW; ++c) acc[c] += (double)to_f(xr[c]);
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

template <typename T, int D>
static park_status kmeans_impl(const T* X, const double* Gbar, int H, int N, int C, int T_,
                               uint64_t seed, int side, const KmeansBufs& kb, int* status,
                               hipStream_t st) {
  constexpr bool fast = sizeof(T) == 2;  // bf16 points: MFMA fast path + float64 refine
  const size_t plane = (size_t)H * C * D;
  PARK_LAUNCH("kmeans_init", k_init_idx, dim3(H), dim3(1024), 0, st, N, C, seed, side, kb.init);
  PARK_LAUNCH("kmeans_seed", k_seed_centroids<T>, dim3(C, H), dim3(D), 0, st, X,
              (const int*)kb.init, N, D, C, kb.mu);
  // refine grid: persistent workgroups per head looping over 256-token chunks
  int rg = (1024 + H - 1) / H;
  const int max_tiles = (N + 255) / 256;
  rg = rg < 2 ? 2 : rg;
  rg = rg > max_tiles ? max_tiles : rg;
  for (int t = 0; t < T_; ++t) {
    const int nbm = (C + 15) / 16;
    PARK_LAUNCH("kmeans_prep", k_prep<D>, dim3(nbm, H), dim3(256), 0, st,
                (const double*)kb.mu, Gbar, C, kb.w, kb.b, fast ? kb.w3 : nullptr, plane, fast ? kb.b32 : nullptr, kmeans_cpad(C),
                fast ? kb.wn : nullptr,
                fast ? kb.eb : nullptr, kb.hmax, kb.nflag);
    if constexpr (fast) {
      if (C >= 512)
        PARK_LAUNCH("kmeans_assign_fast", (k_assign_fast<D, 2>), dim3((N + 255) / 256, H),
                    dim3(256), 0, st, (const bf16_t*)X, (const bf16_t*)kb.w3, plane,
                    (const float*)kb.b32, kmeans_cpad(C), (const float*)kb.wn, (const float*)kb.eb,
                    (const float*)kb.hmax, nbm, N, C, kb.labels, kb.flags, kb.flagu, kb.nflag);
      else
        PARK_LAUNCH("kmeans_assign_fast", (k_assign_fast<D, 3>), dim3((N + 255) / 256, H),
                    dim3(256), 0, st, (const bf16_t*)X, (const bf16_t*)kb.w3, plane,
                    (const float*)kb.b32, kmeans_cpad(C), (const float*)kb.wn, (const float*)kb.eb,
                    (const float*)kb.hmax, nbm, N, C, kb.labels, kb.flags, kb.flagu, kb.nflag);
      PARK_LAUNCH("kmeans_refine64", k_refine_cand<D>, dim3(8 * ((rg * H + 7) / 8)),
                  dim3(256), 0, st, (const bf16_t*)X, (const bf16_t*)kb.w3, plane,
                  (const float*)kb.b32, (const float*)kb.wn, (const float*)kb.eb, kmeans_cpad(C),
                  (const double*)kb.w, (const double*)kb.b, H, N, C, rg, (const int*)kb.flags,
                  (const float*)kb.flagu, (const int*)kb.nflag, kb.labels, status);
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
