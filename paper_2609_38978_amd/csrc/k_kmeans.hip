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
                                              double* __restrict__ wT, bf16_t* __restrict__ w3,
                                              size_t plane, float* __restrict__ b32,
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
      if (wT) wT[((size_t)h * D + a) * C + v0 + r] = acc[k];
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
      b32[(size_t)h * C + v0 + tid] = (float)s;
      wn[(size_t)h * C + v0 + tid] = fn;
      eb[(size_t)h * C + v0 + tid] = fe;
    }
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
// split into three bf16 parts, w = w1 + w2 + w3 + r, |r| <= 2^-24 (1+2^-7)|w|.
// All products are bf16 x bf16, exact in float.  x.w1 is accumulated over the
// D dimensions in one chain of v_mfma_f32_16x16x32_bf16, x.(w2 + w3), whose
// terms are 2^-8 smaller, in a second chain, and the two are added once.
// With delta = 2^-23 per addition inside an MFMA (any faithful rounding) and
// 2^-24 for the VALU roundings, the forward error of t^ = x.w is at most
//   et sum_a |x_a w_a|,  et = 2^-24 1.01 + (D+1) delta (1 + 2^-7)
//                            + 2^-8 1.01 (2D+1) delta + 2^-24 1.01,
// and with sum_a |x_a w_a| <= |x| |w_v|, the float roundings of b_v and of
// the score, and |s^_v| <= |b_v| + 2.01 |x| |w_v|:
//   |s^_v - s_v| <= E_v = Kx |w_v| + eb_v,
//   Kx = 1.1 (2 et + 2.01 2^-24) |x|,  eb_v = 1.1 * 2 * 2^-24 |b_v|
// (the factor 1.1 covers the rounding of |x| and of the bound itself).  A
// token is certified when, for its fast argmin v1, s^_v - E_v > s^_v1 + E_v1
// for every other v: then v1 is the exact argmin.  Otherwise (near-ties,
// exact ties) it is listed for the float64 refinement.
//
// Only scores within E_max = Kx max|w| + max eb of the running best can
// matter, so the per-score bookkeeping runs only when some lane of the
// wavefront holds such a score (a wave-uniform branch); a skipped score
// s^_v > ub + E_max has lower bound s^_v - E_v > ub, above the final best's
// upper bound.
//
// Workgroup = 256 tokens (4 wavefronts x 4 blocks of 16), centroid tiles of 64
// staged in LDS with the next tile prefetched into registers.  MFMA
// orientation: A = 16 centroids x 32 dims, B = 32 dims x 16 tokens, so lane l
// holds centroids 4(l/16)+r of token l%16.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <int D>
__global__ __launch_bounds__(256) void k_assign_fast(const bf16_t* __restrict__ X,
                                                     const bf16_t* __restrict__ w3, size_t plane,
                                                     const float* __restrict__ b32,
                                                     const float* __restrict__ wn,
                                                     const float* __restrict__ eb,
                                                     const float* __restrict__ bmax, int nbm,
                                                     int N, int C,
                                                     int* __restrict__ labels,
                                                     int* __restrict__ flags,
                                                     int* __restrict__ nflag) {
  constexpr int TB = 4, CT = 64, KS = D / 32, WROW = D + 8, CH = D / 8;
  constexpr int NL = CT * CH / 256;  // 16-byte chunks of each part per thread and tile
  constexpr float U24 = 5.9604645e-08f, DEL = 1.1920929e-07f;
  constexpr float ET = U24 * 1.01f + (D + 1) * DEL * 1.0079f + 0.00390625f * 1.01f * (2 * D + 1) * DEL +
                       U24 * 1.01f;
  constexpr float KXC = 1.1f * (2.0f * ET + 2.01f * U24) * 1.0001f;
  __shared__ __attribute__((aligned(16))) bf16_t W1[CT * WROW];
  __shared__ __attribute__((aligned(16))) bf16_t W2[CT * WROW];
  __shared__ __attribute__((aligned(16))) bf16_t W3[CT * WROW];
  __shared__ __attribute__((aligned(16))) float bs[CT];
  __shared__ __attribute__((aligned(16))) float ns[CT];
  __shared__ __attribute__((aligned(16))) float es[CT];
  const int h = blockIdx.y, tid = threadIdx.x, w = tid >> 6, l = tid & 63, g = l >> 4,
            c16 = l & 15;
  const int t0 = blockIdx.x * 256 + w * 64;
  const bf16_t* Xh = X + (size_t)h * N * D;
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
  __shared__ float mx_s[2];
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
  __syncthreads();
  const float nmax = mx_s[0], ebmax = mx_s[1];
  float kx[TB], emax[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    float xs = xsq[tb] + __shfl_xor(xsq[tb], 16, 64);
    xs += __shfl_xor(xs, 32, 64);
    kx[tb] = KXC * sqrtf(xs);
    emax[tb] = fmaf(kx[tb], nmax, ebmax) * 1.0001f;
  }
  // per token and lane: best fast score, its index, its upper bound, the
  // lowest lower bound among the lane's other centroids, and the threshold
  // above which a score cannot matter
  float best[TB], ub[TB], lo2[TB], thr[TB];
  int bidx[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    best[tb] = INFINITY;
    ub[tb] = INFINITY;
    lo2[tb] = INFINITY;
    thr[tb] = INFINITY;
    bidx[tb] = 0;
  }
  const bf16_t* P1 = w3 + (size_t)h * C * D;
  const bf16_t* P2 = P1 + plane;
  const bf16_t* P3 = P2 + plane;
  const f32x4_t zero = {0.0f, 0.0f, 0.0f, 0.0f};
  uint4 r1[NL], r2[NL], r3[NL];
  float rb = INFINITY, rn = 0.0f, re = 0.0f;
  // prefetch tile 0
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int e = tid + 256 * i, r = e / CH, ch = e % CH;
    uint4 v1 = make_uint4(0u, 0u, 0u, 0u), v2 = v1, v3 = v1;
    if (r < C) {
      const size_t o = (size_t)r * D + 8 * ch;
      v1 = *(const uint4*)(P1 + o);
      v2 = *(const uint4*)(P2 + o);
      v3 = *(const uint4*)(P3 + o);
    }
    r1[i] = v1;
    r2[i] = v2;
    r3[i] = v3;
  }
  if (tid < CT && tid < C) {
    rb = b32[(size_t)h * C + tid];
    rn = wn[(size_t)h * C + tid];
    re = eb[(size_t)h * C + tid];
  }
  for (int c0 = 0; c0 < C; c0 += CT) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int e = tid + 256 * i, r = e / CH, ch = e % CH;
      *(uint4*)(W1 + r * WROW + 8 * ch) = r1[i];
      *(uint4*)(W2 + r * WROW + 8 * ch) = r2[i];
      *(uint4*)(W3 + r * WROW + 8 * ch) = r3[i];
    }
    if (tid < CT) {
      bs[tid] = rb;
      ns[tid] = rn;
      es[tid] = re;
    }
    __syncthreads();
    const int c1 = c0 + CT;
    if (c1 < C) {  // prefetch the next tile while this one is scored
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        const int e = tid + 256 * i, r = e / CH, ch = e % CH;
        uint4 v1 = make_uint4(0u, 0u, 0u, 0u), v2 = v1, v3 = v1;
        if (c1 + r < C) {
          const size_t o = (size_t)(c1 + r) * D + 8 * ch;
          v1 = *(const uint4*)(P1 + o);
          v2 = *(const uint4*)(P2 + o);
          v3 = *(const uint4*)(P3 + o);
        }
        r1[i] = v1;
        r2[i] = v2;
        r3[i] = v3;
      }
      rb = INFINITY;
      rn = 0.0f;
      re = 0.0f;
      if (tid < CT && c1 + tid < C) {
        rb = b32[(size_t)h * C + c1 + tid];
        rn = wn[(size_t)h * C + c1 + tid];
        re = eb[(size_t)h * C + c1 + tid];
      }
    }
#pragma unroll
    for (int cb = 0; cb < CT / 16; ++cb) {
      f32x4_t ahi[TB], arest[TB];
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        ahi[tb] = zero;
        arest[tb] = zero;
      }
      const int rowo = (16 * cb + c16) * WROW + 8 * g;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const bf16x8_t a1 = *(const bf16x8_t*)(W1 + rowo + 32 * s);
        const bf16x8_t a2 = *(const bf16x8_t*)(W2 + rowo + 32 * s);
        const bf16x8_t a3 = *(const bf16x8_t*)(W3 + rowo + 32 * s);
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
          ahi[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, xf[tb][s], ahi[tb], 0, 0, 0);
          arest[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a2, xf[tb][s], arest[tb], 0, 0, 0);
          arest[tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a3, xf[tb][s], arest[tb], 0, 0, 0);
        }
      }
      const float4 b4 = *(const float4*)(bs + 16 * cb + 4 * g);
      const float bv[4] = {b4.x, b4.y, b4.z, b4.w};
      float sc[TB][4];
      bool hit = false;
#pragma unroll
      for (int tb = 0; tb < TB; ++tb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          sc[tb][r] = fmaf(-2.0f, ahi[tb][r] + arest[tb][r], bv[r]);
          hit |= !(sc[tb][r] > thr[tb]);
        }
      if (__any(hit)) {
        const float4 n4 = *(const float4*)(ns + 16 * cb + 4 * g);
        const float4 e4 = *(const float4*)(es + 16 * cb + 4 * g);
        const float nv[4] = {n4.x, n4.y, n4.z, n4.w};
        const float ev[4] = {e4.x, e4.y, e4.z, e4.w};
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float x = sc[tb][r];
            const float e = fmaf(kx[tb], nv[r], ev[r]);
            if (x < best[tb]) {
              lo2[tb] = fminf(lo2[tb], 2.0f * best[tb] - ub[tb]);  // old best joins the others
              best[tb] = x;
              ub[tb] = x + e;
              bidx[tb] = c0 + 16 * cb + 4 * g + r;
            } else {
              lo2[tb] = fminf(lo2[tb], x - e);
            }
          }
          thr[tb] = ub[tb] + emax[tb];
        }
      }
    }
  }
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    // merge over the four lane groups holding this token
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float ob = __shfl_xor(best[tb], o, 64), ou = __shfl_xor(ub[tb], o, 64);
      const float ol = __shfl_xor(lo2[tb], o, 64);
      const int oi = __shfl_xor(bidx[tb], o, 64);
      if (ob < best[tb] || (ob == best[tb] && oi < bidx[tb])) {
        lo2[tb] = fminf(fminf(lo2[tb], ol), 2.0f * best[tb] - ub[tb]);
        best[tb] = ob;
        ub[tb] = ou;
        bidx[tb] = oi;
      } else {
        lo2[tb] = fminf(fminf(lo2[tb], ol), 2.0f * ob - ou);
      }
    }
    const int tok = t0 + 16 * tb + c16;
    if (g == 0 && tok < N) {
      const bool ok = isfinite(best[tb]) && isfinite(ub[tb]) && (lo2[tb] > ub[tb]);
      if (ok) {
        labels[(size_t)h * N + tok] = bidx[tb];
      } else {
        const int slot = atomicAdd(nflag + h, 1);
        flags[(size_t)h * N + slot] = tok;
      }
    }
  }
}

// Float64 assignment of the tokens the fast path could not certify: 16 listed
// tokens per workgroup, the centroids split over the four wavefronts (one
// centroid per lane, w read transposed so loads are coalesced), the exact
// minimum (ties to the lowest id) reduced across lanes and wavefronts.
template <typename T, int D>
__global__ __launch_bounds__(256) void k_refine(const T* __restrict__ X,
                                                const double* __restrict__ wT,
                                                const double* __restrict__ b, int N, int C,
                                                const int* __restrict__ flags,
                                                const int* __restrict__ nflag,
                                                int* __restrict__ labels, int* status) {
  constexpr int TT = 16;
  __shared__ double xs[TT][D];
  __shared__ double rs[4][TT];
  __shared__ int ri[4][TT];
  __shared__ int tok_s[TT];
  const int h = blockIdx.y, tid = threadIdx.x, wv = tid >> 6, l = tid & 63;
  const int cnt = min(nflag[h], N);
  const double* wh = wT + (size_t)h * D * C;
  const double* bh = b + (size_t)h * C;
  const int cpw = ((C + 3) / 4 + 63) / 64 * 64;  // centroids per wavefront
  const int v_begin = wv * cpw, v_end = min(C, v_begin + cpw);
  for (int t0 = blockIdx.x * TT; t0 < cnt; t0 += gridDim.x * TT) {
    __syncthreads();
    if (tid < TT) {
      const int tok = t0 + tid < cnt ? flags[(size_t)h * N + t0 + tid] : -1;
      tok_s[tid] = ((unsigned)tok < (unsigned)N) ? tok : -1;
    }
    __syncthreads();
    for (int e = tid; e < TT * D; e += 256) {
      const int t = e / D, a = e % D;
      const int tok = tok_s[t];
      xs[t][a] = tok >= 0 ? (double)to_f(X[((size_t)h * N + tok) * D + a]) : 0.0;
    }
    __syncthreads();
    double best[TT];
    int bidx[TT];
#pragma unroll
    for (int t = 0; t < TT; ++t) {
      best[t] = INFINITY;
      bidx[t] = 0x7fffffff;
    }
    for (int v0 = v_begin; v0 < v_end; v0 += 64) {
      const int v = v0 + l;
      if (v < v_end) {
        double acc[TT];
#pragma unroll
        for (int t = 0; t < TT; ++t) acc[t] = 0.0;
        for (int a0 = 0; a0 < D; a0 += 16) {
          double wa[16];
#pragma unroll
          for (int q = 0; q < 16; ++q) wa[q] = wh[(size_t)(a0 + q) * C + v];  // 16 loads in flight
#pragma unroll
          for (int q = 0; q < 16; ++q)
#pragma unroll
            for (int t = 0; t < TT; ++t) acc[t] = fma(xs[t][a0 + q], wa[q], acc[t]);
        }
        const double bv = bh[v];
#pragma unroll
        for (int t = 0; t < TT; ++t) {
          const double sc = fma(-2.0, acc[t], bv);
          if (sc < best[t]) {
            best[t] = sc;
            bidx[t] = v;
          }
        }
      }
    }
#pragma unroll
    for (int t = 0; t < TT; ++t) {
      double bb = best[t];
      int bi = bidx[t];
      for (int o = 32; o > 0; o >>= 1) {
        const double ob = __shfl_xor(bb, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (ob < bb || (ob == bb && oi < bi)) {
          bb = ob;
          bi = oi;
        }
      }
      if (l == 0) {
        rs[wv][t] = bb;
        ri[wv][t] = bi;
      }
    }
    __syncthreads();
    if (tid < TT && tok_s[tid] >= 0) {
      double bb = rs[0][tid];
      int bi = ri[0][tid];
      for (int q = 1; q < 4; ++q)
        if (rs[q][tid] < bb || (rs[q][tid] == bb && ri[q][tid] < bi)) {
          bb = rs[q][tid];
          bi = ri[q][tid];
        }
      if (!isfinite(bb) || bi >= C) {
        raise_status(status, ST_NONFINITE);
        bi = 0;
      }
      labels[(size_t)h * N + tok_s[tid]] = bi;
    }
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
  // refine grid: persistent workgroups per head looping over 16-token tiles
  int rg = (2048 + H - 1) / H;
  const int max_tiles = (N + 15) / 16;
  rg = rg < 2 ? 2 : rg;
  rg = rg > max_tiles ? max_tiles : rg;
  for (int t = 0; t < T_; ++t) {
    const int nbm = (C + 15) / 16;
    PARK_LAUNCH("kmeans_prep", k_prep<D>, dim3(nbm, H), dim3(256), 0, st,
                (const double*)kb.mu, Gbar, C, kb.w, kb.b, fast ? kb.wT : nullptr,
                fast ? kb.w3 : nullptr, plane, fast ? kb.b32 : nullptr, fast ? kb.wn : nullptr,
                fast ? kb.eb : nullptr, kb.hmax, kb.nflag);
    if constexpr (fast) {
      PARK_LAUNCH("kmeans_assign_fast", k_assign_fast<D>, dim3((N + 255) / 256, H), dim3(256), 0,
                  st, (const bf16_t*)X, (const bf16_t*)kb.w3, plane, (const float*)kb.b32,
                  (const float*)kb.wn, (const float*)kb.eb, (const float*)kb.hmax, nbm, N, C,
                  kb.labels, kb.flags, kb.nflag);
      PARK_LAUNCH("kmeans_refine64", (k_refine<T, D>), dim3(rg, H), dim3(256), 0, st, X,
                  (const double*)kb.wT, (const double*)kb.b, N, C, (const int*)kb.flags,
                  (const int*)kb.nflag, kb.labels, status);
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
