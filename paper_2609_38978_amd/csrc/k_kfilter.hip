// Exact candidate filter for the k-means assignments after the first
// (Sec. 5.2, Alg. 3: T rounds of assignment and update).
//
// Round t >= 1 starts from the labels z of round t-1 (tokens of a cluster are
// contiguous in the order of the counting sort that fed the update) and the
// updated centroids mu.  All distances are in the metric of the side:
// D(x, y)^2 = (x - y)^T Gbar (x - y) for the keys (QRKC, App. D.2), Euclidean
// (Gbar = I) for the queries.  For a token x of cluster a and any centroid v,
// the triangle inequality gives D(x, mu_v) >= D(mu_a, mu_v) - D(x, mu_a), so
// with R_a >= max over the cluster's tokens of D(x, mu_a):
//   D(mu_a, mu_v) > 2 R_a  =>  D(x, mu_v) > D(x, mu_a)  for every x in a,
// i.e. v is strictly farther than mu_a and can be neither the argmin nor tie
// with it.  The candidate set S_a = {v : D(mu_a, mu_v) <= 2 R_a} therefore
// holds every minimiser of every token of a, and the argmin over any superset
// of S_a (lowest id on ties) is the exact argmin over all centroids.
//
// Everything here only has to be conservative: R_a is rounded up and
// D(mu_a, mu_v) rounded down by proven bounds, so rounding can only keep a
// centroid that the exact test would drop.
//   k_gsplit       Gbar in two bf16 parts and its largest absolute row sum
//   k_xnorm        x^T Gbar x per token, plus a bound of its error
//   k_radius       R_a^2 per cluster (float64 from the bounds above)
//   k_cand         the bit matrix of S_a on bf16 MFMA over split operands
//   k_tile_union   per tile of sorted tokens, the union of its clusters' S_a
//   k_assign_cand  the certified bf16-MFMA assignment of each tile of sorted
//                  tokens against the union of its clusters' candidate sets
//   k_refine_union float64 labels of the tokens it cannot certify, against
//                  the same union
#include "common.h"
#include "kernels.h"

namespace park {

typedef __bf16 kf_bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 kf_bf16x2_t __attribute__((ext_vector_type(2)));
typedef float kf_f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ void kf_dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ uint32_t kf_lds_addr(const void* p) {
  return (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)p;
}
template <int D>
__device__ __forceinline__ int kf_swz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
template <int N>
__device__ __forceinline__ void kf_wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// ------------------------------------------------------------ Gbar split
// g2[part][h][D][D] = the two leading bf16 parts of Gbar (residual <= 2^-16
// 1.01 |Gbar_ij|); gmax[h] = max_i sum_j |Gbar_ij| (rounded up), which bounds
// the spectral radius of |Gbar|.  One workgroup per head.
template <int D>
__global__ __launch_bounds__(256) void k_gsplit(const double* __restrict__ Gbar,
                                                bf16_t* __restrict__ g2, size_t plane,
                                                double* __restrict__ gmax) {
  __shared__ double rs[D];
  const int h = blockIdx.x, tid = threadIdx.x;
  const double* G = Gbar + (size_t)h * D * D;
  for (int e = tid; e < D * D; e += 256) {
    const double g = G[e];
    const bf16_t p1 = f2bf((float)g);
    const bf16_t p2 = f2bf((float)(g - (double)bf2f(p1)));
    g2[(size_t)h * D * D + e] = p1;
    g2[plane + (size_t)h * D * D + e] = p2;
  }
  if (tid < D) {
    double s = 0.0;
    for (int j = 0; j < D; ++j) s += fabs(G[(size_t)tid * D + j]);
    rs[tid] = s;
  }
  __syncthreads();
  if (tid == 0) {
    double m = 0.0;
    for (int i = 0; i < D; ++i) m = fmax(m, rs[i]);
    gmax[h] = m * (1.0 + 1e-12);
  }
}

// ------------------------------------------------------------ token norms
// xn[h][j] >= x_j^T Gbar x_j (Euclidean side: |x_j|^2, exact up to float64
// rounding).  QRKC: y = Gbar x on bf16 MFMA with Gbar in two parts (rows of
// Gbar as the A operand, 32 tokens of a wavefront as B), then x . y in float64.
// The products are exact; with 2^-23 per MFMA addition (a chain of 2D
// products) and the split residual, |y^_b - y_b| <= et sum_a |Gbar_ba x_a|,
// et = 2^-16 1.01 + (2D + 1) 2^-23 1.0079 + 2^-24, and |x|^T |Gbar| |x| <=
// gmax |x|^2, so xn = x . y^ + 1.01 et gmax |x|^2 is an upper bound.
// QRKC: a few workgroups per head, each keeping Gbar's two parts in LDS
// (16-byte chunks of a row XOR-swizzled by the row, so the 16 rows of a
// quarter-wavefront's operand read fall in distinct banks) and looping over
// chunks of 512 tokens (4 wavefronts x 4 blocks of 32).
template <int D>
__global__ __launch_bounds__(256) void k_xnorm_euclid(const bf16_t* __restrict__ X, int N,
                                                      double* __restrict__ xn) {
  // |x|^2 in float64 (the squares of bf16 values are exact): 16 lanes per
  // token, four tokens per step
  constexpr int PE = D / 16;
  const int h = blockIdx.y, tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  const int g = l >> 4, sub = l & 15;
  for (int k = 0; k < 32; ++k) {
    const int t = blockIdx.x * 512 + w * 128 + 4 * k + g;
    const bool ok = t < N;
    const bf16_t* r = X + ((size_t)h * N + (ok ? t : 0)) * D + PE * sub;
    uint32_t q[PE / 2];
    if constexpr (PE == 8) {
      const uint4 raw = ok ? *(const uint4*)r : make_uint4(0u, 0u, 0u, 0u);
      q[0] = raw.x; q[1] = raw.y; q[2] = raw.z; q[3] = raw.w;
    } else {
      const uint2 raw = ok ? *(const uint2*)r : make_uint2(0u, 0u);
      q[0] = raw.x; q[1] = raw.y;
    }
    double s2 = 0.0;
#pragma unroll
    for (int e = 0; e < PE / 2; ++e) {
      const double x0 = (double)__uint_as_float(q[e] << 16);
      const double x1 = (double)__uint_as_float(q[e] & 0xffff0000u);
      s2 = fma(x0, x0, fma(x1, x1, s2));
    }
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) s2 += __shfl_xor(s2, o, 64);
    if (sub == 0 && ok) xn[(size_t)h * N + t] = s2 * (1.0 + 1e-13);
  }
}

template <int D>
__global__ __launch_bounds__(256) void k_xnorm(const bf16_t* __restrict__ X,
                                               const bf16_t* __restrict__ g2, size_t plane,
                                               const double* __restrict__ gmax, int N,
                                               double* __restrict__ xn) {
  constexpr int KS = D / 16, CPR = D / 8;
  const int h = blockIdx.y, tid = threadIdx.x, l = tid & 63, hf = l >> 5, c32 = l & 31;
  const int w = tid >> 6;
  const int nchunk = (N + 511) / 512;
  __shared__ __attribute__((aligned(16))) bf16_t Gs[2 * D * D];
  {
    const bf16_t* G1 = g2 + (size_t)h * D * D;
    for (int e = tid; e < 2 * D * CPR; e += 256) {
      const int part = e / (D * CPR), rem = e % (D * CPR), row = rem / CPR, c = rem % CPR;
      const uint4 v = *(const uint4*)(G1 + part * plane + (size_t)row * D + 8 * c);
      *(uint4*)(Gs + part * D * D + row * D + 8 * (c ^ kf_swz<D>(row))) = v;
    }
  }
  __syncthreads();
  const bf16_t* L1 = Gs;
  const bf16_t* L2 = Gs + D * D;
  constexpr double ET = 1.52587890625e-05 * 1.01 + (2 * D + 1) * 1.1920928955078125e-07 * 1.0079 +
                        5.9604644775390625e-08;
  const double gm = gmax[h];
  for (int ck = blockIdx.x; ck < nchunk; ck += gridDim.x)
    for (int tb = 0; tb < 4; ++tb) {
      const int t = ck * 512 + w * 128 + 32 * tb + c32;
      const bool ok = t < N;
      const bf16_t* r = X + ((size_t)h * N + (ok ? t : 0)) * D;
      kf_bf16x8_t xf[KS];
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        uint4 raw = make_uint4(0u, 0u, 0u, 0u);
        if (ok) raw = *(const uint4*)(r + 16 * s + 8 * hf);
        xf[s] = __builtin_bit_cast(kf_bf16x8_t, raw);
      }
      double acc64 = 0.0, xx = 0.0;
#pragma unroll
      for (int rt = 0; rt < D / 32; ++rt) {
        kf_f32x16_t y;
#pragma unroll
        for (int q = 0; q < 16; ++q) y[q] = 0.0f;
        const int row = 32 * rt + c32, ro = row * D, sw = kf_swz<D>(row);
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const kf_bf16x8_t a2 = *(const kf_bf16x8_t*)(L2 + ro + 8 * ((2 * s + hf) ^ sw));
          y = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, xf[s], y, 0, 0, 0);
        }
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const kf_bf16x8_t a1 = *(const kf_bf16x8_t*)(L1 + ro + 8 * ((2 * s + hf) ^ sw));
          y = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, xf[s], y, 0, 0, 0);
        }
        // lane holds y at rows 32 rt + 8 b + 4 hf + r of token c32
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const uint2 raw = ok ? *(const uint2*)(r + 32 * rt + 8 * b + 4 * hf) : make_uint2(0u, 0u);
          const float xv[4] = {__uint_as_float(raw.x << 16), __uint_as_float(raw.x & 0xffff0000u),
                               __uint_as_float(raw.y << 16), __uint_as_float(raw.y & 0xffff0000u)};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            acc64 = fma((double)xv[q], (double)y[4 * b + q], acc64);
            xx = fma((double)xv[q], (double)xv[q], xx);
          }
        }
      }
      acc64 += __shfl_xor(acc64, 32, 64);
      xx += __shfl_xor(xx, 32, 64);
      if (hf == 0 && ok) xn[(size_t)h * N + t] = acc64 + 1.01 * ET * gm * xx;
    }
}

// ------------------------------------------------------------ cluster radii
// r2[h][a] >= max over the tokens x of cluster a (sorted positions
// offsets[a] .. offsets[a+1]) of D(x, mu_a)^2 = x^T Gbar x + b_a - 2 x . w_a,
// from the upper bound xn and float64 b, w (their rounding is covered by a
// relative margin); -1 for an empty cluster.  One wavefront per cluster, one
// lane per token.
template <int D>
__global__ __launch_bounds__(256) void k_radius(const bf16_t* __restrict__ X,
                                                const int* __restrict__ perm,
                                                const int* __restrict__ offsets,
                                                const double* __restrict__ xn,
                                                const double* __restrict__ w,
                                                const double* __restrict__ b, int N, int C,
                                                double* __restrict__ r2) {
  // a wavefront per cluster; 16 lanes per token (each 8 or 4 dimensions of a
  // contiguous row), four tokens per step
  constexpr int PE = D / 16;
  const int h = blockIdx.y, tid = threadIdx.x, l = tid & 63, g = l >> 4, sub = l & 15;
  const int a = blockIdx.x * 4 + (tid >> 6);
  if (a >= C) return;
  const int* off = offsets + (size_t)h * (C + 1);
  const int o0 = min(max(off[a], 0), N), o1 = min(max(off[a + 1], o0), N);
  if (o1 <= o0) {
    if (l == 0) r2[(size_t)h * C + a] = -1.0;
    return;
  }
  double wa[PE];
  const double* wr = w + ((size_t)h * C + a) * D + PE * sub;
#pragma unroll
  for (int e = 0; e < PE; ++e) wa[e] = wr[e];
  const double ba = b[(size_t)h * C + a];
  const int* ph = perm + (size_t)h * N;
  // D^2 rounded up: float64 rounding of x . w_a (D terms), of b_a (computed
  // the same way) and of the sum stays below 1e-12 of the magnitudes involved
  double mx = 0.0;
  for (int base = o0; base < o1; base += 64) {
    // the cluster's token ids, 64 at a time, one per lane
    const int n = min(64, o1 - base);
    int mytok = l < n ? ph[base + l] : -1;
    mytok = (unsigned)mytok < (unsigned)N ? mytok : -1;
    for (int s0 = 0; s0 < n; s0 += 16) {
      // four rows per lane group in flight
      int tk[4];
      uint32_t q[4][PE / 2];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int idx = s0 + 4 * u + g;
        tk[u] = __shfl(mytok, idx, 64);
        tk[u] = idx < n ? tk[u] : -1;
        const bf16_t* xr = X + ((size_t)h * N + (tk[u] >= 0 ? tk[u] : 0)) * D + PE * sub;
        if constexpr (PE == 8) {
          const uint4 raw = tk[u] >= 0 ? *(const uint4*)xr : make_uint4(0u, 0u, 0u, 0u);
          q[u][0] = raw.x; q[u][1] = raw.y; q[u][2] = raw.z; q[u][3] = raw.w;
        } else {
          const uint2 raw = tk[u] >= 0 ? *(const uint2*)xr : make_uint2(0u, 0u);
          q[u][0] = raw.x; q[u][1] = raw.y;
        }
      }
      double xv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) xv[u] = tk[u] >= 0 ? xn[(size_t)h * N + tk[u]] : 0.0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        double dot = 0.0, dab = 0.0;
#pragma unroll
        for (int e = 0; e < PE / 2; ++e) {
          const double x0 = (double)__uint_as_float(q[u][e] << 16);
          const double x1 = (double)__uint_as_float(q[u][e] & 0xffff0000u);
          dot = fma(x0, wa[2 * e], dot);
          dot = fma(x1, wa[2 * e + 1], dot);
          dab = fma(fabs(x0), fabs(wa[2 * e]), dab);
          dab = fma(fabs(x1), fabs(wa[2 * e + 1]), dab);
        }
#pragma unroll
        for (int o = 8; o > 0; o >>= 1) {
          dot += __shfl_xor(dot, o, 64);
          dab += __shfl_xor(dab, o, 64);
        }
        if (tk[u] >= 0)
          mx = fmax(mx, xv[u] + ba - 2.0 * dot + 1e-12 * (xv[u] + fabs(ba) + 2.0 * dab));
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o, 64));
  if (l == 0) r2[(size_t)h * C + a] = mx;
}

// ------------------------------------------------------------ candidate sets
// cand[h][a][word] bit v: v is in S_a.  Per pair, t = mu_a . w_v on bf16 MFMA
// from the two leading parts of each (m1 w1 + m1 w2 + m2 w1; every product
// exact, the dropped parts below 3.2 2^-16 |mu_a| |w_v| elementwise, 2^-23
// per addition over 3D products), |t^ - t| <= ec |mu_a| |w_v| with
// ec = 3.2 2^-16 + (3D + 1) 2^-23 1.02, and, with the float64 rounding of b
// and of the sum below 1e-12 of the magnitudes involved,
//   D(mu_a, mu_v)^2 >= lo = b_a + b_v - 2 t^ - 2 ec |mu_a| |w_v|
//                           - 1e-12 (|b_a| + |b_v| + |mu_a| |w_a| + |mu_v| |w_v|).
// v is dropped from S_a when lo > 4 r2[a] (1 + 1e-9) + 1e-9 (|b_a| + |b_v|):
// then its exact score exceeds mu_a's by far more than the float64 scores
// can err, so the float64 argmin never needs it either.  v = a is always
// kept; rows of empty clusters (r2 < 0) are all zero.  The distance is
// symmetric (t^ bounds mu_v . w_a = mu_a . w_v as well), so each pair of
// tiles is computed once: the pair (A, V) with V >= A writes word V of the
// rows of A (test with r2[a]) and, for V > A, word A of the rows of V (test
// with r2[v], bits gathered across lanes by ballots).  Every word of every
// row has exactly one writer.
// Workgroup: one 32-cluster tile A (the B operand: mu parts, in LDS for the
// four wavefronts) and a group of 16 centroid tiles (the A operand: w parts,
// four per wavefront).
template <int D>
__global__ __launch_bounds__(256, 2) void k_cand(const bf16_t* __restrict__ m2, size_t mplane,
                                                 const bf16_t* __restrict__ w3, size_t wplane,
                                                 const float* __restrict__ mn,
                                                 const float* __restrict__ wn, int Cpad,
                                                 const double* __restrict__ b,
                                                 const double* __restrict__ r2, int C,
                                                 uint32_t* __restrict__ cand) {
  constexpr int KS = D / 16, CPR = D / 8;
  constexpr double EC = 3.2 * 1.52587890625e-05 + (3 * D + 1) * 1.1920928955078125e-07 * 1.02;
  const int h = blockIdx.y, tid = threadIdx.x, l = tid & 63, hf = l >> 5, c32 = l & 31;
  const int w = tid >> 6;
  const int at = blockIdx.x, a0 = at * 32, a = a0 + c32;
  const int nvt = (C + 31) / 32;
  const int vt_beg = max(at, (int)blockIdx.z * 16), vt_end = min(nvt, (int)(blockIdx.z + 1) * 16);
  if (vt_beg >= vt_end) return;  // the transposed writes of other tile pairs cover these
  const bool aval = a < C;
  const int ar = aval ? a : C - 1;
  // the tile's centroids in two bf16 parts, 16-byte chunks swizzled by the row
  __shared__ __attribute__((aligned(16))) bf16_t Ms[2 * 32 * D];
  for (int e = tid; e < 2 * 32 * CPR; e += 256) {
    const int part = e / (32 * CPR), rem = e % (32 * CPR), row = rem / CPR, c = rem % CPR;
    const int rr = min(a0 + row, C - 1);
    const uint4 v = *(const uint4*)(m2 + part * mplane + ((size_t)h * C + rr) * D + 8 * c);
    *(uint4*)(Ms + part * 32 * D + row * D + 8 * (c ^ kf_swz<D>(row))) = v;
  }
  const double ra = aval ? r2[(size_t)h * C + a] : -1.0;
  const double ba = b[(size_t)h * C + ar];
  const double man = (double)mn[(size_t)h * C + ar];
  const double ana = man * (double)wn[(size_t)h * Cpad + ar];
  uint32_t* crow = cand + ((size_t)h * C + ar) * 64;
  // b_v, |w_v|, |mu_v| |w_v| and r2[v] of this workgroup's 16 centroid tiles
  __shared__ double vb_s[512], vw_s[512], vm_s[512], vr_s[512];
  for (int e = tid; e < 512; e += 256) {
    const int v = (int)blockIdx.z * 512 + e, vr = min(v, C - 1);
    const double wv = (double)wn[(size_t)h * Cpad + vr];
    vb_s[e] = b[(size_t)h * C + vr];
    vw_s[e] = wv;
    vm_s[e] = (double)mn[(size_t)h * C + vr] * wv;
    vr_s[e] = v < C ? r2[(size_t)h * C + v] : -1.0;
  }
  __syncthreads();
  const int rowo = c32 * D, swk = kf_swz<D>(c32);
  const bf16_t* M1 = Ms;
  const bf16_t* M2 = Ms + 32 * D;
  for (int vt = vt_beg + w; vt < vt_end; vt += 4) {
    const int v0 = vt * 32;
    kf_bf16x8_t w1f[KS], w2f[KS];
    {
      const int vr = min(v0 + c32, C - 1);
      const bf16_t* W1 = w3 + ((size_t)h * C + vr) * D + 8 * hf;
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2) {
        w1f[s2] = __builtin_bit_cast(kf_bf16x8_t, *(const uint4*)(W1 + 16 * s2));
        w2f[s2] = __builtin_bit_cast(kf_bf16x8_t, *(const uint4*)(W1 + wplane + 16 * s2));
      }
    }

    kf_f32x16_t acc;
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[q] = 0.0f;
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) {
      const kf_bf16x8_t m1 = *(const kf_bf16x8_t*)(M1 + rowo + 8 * ((2 * s2 + hf) ^ swk));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w2f[s2], m1, acc, 0, 0, 0);
    }
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) {
      const int co = rowo + 8 * ((2 * s2 + hf) ^ swk);
      const kf_bf16x8_t m1 = *(const kf_bf16x8_t*)(M1 + co);
      const kf_bf16x8_t mm2 = *(const kf_bf16x8_t*)(M2 + co);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w1f[s2], mm2, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w1f[s2], m1, acc, 0, 0, 0);
    }
    // lane: pairs (a, v0 + 8 bq + 4 hf + r) for q = 4 bq + r
    uint32_t bits = 0u;
    uint32_t tw[16];  // transposed: bit (a, v) of row v, by q
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int vi = 8 * (q >> 2) + 4 * hf + (q & 3), v = v0 + vi;
      const int li = v0 - (int)blockIdx.z * 512 + vi;
      const double bv = vb_s[li];
      const double t = (double)acc[q];
      const double lo = ba + bv - 2.0 * t - 2.0 * EC * man * vw_s[li] -
                        1e-12 * (fabs(ba) + fabs(bv) + ana + vm_s[li]);
      const double gap = 1e-9 * (fabs(ba) + fabs(bv));
      const bool inr = v < C && aval;
      const bool keep = inr && ra >= 0.0 && (v == a || !(lo > 4.0 * ra * (1.0 + 1e-9) + gap));
      const double rv = vr_s[li];
      const bool keept = inr && rv >= 0.0 && !(lo > 4.0 * rv * (1.0 + 1e-9) + gap);
      bits |= keep ? (1u << vi) : 0u;
      const unsigned long long bal = __ballot(keept);
      tw[q] = (uint32_t)(hf == 0 ? bal : (bal >> 32));
    }
    bits |= (uint32_t)__shfl_xor((int)bits, 32, 64);
    if (hf == 0 && aval) crow[vt] = bits;
    if (vt > at) {
      // word `at` of the rows v of this tile: lane (hf, r, bq) with c32 =
      // 8 bq + r (r < 4) writes row v0 + 8 bq + 4 hf + r
      const int r = c32 & 7, bq = c32 >> 3;
      if (r < 4) {
        const int vi = 8 * bq + 4 * hf + r;
        uint32_t word = 0u;
#pragma unroll
        for (int q = 0; q < 16; ++q) word = (q == 4 * bq + r) ? tw[q] : word;
        if (v0 + vi < C) cand[((size_t)h * C + v0 + vi) * 64 + at] = word;
      }
    }
  }
}

// ------------------------------------------------------------ tile unions
// The union of the candidate sets of the clusters a tile of kmeans_tile
// sorted positions spans (from the cluster of its first position to that of
// its last, previous labels): 64 bit words and the first cluster per tile,
// built once per round so that the assignment starts from one load.  One
// wavefront per tile (lane = bit word).
__global__ __launch_bounds__(256) void k_tile_union(const int* __restrict__ perm,
                                                    const int* __restrict__ labels,
                                                    const uint32_t* __restrict__ cand, int H,
                                                    int N, int C, int NT,
                                                    uint32_t* __restrict__ tun,
                                                    int* __restrict__ talo) {
  const int wv = (int)blockIdx.x * 4 + (int)(threadIdx.x >> 6), l = threadIdx.x & 63;
  if (wv >= H * NT) return;
  const int h = wv / NT, t = wv - h * NT;
  const int p0 = t * kmeans_tile, pend = min(N, p0 + kmeans_tile);
  const int* ph = perm + (size_t)h * N;
  const int* zh = labels + (size_t)h * N;
  int z = l == 0 ? 0 : C - 1;
  if (l < 2) {
    const int tk = ph[l == 0 ? p0 : pend - 1];
    if ((unsigned)tk < (unsigned)N) z = zh[tk];
  }
  const int alo = min(max(__shfl(z, 0, 64), 0), C - 1);
  const int ahi = min(max(__shfl(z, 1, 64), alo), C - 1);
  uint32_t x = 0u;
  if (l < (C + 31) / 32) {
    const uint32_t* ch = cand + (size_t)h * C * 64 + l;
    for (int a = alo; a <= ahi; ++a) x |= ch[(size_t)a * 64];
  }
  tun[(size_t)wv * 64 + l] = x;
  if (l == 0) talo[wv] = alo;
}

// ------------------------------------------------------------ filtered assignment
// As k_assign_fast (same split, scores, bookkeeping, certification and listing
// of uncertified tokens), but the workgroup takes kmeans_tile consecutive
// positions of the sorted order of the previous labels and scores them only
// against the union of the candidate sets of the clusters those positions
// belong to (ascending ids, so the first-best tie rule still picks the lowest
// id).  Every candidate set holds its tokens' minimisers and any other
// centroid is strictly farther, so a label certified over the union is the
// exact argmin over all centroids; the certification uses the maxima of the
// error terms over all centroids.  Uncertified tokens are listed for the
// float64 refinement as before.
// workgroups per CU of the two-part filtered assignment (its LDS allows 3;
// 3 caps it at 168 registers, which spills, and measured no faster than 2)
// bf16 parts of w in the filtered assignment at C >= 512 (3 below)
#ifndef PARK_KM_CAND_NP
#define PARK_KM_CAND_NP 2
#endif
#ifndef PARK_KM_CAND_OCC
#define PARK_KM_CAND_OCC 2
#endif
template <int D, int NP>
__global__ __launch_bounds__(256, NP == 2 ? PARK_KM_CAND_OCC : 2) void k_assign_cand(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ w3, size_t plane,
    const float* __restrict__ b32, int Cpad, const float* __restrict__ wn,
    const float* __restrict__ eb, const float* __restrict__ bmax, int nbm, int N, int C,
    const int* __restrict__ perm, const uint32_t* __restrict__ tun,
    const int* __restrict__ talo, int* __restrict__ labels, int* __restrict__ flags,
    float* __restrict__ flagu, int* __restrict__ nflag, const double* __restrict__ xn,
    unsigned long long* __restrict__ dmax) {
  constexpr int TB = PARK_KM_TB, CT = 32, KS = D / 16, CPR = D / 8, RPI = 64 / CPR;
  constexpr int NI = NP * CT / (4 * RPI);
  static_assert(NI * 4 * RPI == NP * CT && (NP == 2 || NP == 3), "tile shape");
  static_assert(kmeans_tile == 128 * TB, "tile tokens");
  constexpr float U24 = 5.9604645e-08f, DEL = 1.1920929e-07f;
  constexpr float ER = NP == 2 ? 1.52587891e-05f : U24;
  constexpr float ET = ER * 1.01f + (D + 1) * DEL * 1.0079f +
                       0.00390625f * 1.01f * ((NP - 1) * D + 1) * DEL + U24 * 1.01f;
  constexpr float KXC = 1.1f * (2.0f * ET + 2.01f * U24) * 1.0001f;
  constexpr int NS = 2;  // ring slots: the union is a few tiles
  __shared__ __attribute__((aligned(16))) bf16_t Wt[NS][NP * CT * D];
  __shared__ uint32_t uw[64];
  __shared__ int wpre[65];
  __shared__ uint16_t ulist[2048 + CT];
  __shared__ __attribute__((aligned(16))) float ub[2048 + CT];
  __shared__ int seg[2];
  __shared__ float mx_s[2];
  __shared__ int wcnt[4];
  __shared__ unsigned long long dm_s[64];  // radius bounds of clusters alo .. alo + 63
  const int h = blockIdx.y, tid = threadIdx.x, l = tid & 63, hf = l >> 5, c32 = l & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int p0 = blockIdx.x * kmeans_tile;
  const int pend = min(N, p0 + kmeans_tile);
  const int* ph = perm + (size_t)h * N;
  const int* zh = labels + (size_t)h * N;
  // the union of the candidate sets of the clusters this tile spans, and its
  // first cluster (k_tile_union, from the previous labels)
  const size_t ti = (size_t)h * gridDim.x + blockIdx.x;
  if (tid < 64) {
    uw[tid] = tun[ti * 64 + tid];
    dm_s[tid] = 0ull;
  }
  if (tid == 0) seg[0] = talo[ti];
  __syncthreads();
  const int alo = min(max(seg[0], 0), C - 1);
  if (tid < 64) {
    const uint32_t x = tid * 32 < C ? uw[tid] : 0u;
    int inc = __popc(x);
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(inc, o, 64);
      if (tid >= o) inc += y;
    }
    wpre[tid + 1] = inc;
    if (tid == 0) wpre[0] = 0;
  }
  __syncthreads();
  const int U = wpre[64];
  for (int e = tid; e < 64 * 32; e += 256) {
    const int word = e >> 5, bit = e & 31;
    const uint32_t x = word * 32 < C ? uw[word] : 0u;
    if ((x >> bit) & 1u) {
      const int pos = wpre[word] + __popc(x & ((1u << bit) - 1u));
      const int v = word * 32 + bit;
      ulist[pos] = (uint16_t)v;
      ub[pos] = b32[(size_t)h * Cpad + v];
    }
  }
  const int ntiles = (U + CT - 1) / CT;
  for (int pos = U + tid; pos < ntiles * CT; pos += 256) {
    ulist[pos] = 0;  // any valid row; its score is +inf
    ub[pos] = INFINITY;
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
  __syncthreads();  // ulist, ub, mx_s ready
  const bf16_t* P1 = w3 + (size_t)h * C * D;
  const int pch = l % CPR;
  auto issue = [&](int tile, int slot) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int row = (w * NI + i) * RPI + l / CPR;
      const int part = row / CT, r = row % CT;
      const int v = min((int)ulist[tile * CT + r], C - 1);
      const bf16_t* src = P1 + part * plane + (size_t)v * D + 8 * (pch ^ kf_swz<D>(r));
      kf_dma16(src, kf_lds_addr(&Wt[slot][0] + (w * NI + i) * 512));
    }
  };
  if (ntiles > 0) issue(0, 0);
  // tokens of this wavefront: sorted positions p0 + w 32 TB + 32 tb + c32
  const bf16_t* Xh = X + (size_t)h * N * D;
  kf_bf16x8_t xf[TB][KS];
  float xsq[TB];
  int toks[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    xsq[tb] = 0.0f;
    const int p = p0 + w * 32 * TB + 32 * tb + c32;
    int tok = p < pend ? ph[p] : -1;
    tok = (unsigned)tok < (unsigned)N ? tok : -1;
    toks[tb] = tok;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      uint4 raw = make_uint4(0u, 0u, 0u, 0u);
      if (tok >= 0) raw = *(const uint4*)(Xh + (size_t)tok * D + 16 * s + 8 * hf);
      xf[tb][s] = __builtin_bit_cast(kf_bf16x8_t, raw);
      const uint32_t q[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const kf_bf16x2_t p2 = __builtin_bit_cast(kf_bf16x2_t, q[e]);
        xsq[tb] = __builtin_amdgcn_fdot2_f32_bf16(p2, p2, xsq[tb], false);
      }
    }
  }
  float kx[TB], best[TB], L[TB];
  int brel[TB], bidx[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    const float xs = xsq[tb] + __shfl_xor(xsq[tb], 32, 64);
    kx[tb] = xs >= 7.88860905e-31f ? KXC * sqrtf(xs) : INFINITY;
    best[tb] = INFINITY;
    L[tb] = INFINITY;
    brel[tb] = -(1 << 30);
  }
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
#pragma unroll
    for (int s = 0; s < KS; ++s) asm volatile("" ::"v"(xf[tb][s]));
    asm volatile("" ::"v"(kx[tb]));
  }
  const int swk = kf_swz<D>(c32);
  const int rowo = c32 * D;
  for (int t = 0; t < ntiles; ++t) {
    kf_wait_vmcnt<0>();
    __syncthreads();  // tile t landed; tile t-1 consumed by every wavefront
    if (t + 1 < ntiles) issue(t + 1, (t + 1) % NS);
    const int slot = t % NS;
    const bf16_t* W1 = &Wt[slot][0];
    const bf16_t* W2 = W1 + CT * D;
    const bf16_t* W3 = W2 + CT * D;
    kf_f32x16_t acc[TB];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[tb][q] = 0.0f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int co = rowo + 8 * ((2 * s + hf) ^ swk);
      const kf_bf16x8_t a2 = *(const kf_bf16x8_t*)(W2 + co);
      kf_bf16x8_t a3;
      if constexpr (NP == 3) a3 = *(const kf_bf16x8_t*)(W3 + co);
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        acc[tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, xf[tb][s], acc[tb], 0, 0, 0);
        if constexpr (NP == 3)
          acc[tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, xf[tb][s], acc[tb], 0, 0, 0);
      }
    }
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int co = rowo + 8 * ((2 * s + hf) ^ swk);
      const kf_bf16x8_t a1 = *(const kf_bf16x8_t*)(W1 + co);
#pragma unroll
      for (int tb = 0; tb < TB; ++tb)
        acc[tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, xf[tb][s], acc[tb], 0, 0, 0);
    }
    float bv[16];
#pragma unroll
    for (int bq = 0; bq < 4; ++bq) {
      const float4 b4 = *(const float4*)(&ub[t * CT + 8 * bq + 4 * hf]);
      bv[4 * bq] = b4.x;
      bv[4 * bq + 1] = b4.y;
      bv[4 * bq + 2] = b4.z;
      bv[4 * bq + 3] = b4.w;
    }
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const float sc = fmaf(-2.0f, acc[tb][q], bv[q]);
        const bool nb = sc < best[tb];
        L[tb] = __builtin_amdgcn_fmed3f(best[tb], L[tb], sc);
        best[tb] = fminf(best[tb], sc);
        brel[tb] = nb ? 8 * (q >> 2) + (q & 3) : brel[tb];
      }
      brel[tb] -= CT;
    }
  }
  // union positions of the best candidates -> centroid ids
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    const int ui = brel[tb] >= -(1 << 29) ? brel[tb] + ntiles * CT + 4 * hf : -1;
    bidx[tb] = (ui >= 0 && ui < U) ? (int)ulist[ui] : -1;
  }
  const float nmax = mx_s[0], ebmax = mx_s[1];
  bool fl[TB];
  float ubv[TB];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
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
    const int tok = toks[tb];
    fl[tb] = false;
    ubv[tb] = INFINITY;
    if (hf == 0 && tok >= 0) {
      bool ok = false;
      float e1 = 0.0f;
      if (bidx[tb] >= 0 && isfinite(best[tb])) {
        const int v = bidx[tb];
        e1 = fmaf(kx[tb], wn[(size_t)h * Cpad + v], eb[(size_t)h * Cpad + v]);
        const float emax = fmaf(kx[tb], nmax, ebmax) * 1.0001f;
        ubv[tb] = best[tb] + e1;
        ok = (L[tb] - emax) > ubv[tb];
      }
      if (ok) {
        const int v = bidx[tb];
        labels[(size_t)h * N + tok] = v;
        // D(x, mu_v)^2 <= x^T Gbar x + (the exact score's upper bound); the
        // 1e-6 e1 term covers the float64 score against the exact one
        const double d2 = fmax(xn[(size_t)h * N + tok] + (double)ubv[tb] + 1e-6 * (double)e1, 0.0);
        const unsigned long long bits = (unsigned long long)__double_as_longlong(d2);
        if ((unsigned)(v - alo) < 64u) atomicMax(&dm_s[v - alo], bits);
        else atomicMax(&dmax[(size_t)h * C + v], bits);
      }
      fl[tb] = !ok;
    }
  }
  uint64_t bal[TB];
  int tot = 0;
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    bal[tb] = __ballot(fl[tb]);
    tot += __popcll(bal[tb]);
  }
  if (l == 0) wcnt[w] = tot;
  __syncthreads();
  if (tid < 64 && alo + tid < C && dm_s[tid] != 0ull)
    atomicMax(&dmax[(size_t)h * C + alo + tid], dm_s[tid]);
  int base = blockIdx.x * kmeans_tile;
  for (int q = 0; q < w; ++q) base += wcnt[q];
  if (tid == 0) nflag[(size_t)h * gridDim.x + blockIdx.x] = wcnt[0] + wcnt[1] + wcnt[2] + wcnt[3];
  if (tot > 0) {
    const uint64_t below = (1ull << l) - 1ull;
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      if (fl[tb]) {
        const int slot = base + __popcll(bal[tb] & below);
        flags[(size_t)h * N + slot] = toks[tb];
        flagu[(size_t)h * N + slot] = ubv[tb];
      }
      base += __popcll(bal[tb]);
    }
  }
}

// ------------------------------------------------------------ refine on the union
// Exact float64 labels of the tokens k_assign_cand could not certify.  A
// listed token keeps its previous label a (the assignment wrote only the
// certified ones), and S_a holds all its minimisers (top of this file), so
// the union of the listed tokens' sets holds every listed token's exact
// argmin.  As in the all-centroid refine (k_refine_cand), every exact score
// lies in [s^_v - E_v, s^_v + E_v] with s^_v on the three-part split of w
// (same error constant), so with U the listed upper bound of a token's
// smallest exact score its argmin lies in {v : s^_v - E_v <= U}; those
// candidates (near-ties leave two or three) are scored in float64 in the
// all-centroid refine's order (16 lanes per pair, D/16 consecutive
// dimensions each, a butterfly over the 16), and the smallest score, ties to
// the lowest id, is the label.  A token with more than KMAX candidates is
// scored against every union row in the same way.
// One wavefront per tile of sorted tokens (a head's tiles on one XCD), no
// LDS ring: each lane reads its union row's three bf16 parts of w directly
// (the A operand of a 32x32x16 MFMA, 32 union rows per step) against 32
// listed tokens (the B operand).  A tile whose union exceeds kUnionMaxRows or
// whose work (token chunks x row steps) exceeds kUnionRefineMax keeps its
// list for the all-centroid refine, which runs next; a tile handled here
// clears its list length.
constexpr int kUnionMaxRows = 512;
constexpr int kUnionRefineMax = 16;

template <int D>
__global__ __launch_bounds__(64) void k_refine_union(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ w3, size_t plane,
    const float* __restrict__ b32, const float* __restrict__ wn, const float* __restrict__ eb,
    int Cpad, const double* __restrict__ w64, const double* __restrict__ b64,
    const uint32_t* __restrict__ cand, int H, int N, int C, int NT, const int* __restrict__ flags,
    const float* __restrict__ flagu, int* __restrict__ nflag, int* __restrict__ labels,
    int* __restrict__ status, const double* __restrict__ xn,
    unsigned long long* __restrict__ dmax) {
  constexpr int KS = D / 16;  // k-steps of a 32x32x16 chain
  constexpr int TC = 32;      // listed tokens per chunk
  constexpr int KMAX = 4;     // candidates kept per token
  constexpr int PL = 16, PE = D / PL, KP = 4;
  constexpr float U24 = 5.9604645e-08f, DEL = 1.1920929e-07f;
  constexpr float ET = U24 * 1.01f + (D + 1) * DEL * 1.0079f +
                       0.00390625f * 1.01f * (2 * D + 1) * DEL + U24 * 1.01f;
  constexpr float KXC = 1.1f * (2.0f * ET + 2.01f * U24) * 1.0001f;
  static_assert(PE == 4 || PE == 8, "lane slice");
  __shared__ uint16_t ul[kUnionMaxRows];
  __shared__ float ubs[kUnionMaxRows], uns[kUnionMaxRows], ues[kUnionMaxRows];
  __shared__ int dl[kmeans_tile];
  __shared__ int ccount[TC], cpos[TC * KMAX], ptk[TC * KMAX], ppos[TC * KMAX];
  __shared__ double cs[TC * KMAX];
  __shared__ int ctok[TC], over[TC], pst[TC];
  __shared__ float cx2[TC];
  __shared__ double obest[TC];
  __shared__ int oidx[TC];
  const int l = threadIdx.x, hf = l >> 5, c32 = l & 31;
  const int nitems = H * NT, per = (nitems + 7) >> 3;
  const int item = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (item >= nitems) return;
  const int h = item / NT, t = item - h * NT;
  const int p0 = t * kmeans_tile, pend = min(N, p0 + kmeans_tile);
  const int n = min(max(nflag[(size_t)h * NT + t], 0), pend - p0);
  if (n <= 0) return;
  const int* fh = flags + (size_t)h * N + p0;
  const float* fu = flagu + (size_t)h * N + p0;
  int* zh = labels + (size_t)h * N;
  // distinct previous labels of the listed tokens (non-decreasing along the
  // list, which follows the sorted order; a repeat only costs a second OR)
  int nd = 0, last = -1;
  for (int i0 = 0; i0 < n; i0 += 64) {
    const int i = i0 + l;
    int a = -1;
    if (i < n) {
      const int tk = fh[i];
      if ((unsigned)tk < (unsigned)N) {
        const int z = zh[tk];
        a = (unsigned)z < (unsigned)C ? z : -1;
      }
    }
    int prev = __shfl_up(a, 1, 64);
    if (l == 0) prev = last;
    const bool st = a >= 0 && a != prev;
    const unsigned long long bal = __ballot(st);
    if (st) dl[nd + __popcll(bal & ((1ull << l) - 1ull))] = a;
    nd += __popcll(bal);
    last = __shfl(a, 63, 64);
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // dl complete for every lane
  // union of their candidate sets: lane = word of the bit rows
  const int nwd = (C + 31) / 32;
  uint32_t bits = 0u;
  if (l < nwd)
    for (int k = 0; k < nd; ++k) bits |= cand[((size_t)h * C + dl[k]) * 64 + l];
  int inc = __popc(bits);
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o, 64);
    if (l >= o) inc += y;
  }
  const int U = __shfl(inc, 63, 64);
  const int nrt = (U + 31) / 32;
  if (U > kUnionMaxRows || ((n + TC - 1) / TC) * nrt > kUnionRefineMax)
    return;  // left to the all-centroid refine
  {
    int pos = inc - __popc(bits);
    while (bits) {
      const int bit = __ffs(bits) - 1;
      ul[pos++] = (uint16_t)(l * 32 + bit);
      bits &= bits - 1u;
    }
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // ul complete
  for (int j = l; j < U; j += 64) {
    const int v = ul[j];
    ubs[j] = b32[(size_t)h * Cpad + v];
    uns[j] = wn[(size_t)h * Cpad + v];
    ues[j] = eb[(size_t)h * Cpad + v];
  }
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
  const bf16_t* Xh = X + (size_t)h * N * D;
  const bf16_t* Wh = w3 + (size_t)h * C * D;
  const double* wh = w64 + (size_t)h * C * D;
  const double* bh = b64 + (size_t)h * C;
  const int g = l >> 4, sub = l & 15;
  for (int i0 = 0; i0 < n; i0 += TC) {
    // token c32 of the chunk: the B operand (dims 16 s + 8 hf) and its bound
    const int i = i0 + c32;
    int tok = i < n ? fh[i] : -1;
    tok = (unsigned)tok < (unsigned)N ? tok : -1;
    float Ub = tok >= 0 ? fu[i] : -INFINITY;
    if (Ub != Ub) Ub = INFINITY;  // NaN: every row is a candidate
    kf_bf16x8_t xf[KS];
    float xsq = 0.0f;
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) {
      uint4 raw = make_uint4(0u, 0u, 0u, 0u);
      if (tok >= 0) raw = *(const uint4*)(Xh + (size_t)tok * D + 16 * s2 + 8 * hf);
      xf[s2] = __builtin_bit_cast(kf_bf16x8_t, raw);
      const uint32_t q[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float lo = __uint_as_float(q[e] << 16), hi = __uint_as_float(q[e] & 0xffff0000u);
        xsq = fmaf(lo, lo, fmaf(hi, hi, xsq));
      }
    }
    xsq += __shfl_xor(xsq, 32, 64);
    const float kx = KXC * sqrtf(xsq);
    if (hf == 0) {
      ccount[c32] = 0;
      ctok[c32] = tok;
      cx2[c32] = xsq;
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    // candidates: union rows 32 rt + 8 bq + 4 hf + r of token c32 (q = 4 bq + r)
    for (int rt = 0; rt < nrt; ++rt) {
      const int v = ul[min(32 * rt + c32, U - 1)];
      const bf16_t* A1 = Wh + (size_t)v * D + 8 * hf;
      kf_f32x16_t ahi, arest;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        ahi[q] = 0.0f;
        arest[q] = 0.0f;
      }
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2) {
        const kf_bf16x8_t a1 = __builtin_bit_cast(kf_bf16x8_t, *(const uint4*)(A1 + 16 * s2));
        const kf_bf16x8_t a2 =
            __builtin_bit_cast(kf_bf16x8_t, *(const uint4*)(A1 + plane + 16 * s2));
        const kf_bf16x8_t a3 =
            __builtin_bit_cast(kf_bf16x8_t, *(const uint4*)(A1 + 2 * plane + 16 * s2));
        ahi = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, xf[s2], ahi, 0, 0, 0);
        arest = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a2, xf[s2], arest, 0, 0, 0);
        arest = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a3, xf[s2], arest, 0, 0, 0);
      }
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int pos = 32 * rt + 8 * (q >> 2) + 4 * hf + (q & 3);
        if (pos < U && tok >= 0) {
          const float sc = fmaf(-2.0f, ahi[q] + arest[q], ubs[pos]);
          const float er = fmaf(kx, uns[pos], ues[pos]);
          if (!(sc - er > Ub)) {
            const int k = atomicAdd(&ccount[c32], 1);
            if (k < KMAX) cpos[c32 * KMAX + k] = pos;
          }
        }
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    // pairs of the tokens with 1 .. KMAX candidates; the others over the union
    int np = 0, nover = 0;
    {
      const int nc = l < TC ? ccount[l] : 0;
      const bool tv = l < TC && ctok[l] >= 0;
      const bool packed = tv && nc >= 1 && nc <= KMAX;
      const int mine = packed ? nc : 0;
      int pinc = mine;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(pinc, o, 64);
        if (l >= o) pinc += y;
      }
      for (int j = 0; j < mine; ++j) {
        ptk[pinc - mine + j] = l;
        ppos[pinc - mine + j] = cpos[l * KMAX + j];
      }
      if (l < TC) pst[l] = pinc - mine;
      np = __shfl(pinc, 63, 64);
      const bool ov = tv && !packed;
      const unsigned long long bo = __ballot(ov);
      if (ov) over[__popcll(bo & ((1ull << l) - 1ull))] = l;
      nover = __popcll(bo);
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    // float64 scores of the pairs, 16 lanes each, KP pairs per group and pass
    for (int base = 0; base < np; base += 4 * KP) {
      double a[KP];
      int pp[KP];
#pragma unroll
      for (int k = 0; k < KP; ++k) {
        const int p = base + 4 * k + g;
        pp[k] = p < np ? p : -1;
        a[k] = 0.0;
        if (p < np) {
          const int tk = ctok[ptk[p]];
          const int v = ul[ppos[p]];
          uint32_t q[PE / 2];
          if constexpr (PE == 8) {
            const uint4 xu = *(const uint4*)(Xh + (size_t)tk * D + sub * PE);
            q[0] = xu.x;
            q[1] = xu.y;
            q[2] = xu.z;
            q[3] = xu.w;
          } else {
            const uint2 xu = *(const uint2*)(Xh + (size_t)tk * D + sub * PE);
            q[0] = xu.x;
            q[1] = xu.y;
          }
          const double* wr = wh + (size_t)v * D + sub * PE;
#pragma unroll
          for (int e = 0; e < PE / 2; ++e) {
            a[k] = fma((double)__uint_as_float(q[e] << 16), wr[2 * e], a[k]);
            a[k] = fma((double)__uint_as_float(q[e] & 0xffff0000u), wr[2 * e + 1], a[k]);
          }
        }
      }
#pragma unroll
      for (int k = 0; k < KP; ++k) {
        double tt = a[k];
#pragma unroll
        for (int o = PL / 2; o > 0; o >>= 1) tt += __shfl_xor(tt, o, 64);
        if (sub == 0 && pp[k] >= 0) cs[pp[k]] = fma(-2.0, tt, bh[ul[ppos[pp[k]]]]);
      }
    }
    // tokens with too many candidates: every union row, 16 lanes per row
    for (int k = 0; k < nover; ++k) {
      const int ot = over[k], tk = ctok[ot];
      uint32_t q[PE / 2];
      if constexpr (PE == 8) {
        const uint4 xu = *(const uint4*)(Xh + (size_t)tk * D + sub * PE);
        q[0] = xu.x;
        q[1] = xu.y;
        q[2] = xu.z;
        q[3] = xu.w;
      } else {
        const uint2 xu = *(const uint2*)(Xh + (size_t)tk * D + sub * PE);
        q[0] = xu.x;
        q[1] = xu.y;
      }
      double bb = INFINITY;
      int bi = 0x7fffffff;
      for (int j0 = g; j0 - g < U; j0 += 4) {
        const int j = min(j0, U - 1);
        const int v = ul[j];
        const double* wr = wh + (size_t)v * D + sub * PE;
        double acc = 0.0;
#pragma unroll
        for (int e = 0; e < PE / 2; ++e) {
          acc = fma((double)__uint_as_float(q[e] << 16), wr[2 * e], acc);
          acc = fma((double)__uint_as_float(q[e] & 0xffff0000u), wr[2 * e + 1], acc);
        }
#pragma unroll
        for (int o = PL / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
        const double sc = fma(-2.0, acc, bh[v]);
        if (j0 < U && (sc < bb || (sc == bb && v < bi))) {
          bb = sc;
          bi = v;
        }
      }
#pragma unroll
      for (int o = 16; o < 64; o <<= 1) {
        const double ob = __shfl_xor(bb, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (ob < bb || (ob == bb && oi < bi)) {
          bb = ob;
          bi = oi;
        }
      }
      if (l == 0) {
        obest[ot] = bb;
        oidx[ot] = bi;
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    // labels: the smallest float64 score, ties to the lowest id
    if (l < TC && ctok[l] >= 0) {
      const int tk = ctok[l], nc = ccount[l];
      double bb = INFINITY;
      int bi = 0x7fffffff;
      if (nc >= 1 && nc <= KMAX) {
        for (int j = 0; j < nc; ++j) {
          const double sc = cs[pst[l] + j];
          const int v = ul[cpos[l * KMAX + j]];
          if (sc < bb || (sc == bb && v < bi)) {
            bb = sc;
            bi = v;
          }
        }
      } else {
        bb = obest[l];
        bi = oidx[l];
      }
      if (!isfinite(bb) || (unsigned)bi >= (unsigned)C) {
        raise_status(status, ST_NONFINITE);
        bi = 0;
      } else {
        // radius bound of the next round: x^T Gbar x + the float64 score,
        // with a margin far above its rounding error
        const double d2 = fmax(xn[(size_t)h * N + tk] + bb +
                                   1e-12 * (fabs(bh[bi]) + 2.0 * sqrt((double)cx2[l]) *
                                                               (double)wn[(size_t)h * Cpad + bi]),
                               0.0);
        atomicMax(&dmax[(size_t)h * C + bi], (unsigned long long)__double_as_longlong(d2));
      }
      zh[tk] = bi;
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // LDS lists consumed before the next chunk
  }
  if (l == 0) nflag[(size_t)h * NT + t] = 0;
}

// ---------------------------------------------------------------- launchers
park_status launch_kfilter_setup(const bf16_t* X, const double* Gbar, int H, int N, int D,
                                 const KfilterBufs& kf, hipStream_t st) {
  const size_t gplane = (size_t)H * D * D;
  if (Gbar) {
    if (D == 128)
      PARK_LAUNCH("kfilter_gsplit", k_gsplit<128>, dim3(H), dim3(256), 0, st, Gbar, kf.g2, gplane,
                  kf.gmax);
    else
      PARK_LAUNCH("kfilter_gsplit", k_gsplit<64>, dim3(H), dim3(256), 0, st, Gbar, kf.g2, gplane,
                  kf.gmax);
  }
  // QRKC: 16 workgroups per head, each with Gbar in LDS for all its chunks
  const int nchunk = (N + 511) / 512;
  const dim3 g(Gbar ? (nchunk < 16 ? nchunk : 16) : nchunk, H);
  const bf16_t* g2 = Gbar ? kf.g2 : nullptr;
  if (!Gbar) {
    if (D == 128)
      PARK_LAUNCH("kfilter_xnorm", k_xnorm_euclid<128>, g, dim3(256), 0, st, X, N, kf.xn);
    else
      PARK_LAUNCH("kfilter_xnorm", k_xnorm_euclid<64>, g, dim3(256), 0, st, X, N, kf.xn);
  } else if (D == 128) {
    PARK_LAUNCH("kfilter_xnorm", k_xnorm<128>, g, dim3(256), 0, st, X, g2, gplane,
                (const double*)kf.gmax, N, kf.xn);
  } else {
    PARK_LAUNCH("kfilter_xnorm", k_xnorm<64>, g, dim3(256), 0, st, X, g2, gplane,
                (const double*)kf.gmax, N, kf.xn);
  }
  return PARK_OK;
}

park_status launch_kfilter_round(const bf16_t* X, int H, int N, int D, int C,
                                 const KmeansBufs& kb, const KfilterBufs& kf, bool measure_radius,
                                 hipStream_t st) {
  const int Cpad = kmeans_cpad(C);
  const size_t plane = (size_t)H * C * D;
  const int nbm = (C + 15) / 16;
  const dim3 gr((C + 3) / 4, H), gc((C + 31) / 32, H, ((C + 31) / 32 + 15) / 16),
      ga((N + kmeans_tile - 1) / kmeans_tile, H);
  // refine on the union: one wavefront per tile, a head's tiles on one XCD
  const int NT = (N + kmeans_tile - 1) / kmeans_tile;
  const dim3 gu(8 * ((H * NT + 7) / 8));
  if (D == 128) {
    if (measure_radius)
      PARK_LAUNCH("kfilter_radius", k_radius<128>, gr, dim3(256), 0, st, X, (const int*)kb.perm,
                  (const int*)kb.offsets, (const double*)kf.xn, (const double*)kb.w,
                  (const double*)kb.b, N, C, kf.r2);
    PARK_LAUNCH("kfilter_cand", k_cand<128>, gc, dim3(256), 0, st, (const bf16_t*)kf.m2, plane,
                (const bf16_t*)kb.w3, plane, (const float*)kf.mn, (const float*)kb.wn, Cpad,
                (const double*)kb.b, (const double*)kf.r2, C, kf.cand);
    PARK_LAUNCH("kfilter_union", k_tile_union, dim3((H * NT + 3) / 4), dim3(256), 0, st,
                (const int*)kb.perm, (const int*)kb.labels, (const uint32_t*)kf.cand, H, N, C, NT,
                kf.tun, kf.talo);
    if (C >= 512 && PARK_KM_CAND_NP == 2)
      PARK_LAUNCH("kmeans_assign_cand", (k_assign_cand<128, 2>), ga, dim3(256), 0, st, X,
                  (const bf16_t*)kb.w3, plane, (const float*)kb.b32, Cpad, (const float*)kb.wn,
                  (const float*)kb.eb, (const float*)kb.hmax, nbm, N, C, (const int*)kb.perm,
                  (const uint32_t*)kf.tun, (const int*)kf.talo, kb.labels, kb.flags, kb.flagu,
                  kb.nflag, (const double*)kf.xn, kf.dmax);
    else
      PARK_LAUNCH("kmeans_assign_cand", (k_assign_cand<128, 3>), ga, dim3(256), 0, st, X,
                  (const bf16_t*)kb.w3, plane, (const float*)kb.b32, Cpad, (const float*)kb.wn,
                  (const float*)kb.eb, (const float*)kb.hmax, nbm, N, C, (const int*)kb.perm,
                  (const uint32_t*)kf.tun, (const int*)kf.talo, kb.labels, kb.flags, kb.flagu,
                  kb.nflag, (const double*)kf.xn, kf.dmax);
    PARK_LAUNCH("kmeans_refine_union", k_refine_union<128>, gu, dim3(64), 0, st, X,
                (const bf16_t*)kb.w3, plane, (const float*)kb.b32, (const float*)kb.wn,
                (const float*)kb.eb, Cpad, (const double*)kb.w, (const double*)kb.b,
                (const uint32_t*)kf.cand, H, N, C, NT, (const int*)kb.flags,
                (const float*)kb.flagu, kb.nflag, kb.labels, kb.status, (const double*)kf.xn,
                kf.dmax);
  } else {
    if (measure_radius)
      PARK_LAUNCH("kfilter_radius", k_radius<64>, gr, dim3(256), 0, st, X, (const int*)kb.perm,
                  (const int*)kb.offsets, (const double*)kf.xn, (const double*)kb.w,
                  (const double*)kb.b, N, C, kf.r2);
    PARK_LAUNCH("kfilter_cand", k_cand<64>, gc, dim3(256), 0, st, (const bf16_t*)kf.m2, plane,
                (const bf16_t*)kb.w3, plane, (const float*)kf.mn, (const float*)kb.wn, Cpad,
                (const double*)kb.b, (const double*)kf.r2, C, kf.cand);
    PARK_LAUNCH("kfilter_union", k_tile_union, dim3((H * NT + 3) / 4), dim3(256), 0, st,
                (const int*)kb.perm, (const int*)kb.labels, (const uint32_t*)kf.cand, H, N, C, NT,
                kf.tun, kf.talo);
    if (C >= 512 && PARK_KM_CAND_NP == 2)
      PARK_LAUNCH("kmeans_assign_cand", (k_assign_cand<64, 2>), ga, dim3(256), 0, st, X,
                  (const bf16_t*)kb.w3, plane, (const float*)kb.b32, Cpad, (const float*)kb.wn,
                  (const float*)kb.eb, (const float*)kb.hmax, nbm, N, C, (const int*)kb.perm,
                  (const uint32_t*)kf.tun, (const int*)kf.talo, kb.labels, kb.flags, kb.flagu,
                  kb.nflag, (const double*)kf.xn, kf.dmax);
    else
      PARK_LAUNCH("kmeans_assign_cand", (k_assign_cand<64, 3>), ga, dim3(256), 0, st, X,
                  (const bf16_t*)kb.w3, plane, (const float*)kb.b32, Cpad, (const float*)kb.wn,
                  (const float*)kb.eb, (const float*)kb.hmax, nbm, N, C, (const int*)kb.perm,
                  (const uint32_t*)kf.tun, (const int*)kf.talo, kb.labels, kb.flags, kb.flagu,
                  kb.nflag, (const double*)kf.xn, kf.dmax);
    PARK_LAUNCH("kmeans_refine_union", k_refine_union<64>, gu, dim3(64), 0, st, X,
                (const bf16_t*)kb.w3, plane, (const float*)kb.b32, (const float*)kb.wn,
                (const float*)kb.eb, Cpad, (const double*)kb.w, (const double*)kb.b,
                (const uint32_t*)kf.cand, H, N, C, NT, (const int*)kb.flags,
                (const float*)kb.flagu, kb.nflag, kb.labels, kb.status, (const double*)kf.xn,
                kf.dmax);
  }
  return PARK_OK;
}

}  // namespace park
