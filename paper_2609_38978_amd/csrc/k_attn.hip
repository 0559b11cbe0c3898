// Block-sparse attention with un-permutation (Eq. (2), Sec. 3.1).
//
// For query block u the key stream is the concatenation of the rows of its
// selected key blocks (ascending block id); the softmax of each query is
// taken over that stream (renormalised), flash-attention style with an
// online maximum, and row i of Q' is written to O[q_perm[i]].  Only the
// last 32-key tile of a stream is partial, whatever the block sizes.
#include "common.h"
#include "kernels.h"

namespace park {

constexpr int AT_MAXC = 2048;

// exclusive prefix of the selected block sizes into cum[0..n] and the first
// row of each selected block into kst[0..n), 256 threads (ids outside
// [0, nblk) count as empty)
__device__ void prefix_sizes(const int* __restrict__ sel, int n, int nblk,
                             const int* __restrict__ koff, int* cum, int* kst, int* tmp) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int x[8];
  int s = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int i = tid * 8 + k;
    x[k] = 0;
    if (i < n) {
      const int v = sel[i];
      int start = -1;
      if ((unsigned)v < (unsigned)nblk) {
        start = koff[v];
        x[k] = max(0, koff[v + 1] - start);
      }
      kst[i] = start;
    }
    s += x[k];
  }
  int inc = s;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  if (lane == 63) tmp[wid] = inc;
  __syncthreads();
  int pre = 0;
  for (int w = 0; w < wid; ++w) pre += tmp[w];
  int run = pre + inc - s;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int i = tid * 8 + k;
    if (i < n) cum[i] = run;
    run += x[k];
    if (i == n - 1) cum[n] = run;
  }
  if (n == 0 && tid == 0) cum[0] = 0;
  __syncthreads();
}

// row of stream position p: binary search of the last m with cum[m] <= p
// (LDS only; -1 past the end of the stream)
__device__ __forceinline__ int stream_row(int p, const int* cum, const int* kst, int n) {
  if (p >= cum[n]) return -1;
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cum[mid] <= p) lo = mid;
    else hi = mid - 1;
  }
  return kst[lo] < 0 ? -1 : kst[lo] + (p - cum[lo]);
}

template <typename OT>
__device__ __forceinline__ void store_out(OT* p, float v);
template <>
__device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store_out<bf16_t>(bf16_t* p, float v) { *p = f2bf(v); }

// fp32 VALU kernel (fp32 inputs): 32 query rows x 32 keys per step, 8 threads
// per row.
template <typename T, typename OT, int D>
__global__ __launch_bounds__(256) void k_attn_valu(const T* __restrict__ Qp, const T* __restrict__ Kp,
                                                   const T* __restrict__ Vp,
                                                   const int* __restrict__ q_offsets,
                                                   const int* __restrict__ k_offsets,
                                                   const int* __restrict__ kv_count,
                                                   const int* __restrict__ kv_index,
                                                   const int* __restrict__ q_perm, int N, int CQ,
                                                   int CK, OT* __restrict__ O) {
  constexpr int RT = 32, KT = 32, TPR = 8, CPT = D / TPR, KPT = KT / TPR;
  __shared__ float qs[RT][D + 1];
  __shared__ float ks[KT][D + 1];
  __shared__ float vs[KT][D + 1];
  __shared__ float ps[RT][KT + 1];
  __shared__ int cum[AT_MAXC + 1];
  __shared__ int kst[AT_MAXC];
  __shared__ int krow[KT];
  __shared__ int tmp[4];
  const int h = blockIdx.y, u = blockIdx.x, tid = threadIdx.x;
  const int* qo = q_offsets + (size_t)h * (CQ + 1);
  const int q0 = min(max(qo[u], 0), N), q1 = min(max(qo[u + 1], q0), N);
  if (q1 <= q0) return;
  const int* koff = k_offsets + (size_t)h * (CK + 1);
  const size_t row = (size_t)h * CQ + u;
  int nsel = kv_count[row];
  nsel = nsel < 0 ? 0 : (nsel > CK ? CK : nsel);
  const int* sel = kv_index + row * CK;
  prefix_sizes(sel, nsel, CK, koff, cum, kst, tmp);
  const int nk = cum[nsel];
  const T* Qh = Qp + (size_t)h * N * D;
  const T* Kh = Kp + (size_t)h * N * D;
  const T* Vh = Vp + (size_t)h * N * D;
  const int r = tid / TPR, sub = tid % TPR;
  const float scale = 1.0f / sqrtf((float)D);
  for (int r0 = q0; r0 < q1; r0 += RT) {
    const int nr = min(RT, q1 - r0);
    __syncthreads();
    for (int e = tid; e < RT * D; e += 256) {
      const int rr = e / D, c = e % D;
      qs[rr][c] = rr < nr ? to_f(Qh[(size_t)(r0 + rr) * D + c]) : 0.0f;
    }
    float mrow = -INFINITY, lrow = 0.0f;
    float acc[CPT];
#pragma unroll
    for (int c = 0; c < CPT; ++c) acc[c] = 0.0f;
    for (int k0 = 0; k0 < nk; k0 += KT) {
      __syncthreads();
      if (tid < KT) krow[tid] = stream_row(k0 + tid, cum, kst, nsel);
      __syncthreads();
      for (int e = tid; e < KT * D; e += 256) {
        const int kr = e / D, c = e % D;
        const int src = krow[kr];
        const bool ok = (unsigned)src < (unsigned)N;
        ks[kr][c] = ok ? to_f(Kh[(size_t)src * D + c]) : 0.0f;
        vs[kr][c] = ok ? to_f(Vh[(size_t)src * D + c]) : 0.0f;
      }
      __syncthreads();
      float s[KPT];
      float tmax = -INFINITY;
#pragma unroll
      for (int j = 0; j < KPT; ++j) {
        const int kk = sub + TPR * j;
        float dot = 0.0f;
#pragma unroll 8
        for (int a = 0; a < D; ++a) dot = fmaf(qs[r][a], ks[kk][a], dot);
        s[j] = (k0 + kk < nk) ? dot * scale : -INFINITY;
        tmax = fmaxf(tmax, s[j]);
      }
#pragma unroll
      for (int o = 1; o < TPR; o <<= 1) tmax = fmaxf(tmax, __shfl_xor(tmax, o, 64));
      const float mnew = fmaxf(mrow, tmax);
      const float alpha = (mrow == -INFINITY) ? 0.0f : expf(mrow - mnew);
      float psum = 0.0f;
#pragma unroll
      for (int j = 0; j < KPT; ++j) {
        const float p = (s[j] == -INFINITY) ? 0.0f : expf(s[j] - mnew);
        ps[r][sub + TPR * j] = p;
        psum += p;
      }
#pragma unroll
      for (int o = 1; o < TPR; o <<= 1) psum += __shfl_xor(psum, o, 64);
      lrow = lrow * alpha + psum;
      mrow = mnew;
#pragma unroll
      for (int c = 0; c < CPT; ++c) acc[c] *= alpha;
      __syncthreads();
      for (int kk = 0; kk < KT; ++kk) {
        const float p = ps[r][kk];
#pragma unroll
        for (int c = 0; c < CPT; ++c) acc[c] = fmaf(p, vs[kk][sub * CPT + c], acc[c]);
      }
    }
    if (r < nr) {
      const int dst = q_perm[(size_t)h * N + r0 + r];
      if ((unsigned)dst < (unsigned)N) {
        const float inv = lrow > 0.0f ? 1.0f / lrow : 0.0f;
        OT* o = O + ((size_t)h * N + dst) * D + sub * CPT;
#pragma unroll
        for (int c = 0; c < CPT; ++c) store_out<OT>(o + c, acc[c] * inv);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel (v_mfma_f32_16x16x32_bf16).  Workgroup = (query block, head),
// 4 wavefronts of 16 query rows each; 64-key tiles of the key stream are staged
// in LDS (K row-major, V transposed).  Per tile and wavefront:
//   S^T = K Q^T  (16 keys x 16 queries per MFMA): lane l holds keys
//                16b + 4(l/16) + r of query l%16, so the online softmax of a
//                query reduces over 16 registers and two lane groups only;
//   O^T += V^T P^T: the probabilities are reused from registers as the B
//                operand (k-slot 8g+r <-> key 32c+4g+r, 8g+4+r <-> 32c+16+4g+r)
//                and V^T supplies the matching keys from LDS.
// Softmax in base 2: the running maximum is taken on raw scores and each
// probability costs one FMA and one v_exp_f32; probabilities are rounded to
// bf16 (RNE) by the packed hardware conversion.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

template <typename OT>
__device__ __forceinline__ void store_out4(OT* p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void store_out4<float>(float* p, float a, float b, float c, float d) {
  *(float4*)p = make_float4(a, b, c, d);
}
template <>
__device__ __forceinline__ void store_out4<bf16_t>(bf16_t* p, float a, float b, float c, float d) {
  const uint32_t lo = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
  const uint32_t hi = (uint32_t)f2bf(c) | ((uint32_t)f2bf(d) << 16);
  *(uint2*)p = make_uint2(lo, hi);
}

// Loads one 64-key tile of K' and V' (rows krow[buf][0..63], -1 = padding)
// into registers: NKL 16-byte chunks of K and NVL key pairs of V per thread.
template <int D, int KT, int NKL, int NVL>
__device__ __forceinline__ void stage_kv(uint4 (&kreg)[NKL], uint4 (&va)[NVL], uint4 (&vb)[NVL],
                                         const int (&krow)[2][KT], int buf,
                                         const bf16_t* __restrict__ Kh,
                                         const bf16_t* __restrict__ Vh, int N, int tid) {
  constexpr int CH = D / 8;
#pragma unroll
  for (int i = 0; i < NKL; ++i) {
    const int e = tid + 256 * i, key = e / CH, ch = e % CH;
    const int src = krow[buf][key];
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if ((unsigned)src < (unsigned)N) v = *(const uint4*)(Kh + (size_t)src * D + 8 * ch);
    kreg[i] = v;
  }
#pragma unroll
  for (int i = 0; i < NVL; ++i) {
    const int e = tid + 256 * i, kp = e % (KT / 2), ch = e / (KT / 2);
    const int s0 = krow[buf][2 * kp], s1 = krow[buf][2 * kp + 1];
    uint4 a = make_uint4(0u, 0u, 0u, 0u), b = a;
    if ((unsigned)s0 < (unsigned)N) a = *(const uint4*)(Vh + (size_t)s0 * D + 8 * ch);
    if ((unsigned)s1 < (unsigned)N) b = *(const uint4*)(Vh + (size_t)s1 * D + 8 * ch);
    va[i] = a;
    vb[i] = b;
  }
}

template <typename OT, int D>
__global__ __launch_bounds__(256) void k_attn_mfma(const bf16_t* __restrict__ Qp,
                                                   const bf16_t* __restrict__ Kp,
                                                   const bf16_t* __restrict__ Vp,
                                                   const int* __restrict__ q_offsets,
                                                   const int* __restrict__ k_offsets,
                                                   const int* __restrict__ kv_count,
                                                   const int* __restrict__ kv_index,
                                                   const int* __restrict__ q_perm, int N, int CQ,
                                                   int CK, float scale_log2, OT* __restrict__ O) {
  constexpr int KT = 64;        // keys per tile
  constexpr int KS = D / 32;    // k-steps of S
  constexpr int DB = D / 16;    // 16-column blocks of O
  constexpr int KROW = D + 8;   // padded K row (bf16)
  constexpr int VROW = KT + 4;  // padded V^T row (bf16): 136 B, conflict-free 8-byte reads
  constexpr int CH = D / 8;     // 16-byte chunks per row
  constexpr int NKL = KT * CH / 256;        // K chunks loaded per thread
  constexpr int NVL = (KT / 2) * CH / 256;  // V key-pair chunks loaded per thread
  __shared__ __attribute__((aligned(16))) bf16_t Ks[KT * KROW];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[D * VROW];
  __shared__ int cum[AT_MAXC + 1];
  __shared__ int kst[AT_MAXC];
  __shared__ int krow[2][KT];
  __shared__ int tmp[4];
  const int h = blockIdx.y, u = blockIdx.x, tid = threadIdx.x;
  const int* qo = q_offsets + (size_t)h * (CQ + 1);
  const int q0 = min(max(qo[u], 0), N), q1 = min(max(qo[u + 1], q0), N);
  if (q1 <= q0) return;
  const int* koff = k_offsets + (size_t)h * (CK + 1);
  const size_t row = (size_t)h * CQ + u;
  int nsel = kv_count[row];
  nsel = nsel < 0 ? 0 : (nsel > CK ? CK : nsel);
  const int* sel = kv_index + row * CK;
  prefix_sizes(sel, nsel, CK, koff, cum, kst, tmp);
  const int nk = cum[nsel];
  const bf16_t* Qh = Qp + (size_t)h * N * D;
  const bf16_t* Kh = Kp + (size_t)h * N * D;
  const bf16_t* Vh = Vp + (size_t)h * N * D;
  const int w = tid >> 6, l = tid & 63, g = l >> 4, c16 = l & 15;
  // register staging of one K/V tile (prefetched one tile ahead); the tile's
  // stream rows come from krow[buf][*], filled by the first 64 threads.
  uint4 kreg[NKL], va[NVL], vb[NVL];

  for (int r0 = q0; r0 < q1; r0 += 64) {
    const int qr = r0 + 16 * w + c16;
    const bool qvalid = qr < q1;
    const bool wave_on = r0 + 16 * w < q1;
    bf16x8_t qf[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      uint4 raw = make_uint4(0u, 0u, 0u, 0u);
      if (qvalid) raw = *(const uint4*)(Qh + (size_t)qr * D + 32 * s + 8 * g);
      qf[s] = __builtin_bit_cast(bf16x8_t, raw);
    }
    float m = -INFINITY, lpart = 0.0f;
    f32x4_t acc[DB];
#pragma unroll
    for (int b = 0; b < DB; ++b) acc[b] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    if (nk > 0) {
      if (tid < KT) krow[0][tid] = stream_row(tid, cum, kst, nsel);
      __syncthreads();
      stage_kv<D, KT, NKL, NVL>(kreg, va, vb, krow, 0, Kh, Vh, N, tid);
    }
    int buf = 0;
    for (int k0 = 0; k0 < nk; k0 += KT) {
      __syncthreads();  // previous tile fully consumed
#pragma unroll
      for (int i = 0; i < NKL; ++i) {
        const int e = tid + 256 * i, key = e / CH, ch = e % CH;
        *(uint4*)(Ks + key * KROW + 8 * ch) = kreg[i];
      }
#pragma unroll
      for (int i = 0; i < NVL; ++i) {
        const int e = tid + 256 * i, kp = e % (KT / 2), ch = e / (KT / 2);
        const uint32_t a0 = va[i].x, a1 = va[i].y, a2 = va[i].z, a3 = va[i].w;
        const uint32_t b0 = vb[i].x, b1 = vb[i].y, b2 = vb[i].z, b3 = vb[i].w;
        bf16_t* vt = Vt + (8 * ch) * VROW + 2 * kp;
        *(uint32_t*)(vt + 0 * VROW) = (a0 & 0xffffu) | (b0 << 16);
        *(uint32_t*)(vt + 1 * VROW) = (a0 >> 16) | (b0 & 0xffff0000u);
        *(uint32_t*)(vt + 2 * VROW) = (a1 & 0xffffu) | (b1 << 16);
        *(uint32_t*)(vt + 3 * VROW) = (a1 >> 16) | (b1 & 0xffff0000u);
        *(uint32_t*)(vt + 4 * VROW) = (a2 & 0xffffu) | (b2 << 16);
        *(uint32_t*)(vt + 5 * VROW) = (a2 >> 16) | (b2 & 0xffff0000u);
        *(uint32_t*)(vt + 6 * VROW) = (a3 & 0xffffu) | (b3 << 16);
        *(uint32_t*)(vt + 7 * VROW) = (a3 >> 16) | (b3 & 0xffff0000u);
      }
      const bool more = k0 + KT < nk;
      if (more && tid < KT) krow[buf ^ 1][tid] = stream_row(k0 + KT + tid, cum, kst, nsel);
      __syncthreads();
      buf ^= 1;
      if (more) stage_kv<D, KT, NKL, NVL>(kreg, va, vb, krow, buf, Kh, Vh, N, tid);
      if (!wave_on) continue;
      f32x4_t st[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        st[b] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const bf16x8_t a = *(const bf16x8_t*)(Ks + (16 * b + c16) * KROW + 32 * s + 8 * g);
          st[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[s], st[b], 0, 0, 0);
        }
      }
      // online softmax on raw scores; exp2 argument = (s - m) * scale * log2(e)
      if (k0 + KT > nk) {  // last tile: mask the keys past the end of the stream
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (k0 + 16 * b + 4 * g + r >= nk) st[b][r] = -INFINITY;
      }
      float tmax = st[0][0];
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) tmax = fmaxf(tmax, st[b][r]);
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
      const float mnew = fmaxf(m, tmax);
      if (__any(mnew != m)) {  // rescale only when some running maximum moved
        const float alpha = __builtin_amdgcn_exp2f((m - mnew) * scale_log2);
        lpart *= alpha;
#pragma unroll
        for (int b = 0; b < DB; ++b) acc[b] *= alpha;
      }
      m = mnew;
      const float nms = -mnew * scale_log2;
      bf16x8_t pb[2];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        float p[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          p[r] = __builtin_amdgcn_exp2f(fmaf(st[b][r], scale_log2, nms));
          lpart += p[r];
        }
        const bf16x2_t lo = __builtin_convertvector(f32x2_t{p[0], p[1]}, bf16x2_t);
        const bf16x2_t hi = __builtin_convertvector(f32x2_t{p[2], p[3]}, bf16x2_t);
        pb[b >> 1][(b & 1) * 4 + 0] = lo[0];
        pb[b >> 1][(b & 1) * 4 + 1] = lo[1];
        pb[b >> 1][(b & 1) * 4 + 2] = hi[0];
        pb[b >> 1][(b & 1) * 4 + 3] = hi[1];
      }
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int mb = 0; mb < DB; ++mb) {
          const bf16_t* vrow = Vt + (16 * mb + c16) * VROW + 32 * c + 4 * g;
          const uint2 lo = *(const uint2*)vrow;
          const uint2 hi = *(const uint2*)(vrow + 16);
          const bf16x8_t a = __builtin_bit_cast(bf16x8_t, make_uint4(lo.x, lo.y, hi.x, hi.y));
          acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[c], acc[mb], 0, 0, 0);
        }
    }
    float lsum = lpart + __shfl_xor(lpart, 16, 64);
    lsum += __shfl_xor(lsum, 32, 64);
    if (qvalid) {
      const int dst = q_perm[(size_t)h * N + qr];
      if ((unsigned)dst < (unsigned)N) {
        const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
        OT* o = O + ((size_t)h * N + dst) * D + 4 * g;
#pragma unroll
        for (int mb = 0; mb < DB; ++mb)
          store_out4<OT>(o + 16 * mb, acc[mb][0] * inv, acc[mb][1] * inv, acc[mb][2] * inv,
                         acc[mb][3] * inv);
      }
    }
    __syncthreads();
  }
}

template <typename T, typename OT>
static park_status attn_dispatch_d(const void* Qp, const void* Kp, const void* Vp, const int* qo,
                                   const int* ko, const int* kc, const int* ki, const int* qp,
                                   int H, int N, int D, int CQ, int CK, void* O, hipStream_t st) {
  dim3 g(CQ, H);
  if (D == 128)
    PARK_LAUNCH("attn_valu", (k_attn_valu<T, OT, 128>), g, dim3(256), 0, st, (const T*)Qp,
                (const T*)Kp, (const T*)Vp, qo, ko, kc, ki, qp, N, CQ, CK, (OT*)O);
  else
    PARK_LAUNCH("attn_valu", (k_attn_valu<T, OT, 64>), g, dim3(256), 0, st, (const T*)Qp,
                (const T*)Kp, (const T*)Vp, qo, ko, kc, ki, qp, N, CQ, CK, (OT*)O);
  return PARK_OK;
}

template <typename OT>
static park_status attn_mfma_d(const void* Qp, const void* Kp, const void* Vp, const int* qo,
                               const int* ko, const int* kc, const int* ki, const int* qp, int H,
                               int N, int D, int CQ, int CK, void* O, hipStream_t st) {
  dim3 g(CQ, H);
  const float sl2 = (float)(1.4426950408889634 / sqrt((double)D));
  if (D == 128)
    PARK_LAUNCH("attn_mfma", (k_attn_mfma<OT, 128>), g, dim3(256), 0, st, (const bf16_t*)Qp,
                (const bf16_t*)Kp, (const bf16_t*)Vp, qo, ko, kc, ki, qp, N, CQ, CK, sl2, (OT*)O);
  else
    PARK_LAUNCH("attn_mfma", (k_attn_mfma<OT, 64>), g, dim3(256), 0, st, (const bf16_t*)Qp,
                (const bf16_t*)Kp, (const bf16_t*)Vp, qo, ko, kc, ki, qp, N, CQ, CK, sl2, (OT*)O);
  return PARK_OK;
}

park_status launch_attention(const void* Qp, const void* Kp, const void* Vp, const int* q_offsets,
                             const int* k_offsets, const int* kv_count, const int* kv_index,
                             const int* q_perm, int H, int N, int D, int dtype, int CQ, int CK,
                             void* O, int out_dtype, hipStream_t st) {
  if (dtype == PARK_BF16) {
    if (out_dtype == PARK_BF16)
      return attn_mfma_d<bf16_t>(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index, q_perm, H,
                                 N, D, CQ, CK, O, st);
    return attn_mfma_d<float>(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index, q_perm, H, N,
                              D, CQ, CK, O, st);
  }
  // fp32 inputs: VALU kernel in fp32 (the contraction cannot use bf16 MFMA exactly)
  if (out_dtype == PARK_BF16)
    return attn_dispatch_d<float, bf16_t>(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index,
                                          q_perm, H, N, D, CQ, CK, O, st);
  return attn_dispatch_d<float, float>(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index,
                                       q_perm, H, N, D, CQ, CK, O, st);
}

}  // namespace park
