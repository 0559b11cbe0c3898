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

// exclusive prefix of the selected block sizes into cum[0..n], 256 threads
// (ids outside [0, nblk) count as empty)
__device__ void prefix_sizes(const int* __restrict__ sel, int n, int nblk,
                             const int* __restrict__ koff, int* cum, int* tmp) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int x[8];
  int s = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int i = tid * 8 + k;
    x[k] = 0;
    if (i < n) {
      const int v = sel[i];
      if ((unsigned)v < (unsigned)nblk) x[k] = max(0, koff[v + 1] - koff[v]);
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
__device__ __forceinline__ int stream_row(int p, const int* cum, int n, const int* sel,
                                          int nblk, const int* koff) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cum[mid] <= p) lo = mid;
    else hi = mid - 1;
  }
  const int v = sel[lo];
  return (unsigned)v < (unsigned)nblk ? koff[v] + (p - cum[lo]) : -1;
}

template <typename OT>
__device__ __forceinline__ void store_out(OT* p, float v);
template <>
__device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store_out<bf16_t>(bf16_t* p, float v) { *p = f2bf(v); }

// fp32 VALU kernel: 32 query rows x 32 keys per step, 8 threads per row.
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
  prefix_sizes(sel, nsel, CK, koff, cum, tmp);
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
      if (tid < KT) krow[tid] = (k0 + tid < nk) ? stream_row(k0 + tid, cum, nsel, sel, CK, koff) : -1;
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

park_status launch_attention(const void* Qp, const void* Kp, const void* Vp, const int* q_offsets,
                             const int* k_offsets, const int* kv_count, const int* kv_index,
                             const int* q_perm, int H, int N, int D, int dtype, int CQ, int CK,
                             void* O, int out_dtype, hipStream_t st) {
  if (dtype == PARK_BF16) {
    if (out_dtype == PARK_BF16)
      return attn_dispatch_d<bf16_t, bf16_t>(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index,
                                             q_perm, H, N, D, CQ, CK, O, st);
    return attn_dispatch_d<bf16_t, float>(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index,
                                          q_perm, H, N, D, CQ, CK, O, st);
  }
  if (out_dtype == PARK_BF16)
    return attn_dispatch_d<float, bf16_t>(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index,
                                          q_perm, H, N, D, CQ, CK, O, st);
  return attn_dispatch_d<float, float>(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index,
                                       q_perm, H, N, D, CQ, CK, O, st);
}

}  // namespace park
