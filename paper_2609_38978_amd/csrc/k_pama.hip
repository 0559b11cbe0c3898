// PAMA block importance (Sec. 5.1, Eqs. (8)-(9)) and mask selection
// (Sec. 3.2 top-p, App. J top-k).
//
//   S^_iv = q_i . c_v / sqrt(d) + log n_v   (n_v = 0: block left out)
//   P^_iv = softmax_v S^_iv;   W^_uv = (1 / n_u) sum_{i in Q_u} P^_iv
//
// k_pama64 evaluates this in float64 with one workgroup per (query block,
// head): the logit row of every query stays in registers and the column sums
// in registers of the thread that owns the key block (no HBM round trip, no
// atomics, fixed summation order).
#include "common.h"
#include "kernels.h"

namespace park {

constexpr int MAXC = 2048;

// ---------------------------------------------------------------- helpers
// exclusive scan of up to 2048 ints held in LDS `a[0..n)`, 256 threads;
// returns the total.  `tmp` needs 4 ints.
__device__ int block_exclusive_scan_2048(int* a, int n, int* tmp) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int x[8];
  int s = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int i = tid * 8 + k;
    x[k] = i < n ? a[i] : 0;
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
  int pre = 0, tot = 0;
  for (int w = 0; w < 4; ++w) {
    if (w < wid) pre += tmp[w];
    tot += tmp[w];
  }
  int run = pre + inc - s;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int i = tid * 8 + k;
    if (i < n) a[i] = run;
    run += x[k];
  }
  __syncthreads();
  return tot;
}

// ---------------------------------------------------------------- PAMA f64
template <typename T, int D>
__global__ __launch_bounds__(256) void k_pama64(const T* __restrict__ Qp, const int* __restrict__ q_offsets,
                                                const float* __restrict__ cen,
                                                const int* __restrict__ k_sizes, int N, int CQ, int CK,
                                                double* __restrict__ W64, float* __restrict__ W32,
                                                int* status) {
  constexpr int QT = 4;                 // queries per step
  constexpr int MV = MAXC / 256;        // key blocks per thread
  __shared__ double qs[QT][D];
  __shared__ double red[4][QT];
  const int h = blockIdx.y, u = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int* off = q_offsets + (size_t)h * (CQ + 1);
  const int q0 = min(max(off[u], 0), N), q1 = min(max(off[u + 1], q0), N);
  const int nu = q1 - q0;
  const size_t wrow = ((size_t)h * CQ + u) * CK;
  double lg[MV], acc[MV];
  bool on[MV];
#pragma unroll
  for (int m = 0; m < MV; ++m) {
    const int v = tid + 256 * m;
    const int n = v < CK ? k_sizes[(size_t)h * CK + v] : 0;
    on[m] = n > 0;
    lg[m] = on[m] ? log((double)n) : 0.0;
    acc[m] = 0.0;
  }
  const double sqd = sqrt((double)D);
  const float* ch = cen + (size_t)h * CK * D;
  for (int i0 = q0; i0 < q1; i0 += QT) {
    const int nq = min(QT, q1 - i0);
    __syncthreads();
    for (int e = tid; e < QT * D; e += 256) {
      const int k = e / D, a = e % D;
      qs[k][a] = k < nq ? (double)to_f(Qp[((size_t)h * N + i0 + k) * D + a]) : 0.0;
    }
    __syncthreads();
    double S[QT][MV];
#pragma unroll
    for (int m = 0; m < MV; ++m) {
      const int v = tid + 256 * m;
#pragma unroll
      for (int k = 0; k < QT; ++k) S[k][m] = 0.0;
      if (on[m]) {
        const float* cv = ch + (size_t)v * D;
        for (int a = 0; a < D; ++a) {
          const double c = (double)cv[a];
#pragma unroll
          for (int k = 0; k < QT; ++k) S[k][m] = fma(qs[k][a], c, S[k][m]);
        }
      }
    }
    // logits, row maxima
    double mx[QT];
#pragma unroll
    for (int k = 0; k < QT; ++k) {
      mx[k] = -INFINITY;
#pragma unroll
      for (int m = 0; m < MV; ++m)
        if (on[m]) {
          S[k][m] = S[k][m] / sqd + lg[m];
          mx[k] = fmax(mx[k], S[k][m]);
        }
      for (int o = 32; o > 0; o >>= 1) mx[k] = fmax(mx[k], __shfl_xor(mx[k], o, 64));
    }
    if (lane == 0)
#pragma unroll
      for (int k = 0; k < QT; ++k) red[wid][k] = mx[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < QT; ++k) mx[k] = fmax(fmax(red[0][k], red[1][k]), fmax(red[2][k], red[3][k]));
    __syncthreads();
    // exponentials and row sums
    double sm[QT];
#pragma unroll
    for (int k = 0; k < QT; ++k) {
      sm[k] = 0.0;
#pragma unroll
      for (int m = 0; m < MV; ++m)
        if (on[m]) {
          S[k][m] = exp(S[k][m] - mx[k]);
          sm[k] += S[k][m];
        }
      for (int o = 32; o > 0; o >>= 1) sm[k] += __shfl_xor(sm[k], o, 64);
    }
    if (lane == 0)
#pragma unroll
      for (int k = 0; k < QT; ++k) red[wid][k] = sm[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < QT; ++k) sm[k] = ((red[0][k] + red[1][k]) + red[2][k]) + red[3][k];
    // column sums over the queries of the block, in query order
#pragma unroll
    for (int k = 0; k < QT; ++k)
      if (k < nq)
#pragma unroll
        for (int m = 0; m < MV; ++m)
          if (on[m]) acc[m] += S[k][m] / sm[k];
  }
#pragma unroll
  for (int m = 0; m < MV; ++m) {
    const int v = tid + 256 * m;
    if (v < CK) {
      const double wv = nu > 0 ? acc[m] / (double)nu : 0.0;
      if (!isfinite(wv)) raise_status(status, ST_NONFINITE);
      if (W64) W64[wrow + v] = wv;
      if (W32) W32[wrow + v] = (float)wv;
    }
  }
}

// ---------------------------------------------------------------- select
// One workgroup per (query block, head).  Valid key blocks are sorted by
// (W^ descending, id ascending) with an LDS bitonic sort; the kept prefix is
// then marked and compacted into ascending ids.
__global__ __launch_bounds__(256) void k_select64(const double* __restrict__ W64,
                                                  const int* __restrict__ q_offsets,
                                                  const int* __restrict__ k_sizes, int CQ, int CK,
                                                  int P, int mode, double param, int kcount,
                                                  int* __restrict__ kv_count,
                                                  int* __restrict__ kv_index) {
  __shared__ double key[MAXC];
  __shared__ int id[MAXC];
  __shared__ int flag[MAXC];
  __shared__ int tmp[4];
  __shared__ int nvalid_s, m_s;
  const int h = blockIdx.y, u = blockIdx.x, tid = threadIdx.x;
  const int* off = q_offsets + (size_t)h * (CQ + 1);
  const int nu = off[u + 1] - off[u];
  const size_t row = (size_t)h * CQ + u;
  if (nu <= 0) {
    if (tid == 0) kv_count[row] = 0;
    return;
  }
  if (tid == 0) nvalid_s = 0;
  __syncthreads();
  int myvalid = 0;
  for (int e = tid; e < P; e += 256) {
    const bool ok = e < CK && k_sizes[(size_t)h * CK + e] > 0;
    key[e] = ok ? W64[row * CK + e] : -1.0;
    id[e] = e;
    if (e < CK) flag[e] = 0;
    myvalid += ok;
  }
  atomicAdd(&nvalid_s, myvalid);
  __syncthreads();
  // bitonic sort, "before" = larger key, then smaller id
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int t = tid; t < P / 2; t += 256) {
        const int i = 2 * t - (t & (j - 1));
        const int l = i + j;
        const bool up = (i & k) == 0;
        const double ka = key[i], kb = key[l];
        const int ia = id[i], ib = id[l];
        const bool a_first = (ka > kb) || (ka == kb && ia < ib);
        if (a_first != up) {
          key[i] = kb;
          key[l] = ka;
          id[i] = ib;
          id[l] = ia;
        }
      }
      __syncthreads();
    }
  }
  const int nvalid = nvalid_s;
  if (tid == 0) {
    int m;
    if (mode == PARK_SELECT_TOPK) {
      m = kcount < 1 ? 1 : kcount;
      if (m > nvalid) m = nvalid;
    } else {
      double cs = 0.0;
      m = nvalid;
      for (int r = 0; r < nvalid; ++r) {
        cs += key[r];
        if (cs >= param) {
          m = r + 1;
          break;
        }
      }
    }
    if (m < 1 && nvalid > 0) m = 1;
    m_s = m;
  }
  __syncthreads();
  const int m = m_s;
  for (int r = tid; r < m; r += 256) flag[id[r]] = 1;
  __syncthreads();
  // ascending compaction: flag -> exclusive prefix positions
  for (int e = tid; e < CK; e += 256) id[e] = flag[e];
  __syncthreads();
  block_exclusive_scan_2048(id, CK, tmp);
  int* out = kv_index + row * CK;
  for (int e = tid; e < CK; e += 256)
    if (flag[e]) out[id[e]] = e;
  if (tid == 0) kv_count[row] = m;
}

// ---------------------------------------------------------------- launchers
park_status launch_pama64(const void* Qp, const int* q_offsets, const float* cen,
                          const int* k_sizes, int H, int N, int D, int dtype, int CQ, int CK,
                          double* W64, float* W32, int* status, hipStream_t st) {
  dim3 g(CQ, H);
  if (D == 128) {
    if (dtype == PARK_BF16)
      PARK_LAUNCH("pama64", (k_pama64<bf16_t, 128>), g, dim3(256), 0, st, (const bf16_t*)Qp,
                  q_offsets, cen, k_sizes, N, CQ, CK, W64, W32, status);
    else
      PARK_LAUNCH("pama64", (k_pama64<float, 128>), g, dim3(256), 0, st, (const float*)Qp,
                  q_offsets, cen, k_sizes, N, CQ, CK, W64, W32, status);
  } else {
    if (dtype == PARK_BF16)
      PARK_LAUNCH("pama64", (k_pama64<bf16_t, 64>), g, dim3(256), 0, st, (const bf16_t*)Qp,
                  q_offsets, cen, k_sizes, N, CQ, CK, W64, W32, status);
    else
      PARK_LAUNCH("pama64", (k_pama64<float, 64>), g, dim3(256), 0, st, (const float*)Qp,
                  q_offsets, cen, k_sizes, N, CQ, CK, W64, W32, status);
  }
  return PARK_OK;
}

park_status launch_select(const double* W64, const int* q_offsets, const int* k_sizes, int H,
                          int CQ, int CK, int mode, double param, int* kv_count, int* kv_index,
                          hipStream_t st) {
  int P = 1;
  while (P < CK) P <<= 1;
  if (P < 2) P = 2;
  int kcount = 0;
  if (mode == PARK_SELECT_TOPK) {
    // ceil(rho * N_K) blocks, clamped on the device to [1, #nonempty]
    double x = param * (double)CK - 1e-9;
    kcount = (int)x;
    if ((double)kcount < x) ++kcount;
    if (kcount < 1) kcount = 1;
  }
  PARK_LAUNCH("select", k_select64, dim3(CQ, H), dim3(256), 0, st, W64, q_offsets, k_sizes, CQ,
              CK, P, mode, param, kcount, kv_count, kv_index);
  return PARK_OK;
}

}  // namespace park
