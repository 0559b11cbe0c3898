// PAMA block importance (Sec. 5.1, Eqs. (8)-(9)) and mask selection
// (Sec. 3.2 top-p, App. J top-k).
//
//   S^_iv = q_i . c_v / sqrt(d) + log n_v   (n_v = 0: block left out)
//   P^_iv = softmax_v S^_iv;   W^_uv = (1 / n_u) sum_{i in Q_u} P^_iv
//
// k_pama64 evaluates this in float64 (float64 MFMA) over items of whole
// chunks of 64 queries; an item's column sums stay in LDS, and the items of
// a query block are added up in item order (deterministic, no atomics on
// values).
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
// Float64 PAMA rows on float64 MFMA (v_mfma_f64_16x16x4_f64: A[i][k] and
// B[k][j] in lane 16k + i / 16k + j, D[g + 4r][c] in lane 16g + c, item r).
// Workgroup = one (query block, head) at a time; the block's rows in chunks
// of 64 (4 wavefronts x 16 queries), each chunk streaming the float32
// centroids twice (normaliser pass, probability pass) through a two-slot LDS
// ring filled by LDS DMA (rows swizzled in 16-byte chunks so the B-operand
// reads are free of bank conflicts).  Logits, exponentials and all sums in
// float64; a tile's per-wavefront column sums go through LDS and are added to
// the row's column sums in wavefront order, chunk after chunk (deterministic).
// With a row list it recomputes only the listed query blocks (the rows the
// fast path could not certify); the workgroups of a head run on one XCD.
//
// Given the fast path's W^ and its certified relative error delta_u (plus
// 4 2^-126 absolute near float's underflow), the normaliser pass leaves out
// the blocks that cannot matter to it: every query i of block u has
// P_iv <= n_u W_uv, so a block with n_u CK (W^_uv (1 + delta_u) + 4 2^-126)
// below P64_DROP carries less than P64_DROP / CK of every Z_i, all such
// blocks together less than P64_DROP.  Each Z_i then comes out between
// (1 - P64_DROP) Z_i and Z_i, each W^ of the row between W^ and
// W^ (1 + 2 P64_DROP): far inside float32's resolution, and far below the
// near-tie gaps the float64 selection is meant to resolve.  On clustered
// DiT activations only a few percent of the blocks of a row remain.
__device__ __forceinline__ void p64_dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ uint32_t p64_lds_addr(const void* p) {
  return (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)p;
}
typedef double f64x4_t __attribute__((ext_vector_type(4)));
constexpr double P64_DROP = 0x1p-33;

// exclusive scan of one int per thread over a 256-thread workgroup; `tmp`
// needs 4 ints
__device__ int wg256_exclusive(int x, int* tmp, int& total) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int inc = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  if (lane == 63) tmp[wid] = inc;
  __syncthreads();
  int pre = 0;
  total = 0;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int t = tmp[v];
    if (v < wid) pre += t;
    total += t;
  }
  __syncthreads();  // tmp is free for the next scan
  return pre + inc - x;
}

// W2: two wavefronts per SIMD (centroid blocks of a tile one after the other,
// registers within 256); otherwise one wavefront per SIMD with the two blocks
// of a tile unrolled together (shorter steps, for small item counts).
template <typename T, int D, bool W2>
__global__ __launch_bounds__(256, W2 ? 2 : 1) void k_pama64(const T* __restrict__ Qp,
                                                const int* __restrict__ q_offsets,
                                                const float* __restrict__ cen,
                                                const int* __restrict__ k_sizes, int H, int N,
                                                int CQ, int CK, const int4* __restrict__ items,
                                                int* __restrict__ cnt, double* __restrict__ part,
                                                double* __restrict__ W64, float* __restrict__ W32,
                                                const int* __restrict__ bandc,
                                                const int* __restrict__ kv_index,
                                                const float* __restrict__ wfast,
                                                const float* __restrict__ dfast, int plist,
                                                int* status) {
  constexpr int CT = 32, CPR = D / 4, RPI = 64 / CPR, NI = CT / (4 * RPI), KS = D / 4;
  static_assert(NI * 4 * RPI == CT, "tile shape");
  constexpr int NS = 3;  // centroid ring: one tile in flight while one is used
  __shared__ __attribute__((aligned(16))) float Ct[NS][CT * D];
  __shared__ double Lt[NS][CT];
  __shared__ double stg[2][4][CT];  // per-wavefront column sums of a tile (by step parity)
  extern __shared__ double wacc64[];  // [CK] column sums of the item, in chunk and wavefront order
  int* keep = (int*)(wacc64 + CK);    // [CK] blocks of the normaliser pass, ascending
  __shared__ int item_s, ktmp[4];
  const int tid = threadIdx.x, l = tid & 63, g = l >> 4, c16 = l & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const double isd = 1.0 / sqrt((double)D);
  const int ntf = (CK + CT - 1) / CT;
  const int pch = l % CPR;
  const int nall = H * CQ, per = (nall + 7) >> 3;
  for (int k = -1;;) {
    // next item: from the queue, or (no item list) this workgroup's one row,
    // rows of a head on one XCD
    int rid, cb = 0, ce = 1 << 30, slot = -1;
    if (items) {
      __syncthreads();  // the previous item is finished with LDS and item_s
      if (tid == 0) item_s = atomicAdd(&cnt[2], 1);
      __syncthreads();
      k = item_s;
      if (k >= cnt[0]) break;
      const int4 it = items[k];
      rid = it.x;
      cb = it.y;
      ce = it.z;
      slot = it.w;
    } else {
      if (k >= 0) break;
      k = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
      if (k >= nall) break;
      rid = k;
    }
    const int h = rid / CQ, u = rid - h * CQ;
    const float* ch = cen + (size_t)h * CK * D;
    const int* nh = k_sizes + (size_t)h * CK;
    const int* off = q_offsets + (size_t)h * (CQ + 1);
    const T* Qh = Qp + (size_t)h * N * D;
    // band rows: the probability pass covers only the listed (ambiguous)
    // blocks, which sit at the end of the row of kv_index; the normaliser
    // pass covers every block that can matter to it (n0 blocks: keep[], or
    // all of them)
    const int nb = bandc ? min(bandc[rid], CK) : -1;
    const int* blist = nb >= 0 ? kv_index + (size_t)rid * CK + (CK - nb) : nullptr;
    int nt2 = nb >= 0 ? (nb + CT - 1) / CT : ntf;
    int n0 = CK, nt = ntf;
    bool lst = false;
    // with plist, whole rows (top-p) take the list in the probability pass
    // too: the blocks left out weigh less than P64_DROP / n_u together, so a
    // cut at p < 1 - P64_DROP lies among the listed ones; theirs stay 0
    const bool pl = plist && nb < 0;
    // column of tile row r in a pass (-1: none)
    auto column = [&](int pass, int tile, int r) {
      const int ix = tile * CT + r;
      if (pass == 1 && nb >= 0) return ix < nb ? min(max(blist[ix], 0), CK - 1) : -1;
      if (pass == 0 || pl) return ix < n0 ? (lst ? keep[ix] : ix) : -1;
      return ix < CK ? ix : -1;
    };
    int Lc = nt + nt2;  // steps per chunk of 64 queries
    auto issue = [&](int step, int slot) {
      const int j = step % Lc, pass = j >= nt ? 1 : 0, tile = pass ? j - nt : j;
      // the step's columns first (list reads go out together), then the DMAs
      int vs[NI];
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int c = column(pass, tile, (w * NI + i) * RPI + l / CPR);
        vs[i] = c >= 0 ? c : CK - 1;
      }
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int r = (w * NI + i) * RPI + l / CPR;
        const float* src = ch + (size_t)vs[i] * D + 4 * (pch ^ (r & (CPR - 1)));
        p64_dma16(src, p64_lds_addr(&Ct[slot][0] + (w * NI + i) * 256));
      }
      if (tid < CT) {
        const int v = column(pass, tile, tid);
        const int n = v >= 0 ? nh[v] : 0;
        Lt[slot][tid] = n > 0 ? log((double)n) : -INFINITY;
      }
    };
    const int q0 = min(max(off[u], 0), N), q1 = min(max(off[u + 1], q0), N);
    const int nu = q1 - q0;
    const size_t wrow = (size_t)rid * CK;
    if (nu <= 0) {
      for (int v = tid; v < CK; v += 256) {
        if (W64) W64[wrow + v] = 0.0;
        if (W32) W32[wrow + v] = 0.0f;
      }
      continue;
    }
    __syncthreads();  // the previous item's column sums and block list have been read
    for (int v = tid; v < CK; v += 256) wacc64[v] = 0.0;
    if (wfast) {
      // the normaliser's blocks: thread t tests blocks 8t .. 8t + 7
      const float* wr = wfast + wrow;
      const double dl = (double)dfast[rid];
      const double thr = P64_DROP / ((double)nu * (double)CK);
      int fl = 0, c = 0;
      int ns[8];
      float ws8[8];  // loads first (clamped ids), so that they go out together
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int e = min(8 * tid + k, CK - 1);
        ns[k] = nh[e];
        ws8[k] = wr[e];
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int e = 8 * tid + k;
        // NaN / infinite bounds keep the block
        const bool kp = e < CK && ns[k] > 0 &&
                        !((double)ws8[k] * (1.0 + dl) + 4.0 * 1.1754943508222875e-38 < thr);
        fl |= (int)kp << k;
        c += kp;
      }
      int tot;
      int pos = wg256_exclusive(c, ktmp, tot);
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if ((fl >> k) & 1) keep[pos++] = 8 * tid + k;
      __syncthreads();
      if (tot > 0) {  // a row always holds a block of weight >= 1 / CK
        lst = true;
        n0 = tot;
        nt = (tot + CT - 1) / CT;
        if (pl) nt2 = nt;
        Lc = nt + nt2;
      }
    }
    const int nch = min(ce, (nu + 63) / 64) - cb;  // chunks of 64 queries from cb on
    const int total = nch * Lc;
    float qa[KS];  // float holds bf16 and float32 inputs exactly
    double m[4], z[4], mf[4];
    bool qv[4];
    issue(0, 0);
    if (total > 1) issue(1, 1);
    int prev_t = -1;  // the previous step's tile, when it was a probability-pass tile
    for (int it = 0; it < total; ++it) {
      const int j = it % Lc, pass = j >= nt ? 1 : 0, tile = pass ? j - nt : j;
      const int r0 = q0 + 64 * (cb + it / Lc);
      if (tile == 0 && pass == 0) {
        // A operand: query r0 + 16w + c16, dimensions 4s + g (loads from a
        // clamped row, so that they go out together; rows past the block 0)
        const int qi = r0 + 16 * w + c16;
        const T* qrow = Qh + (size_t)min(qi, q1 - 1) * D + g;
#pragma unroll
        for (int s = 0; s < KS; ++s) qa[s] = to_f(qrow[4 * s]);
#pragma unroll
        for (int s = 0; s < KS; ++s) qa[s] = qi < q1 ? qa[s] : 0.0f;
#pragma unroll
        for (int s = 0; s < KS; ++s) asm volatile("" ::"v"(qa[s]));
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          qv[r] = r0 + 16 * w + g + 4 * r < q1;  // this lane's output queries g + 4r
          m[r] = -INFINITY;
          z[r] = 0.0;
        }
      }
      if (tile == 0 && pass == 1) {
        // merge (max, sum) over the 16 lanes holding the same queries
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          double mm = m[r], zz = z[r];
#pragma unroll
          for (int o = 1; o < 16; o <<= 1) {
            const double om = __shfl_xor(mm, o, 64), oz = __shfl_xor(zz, o, 64);
            const double nm = fmax(mm, om);
            zz = (nm == -INFINITY) ? 0.0 : zz * exp(mm - nm) + oz * exp(om - nm);
            mm = nm;
          }
          // P = exp(S - (m + log z)); rows past the block get exp(-inf) = 0
          mf[r] = qv[r] && zz > 0.0 ? mm + log(zz) : INFINITY;
        }
      }
      // own DMAs of this tile done (the next one may stay in flight)
      if (it + 1 < total) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NI) : "memory");
      else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();  // tile landed everywhere; tile it-1 consumed (its slot is free)
      if (it + 2 < total) issue(it + 2, (it + 2) % NS);
      // the previous probability-pass tile's wavefront sums, in wavefront order
      if (prev_t >= 0 && tid < CT) {
        const int col = column(1, prev_t, tid);
        const double (*sg)[CT] = stg[(it - 1) & 1];
        if (col >= 0) wacc64[col] += ((sg[0][tid] + sg[1][tid]) + sg[2][tid]) + sg[3][tid];
      }
      const int slot = it % NS;
      const float* cs = &Ct[slot][0];
      if (r0 + 16 * w >= q1) {
        // no query of this wavefront is in the block (the last chunk of a
        // block that is not a multiple of 64): its column sums are zero, as
        // the exponentials of its rows would be, and its SIMD is left to the
        // other workgroup
        if (pass == 1 && g == 0) {
#pragma unroll
          for (int cb = 0; cb < CT / 16; ++cb) stg[it & 1][w][16 * cb + c16] = 0.0;
        }
        prev_t = pass == 1 ? tile : -1;
        continue;
      }
      constexpr int UNR = W2 ? 1 : CT / 16;
#pragma unroll UNR
      for (int cb = 0; cb < CT / 16; ++cb) {
        const int row = 16 * cb + c16;  // B operand: centroid row, dimension 4s + g
        const float* crow = cs + row * D + g;
        const int sw = row & (CPR - 1);
        float bf[KS];  // all LDS reads first, then the MFMA chains
#pragma unroll
        for (int s = 0; s < KS; ++s) bf[s] = crow[4 * (s ^ sw)];
        f64x4_t acc = {0.0, 0.0, 0.0, 0.0}, acc1 = acc;  // two chains (even / odd k-steps)
#pragma unroll
        for (int s = 0; s < KS; s += 2) {
          // widened next to their MFMA (the float64 copies would need twice the registers)
          float a0 = qa[s], a1 = qa[s + 1];
          asm volatile("" : "+v"(a0), "+v"(a1));
          acc = __builtin_amdgcn_mfma_f64_16x16x4f64((double)a0, (double)bf[s], acc, 0, 0, 0);
          acc1 = __builtin_amdgcn_mfma_f64_16x16x4f64((double)a1, (double)bf[s + 1], acc1, 0, 0, 0);
        }
        acc += acc1;
        const double lg = Lt[slot][row];  // this lane's centroid (column c16)
        if (pass == 0) {
          if (lg != -INFINITY) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              // one exp per logit: d = S - m; z += e^d (d <= 0), else z = z e^-d + 1, m = S
              const double sv = acc[r] * isd + lg;
              const double d = sv - m[r];
              const double e = exp(-fabs(d));
              z[r] = d <= 0.0 ? z[r] + e : fma(z[r], e, 1.0);
              m[r] = fmax(m[r], sv);
            }
          }
        } else {
          double cs4 = 0.0;
          if (lg != -INFINITY) {
#pragma unroll
            for (int r = 0; r < 4; ++r) cs4 += exp(fma(acc[r], isd, lg - mf[r]));
          }
          cs4 += __shfl_xor(cs4, 16, 64);
          cs4 += __shfl_xor(cs4, 32, 64);
          if (g == 0) stg[it & 1][w][row] = cs4;
        }
      }
      prev_t = pass == 1 ? tile : -1;
    }
    __syncthreads();
    if (prev_t >= 0 && tid < CT) {
      const int col = column(1, prev_t, tid);
      const double (*sg)[CT] = stg[(total - 1) & 1];
      if (col >= 0) wacc64[col] += ((sg[0][tid] + sg[1][tid]) + sg[2][tid]) + sg[3][tid];
    }
    __syncthreads();
    if (slot != -1) {  // part of a split row: raw column sums, added up by k_p64_combine
      double* dst = slot == -2 ? W64 + wrow : part + (size_t)slot * CK;
      for (int v = tid; v < CK; v += 256) dst[v] = wacc64[v];
    } else {
      const double inv_n = 1.0 / (double)nu;
      for (int v = tid; v < CK; v += 256) {
        const double wv = wacc64[v] * inv_n;
        if (!isfinite(wv)) raise_status(status, ST_NONFINITE);
        if (W64) W64[wrow + v] = wv;
        if (W32) W32[wrow + v] = (float)wv;
      }
    }
  }
}

// Query-centroid estimate (Sec. 4.1; the "w/o PAMA" variant of Sec. 6):
//   W^_uv = softmax_v (qbar_u . c_v / sqrt(d) + log n_v)
// for the float mean qbar_u of each nonempty query block (an empty block's
// row is 0), in float64.  The float64 MFMA tiles of k_pama64, but each of a
// tile's 64 query rows is a block of its own: a wavefront holds 16 blocks,
// the normaliser pass keeps an online (max, sum) per block, and the
// probability pass writes every block's row directly (no column sums).
// Workgroup = 64 consecutive blocks of one head, the workgroups of a head on
// one XCD.
template <int D>
__global__ __launch_bounds__(256, 2) void k_qcen64(const float* __restrict__ qbar,
                                                  const int* __restrict__ qsizes,
                                                  const float* __restrict__ cen,
                                                  const int* __restrict__ k_sizes, int H, int CQ,
                                                  int CK, double* __restrict__ W64,
                                                  float* __restrict__ W32,
                                                  float* __restrict__ delta, int* status) {
  constexpr int CT = 32, CPR = D / 4, RPI = 64 / CPR, NI = CT / (4 * RPI), KS = D / 4;
  static_assert(NI * 4 * RPI == CT, "tile shape");
  constexpr int NS = 3;  // centroid ring: one tile in flight while one is used
  __shared__ __attribute__((aligned(16))) float Ct[NS][CT * D];
  __shared__ double Lt[NS][CT];
  const int tid = threadIdx.x, l = tid & 63, g = l >> 4, c16 = l & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const double isd = 1.0 / sqrt((double)D);
  const int nt = (CK + CT - 1) / CT, total = 2 * nt;  // normaliser tiles, then probability tiles
  const int pch = l % CPR;
  const int nchunk = (CQ + 63) / 64, nall = H * nchunk, per = (nall + 7) >> 3;
  const int k = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (k >= nall) return;
  const int h = k / nchunk, u0 = 64 * (k - h * nchunk);
  const float* ch = cen + (size_t)h * CK * D;
  const int* nh = k_sizes + (size_t)h * CK;
  const int* qs = qsizes + (size_t)h * CQ;
  auto issue = [&](int step, int slot) {
    const int tile = step % nt;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = (w * NI + i) * RPI + l / CPR;
      const int v = min(tile * CT + r, CK - 1);
      const float* src = ch + (size_t)v * D + 4 * (pch ^ (r & (CPR - 1)));
      p64_dma16(src, p64_lds_addr(&Ct[slot][0] + (w * NI + i) * 256));
    }
    if (tid < CT) {
      const int v = tile * CT + tid;
      const int n = v < CK ? nh[v] : 0;
      Lt[slot][tid] = n > 0 ? log((double)n) : -INFINITY;
    }
  };
  // A operand: block u0 + 16w + c16, dimensions 4s + g
  float qa[KS];
  {
    const int ua = u0 + 16 * w + c16;
    const bool ok = ua < CQ && qs[min(ua, CQ - 1)] > 0;
    const float* qr = qbar + ((size_t)h * CQ + min(ua, CQ - 1)) * D;
#pragma unroll
    for (int s = 0; s < KS; ++s) qa[s] = qr[4 * s + g];  // loads together, then masked
#pragma unroll
    for (int s = 0; s < KS; ++s) qa[s] = ok ? qa[s] : 0.0f;
  }
  // this lane's output blocks g + 4r of the wavefront
  double m[4], z[4], mf[4];
  bool qv[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int uo = u0 + 16 * w + g + 4 * r;
    qv[r] = uo < CQ && qs[min(uo, CQ - 1)] > 0;
    m[r] = -INFINITY;
    z[r] = 0.0;
  }
  issue(0, 0);
  if (total > 1) issue(1, 1);
  for (int it = 0; it < total; ++it) {
    const int pass = it >= nt ? 1 : 0, tile = pass ? it - nt : it;
    if (it == nt) {
      // merge (max, sum) over the 16 lanes holding the same blocks
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        double mm = m[r], zz = z[r];
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          const double om = __shfl_xor(mm, o, 64), oz = __shfl_xor(zz, o, 64);
          const double nm = fmax(mm, om);
          zz = (nm == -INFINITY) ? 0.0 : zz * exp(mm - nm) + oz * exp(om - nm);
          mm = nm;
        }
        // P = exp(S - (m + log z)); empty blocks get exp(-inf) = 0
        mf[r] = qv[r] && zz > 0.0 ? mm + log(zz) : INFINITY;
        // the float row is the float64 one rounded once (2^-24), the float64
        // row within ~1e-13 of exact: 2^-23 bounds the float row's error
        const int uo = u0 + 16 * w + g + 4 * r;
        if (c16 == 0 && uo < CQ) delta[(size_t)h * CQ + uo] = 0x1p-23f;
      }
    }
    // own DMAs of this tile done (the next one may stay in flight)
    if (it + 1 < total) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NI) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();  // tile landed everywhere; tile it-1 consumed (its slot is free)
    if (it + 2 < total) issue(it + 2, (it + 2) % NS);
    if (u0 + 16 * w >= CQ) continue;  // no block of this wavefront (the head's last chunk)
    const int slot = it % NS;
    const float* cs = &Ct[slot][0];
#pragma unroll 1
    for (int cb = 0; cb < CT / 16; ++cb) {
      const int row = 16 * cb + c16;  // B operand: centroid row, dimension 4s + g
      const float* crow = cs + row * D + g;
      const int sw = row & (CPR - 1);
      float bf[KS];
#pragma unroll
      for (int s = 0; s < KS; ++s) bf[s] = crow[4 * (s ^ sw)];
      f64x4_t acc = {0.0, 0.0, 0.0, 0.0}, acc1 = acc;
#pragma unroll
      for (int s = 0; s < KS; s += 2) {
        float a0 = qa[s], a1 = qa[s + 1];
        asm volatile("" : "+v"(a0), "+v"(a1));
        acc = __builtin_amdgcn_mfma_f64_16x16x4f64((double)a0, (double)bf[s], acc, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f64_16x16x4f64((double)a1, (double)bf[s + 1], acc1, 0, 0, 0);
      }
      acc += acc1;
      const double lg = Lt[slot][row];
      if (pass == 0) {
        if (lg != -INFINITY) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const double sv = acc[r] * isd + lg;
            const double d = sv - m[r];
            const double e = exp(-fabs(d));
            z[r] = d <= 0.0 ? z[r] + e : fma(z[r], e, 1.0);
            m[r] = fmax(m[r], sv);
          }
        }
      } else {
        const int col = tile * CT + row;
        if (col < CK) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int uo = u0 + 16 * w + g + 4 * r;
            if (uo >= CQ) continue;
            const double pv = lg != -INFINITY ? exp(fma(acc[r], isd, lg - mf[r])) : 0.0;
            if (!isfinite(pv)) raise_status(status, ST_NONFINITE);
            const size_t o = ((size_t)h * CQ + uo) * CK + col;
            W64[o] = pv;
            W32[o] = (float)pv;
          }
        }
      }
    }
  }
}

// 1024-thread exclusive scan of one int per thread; `tmp` needs 16 ints.
__device__ int wg1024_exclusive(int x, int* tmp, int& total) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int inc = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  if (lane == 63) tmp[wid] = inc;
  __syncthreads();
  int pre = 0;
  total = 0;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int t = tmp[v];
    if (v < wid) pre += t;
    total += t;
  }
  __syncthreads();  // tmp is free for the next scan
  return pre + inc - x;
}

// Work list of the float64 pass over the listed rows.  Each row is cut into
// items of m chunks of 64 queries, m the smallest power of two for which the
// extra partial-sum rows (one per item after the first of a row) fit in
// `cap`; a row of one item is finished by its item.  items[k] = {h CQ + u,
// first chunk, end chunk, slot}: slot -1 finishes the row, -2 leaves the raw
// column sums in the row's W64 slot, s >= 0 in part[s].  srows[j] = {h CQ +
// u, first part slot, number of part slots, n_u} for every split row, in row
// order.  cnt = {items, split rows, queue head, 0}.  One workgroup.
__global__ __launch_bounds__(1024) void k_p64_plan(const int* __restrict__ q_offsets,
                                                   const int* __restrict__ rows,
                                                   const int* __restrict__ nrows, int H, int N,
                                                   int CQ, int cap, int4* __restrict__ items,
                                                   int4* __restrict__ srows, int* __restrict__ cnt) {
  constexpr int NM = 16;    // candidate m = 1, 2, 4, ..., 2^15
  constexpr int HG = 4096;  // heads per group (the listed rows are walked group by group)
  __shared__ int tmp[16];
  __shared__ long long red[16][NM];
  __shared__ int hp[HG + 1];
  __shared__ int m_s;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  // hp[k] = listed rows of heads h0 .. h0+k-1; returns the rows of the group
  auto head_prefix = [&](int h0, int nh) {
    int base = 0;
    for (int k0 = 0; k0 < nh; k0 += 1024) {
      const int k = k0 + tid;
      const int n = k < nh ? min(max(nrows[h0 + k], 0), CQ) : 0;
      int t;
      const int x = wg1024_exclusive(n, tmp, t);
      if (k < nh) hp[k] = base + x;
      base += t;
    }
    if (tid == 0) hp[nh] = base;
    __syncthreads();
    return base;
  };
  // listed row j of the group: head h, block u (-1: invalid) and its length
  auto row_at = [&](int h0, int nh, int j, int& h, int& u) {
    int lo = 0, hi = nh - 1;  // the last head whose rows start at or before j
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (hp[mid] <= j) lo = mid;
      else hi = mid - 1;
    }
    h = h0 + lo;
    u = rows[(size_t)h * CQ + (j - hp[lo])];
    if ((unsigned)u >= (unsigned)CQ) {
      u = -1;
      return 0;
    }
    const int* off = q_offsets + (size_t)h * (CQ + 1);
    const int a = min(max(off[u], 0), N), b = min(max(off[u + 1], a), N);
    return b - a;
  };
  long long e[NM];
#pragma unroll
  for (int j = 0; j < NM; ++j) e[j] = 0;
  for (int h0 = 0; h0 < H; h0 += HG) {
    const int nh = min(HG, H - h0);
    const int U = head_prefix(h0, nh);
    for (int j = tid; j < U; j += 1024) {
      int h, u;
      const int nch = (row_at(h0, nh, j, h, u) + 63) >> 6;
#pragma unroll
      for (int k = 0; k < NM; ++k) e[k] += nch > 0 ? ((nch - 1) >> k) : 0;
    }
  }
#pragma unroll
  for (int j = 0; j < NM; ++j) {
    long long x = e[j];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    if (lane == 0) red[wid][j] = x;
  }
  __syncthreads();
  if (tid == 0) {
    int m = 1 << 30;  // one item per row
    for (int j = NM - 1; j >= 0; --j) {
      long long t = 0;
      for (int v = 0; v < 16; ++v) t += red[v][j];
      if (t <= (long long)cap) m = 1 << j;
    }
    m_s = m;
  }
  __syncthreads();
  const int m = m_s;
  int ib = 0, sb = 0, rb = 0;  // items, part slots and split rows so far (uniform)
  for (int h0 = 0; h0 < H; h0 += HG) {
    const int nh = min(HG, H - h0);
    const int U = head_prefix(h0, nh);
    for (int j0 = 0; j0 < U; j0 += 1024) {
      int h = 0, u = -1, nu = 0;
      if (j0 + tid < U) nu = row_at(h0, nh, j0 + tid, h, u);
      const int nch = (nu + 63) >> 6;
      const int ns = u < 0 ? 0 : (nch > 0 ? (nch - 1) / m + 1 : 1);
      int t1, t2, t3;
      const int x1 = wg1024_exclusive(ns, tmp, t1);
      const int x2 = wg1024_exclusive(ns > 1 ? ns - 1 : 0, tmp, t2);
      const int x3 = wg1024_exclusive(ns > 1 ? 1 : 0, tmp, t3);
      const int rid = h * CQ + u;
      for (int k = 0; k < ns; ++k) {
        const int sl = ns == 1 ? -1 : (k == 0 ? -2 : sb + x2 + k - 1);
        items[ib + x1 + k] = make_int4(rid, k * m, k + 1 < ns ? (k + 1) * m : nch, sl);
      }
      if (ns > 1) srows[rb + x3] = make_int4(rid, sb + x2, ns - 1, nu);
      ib += t1;
      sb += t2;
      rb += t3;
    }
  }
  if (tid == 0) {
    cnt[0] = ib;
    cnt[1] = rb;
    cnt[2] = 0;
    cnt[3] = 0;
  }
}

// Rows split over several items: W^ = (raw sums in the W64 slot + the part
// slots, in item order) / n_u.  Grid-stride over the split rows.
__global__ __launch_bounds__(256) void k_p64_combine(const int4* __restrict__ srows,
                                                     const int* __restrict__ cnt,
                                                     const double* __restrict__ part, int CK,
                                                     double* __restrict__ W64,
                                                     float* __restrict__ W32, int* status) {
  const int nr = cnt[1];
  for (int r = blockIdx.x; r < nr; r += gridDim.x) {
    const int4 sr = srows[r];
    const double inv_n = 1.0 / (double)sr.w;
    double* wr = W64 + (size_t)sr.x * CK;
    for (int v = threadIdx.x; v < CK; v += 256) {
      double a = wr[v];
      for (int j = 0; j < sr.z; ++j) a += part[(size_t)(sr.y + j) * CK + v];
      const double wv = a * inv_n;
      if (!isfinite(wv)) raise_status(status, ST_NONFINITE);
      wr[v] = wv;
      if (W32) W32[(size_t)sr.x * CK + v] = (float)wv;
    }
  }
}

// ---------------------------------------------------------------- select
// One workgroup per (query block, head).  Valid key blocks are sorted by
// (W^ descending, id ascending) with an LDS bitonic sort; the kept prefix is
// then marked and compacted into ascending ids.
__device__ void select64_row(const double* __restrict__ W64, const int* __restrict__ q_offsets,
                             const int* __restrict__ k_sizes, int h, int u, int CQ, int CK, int P,
                             int mode, double param, int kcount, int* __restrict__ kv_count,
                             int* __restrict__ kv_index) {
  __shared__ double key[MAXC];
  __shared__ int id[MAXC];
  __shared__ int flag[MAXC];
  __shared__ int tmp[4];
  __shared__ int nvalid_s, m_s;
  const int tid = threadIdx.x;
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
    // a NaN weight (non-finite input, already reported) ranks as 0, as in the
    // fast selection, so the order stays total and the kept prefix only holds
    // valid ids
    const double wv = ok ? W64[row * CK + e] : -1.0;
    key[e] = ok ? (wv == wv ? wv : 0.0) : -1.0;
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
  __syncthreads();
}

// float64 selection of every query block, or (rows != null) of the listed ones.
__global__ __launch_bounds__(256) void k_select64(const double* __restrict__ W64,
                                                  const int* __restrict__ q_offsets,
                                                  const int* __restrict__ k_sizes, int CQ, int CK,
                                                  int P, int mode, double param, int kcount,
                                                  const int* __restrict__ rows,
                                                  const int* __restrict__ nrows,
                                                  int* __restrict__ kv_count,
                                                  int* __restrict__ kv_index,
                                                  const int* __restrict__ bandc) {
  const int h = blockIdx.y;
  const int cnt = rows ? min(nrows[h], CQ) : blockIdx.x + 1;
  const int step = rows ? gridDim.x : 1;
  for (int r = blockIdx.x; r < cnt; r += step) {
    const int u = rows ? rows[(size_t)h * CQ + r] : r;
    if ((unsigned)u >= (unsigned)CQ) continue;
    if (bandc && bandc[(size_t)h * CQ + u] >= 0) continue;  // k_select_band's row
    select64_row(W64, q_offsets, k_sizes, h, u, CQ, CK, P, mode, param, kcount, kv_count,
                 kv_index);
  }
}

// Top-k rows settled by their band (see select_topk_radix): the certain
// blocks (the row's first kv_count[row] entries) plus the top m - kv_count
// band blocks (the row's last bandc[row] entries) by float64 W^ (descending,
// ties to the lowest id), written in ascending id order.  The band is small:
// ranks by pairwise comparison.
__global__ __launch_bounds__(256) void k_select_band(const double* __restrict__ W64,
                                                     const int* __restrict__ k_sizes, int CQ,
                                                     int CK, int kcount,
                                                     const int* __restrict__ rows,
                                                     const int* __restrict__ nrows,
                                                     const int* __restrict__ bandc,
                                                     int* __restrict__ kv_count,
                                                     int* __restrict__ kv_index) {
  __shared__ int flag[MAXC];
  __shared__ int bid[MAXC];
  __shared__ double bval[MAXC];
  __shared__ int tmp[4];
  const int h = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int cnt = min(nrows[h], CQ);
  for (int r = blockIdx.x; r < cnt; r += gridDim.x) {
    const int u = rows[(size_t)h * CQ + r];
    if ((unsigned)u >= (unsigned)CQ) continue;
    const size_t row = (size_t)h * CQ + u;
    const int nb = min(bandc[row], CK);
    if (nb < 0) continue;
    const int nin = min(max(kv_count[row], 0), CK - nb);
    int* out = kv_index + row * CK;
    int nv = 0;
    for (int e = tid; e < CK; e += 256) {
      nv += k_sizes[(size_t)h * CK + e] > 0;
      flag[e] = 0;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) nv += __shfl_xor(nv, o, 64);
    __syncthreads();  // flag cleared; tmp free
    if (lane == 0) tmp[wid] = nv;
    for (int i = tid; i < nb; i += 256) {
      const int v = min(max(out[CK - nb + i], 0), CK - 1);
      const double x = W64[row * CK + v];
      bid[i] = v;
      bval[i] = x == x ? x : 0.0;  // a NaN weight (already reported) ranks as 0
    }
    for (int i = tid; i < nin; i += 256) flag[min(max(out[i], 0), CK - 1)] = 1;
    __syncthreads();
    const int nvalid = tmp[0] + tmp[1] + tmp[2] + tmp[3];
    const int m = min(max(kcount, 1), nvalid);
    const int need = m - nin;
    for (int i = tid; i < nb; i += 256) {
      const double x = bval[i];
      const int v = bid[i];
      int rank = 0;
      for (int j = 0; j < nb; ++j) rank += (bval[j] > x) || (bval[j] == x && bid[j] < v);
      if (rank < need) flag[v] = 1;
    }
    __syncthreads();
    for (int e = tid; e < CK; e += 256) bid[e] = flag[e];
    __syncthreads();
    block_exclusive_scan_2048(bid, CK, tmp);
    for (int e = tid; e < CK; e += 256)
      if (flag[e]) out[bid[e]] = e;
    if (tid == 0) kv_count[row] = m;
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Fast PAMA on bf16 MFMA (bf16 queries), with a per-row error bound.
//
// Centroids (float) are split into three bf16 parts, c = c1 + c2 + c3 + r with
// |r| <= 2^-24 |c|.  t = q.c is accumulated as q.(c2 + c3) in one chain over
// all dimensions plus q.c1 in 32-dimension segments, each a fresh
// accumulator except the last, which starts from the finished c2 + c3 chain;
// the D/32 segment results are added on the VALU.  With 2^-23 per MFMA
// addition and 2^-24 per VALU rounding,
//   |t^ - t| <= et |q| |c|,  et = 2^-24 1.01 + (32 2^-23 + (D/32-1) 2^-24) 1.01
//                                + 2^-8 1.01 (2D) 2^-23 + 2^-24 1.01
// (residual r; the c1 segments and their sum; the c2 + c3 chain; the last
// segment's 32 additions onto the seed, 32 2^-23 |q.(c2 + c3)| < 2^-24 |q||c|).
// The logit adds log2(e) log n_v, precomputed in float (k_cen_prep).
// The logit S = t/sqrt(d) + log n is formed with one FMA; its error
//   e_i = isd (et + 1.01 2^-24) |q_i| cmax + 1.01 2^-24 (2 lgmax + 1.01 isd |q_i| cmax)
// bounds every centroid of query i (cmax = max |c_v|, lgmax = max log n_v).
// Pass 1 keeps, per lane and query, an online (max, sum of exp2); lanes are
// merged at the end.  Pass 2 recomputes the logits and accumulates
// P = exp2((S - m) log2 e) / Z over the queries into per-wavefront LDS
// columns, which are added in wavefront order (deterministic).
// Relative error of each W^_uv:
//   delta_u = max_i (2.02 e_i + dZ_i + 2^-23 (3 + 1.5 argmax_i)) + 17 2^-24
// where argmax_i = 2 (isd |q_i| cmax + lgmax) log2 e bounds the exp2
// arguments (an argument x carries a relative exp2 error <= 2^-23 (2 + 1.5|x|))
// and dZ_i bounds the float normaliser (see the kernel); values below float's
// normal range carry an extra absolute error, handled by the selection.  Rows whose selection this bound cannot certify are recomputed
// in float64.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Splits the centroids into three bf16 planes and records log2(e) log n_v
// (-inf for empty blocks; the logits are in base 2), |c_v| rounded up, and
// per-block maxima of |c_v| and |log n_v|.
template <int D>
__global__ __launch_bounds__(256) void k_cen_prep(const float* __restrict__ cen,
                                                  const int* __restrict__ k_sizes, int CK,
                                                  bf16_t* __restrict__ c3, size_t plane,
                                                  float* __restrict__ lg, int CKpad,
                                                  float* __restrict__ cn,
                                                  float* __restrict__ bmax) {
  constexpr int CB = 16, TPC = 256 / CB, EPT = D / TPC;
  __shared__ float part[CB][TPC];
  const int h = blockIdx.y, v0 = blockIdx.x * CB, tid = threadIdx.x;
  const int r = tid / TPC, j = tid % TPC, v = v0 + r;
  float ss = 0.0f;
  if (v < CK) {
    const size_t o = ((size_t)h * CK + v) * D + j * EPT;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const float x = cen[o + e];
      const bf16_t p1 = f2bf(x);
      const float r1 = x - bf2f(p1);
      const bf16_t p2 = f2bf(r1);
      const float r2 = r1 - bf2f(p2);
      c3[o + e] = p1;
      c3[o + e + plane] = p2;
      c3[o + e + 2 * plane] = f2bf(r2);
      ss = fmaf(x, x, ss);
    }
  }
  part[r][j] = ss;
  __syncthreads();
  float fn = 0.0f, fl = 0.0f;
  if (tid < CB) {
    const int vv = v0 + tid;
    if (vv < CK) {
      float s2 = 0.0f;
      for (int q = 0; q < TPC; ++q) s2 += part[tid][q];
      fn = sqrtf(s2) * 1.0001f;
      const int n = k_sizes[(size_t)h * CK + vv];
      const float l = n > 0 ? (float)log((double)n) : -INFINITY;
      cn[(size_t)h * CK + vv] = fn;
      lg[(size_t)h * CKpad + vv] = l * 1.4426950408889634f;  // log2(e) log n, one rounding
      fl = n > 0 ? fabsf(l) : 0.0f;
    }
  }
  if (blockIdx.x == gridDim.x - 1)  // padding blocks: never scored
    for (int vv = CK + tid; vv < CKpad; vv += 256) lg[(size_t)h * CKpad + vv] = -INFINITY;
  if (tid < 64) {
    for (int o = 8; o > 0; o >>= 1) {
      fn = fmaxf(fn, __shfl_xor(fn, o, 64));
      fl = fmaxf(fl, __shfl_xor(fl, o, 64));
    }
    if (tid == 0) {
      bmax[((size_t)h * gridDim.x + blockIdx.x) * 2] = fn;
      bmax[((size_t)h * gridDim.x + blockIdx.x) * 2 + 1] = fl;
    }
  }
}

// One wave-wide LDS DMA (lane l's 16 bytes at g land at LDS byte lds + 16 l),
// as inline assembly so that the compiler does not drain every DMA in flight
// before each LDS read; completion is waited for explicitly.
__device__ __forceinline__ void pm_dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ uint32_t pm_lds_addr(const void* p) {
  return (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)p;
}
template <int D>
__device__ __forceinline__ int pm_swz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
// waits until at most N vector-memory operations of this wavefront are outstanding
template <int N>
__device__ __forceinline__ void pm_wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Work list of the fast retrieval: per head, every query block in chunks of
// 32 queries, in block order; a wavefront takes two consecutive chunks (they
// may belong to different blocks) and a workgroup eight.
// items[h][k] = {block u, chunk r, part slot (-1 for chunk 0), chunks of u};
// chunk 0 writes the block's row of W^, later chunks a row of `part`
// (slot = pstart[u] + r - 1), added up in chunk order by k_pama_combine.
// nitem[h] = number of items, pstart[h][u] = rows of `part` taken by the
// blocks before u (every chunk after a block's first takes one).  The
// per-row error bounds are cleared for the workgroups' atomic maxima.  One
// workgroup of 1024 threads per head, CQ <= 2048.
__global__ __launch_bounds__(1024) void k_pama_plan(const int* __restrict__ q_offsets, int N,
                                                    int CQ, int icap, int4* __restrict__ items,
                                                    int* __restrict__ nitem,
                                                    int* __restrict__ pstart,
                                                    float* __restrict__ delta) {
  __shared__ int st[MAXC + 1];
  __shared__ int ps[MAXC + 1];
  const int h = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int* off = q_offsets + (size_t)h * (CQ + 1);
  // two blocks per thread: chunks, then a workgroup scan
  int c[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int u = 2 * tid + k;
    c[k] = 0;
    if (u < CQ) {
      const int a = min(max(off[u], 0), N), b = min(max(off[u + 1], a), N);
      c[k] = (b - a + 31) >> 5;
      delta[(size_t)h * CQ + u] = 0.0f;
    }
  }
  // exclusive scans of the chunks (items) and of the chunks after the first
  // (part rows), packed in one 64-bit word (32 bits each)
  const int e0 = c[0] > 1 ? c[0] - 1 : 0, e1 = c[1] > 1 ? c[1] - 1 : 0;
  const long long sum = (long long)(c[0] + c[1]) | ((long long)(e0 + e1) << 32);
  long long inc = sum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const long long y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  __shared__ long long tmp64[16];
  if (lane == 63) tmp64[wid] = inc;
  __syncthreads();
  long long pre = inc - sum, tot = 0;
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    pre += q < wid ? tmp64[q] : 0;
    tot += tmp64[q];
  }
  const int pi = (int)(pre & 0xffffffffll), pp = (int)(pre >> 32);
  if (2 * tid < CQ) {
    st[2 * tid] = pi;
    ps[2 * tid] = pp;
  }
  if (2 * tid + 1 < CQ) {
    st[2 * tid + 1] = pi + c[0];
    ps[2 * tid + 1] = pp + e0;
  }
  if (tid == 0) {
    st[CQ] = (int)(tot & 0xffffffffll);
    ps[CQ] = (int)(tot >> 32);
  }
  __syncthreads();
  const int tot_items = st[CQ];
  for (int u = tid; u <= CQ; u += 1024) pstart[(size_t)h * (CQ + 1) + u] = ps[u];
  if (tid == 0) nitem[h] = min(tot_items, icap);
  const int T = min(tot_items, icap);
  for (int k = tid; k < T; k += 1024) {
    int lo = 0, hi = CQ - 1;  // the last block whose items start at or before k
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (st[mid] <= k) lo = mid;
      else hi = mid - 1;
    }
    const int r = k - st[lo], nr = st[lo + 1] - st[lo];
    items[(size_t)h * icap + k] = make_int4(lo, r, r == 0 ? -1 : ps[lo] + r - 1, nr);
  }
}

// Fast retrieval.  A workgroup takes four items of one head (one round of 64
// queries of a query block per wavefront, from the plan) and streams the
// head's key-block centroids through an NS-slot LDS ring (32 rows of the
// three bf16 parts per tile, LDS DMA, rows swizzled in 16-byte chunks),
// twice: pass 1 builds each query's normaliser, pass 2 sums the
// probabilities over the round's queries.  Every tile serves 256 queries.
//
// MFMA 32x32x16 on two 32-query groups per wavefront.  The query fragment
// (query l%32, dims 16 s + 8 (l/32) ..) and the centroid fragment (centroid
// l%32, same dims) serve as either operand, so pass 1 computes S^T (lane:
// one query, centroids 8b + 4(l/32) + r) and pass 2 computes S (lane: one
// centroid, queries 8b + 4(l/32) + r); each pass then reduces within lanes.
// Accuracy as in the float error bound below: the c1 part is accumulated in
// 32-dimension segments (two MFMAs from zero) added in float, the two small
// parts in one chain over all dimensions.
//
// Scores are kept in log2 units, s' = (q.c / sqrt(d) + log n_v) log2 e.
// Pass 1 keeps per query a reference maximum m and z = sum 2^(s' - m) (one
// rescale per tile, tile terms added in a tree); pass 2 uses
// c_q = m + log2 z, so p = 2^(s' - c_q).
template <int D>
__global__ __launch_bounds__(256, 2) void k_pama_fast(const bf16_t* __restrict__ Qp,
                                                      const int* __restrict__ q_offsets,
                                                      const int4* __restrict__ items,
                                                      const int* __restrict__ nitem, int icap,
                                                      float* __restrict__ part, int pcap,
                                                      const bf16_t* __restrict__ c3, size_t plane,
                                                      const float* __restrict__ lg, int CKpad,
                                                      const float* __restrict__ bmax, int nbm, int H,
                                                      int N, int CQ, int CK, float* __restrict__ W32,
                                                      float* __restrict__ delta) {
  constexpr int CT = 32, KS = D / 16, CPR = D / 8, RPI = 64 / CPR;
  constexpr int NI = 3 * CT / (4 * RPI);  // DMAs per wavefront and tile
  static_assert(NI * 4 * RPI == 3 * CT && KS % 2 == 0, "tile shape");
  constexpr int NS = 3;
  constexpr float U24 = 5.9604645e-08f, DEL = 1.1920929e-07f, L2E = 1.4426950408889634f;
  constexpr float ET = U24 * 1.01f + (32.0f * DEL + (KS / 2 - 1) * U24) * 1.01f +
                       0.00390625f * 1.01f * (2 * D) * DEL + U24 * 1.01f;
  __shared__ __attribute__((aligned(16))) bf16_t Ct[NS][3 * CT * D];  // [slot][part][row][D]
  __shared__ __attribute__((aligned(16))) float Lt[NS][CT];
  __shared__ __attribute__((aligned(16))) float cbuf[4][64];  // c_q of each wavefront's chunk
  __shared__ float mx_s[2];
  // workgroups of a head on one XCD (its L2 holds the head's centroids)
  const int G = (icap + 7) / 8, nwgs = G * H, per = (nwgs + 7) >> 3;
  const int wgi = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (wgi >= nwgs) return;
  const int h = wgi / G, grp8 = wgi - h * G;
  const int T = min(nitem[h], icap);
  if (8 * grp8 >= T) return;
  const int tid = threadIdx.x, l = tid & 63, hf = l >> 5, c32 = l & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int* off = q_offsets + (size_t)h * (CQ + 1);
  // this wavefront's two chunks (group g: queries q0[g] + 32 rc[g] + l % 32)
  int ug[2], rc[2], q0[2], q1[2], nu[2];
  float* orow[2];
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    const int k = 8 * grp8 + 2 * w + g;
    const int4 itm = k < T ? items[(size_t)h * icap + k] : make_int4(-1, 0, -1, 0);
    const int u = (unsigned)itm.x < (unsigned)CQ ? itm.x : -1;
    ug[g] = u;
    rc[g] = itm.y;
    q0[g] = u >= 0 ? min(max(off[u], 0), N) : 0;
    q1[g] = u >= 0 ? min(max(off[u + 1], q0[g]), N) : 0;
    nu[g] = q1[g] - q0[g];
    if (u >= 0 && 32 * rc[g] < nu[g] && rc[g] == 0) orow[g] = W32 + ((size_t)h * CQ + u) * CK;
    else if (u >= 0 && 32 * rc[g] < nu[g] && itm.z >= 0 && itm.z < pcap)
      orow[g] = part + ((size_t)h * pcap + itm.z) * CK;
    else orow[g] = nullptr;
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
  __syncthreads();
  const float cmax = mx_s[0], lgmax = mx_s[1];
  const float isd = 1.0f / sqrtf((float)D), isdL = isd * L2E;
  const bf16_t* P1 = c3 + (size_t)h * CK * D;
  const float* lgh = lg + (size_t)h * CKpad;
  const int pch = l % CPR;
  const int nt = (CK + CT - 1) / CT;
  auto issue = [&](int tile, int slot) {
    const int c0 = tile * CT;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int row = (w * NI + i) * RPI + l / CPR;
      const int part = row / CT, r = row % CT;
      const int v = min(c0 + r, CK - 1);
      const bf16_t* src = P1 + part * plane + (size_t)v * D + 8 * (pch ^ pm_swz<D>(r));
      pm_dma16(src, pm_lds_addr(&Ct[slot][0] + (w * NI + i) * 512));
    }
    if (w == 0 && l < CT / 4) pm_dma16(lgh + c0 + 4 * l, pm_lds_addr(&Lt[slot][0]));
  };
  // the centroid fragment of this lane: row c32 of a tile, dims 16 s + 8 hf ..
  const int crow = c32 * D, cswz = pm_swz<D>(c32);

  float dmax[2] = {0.0f, 0.0f};  // relative error bound of each chunk
  const int total = 2 * nt;
#pragma unroll
  for (int p = 0; p < NS - 1; ++p)
    if (p < total) issue(p % nt, p);
  // ring step of tile `it`: own DMAs done, barrier, next tile issued; its slot
  int it = 0;
  auto ring_step = [&]() {
    if (it + 1 < total) {
      if (w == 0) pm_wait_vmcnt<NI + 1>();
      else pm_wait_vmcnt<NI>();
    } else {
      pm_wait_vmcnt<0>();
    }
    __syncthreads();  // tile landed everywhere; the tile before consumed (its slot is free)
    if (it + NS - 1 < total) issue((it + NS - 1) % nt, (it + NS - 1) % NS);
    return it % NS;
  };
  // products of both query groups with one tile: S^T (pass 1: lane = query,
  // 16 centroids) or S (pass 2: lane = centroid, 16 queries); c2 + c3 in one
  // chain over all dimensions, c1 in 32-dimension segments (two MFMAs from
  // zero, the last from the finished c2 + c3 chain) added in float
  auto products = [&](const bf16x8_t (*q2)[KS], const bf16_t* B1, bool qa_left, f32x16_t* hi) {
    const bf16_t* B2 = B1 + CT * D;
    const bf16_t* B3 = B2 + CT * D;
    constexpr int LS = KS / 2 - 1;  // the last segment
    auto mm = [&](const bf16x8_t& b, const bf16x8_t& q, const f32x16_t& c) {
      return qa_left ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(q, b, c, 0, 0, 0)
                     : __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, q, c, 0, 0, 0);
    };
    f32x16_t rest[2];
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int q = 0; q < 16; ++q) rest[g][q] = 0.0f;
    bf16x8_t bl[2];  // c1 fragments of the last segment
#pragma unroll
    for (int sp = 0; sp < KS / 2; ++sp) {
      f32x16_t seg[2];
#pragma unroll
      for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int q = 0; q < 16; ++q) seg[g][q] = 0.0f;
#pragma unroll
      for (int s = 2 * sp; s < 2 * sp + 2; ++s) {
        const int co = crow + 8 * ((2 * s + hf) ^ cswz);
        const bf16x8_t b1 = *(const bf16x8_t*)(B1 + co);
        const bf16x8_t b2 = *(const bf16x8_t*)(B2 + co);
        const bf16x8_t b3 = *(const bf16x8_t*)(B3 + co);
        if (sp == LS) bl[s - 2 * sp] = b1;
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          if (sp < LS) seg[g] = mm(b1, q2[g][s], seg[g]);
          rest[g] = mm(b2, q2[g][s], rest[g]);
          rest[g] = mm(b3, q2[g][s], rest[g]);
        }
      }
      if (sp < LS) {
#pragma unroll
        for (int g = 0; g < 2; ++g) hi[g] = sp == 0 ? seg[g] : hi[g] + seg[g];
      }
    }
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      f32x16_t seg = rest[g];
#pragma unroll
      for (int s = 2 * LS; s < 2 * LS + 2; ++s) seg = mm(bl[s - 2 * LS], q2[g][s], seg);
      hi[g] = LS == 0 ? seg : hi[g] + seg;
    }
  };
  bf16x8_t qf[2][KS];
  {
    bool ong[2];
#pragma unroll
    for (int g = 0; g < 2; ++g) ong[g] = orow[g] != nullptr;
    const bool on = ong[0] || ong[1];
    float m[2], z[2];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const int qa = q0[g] + 32 * rc[g] + c32;
      const bool qv = ong[g] && qa < q1[g];
      float qsq = 0.0f;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        uint4 raw = make_uint4(0u, 0u, 0u, 0u);
        if (qv) raw = *(const uint4*)(Qp + ((size_t)h * N + qa) * D + 16 * s + 8 * hf);
        qf[g][s] = __builtin_bit_cast(bf16x8_t, raw);
        asm volatile("" ::"v"(qf[g][s]));  // loads complete here, not inside the ring waits
        const uint32_t q[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = __uint_as_float(q[e] << 16), hi = __uint_as_float(q[e] & 0xffff0000u);
          qsq = fmaf(lo, lo, fmaf(hi, hi, qsq));
        }
      }
      qsq += __shfl_xor(qsq, 32, 64);
      if (qv) {
        // row error bound of this query (|q| rounded up)
        const float qn = sqrtf(qsq) * 1.0001f;
        const float ei = isd * (ET + 1.01f * U24) * qn * cmax +
                         1.01f * U24 * (3.0f * lgmax + 2.02f * isd * qn * cmax);
        const float argmax = 2.0f * (isd * qn * cmax + lgmax) * L2E;
        const float nadd = fmaxf((float)(CK / 16 + 1), (float)(CK / 32 + 5));
        const float dZ = DEL * (10.0f + 3.0f * log2f((float)CK + 1.0f) + 2.0f * nadd +
                                3.0f * argmax) +
                         2.0f * U24 * (nadd + 24.0f);
        dmax[g] = fmaxf(dmax[g], 2.02f * ei + dZ +
                                     DEL * (3.0f + 2.5f * argmax + 2.0f * log2f((float)CK + 1.0f)));
      }
      m[g] = -INFINITY;
      z[g] = 0.0f;
    }
    // pass 1: lane holds query c32 of each group, centroids c0 + 8b + 4hf + r
    for (int tile = 0; tile < nt; ++tile, ++it) {
      const int slot = ring_step();
      if (!on) continue;
      f32x16_t hi[2];
      products(qf, &Ct[slot][0], false, hi);
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        float sv[16];
#pragma unroll
        for (int bq = 0; bq < 4; ++bq) {
          const float4 l4 = *(const float4*)(&Lt[slot][8 * bq + 4 * hf]);
          const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
          for (int r = 0; r < 4; ++r)
            sv[4 * bq + r] = fmaf(hi[g][4 * bq + r], isdL, lv[r]);
        }
        float tmax = fmaxf(sv[0], sv[1]);
#pragma unroll
        for (int q = 2; q < 16; ++q) tmax = fmaxf(tmax, sv[q]);
        const float mn = fmaxf(m[g], tmax);
        if (mn != -INFINITY) {
#pragma unroll
          for (int q = 0; q < 16; ++q) sv[q] = __builtin_amdgcn_exp2f(sv[q] - mn);
#pragma unroll
          for (int o = 8; o > 0; o >>= 1)
#pragma unroll
            for (int q = 0; q < o; ++q) sv[q] += sv[q + o];
          z[g] = (m[g] == mn ? z[g] : z[g] * __builtin_amdgcn_exp2f(m[g] - mn)) + sv[0];
          m[g] = mn;
        }
      }
    }
    // c_q = m + log2 z per query (halves merged); invalid queries +inf
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const float om = __shfl_xor(m[g], 32, 64), oz = __shfl_xor(z[g], 32, 64);
      const float M = fmaxf(m[g], om);
      float zz = 0.0f;
      if (M != -INFINITY)
        zz = z[g] * __builtin_amdgcn_exp2f(m[g] - M) + oz * __builtin_amdgcn_exp2f(om - M);
      const int qa = q0[g] + 32 * rc[g] + c32;
      const float c = (ong[g] && qa < q1[g] && zz > 0.0f) ? M + __builtin_amdgcn_logf(zz) : INFINITY;
      if (hf == 0) cbuf[w][32 * g + c32] = c;
    }
    // pass 2: lane holds centroid c0 + c32, queries 8b + 4hf + r of each group
    for (int tile = 0; tile < nt; ++tile, ++it) {
      const int slot = ring_step();
      if (!on) continue;
      const float lgj = Lt[slot][c32];
      float ws[2];
      f32x16_t hi[2];
      products(qf, &Ct[slot][0], true, hi);
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        float e[16];
#pragma unroll
        for (int bq = 0; bq < 4; ++bq) {
          const float4 c4 = *(const float4*)(&cbuf[w][32 * g + 8 * bq + 4 * hf]);
          const float cv[4] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
          for (int r = 0; r < 4; ++r)
            e[4 * bq + r] = __builtin_amdgcn_exp2f(
                fmaf(hi[g][4 * bq + r], isdL, lgj) - cv[r]);
        }
#pragma unroll
        for (int o = 8; o > 0; o >>= 1)
#pragma unroll
          for (int q = 0; q < o; ++q) e[q] += e[q + o];
        ws[g] = e[0] + __shfl_xor(e[0], 32, 64);
      }
      // lanes of half g write chunk g's sums
      const int v = tile * CT + c32;
      float* dst = hf ? orow[1] : orow[0];
      if (dst && v < CK) dst[v] = (hf ? ws[1] : ws[0]) / (float)(hf ? nu[1] : nu[0]);
    }
  }
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    if (orow[g]) {
      // the row's bound: the largest over its chunks (non-negative floats
      // order as their bit patterns), finished by k_pama_combine
      float dm = dmax[g];
      for (int o = 32; o > 0; o >>= 1) dm = fmaxf(dm, __shfl_xor(dm, o, 64));
      if (l == 0) atomicMax((int*)&delta[(size_t)h * CQ + ug[g]], __float_as_int(dm));
    }
  }
}

// centroid tiles of the single-sweep retrieval (its logits stay in registers)
constexpr int FULLK_NT = 8;

// Full-K retrieval (Alg. 1) for small key-block counts (CK <= 32 FK_NT): one
// sweep over the centroids instead of two.  A wavefront takes one 32-query
// chunk (items as in the fast retrieval, four per workgroup) and computes S^T
// (lane: one query, 16 of each tile's 32 centroids) exactly as the fast
// path's first pass, keeping every final logit of its query row in
// registers; the online normaliser (m, z) is the fast path's, so the row
// bound delta_u is the same.  The probabilities then come from the kept
// logits, and each centroid's sum over the chunk's 32 queries is a fixed
// five-level butterfly over the lanes (the fast path's pass 2 sums the same
// values in a five-level tree), written to the chunk's row as before.
template <int D, int FK_NT>
__global__ __launch_bounds__(256, 2) void k_pama_fullk(const bf16_t* __restrict__ Qp,
                                                       const int* __restrict__ q_offsets,
                                                       const int4* __restrict__ items,
                                                       const int* __restrict__ nitem, int icap,
                                                       float* __restrict__ part, int pcap,
                                                       const bf16_t* __restrict__ c3,
                                                       size_t plane, const float* __restrict__ lg,
                                                       int CKpad, const float* __restrict__ bmax,
                                                       int nbm, int H, int N, int CQ, int CK,
                                                       float* __restrict__ W32,
                                                       float* __restrict__ delta) {
  constexpr int CT = 32, KS = D / 16, CPR = D / 8, RPI = 64 / CPR;
  constexpr int NI = 3 * CT / (4 * RPI);  // DMAs per wavefront and tile
  static_assert(NI * 4 * RPI == 3 * CT && KS % 2 == 0, "tile shape");
  constexpr int NS = 3;
  constexpr float U24 = 5.9604645e-08f, DEL = 1.1920929e-07f, L2E = 1.4426950408889634f;
  constexpr float ET = U24 * 1.01f + (32.0f * DEL + (KS / 2 - 1) * U24) * 1.01f +
                       0.00390625f * 1.01f * (2 * D) * DEL + U24 * 1.01f;
  __shared__ __attribute__((aligned(16))) bf16_t Ct[NS][3 * CT * D];  // [slot][part][row][D]
  __shared__ __attribute__((aligned(16))) float Lt[NS][CT];
  __shared__ float mx_s[2];
  // workgroups of a head on one XCD (its L2 holds the head's centroids)
  const int G = (icap + 3) / 4, nwgs = G * H, per = (nwgs + 7) >> 3;
  const int wgi = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (wgi >= nwgs) return;
  const int h = wgi / G, grp4 = wgi - h * G;
  const int T = min(nitem[h], icap);
  if (4 * grp4 >= T) return;
  const int tid = threadIdx.x, l = tid & 63, hf = l >> 5, c32 = l & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int* off = q_offsets + (size_t)h * (CQ + 1);
  // this wavefront's chunk: queries q0 + 32 rc + l % 32
  const int k = 4 * grp4 + w;
  const int4 itm = k < T ? items[(size_t)h * icap + k] : make_int4(-1, 0, -1, 0);
  const int u = (unsigned)itm.x < (unsigned)CQ ? itm.x : -1;
  const int rc = itm.y;
  const int q0 = u >= 0 ? min(max(off[u], 0), N) : 0;
  const int q1 = u >= 0 ? min(max(off[u + 1], q0), N) : 0;
  const int nu = q1 - q0;
  float* orow = nullptr;
  if (u >= 0 && 32 * rc < nu) {
    if (rc == 0) orow = W32 + ((size_t)h * CQ + u) * CK;
    else if (itm.z >= 0 && itm.z < pcap) orow = part + ((size_t)h * pcap + itm.z) * CK;
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
  __syncthreads();
  const float cmax = mx_s[0], lgmax = mx_s[1];
  const float isd = 1.0f / sqrtf((float)D), isdL = isd * L2E;
  const bf16_t* P1 = c3 + (size_t)h * CK * D;
  const float* lgh = lg + (size_t)h * CKpad;
  const int pch = l % CPR;
  const int nt = (CK + CT - 1) / CT;  // <= FK_NT (the launcher checks)
  auto issue = [&](int tile, int slot) {
    const int c0 = tile * CT;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int row = (w * NI + i) * RPI + l / CPR;
      const int part = row / CT, r = row % CT;
      const int v = min(c0 + r, CK - 1);
      const bf16_t* src = P1 + part * plane + (size_t)v * D + 8 * (pch ^ pm_swz<D>(r));
      pm_dma16(src, pm_lds_addr(&Ct[slot][0] + (w * NI + i) * 512));
    }
    if (w == 0 && l < CT / 4) pm_dma16(lgh + c0 + 4 * l, pm_lds_addr(&Lt[slot][0]));
  };
  const int crow = c32 * D, cswz = pm_swz<D>(c32);
  const bool on = orow != nullptr;
  // the query fragment and the row bound of this lane's query
  const int qa = q0 + 32 * rc + c32;
  const bool qv = on && qa < q1;
  bf16x8_t qf[KS];
  float dmax = 0.0f;
  {
    float qsq = 0.0f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      uint4 raw = make_uint4(0u, 0u, 0u, 0u);
      if (qv) raw = *(const uint4*)(Qp + ((size_t)h * N + qa) * D + 16 * s + 8 * hf);
      qf[s] = __builtin_bit_cast(bf16x8_t, raw);
      asm volatile("" ::"v"(qf[s]));  // loads complete here, not inside the ring waits
      const uint32_t q[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float lo = __uint_as_float(q[e] << 16), hi = __uint_as_float(q[e] & 0xffff0000u);
        qsq = fmaf(lo, lo, fmaf(hi, hi, qsq));
      }
    }
    qsq += __shfl_xor(qsq, 32, 64);
    if (qv) {
      // the row error bound of this query, as in the fast path
      const float qn = sqrtf(qsq) * 1.0001f;
      const float ei = isd * (ET + 1.01f * U24) * qn * cmax +
                       1.01f * U24 * (3.0f * lgmax + 2.02f * isd * qn * cmax);
      const float argmax = 2.0f * (isd * qn * cmax + lgmax) * L2E;
      const float nadd = fmaxf((float)(CK / 16 + 1), (float)(CK / 32 + 5));
      const float dZ = DEL * (10.0f + 3.0f * log2f((float)CK + 1.0f) + 2.0f * nadd +
                              3.0f * argmax) +
                       2.0f * U24 * (nadd + 24.0f);
      dmax = 2.02f * ei + dZ + DEL * (3.0f + 2.5f * argmax + 2.0f * log2f((float)CK + 1.0f));
    }
  }
#pragma unroll
  for (int p = 0; p < NS - 1; ++p)
    if (p < nt) issue(p, p);
  // the sweep: S^T of each tile (lane: query c32, centroids 8b + 4hf + r),
  // kept in registers, and the online normaliser
  float L[FK_NT][16];
  float m = -INFINITY, z = 0.0f;
#pragma unroll
  for (int tile = 0; tile < FK_NT; ++tile) {
    if (tile < nt) {
      if (tile + 1 < nt) {
        if (w == 0) pm_wait_vmcnt<NI + 1>();
        else pm_wait_vmcnt<NI>();
      } else {
        pm_wait_vmcnt<0>();
      }
      __syncthreads();  // tile landed everywhere; the tile before consumed (its slot is free)
      if (tile + NS - 1 < nt) issue(tile + NS - 1, (tile + NS - 1) % NS);
      const int slot = tile % NS;
      if (!on) continue;  // no chunk: the ring steps only
      const bf16_t* B1 = &Ct[slot][0];
      const bf16_t* B2 = B1 + CT * D;
      const bf16_t* B3 = B2 + CT * D;
      // c2 + c3 in one chain, c1 in 32-dimension segments (the last one
      // from the finished c2 + c3 chain) added in float, as the fast path
      constexpr int LS = KS / 2 - 1;
      f32x16_t hi, rest;
#pragma unroll
      for (int q = 0; q < 16; ++q) rest[q] = 0.0f;
      bf16x8_t bl[2];
#pragma unroll
      for (int sp = 0; sp < KS / 2; ++sp) {
        f32x16_t seg;
#pragma unroll
        for (int q = 0; q < 16; ++q) seg[q] = 0.0f;
#pragma unroll
        for (int s = 2 * sp; s < 2 * sp + 2; ++s) {
          const int co = crow + 8 * ((2 * s + hf) ^ cswz);
          const bf16x8_t b1 = *(const bf16x8_t*)(B1 + co);
          const bf16x8_t b2 = *(const bf16x8_t*)(B2 + co);
          const bf16x8_t b3 = *(const bf16x8_t*)(B3 + co);
          if (sp == LS) bl[s - 2 * sp] = b1;
          else seg = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b1, qf[s], seg, 0, 0, 0);
          rest = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b2, qf[s], rest, 0, 0, 0);
          rest = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b3, qf[s], rest, 0, 0, 0);
        }
        if (sp < LS) hi = sp == 0 ? seg : hi + seg;
      }
      {
        f32x16_t seg = rest;
#pragma unroll
        for (int s = 2 * LS; s < 2 * LS + 2; ++s)
          seg = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bl[s - 2 * LS], qf[s], seg, 0, 0, 0);
        hi = LS == 0 ? seg : hi + seg;
      }
#pragma unroll
      for (int bq = 0; bq < 4; ++bq) {
        const float4 l4 = *(const float4*)(&Lt[slot][8 * bq + 4 * hf]);
        const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
        for (int r = 0; r < 4; ++r)
          L[tile][4 * bq + r] = fmaf(hi[4 * bq + r], isdL, lv[r]);
      }
      {
        float tmax = fmaxf(L[tile][0], L[tile][1]);
#pragma unroll
        for (int q = 2; q < 16; ++q) tmax = fmaxf(tmax, L[tile][q]);
        const float mn = fmaxf(m, tmax);
        if (mn != -INFINITY) {
          float sv[16];
#pragma unroll
          for (int q = 0; q < 16; ++q) sv[q] = __builtin_amdgcn_exp2f(L[tile][q] - mn);
#pragma unroll
          for (int o = 8; o > 0; o >>= 1)
#pragma unroll
            for (int q = 0; q < o; ++q) sv[q] += sv[q + o];
          z = (m == mn ? z : z * __builtin_amdgcn_exp2f(m - mn)) + sv[0];
          m = mn;
        }
      }
    }
  }
  // c_q = m + log2 z per query (the two halves of a query merged); invalid
  // queries +inf, so their probabilities are zero
  float cq;
  {
    const float om = __shfl_xor(m, 32, 64), oz = __shfl_xor(z, 32, 64);
    const float M = fmaxf(m, om);
    float zz = 0.0f;
    if (M != -INFINITY) zz = z * __builtin_amdgcn_exp2f(m - M) + oz * __builtin_amdgcn_exp2f(om - M);
    cq = (qv && zz > 0.0f) ? M + __builtin_amdgcn_logf(zz) : INFINITY;
  }
  // probabilities from the kept logits, summed over the chunk's 32 queries
  // per centroid: each tile's 32 x 32 probabilities go through LDS (this
  // wavefront's part of the ring, free after the sweep) from query lanes to
  // centroid lanes; lane (c, half) sums queries 16 half .. 16 half + 15 of
  // centroid c in a four-level tree and adds the other half's sum (the
  // five-level depth of the fast path's in-chunk sums)
  __syncthreads();  // every wavefront is done with the ring
  if (on) {
    constexpr int TS = 36;  // row stride (floats) of the transpose buffer
    float* tb = (float*)&Ct[0][0] + w * (32 * TS);
    const float fnu = (float)nu;
#pragma unroll
    for (int tile = 0; tile < FK_NT; ++tile) {
      if (tile < nt) {
        float e[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) e[q] = __builtin_amdgcn_exp2f(L[tile][q] - cq);
        // lane (query c32, hf) holds centroids 8b + 4hf + r
#pragma unroll
        for (int b = 0; b < 4; ++b)
          *(float4*)&tb[c32 * TS + 8 * b + 4 * hf] =
              make_float4(e[4 * b], e[4 * b + 1], e[4 * b + 2], e[4 * b + 3]);
        float x[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) x[j] = tb[(16 * hf + j) * TS + c32];
#pragma unroll
        for (int o = 8; o > 0; o >>= 1)
#pragma unroll
          for (int j = 0; j < o; ++j) x[j] += x[j + o];
        const float other = __shfl_xor(x[0], 32, 64);
        const float sum = hf ? other + x[0] : x[0] + other;
        const int v = tile * CT + c32;
        if (hf == 0 && v < CK) orow[v] = sum / fnu;
      }
    }
    // the row's bound: the largest over its chunks, finished by k_pama_combine
    float dm = dmax;
    for (int o = 32; o > 0; o >>= 1) dm = fmaxf(dm, __shfl_xor(dm, o, 64));
    if (l == 0) atomicMax((int*)&delta[(size_t)h * CQ + u], __float_as_int(dm));
  }
}

// Rows of the fast retrieval: W^ = chunk 0 + chunk 1 + ... in chunk order,
// empty blocks a zero row; the bound becomes delta_u = (max over chunks +
// (17 + 2 chunks) 2^-24) 1.01.  One workgroup per (query block, head).
__global__ __launch_bounds__(256) void k_pama_combine(const int* __restrict__ q_offsets,
                                                      const int* __restrict__ pstart, int H,
                                                      int N, int CQ, int CK,
                                                      const float* __restrict__ part, int pcap,
                                                      float* __restrict__ W32,
                                                      float* __restrict__ delta) {
  constexpr float U24 = 5.9604645e-08f;
  constexpr int E = MAXC / 256;  // columns per thread, loads issued together
  const int h = blockIdx.y, u = blockIdx.x, row = h * CQ + u;
  const int* off = q_offsets + (size_t)h * (CQ + 1);
  const int a = min(max(off[u], 0), N), b = min(max(off[u + 1], a), N);
  const int nch = (b - a + 31) >> 5;
  float* wr = W32 + (size_t)row * CK;
  if (nch == 0) {
    for (int v = threadIdx.x; v < CK; v += 256) wr[v] = 0.0f;
    if (threadIdx.x == 0) delta[row] = 0.0f;
    return;
  }
  if (threadIdx.x == 0) delta[row] = (delta[row] + (17.0f + 2.0f * nch) * U24) * 1.01f;
  if (nch == 1) return;
  const int s0 = pstart[(size_t)h * (CQ + 1) + u];  // part row of chunk 1
  float acc[E];
#pragma unroll
  for (int k = 0; k < E; ++k) {
    const int v = threadIdx.x + 256 * k;
    acc[k] = v < CK ? wr[v] : 0.0f;
  }
  for (int r = 1; r < nch; ++r) {
    const int sl = s0 + r - 1;
    if (sl >= pcap) break;
    const float* pr = part + ((size_t)h * pcap + sl) * CK;
    float x[E];  // loads first (clamped columns), so that they go out together
#pragma unroll
    for (int k = 0; k < E; ++k) x[k] = pr[min((int)threadIdx.x + 256 * k, CK - 1)];
#pragma unroll
    for (int k = 0; k < E; ++k)
      if ((int)threadIdx.x + 256 * k < CK) acc[k] = acc[k] + x[k];
  }
#pragma unroll
  for (int k = 0; k < E; ++k) {
    const int v = threadIdx.x + 256 * k;
    if (v < CK) wr[v] = acc[k];
  }
}

// Top-k on the float W^ of one row by radix selection (no sort): the m-th
// largest value a (m = kcount clamped to [1, #nonempty]) is found 8 bits at a
// time (W^ >= 0, so float order is the order of the bit patterns), then the
// number of values >= a and the largest value below a give the (m+1)-th
// largest b (= a on a tie).  The row is certified when a (1 - delta) - eps >
// b (1 + delta) + eps, and then the kept set is exactly {W^ >= a}; otherwise
// it is listed for the float64 path.  256 threads; `hist` and `aux` need 2048
// ints, `tmp` 4.
__device__ void select_topk_radix(const float* __restrict__ w, const int* __restrict__ ksz, int CK,
                                  int kcount, double dl, int* __restrict__ kv_count,
                                  int* __restrict__ out, int* __restrict__ rows,
                                  int* __restrict__ nrows, int u, int* hist, int* aux, int* tmp,
                                  int* __restrict__ bandc) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  constexpr int E = MAXC / 256;
  uint32_t kv[E];
  int nv = 0;
  int ks[E];
  float xs[E];  // loads first (clamped columns), so that they go out together
#pragma unroll
  for (int k = 0; k < E; ++k) {
    const int e = min(tid + 256 * k, CK - 1);
    ks[k] = ksz[e];
    xs[k] = w[e];
  }
#pragma unroll
  for (int k = 0; k < E; ++k) {
    const int e = tid + 256 * k;
    const bool ok = e < CK && ks[k] > 0;
    // valid keys have bit 31 clear (W^ >= 0); invalid ones are all ones and never match
    const float x = xs[k];
    kv[k] = ok ? (x > 0.0f ? __float_as_uint(x) : 0u) : 0xffffffffu;
    nv += ok;
  }
  // block sum (wave shuffles, then the four wavefront totals)
  auto block_sum = [&](int x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    __syncthreads();
    if (lane == 0) tmp[wid] = x;
    __syncthreads();
    return tmp[0] + tmp[1] + tmp[2] + tmp[3];
  };
  const int nvalid = block_sum(nv);
  if (nvalid == 0) {
    if (tid == 0) *kv_count = 0;
    return;
  }
  const int m = min(max(kcount, 1), nvalid);
  // rank m from the top, 8 bits per pass
  uint32_t prefix = 0u, pmask = 0u;
  int r = m;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    hist[tid] = 0;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < E; ++k)
      if ((kv[k] >> 31) == 0u && (kv[k] & pmask) == prefix) atomicAdd(&hist[(kv[k] >> shift) & 255u], 1);
    __syncthreads();
    // counts from the highest digit down: thread t holds digit 255 - t
    const int c = hist[255 - tid];
    int inc = c;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(inc, o, 64);
      if (lane >= o) inc += y;
    }
    if (lane == 63) tmp[wid] = inc;
    __syncthreads();
    for (int w2 = 0; w2 < wid; ++w2) inc += tmp[w2];
    if (inc >= r && inc - c < r) {
      aux[0] = 255 - tid;
      aux[1] = r - (inc - c);
    }
    __syncthreads();
    prefix |= (uint32_t)aux[0] << shift;
    pmask |= 255u << shift;
    r = aux[1];
    __syncthreads();
  }
  const uint32_t a_bits = prefix;
  int ge = 0;
  uint32_t lt = 0u;  // the largest value below a (0: none)
#pragma unroll
  for (int k = 0; k < E; ++k) {
    const bool v = (kv[k] >> 31) == 0u;
    ge += v && kv[k] >= a_bits;
    if (v && kv[k] < a_bits) lt = max(lt, kv[k]);
  }
  const int cnt_ge = block_sum(ge);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) lt = max(lt, (uint32_t)__shfl_xor((int)lt, o, 64));
  __syncthreads();
  if (lane == 0) tmp[wid] = (int)lt;
  __syncthreads();
  lt = max(max((uint32_t)tmp[0], (uint32_t)tmp[1]), max((uint32_t)tmp[2], (uint32_t)tmp[3]));
  const double eps = 4.0 * 1.1754943508222875e-38;  // absolute error near underflow
  bool ok = cnt_ge == m;
  if (ok && m < nvalid) {
    const double a = (double)__uint_as_float(a_bits) * (1.0 - dl) - eps;
    const double b = (double)__uint_as_float(lt) * (1.0 + dl) + eps;
    ok = a > b;
  }
  if (!ok && bandc) {
    // the blocks the bound places for certain: in the exact top m when their
    // lower bound exceeds the upper bound of the (m+1)-th largest W^ (every
    // block from position m + 1 on is then below them), out of it when their
    // upper bound is below the lower bound of the m-th (m blocks are above
    // them); the others (the band) are settled by their float64 weights.
    // Certain blocks go to the row's start, the band to its end (ascending).
    const double wm = (double)__uint_as_float(a_bits);
    const double wm1 = cnt_ge > m ? wm : (double)__uint_as_float(lt);
    const double tin = wm1 * (1.0 + dl) + eps, tout = wm * (1.0 - dl) - eps;
#pragma unroll
    for (int k = 0; k < E; ++k) {
      const int e = tid + 256 * k;
      const bool v = (kv[k] >> 31) == 0u;
      const double x = (double)__uint_as_float(kv[k]);
      const bool sin = v && x * (1.0 - dl) - eps > tin;
      const bool sout = v && x * (1.0 + dl) + eps < tout;
      if (e < MAXC) {
        hist[e] = sin ? 1 : 0;
        aux[e] = (v && !sin && !sout) ? 1 : 0;
      }
    }
    __syncthreads();
    const int nin = block_exclusive_scan_2048(hist, CK, tmp);
    const int nb = block_exclusive_scan_2048(aux, CK, tmp);
#pragma unroll
    for (int k = 0; k < E; ++k) {
      const int e = tid + 256 * k;
      if (e < CK && (kv[k] >> 31) == 0u) {
        const double x = (double)__uint_as_float(kv[k]);
        const bool sin = x * (1.0 - dl) - eps > tin;
        const bool sout = x * (1.0 + dl) + eps < tout;
        if (sin) out[hist[e]] = e;
        else if (!sout) out[CK - nb + aux[e]] = e;
      }
    }
    if (tid == 0) {
      *kv_count = nin;
      *bandc = nb;
      rows[atomicAdd(nrows, 1)] = u;
    }
    return;
  }
  if (!ok) {
    if (tid == 0) {
      if (bandc) *bandc = -1;
      rows[atomicAdd(nrows, 1)] = u;
    }
    return;
  }
  // kept: W^ >= a; written in ascending id order
#pragma unroll
  for (int k = 0; k < E; ++k) {
    const int e = tid + 256 * k;
    if (e < MAXC) hist[e] = ((kv[k] >> 31) == 0u && kv[k] >= a_bits) ? 1 : 0;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < E; ++k) aux[tid + 256 * k] = hist[tid + 256 * k];
  __syncthreads();
  block_exclusive_scan_2048(aux, CK, tmp);
  for (int e = tid; e < CK; e += 256)
    if (hist[e]) out[aux[e]] = e;
  if (tid == 0) *kv_count = m;
}

// Top-p on the float W^ of one row without sorting: the value T of the last
// kept block (the largest T whose mass {W^ >= T} reaches p) is found 8 bits at
// a time from per-digit counts and float64 masses.  Those masses are summed
// with atomics, so T may come out wrong near rounding ties; the certification
// below uses deterministic sums and only passes for the unique correct set
// (it reaches p with margin, without its smallest member it does not, and its
// smallest value is separated from the next one), so an accepted row is right
// and the others go to the float64 path.  All blocks are kept when the total
// mass is below p.  256 threads; `hist`, `aux` need 2048 ints, `dh` 256
// doubles, `tmp` 4 ints, `dtmp` 4 doubles.
__device__ void select_topp_radix(const float* __restrict__ w, const int* __restrict__ ksz, int CK,
                                  double p, double dl, int* __restrict__ kv_count,
                                  int* __restrict__ out, int* __restrict__ rows,
                                  int* __restrict__ nrows, int u, int* hist, int* aux, double* dh,
                                  int* tmp, double* dtmp) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  constexpr int E = MAXC / 256;
  uint32_t kv[E];
  int nv = 0;
  int ks[E];
  float xs[E];  // loads first (clamped columns), so that they go out together
#pragma unroll
  for (int k = 0; k < E; ++k) {
    const int e = min(tid + 256 * k, CK - 1);
    ks[k] = ksz[e];
    xs[k] = w[e];
  }
#pragma unroll
  for (int k = 0; k < E; ++k) {
    const int e = tid + 256 * k;
    const bool ok = e < CK && ks[k] > 0;
    const float x = xs[k];
    kv[k] = ok ? (x > 0.0f ? __float_as_uint(x) : 0u) : 0xffffffffu;
    nv += ok;
  }
  auto valid = [&](int k) { return (kv[k] >> 31) == 0u; };
  auto isum = [&](int x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    __syncthreads();
    if (lane == 0) tmp[wid] = x;
    __syncthreads();
    return tmp[0] + tmp[1] + tmp[2] + tmp[3];
  };
  // deterministic float64 sum: fixed order per thread, shuffles, wavefronts
  auto dsum = [&](double x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    __syncthreads();
    if (lane == 0) dtmp[wid] = x;
    __syncthreads();
    return (dtmp[0] + dtmp[1]) + (dtmp[2] + dtmp[3]);
  };
  auto umax = [&](uint32_t x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x = max(x, (uint32_t)__shfl_xor((int)x, o, 64));
    __syncthreads();
    if (lane == 0) tmp[wid] = (int)x;
    __syncthreads();
    return max(max((uint32_t)tmp[0], (uint32_t)tmp[1]), max((uint32_t)tmp[2], (uint32_t)tmp[3]));
  };
  const int nvalid = isum(nv);
  if (nvalid == 0) {
    if (tid == 0) *kv_count = 0;
    return;
  }
  double tl = 0.0;
#pragma unroll
  for (int k = 0; k < E; ++k)
    if (valid(k)) tl += (double)__uint_as_float(kv[k]);
  const double total = dsum(tl);
  uint32_t T = 0u;  // bits of the last kept value
  if (total >= p) {
    uint32_t prefix = 0u, pmask = 0u;
    double above = 0.0;  // mass of the values above the current prefix range
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      hist[tid] = 0;
      dh[tid] = 0.0;
      __syncthreads();
#pragma unroll
      for (int k = 0; k < E; ++k)
        if (valid(k) && (kv[k] & pmask) == prefix) {
          const int d = (kv[k] >> shift) & 255u;
          atomicAdd(&hist[d], 1);
          atomicAdd(&dh[d], (double)__uint_as_float(kv[k]));
        }
      __syncthreads();
      // masses from the highest digit down: thread t holds digit 255 - t
      const double ms = dh[255 - tid];
      double inc = ms;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const double y = __shfl_up(inc, o, 64);
        if (lane >= o) inc += y;
      }
      if (lane == 63) dtmp[wid] = inc;
      __syncthreads();
      for (int w2 = 0; w2 < wid; ++w2) inc += dtmp[w2];
      // the first digit (from the top) at which the mass reaches p; the
      // lowest digit with values when it is never reached (rounding)
      const bool cross = above + inc >= p && above + inc - ms < p;
      const int last = hist[255 - tid] > 0 ? tid : -1;
      int lastv = last;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) lastv = max(lastv, __shfl_xor(lastv, o, 64));
      __syncthreads();
      if (lane == 0) tmp[wid] = lastv;
      if (tid == 0) aux[0] = -1;
      __syncthreads();
      const int lastt = max(max(tmp[0], tmp[1]), max(tmp[2], tmp[3]));
      if (cross) {
        aux[0] = 255 - tid;
        dtmp[0] = above + inc - ms;
      }
      __syncthreads();
      int d = aux[0];
      double ab = dtmp[0];
      if (d < 0) {  // not reached inside this range: take its lowest digit
        d = 255 - lastt;
        __syncthreads();
        if (tid == lastt) dtmp[0] = above + inc - ms;
        __syncthreads();
        ab = dtmp[0];
      }
      above = ab;
      prefix |= (uint32_t)d << shift;
      pmask |= 255u << shift;
      __syncthreads();
    }
    T = prefix;
  } else {
    // every nonempty block is kept: T = the smallest value
    uint32_t mn = 0xffffffffu;
#pragma unroll
    for (int k = 0; k < E; ++k)
      if (valid(k)) mn = min(mn, kv[k]);
    T = ~umax(~mn);
  }
  int gt = 0, eq = 0;
  double ms = 0.0;
  uint32_t lt = 0u;
#pragma unroll
  for (int k = 0; k < E; ++k) {
    if (!valid(k)) continue;
    gt += kv[k] > T;
    eq += kv[k] == T;
    if (kv[k] >= T) ms += (double)__uint_as_float(kv[k]);
    else lt = max(lt, kv[k]);
  }
  const int ngt = isum(gt), neq = isum(eq);
  const double csum = dsum(ms);
  lt = umax(lt);
  const int m = ngt + neq;
  // certification (delta: the row's relative error; eps: absolute error near underflow)
  const double eps = 4.0 * 1.1754943508222875e-38;
  const double tv = (double)__uint_as_float(T);
  const double slo = csum * (1.0 - dl) - m * eps, shi = csum * (1.0 + dl) + m * eps;
  const double minlo = tv * (1.0 - dl) - eps;
  bool ok = m >= 1 && shi - minlo < p * (1.0 - 1e-12);
  if (m < nvalid) {
    ok = ok && neq == 1 && slo >= p * (1.0 + 1e-12);
    ok = ok && minlo > (double)__uint_as_float(lt) * (1.0 + dl) + eps;
  }
  if (!ok) {
    if (tid == 0) rows[atomicAdd(nrows, 1)] = u;
    return;
  }
  // kept: W^ >= T; written in ascending id order
#pragma unroll
  for (int k = 0; k < E; ++k) hist[tid + 256 * k] = (valid(k) && kv[k] >= T) ? 1 : 0;
  __syncthreads();
#pragma unroll
  for (int k = 0; k < E; ++k) aux[tid + 256 * k] = hist[tid + 256 * k];
  __syncthreads();
  block_exclusive_scan_2048(aux, CK, tmp);
  for (int e = tid; e < CK; e += 256)
    if (hist[e]) out[aux[e]] = e;
  if (tid == 0) *kv_count = m;
}

// Certified selection on the float W^: sort (W^ descending, id ascending),
// take the cut, and accept the row only if the cut is robust to the row's
// relative error delta_u plus an absolute error for values below float's
// normal range: the last kept block's lower bound must exceed the first
// dropped block's upper bound and, for top-p, the kept set's bounds must
// still straddle p.  Accepted rows are written; the others are listed for
// the float64 path.
__global__ __launch_bounds__(256) void k_select_fast(const float* __restrict__ W32,
                                                     const float* __restrict__ delta,
                                                     const int* __restrict__ q_offsets,
                                                     const int* __restrict__ k_sizes, int CQ,
                                                     int CK, int P, int mode, double param,
                                                     int kcount, int* __restrict__ kv_count,
                                                     int* __restrict__ kv_index,
                                                     int* __restrict__ rows,
                                                     int* __restrict__ nrows,
                                                     int* __restrict__ bandc) {
  __shared__ int flag[MAXC], aux[MAXC];
  __shared__ double dh[256], dtmp[4];
  __shared__ int tmp[4];
  const int h = blockIdx.y, u = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int* off = q_offsets + (size_t)h * (CQ + 1);
  const int nu = off[u + 1] - off[u];
  const size_t row = (size_t)h * CQ + u;
  if (nu <= 0) {
    if (tid == 0) kv_count[row] = 0;
    return;
  }
  if (mode == PARK_SELECT_TOPK) {
    select_topk_radix(W32 + row * CK, k_sizes + (size_t)h * CK, CK, kcount, (double)delta[row],
                      kv_count + row, kv_index + row * CK, rows + (size_t)h * CQ, nrows + h, u,
                      flag, aux, tmp, bandc ? bandc + row : nullptr);
    return;
  }
  if (bandc && tid == 0) bandc[row] = -1;  // a top-p row left to float64 is recomputed whole
  select_topp_radix(W32 + row * CK, k_sizes + (size_t)h * CK, CK, param, (double)delta[row],
                    kv_count + row, kv_index + row * CK, rows + (size_t)h * CQ, nrows + h, u, flag,
                    aux, dh, tmp, dtmp);
}

__global__ void k_zero_counts(int* __restrict__ c, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) c[i] = 0;
}

// ---------------------------------------------------------------- launchers
static int topk_count(int CK, double param) {
  // ceil(rho * N_K) blocks, clamped on the device to [1, #nonempty]
  const double x = param * (double)CK - 1e-9;
  int k = (int)x;
  if ((double)k < x) ++k;
  return k < 1 ? 1 : k;
}

static int pow2_at_least(int n) {
  int P = 2;
  while (P < n) P <<= 1;
  return P;
}

park_status launch_retrieve(const void* Qp, const int* q_offsets, const float* cen,
                            const int* k_sizes, int H, int N, int D, int dtype, int CQ, int CK,
                            int mode, double param, const RetrieveBufs& rb, float* W_out,
                            int* kv_count, int* kv_index, int* status, hipStream_t st) {
  const int P = pow2_at_least(CK);
  const int kcount = mode == PARK_SELECT_TOPK ? topk_count(CK, param) : 0;
  if (dtype != PARK_BF16) {  // float32 queries: float64 PAMA and selection of every row
    PARK_TRY(launch_pama64(Qp, q_offsets, cen, k_sizes, H, N, D, dtype, CQ, CK, nullptr, nullptr,
                           nullptr, rb.W64, W_out, nullptr, nullptr, nullptr, nullptr, 0, status,
                           st));
    PARK_LAUNCH("select", k_select64, dim3(CQ, H), dim3(256), 0, st, (const double*)rb.W64,
                q_offsets, k_sizes, CQ, CK, P, mode, param, kcount, (const int*)nullptr,
                (const int*)nullptr, kv_count, kv_index, (const int*)nullptr);
    return PARK_OK;
  }
  const size_t plane = (size_t)H * CK * D;
  const int nbm = (CK + 15) / 16;
  float* W32 = W_out ? W_out : rb.W32;
  const int CKpad = pama_ckpad(CK);
  // chunks of 32 queries, eight per workgroup (work list per head)
  const int icap = pama_icap(N, CQ), pcap = pama_pcap(N);
  const unsigned nwg = 8u * ((((unsigned)icap + 7u) / 8u * (unsigned)H + 7u) / 8u);
  float* part = (float*)rb.W64;  // free until the float64 rows are computed
  PARK_LAUNCH("pama_plan", k_pama_plan, dim3(H), dim3(1024), 0, st, q_offsets, N, CQ, icap,
              rb.qitems, rb.nitem, rb.qstart, rb.delta);
  // at most FULLK_NT centroid tiles: the single-sweep (Full-K) retrieval,
  // one chunk per wavefront, four per workgroup
  const bool fullk = CK <= 32 * FULLK_NT;
  const unsigned nwg4 = 8u * ((((unsigned)icap + 3u) / 4u * (unsigned)H + 7u) / 8u);
  if (fullk) {
    if (D == 128) {
      PARK_LAUNCH("pama_cen_prep", k_cen_prep<128>, dim3(nbm, H), dim3(256), 0, st, cen, k_sizes,
                  CK, rb.c3, plane, rb.lg, CKpad, rb.cn, rb.bmax);
      PARK_LAUNCH("pama_fullk", (k_pama_fullk<128, FULLK_NT>), dim3(nwg4), dim3(256), 0, st,
                  (const bf16_t*)Qp, q_offsets, (const int4*)rb.qitems, (const int*)rb.nitem,
                  icap, part, pcap, (const bf16_t*)rb.c3, plane, (const float*)rb.lg, CKpad,
                  (const float*)rb.bmax, nbm, H, N, CQ, CK, W32, rb.delta);
    } else {
      PARK_LAUNCH("pama_cen_prep", k_cen_prep<64>, dim3(nbm, H), dim3(256), 0, st, cen, k_sizes,
                  CK, rb.c3, plane, rb.lg, CKpad, rb.cn, rb.bmax);
      PARK_LAUNCH("pama_fullk", (k_pama_fullk<64, FULLK_NT>), dim3(nwg4), dim3(256), 0, st,
                  (const bf16_t*)Qp, q_offsets, (const int4*)rb.qitems, (const int*)rb.nitem,
                  icap, part, pcap, (const bf16_t*)rb.c3, plane, (const float*)rb.lg, CKpad,
                  (const float*)rb.bmax, nbm, H, N, CQ, CK, W32, rb.delta);
    }
  } else if (D == 128) {
    PARK_LAUNCH("pama_cen_prep", k_cen_prep<128>, dim3(nbm, H), dim3(256), 0, st, cen, k_sizes, CK,
                rb.c3, plane, rb.lg, CKpad, rb.cn, rb.bmax);
    PARK_LAUNCH("pama_fast", k_pama_fast<128>, dim3(nwg), dim3(256), 0, st, (const bf16_t*)Qp,
                q_offsets, (const int4*)rb.qitems, (const int*)rb.nitem, icap, part, pcap,
                (const bf16_t*)rb.c3, plane,
                (const float*)rb.lg, CKpad, (const float*)rb.bmax, nbm, H, N, CQ, CK, W32, rb.delta);
  } else {
    PARK_LAUNCH("pama_cen_prep", k_cen_prep<64>, dim3(nbm, H), dim3(256), 0, st, cen, k_sizes, CK,
                rb.c3, plane, rb.lg, CKpad, rb.cn, rb.bmax);
    PARK_LAUNCH("pama_fast", k_pama_fast<64>, dim3(nwg), dim3(256), 0, st, (const bf16_t*)Qp,
                q_offsets, (const int4*)rb.qitems, (const int*)rb.nitem, icap, part, pcap,
                (const bf16_t*)rb.c3, plane,
                (const float*)rb.lg, CKpad, (const float*)rb.bmax, nbm, H, N, CQ, CK, W32, rb.delta);
  }
  PARK_LAUNCH("pama_combine", k_pama_combine, dim3(CQ, H), dim3(256), 0, st, q_offsets,
              (const int*)rb.qstart, H, N, CQ, CK, (const float*)part, pcap, W32, rb.delta);
  PARK_LAUNCH("pama_reset", k_zero_counts, dim3((H + 63) / 64), dim3(64), 0, st, rb.nrows, H);
  // top-k rows the bound cannot settle are settled by their band of
  // ambiguous blocks (float64 weights of those blocks only); not when the
  // caller asked for W^ (its float64 rows are then written whole)
  int* bandc = (mode == PARK_SELECT_TOPK && !W_out) ? rb.bandc : nullptr;
  float* W32r = bandc ? nullptr : W32;
  PARK_LAUNCH("select_fast", k_select_fast, dim3(CQ, H), dim3(256), 0, st, (const float*)W32,
              (const float*)rb.delta, q_offsets, k_sizes, CQ, CK, P, mode, param, kcount,
              kv_count, kv_index, rb.rows, rb.nrows, bandc);
  // rows the float bound could not certify: float64 PAMA over chunks of 64
  // queries (work list, queue), split rows added up, then selection
  int rg = (1024 + H - 1) / H;
  rg = rg < 1 ? 1 : (rg > CQ ? CQ : rg);
  PARK_LAUNCH("pama_plan64", k_p64_plan, dim3(1), dim3(1024), 0, st, q_offsets,
              (const int*)rb.rows, (const int*)rb.nrows, H, N, CQ, p64_cap(H, CQ), rb.items,
              rb.srows, rb.pcnt);
  // the fast W^ rows and their bounds prune the normaliser pass (a row's
  // float32 W^ is written only at the end of its last item), and the
  // probability pass of top-p rows when W^ is not asked for
  const int plist = (mode == PARK_SELECT_TOPP && !W_out) ? 1 : 0;
  PARK_TRY(launch_pama64(Qp, q_offsets, cen, k_sizes, H, N, D, dtype, CQ, CK, rb.items, rb.pcnt,
                         rb.part, rb.W64, W32r, bandc, kv_index, W32, rb.delta, plist, status,
                         st));
  PARK_LAUNCH("pama_combine64", k_p64_combine, dim3(256), dim3(256), 0, st,
              (const int4*)rb.srows, (const int*)rb.pcnt, (const double*)rb.part, CK, rb.W64, W32r,
              status);
  PARK_LAUNCH("select_refine", k_select64, dim3(rg, H), dim3(256), 0, st, (const double*)rb.W64,
              q_offsets, k_sizes, CQ, CK, P, mode, param, kcount, (const int*)rb.rows,
              (const int*)rb.nrows, kv_count, kv_index, (const int*)bandc);
  if (bandc)
    PARK_LAUNCH("select_band", k_select_band, dim3(rg, H), dim3(256), 0, st,
                (const double*)rb.W64, k_sizes, CQ, CK, kcount, (const int*)rb.rows,
                (const int*)rb.nrows, (const int*)bandc, kv_count, kv_index);
  return PARK_OK;
}

template <int D, bool W2>
static park_status pama64_launch(const char* nm, unsigned nwg, size_t lds, const void* Qp,
                                 int dtype, const int* q_offsets, const float* cen,
                                 const int* k_sizes, int H, int N, int CQ, int CK,
                                 const int4* items, int* cnt, double* part, double* W64,
                                 float* W32, const int* bandc, const int* kv_index,
                                 const float* wfast, const float* dfast, int plist,
                                 int* status, hipStream_t st) {
  // reserved once for the largest CK (2048), outside any stream capture that may follow
  static const int lds_max = (int)(MAXC * (sizeof(double) + sizeof(int)));
  static const hipError_t a1 = hipFuncSetAttribute(
      (const void*)k_pama64<bf16_t, D, W2>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
  static const hipError_t a2 = hipFuncSetAttribute(
      (const void*)k_pama64<float, D, W2>, hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
  if (a1 != hipSuccess || a2 != hipSuccess)
    return fail(PARK_ERR_HIP, "retrieval: cannot reserve %zu bytes of LDS", lds);
  if (dtype == PARK_BF16)
    PARK_LAUNCH(nm, (k_pama64<bf16_t, D, W2>), dim3(nwg), dim3(256), lds, st, (const bf16_t*)Qp,
                q_offsets, cen, k_sizes, H, N, CQ, CK, items, cnt, part, W64, W32, bandc, kv_index,
                wfast, dfast, plist, status);
  else
    PARK_LAUNCH(nm, (k_pama64<float, D, W2>), dim3(nwg), dim3(256), lds, st, (const float*)Qp,
                q_offsets, cen, k_sizes, H, N, CQ, CK, items, cnt, part, W64, W32, bandc, kv_index,
                wfast, dfast, plist, status);
  return PARK_OK;
}

park_status launch_pama64(const void* Qp, const int* q_offsets, const float* cen,
                          const int* k_sizes, int H, int N, int D, int dtype, int CQ, int CK,
                          const int4* items, int* cnt, double* part, double* W64, float* W32,
                          const int* bandc, const int* kv_index, const float* wfast,
                          const float* dfast, int plist, int* status, hipStream_t st) {
  // with an item list: a queue drained by a fixed grid; without: one
  // workgroup per row, the rows of a head on one XCD
  const unsigned nwg = items ? 512u : 8u * (((unsigned)H * (unsigned)CQ + 7u) / 8u);
  const size_t lds = (size_t)CK * (sizeof(double) + sizeof(int));
  const char* nm = items ? "pama_refine64" : "pama64";
  // small layers have few items: the shorter steps of one wavefront per SIMD
  // win; large ones fill the chip, and two wavefronts per SIMD hide latency
  const bool w2 = (long)H * CQ >= 8192;
  if (D == 128)
    return w2 ? pama64_launch<128, true>(nm, nwg, lds, Qp, dtype, q_offsets, cen, k_sizes, H, N,
                                         CQ, CK, items, cnt, part, W64, W32, bandc, kv_index,
                                         wfast, dfast, plist, status, st)
              : pama64_launch<128, false>(nm, nwg, lds, Qp, dtype, q_offsets, cen, k_sizes, H, N,
                                          CQ, CK, items, cnt, part, W64, W32, bandc, kv_index,
                                          wfast, dfast, plist, status, st);
  return w2 ? pama64_launch<64, true>(nm, nwg, lds, Qp, dtype, q_offsets, cen, k_sizes, H, N, CQ,
                                      CK, items, cnt, part, W64, W32, bandc, kv_index, wfast,
                                      dfast, plist, status, st)
            : pama64_launch<64, false>(nm, nwg, lds, Qp, dtype, q_offsets, cen, k_sizes, H, N, CQ,
                                       CK, items, cnt, part, W64, W32, bandc, kv_index, wfast,
                                       dfast, plist, status, st);
}

// Query-centroid estimate and its selection: the float rows through the
// certified float selection, the rows it cannot settle by float64 weights.
park_status launch_qcen_retrieve(const float* qbar, const int* qsizes, const int* uoff,
                                 const float* cen, const int* k_sizes, int H, int D, int CQ,
                                 int CK, int mode, double param, const RetrieveBufs& rb,
                                 float* W_out, int* kv_count, int* kv_index, int* status,
                                 hipStream_t st) {
  const int nall = H * ((CQ + 63) / 64);
  const unsigned nwg = 8u * (((unsigned)nall + 7u) / 8u);
  float* W32 = W_out ? W_out : rb.W32;
  if (D == 128)
    PARK_LAUNCH("qcen64", k_qcen64<128>, dim3(nwg), dim3(256), 0, st, qbar, qsizes, cen, k_sizes,
                H, CQ, CK, rb.W64, W32, rb.delta, status);
  else
    PARK_LAUNCH("qcen64", k_qcen64<64>, dim3(nwg), dim3(256), 0, st, qbar, qsizes, cen, k_sizes,
                H, CQ, CK, rb.W64, W32, rb.delta, status);
  const int P = pow2_at_least(CK);
  const int kcount = mode == PARK_SELECT_TOPK ? topk_count(CK, param) : 0;
  PARK_LAUNCH("pama_reset", k_zero_counts, dim3((H + 63) / 64), dim3(64), 0, st, rb.nrows, H);
  PARK_LAUNCH("select_fast", k_select_fast, dim3(CQ, H), dim3(256), 0, st, (const float*)W32,
              (const float*)rb.delta, uoff, k_sizes, CQ, CK, P, mode, param, kcount, kv_count,
              kv_index, rb.rows, rb.nrows, (int*)nullptr);
  int rg = (1024 + H - 1) / H;
  rg = rg < 1 ? 1 : (rg > CQ ? CQ : rg);
  PARK_LAUNCH("select_refine", k_select64, dim3(rg, H), dim3(256), 0, st, (const double*)rb.W64,
              uoff, k_sizes, CQ, CK, P, mode, param, kcount, (const int*)rb.rows,
              (const int*)rb.nrows, kv_count, kv_index, (const int*)nullptr);
  return PARK_OK;
}

}  // namespace park
