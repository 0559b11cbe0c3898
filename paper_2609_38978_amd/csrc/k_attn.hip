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
                                                   int CK, OT* __restrict__ O,
                                                   float* __restrict__ lse) {
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
        // natural-log normaliser of the row: mrow is the largest scaled score
        if (lse && sub == 0) lse[(size_t)h * N + dst] = lrow > 0.0f ? mrow + logf(lrow) : -INFINITY;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA path: operand and accumulator vector types, output stores.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

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

// MinHash of a selected key-block set: min over the selected ids of a fixed
// integer hash (an avalanche mixer), used to order query blocks so that blocks
// selecting nearly the same key blocks are neighbours.
__device__ __forceinline__ uint32_t attn_hash(uint32_t v) {
  v ^= v >> 16;
  v *= 0x7feb352du;
  v ^= v >> 15;
  v *= 0x846ca68bu;
  v ^= v >> 16;
  return v;
}

// XOR swizzle of the 16-byte chunk index within a K row (an involution): the
// 16 rows one S^T MFMA reads land in 16 different bank groups.
template <int D>
__device__ __forceinline__ int swz_k(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }

// One wave-wide LDS DMA: lane l's 16 bytes at g land at LDS byte address
// lds + 16 l (lds wave-uniform).  Written as inline assembly so that the
// compiler does not treat the transfer as a pending LDS store: it would
// otherwise wait for every DMA in flight before each LDS read.  Completion
// is tracked explicitly with wait_vmcnt() and a barrier.
__device__ __forceinline__ void lds_dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds)
               : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)p;
}

// waits until at most N vector-memory operations of this wavefront are outstanding
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// ------------------------------------------------------------------------
// Grouped block-sparse attention.
//
// Query blocks that select nearly the same key blocks share one key/value
// stream: the plan orders the query blocks of a head by two MinHash values of
// their selected key-block sets and cuts the concatenated rows into groups of
// at most ATTN_R rows and ATTN_LB query blocks.  A workgroup streams the
// union of its blocks' selections once (ascending key-block id) and each row
// keeps only the keys of the key blocks its own query block selected, so the
// result per row is the same renormalised softmax over its own selection.

#ifndef PARK_ATTN_R
#define PARK_ATTN_R 128
#endif
#ifndef PARK_ATTN_RING
#define PARK_ATTN_RING 3
#endif
#ifndef PARK_ATTN_HEADMAJOR
#define PARK_ATTN_HEADMAJOR 1
#endif
constexpr int ATTN_R = PARK_ATTN_R;  // rows per group (32 per wavefront)
constexpr int ATTN_KSLOTS = PARK_ATTN_RING;  // K tiles in LDS (V: one more)
constexpr int ATTN_UCAP = 1024;  // key blocks of the union per stream chunk
constexpr int ATTN_LB = 16;          // query blocks per group (bits of a selection word)

static int attn_windows(int N) { return (N + ATTN_R - 1) / ATTN_R; }
// groups per head: every window of ATTN_R rows, split further when it holds
// more than ATTN_LB query blocks (a window boundary cuts at most one block)
int attn_groups_per_head(int N, int CQ) {
  const int W = attn_windows(N);
  return W + (CQ + W + ATTN_LB - 1) / ATTN_LB + 1;
}

// Selection families.  fam[h][u] = the smallest query block v (u itself
// included) whose selected key-block set overlaps u's with Jaccard index above
// 1/2 (3 |S_u & S_v| > |S_u| + |S_v|).  Blocks whose selections are nearly the
// same (on video latents: query clusters of the same content) then share one
// value, and sorting by fam[fam[u]] makes the blocks of a family neighbours in
// the group plan.
//
// k_attn_selbits: the selection of every (head, query block) as a 64-word bit
// row (CK <= 2048), one wavefront per row, fam = u, and the parts of the
// plan's sort key that come from the selection (MinHash values, key tiles).
__global__ __launch_bounds__(256) void k_attn_selbits(const int* __restrict__ kv_count,
                                                      const int* __restrict__ kv_index,
                                                      const int* __restrict__ q_offsets,
                                                      const int* __restrict__ k_offsets, int H,
                                                      int N, int CQ, int CK,
                                                      uint32_t* __restrict__ bits,
                                                      int* __restrict__ fam,
                                                      uint4* __restrict__ rkey) {
  __shared__ uint32_t rowb[4][64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const size_t row = (size_t)blockIdx.x * 4 + wid;
  const bool valid = row < (size_t)H * CQ;
  rowb[wid][lane] = 0u;
  __syncthreads();
  uint32_t m1 = 0xffffffffu, m2 = 0xffffffffu;
  int nkey = 0;
  if (valid) {
    const int h = (int)(row / (size_t)CQ);
    const int* koff = k_offsets + (size_t)h * (CK + 1);
    const int n = min(max(kv_count[row], 0), CK);
    const int* sel = kv_index + row * CK;
    for (int j = lane; j < n; j += 64) {
      const int v = sel[j];
      m1 = min(m1, attn_hash((uint32_t)v));
      m2 = min(m2, attn_hash((uint32_t)v + 7919u));
      if ((unsigned)v < (unsigned)CK) {
        atomicOr(&rowb[wid][v >> 5], 1u << (v & 31));
        nkey += max(0, koff[v + 1] - koff[v]);
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    m1 = min(m1, (uint32_t)__shfl_xor((int)m1, o, 64));
    m2 = min(m2, (uint32_t)__shfl_xor((int)m2, o, 64));
    nkey += __shfl_xor(nkey, o, 64);
  }
  __syncthreads();
  if (valid) {
    bits[row * 64 + lane] = rowb[wid][lane];
    if (lane == 0) {
      const int h = (int)(row / (size_t)CQ), u = (int)(row % (size_t)CQ);
      const int* qo = q_offsets + (size_t)h * (CQ + 1);
      const int a = min(max(qo[u], 0), N), b = min(max(qo[u + 1], a), N);
      fam[row] = u;
      // the plan's sort-key parts: the two MinHash values, the key tiles of
      // the block's own selection, whether the block has rows
      rkey[row] = make_uint4(m1, m2, (uint32_t)((nkey + 31) >> 5), b > a ? 1u : 0u);
    }
  }
}

// k_attn_family: workgroup = a pair of 64-block tiles (tu, tv <= tu) of a
// head; thread (r, kk) holds row u = 64 tu + r in registers and compares it
// with rows v = 64 tv + kk + 4 j < u (LDS); the smallest qualifying v goes to
// fam[u] by atomicMin (order-independent).
__global__ __launch_bounds__(256) void k_attn_family(const int* __restrict__ kv_count,
                                                     const uint32_t* __restrict__ bits, int CQ,
                                                     int CK, int* __restrict__ fam) {
  __shared__ uint4 vb[64][17];  // 64 bit rows of the v tile (+1 chunk: conflict-free)
  __shared__ int vcnt[64];
  const int h = blockIdx.y, p = (int)blockIdx.x, tid = threadIdx.x;
  int tu = (int)((sqrtf(8.0f * (float)p + 1.0f) - 1.0f) * 0.5f);
  while ((tu + 1) * (tu + 2) / 2 <= p) ++tu;
  while (tu * (tu + 1) / 2 > p) --tu;
  const int tv = p - tu * (tu + 1) / 2;
  const int W4 = ((CK + 31) / 32 + 3) / 4;  // 16-byte chunks holding the selection bits
  const uint4* bh = (const uint4*)(bits + (size_t)h * CQ * 64);
  for (int e = tid; e < 64 * 16; e += 256) {
    const int k = e >> 4, c = e & 15, v = tv * 64 + k;
    vb[k][c] = v < CQ ? bh[(size_t)v * 16 + c] : make_uint4(0u, 0u, 0u, 0u);
  }
  if (tid < 64) {
    const int v = tv * 64 + tid;
    vcnt[tid] = v < CQ ? min(max(kv_count[(size_t)h * CQ + v], 0), CK) : 0;
  }
  const int r = tid & 63, kk = tid >> 6, u = tu * 64 + r;
  uint4 ur[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) ur[c] = u < CQ ? bh[(size_t)u * 16 + c] : make_uint4(0u, 0u, 0u, 0u);
  const int cu = u < CQ ? min(max(kv_count[(size_t)h * CQ + u], 0), CK) : 0;
  __syncthreads();
  if (u >= CQ || cu == 0) return;  // no barrier follows
  int cand = 0x7fffffff;
  for (int j = 0; j < 16; ++j) {
    const int k = kk + 4 * j, v = tv * 64 + k;
    if (v >= u) break;
    int inter = 0;
#pragma unroll
    for (int c = 0; c < 16; ++c)
      if (c < W4) {
        const uint4 y = vb[k][c];
        inter += __popc(ur[c].x & y.x) + __popc(ur[c].y & y.y) + __popc(ur[c].z & y.z) +
                 __popc(ur[c].w & y.w);
      }
    if (3 * inter > cu + vcnt[k]) {
      cand = v;
      break;
    }
  }
  if (cand != 0x7fffffff) atomicMin(&fam[(size_t)h * CQ + u], cand);
}

// Group plan of one head (1024 threads, CQ <= 2048):
//   order[h][i]  query block at sorted position i (-1 past the blocks with rows)
//   spre[h][i]   rows of the sorted blocks before position i (i <= CQ)
//   grp[h][g]    {first row, end row, first position, end position}: rows in
//                the coordinates of the sorted concatenation; {0,0,0,0} when
//                g is past the last group.
__global__ __launch_bounds__(1024) void k_attn_gplan(const int* __restrict__ q_offsets,
                                                     const uint4* __restrict__ rkey,
                                                     const int* __restrict__ fam, int N,
                                                     int CQ, int CK, int GPH,
                                                     int* __restrict__ order,
                                                     int* __restrict__ spre,
                                                     int4* __restrict__ grp) {
  __shared__ unsigned long long key[2048];
  __shared__ int pre[2049];
  __shared__ int tiles[2048];  // key tiles of each query block's own selection (by block id)
  __shared__ int tpos[2048];   // the same by sorted position
  __shared__ int wsum[16];
  const int h = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int* qo = q_offsets + (size_t)h * (CQ + 1);
  int SZ = 2;
  while (SZ < CQ) SZ <<= 1;
  // sort keys (selection family, top bits of the first MinHash, top bits of
  // the second, block id); blocks without rows sort last with the key ~0.
  // One thread per block.
  for (int u = tid; u < SZ; u += 1024) {
    unsigned long long kk = ~0ull;
    if (u < CQ) {
      // MinHash values and key tiles of the selection (k_attn_selbits)
      const uint4 rk = rkey[(size_t)h * CQ + u];
      tiles[u] = (int)rk.z;
      if (rk.w) {
        // family label: the partner of u's smallest partner (one pointer jump)
        const int* fh = fam + (size_t)h * CQ;
        int f = fh[u];
        f = (unsigned)f < (unsigned)CQ ? fh[f] : u;
        f = (unsigned)f < (unsigned)CQ ? f : u;
        kk = ((unsigned long long)f << 52) | ((unsigned long long)(rk.x >> 12) << 32) |
             (rk.y & 0xfffff800u) | (uint32_t)u;
      }
    }
    key[u] = kk;
  }
  __syncthreads();
  for (int len = 2; len <= SZ; len <<= 1)
    for (int j = len >> 1; j > 0; j >>= 1) {
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int i = tid + 1024 * k, ixj = i ^ j;
        if (i < SZ && ixj > i) {
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
  // rows of the sorted blocks and their exclusive prefix
  int x[2], uu[2];
  int s = 0;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int pos = 2 * tid + k;
    uu[k] = -1;
    x[k] = 0;
    if (pos < CQ && key[pos] != ~0ull) {
      const int u = (int)(key[pos] & 0x7ffu);
      const int a = min(max(qo[u], 0), N), b = min(max(qo[u + 1], a), N);
      uu[k] = u;
      x[k] = b - a;
    }
    s += x[k];
  }
  int inc = s;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  if (lane == 63) wsum[wid] = inc;
  __syncthreads();
  int run = inc - s, total = 0;
  for (int i = 0; i < 16; ++i) {
    run += i < wid ? wsum[i] : 0;
    total += wsum[i];
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int pos = 2 * tid + k;
    if (pos < CQ) {
      pre[pos] = run;
      tpos[pos] = uu[k] >= 0 ? tiles[uu[k]] : 0;
      order[(size_t)h * CQ + pos] = uu[k];
      spre[(size_t)h * (CQ + 1) + pos] = run;
    }
    run += x[k];
  }
  if (tid == 0) {
    pre[CQ] = total;
    spre[(size_t)h * (CQ + 1) + CQ] = total;
  }
  __syncthreads();
  // windows of ATTN_R rows; a window with more than ATTN_LB blocks is split
  // into runs of ATTN_LB blocks.  With at most 2048 groups they are ordered
  // longest first (summed key tiles of their query blocks), so that the
  // longest ones start first.
  int4* gh = grp + (size_t)h * GPH;
  const int W = (total + ATTN_R - 1) / ATTN_R;
  const bool lpt = GPH <= 2048 && W < (1 << 23);
  // blocks of window wdw: sorted positions [i0, i1)
  auto window = [&](int wdw, int& i0, int& i1) {
    const int ra = wdw * ATTN_R, rb = min(ra + ATTN_R, total);
    int lo = 0, hi = CQ;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (pre[mid + 1] > ra) hi = mid;
      else lo = mid + 1;
    }
    i0 = lo;
    hi = CQ;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (pre[mid] >= rb) hi = mid;
      else lo = mid + 1;
    }
    i1 = lo;
  };
  auto desc = [&](int wdw, int k, int i0, int i1) {
    const int ra = wdw * ATTN_R, rb = min(ra + ATTN_R, total);
    const int ib = i0 + k * ATTN_LB, ie = min(ib + ATTN_LB, i1);
    return make_int4(max(ra, pre[ib]), min(rb, pre[ie]), ib, ie);
  };
  int gbase = 0;
  for (int w0 = 0; w0 < W; w0 += 1024) {
    const int wdw = w0 + tid;
    int i0 = 0, i1 = 0, nsub = 0;
    if (wdw < W) {
      window(wdw, i0, i1);
      nsub = (i1 - i0 + ATTN_LB - 1) / ATTN_LB;
    }
    int sinc = nsub;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(sinc, o, 64);
      if (lane >= o) sinc += y;
    }
    __syncthreads();
    if (lane == 63) wsum[wid] = sinc;
    __syncthreads();
    int g = gbase + sinc - nsub, ctot = 0;
    for (int i = 0; i < 16; ++i) {
      g += i < wid ? wsum[i] : 0;
      ctot += wsum[i];
    }
    for (int k = 0; k < nsub; ++k, ++g) {
      if (g >= GPH) continue;
      const int4 gd = desc(wdw, k, i0, i1);
      if (lpt) {
        uint32_t c = 0;
        for (int i = gd.z; i < gd.w; ++i) c += (uint32_t)tpos[i];
        key[g] = ((unsigned long long)(0xffffffffu - c) << 32) | ((uint32_t)wdw << 8) | (uint32_t)k;
      } else {
        gh[g] = gd;
      }
    }
    gbase += ctot;
  }
  if (lpt) {
    const int G = min(gbase, GPH);
    int SG = 2;
    while (SG < G) SG <<= 1;
    for (int g = G + tid; g < SG; g += 1024) key[g] = ~0ull;
    __syncthreads();
    for (int len = 2; len <= SG; len <<= 1)
      for (int j = len >> 1; j > 0; j >>= 1) {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const int i = tid + 1024 * k, ixj = i ^ j;
          if (i < SG && ixj > i) {
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
    for (int g = tid; g < G; g += 1024) {
      const uint32_t lo = (uint32_t)key[g];
      const int wdw = (int)(lo >> 8), k = (int)(lo & 255u);
      int i0, i1;
      window(wdw, i0, i1);
      gh[g] = desc(wdw, k, i0, i1);
    }
  }
  for (int g = gbase + tid; g < GPH; g += 1024) gh[g] = make_int4(0, 0, 0, 0);
}

// maximum of v over lanes l and l ^ 32 (a cross-half lane swap, no LDS traffic)
__device__ __forceinline__ float max_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(v, fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1])));
}

// makes all K fragments of a tile live at once, so that their LDS reads are
// issued together instead of one read-wait-MFMA step at a time
template <int KS>
__device__ __forceinline__ void frags_ready(const bf16x8_t (&a)[KS]) {
  if constexpr (KS == 8)
    asm volatile("" ::"v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]),
                 "v"(a[7]));
  else
    asm volatile("" ::"v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]));
}

// waits until this wavefront's DMAs of the oldest tile in flight are done,
// `younger` (0 .. NS - 2) newer tiles of PER operations each may stay in flight
template <int PER, int NS>
__device__ __forceinline__ void wait_oldest(int younger) {
  static_assert(NS >= 2 && NS <= 8, "ring depth");
  switch (NS >= 3 ? min(younger, NS - 2) : 0) {
    case 6: wait_vmcnt<6 * PER>(); break;
    case 5: wait_vmcnt<5 * PER>(); break;
    case 4: wait_vmcnt<4 * PER>(); break;
    case 3: wait_vmcnt<3 * PER>(); break;
    case 2: wait_vmcnt<2 * PER>(); break;
    case 1: wait_vmcnt<1 * PER>(); break;
    default: wait_vmcnt<0>(); break;
  }
}

// rotation of the rows of block b in a bias tile (a multiple of 4)
__device__ __forceinline__ int bias_rot(int b) { return 4 * ((b >> 1) & 7); }

template <int D, int KT, int NW>
struct GrpTile {
  static constexpr int CPR = D / 8;           // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;        // rows one wave-wide DMA fills
  // DMAs per wavefront, tensor and tile, and the wavefronts that issue them
  static constexpr int NI = KT / (NW * RPI) >= 1 ? KT / (NW * RPI) : 1;
  static constexpr int DW = KT / (NI * RPI);
  static constexpr int ELEMS = KT * D;  // bf16 elements of one K or V tile
  static_assert(DW >= 1 && DW <= NW && NI * DW * RPI == KT, "tile shape");
};

// V swizzle of the 32x32 transpose reads: the 4 rows x 64 bytes that one
// half-wavefront reads cover the 64 banks once
template <int D>
__device__ __forceinline__ int swz_v32(int r) { return D == 128 ? 4 * (r & 3) : 4 * ((r >> 1) & 1); }

template <typename OT, int D, int NW>
__global__ __launch_bounds__(64 * NW, 8 / NW) void k_attn_grp(
    const bf16_t* __restrict__ Qp, const bf16_t* __restrict__ Kp, const bf16_t* __restrict__ Vp,
    const int* __restrict__ q_offsets, const int* __restrict__ k_offsets,
    const int* __restrict__ kv_count, const int* __restrict__ kv_index,
    const int* __restrict__ q_perm, const int* __restrict__ order, const int* __restrict__ spre,
    const int4* __restrict__ grp, int H, int N, int CQ, int CK, int GPH, float scale_log2,
    OT* __restrict__ O, float* __restrict__ lse) {
  constexpr int KT = 32, NT = 64 * NW;
  constexpr int NSK = ATTN_KSLOTS, NSV = ATTN_KSLOTS + 1;  // K and V ring slots
  using TS = GrpTile<D, KT, NW>;
  constexpr int KS = D / 16;         // k-steps of S^T
  constexpr int DB = D / 32;         // 32-dimension blocks of O^T
  constexpr int EPT = AT_MAXC / NT;  // key blocks per thread in the union scan
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  bf16_t* Ks = (bf16_t*)smem;                        // [NSK][KT][D], swizzled chunks
  bf16_t* Vs = Ks + NSK * TS::ELEMS;                 // [NSV][KT][D], swizzled chunks
  float* bias = (float*)(Vs + NSV * TS::ELEMS);      // [NSK][ATTN_LB][KT]: 0 or -inf
  uint32_t* flg = (uint32_t*)(bias + NSK * ATTN_LB * KT);  // [AT_MAXC / 2]: 16 bits per key block
  int2* ut = (int2*)(flg + AT_MAXC / 2);            // [ATTN_UCAP + 1]
  uint16_t* selw = (uint16_t*)(ut + ATTN_UCAP + 1);  // [ATTN_UCAP]
  __shared__ int sg_row[ATTN_LB], sg_lr[ATTN_LB + 1], sg_u[ATTN_LB], sg_n[ATTN_LB + 1];
  __shared__ int tmp[2][NW];
  static_assert(ATTN_LB <= 16, "selection words are 16 bits");

  const int nitems = H * GPH;
#if PARK_ATTN_HEADMAJOR
  // head-major over the whole chip: consecutive workgroups (dealt to the 8
  // XCDs in turn) take the groups of one head, so only a head or two are in
  // flight at a time and their keys and values stay in the Infinity Cache
  const int item = (int)blockIdx.x;
#else
  // XCD-aware work item: XCD x (= blockIdx % 8) takes items [x*per, (x+1)*per)
  const int per = (nitems + 7) >> 3;
  const int item = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
#endif
  if (item >= nitems) return;
  const int h = item / GPH;
  const int4 gd = grp[item];
  const int ib = gd.z, ie = gd.w;
  if (gd.y <= gd.x || ib < 0 || ie <= ib || ie - ib > ATTN_LB || ie > CQ || gd.y - gd.x > 32 * NW)
    return;
  const int nb = ie - ib, tid = threadIdx.x;
  const int* qo = q_offsets + (size_t)h * (CQ + 1);
  const int* koff = k_offsets + (size_t)h * (CK + 1);
  if (tid < nb) {
    const int i = ib + tid;
    const int u = min(max(order[(size_t)h * CQ + i], 0), CQ - 1);
    const int s0 = spre[(size_t)h * (CQ + 1) + i];
    const int a = max(gd.x, s0);
    sg_u[tid] = u;
    sg_row[tid] = min(max(qo[u], 0), N) + (a - s0);
    sg_lr[tid] = a - gd.x;
    sg_n[tid] = min(max(kv_count[(size_t)h * CQ + u], 0), CK);
  }
  if (tid == 0) sg_lr[nb] = gd.y - gd.x;
  for (int v = tid; v < AT_MAXC / 2; v += NT) flg[v] = 0u;
  __syncthreads();
  // selection entries of the group's blocks, end-to-end (a prefix over the
  // few blocks, then one parallel pass: the entries' loads go out together)
  if (tid == 0) {
    int c = 0;
    for (int b = 0; b < nb; ++b) {
      const int n = sg_n[b];
      sg_n[b] = c;
      c += n;
    }
    sg_n[nb] = c;
  }
  __syncthreads();
  // bit b of key block v's flag: query block b of the group selected v
  for (int e = tid; e < sg_n[nb]; e += NT) {
    int b = 0;
    while (b + 1 < nb && sg_n[b + 1] <= e) ++b;
    const int v = kv_index[((size_t)h * CQ + sg_u[b]) * CK + (e - sg_n[b])];
    if ((unsigned)v < (unsigned)CK) atomicOr(&flg[v >> 1], (1u << b) << (16 * (v & 1)));
  }
  __syncthreads();
  const bf16_t* Qh = Qp + (size_t)h * N * D;
  const bf16_t* Kh = Kp + (size_t)h * N * D;
  const bf16_t* Vh = Vp + (size_t)h * N * D;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l = tid & 63, hf = l >> 5, c32 = l & 31;

  // this lane's query row: group row 32 w + c32, query block bq of the group
  const int gr = 32 * w + c32;
  const int grows = sg_lr[nb];
  int bq = 0;
  while (bq + 1 < nb && sg_lr[bq + 1] <= gr) ++bq;
  const int qr0 = sg_row[bq] + (gr - sg_lr[bq]);
  const bool qvalid = gr < grows && (unsigned)qr0 < (unsigned)N;
  const int qr = qvalid ? qr0 : 0;
  bf16x8_t qf[KS];
#pragma unroll
  for (int s2 = 0; s2 < KS; ++s2) {
    uint4 raw = make_uint4(0u, 0u, 0u, 0u);
    if (qvalid) raw = *(const uint4*)(Qh + (size_t)qr * D + 16 * s2 + 8 * hf);
    qf[s2] = __builtin_bit_cast(bf16x8_t, raw);
  }
#pragma unroll
  for (int s2 = 0; s2 < KS; ++s2) asm volatile("" ::"v"(qf[s2]));
  // the bias row of this lane
  const int bqq = qvalid ? bq : 0;
  const int brow = bqq * KT, bcol = 4 * hf + bias_rot(bqq);

  // LDS read offsets (bf16 elements, relative to a slot)
  // K (A operand of S^T): key row c32, chunk 2 s + hf
  int kofs[KS];
#pragma unroll
  for (int s2 = 0; s2 < KS; ++s2) kofs[s2] = c32 * D + 8 * ((2 * s2 + hf) ^ swz_k<D>(c32));
  // V^T (A operand of O^T) by transpose reads: in 16-lane group G, lane j
  // gives row 4 hf + j/4 (+ 16 kappa, + 8 for the second read) and dims
  // 32 db + 16 (G % 2) + 4 (j % 4); it receives dim 32 db + 16 (G % 2) + j
  const int G = l >> 4, jg = l & 15;
  const int vr0 = 4 * hf + (jg >> 2);
  int vofs[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const int col = 32 * db + 16 * (G & 1) + 4 * (jg & 3);
    vofs[db] = vr0 * D + 8 * ((col >> 3) ^ swz_v32<D>(vr0)) + (col & 7);
  }

  float m = -INFINITY, lpart = 0.0f;
  f32x16_t acc[DB];
#pragma unroll
  for (int b = 0; b < DB; ++b)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[b][q] = 0.0f;

  // DMA lanes: tile row rr[i], chunk position pch; a cursor into ut per row;
  // kb[i]: selection bits of the row's key block (all lanes of a row agree)
  const int pch = l % TS::CPR;
  const bool dma_w = w < TS::DW;
  int rr[TS::NI];
#pragma unroll
  for (int i = 0; i < TS::NI; ++i) rr[i] = (w * TS::NI + i) * TS::RPI + l / TS::CPR;

  // the union (U key blocks) is streamed in chunks of at most ATTN_UCAP key
  // blocks; the online softmax state carries over from one chunk to the next
  const int lane = tid & 63, wv = tid >> 6;
  int U = ATTN_UCAP;
  for (int ch = 0; ch * ATTN_UCAP < U; ++ch) {
    // stream table of this chunk: ut[j] = {stream position, first row of Kp}
    // of its j-th key block, ut[Uc] = {end position, -1}; selw[j] its bits
    {
      uint32_t f[EPT];
      int x[EPT], kst[EPT], c = 0, s = 0;
      int2 kb2[EPT];  // block boundaries, loaded together (clamped ids)
#pragma unroll
      for (int k = 0; k < EPT; ++k) kb2[k] = *(const int2*)(koff + min(tid * EPT + k, CK - 1));
#pragma unroll
      for (int k = 0; k < EPT; ++k) {
        const int v = tid * EPT + k;
        f[k] = v < CK ? (flg[v >> 1] >> (16 * (v & 1))) & 0xffffu : 0u;
        x[k] = 0;
        kst[k] = -1;
        if (f[k]) {
          kst[k] = kb2[k].x;
          x[k] = max(0, kb2[k].y - kst[k]);
          ++c;
        }
        s += x[k];
      }
      int ic = c, is = s;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int yc = __shfl_up(ic, o, 64), ys = __shfl_up(is, o, 64);
        if (lane >= o) {
          ic += yc;
          is += ys;
        }
      }
      if (lane == 63) {
        tmp[0][wv] = ic;
        tmp[1][wv] = is;
      }
      __syncthreads();
      int jc = ic - c, js = is - s;
      U = 0;
      for (int w2 = 0; w2 < NW; ++w2) {
        jc += w2 < wv ? tmp[0][w2] : 0;
        js += w2 < wv ? tmp[1][w2] : 0;
        U += tmp[0][w2];
      }
      const int jlo = ch * ATTN_UCAP, jhi = min(jlo + ATTN_UCAP, U);
#pragma unroll
      for (int k = 0; k < EPT; ++k)
        if (f[k]) {
          if (jc >= jlo && jc < jhi) {
            ut[jc - jlo] = make_int2(js, kst[k]);
            selw[jc - jlo] = (uint16_t)f[k];
            if (jc == jhi - 1) ut[jc - jlo + 1] = make_int2(js + x[k], -1);
          }
          ++jc;
          js += x[k];
        }
      __syncthreads();
    }
    if (U == 0) break;
    const int Uc = min(ATTN_UCAP, U - ch * ATTN_UCAP);
    const int base = ut[0].x, nk = ut[Uc].x - base;
    int jj[TS::NI], cj[TS::NI], kj[TS::NI], src[TS::NI];
    uint32_t sw[TS::NI], kb[TS::NI];
    int2 nx[TS::NI];
#pragma unroll
    for (int i = 0; i < TS::NI; ++i) {
      jj[i] = 0;
      cj[i] = base;
      kj[i] = ut[0].y;
      sw[i] = selw[0];
      nx[i] = ut[1];
      src[i] = 0;
      kb[i] = 0u;
    }
    auto advance = [&](int t) {
      if (!dma_w) return;
#pragma unroll
      for (int i = 0; i < TS::NI; ++i) {
        const int pos = base + t * KT + rr[i];
        while (pos >= nx[i].x && jj[i] + 1 < Uc) {
          ++jj[i];
          cj[i] = nx[i].x;
          kj[i] = nx[i].y;
          sw[i] = selw[jj[i]];
          nx[i] = ut[jj[i] + 1];
        }
        const int r = kj[i] + (pos - cj[i]);
        const bool ok = pos < base + nk && (unsigned)r < (unsigned)N;
        src[i] = ok ? r : 0;
        kb[i] = ok ? sw[i] : 0u;
      }
    };
    // tile T: K into slot T % NSK, V into slot T % NSV, with the score bias
    // of every (query block, tile row)
    auto issue = [&](int T) {
      if (!dma_w) return;
      const int sk = T % NSK, sv = T % NSV;
      bf16_t* ks = Ks + sk * TS::ELEMS;
      bf16_t* vs = Vs + sv * TS::ELEMS;
#pragma unroll
      for (int i = 0; i < TS::NI; ++i) {
        const int off = (w * TS::NI + i) * 512;  // 1 KB per wave-wide DMA
        lds_dma16(Kh + (size_t)src[i] * D + 8 * (pch ^ swz_k<D>(rr[i])), lds_addr(ks + off));
      }
#pragma unroll
      for (int i = 0; i < TS::NI; ++i) {
        const int off = (w * TS::NI + i) * 512;
        lds_dma16(Vh + (size_t)src[i] * D + 8 * (pch ^ swz_v32<D>(rr[i])), lds_addr(vs + off));
      }
      // row r of block b sits at b * KT + ((r + bias_rot(b)) % KT): groups of
      // four rows stay contiguous and the 16 blocks of one row land in 16
      // different banks
      float* bs = bias + sk * ATTN_LB * KT;
#pragma unroll
      for (int i = 0; i < TS::NI; ++i)
#pragma unroll
        for (int b = pch; b < ATTN_LB; b += TS::CPR)
          bs[b * KT + ((rr[i] + bias_rot(b)) & (KT - 1))] = ((kb[i] >> b) & 1u) ? 0.0f : -INFINITY;
    };
    // S^T of tile T (32 keys x 32 queries; lane: keys 8 b + 4 hf + r of query
    // c32), starting from the bias of those keys
    auto scores = [&](int T, f32x16_t& st) {
      const int sk = T % NSK;
      const bf16_t* ks = Ks + sk * TS::ELEMS;
      bf16x8_t kf[KS];
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2) kf[s2] = *(const bf16x8_t*)(ks + kofs[s2]);
      const float* br = bias + sk * ATTN_LB * KT + brow;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const float4 y = *(const float4*)(br + ((bcol + 8 * b) & (KT - 1)));
        st[4 * b + 0] = y.x;
        st[4 * b + 1] = y.y;
        st[4 * b + 2] = y.z;
        st[4 * b + 3] = y.w;
      }
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2)
        st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s2], qf[s2], st, 0, 0, 0);
    };
    const int ntiles = (nk + KT - 1) / KT;
    // tiles 0 .. NSK - 1 in flight, then S^T of tile 0
#pragma unroll
    for (int p = 0; p < NSK; ++p)
      if (p < ntiles) {
        advance(p);
        issue(p);
      }
    f32x16_t st_next;
    if (ntiles > 0) {
      wait_oldest<2 * TS::NI, NSK + 1>(ntiles - 1);
      __syncthreads();
      scores(0, st_next);
    }
    for (int t = 0; t < ntiles; ++t) {
      // at the top: S^T(t) is in st_next; tiles t+1 .. t+NSK-1 are in flight
      const f32x16_t st = st_next;
      const int nxt = t + NSK;
      if (nxt < ntiles) advance(nxt);
      // K(t+1) (and with it everything issued before: V(t)) has landed; V(t+1)
      // and the tiles after t+1 may stay in flight
      if (t + 2 < ntiles) wait_oldest<TS::NI, 8>(2 * (min(ntiles - 2 - t, NSK - 2)) + 1);
      else if (t + 1 < ntiles) wait_vmcnt<TS::NI>();
      else wait_vmcnt<0>();
      __syncthreads();  // K(t+1), V(t) visible; K(t) and V(t-1) are free
      // softmax of tile t and O^T += V^T P^T; the scores of tile t+1 are
      // computed in the same block so that their MFMAs overlap this VALU work
      // row maximum of tile t and the (lazy) rescale of the running state
      auto rescale = [&]() {
        float tmax = fmaxf(st[0], st[1]);
#pragma unroll
        for (int q = 2; q < 16; ++q) tmax = fmaxf(tmax, st[q]);
        tmax = max_xor32(tmax);
        // the reference maximum moves only when a row maximum exceeds it by
        // more than 2^8 in probability (softmax is invariant to the shift; p <= 2^8)
        if (__any((tmax - m) * scale_log2 > 8.0f)) {
          // rows without a kept key so far keep m = -inf (and alpha = 1)
          const float mnew = fmaxf(m, tmax);
          const float alpha = mnew == m ? 1.0f : __builtin_amdgcn_exp2f((m - mnew) * scale_log2);
          lpart *= alpha;
#pragma unroll
          for (int b = 0; b < DB; ++b) acc[b] *= alpha;
          m = mnew;
        }
      };
      // probabilities of tile t and O^T += V^T P^T in two 16-key steps; step
      // kp takes scores 8 kp .. 8 kp + 7 (keys 16 kp + 4 hf + r and
      // 16 kp + 8 + 4 hf + r)
      auto pv = [&]() {
        const float nms = m == -INFINITY ? 0.0f : -m * scale_log2;
        const bf16_t* vs = Vs + (t % NSV) * TS::ELEMS;
#pragma unroll
        for (int kp = 0; kp < 2; ++kp) {
          float p[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            p[e] = __builtin_amdgcn_exp2f(fmaf(st[8 * kp + e], scale_log2, nms));
            lpart += p[e];
          }
          bf16x8_t pb;
#pragma unroll
          for (int e = 0; e < 8; e += 2) {
            const bf16x2_t two = __builtin_convertvector(f32x2_t{p[e], p[e + 1]}, bf16x2_t);
            pb[e] = two[0];
            pb[e + 1] = two[1];
          }
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            const bf16_t* v1 = vs + vofs[db] + 16 * kp * D;
            const i16x4_t t1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)v1);
            const i16x4_t t2 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(v1 + 8 * D));
            const bf16x8_t a = __builtin_bit_cast(
                bf16x8_t, (short __attribute__((ext_vector_type(8)))){t1[0], t1[1], t1[2], t1[3],
                                                                      t2[0], t2[1], t2[2], t2[3]});
            acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, acc[db], 0, 0, 0);
          }
        }
      };
      // every tile is computed by every wavefront (keys that its query blocks
      // did not select have score -inf, so they add nothing); the scores of
      // tile t+1 (past the end: a stale slot, never used) are computed in the
      // same block as the probabilities of tile t so that their MFMAs overlap
      // that VALU work
      rescale();
      scores(t + 1, st_next);
      pv();
      // the DMAs of tile t+NSK go out after this step's compute: a DMA issue
      // that stalls on a busy memory system then does not hold the MFMAs back
      if (nxt < ntiles) issue(nxt);
    }
    __syncthreads();  // every wavefront is done with this chunk's tables and ring
  }
  float lsum = lpart + __shfl_xor(lpart, 32, 64);
  if (qvalid) {
    const int dst = q_perm[(size_t)h * N + qr];
    if ((unsigned)dst < (unsigned)N) {
      const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
      // natural-log normaliser: the probabilities are exp2((s - m) scale_log2)
      // of raw scores s, so sum_j exp(s_j / sqrt(d)) = exp(m / sqrt(d)) lsum
      if (lse && hf == 0)
        lse[(size_t)h * N + dst] =
            lsum > 0.0f ? m * (scale_log2 * 0.69314718055994531f) + logf(lsum) : -INFINITY;
      OT* o = O + ((size_t)h * N + dst) * D + 4 * hf;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int bq4 = 0; bq4 < 4; ++bq4)
          store_out4<OT>(o + 32 * db + 8 * bq4, acc[db][4 * bq4 + 0] * inv,
                         acc[db][4 * bq4 + 1] * inv, acc[db][4 * bq4 + 2] * inv,
                         acc[db][4 * bq4 + 3] * inv);
    }
  }
}

template <typename T, typename OT>
static park_status attn_dispatch_d(const void* Qp, const void* Kp, const void* Vp, const int* qo,
                                   const int* ko, const int* kc, const int* ki, const int* qp,
                                   int H, int N, int D, int CQ, int CK, void* O, float* lse,
                                   hipStream_t st) {
  dim3 g(CQ, H);
  if (D == 128)
    PARK_LAUNCH("attn_valu", (k_attn_valu<T, OT, 128>), g, dim3(256), 0, st, (const T*)Qp,
                (const T*)Kp, (const T*)Vp, qo, ko, kc, ki, qp, N, CQ, CK, (OT*)O, lse);
  else
    PARK_LAUNCH("attn_valu", (k_attn_valu<T, OT, 64>), g, dim3(256), 0, st, (const T*)Qp,
                (const T*)Kp, (const T*)Vp, qo, ko, kc, ki, qp, N, CQ, CK, (OT*)O, lse);
  return PARK_OK;
}

size_t attn_grp_offset(int H, int CQ);
// the families [H][CQ], padded to 16 bytes (the bit rows follow)
static size_t attn_fam_bytes(int H, int CQ) { return ((size_t)H * CQ * sizeof(int) + 15) & ~(size_t)15; }

template <typename OT, int D, int NW>
static park_status attn_grp_launch(const void* Qp, const void* Kp, const void* Vp, const int* qo,
                                   const int* ko, const int* kc, const int* ki, const int* qp,
                                   int H, int N, int CQ, int CK, void* plan, float sl2, void* O,
                                   float* lse, hipStream_t st) {
  const int GPH = attn_groups_per_head(N, CQ);
  int* order = (int*)plan;
  int* spre = order + (size_t)H * CQ;
  int4* grp = (int4*)((char*)plan + attn_grp_offset(H, CQ));
  int* fam = (int*)(grp + (size_t)H * GPH);
  uint32_t* bits = (uint32_t*)((char*)fam + attn_fam_bytes(H, CQ));
  uint4* rkey = (uint4*)(bits + (size_t)H * CQ * 64);
  const unsigned nrow = (unsigned)H * (unsigned)CQ, ntile = (unsigned)(CQ + 63) / 64;
  PARK_LAUNCH("attn_selbits", k_attn_selbits, dim3((nrow + 3) / 4), dim3(256), 0, st, kc, ki, qo,
              ko, H, N, CQ, CK, bits, fam, rkey);
  PARK_LAUNCH("attn_family", k_attn_family, dim3(ntile * (ntile + 1) / 2, H), dim3(256), 0, st,
              kc, bits, CQ, CK, fam);
  PARK_LAUNCH("attn_plan", k_attn_gplan, dim3(H), dim3(1024), 0, st, qo, (const uint4*)rkey,
              (const int*)fam, N, CQ, CK, GPH, order, spre, grp);
  // K ring, V ring, score biases, key-block flags, stream table, selection words
  constexpr size_t lds = (size_t)(2 * ATTN_KSLOTS + 1) * 32 * D * sizeof(bf16_t) +
                         (size_t)ATTN_KSLOTS * ATTN_LB * 32 * 4 + (size_t)AT_MAXC / 2 * 4 +
                         (size_t)(ATTN_UCAP + 1) * sizeof(int2) + (size_t)ATTN_UCAP * 2;
  static const hipError_t attr = hipFuncSetAttribute(
      (const void*)k_attn_grp<OT, D, NW>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (attr != hipSuccess)
    return fail(PARK_ERR_HIP, "attention: cannot reserve %zu bytes of LDS", lds);
  // 8 * ceil(items / 8) workgroups: every item owns one (see the remap in the kernel)
  const unsigned nwg = 8u * (((unsigned)H * (unsigned)GPH + 7u) / 8u);
  PARK_LAUNCH("attn_mfma", (k_attn_grp<OT, D, NW>), dim3(nwg), dim3(64 * NW), lds, st,
              (const bf16_t*)Qp, (const bf16_t*)Kp, (const bf16_t*)Vp, qo, ko, kc, ki, qp, order,
              spre, grp, H, N, CQ, CK, GPH, sl2, (OT*)O, lse);
  return PARK_OK;
}

template <typename OT>
static park_status attn_mfma_d(const void* Qp, const void* Kp, const void* Vp, const int* qo,
                               const int* ko, const int* kc, const int* ki, const int* qp, int H,
                               int N, int D, int CQ, int CK, void* plan, void* O, float* lse,
                               hipStream_t st) {
  const float sl2 = (float)(1.4426950408889634 / sqrt((double)D));
  if (D == 128)
    return attn_grp_launch<OT, 128, ATTN_R / 32>(Qp, Kp, Vp, qo, ko, kc, ki, qp, H, N, CQ, CK,
                                                  plan, sl2, O, lse, st);
  return attn_grp_launch<OT, 64, ATTN_R / 32>(Qp, Kp, Vp, qo, ko, kc, ki, qp, H, N, CQ, CK, plan,
                                              sl2, O, lse, st);
}

// order [H][CQ], spre [H][CQ + 1], then the groups [H][GPH] at 16-byte
// alignment, the selection families [H][CQ] (padded to 16 bytes), the
// selection bit rows [H][CQ][64] and the sort-key parts [H][CQ] (uint4)
size_t attn_grp_offset(int H, int CQ) {
  return (((size_t)H * CQ + (size_t)H * (CQ + 1)) * sizeof(int) + 15) & ~(size_t)15;
}

size_t attn_plan_bytes(int H, int N, int CQ) {
  return attn_grp_offset(H, CQ) + (size_t)H * attn_groups_per_head(N, CQ) * sizeof(int4) +
         attn_fam_bytes(H, CQ) + (size_t)H * CQ * 64 * sizeof(uint32_t) +
         (size_t)H * CQ * sizeof(uint4);
}

park_status launch_attention(const void* Qp, const void* Kp, const void* Vp, const int* q_offsets,
                             const int* k_offsets, const int* kv_count, const int* kv_index,
                             const int* q_perm, int H, int N, int D, int dtype, int CQ, int CK,
                             void* O, int out_dtype, float* lse, void* plan,
                             hipStream_t st) {
  if (dtype == PARK_BF16) {
    if (out_dtype == PARK_BF16)
      return attn_mfma_d<bf16_t>(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index, q_perm, H,
                                 N, D, CQ, CK, plan, O, lse, st);
    return attn_mfma_d<float>(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index, q_perm, H, N,
                              D, CQ, CK, plan, O, lse, st);
  }
  // fp32 inputs: VALU kernel in fp32 (the contraction cannot use bf16 MFMA exactly)
  if (out_dtype == PARK_BF16)
    return attn_dispatch_d<float, bf16_t>(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index,
                                          q_perm, H, N, D, CQ, CK, O, lse, st);
  return attn_dispatch_d<float, float>(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index,
                                       q_perm, H, N, D, CQ, CK, O, lse, st);
}

}  // namespace park
