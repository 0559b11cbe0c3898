// Stable counting sort of cluster labels (pi = argsort(z), Alg. 3) and the
// row gathers X' = X[pi].  Two passes: per-tile histograms, then a stable
// scatter in which each tile's workgroup first derives its own bases from the
// histogram table (cluster totals scanned over clusters, plus the counts of
// the earlier tiles) and then walks its tokens in order one wavefront (64
// tokens) at a time.  All integer work; the result is unique, so it is
// bit-exact and deterministic.
#include "common.h"
#include "kernels.h"

namespace park {

// Tokens per sort tile: the smallest power of two >= 256 for which the
// per-head histogram table (C x tiles) stays below 64K entries, so that each
// scatter workgroup's pass over the table stays short while the scatter gets
// as many workgroups as possible.
int sort_tile(int H, int N, int C) {
  (void)H;
  int t = 256;
  while ((long)C * ((N + t - 1) / t) > 65536 && t < (1 << 30)) t *= 2;
  return t;
}

int sort_tiles(int H, int N, int C) {
  const int t = sort_tile(H, N, C);
  return (N + t - 1) / t;
}

// thist[h][tile][v] = #{ i in tile : z_i = v }
__global__ __launch_bounds__(256) void k_sort_hist(const int* __restrict__ labels, int N, int C,
                                                   int tile_sz, int* __restrict__ thist) {
  extern __shared__ int hist[];
  const int h = blockIdx.y, tile = blockIdx.x, nt = gridDim.x;
  for (int v = threadIdx.x; v < C; v += 256) hist[v] = 0;
  __syncthreads();
  const int i0 = tile * tile_sz, i1 = min(N, i0 + tile_sz);
  const int* z = labels + (size_t)h * N;
  // eight loads in flight per thread
  for (int c0 = i0; c0 < i1; c0 += 8 * 256) {
    int v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int i = c0 + 256 * k + threadIdx.x;
      v[k] = i < i1 ? z[i] : -1;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if ((unsigned)v[k] < (unsigned)C) atomicAdd(&hist[v[k]], 1);
  }
  __syncthreads();
  int* out = thist + ((size_t)h * nt + tile) * C;
  for (int v = threadIdx.x; v < C; v += 256) out[v] = hist[v];
}

// Stable scatter.  Bases first: thread v sums cluster v's counts over the
// tiles before this one and over all tiles (table rows read coalesced, eight
// in flight), the totals are scanned over clusters, and base_v = start_v +
// earlier counts; tile 0 also writes the cluster offsets (o[C] = N).  Then
// wavefront 0 walks the tile's tokens in increasing order; equal labels
// inside the wavefront are matched with one ballot per label bit.
__global__ __launch_bounds__(256) void k_sort_scatter(const int* __restrict__ labels, int N, int C,
                                                      int nbits, int tile_sz,
                                                      const int* __restrict__ thist,
                                                      int* __restrict__ perm,
                                                      int* __restrict__ offsets) {
  extern __shared__ int run[];  // [C] bases, then [C] totals
  __shared__ int wsum[4];
  const int h = blockIdx.y, tile = blockIdx.x, nt = gridDim.x, tid = threadIdx.x;
  const int lane = tid & 63, wid = tid >> 6;
  const int* b = thist + (size_t)h * nt * C;
  int* tot = run + C;
  for (int v = tid; v < C; v += 256) {
    int before = 0, all = 0;
    for (int t0 = 0; t0 < nt; t0 += 8) {
      int c[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) c[k] = t0 + k < nt ? b[(size_t)(t0 + k) * C + v] : 0;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        all += c[k];
        before += t0 + k < tile ? c[k] : 0;
      }
    }
    run[v] = before;
    tot[v] = all;
  }
  __syncthreads();
  // exclusive scan of tot over the clusters: thread tid owns clusters
  // [tid * per, (tid + 1) * per)
  const int per = (C + 255) / 256;
  int s = 0;
  for (int k = 0; k < per; ++k) {
    const int v = tid * per + k;
    s += v < C ? tot[v] : 0;
  }
  int inc = s;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  if (lane == 63) wsum[wid] = inc;
  __syncthreads();
  int pre = inc - s;
  for (int q = 0; q < wid; ++q) pre += wsum[q];
  int* off = offsets + (size_t)h * (C + 1);
  for (int k = 0; k < per; ++k) {
    const int v = tid * per + k;
    if (v < C) {
      const int start = pre;
      pre += tot[v];
      run[v] += start;
      if (tile == 0) off[v] = start;
    }
  }
  if (tile == 0 && tid == 0) off[C] = N;
  __syncthreads();
  if (wid != 0) return;
  const int i0 = tile * tile_sz, i1 = min(N, i0 + tile_sz);
  const int* z = labels + (size_t)h * N;
  int* p = perm + (size_t)h * N;
  const uint64_t lt = (1ull << lane) - 1ull;
  const uint64_t gt = ~((2ull << lane) - 1ull);
  // the labels of 16 wavefront steps are loaded together (latency once per
  // 1024 tokens instead of once per step)
  constexpr int UN = 16;
  for (int c00 = i0; c00 < i1; c00 += 64 * UN) {
    int vv[UN];
#pragma unroll
    for (int k = 0; k < UN; ++k) {
      const int i = c00 + 64 * k + lane;
      vv[k] = i < i1 ? z[i] : -1;
    }
#pragma unroll
    for (int k = 0; k < UN; ++k) {
      if (c00 + 64 * k >= i1) break;
      const int i = c00 + 64 * k + lane;
      const int v = vv[k];
      const bool ok = i < i1 && (unsigned)v < (unsigned)C;
      uint64_t m = __ballot(ok);
      for (int bit = 0; bit < nbits; ++bit) {
        const bool set = (v >> bit) & 1;
        const uint64_t B = __ballot(ok && set);
        m &= set ? B : ~B;
      }
      const int rank = __popcll(m & lt);
      if (ok) p[run[v] + rank] = i;
      // one wavefront, whose LDS accesses complete in order; the fences keep
      // the compiler from moving the base reads and updates across each other
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      if (ok && (m & gt) == 0) run[v] += rank + 1;
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
  }
}

park_status launch_count_sort(const int* labels, int H, int N, int C, int* thist, int* perm,
                              int* offsets, hipStream_t st) {
  const int tsz = sort_tile(H, N, C);
  const int nt = (N + tsz - 1) / tsz;
  int nbits = 1;
  while ((1 << nbits) < C) ++nbits;
  PARK_LAUNCH("sort_hist", k_sort_hist, dim3(nt, H), dim3(256), (size_t)C * sizeof(int), st, labels,
              N, C, tsz, thist);
  PARK_LAUNCH("sort_scatter", k_sort_scatter, dim3(nt, H), dim3(256), (size_t)2 * C * sizeof(int),
              st, labels, N, C, nbits, tsz, (const int*)thist, perm, offsets);
  return PARK_OK;
}

// Xp[h][i] = X[h][perm[h][i]], 16-byte vectors.
__global__ __launch_bounds__(256) void k_gather(const uint4* __restrict__ X, const int* __restrict__ perm,
                                                int N, int vpr, uint4* __restrict__ Xp) {
  const int h = blockIdx.y;
  const size_t t = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t total = (size_t)N * vpr;
  if (t >= total) return;
  const int i = (int)(t / vpr), c = (int)(t % vpr);
  const int src = perm[(size_t)h * N + i];
  uint4 val = make_uint4(0u, 0u, 0u, 0u);
  if ((unsigned)src < (unsigned)N) val = X[((size_t)h * N + src) * vpr + c];
  Xp[((size_t)h * N + i) * vpr + c] = val;
}

park_status launch_gather(const void* X, const int* perm, int H, int N, int D, int dtype, void* Xp,
                          hipStream_t st) {
  const int vpr = (int)(D * elem_size(dtype) / 16);
  const size_t total = (size_t)N * vpr;
  dim3 g((unsigned)((total + 255) / 256), H);
  PARK_LAUNCH("gather_rows", k_gather, g, dim3(256), 0, st, (const uint4*)X, perm, N, vpr,
              (uint4*)Xp);
  return PARK_OK;
}

// Fixed-tile blocks of the cluster-ordered tokens: offsets[h][v] =
// min(v b, N) for v = 0..C, b = ceil(N / C).
__global__ __launch_bounds__(256) void k_fixed_offsets(int N, int C, int b,
                                                       int* __restrict__ offsets) {
  const int h = blockIdx.y;
  const int v = blockIdx.x * 256 + threadIdx.x;
  if (v > C) return;
  const long o = (long)v * b;
  offsets[(size_t)h * (C + 1) + v] = o < (long)N ? (int)o : N;
}

park_status launch_fixed_offsets(int H, int N, int C, int* offsets, hipStream_t st) {
  const int b = (N + C - 1) / C;
  PARK_LAUNCH("fixed_offsets", k_fixed_offsets, dim3((C + 1 + 255) / 256, H), dim3(256), 0, st,
              N, C, b, offsets);
  return PARK_OK;
}

// Rows of the nonempty blocks packed in block order: row u of x (sizes[u] >
// 0) moves to row r_u = #{w < u : sizes[w] > 0} of out, and the unit
// offsets uoff[h][u] = r_u (uoff[h][C] = the count) give each nonempty block
// exactly that one row.  One workgroup per (block, head).
__global__ __launch_bounds__(256) void k_compact_rows(const float* __restrict__ x,
                                                      const int* __restrict__ sizes, int C, int D,
                                                      float* __restrict__ out,
                                                      int* __restrict__ uoff) {
  __shared__ int red[4];
  const int h = blockIdx.y, u = blockIdx.x, tid = threadIdx.x;
  const int* sz = sizes + (size_t)h * C;
  int cnt = 0;
  for (int w = tid; w < u; w += 256) cnt += sz[w] > 0 ? 1 : 0;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o);
  if ((tid & 63) == 0) red[tid >> 6] = cnt;
  __syncthreads();
  const int r = red[0] + red[1] + red[2] + red[3];
  const bool keep = sz[u] > 0;
  if (tid == 0) {
    uoff[(size_t)h * (C + 1) + u] = r;
    if (u == C - 1) uoff[(size_t)h * (C + 1) + C] = r + (keep ? 1 : 0);
  }
  if (keep)
    for (int a = tid; a < D; a += 256)
      out[((size_t)h * C + r) * D + a] = x[((size_t)h * C + u) * D + a];
}

park_status launch_compact_rows(const float* x, const int* sizes, int H, int C, int D, float* out,
                                int* uoff, hipStream_t st) {
  PARK_LAUNCH("compact_rows", k_compact_rows, dim3(C, H), dim3(256), 0, st, x, sizes, C, D, out,
              uoff);
  return PARK_OK;
}

}  // namespace park
