// Stable counting sort of cluster labels (pi = argsort(z), Alg. 3) and the
// row gathers X' = X[pi].  Three passes: per-tile histograms, one exclusive
// scan per head in (cluster, tile) order, and a stable scatter in which each
// tile walks its tokens in order one wavefront (64 tokens) at a time.  All
// integer work; the result is unique, so it is bit-exact and deterministic.
#include "common.h"
#include "kernels.h"

namespace park {

// Tokens per scatter tile: the smallest power of two >= 256 for which the
// per-head histogram table (C x tiles) stays below 64K entries, so that the
// single-workgroup scan stays short while the scatter (one wavefront per
// tile, serial within the tile) gets as many wavefronts as possible.
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

// thist[h][v][tile] = #{ i in tile : z_i = v }
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
  int* out = thist + (size_t)h * C * nt;
  for (int v = threadIdx.x; v < C; v += 256) out[(size_t)v * nt + tile] = hist[v];
}

// In-place exclusive scan of thist[h] (C*nt entries, cluster-major) and the
// cluster offsets o[v] = first position of cluster v, o[C] = N.  A pass covers
// SP sub-passes of 4096 entries (4 consecutive per thread, coalesced); all its
// loads are issued together and the SP block scans share one barrier.
__global__ __launch_bounds__(1024) void k_sort_scan(int* __restrict__ thist, int C, int nt, int N,
                                                    int* __restrict__ offsets) {
  constexpr int SP = 4;
  __shared__ int wsum[2][SP][16];
  const int h = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int* a = thist + (size_t)h * C * nt;
  int* off = offsets + (size_t)h * (C + 1);
  const int total = C * nt;
  int carry = 0;
  for (int pass = 0, base = 0; base < total; ++pass, base += SP * 4096) {
    int x[SP][4], sv[SP], inc[SP];
#pragma unroll
    for (int j = 0; j < SP; ++j)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = base + 4096 * j + 4 * tid + k;
        x[j][k] = e < total ? a[e] : 0;
      }
#pragma unroll
    for (int j = 0; j < SP; ++j) {
      sv[j] = (x[j][0] + x[j][1]) + (x[j][2] + x[j][3]);
      inc[j] = sv[j];
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(inc[j], o, 64);
        if (lane >= o) inc[j] += y;
      }
      if (lane == 63) wsum[pass & 1][j][wid] = inc[j];
    }
    __syncthreads();
    int run0 = carry;
#pragma unroll
    for (int j = 0; j < SP; ++j) {
      int wpre = 0, blk = 0;
#pragma unroll
      for (int w = 0; w < 16; ++w) {
        const int ws = wsum[pass & 1][j][w];
        wpre += w < wid ? ws : 0;
        blk += ws;
      }
      int run = run0 + wpre + inc[j] - sv[j];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = base + 4096 * j + 4 * tid + k;
        if (e < total) {
          a[e] = run;
          if (e % nt == 0) off[e / nt] = run;
        }
        run += x[j][k];
      }
      run0 += blk;
    }
    carry = run0;  // wsum[pass & 1] is rewritten two passes later, after another barrier
  }
  if (tid == 0) off[C] = N;
}

// Stable scatter: one wavefront per tile, tokens in increasing order.
// Equal labels inside a wave are matched with one ballot per label bit.
__global__ __launch_bounds__(64) void k_sort_scatter(const int* __restrict__ labels, int N, int C,
                                                     int nbits, int tile_sz,
                                                     const int* __restrict__ tbase,
                                                     int* __restrict__ perm) {
  extern __shared__ int run[];
  const int h = blockIdx.y, tile = blockIdx.x, nt = gridDim.x, lane = threadIdx.x;
  const int* b = tbase + (size_t)h * C * nt;
  for (int v = lane; v < C; v += 64) run[v] = b[(size_t)v * nt + tile];
  __syncthreads();
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
      __syncthreads();
      if (ok && (m & gt) == 0) run[v] += rank + 1;
      __syncthreads();
    }
  }
}

park_status launch_count_sort(const int* labels, int H, int N, int C, int* thist, int* perm,
                              int* offsets, hipStream_t st) {
  const int tsz = sort_tile(H, N, C);
  const int nt = (N + tsz - 1) / tsz;
  const size_t lds = (size_t)C * sizeof(int);
  int nbits = 1;
  while ((1 << nbits) < C) ++nbits;
  PARK_LAUNCH("sort_hist", k_sort_hist, dim3(nt, H), dim3(256), lds, st, labels, N, C, tsz, thist);
  PARK_LAUNCH("sort_scan", k_sort_scan, dim3(H), dim3(1024), 0, st, thist, C, nt, N, offsets);
  PARK_LAUNCH("sort_scatter", k_sort_scatter, dim3(nt, H), dim3(64), lds, st, labels, N, C, nbits,
              tsz, (const int*)thist, perm);
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

}  // namespace park
