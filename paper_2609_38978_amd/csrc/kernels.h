// Host launchers of the PARK kernels (one group per .hip file).
#pragma once

#include "common.h"

namespace park {

// k_metric.hip --------------------------------------------------------------
size_t gram_chunks(int H, int N);
// G = Q^T Q / N and Gbar (Eq. (11)); then, separately, the Cholesky factor R of
// Gbar (the k-means only needs Gbar)
park_status launch_metric(const void* Q, int H, int N, int D, int dtype, double alpha, double eps,
                          double s_min, double* part, double* G, double* Gbar, int* status,
                          hipStream_t st);
park_status launch_metric_factor(const double* Gbar, int H, int D, double* R, int* status,
                                 hipStream_t st);
park_status launch_transform(const void* X, const double* R, int H, int N, int D, int dtype,
                             float* Xt, hipStream_t st);

// k_sort.hip ----------------------------------------------------------------
int sort_tiles(int H, int N, int C);
// Stable counting sort of labels[h][0..N) into perm/offsets (+ sizes).
park_status launch_count_sort(const int* labels, int H, int N, int C, int* thist, int* perm,
                              int* offsets, hipStream_t st);
park_status launch_gather(const void* X, const int* perm, int H, int N, int D, int dtype, void* Xp,
                          hipStream_t st);
// fixed-tile block boundaries min(v ceil(N/C), N), v = 0..C, for every head
park_status launch_fixed_offsets(int H, int N, int C, int* offsets, hipStream_t st);
// rows of the nonempty blocks (sizes > 0) of x [H][C][D] packed into out
// [H][C][D] in block order, with offsets [H][C+1] giving each such block its row
park_status launch_compact_rows(const float* x, const int* sizes, int H, int C, int D, float* out,
                                int* uoff, hipStream_t st);

// k_kmeans.hip --------------------------------------------------------------
// centroid count padded to the fast assignment's tile multiple
inline int kmeans_cpad(int C) { return (C + 63) / 64 * 64; }

// tokens per fast-assignment workgroup, 128 per block of 32 tokens a
// wavefront holds; the tokens left for the float64 refine are listed per such tile
#ifndef PARK_KM_TB
#define PARK_KM_TB 2
#endif
constexpr int kmeans_tile = 128 * PARK_KM_TB;

// key-block count padded to the fast retrieval's tile multiple
inline int pama_ckpad(int CK) { return (CK + 63) / 64 * 64; }

// exact candidate filter of the k-means rounds after the first (k_kfilter.hip)
struct KfilterBufs {
  bf16_t* g2;       // [2][H][D][D] Gbar in two bf16 parts (QRKC side)
  double* gmax;     // [H] largest absolute row sum of Gbar
  double* xn;       // [H][N] upper bound of x^T Gbar x (|x|^2 on the Euclidean side)
  double* r2;       // [H][C] squared cluster radius bound, -1 for an empty cluster
  uint32_t* cand;   // [H][C][64] candidate-set bit rows
  bf16_t* m2;       // [2][H][C][D] centroids in two bf16 parts
  float* mn;        // [H][C] |mu_v| rounded up
  // [H][C] bit patterns of non-negative doubles: per cluster, the largest
  // upper bound of D(x, mu_a)^2 over the tokens an assignment gave label a
  // (the radius of the next round, before the centroid's move)
  unsigned long long* dmax;
  // per tile of kmeans_tile sorted positions: the union of the candidate
  // sets of the clusters it spans ([H][tiles][64] bit words) and its first
  // cluster ([H][tiles])
  uint32_t* tun;
  int* talo;
};

struct KmeansBufs {
  int* init;      // [H][C]
  double* mu;     // [H][C][D] centroids in the input space
  double* w;      // [H][C][D] metric applied to the centroids
  double* b;      // [H][C]    mu^T w
  int* labels;    // [H][N]
  int* thist;     // sort tile histograms
  int* perm;      // [H][N]
  int* offsets;   // [H][C+1]
  int* status;    // sticky device status word
  // fast path (bf16 points)
  bf16_t* w3;     // [3][H][C][D] w as three bf16 parts
  float* b32;     // [H][kmeans_cpad(C)], padding +inf
  float* wn;      // [H][kmeans_cpad(C)] |w_v| (rounded up), padding 0
  float* eb;      // [H][kmeans_cpad(C)] |b_v| term of the fast-path bound, padding 0
  float* hmax;    // [H][ceil(C/16)][2] per-block max |w_v|, max eb_v
  int* nflag;     // [H][ceil(N/kmeans_tile)] tokens of each tile left for the float64 refine
  int* flags;     // [H][N]    their indices, tile t's list at kmeans_tile * t
  float* flagu;   // [H][N]    and an upper bound of their smallest exact score
  const KfilterBufs* kf = nullptr;  // candidate filter (bf16 points; null: every round dense)
  const double* mu_init = nullptr;  // [H][C][D] starting centroids (null: seeded init)
  double* mu_out = nullptr;         // [H][C][D] receives the means of the final clusters
};
park_status launch_kmeans(const void* X, const double* Gbar /* null = Euclidean */, int H, int N,
                          int D, int dtype, int C, int T, uint64_t seed, int side,
                          const KmeansBufs& kb, hipStream_t st);
park_status launch_segment_mean(const void* X, const int* perm, const int* offsets, int H, int N,
                                int D, int dtype, int C, double* mu64, float* c32, int* sizes,
                                hipStream_t st);

// k_pama.hip ----------------------------------------------------------------
struct RetrieveBufs {
  double* W64;    // [H][CQ][CK] float64 W^ (rows recomputed in float64)
  float* W32;     // [H][CQ][CK] float W^ when the caller gives no W_out
  float* delta;   // [H][CQ]     relative error bound of each fast row
  int* rows;      // [H][CQ]     rows left for the float64 path
  int* nrows;     // [H]
  bf16_t* c3;     // [3][H][CK][D] centroids as three bf16 parts
  float* lg;      // [H][pama_ckpad(CK)] log2(e) log n_v (-inf: empty and padding blocks)
  float* cn;      // [H][CK]     |c_v|
  float* bmax;    // [H][ceil(CK/16)][2] per-block max |c_v|, |log n_v|
  int4* qitems;   // [H][pama_icap] fast-retrieval work list (chunks of 32 queries)
  int* nitem;     // [H] items per head
  int* qstart;    // [H][CQ+1] first item of each query block
  double* part;   // [p64_cap][CK] raw column sums of the later items of split rows
  int4* items;    // [H CQ + p64_cap] float64 work list
  int4* srows;    // [p64_cap] split rows
  int* pcnt;      // [4] items, split rows, queue head
  // [H][CQ] top-k rows the float bound could not settle: the number of
  // ambiguous blocks ("band") whose float64 weights decide the cut, -1 for a
  // row recomputed whole; the certain blocks and the band are listed in the
  // row of kv_index until the float64 selection writes it
  int* bandc;
};
// fast retrieval: items (rounds of 64 queries) per head, and rows of round
// partial sums per head (every round after a block's first), kept in the
// float64 W^ buffer, which is free until the float64 rows are computed
inline int pama_icap(int N, int CQ) { return (N + 31) / 32 + CQ + 8; }
inline int pama_pcap(int N) { return (N + 31) / 32 + 1; }
// partial-sum rows available to the float64 pass (a quarter of the rows)
inline int p64_cap(int H, int CQ) { return (H * CQ + 3) / 4; }
park_status launch_pama64(const void* Qp, const int* q_offsets, const float* cen,
                          const int* k_sizes, int H, int N, int D, int dtype, int CQ, int CK,
                          const int4* items, int* cnt, double* part, double* W64, float* W32,
                          const int* bandc, const int* kv_index, const float* wfast,
                          const float* dfast, int plist, int* status, hipStream_t st);
park_status launch_qcen_retrieve(const float* qbar, const int* qsizes, const int* uoff,
                                 const float* cen, const int* k_sizes, int H, int D, int CQ,
                                 int CK, int mode, double param, const RetrieveBufs& rb,
                                 float* W_out, int* kv_count, int* kv_index, int* status,
                                 hipStream_t st);
park_status launch_retrieve(const void* Qp, const int* q_offsets, const float* cen,
                            const int* k_sizes, int H, int N, int D, int dtype, int CQ, int CK,
                            int mode, double param, const RetrieveBufs& rb, float* W_out,
                            int* kv_count, int* kv_index, int* status, hipStream_t st);

// k_attn.hip ----------------------------------------------------------------
// `plan` is device scratch of attn_plan_bytes(H, N, CQ) bytes (bf16 inputs only)
size_t attn_plan_bytes(int H, int N, int CQ);
park_status launch_attention(const void* Qp, const void* Kp, const void* Vp, const int* q_offsets,
                             const int* k_offsets, const int* kv_count, const int* kv_index,
                             const int* q_perm, int H, int N, int D, int dtype, int CQ, int CK,
                             void* O, int out_dtype, float* lse, void* plan, hipStream_t st);

// k_kfilter.hip -------------------------------------------------------------
// once per k-means call: Gbar's parts (QRKC) and the token norms
park_status launch_kfilter_setup(const bf16_t* X, const double* Gbar, int H, int N, int D,
                                 const KfilterBufs& kf, hipStream_t st);
// one round t >= 1: radii, candidate sets, filtered assignment (listing the
// uncertified tokens for k_refine_cand as the dense assignment does)
// measure_radius: r2 from k_radius (otherwise k_prep has bounded it from the
// previous assignment's distances)
park_status launch_kfilter_round(const bf16_t* X, int H, int N, int D, int C,
                                 const KmeansBufs& kb, const KfilterBufs& kf, bool measure_radius,
                                 hipStream_t st);

// k_probe.hip ---------------------------------------------------------------
park_status launch_probe_exp2(const float* x, float* y, long n, hipStream_t st);
park_status launch_probe_mfma(const bf16_t* A, const bf16_t* Bt, const float* C0, float* C,
                              int nprob, int K, hipStream_t st);

// misc ----------------------------------------------------------------------
park_status launch_clear_status(int* status, hipStream_t st);

}  // namespace park
