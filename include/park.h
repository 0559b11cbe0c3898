/*
 * park.h -- C ABI of the PARK sparse-attention forward on AMD Instinct MI355X
 * (gfx950).  One DiT attention layer, all heads, one GPU.
 *
 * PARK ("Accurate Block Retrieval for Sparse Attention in Video Diffusion
 * Transformers") computes, per attention head:
 *   1. Euclidean k-means of the queries and QRKC k-means of the keys (keys
 *      clustered under the stabilised query second-moment metric), then a
 *      stable token permutation that makes every cluster a contiguous block
 *      (Sec. 5.2, Alg. 3);
 *   2. original-space key-block centroids c_v and sizes n_v (Eq. (8));
 *   3. PAMA block importance W^_uv (every query scored against the key
 *      centroids with a log n_v correction, softmax per query, averaged
 *      within the query block, Eqs. (8)-(9)) and a top-k / top-p block mask
 *      (Sec. 3.2, App. J);
 *   4. block-sparse attention over the selected blocks, written back in the
 *      original token order (Eq. (2)).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Tensors are [H][N][d] row-major and contiguous.  Q/K/V/Q'/K'/V' hold
 *    dims->dtype elements (PARK_F32 or PARK_BF16); d must be 64 or 128.
 *  - Every pointer argument except `dims`, `params` and `state` (which are
 *    host structs) is a DEVICE pointer owned by the caller; the library
 *    never allocates or frees device memory.  Device pointers must be
 *    16-byte aligned.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Every call only enqueues work on it and returns without synchronising,
 *    except park_check().
 *  - Argument errors are detected on the host before anything is enqueued
 *    and returned synchronously (PARK_ERR_INVALID_ARG, PARK_ERR_UNSUPPORTED,
 *    PARK_ERR_WORKSPACE); the message is available from park_last_error()
 *    (thread-local).  A failed launch returns PARK_ERR_HIP.  Numeric failures
 *    found on the device (a metric that is not positive definite, non-finite
 *    values) set bits of a status word kept in the first bytes of the
 *    workspace.  Every call taking a workspace clears that word when it
 *    starts, so it describes the most recent such call; read it with
 *    park_check().  The workspace needs no initialisation.
 *  - Cluster ids are int32 in [0, C); offsets arrays have C+1 entries with
 *    offsets[0] = 0 and offsets[C] = N; permutations map a position of the
 *    permuted order to the original token index (X'[i] = X[perm[i]]).
 *  - Empty clusters are allowed (n_v = 0).  An empty key block is never
 *    scored or selected; an empty query block gets kv_count = 0.
 *  - Limits: 1 <= H, 1 <= C <= N, C <= 2048, N * d < 2^31, 1 <= T <= 1000.
 */
#ifndef PARK_H
#define PARK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum park_status {
  PARK_OK = 0,
  PARK_ERR_INVALID_ARG = 1, /* null pointer, bad size, misalignment, bad enum */
  PARK_ERR_UNSUPPORTED = 2, /* d not in {64,128}, C > 2048, ...              */
  PARK_ERR_WORKSPACE = 3,   /* workspace smaller than park_workspace_size()  */
  PARK_ERR_HIP = 4,         /* a HIP launch or runtime call failed           */
  PARK_ERR_NUMERIC = 5      /* device-detected numeric failure (park_check)  */
} park_status;

typedef enum park_dtype { PARK_F32 = 0, PARK_BF16 = 1 } park_dtype;

/* PARK_METRIC_EUCLID: plain Euclidean k-means (the query side, Sec. 5.2, and
 * the "w/o QRKC" key side).  PARK_METRIC_QRKC: Euclidean k-means of K R where
 * Gbar = R R^T is the stabilised query second moment (Alg. 3). */
typedef enum park_metric { PARK_METRIC_EUCLID = 0, PARK_METRIC_QRKC = 1 } park_metric;

/* PARK_SELECT_TOPK: keep ceil(ratio * CK) key blocks per query block (App. J).
 * PARK_SELECT_TOPP: keep the shortest prefix, by decreasing W^ (ties by
 * increasing block id), whose cumulative W^ reaches p (Sec. 3.2). */
typedef enum park_select { PARK_SELECT_TOPK = 0, PARK_SELECT_TOPP = 1 } park_select;

/* What park_forward recomputes (clustering/mask reuse across diffusion
 * steps, Sec. 5.2 "Clustering and Reuse Strategy"). */
typedef enum park_reuse {
  PARK_RECOMPUTE = 0,              /* everything                                */
  PARK_REUSE_CLUSTERS = 1,         /* keep permutations/offsets, redo the rest  */
  PARK_REUSE_CLUSTERS_AND_MASK = 2 /* keep permutations, offsets and the mask   */
} park_reuse;

/* How park_forward estimates block importance (Sec. 5.1 and the ablation of
 * Sec. 6).  PARK_EST_PAMA: per-query softmax over the key-block scores, then
 * the mean over the query block (Eqs. (8)-(9)).  PARK_EST_QCENTROID: the
 * query-centroid estimate of Sec. 4.1, softmax_v(qbar_u . c_v / sqrt(d) +
 * log n_v) with qbar_u the mean of the block's queries rounded to float (the
 * "w/o PAMA" variant); its rows are computed in float64. */
typedef enum park_estimator { PARK_EST_PAMA = 0, PARK_EST_QCENTROID = 1 } park_estimator;

/* What a block is.  PARK_BLOCKS_CLUSTER: block v is k-means cluster v (Alg. 3:
 * K_v = {j : z_j = v}, variable sizes).  PARK_BLOCKS_FIXED: the tokens are
 * still ordered by cluster (stable argsort of the labels), but block v is the
 * fixed chunk [v b, min((v+1) b, N)) of that order with b = ceil(N / C), so
 * every block has b tokens except a shorter last one (and empty trailing
 * blocks when C b - N >= b). */
typedef enum park_block_mode { PARK_BLOCKS_CLUSTER = 0, PARK_BLOCKS_FIXED = 1 } park_block_mode;

/* How park_forward's recomputation initialises the two k-means.
 * PARK_INIT_SEEDED: from C distinct tokens drawn by the seeded shuffle (as
 * park_cluster_keys).  PARK_INIT_WARM: from the centroids in state.q_mu and
 * state.k_mu, the means of the final clusters of the previous recompute
 * (clusters change little between diffusion steps, Sec. 5.2). */
typedef enum park_init { PARK_INIT_SEEDED = 0, PARK_INIT_WARM = 1 } park_init;

typedef struct park_dims {
  int32_t H;     /* attention heads                      */
  int32_t N;     /* tokens per head (L in the paper)     */
  int32_t d;     /* head dimension: 64 or 128            */
  int32_t dtype; /* park_dtype of Q, K, V and Q', K', V' */
} park_dims;

typedef struct park_params {
  int32_t CQ;        /* query blocks N_Q (query clusters)                   */
  int32_t CK;        /* key blocks N_K (key clusters)                       */
  int32_t T;         /* k-means iterations (assign + update rounds)         */
  int32_t select;    /* park_select                                          */
  double topk_ratio; /* rho in (0, 1] for PARK_SELECT_TOPK                   */
  double topp;       /* p in (0, 1] for PARK_SELECT_TOPP                     */
  double alpha;      /* shrinkage in [0, 1] (paper: 0.05)                    */
  double eps;        /* stability constant >= 0 (1e-6)                       */
  double s_min;      /* floor of the metric scale (paper: 1e-12)             */
  uint64_t seed;     /* k-means initialisation seed                          */
  int32_t key_metric;/* park_metric for the keys (PARK_METRIC_QRKC)          */
  int32_t out_dtype; /* park_dtype of O                                      */
  int32_t estimator; /* park_estimator (PARK_EST_PAMA)                        */
  int32_t block_mode;/* park_block_mode (PARK_BLOCKS_CLUSTER)                 */
  int32_t init;      /* park_init of a recomputation (PARK_INIT_SEEDED)      */
} park_params;

/* Caller-allocated device buffers carried across park_forward calls. */
typedef struct park_state {
  int32_t* q_perm;     /* [H][N]                                  */
  int32_t* k_perm;     /* [H][N]                                  */
  int32_t* q_offsets;  /* [H][CQ+1]                               */
  int32_t* k_offsets;  /* [H][CK+1]                               */
  float* k_centroids;  /* [H][CK][d]  original-space c_v          */
  int32_t* k_sizes;    /* [H][CK]     n_v                         */
  int32_t* kv_count;   /* [H][CQ]     selected key blocks per row */
  int32_t* kv_index;   /* [H][CQ][CK] ascending block ids         */
  void* Qp;            /* [H][N][d]   permuted queries (dtype)    */
  void* Kp;            /* [H][N][d]   permuted keys               */
  void* Vp;            /* [H][N][d]   permuted values             */
  float* W;            /* [H][CQ][CK] W^ (optional, may be NULL)  */
  double* q_mu;        /* [H][CQ][d]  query centroids (may be NULL): written with the means
                          of the final query clusters by every recomputation, read as the
                          starting centroids by PARK_INIT_WARM                            */
  double* k_mu;        /* [H][CK][d]  key centroids in the original key space, likewise */
} park_state;

/* Byte sizes of the caller-allocated park_state buffers for these dims and
 * block counts, in the order the members are declared (q_perm, k_perm,
 * q_offsets, k_offsets, k_centroids, k_sizes, kv_count, kv_index, Qp, Kp,
 * Vp, W, q_mu, k_mu): bytes[i] for member i, PARK_STATE_NBUF entries.
 * Host-only.  PARK_ERR_INVALID_ARG if bytes is NULL or n < PARK_STATE_NBUF. */
#define PARK_STATE_NBUF 14
park_status park_state_sizes(const park_dims* dims, int32_t CQ, int32_t CK, size_t* bytes,
                             int32_t n);

/* Bytes of workspace any call below needs for these sizes (the maximum over
 * park_cluster_keys with C = max(CQ, CK), park_retrieve_blocks and
 * park_forward).  Host-only; never fails for valid dims. */
park_status park_workspace_size(const park_dims* dims, int32_t CQ, int32_t CK, size_t* bytes);

/* Stage 1 -- k-means clustering of one side and its stable permutation.
 * Sec. 5.2 "Clustering and Reuse Strategy" and Alg. 3 (QRKC).
 *   X        [H][N][d] dtype   points to cluster (queries or keys)
 *   Qmetric  [H][N][d] dtype   queries defining Gbar (QRKC only, else NULL)
 *   C, T, seed, side           clusters, iterations, seed; side 0 = queries,
 *                              1 = keys (selects the initialisation stream)
 *   metric                     park_metric
 *   alpha, eps, s_min          metric stabilisation (QRKC only)
 *   labels   [H][N] int32      labels of the T-th assignment (may be NULL)
 *   perm     [H][N] int32      stable argsort of the labels
 *   offsets  [H][C+1] int32    cluster boundaries in the permuted order
 *   R_out    [H][d][d] double  lower Cholesky factor, Gbar = R R^T (QRKC,
 *                              may be NULL)
 *   Xt_out   [H][N][d] float   transformed points X R (QRKC, may be NULL;
 *                              diagnostic, not needed by the hot path)
 * Metric (App. D): the k-means needs only Gbar -- its quadratic form
 * (k - mu)^T Gbar (k - mu) is the squared distance of both the Cholesky and
 * the symmetric-square-root realisation -- so any positive semidefinite Gbar
 * works, including a rank-deficient one (alpha = eps = 0 with rank-deficient
 * queries).  The Cholesky factor is taken only when R_out or Xt_out is given;
 * then a Gbar that is not positive definite is PARK_ERR_NUMERIC (park_check).
 * Initialisation: the first C entries of a Fisher-Yates shuffle of the token
 * indices driven by SplitMix64 seeded with seed ^ (0x9E3779B97F4A7C15 *
 * (2*h + side + 1)).  Labels are exact argmins of the float64 distances
 * (ties to the lowest id); an empty cluster keeps its centroid. */
park_status park_cluster_keys(const void* X, const void* Qmetric, const park_dims* dims,
                              int32_t C, int32_t T, uint64_t seed, int32_t side,
                              int32_t metric, double alpha, double eps, double s_min,
                              int32_t* labels, int32_t* perm, int32_t* offsets,
                              double* R_out, float* Xt_out, void* ws, size_t ws_bytes,
                              void* stream);

/* Row gather X'[h][i] = X[h][perm[h][i]] (Alg. 3, K' and V').
 *   X, Xp  [H][N][d] dtype;  perm [H][N] int32 (a permutation of 0..N-1). */
park_status park_gather_rows(const void* X, const int32_t* perm, const park_dims* dims,
                             void* Xp, void* stream);

/* Stage 2 -- key-block centroids in the original key space (Eq. (8), Alg. 3):
 * c_v = mean of X[perm[i]] over offsets[v] <= i < offsets[v+1], accumulated
 * in float64 and rounded to float; sizes[v] = n_v.  Empty blocks give c = 0.
 * Passing X' with the identity permutation is equivalent.
 *   centroids [H][C][d] float;  sizes [H][C] int32. */
park_status park_block_centroids(const void* X, const int32_t* perm, const int32_t* offsets,
                                 const park_dims* dims, int32_t C, float* centroids,
                                 int32_t* sizes, void* stream);

/* Stage 3 -- PAMA retrieval and mask selection (Eqs. (8)-(9), Alg. 1-2,
 * Sec. 3.2, App. J).
 *   Qp         [H][N][d] dtype   permuted queries
 *   q_offsets  [H][CQ+1]         query-block boundaries
 *   centroids  [H][CK][d] float  key-block centroids;  k_sizes [H][CK] int32
 *   select     park_select;  param = ratio (TOPK) or p (TOPP), in (0, 1]
 *   W_out      [H][CQ][CK] float W^ (may be NULL)
 *   kv_count   [H][CQ] int32;  kv_index [H][CQ][CK] int32, the first
 *              kv_count entries of each row hold the selected ids ascending.
 * The mask equals the one obtained from float64 W^ (rows whose fast-path
 * margin is below its error bound are recomputed in float64; that pass
 * leaves out of each query's normaliser the blocks whose certified bound
 * keeps them below 2^-33 of it, so a recomputed W^ is within 2^-32 relative
 * of its float64 value before the rounding to float). */
park_status park_retrieve_blocks(const void* Qp, const int32_t* q_offsets, const float* centroids,
                                 const int32_t* k_sizes, const park_dims* dims, int32_t CQ,
                                 int32_t CK, int32_t select, double param, float* W_out,
                                 int32_t* kv_count, int32_t* kv_index, void* ws,
                                 size_t ws_bytes, void* stream);

/* Stage 4 -- block-sparse attention with un-permutation (Eq. (2)).
 * For each query block u and each permuted query row i in it:
 *   O[h][q_perm[h][i]] = softmax_j(q_i . k_j / sqrt(d)) v_j over the keys j of
 *   the selected key blocks of u (softmax renormalised over those keys).
 *   Qp, Kp, Vp [H][N][d] dtype;  O [H][N][d] out_dtype (PARK_F32 or PARK_BF16,
 *   bf16 by round-to-nearest-even).  Rows of empty query blocks do not exist;
 *   every token is written exactly once; the rows of a query block with
 *   kv_count = 0 are written as zeros.
 *   lse [H][N] float (may be NULL): the natural-log normaliser of each row,
 *   log sum_j exp(q_i . k_j / sqrt(d)) over the same keys, in the original
 *   token order like O (lse[h][q_perm[h][i]]); -inf for a row whose query
 *   block selected no key.  It is what merges this output with attention
 *   over other keys (the log-sum-exp of the two normalisers).
 *   ws: device workspace of at least park_workspace_size() bytes for these
 *   dims, CQ and CK (it holds the per-call work plan); PARK_ERR_WORKSPACE if
 *   smaller than the attention part of it. */
park_status park_block_sparse_attn(const void* Qp, const void* Kp, const void* Vp,
                                   const int32_t* q_offsets, const int32_t* k_offsets,
                                   const int32_t* kv_count, const int32_t* kv_index,
                                   const int32_t* q_perm, const park_dims* dims, int32_t CQ,
                                   int32_t CK, void* O, int32_t out_dtype, float* lse, void* ws,
                                   size_t ws_bytes, void* stream);

/* park_block_sparse_attn for callers that cannot allocate device memory
 * (code under HIP graph capture, serving loops, harnesses that forbid
 * hipMalloc): the same computation and arguments without the workspace.  The
 * status word and the per-call work plan live in a static device array of the
 * library, 32 MiB per device (held until the process ends), so the call needs
 * no buffer beyond its inputs and outputs and allocates nothing.  The plan
 * takes about H (284 CQ + 16 (N/128 + (CQ + N/128)/16 + 2)) bytes;
 * PARK_ERR_WORKSPACE (nothing enqueued) when it does not fit.  Every call on
 * one device uses that device's array, so calls that overlap on one device
 * (concurrent streams or host threads) race: order them on one stream. */
park_status park_block_sparse_attn_static(const void* Qp, const void* Kp, const void* Vp,
                                          const int32_t* q_offsets, const int32_t* k_offsets,
                                          const int32_t* kv_count, const int32_t* kv_index,
                                          const int32_t* q_perm, const park_dims* dims,
                                          int32_t CQ, int32_t CK, void* O, int32_t out_dtype,
                                          float* lse, void* stream);

/* The whole layer: stages 1-4 on Q, K, V [H][N][d] (dtype), output O
 * [H][N][d] (params->out_dtype) in the original token order.  `state` holds
 * caller-allocated buffers that receive (RECOMPUTE) or supply (REUSE_*) the
 * clustering and mask.  With PARK_REUSE_CLUSTERS the permutations and offsets
 * of `state` are reused and gathers, centroids, retrieval and attention run
 * on the new tensors; PARK_REUSE_CLUSTERS_AND_MASK also reuses the mask.
 * A recomputation with params->init = PARK_INIT_WARM starts both k-means
 * from state.q_mu / state.k_mu (then required, PARK_ERR_INVALID_ARG
 * otherwise); any recomputation given those buffers leaves the means of its
 * final clusters there.
 * With RECOMPUTE the query side's clustering runs on a side stream of the
 * device (created by the library, default priority) that forks from `stream`
 * and joins back into it, beside the key side's on `stream`: work queued on
 * `stream` before and after the call stays ordered with the whole layer, and
 * a capture of `stream` records the fork and the join.  Calls on one device
 * share that side stream. */
park_status park_forward(const void* Q, const void* K, const void* V, const park_dims* dims,
                         const park_params* params, int32_t reuse, const park_state* state,
                         void* O, void* ws, size_t ws_bytes, void* stream);

/* Recomputation schedule across denoising steps (Sec. 5.2 "Clustering and
 * Reuse Strategy"; App. "Clustering and Sparse-Mask Reuse"): the clustering
 * and the mask are computed at the steps of the set `steps` and reused at the
 * steps in between.  Host-only, touches no device.
 *   step       denoising step index >= 0
 *   steps      [n_steps] strictly increasing step indices >= 0 (host memory)
 *   reuse_out  receives PARK_RECOMPUTE when step is in `steps`,
 *              PARK_REUSE_CLUSTERS_AND_MASK after the first of them, and
 *              PARK_STEP_DENSE before it (no clustering or mask exists yet:
 *              the caller runs dense attention, the warm-up of the schedule).
 * PARK_ERR_INVALID_ARG for a null pointer, n_steps < 1, a negative step or a
 * schedule that is not strictly increasing. */
#define PARK_STEP_DENSE (-1)
park_status park_schedule_step(int32_t step, const int32_t* steps, int32_t n_steps,
                               int32_t* reuse_out);

/* Hardware probes (used by tests of the error models behind the certified
 * fast paths of park_cluster_keys and park_retrieve_blocks; not part of the
 * forward).  Device pointers, asynchronous on `stream`.
 *   park_probe_exp2: y[i] = 2^x[i] by the v_exp_f32 instruction the retrieval
 *     and attention kernels use;  x, y [n] float, n >= 0.
 *   park_probe_mfma_bf16: for each of nprob problems, C = C0 + A B as a chain
 *     of K/16 v_mfma_f32_32x32x16_bf16 in increasing k (the score chains of
 *     the k-means and PAMA kernels);  A [nprob][32][K] and Bt [nprob][32][K]
 *     bf16 (Bt holds the columns of B), C0, C [nprob][32][32] float;  K a
 *     positive multiple of 16, at most 4096.
 * PARK_ERR_INVALID_ARG for a null or misaligned pointer or a bad size. */
park_status park_probe_exp2(const float* x, float* y, int64_t n, void* stream);
park_status park_probe_mfma_bf16(const uint16_t* A, const uint16_t* Bt, const float* C0, float* C,
                                 int32_t nprob, int32_t K, void* stream);

/* Synchronises `stream`, returns the sticky device status recorded in the
 * workspace `ws` (PARK_OK or PARK_ERR_NUMERIC) and clears it. */
park_status park_check(void* ws, void* stream);

/* Static description of a status code. */
const char* park_status_string(park_status s);

/* Message of the last failed call on this thread ("" if none). */
const char* park_last_error(void);

/* Per-kernel timing with HIP events on the launch stream (off by default).
 * park_profile_enable(1) starts recording around every kernel launch;
 * park_profile_read() synchronises outstanding events and writes a JSON object
 * {"kernel": {"launches": n, "ms": total}, ...} into buf (truncated to cap). */
park_status park_profile_enable(int32_t on);
park_status park_profile_reset(void);
park_status park_profile_read(char* buf, size_t cap);

#ifdef __cplusplus
}
#endif

#endif /* PARK_H */
