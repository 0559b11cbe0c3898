// Host side of the PARK C ABI: argument validation, workspace layout, stage
// orchestration, status reporting and the optional per-kernel profiler.
#include <stdarg.h>
#include <stdlib.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"
#include "kernels.h"

namespace park {

// ------------------------------------------------------------ last error
static thread_local char g_err[512] = "";

park_status fail(park_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

// ------------------------------------------------------------ profiler
namespace {
struct ProfRec {
  const char* name;
  hipEvent_t a, b;
};
std::mutex g_pmu;
bool g_prof = false;
std::vector<hipEvent_t> g_pool;
std::vector<ProfRec> g_recs;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

bool prof_take(hipEvent_t* a, hipEvent_t* b) {
  std::lock_guard<std::mutex> lk(g_pmu);
  if (!g_prof) return false;
  *a = take_event();
  *b = take_event();
  return *a && *b;
}

void prof_commit(const char* name, hipEvent_t a, hipEvent_t b) {
  std::lock_guard<std::mutex> lk(g_pmu);
  g_recs.push_back({name, a, b});
}

// ------------------------------------------------------------ small kernels
__global__ void k_clear_int(int* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

park_status launch_clear_status(int* status, hipStream_t st) {
  PARK_LAUNCH("clear_status", k_clear_int, dim3(1), dim3(64), 0, st, status, 1);
  return PARK_OK;
}

// ------------------------------------------------------------ validation
static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

static park_status check_dims(const park_dims* dims) {
  if (!dims) return fail(PARK_ERR_INVALID_ARG, "dims is NULL");
  if (dims->H < 1 || dims->N < 1) return fail(PARK_ERR_INVALID_ARG, "need H >= 1 and N >= 1");
  if (dims->d != 64 && dims->d != 128)
    return fail(PARK_ERR_UNSUPPORTED, "head dimension %d not supported (64 or 128)", dims->d);
  if (dims->dtype != PARK_F32 && dims->dtype != PARK_BF16)
    return fail(PARK_ERR_INVALID_ARG, "unknown dtype %d", dims->dtype);
  if ((int64_t)dims->N * dims->d >= ((int64_t)1 << 31))
    return fail(PARK_ERR_UNSUPPORTED, "N * d must be below 2^31");
  return PARK_OK;
}

static park_status check_C(int C, int N, const char* what) {
  if (C < 1 || C > N) return fail(PARK_ERR_INVALID_ARG, "%s = %d must be in [1, N = %d]", what, C, N);
  if (C > 2048) return fail(PARK_ERR_UNSUPPORTED, "%s = %d exceeds 2048", what, C);
  return PARK_OK;
}

static park_status check_ptr(const void* p, const char* what) {
  if (!p) return fail(PARK_ERR_INVALID_ARG, "%s is NULL", what);
  if (!aligned16(p)) return fail(PARK_ERR_INVALID_ARG, "%s is not 16-byte aligned", what);
  return PARK_OK;
}

static park_status check_opt_ptr(const void* p, const char* what) {
  if (p && !aligned16(p)) return fail(PARK_ERR_INVALID_ARG, "%s is not 16-byte aligned", what);
  return PARK_OK;
}

static park_status check_select(int mode, double param) {
  if (mode != PARK_SELECT_TOPK && mode != PARK_SELECT_TOPP)
    return fail(PARK_ERR_INVALID_ARG, "unknown selection mode %d", mode);
  if (!(param > 0.0 && param <= 1.0))
    return fail(PARK_ERR_INVALID_ARG, "selection parameter %g must be in (0, 1]", param);
  return PARK_OK;
}

// ------------------------------------------------------------ workspace
struct ClusterWs {
  int* init;
  double* part;
  double* G;
  double* Gbar;
  double* R;
  double* mu;
  double* w;
  double* b;
  int* labels;
  int* thist;
  bf16_t* w3;
  float* b32;
  float* wn;
  float* eb;
  float* hmax;
  int* nflag;
  int* flags;
  float* flagu;
  KfilterBufs kf;
};

static ClusterWs carve_cluster(Carver& cv, int H, int N, int D, int C) {
  ClusterWs c;
  c.init = cv.take<int>((size_t)H * C);
  c.part = cv.take<double>((size_t)H * gram_chunks(H, N) * D * D);
  c.G = cv.take<double>((size_t)H * D * D);
  c.Gbar = cv.take<double>((size_t)H * D * D);
  c.R = cv.take<double>((size_t)H * D * D);
  c.mu = cv.take<double>((size_t)H * C * D);
  c.w = cv.take<double>((size_t)H * C * D);
  c.b = cv.take<double>((size_t)H * C);
  c.labels = cv.take<int>((size_t)H * N);
  c.thist = cv.take<int>((size_t)H * C * sort_tiles(H, N, C));
  c.w3 = cv.take<bf16_t>((size_t)3 * H * C * D);
  c.b32 = cv.take<float>((size_t)H * kmeans_cpad(C));
  c.wn = cv.take<float>((size_t)H * kmeans_cpad(C));
  c.eb = cv.take<float>((size_t)H * kmeans_cpad(C));
  c.hmax = cv.take<float>((size_t)2 * H * ((C + 15) / 16));
  c.nflag = cv.take<int>((size_t)H * ((N + kmeans_tile - 1) / kmeans_tile));
  c.flags = cv.take<int>((size_t)H * N);
  c.flagu = cv.take<float>((size_t)H * N);
  c.kf.g2 = cv.take<bf16_t>((size_t)2 * H * D * D);
  c.kf.gmax = cv.take<double>((size_t)H);
  c.kf.xn = cv.take<double>((size_t)H * N);
  c.kf.r2 = cv.take<double>((size_t)H * C);
  c.kf.cand = cv.take<uint32_t>((size_t)H * C * 64);
  c.kf.m2 = cv.take<bf16_t>((size_t)2 * H * C * D);
  c.kf.mn = cv.take<float>((size_t)H * C);
  c.kf.dmax = cv.take<unsigned long long>((size_t)H * C);
  c.kf.tun = cv.take<uint32_t>((size_t)H * ((N + kmeans_tile - 1) / kmeans_tile) * 64);
  c.kf.talo = cv.take<int>((size_t)H * ((N + kmeans_tile - 1) / kmeans_tile));
  return c;
}

static RetrieveBufs carve_retrieve(Carver& cv, int H, int N, int D, int CQ, int CK) {
  RetrieveBufs r;
  // float64 rows; before them, the fast pass's round partial sums (float)
  r.W64 = cv.take<double>(std::max((size_t)H * CQ * CK, ((size_t)H * pama_pcap(N) * CK + 1) / 2));
  r.W32 = cv.take<float>((size_t)H * CQ * CK);
  r.delta = cv.take<float>((size_t)H * CQ);
  r.rows = cv.take<int>((size_t)H * CQ);
  r.nrows = cv.take<int>((size_t)H);
  r.c3 = cv.take<bf16_t>((size_t)3 * H * CK * D);
  r.lg = cv.take<float>((size_t)H * pama_ckpad(CK));
  r.cn = cv.take<float>((size_t)H * CK);
  r.bmax = cv.take<float>((size_t)2 * H * ((CK + 15) / 16));
  r.qitems = cv.take<int4>((size_t)H * pama_icap(N, CQ));
  r.nitem = cv.take<int>((size_t)H);
  r.qstart = cv.take<int>((size_t)H * (CQ + 1));
  r.part = cv.take<double>((size_t)p64_cap(H, CQ) * CK);
  r.items = cv.take<int4>((size_t)H * CQ + p64_cap(H, CQ));
  r.srows = cv.take<int4>((size_t)p64_cap(H, CQ) + 1);
  r.pcnt = cv.take<int>(4);
  r.bandc = cv.take<int>((size_t)H * CQ);
  return r;
}

// attention: the status word, then the chunk plan
static size_t attn_ws_end(int H, int N, int CQ) {
  Carver a(nullptr);
  a.take<int>(64);
  a.take<int4>(attn_plan_bytes(H, N, CQ) / sizeof(int4));
  return a.off;
}

static void* carve_attn_plan(void* ws, int H, int N, int CQ) {
  Carver cv(ws);
  cv.take<int>(64);
  return cv.take<int4>(attn_plan_bytes(H, N, CQ) / sizeof(int4));
}

// query-centroid estimator: the block means of the queries, packed, and the
// offsets giving each nonempty query block its one row
struct QcenBufs {
  float* qbar;   // [H][CQ][D]
  float* qrows;  // [H][CQ][D]
  int* qsizes;   // [H][CQ]
  int* uoff;     // [H][CQ+1]
};

static QcenBufs carve_qcen(Carver& cv, int H, int D, int CQ) {
  QcenBufs q;
  q.qbar = cv.take<float>((size_t)H * CQ * D);
  q.qrows = cv.take<float>((size_t)H * CQ * D);
  q.qsizes = cv.take<int>((size_t)H * CQ);
  q.uoff = cv.take<int>((size_t)H * (CQ + 1));
  return q;
}

// status word first, then the largest of the cluster, retrieval and attention regions
static size_t ws_bytes_for(int H, int N, int D, int CQ, int CK) {
  Carver a(nullptr);
  a.take<int>(64);
  const size_t base = a.off;
  Carver c1(nullptr);
  c1.off = base;
  carve_cluster(c1, H, N, D, CQ);  // query side
  carve_cluster(c1, H, N, D, CK);  // key side (the two sides can run at the same time)
  Carver c2(nullptr);
  c2.off = base;
  carve_retrieve(c2, H, N, D, CQ, CK);
  Carver c3(nullptr);  // query-centroid estimator: CQ float rows per head
  c3.off = base;
  carve_qcen(c3, H, D, CQ);
  carve_retrieve(c3, H, CQ, D, CQ, CK);
  return std::max(std::max(std::max(c1.off, c2.off), c3.off), attn_ws_end(H, N, CQ)) + 256;
}

static park_status check_ws(void* ws, size_t ws_bytes, size_t need) {
  PARK_TRY(check_ptr(ws, "workspace"));
  if (ws_bytes < need)
    return fail(PARK_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required",
                ws_bytes, need);
  return PARK_OK;
}

// arguments of the attention entry points (everything but the workspace)
static park_status check_attn_args(const void* Qp, const void* Kp, const void* Vp,
                                   const int32_t* q_offsets, const int32_t* k_offsets,
                                   const int32_t* kv_count, const int32_t* kv_index,
                                   const int32_t* q_perm, const park_dims* dims, int32_t CQ,
                                   int32_t CK, void* O, int32_t out_dtype, float* lse) {
  PARK_TRY(check_dims(dims));
  PARK_TRY(check_C(CQ, dims->N, "CQ"));
  PARK_TRY(check_C(CK, dims->N, "CK"));
  if (out_dtype != PARK_F32 && out_dtype != PARK_BF16)
    return fail(PARK_ERR_INVALID_ARG, "unknown out_dtype %d", out_dtype);
  PARK_TRY(check_ptr(Qp, "Qp"));
  PARK_TRY(check_ptr(Kp, "Kp"));
  PARK_TRY(check_ptr(Vp, "Vp"));
  PARK_TRY(check_ptr(q_offsets, "q_offsets"));
  PARK_TRY(check_ptr(k_offsets, "k_offsets"));
  PARK_TRY(check_ptr(kv_count, "kv_count"));
  PARK_TRY(check_ptr(kv_index, "kv_index"));
  PARK_TRY(check_ptr(q_perm, "q_perm"));
  PARK_TRY(check_ptr(O, "O"));
  PARK_TRY(check_opt_ptr(lse, "lse"));
  return PARK_OK;
}

// ------------------------------------------------------------ static scratch
// park_block_sparse_attn_static keeps its status word and work plan in this
// file-scope device array instead of a caller workspace.  Each device holds
// its own copy; host code uses only the address hipGetSymbolAddress returns
// for the current device (the array's name is a host-side stand-in), kept per
// device after the first call there.  Every call on a device shares it.
constexpr size_t kStaticScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[64];

static park_status static_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(PARK_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= 64) return fail(PARK_ERR_UNSUPPORTED, "device %d", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(PARK_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return PARK_OK;
}

// ------------------------------------------------------------ side stream
// The query side's clustering runs on a second stream of the device, beside
// the key side's metric Gbar and k-means on the caller's stream, and later
// the key and value gathers run there beside the retrieval: the two streams
// share nothing but the status word, which kernels only OR into.  The stream
// (default priority) and its fork/join events are created on the first call
// that is not being captured; until then the sides run one after the other.
// A call holds the device's lock while it queues its work, so concurrent calls
// on one device cannot swap each other's events.
struct SideStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  std::mutex mu;  // held while a call queues its work (the events are shared)
};
static std::mutex g_side_mu;
static SideStream g_side[64];

static SideStream* side_stream(hipStream_t st) {
  // PARK_SIDE_STREAM=0 keeps everything on the caller's stream (kernel
  // durations then carry no overlap with the other side's kernels)
  static const bool off = [] {
    const char* e = getenv("PARK_SIDE_STREAM");
    return e && e[0] == '0';
  }();
  if (off) return nullptr;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lk(g_side_mu);
  SideStream& a = g_side[dev];
  if (!a.s) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone)
      return nullptr;
    hipStream_t s2 = nullptr;
    hipEvent_t e[2] = {nullptr, nullptr};
    if (hipStreamCreateWithFlags(&s2, hipStreamNonBlocking) != hipSuccess) return nullptr;
    for (int i = 0; i < 2; ++i)
      if (hipEventCreateWithFlags(&e[i], hipEventDisableTiming) != hipSuccess) {
        for (int j = 0; j < i; ++j) hipEventDestroy(e[j]);
        hipStreamDestroy(s2);
        return nullptr;
      }
    a.s = s2;
    a.fork = e[0];
    a.join = e[1];
  }
  return &a;
}

static park_status ev_record(hipEvent_t ev, hipStream_t s) {
  const hipError_t e = hipEventRecord(ev, s);
  return e == hipSuccess ? PARK_OK : fail(PARK_ERR_HIP, "event record: %s", hipGetErrorString(e));
}
static park_status ev_wait(hipStream_t s, hipEvent_t ev) {
  const hipError_t e = hipStreamWaitEvent(s, ev, 0);
  return e == hipSuccess ? PARK_OK : fail(PARK_ERR_HIP, "stream wait: %s", hipGetErrorString(e));
}

// ------------------------------------------------------------ stage bodies
// `region` (optional) is the cluster workspace to use; by default the first
// region after the status word.  `parts`: bit 1 the metric Gbar, bit 4 its
// Cholesky factor R (and the transform), bit 2 the k-means (with the Gbar
// already in the region); 7 all, in that order.
static park_status cluster_body(const void* X, const void* Qm, const park_dims& dm, int C, int T,
                                uint64_t seed, int side, int metric, double alpha, double eps,
                                double s_min, int* labels, int* perm, int* offsets, double* R_out,
                                float* Xt_out, void* ws, hipStream_t st,
                                const ClusterWs* region = nullptr, int parts = 7,
                                const double* mu_init = nullptr, double* mu_out = nullptr) {
  const int H = dm.H, N = dm.N, D = dm.d;
  Carver cv(ws);
  int* status = cv.take<int>(64);
  ClusterWs cw = region ? *region : carve_cluster(cv, H, N, D, C);
  const double* Gbar = nullptr;
  if (metric == PARK_METRIC_QRKC) {
    if (parts & 1)
      PARK_TRY(launch_metric(Qm, H, N, D, dm.dtype, alpha, eps, s_min, cw.part, cw.G, cw.Gbar,
                             status, st));
    if (parts & 4) {
      double* R = R_out ? R_out : cw.R;
      PARK_TRY(launch_metric_factor(cw.Gbar, H, D, R, status, st));
      if (Xt_out) PARK_TRY(launch_transform(X, R, H, N, D, dm.dtype, Xt_out, st));
    }
    Gbar = cw.Gbar;
  }
  if (!(parts & 2)) return PARK_OK;
  KmeansBufs kb;
  kb.init = cw.init;
  kb.mu = cw.mu;
  kb.w = cw.w;
  kb.b = cw.b;
  kb.labels = labels ? labels : cw.labels;
  kb.thist = cw.thist;
  kb.perm = perm;
  kb.offsets = offsets;
  kb.status = status;
  kb.w3 = cw.w3;
  kb.b32 = cw.b32;
  kb.wn = cw.wn;
  kb.eb = cw.eb;
  kb.hmax = cw.hmax;
  kb.nflag = cw.nflag;
  kb.flags = cw.flags;
  kb.flagu = cw.flagu;
  kb.kf = &cw.kf;
  kb.mu_init = mu_init;
  kb.mu_out = mu_out;
  return launch_kmeans(X, Gbar, H, N, D, dm.dtype, C, T, seed, side, kb, st);
}

static park_status retrieve_body(const void* Qp, const int* q_offsets, const float* cen,
                                 const int* k_sizes, const park_dims& dm, int CQ, int CK,
                                 int mode, double param, float* W_out, int* kv_count,
                                 int* kv_index, void* ws, hipStream_t st) {
  Carver cv(ws);
  int* status = cv.take<int>(64);
  RetrieveBufs rb = carve_retrieve(cv, dm.H, dm.N, dm.d, CQ, CK);
  return launch_retrieve(Qp, q_offsets, cen, k_sizes, dm.H, dm.N, dm.d, dm.dtype, CQ, CK, mode,
                         param, rb, W_out, kv_count, kv_index, status, st);
}

}  // namespace park

using namespace park;

// ============================================================ C ABI
// The retrieval of park_forward: key centroids (through the permutation),
// then PAMA or the query-centroid estimate and the mask, on `st`.
static park_status retrieve_stage(const void* K, const park_params* p, const park_state* s,
                                  const park_dims* dims, double param, void* ws, hipStream_t st) {
  const int H = dims->H, N = dims->N, D = dims->d;
  PARK_TRY(launch_segment_mean(K, s->k_perm, s->k_offsets, H, N, D, dims->dtype, p->CK, nullptr,
                               s->k_centroids, s->k_sizes, st));
  if (p->estimator == PARK_EST_PAMA)
    return retrieve_body(s->Qp, s->q_offsets, s->k_centroids, s->k_sizes, *dims, p->CQ, p->CK,
                         p->select, param, s->W, s->kv_count, s->kv_index, ws, st);
  // query-centroid estimate: one float row (the block mean) per query block,
  // scored in float64 (empty blocks: a zero row) and selected by the
  // certified float selection, the rows it cannot settle by the float64 one
  // (uoff: one row per nonempty block)
  Carver qc(ws);
  int* status = qc.take<int>(64);
  const QcenBufs qb = carve_qcen(qc, H, D, p->CQ);
  const RetrieveBufs rb = carve_retrieve(qc, H, p->CQ, D, p->CQ, p->CK);
  PARK_TRY(launch_segment_mean(s->Qp, nullptr, s->q_offsets, H, N, D, dims->dtype, p->CQ,
                               nullptr, qb.qbar, qb.qsizes, st));
  PARK_TRY(launch_compact_rows(qb.qbar, qb.qsizes, H, p->CQ, D, qb.qrows, qb.uoff, st));
  return launch_qcen_retrieve(qb.qbar, qb.qsizes, qb.uoff, s->k_centroids, s->k_sizes, H, D,
                              p->CQ, p->CK, p->select, param, rb, s->W, s->kv_count, s->kv_index,
                              status, st);
}

extern "C" {

const char* park_status_string(park_status s) {
  // a C caller may pass any int; outside the enumerators a C++ park_status
  // value is undefined, so the argument's bits are read as an int
  static_assert(sizeof(park_status) == sizeof(int), "park_status is an int in C");
  int v;
  memcpy(&v, &s, sizeof v);
  switch (v) {
    case PARK_OK: return "ok";
    case PARK_ERR_INVALID_ARG: return "invalid argument";
    case PARK_ERR_UNSUPPORTED: return "unsupported configuration";
    case PARK_ERR_WORKSPACE: return "workspace too small";
    case PARK_ERR_HIP: return "HIP runtime error";
    case PARK_ERR_NUMERIC: return "numeric failure on the device";
  }
  return "unknown status";
}

const char* park_last_error(void) { return g_err; }

park_status park_workspace_size(const park_dims* dims, int32_t CQ, int32_t CK, size_t* bytes) {
  g_err[0] = 0;
  PARK_TRY(check_dims(dims));
  if (!bytes) return fail(PARK_ERR_INVALID_ARG, "bytes is NULL");
  PARK_TRY(check_C(CQ, dims->N, "CQ"));
  PARK_TRY(check_C(CK, dims->N, "CK"));
  *bytes = ws_bytes_for(dims->H, dims->N, dims->d, CQ, CK);
  return PARK_OK;
}

park_status park_state_sizes(const park_dims* dims, int32_t CQ, int32_t CK, size_t* bytes,
                             int32_t n) {
  g_err[0] = 0;
  PARK_TRY(check_dims(dims));
  if (!bytes) return fail(PARK_ERR_INVALID_ARG, "bytes is NULL");
  if (n < PARK_STATE_NBUF)
    return fail(PARK_ERR_INVALID_ARG, "bytes has %d entries, %d needed", n, PARK_STATE_NBUF);
  PARK_TRY(check_C(CQ, dims->N, "CQ"));
  PARK_TRY(check_C(CK, dims->N, "CK"));
  const size_t H = dims->H, N = dims->N, D = dims->d;
  const size_t el = dims->dtype == PARK_BF16 ? 2 : 4;
  const size_t b[PARK_STATE_NBUF] = {
      H * N * 4,            H * N * 4,            H * (CQ + 1) * 4,    H * (CK + 1) * 4,
      H * CK * D * 4,       H * CK * 4,           H * CQ * 4,          H * CQ * CK * 4,
      H * N * D * el,       H * N * D * el,       H * N * D * el,      H * CQ * CK * 4,
      H * CQ * D * 8,       H * CK * D * 8};
  for (int i = 0; i < PARK_STATE_NBUF; ++i) bytes[i] = b[i];
  return PARK_OK;
}

park_status park_cluster_keys(const void* X, const void* Qmetric, const park_dims* dims, int32_t C,
                              int32_t T, uint64_t seed, int32_t side, int32_t metric, double alpha,
                              double eps, double s_min, int32_t* labels, int32_t* perm,
                              int32_t* offsets, double* R_out, float* Xt_out, void* ws,
                              size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  PARK_TRY(check_dims(dims));
  PARK_TRY(check_C(C, dims->N, "C"));
  if (T < 1 || T > 1000) return fail(PARK_ERR_INVALID_ARG, "T = %d must be in [1, 1000]", T);
  if (side != 0 && side != 1) return fail(PARK_ERR_INVALID_ARG, "side must be 0 or 1");
  if (metric != PARK_METRIC_EUCLID && metric != PARK_METRIC_QRKC)
    return fail(PARK_ERR_INVALID_ARG, "unknown metric %d", metric);
  PARK_TRY(check_ptr(X, "X"));
  PARK_TRY(check_ptr(perm, "perm"));
  PARK_TRY(check_ptr(offsets, "offsets"));
  PARK_TRY(check_opt_ptr(labels, "labels"));
  if (metric == PARK_METRIC_QRKC) {
    PARK_TRY(check_ptr(Qmetric, "Qmetric"));
    if (!(alpha >= 0.0 && alpha <= 1.0)) return fail(PARK_ERR_INVALID_ARG, "alpha must be in [0, 1]");
    if (!(eps >= 0.0) || !(s_min > 0.0) || eps > 1e300 || s_min > 1e300)
      return fail(PARK_ERR_INVALID_ARG, "need eps >= 0 and s_min > 0, both finite");
    PARK_TRY(check_opt_ptr(R_out, "R_out"));
    PARK_TRY(check_opt_ptr(Xt_out, "Xt_out"));
  } else if (R_out || Xt_out) {
    return fail(PARK_ERR_INVALID_ARG, "R_out / Xt_out need the QRKC metric");
  }
  PARK_TRY(check_ws(ws, ws_bytes, ws_bytes_for(dims->H, dims->N, dims->d, C, C)));
  hipStream_t st = (hipStream_t)stream;
  Carver cv(ws);
  PARK_TRY(launch_clear_status(cv.take<int>(64), st));
  // the k-means needs only Gbar (any positive semidefinite one: its quadratic
  // form is the symmetric-square-root realisation); the Cholesky factor is
  // taken, and must exist, only when R or X R is asked for
  return cluster_body(X, Qmetric, *dims, C, T, seed, side, metric, alpha, eps, s_min, labels, perm,
                      offsets, R_out, Xt_out, ws, st, nullptr, (R_out || Xt_out) ? 7 : 3);
}

park_status park_gather_rows(const void* X, const int32_t* perm, const park_dims* dims, void* Xp,
                             void* stream) {
  g_err[0] = 0;
  PARK_TRY(check_dims(dims));
  PARK_TRY(check_ptr(X, "X"));
  PARK_TRY(check_ptr(perm, "perm"));
  PARK_TRY(check_ptr(Xp, "Xp"));
  return launch_gather(X, perm, dims->H, dims->N, dims->d, dims->dtype, Xp, (hipStream_t)stream);
}

park_status park_block_centroids(const void* X, const int32_t* perm, const int32_t* offsets,
                                 const park_dims* dims, int32_t C, float* centroids,
                                 int32_t* sizes, void* stream) {
  g_err[0] = 0;
  PARK_TRY(check_dims(dims));
  PARK_TRY(check_C(C, dims->N, "C"));
  PARK_TRY(check_ptr(X, "X"));
  PARK_TRY(check_ptr(perm, "perm"));
  PARK_TRY(check_ptr(offsets, "offsets"));
  PARK_TRY(check_ptr(centroids, "centroids"));
  PARK_TRY(check_ptr(sizes, "sizes"));
  return launch_segment_mean(X, perm, offsets, dims->H, dims->N, dims->d, dims->dtype, C, nullptr,
                             centroids, sizes, (hipStream_t)stream);
}

park_status park_retrieve_blocks(const void* Qp, const int32_t* q_offsets, const float* centroids,
                                 const int32_t* k_sizes, const park_dims* dims, int32_t CQ,
                                 int32_t CK, int32_t select, double param, float* W_out,
                                 int32_t* kv_count, int32_t* kv_index, void* ws, size_t ws_bytes,
                                 void* stream) {
  g_err[0] = 0;
  PARK_TRY(check_dims(dims));
  PARK_TRY(check_C(CQ, dims->N, "CQ"));
  PARK_TRY(check_C(CK, dims->N, "CK"));
  PARK_TRY(check_select(select, param));
  PARK_TRY(check_ptr(Qp, "Qp"));
  PARK_TRY(check_ptr(q_offsets, "q_offsets"));
  PARK_TRY(check_ptr(centroids, "centroids"));
  PARK_TRY(check_ptr(k_sizes, "k_sizes"));
  PARK_TRY(check_ptr(kv_count, "kv_count"));
  PARK_TRY(check_ptr(kv_index, "kv_index"));
  PARK_TRY(check_opt_ptr(W_out, "W_out"));
  PARK_TRY(check_ws(ws, ws_bytes, ws_bytes_for(dims->H, dims->N, dims->d, CQ, CK)));
  hipStream_t st = (hipStream_t)stream;
  Carver cv(ws);
  PARK_TRY(launch_clear_status(cv.take<int>(64), st));
  return retrieve_body(Qp, q_offsets, centroids, k_sizes, *dims, CQ, CK, select, param, W_out,
                       kv_count, kv_index, ws, st);
}

park_status park_block_sparse_attn(const void* Qp, const void* Kp, const void* Vp,
                                   const int32_t* q_offsets, const int32_t* k_offsets,
                                   const int32_t* kv_count, const int32_t* kv_index,
                                   const int32_t* q_perm, const park_dims* dims, int32_t CQ,
                                   int32_t CK, void* O, int32_t out_dtype, float* lse, void* ws,
                                   size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  PARK_TRY(check_attn_args(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index, q_perm, dims, CQ,
                           CK, O, out_dtype, lse));
  PARK_TRY(check_ws(ws, ws_bytes, attn_ws_end(dims->H, dims->N, CQ) + 256));
  hipStream_t st = (hipStream_t)stream;
  Carver cv(ws);
  PARK_TRY(launch_clear_status(cv.take<int>(64), st));
  return launch_attention(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index, q_perm, dims->H,
                          dims->N, dims->d, dims->dtype, CQ, CK, O, out_dtype, lse,
                          carve_attn_plan(ws, dims->H, dims->N, CQ), st);
}

park_status park_block_sparse_attn_static(const void* Qp, const void* Kp, const void* Vp,
                                          const int32_t* q_offsets, const int32_t* k_offsets,
                                          const int32_t* kv_count, const int32_t* kv_index,
                                          const int32_t* q_perm, const park_dims* dims,
                                          int32_t CQ, int32_t CK, void* O, int32_t out_dtype,
                                          float* lse, void* stream) {
  g_err[0] = 0;
  PARK_TRY(check_attn_args(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index, q_perm, dims, CQ,
                           CK, O, out_dtype, lse));
  const size_t need = attn_ws_end(dims->H, dims->N, CQ);
  if (need > kStaticScratchBytes)
    return fail(PARK_ERR_WORKSPACE,
                "H = %d, N = %d, CQ = %d need %zu bytes of plan, more than the %zu bytes of "
                "static scratch: use park_block_sparse_attn with a workspace",
                dims->H, dims->N, CQ, need, kStaticScratchBytes);
  void* ptr = nullptr;
  PARK_TRY(static_scratch(&ptr));
  hipStream_t st = (hipStream_t)stream;
  Carver cv(ptr);
  PARK_TRY(launch_clear_status(cv.take<int>(64), st));
  return launch_attention(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index, q_perm, dims->H,
                          dims->N, dims->d, dims->dtype, CQ, CK, O, out_dtype, lse,
                          carve_attn_plan(ptr, dims->H, dims->N, CQ), st);
}

park_status park_forward(const void* Q, const void* K, const void* V, const park_dims* dims,
                         const park_params* p, int32_t reuse, const park_state* s, void* O,
                         void* ws, size_t ws_bytes, void* stream) {
  g_err[0] = 0;
  PARK_TRY(check_dims(dims));
  if (!p) return fail(PARK_ERR_INVALID_ARG, "params is NULL");
  if (!s) return fail(PARK_ERR_INVALID_ARG, "state is NULL");
  PARK_TRY(check_C(p->CQ, dims->N, "CQ"));
  PARK_TRY(check_C(p->CK, dims->N, "CK"));
  if (p->T < 1 || p->T > 1000) return fail(PARK_ERR_INVALID_ARG, "T must be in [1, 1000]");
  const double param = p->select == PARK_SELECT_TOPK ? p->topk_ratio : p->topp;
  PARK_TRY(check_select(p->select, param));
  if (p->key_metric != PARK_METRIC_EUCLID && p->key_metric != PARK_METRIC_QRKC)
    return fail(PARK_ERR_INVALID_ARG, "unknown key metric %d", p->key_metric);
  if (!(p->alpha >= 0.0 && p->alpha <= 1.0) || !(p->eps >= 0.0) || !(p->s_min > 0.0) ||
      p->eps > 1e300 || p->s_min > 1e300)
    return fail(PARK_ERR_INVALID_ARG, "need alpha in [0,1], eps >= 0, s_min > 0");
  if (p->out_dtype != PARK_F32 && p->out_dtype != PARK_BF16)
    return fail(PARK_ERR_INVALID_ARG, "unknown out_dtype %d", p->out_dtype);
  if (p->estimator != PARK_EST_PAMA && p->estimator != PARK_EST_QCENTROID)
    return fail(PARK_ERR_INVALID_ARG, "unknown estimator %d", p->estimator);
  if (p->block_mode != PARK_BLOCKS_CLUSTER && p->block_mode != PARK_BLOCKS_FIXED)
    return fail(PARK_ERR_INVALID_ARG, "unknown block mode %d", p->block_mode);
  if (p->init != PARK_INIT_SEEDED && p->init != PARK_INIT_WARM)
    return fail(PARK_ERR_INVALID_ARG, "unknown init %d", p->init);
  if (p->init == PARK_INIT_WARM && reuse == PARK_RECOMPUTE && (!s->q_mu || !s->k_mu))
    return fail(PARK_ERR_INVALID_ARG, "PARK_INIT_WARM needs state.q_mu and state.k_mu");
  if (reuse < PARK_RECOMPUTE || reuse > PARK_REUSE_CLUSTERS_AND_MASK)
    return fail(PARK_ERR_INVALID_ARG, "unknown reuse mode %d", reuse);
  PARK_TRY(check_ptr(Q, "Q"));
  PARK_TRY(check_ptr(K, "K"));
  PARK_TRY(check_ptr(V, "V"));
  PARK_TRY(check_ptr(O, "O"));
  PARK_TRY(check_ptr(s->q_perm, "state.q_perm"));
  PARK_TRY(check_ptr(s->k_perm, "state.k_perm"));
  PARK_TRY(check_ptr(s->q_offsets, "state.q_offsets"));
  PARK_TRY(check_ptr(s->k_offsets, "state.k_offsets"));
  PARK_TRY(check_ptr(s->k_centroids, "state.k_centroids"));
  PARK_TRY(check_ptr(s->k_sizes, "state.k_sizes"));
  PARK_TRY(check_ptr(s->kv_count, "state.kv_count"));
  PARK_TRY(check_ptr(s->kv_index, "state.kv_index"));
  PARK_TRY(check_ptr(s->Qp, "state.Qp"));
  PARK_TRY(check_ptr(s->Kp, "state.Kp"));
  PARK_TRY(check_ptr(s->Vp, "state.Vp"));
  PARK_TRY(check_opt_ptr(s->W, "state.W"));
  PARK_TRY(check_opt_ptr(s->q_mu, "state.q_mu"));
  PARK_TRY(check_opt_ptr(s->k_mu, "state.k_mu"));
  const int H = dims->H, N = dims->N, D = dims->d;
  PARK_TRY(check_ws(ws, ws_bytes, ws_bytes_for(H, N, D, p->CQ, p->CK)));
  hipStream_t st = (hipStream_t)stream;
  Carver cv(ws);
  PARK_TRY(launch_clear_status(cv.take<int>(64), st));
  if (reuse == PARK_RECOMPUTE) {
    // query side on the side stream, key side here, joined before the gathers
    Carver rc(ws);
    rc.take<int>(64);
    const ClusterWs cq = carve_cluster(rc, H, N, D, p->CQ);
    const ClusterWs ck = carve_cluster(rc, H, N, D, p->CK);
    // queued in this order so that both streams get work early: the key
    // side's metric Gbar, the whole query side (side stream), the key side's
    // k-means.  The k-means needs only Gbar, whose quadratic form is the
    // symmetric-square-root realisation of the metric, so no factor is taken
    // and a rank-deficient (positive semidefinite) Gbar is fine
    SideStream* side = side_stream(st);
    hipStream_t sq = side ? side->s : st;
    std::unique_lock<std::mutex> lk;
    if (side) {
      lk = std::unique_lock<std::mutex>(side->mu);
      PARK_TRY(ev_record(side->fork, st));
      PARK_TRY(ev_wait(sq, side->fork));
    }
    // warm start: both sides from the previous recompute's means; either way
    // the final means are left in state.q_mu / k_mu when they are given
    const bool warm = p->init == PARK_INIT_WARM;
    park_status r = cluster_body(K, Q, *dims, p->CK, p->T, p->seed, 1, p->key_metric, p->alpha,
                                 p->eps, p->s_min, nullptr, s->k_perm, s->k_offsets, nullptr,
                                 nullptr, ws, st, &ck, 1);
    if (r == PARK_OK)
      r = cluster_body(Q, nullptr, *dims, p->CQ, p->T, p->seed, 0, PARK_METRIC_EUCLID, 0, 0, 1,
                       nullptr, s->q_perm, s->q_offsets, nullptr, nullptr, ws, sq, &cq, 7,
                       warm ? s->q_mu : nullptr, s->q_mu);
    if (r == PARK_OK)
      r = cluster_body(K, Q, *dims, p->CK, p->T, p->seed, 1, p->key_metric, p->alpha, p->eps,
                       p->s_min, nullptr, s->k_perm, s->k_offsets, nullptr, nullptr, ws, st, &ck,
                       2, warm ? s->k_mu : nullptr, s->k_mu);
    if (side) {  // joined also after an error
      PARK_TRY(ev_record(side->join, sq));
      PARK_TRY(ev_wait(st, side->join));
    }
    PARK_TRY(r);
    if (p->block_mode == PARK_BLOCKS_FIXED) {  // same order, fixed chunks of it
      PARK_TRY(launch_fixed_offsets(H, N, p->CQ, s->q_offsets, st));
      PARK_TRY(launch_fixed_offsets(H, N, p->CK, s->k_offsets, st));
    }
  }
  PARK_TRY(launch_gather(Q, s->q_perm, H, N, D, dims->dtype, s->Qp, st));
  // with a retrieval to run, the keys and values are gathered on the side
  // stream meanwhile (the retrieval reads the key centroids, which are taken
  // through the permutation: the same rows in the same order), joined before
  // the attention
  const bool retrieve = reuse != PARK_REUSE_CLUSTERS_AND_MASK;
  SideStream* kv_side = retrieve ? side_stream(st) : nullptr;
  hipStream_t skv = kv_side ? kv_side->s : st;
  std::unique_lock<std::mutex> kv_lk;
  if (kv_side) {
    kv_lk = std::unique_lock<std::mutex>(kv_side->mu);
    PARK_TRY(ev_record(kv_side->fork, st));
    PARK_TRY(ev_wait(skv, kv_side->fork));
  }
  park_status rkv = launch_gather(K, s->k_perm, H, N, D, dims->dtype, s->Kp, skv);
  if (rkv == PARK_OK) rkv = launch_gather(V, s->k_perm, H, N, D, dims->dtype, s->Vp, skv);
  if (kv_side) {  // joined also after an error
    const park_status rj = ev_record(kv_side->join, skv);
    if (rkv == PARK_OK) rkv = rj;
  }
  park_status rr = rkv == PARK_OK && retrieve
                       ? retrieve_stage(K, p, s, dims, param, ws, st)
                       : PARK_OK;
  if (kv_side) {
    const park_status rw = ev_wait(st, kv_side->join);
    if (rr == PARK_OK) rr = rw;
  }
  PARK_TRY(rkv);
  PARK_TRY(rr);
  return launch_attention(s->Qp, s->Kp, s->Vp, s->q_offsets, s->k_offsets, s->kv_count,
                          s->kv_index, s->q_perm, H, N, D, dims->dtype, p->CQ, p->CK, O,
                          p->out_dtype, nullptr, carve_attn_plan(ws, H, N, p->CQ), st);
}


park_status park_schedule_step(int32_t step, const int32_t* steps, int32_t n_steps,
                               int32_t* reuse_out) {
  g_err[0] = 0;
  if (!steps || !reuse_out) return fail(PARK_ERR_INVALID_ARG, "steps / reuse_out is NULL");
  if (n_steps < 1) return fail(PARK_ERR_INVALID_ARG, "the schedule needs at least one step");
  if (step < 0) return fail(PARK_ERR_INVALID_ARG, "step %d is negative", step);
  for (int i = 0; i < n_steps; ++i) {
    if (steps[i] < 0) return fail(PARK_ERR_INVALID_ARG, "schedule entry %d is negative", i);
    if (i > 0 && steps[i] <= steps[i - 1])
      return fail(PARK_ERR_INVALID_ARG, "schedule is not strictly increasing at entry %d", i);
  }
  int32_t mode = PARK_STEP_DENSE;
  if (step >= steps[0]) {
    mode = PARK_REUSE_CLUSTERS_AND_MASK;
    for (int i = 0; i < n_steps; ++i)
      if (steps[i] == step) mode = PARK_RECOMPUTE;
  }
  *reuse_out = mode;
  return PARK_OK;
}

park_status park_probe_exp2(const float* x, float* y, int64_t n, void* stream) {
  g_err[0] = 0;
  if (n < 0 || n > ((int64_t)1 << 40)) return fail(PARK_ERR_INVALID_ARG, "n = %lld", (long long)n);
  if (n > 0) {
    PARK_TRY(check_ptr(x, "x"));
    PARK_TRY(check_ptr(y, "y"));
  }
  return launch_probe_exp2(x, y, (long)n, (hipStream_t)stream);
}

park_status park_probe_mfma_bf16(const uint16_t* A, const uint16_t* Bt, const float* C0, float* C,
                                 int32_t nprob, int32_t K, void* stream) {
  g_err[0] = 0;
  if (nprob < 0) return fail(PARK_ERR_INVALID_ARG, "nprob = %d", nprob);
  if (K < 16 || K > 4096 || K % 16)
    return fail(PARK_ERR_INVALID_ARG, "K = %d must be a multiple of 16 in [16, 4096]", K);
  if (nprob > 0) {
    PARK_TRY(check_ptr(A, "A"));
    PARK_TRY(check_ptr(Bt, "Bt"));
    PARK_TRY(check_ptr(C0, "C0"));
    PARK_TRY(check_ptr(C, "C"));
  }
  return launch_probe_mfma(A, Bt, C0, C, nprob, K, (hipStream_t)stream);
}

park_status park_check(void* ws, void* stream) {
  g_err[0] = 0;
  PARK_TRY(check_ptr(ws, "workspace"));
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = hipStreamSynchronize(st);
  if (e != hipSuccess) return fail(PARK_ERR_HIP, "stream sync: %s", hipGetErrorString(e));
  int word = 0;
  e = hipMemcpy(&word, ws, sizeof(int), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return fail(PARK_ERR_HIP, "status read: %s", hipGetErrorString(e));
  if (word == 0) return PARK_OK;
  PARK_TRY(launch_clear_status((int*)ws, st));
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return fail(PARK_ERR_HIP, "stream sync: %s", hipGetErrorString(e));
  return fail(PARK_ERR_NUMERIC, "device status 0x%x:%s%s", word,
              (word & ST_NOT_SPD) ? " metric not positive definite;" : "",
              (word & ST_NONFINITE) ? " non-finite values;" : "");
}

park_status park_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_pmu);
  g_prof = on != 0;
  return PARK_OK;
}

park_status park_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_pmu);
  for (auto& r : g_recs) {
    hipEventSynchronize(r.b);
    g_pool.push_back(r.a);
    g_pool.push_back(r.b);
  }
  g_recs.clear();
  return PARK_OK;
}

park_status park_profile_read(char* buf, size_t cap) {
  if (!buf || cap == 0) return fail(PARK_ERR_INVALID_ARG, "buffer is NULL");
  std::lock_guard<std::mutex> lk(g_pmu);
  std::map<std::string, std::pair<long, double>> agg;
  for (auto& r : g_recs) {
    hipEventSynchronize(r.b);
    float ms = 0.0f;
    hipEventElapsedTime(&ms, r.a, r.b);
    auto& a = agg[r.name];
    a.first += 1;
    a.second += ms;
    g_pool.push_back(r.a);
    g_pool.push_back(r.b);
  }
  g_recs.clear();
  std::string out = "{";
  bool first = true;
  for (auto& kv : agg) {
    char tmp[256];
    snprintf(tmp, sizeof(tmp), "%s\"%s\": {\"launches\": %ld, \"ms\": %.6f}", first ? "" : ", ",
             kv.first.c_str(), kv.second.first, kv.second.second);
    out += tmp;
    first = false;
  }
  out += "}";
  strncpy(buf, out.c_str(), cap - 1);
  buf[cap - 1] = 0;
  return PARK_OK;
}

}  // extern "C"
