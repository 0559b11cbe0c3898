// Host-side checks of the C ABI, built with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code only (see test_host_sanitizers.py).
// Every call here returns before anything is enqueued: size queries, the
// schedule helper, status strings and argument validation of each entry
// point.  No GPU is touched; the fake device addresses are never dereferenced.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "park.h"

extern "C" int host_check_status_strings(void);  // host_checks_c.c

static int failures = 0;

#define EXPECT(cond)                                                   \
  do {                                                                 \
    if (!(cond)) {                                                     \
      std::fprintf(stderr, "%s:%d: failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                      \
    }                                                                  \
  } while (0)

static void* const FAKE = (void*)(uintptr_t)(1u << 20);  // 256-byte aligned, never read

static park_params params(int CQ, int CK) {
  park_params p;
  std::memset(&p, 0, sizeof p);
  p.CQ = CQ;
  p.CK = CK;
  p.T = 10;
  p.select = PARK_SELECT_TOPK;
  p.topk_ratio = 0.1;
  p.topp = 0.9;
  p.alpha = 0.05;
  p.eps = 1e-6;
  p.s_min = 1e-12;
  p.seed = 1;
  p.key_metric = PARK_METRIC_QRKC;
  p.out_dtype = PARK_F32;
  p.estimator = PARK_EST_PAMA;
  p.block_mode = PARK_BLOCKS_CLUSTER;
  p.init = PARK_INIT_SEEDED;
  return p;
}

static void sizes() {
  // size queries over a grid of shapes up to the largest layers (and past the
  // 32-bit range of H*N*d), each monotone in the block counts
  const int Hs[] = {1, 3, 24, 40, 96};
  const int Ns[] = {1, 63, 1000, 75600, 119056, 1 << 20};
  const int ds[] = {64, 128};
  const int dts[] = {PARK_F32, PARK_BF16};
  for (int H : Hs)
    for (int N : Ns)
      for (int d : ds)
        for (int dt : dts) {
          park_dims dims = {H, N, d, dt};
          size_t prev = 0;
          for (int C : {1, 16, 64, 256, 1182, 1861, 2048}) {
            if (C > N) continue;
            size_t ws = 0;
            EXPECT(park_workspace_size(&dims, C, C, &ws) == PARK_OK);
            EXPECT(ws >= prev);
            prev = ws;
            std::vector<size_t> b(PARK_STATE_NBUF, 0);
            EXPECT(park_state_sizes(&dims, C, C, b.data(), PARK_STATE_NBUF) == PARK_OK);
            EXPECT(b[0] == (size_t)H * N * 4);
            EXPECT(b[7] == (size_t)H * C * C * 4);
            EXPECT(b[8] == (size_t)H * N * d * (dt == PARK_F32 ? 4 : 2));
          }
        }
  park_dims dims = {2, 1000, 128, PARK_BF16};
  size_t ws = 0;
  EXPECT(park_workspace_size(&dims, 0, 16, &ws) == PARK_ERR_INVALID_ARG);
  EXPECT(park_workspace_size(&dims, 1001, 16, &ws) == PARK_ERR_INVALID_ARG);
  EXPECT(park_workspace_size(nullptr, 16, 16, &ws) == PARK_ERR_INVALID_ARG);
  EXPECT(park_workspace_size(&dims, 16, 16, nullptr) == PARK_ERR_INVALID_ARG);
  park_dims bad = {2, 1000, 96, PARK_BF16};
  EXPECT(park_workspace_size(&bad, 16, 16, &ws) == PARK_ERR_UNSUPPORTED);
  bad = {-1, 1000, 128, PARK_BF16};
  EXPECT(park_workspace_size(&bad, 16, 16, &ws) == PARK_ERR_INVALID_ARG);
  bad = {2, 1000, 128, 7};
  EXPECT(park_workspace_size(&bad, 16, 16, &ws) == PARK_ERR_INVALID_ARG);
  EXPECT(std::strstr(park_last_error(), "dtype") != nullptr);
  size_t b[PARK_STATE_NBUF];
  EXPECT(park_state_sizes(&dims, 16, 16, b, PARK_STATE_NBUF - 1) == PARK_ERR_INVALID_ARG);
  EXPECT(park_state_sizes(&dims, 16, 16, nullptr, PARK_STATE_NBUF) == PARK_ERR_INVALID_ARG);
}

static void strings_and_schedule() {
  EXPECT(host_check_status_strings() == 0);
  EXPECT(std::strcmp(park_status_string(PARK_ERR_WORKSPACE), "workspace too small") == 0);
  const int32_t sched[] = {10, 20, 30};
  for (int t = 0; t < 50; ++t) {
    int32_t r = -7;
    EXPECT(park_schedule_step(t, sched, 3, &r) == PARK_OK);
    if (t < 10) EXPECT(r == PARK_STEP_DENSE);
    else if (t == 10 || t == 20 || t == 30) EXPECT(r == PARK_RECOMPUTE);
    else EXPECT(r == PARK_REUSE_CLUSTERS_AND_MASK);
  }
  int32_t r;
  const int32_t unsorted[] = {5, 2};
  EXPECT(park_schedule_step(4, unsorted, 2, &r) == PARK_ERR_INVALID_ARG);
  EXPECT(park_schedule_step(-1, sched, 3, &r) == PARK_ERR_INVALID_ARG);
  EXPECT(park_schedule_step(1, sched, 0, &r) == PARK_ERR_INVALID_ARG);
  EXPECT(park_schedule_step(1, nullptr, 3, &r) == PARK_ERR_INVALID_ARG);
  EXPECT(park_schedule_step(1, sched, 3, nullptr) == PARK_ERR_INVALID_ARG);
  EXPECT(park_profile_enable(1) == PARK_OK);
  EXPECT(park_profile_reset() == PARK_OK);
  char buf[64];
  EXPECT(park_profile_read(buf, sizeof buf) == PARK_OK);
  EXPECT(park_profile_enable(0) == PARK_OK);
}

static void argument_errors() {
  park_dims d = {2, 1000, 128, PARK_BF16};
  const size_t big = (size_t)1 << 40;
  auto cluster = [&](const void* X, const void* Q, int C, int T, int side, int metric,
                     double alpha, double s_min, size_t wsb, park_dims* dd) {
    return park_cluster_keys(X, Q, dd ? dd : &d, C, T, 1, side, metric, alpha, 1e-6, s_min,
                             (int32_t*)FAKE, (int32_t*)FAKE, (int32_t*)FAKE, nullptr, nullptr,
                             FAKE, wsb, nullptr);
  };
  EXPECT(cluster(nullptr, FAKE, 16, 10, 1, PARK_METRIC_QRKC, 0.05, 1e-12, big, nullptr) ==
         PARK_ERR_INVALID_ARG);
  EXPECT(cluster((char*)FAKE + 4, FAKE, 16, 10, 1, PARK_METRIC_QRKC, 0.05, 1e-12, big,
                 nullptr) == PARK_ERR_INVALID_ARG);
  EXPECT(cluster(FAKE, nullptr, 16, 10, 1, PARK_METRIC_QRKC, 0.05, 1e-12, big, nullptr) ==
         PARK_ERR_INVALID_ARG);
  EXPECT(cluster(FAKE, FAKE, 0, 10, 1, PARK_METRIC_QRKC, 0.05, 1e-12, big, nullptr) ==
         PARK_ERR_INVALID_ARG);
  EXPECT(cluster(FAKE, FAKE, 16, 0, 1, PARK_METRIC_QRKC, 0.05, 1e-12, big, nullptr) ==
         PARK_ERR_INVALID_ARG);
  EXPECT(cluster(FAKE, FAKE, 16, 10, 2, PARK_METRIC_QRKC, 0.05, 1e-12, big, nullptr) ==
         PARK_ERR_INVALID_ARG);
  EXPECT(cluster(FAKE, FAKE, 16, 10, 1, PARK_METRIC_QRKC, NAN, 1e-12, big, nullptr) ==
         PARK_ERR_INVALID_ARG);
  EXPECT(cluster(FAKE, FAKE, 16, 10, 1, PARK_METRIC_QRKC, 0.05, 0.0, big, nullptr) ==
         PARK_ERR_INVALID_ARG);
  EXPECT(cluster(FAKE, FAKE, 16, 10, 1, PARK_METRIC_QRKC, 0.05, 1e-12, 100, nullptr) ==
         PARK_ERR_WORKSPACE);
  park_dims d32 = {2, 1000, 32, PARK_BF16};
  EXPECT(cluster(FAKE, FAKE, 16, 10, 1, PARK_METRIC_QRKC, 0.05, 1e-12, big, &d32) ==
         PARK_ERR_UNSUPPORTED);

  EXPECT(park_retrieve_blocks(FAKE, (int32_t*)FAKE, (float*)FAKE, (int32_t*)FAKE, &d, 16, 16,
                              PARK_SELECT_TOPP, 1.5, nullptr, (int32_t*)FAKE, (int32_t*)FAKE,
                              FAKE, big, nullptr) == PARK_ERR_INVALID_ARG);
  EXPECT(park_retrieve_blocks(FAKE, (int32_t*)FAKE, (float*)FAKE, (int32_t*)FAKE, &d, 16, 3000,
                              PARK_SELECT_TOPP, 0.9, nullptr, (int32_t*)FAKE, (int32_t*)FAKE,
                              FAKE, big, nullptr) == PARK_ERR_INVALID_ARG);
  EXPECT(park_retrieve_blocks(FAKE, (int32_t*)FAKE, (float*)FAKE, (int32_t*)FAKE, &d, 16, 16,
                              PARK_SELECT_TOPP, 0.9, nullptr, (int32_t*)FAKE, (int32_t*)FAKE,
                              FAKE, 8, nullptr) == PARK_ERR_WORKSPACE);

  auto attn = [&](const void* V, int odt, float* lse, size_t wsb) {
    return park_block_sparse_attn(FAKE, FAKE, V, (int32_t*)FAKE, (int32_t*)FAKE, (int32_t*)FAKE,
                                  (int32_t*)FAKE, (int32_t*)FAKE, &d, 16, 16, FAKE, odt, lse,
                                  FAKE, wsb, nullptr);
  };
  EXPECT(attn(FAKE, 7, nullptr, big) == PARK_ERR_INVALID_ARG);
  EXPECT(attn(nullptr, PARK_F32, nullptr, big) == PARK_ERR_INVALID_ARG);
  EXPECT(attn(FAKE, PARK_F32, (float*)((char*)FAKE + 4), big) == PARK_ERR_INVALID_ARG);
  EXPECT(attn(FAKE, PARK_F32, nullptr, 8) == PARK_ERR_WORKSPACE);
  EXPECT(park_block_sparse_attn_static(FAKE, FAKE, nullptr, (int32_t*)FAKE, (int32_t*)FAKE,
                                       (int32_t*)FAKE, (int32_t*)FAKE, (int32_t*)FAKE, &d, 16, 16,
                                       FAKE, PARK_F32, nullptr, nullptr) == PARK_ERR_INVALID_ARG);

  park_state st;
  std::memset(&st, 0, sizeof st);
  int32_t** ip[] = {&st.q_perm, &st.k_perm, &st.q_offsets, &st.k_offsets};
  for (auto p : ip) *p = (int32_t*)FAKE;
  st.k_centroids = (float*)FAKE;
  st.k_sizes = (int32_t*)FAKE;
  st.kv_count = (int32_t*)FAKE;
  st.kv_index = (int32_t*)FAKE;
  st.Qp = FAKE;
  st.Kp = FAKE;
  st.Vp = FAKE;
  park_params p = params(16, 16);
  EXPECT(park_forward(FAKE, FAKE, FAKE, &d, &p, 3, &st, FAKE, FAKE, big, nullptr) ==
         PARK_ERR_INVALID_ARG);
  EXPECT(park_forward(FAKE, FAKE, FAKE, &d, nullptr, 0, &st, FAKE, FAKE, big, nullptr) ==
         PARK_ERR_INVALID_ARG);
  EXPECT(park_forward(FAKE, FAKE, FAKE, &d, &p, 0, &st, FAKE, FAKE, 64, nullptr) ==
         PARK_ERR_WORKSPACE);
  park_params q = p;
  q.topk_ratio = 0.0;
  EXPECT(park_forward(FAKE, FAKE, FAKE, &d, &q, 0, &st, FAKE, FAKE, big, nullptr) ==
         PARK_ERR_INVALID_ARG);
  q = p;
  q.init = PARK_INIT_WARM;  // needs q_mu and k_mu
  EXPECT(park_forward(FAKE, FAKE, FAKE, &d, &q, 0, &st, FAKE, FAKE, big, nullptr) ==
         PARK_ERR_INVALID_ARG);
  EXPECT(std::strstr(park_last_error(), "q_mu") != nullptr);
  park_state s2 = st;
  s2.Vp = nullptr;
  EXPECT(park_forward(FAKE, FAKE, FAKE, &d, &p, 0, &s2, FAKE, FAKE, big, nullptr) ==
         PARK_ERR_INVALID_ARG);

  EXPECT(park_probe_exp2((float*)FAKE, (float*)FAKE, -1, nullptr) == PARK_ERR_INVALID_ARG);
  EXPECT(park_probe_exp2(nullptr, nullptr, 0, nullptr) == PARK_OK);
  for (int K : {0, 8, 24, 4112})
    EXPECT(park_probe_mfma_bf16((uint16_t*)FAKE, (uint16_t*)FAKE, (float*)FAKE, (float*)FAKE, 1, K,
                                nullptr) == PARK_ERR_INVALID_ARG);
}

int main() {
  sizes();
  strings_and_schedule();
  argument_errors();
  if (failures) {
    std::fprintf(stderr, "%d host check(s) failed\n", failures);
    return 1;
  }
  std::printf("host checks passed\n");
  return 0;
}
