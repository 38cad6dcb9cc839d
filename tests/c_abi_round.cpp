// The C ABI used directly from C++, without Python or PyTorch: device
// buffers from hipMalloc, one outer round over two units through
// edit_outer_step_round, the decision read back with edit_outer_state_get,
// and the argument checks of the boundary; then the same round as K
// sync-group workers (edit_group_*), the collectives done by hand.  Run by
// tests/test_gpu_c_abi.py; built by __graft_entry__.build().
//
// The inputs make the expected result a closed form.  theta is a multiple of
// 1/64 and worker j's replica is theta + (j + 1)/256 exactly (both exact in
// bf16), so Delta_j = c_j = (j + 1)/256 everywhere and G_j = c_j sqrt(n).
// Round 0 is inside the EMA warm-up, so no worker is flagged; the weights are
// the softmax of -G (Eq. 2), Gbar = |sum_j w_j c_j| sqrt(n), beta = 1 (Eq. 4
// with phi = 10), and with zero momentum the Nesterov step gives
// theta' = theta + nu (1 + rho) sum_j w_j c_j.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "edit_outer.h"

#define CHECK(cond, ...)                                   \
  do {                                                     \
    if (!(cond)) {                                         \
      std::printf("FAIL (line %d): ", __LINE__);           \
      std::printf(__VA_ARGS__);                            \
      std::printf("\n");                                   \
      return 1;                                            \
    }                                                      \
  } while (0)

static float from_bf16(uint16_t h) {
  const uint32_t u = static_cast<uint32_t>(h) << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

// Exact for the multiples of 1/256 used here (they need at most 8 bits).
static uint16_t to_bf16_exact(float x) {
  uint32_t u;
  std::memcpy(&u, &x, 4);
  return static_cast<uint16_t>(u >> 16);
}

int main() {
  const int K = 4;
  const int64_t numel[2] = {10007, 3};
  const double nu = 0.8, rho = 0.85;
  edit_outer_config_t cfg = {K, 2, numel, EDIT_BF16, EDIT_AE | EDIT_WA | EDIT_GC, nu, rho,
                             10.0, 1e-6, 0.02, 3.0, 10};
  edit_outer_t h = nullptr;
  CHECK(edit_outer_init(&cfg, &h) == EDIT_OK, "init: %s", edit_outer_last_error());

  float* theta[2];
  float* mom[2];
  void* reps[2 * K];
  std::vector<std::vector<float>> theta_h(2);
  for (int u = 0; u < 2; ++u) {
    const int64_t n = numel[u];
    theta_h[u].resize(n);
    for (int64_t i = 0; i < n; ++i) theta_h[u][i] = static_cast<float>(i % 41 - 20) / 64.0f;
    CHECK(hipMalloc(&theta[u], 4 * n) == hipSuccess, "hipMalloc");
    CHECK(hipMalloc(&mom[u], 4 * n) == hipSuccess, "hipMalloc");
    CHECK(hipMemcpy(theta[u], theta_h[u].data(), 4 * n, hipMemcpyHostToDevice) == hipSuccess, "copy");
    CHECK(hipMemset(mom[u], 0, 4 * n) == hipSuccess, "memset");
    for (int j = 0; j < K; ++j) {
      std::vector<uint16_t> r(n);
      for (int64_t i = 0; i < n; ++i) r[i] = to_bf16_exact(theta_h[u][i] + (j + 1) / 256.0f);
      CHECK(hipMalloc(&reps[u * K + j], 2 * n) == hipSuccess, "hipMalloc");
      CHECK(hipMemcpy(reps[u * K + j], r.data(), 2 * n, hipMemcpyHostToDevice) == hipSuccess, "copy");
    }
  }

  // one round, both units, on the default stream
  const int32_t layers[2] = {0, 1};
  CHECK(edit_outer_step_round(h, 2, layers, theta, mom, reps, nullptr) == EDIT_OK, "round: %s",
        edit_outer_last_error());
  CHECK(hipDeviceSynchronize() == hipSuccess, "sync");

  for (int u = 0; u < 2; ++u) {
    const int64_t n = numel[u];
    edit_layer_state_t st;
    CHECK(edit_outer_state_get(h, u, &st) == EDIT_OK, "state_get: %s", edit_outer_last_error());
    CHECK(st.round == 1 && !st.rolled_back && !st.z_tested, "unit %d: round %lld", u, (long long)st.round);
    // expected decision
    double G[K], w[K], sum_e = 0.0, dbar = 0.0;
    for (int j = 0; j < K; ++j) G[j] = (j + 1) / 256.0 * std::sqrt(static_cast<double>(n));
    for (int j = 0; j < K; ++j) sum_e += std::exp(-(G[j] - G[0]));
    for (int j = 0; j < K; ++j) {
      w[j] = std::exp(-(G[j] - G[0])) / sum_e;
      dbar += w[j] * (j + 1) / 256.0;
    }
    for (int j = 0; j < K; ++j) {
      CHECK(!st.anomalous[j], "unit %d worker %d flagged", u, j);
      CHECK(std::fabs(st.norm[j] - G[j]) <= 1e-12 * G[j], "unit %d G_%d %.17g vs %.17g", u, j,
            st.norm[j], G[j]);
      CHECK(std::fabs(st.weight[j] - w[j]) <= 1e-12, "unit %d w_%d %.17g vs %.17g", u, j, st.weight[j], w[j]);
      CHECK(std::fabs(st.ema_mean[j] - 0.02 * G[j]) <= 1e-12 * G[j], "unit %d mu_%d", u, j);
    }
    const double gbar = dbar * std::sqrt(static_cast<double>(n));
    CHECK(std::fabs(st.synced_norm - gbar) <= 1e-9 * gbar, "unit %d Gbar %.17g vs %.17g", u, st.synced_norm, gbar);
    CHECK(st.clip_coef == 1.0, "unit %d beta %g", u, st.clip_coef);
    // theta' and the replicas
    std::vector<float> th(n), b(n);
    CHECK(hipMemcpy(th.data(), theta[u], 4 * n, hipMemcpyDeviceToHost) == hipSuccess, "copy back");
    CHECK(hipMemcpy(b.data(), mom[u], 4 * n, hipMemcpyDeviceToHost) == hipSuccess, "copy back");
    for (int64_t i = 0; i < n; ++i) {
      const double expect = theta_h[u][i] + nu * (1.0 + rho) * dbar;
      CHECK(std::fabs(th[i] - expect) <= 1e-6 * (std::fabs(expect) + 1e-3), "unit %d theta[%lld] %.9g vs %.9g",
            u, (long long)i, th[i], expect);
      CHECK(std::fabs(b[i] + dbar) <= 1e-6 * dbar, "unit %d b[%lld]", u, (long long)i);
    }
    for (int j = 0; j < K; ++j) {
      std::vector<uint16_t> r(n);
      CHECK(hipMemcpy(r.data(), reps[u * K + j], 2 * n, hipMemcpyDeviceToHost) == hipSuccess, "copy back");
      for (int64_t i = 0; i < n; ++i) {
        const float back = from_bf16(r[i]);
        // the cast of theta' to bf16: within half a bf16 step
        CHECK(std::fabs(back - th[i]) <= std::ldexp(std::fabs(th[i]), -8) + 1e-30, "unit %d replica %d [%lld]", u,
              j, (long long)i);
      }
    }
  }

  // the boundary's argument checks
  CHECK(edit_outer_step_round(h, 0, layers, theta, mom, reps, nullptr) == EDIT_EINVAL, "count 0 accepted");
  float* misaligned[2] = {theta[0] + 1, theta[1]};
  CHECK(edit_outer_step_round(h, 2, layers, misaligned, mom, reps, nullptr) == EDIT_EINVAL, "misaligned accepted");
  CHECK(std::strstr(edit_outer_last_error(), "aligned") != nullptr, "message: %s", edit_outer_last_error());
  void* aliased[2 * K];
  for (int k = 0; k < 2 * K; ++k) aliased[k] = reps[k];
  aliased[1] = reps[0];
  CHECK(edit_outer_step_round(h, 2, layers, theta, mom, aliased, nullptr) == EDIT_EINVAL, "aliasing accepted");
  const int32_t twice[2] = {0, 0};
  CHECK(edit_outer_step_round(h, 2, twice, theta, mom, reps, nullptr) == EDIT_EINVAL, "repeated unit accepted");
  edit_layer_state_t st;
  CHECK(edit_outer_state_get(h, 2, &st) == EDIT_EINVAL, "bad layer accepted");

  edit_outer_destroy(h);
  for (int u = 0; u < 2; ++u) {
    (void)hipFree(theta[u]);
    (void)hipFree(mom[u]);
  }
  for (int k = 0; k < 2 * K; ++k) (void)hipFree(reps[k]);

  // The same round as K sync-group workers (one replica each), the two
  // collectives done by hand: the all-gather by copying the K pairs into
  // one array, the all-reduce by forming sum_j w_j delta_j on the host.
  {
    const int64_t n = numel[0];
    edit_outer_config_t gcfg = cfg;
    gcfg.num_layers = 1;
    edit_group_t g[K];
    float *gth[K], *gmo[K], *gdelta[K], *dbar;
    void* grep[K];
    double *pair[K], *gathered, *wout[K];
    for (int r = 0; r < K; ++r) {
      CHECK(edit_group_init(&gcfg, r, &g[r]) == EDIT_OK, "group init: %s", edit_outer_last_error());
      CHECK(hipMalloc(&gth[r], 4 * n) == hipSuccess && hipMalloc(&gmo[r], 4 * n) == hipSuccess &&
                hipMalloc(&gdelta[r], 4 * n) == hipSuccess && hipMalloc(&grep[r], 2 * n) == hipSuccess &&
                hipMalloc(&pair[r], 16) == hipSuccess && hipMalloc(&wout[r], 8) == hipSuccess,
            "hipMalloc");
      CHECK(hipMemcpy(gth[r], theta_h[0].data(), 4 * n, hipMemcpyHostToDevice) == hipSuccess, "copy");
      CHECK(hipMemset(gmo[r], 0, 4 * n) == hipSuccess, "memset");
      std::vector<uint16_t> rr(n);
      for (int64_t i = 0; i < n; ++i) rr[i] = to_bf16_exact(theta_h[0][i] + (r + 1) / 256.0f);
      CHECK(hipMemcpy(grep[r], rr.data(), 2 * n, hipMemcpyHostToDevice) == hipSuccess, "copy");
    }
    CHECK(hipMalloc(&gathered, 16 * K) == hipSuccess && hipMalloc(&dbar, 4 * n) == hipSuccess, "hipMalloc");
    for (int r = 0; r < K; ++r)
      CHECK(edit_group_norm(g[r], 0, gth[r], grep[r], gdelta[r], pair[r], nullptr) == EDIT_OK, "norm: %s",
            edit_outer_last_error());
    for (int r = 0; r < K; ++r)  // the all-gather
      CHECK(hipMemcpy(gathered + 2 * r, pair[r], 16, hipMemcpyDeviceToDevice) == hipSuccess, "gather");
    for (int r = 0; r < K; ++r)
      CHECK(edit_group_weights(g[r], 0, gathered, wout[r], gdelta[r], nullptr) == EDIT_OK, "weights: %s",
            edit_outer_last_error());
    // the all-reduce: dbar = sum_r w_r delta_r, on the host in fp32
    std::vector<float> acc(n, 0.f), d(n);
    double w[K], G[K], sum_e = 0.0, cbar = 0.0;
    for (int r = 0; r < K; ++r) {
      CHECK(hipMemcpy(&w[r], wout[r], 8, hipMemcpyDeviceToHost) == hipSuccess, "copy back");
      CHECK(hipMemcpy(d.data(), gdelta[r], 4 * n, hipMemcpyDeviceToHost) == hipSuccess, "copy back");
      for (int64_t i = 0; i < n; ++i) acc[i] += static_cast<float>(w[r]) * d[i];
      G[r] = (r + 1) / 256.0 * std::sqrt(static_cast<double>(n));
      sum_e += std::exp(-(G[r] - G[0]));
    }
    for (int r = 0; r < K; ++r) {
      const double expect_w = std::exp(-(G[r] - G[0])) / sum_e;
      CHECK(std::fabs(w[r] - expect_w) <= 1e-12, "group w_%d %.17g vs %.17g", r, w[r], expect_w);
      cbar += expect_w * (r + 1) / 256.0;
    }
    CHECK(hipMemcpy(dbar, acc.data(), 4 * n, hipMemcpyHostToDevice) == hipSuccess, "copy");
    for (int r = 0; r < K; ++r)
      CHECK(edit_group_apply(g[r], 0, dbar, gth[r], gmo[r], grep[r], nullptr) == EDIT_OK, "apply: %s",
            edit_outer_last_error());
    CHECK(hipDeviceSynchronize() == hipSuccess, "sync");
    for (int r = 0; r < K; ++r) {
      edit_layer_state_t st;
      CHECK(edit_group_state_get(g[r], 0, &st) == EDIT_OK, "group state_get: %s", edit_outer_last_error());
      CHECK(st.round == 1 && !st.rolled_back && st.clip_coef == 1.0, "rank %d: round/rollback/beta", r);
      CHECK(std::fabs(st.norm[r] - G[r]) <= 1e-12 * G[r], "rank %d: G", r);
      CHECK(std::fabs(st.ema_mean[r] - 0.02 * G[r]) <= 1e-12 * G[r], "rank %d: mu", r);
      const double gbar = cbar * std::sqrt(static_cast<double>(n));
      CHECK(std::fabs(st.synced_norm - gbar) <= 1e-6 * gbar, "rank %d: Gbar %.9g vs %.9g", r, st.synced_norm, gbar);
      std::vector<float> th(n), b(n);
      CHECK(hipMemcpy(th.data(), gth[r], 4 * n, hipMemcpyDeviceToHost) == hipSuccess, "copy back");
      CHECK(hipMemcpy(b.data(), gmo[r], 4 * n, hipMemcpyDeviceToHost) == hipSuccess, "copy back");
      for (int64_t i = 0; i < n; ++i) {
        const double expect = theta_h[0][i] + nu * (1.0 + rho) * cbar;
        CHECK(std::fabs(th[i] - expect) <= 1e-6 * (std::fabs(expect) + 1e-3), "rank %d theta[%lld]", r,
              (long long)i);
        CHECK(std::fabs(b[i] + cbar) <= 1e-6 * cbar, "rank %d b[%lld]", r, (long long)i);
      }
    }
    // argument checks of the group entry points
    edit_group_t bad = nullptr;
    CHECK(edit_group_init(&gcfg, K, &bad) == EDIT_EINVAL, "rank K accepted");
    CHECK(edit_group_norm(g[0], 1, gth[0], grep[0], gdelta[0], pair[0], nullptr) == EDIT_EINVAL, "bad layer accepted");
    CHECK(edit_group_norm(g[0], 0, gth[0], grep[0], gth[0], pair[0], nullptr) == EDIT_EINVAL, "aliasing accepted");
    CHECK(edit_group_apply(g[0], 0, gth[0], gth[0], gmo[0], grep[0], nullptr) == EDIT_EINVAL, "dbar aliasing accepted");
    for (int r = 0; r < K; ++r) {
      edit_group_destroy(g[r]);
      (void)hipFree(gth[r]);
      (void)hipFree(gmo[r]);
      (void)hipFree(gdelta[r]);
      (void)hipFree(grep[r]);
      (void)hipFree(pair[r]);
      (void)hipFree(wout[r]);
    }
    (void)hipFree(gathered);
    (void)hipFree(dbar);
  }
  std::printf("ok\n");
  return 0;
}
