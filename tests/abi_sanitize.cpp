// Host-side driver for an AddressSanitizer + UndefinedBehaviorSanitizer build of
// libpspo's host code (the device code is compiled without sanitizers): every
// argument check of the C ABI, the host validation of survival tables and the
// workspace queries at extreme sizes.  No call here reaches a kernel launch, so
// it runs without a GPU.  Exit status 0 iff every check holds; a sanitizer
// report aborts the process.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>
#include <vector>

#include "pspo.h"

static int g_fail = 0;
#define CHECK(cond)                                                           \
  do {                                                                        \
    if (!(cond)) {                                                            \
      std::fprintf(stderr, "%s:%d: CHECK failed: %s\n", __FILE__, __LINE__, #cond); \
      g_fail = 1;                                                             \
    }                                                                         \
  } while (0)

// aligned, never dereferenced on these paths
static void* fake(uintptr_t extra = 0) { return reinterpret_cast<void*>((uintptr_t(1) << 20) + extra); }

static void xi_tables() {
  // valid, increasing, out of range, NaN, empty prompts
  std::vector<double> ok = {1.0, 0.5, 0.5, 0.1, 1.0, std::ldexp(1.0, -40)};
  std::vector<int64_t> off = {0, 4, 6};
  CHECK(pspo_validate_xi_host(ok.data(), off.data(), 2) == PSPO_OK);
  std::vector<double> inc = {1.0, 0.5, 0.6};
  std::vector<int64_t> off3 = {0, 3};
  CHECK(pspo_validate_xi_host(inc.data(), off3.data(), 1) == PSPO_ERR_BAD_XI);
  CHECK(std::strstr(pspo_last_error(), "increases at t = 3") != nullptr);
  double nanv[1] = {std::nan("")};
  int64_t off1[2] = {0, 1};
  CHECK(pspo_validate_xi_host(nanv, off1, 1) == PSPO_ERR_BAD_XI);
  double big[1] = {1.25};
  CHECK(pspo_validate_xi_host(big, off1, 1) == PSPO_ERR_BAD_XI);
  int64_t bad_off[3] = {0, 2, 1};
  CHECK(pspo_validate_xi_host(ok.data(), bad_off, 2) == PSPO_ERR_INVALID_ARG);
  int64_t empty[4] = {0, 0, 0, 0};
  CHECK(pspo_validate_xi_host(nullptr, empty, 3) == PSPO_OK);
  CHECK(pspo_validate_xi_host(nullptr, nullptr, 0) == PSPO_OK);
  CHECK(pspo_validate_xi_host(nullptr, off1, 1) == PSPO_ERR_INVALID_ARG);
  CHECK(pspo_validate_xi_host(ok.data(), off.data(), -1) == PSPO_ERR_INVALID_ARG);
  // a long table, every entry visited
  std::vector<double> lng(1 << 16);
  for (size_t t = 0; t < lng.size(); ++t) lng[t] = std::exp(-1e-4 * double(t));
  int64_t offl[2] = {0, int64_t(lng.size())};
  CHECK(pspo_validate_xi_host(lng.data(), offl, 1) == PSPO_OK);
}

static void sampler_and_packer() {
  CHECK(pspo_sample_cutoffs(static_cast<double*>(fake()), static_cast<int64_t*>(fake()),
                            static_cast<int32_t*>(fake()), -1, 1, 0, 0, static_cast<int32_t*>(fake()), nullptr,
                            nullptr) == PSPO_ERR_INVALID_ARG);
  CHECK(pspo_sample_cutoffs(nullptr, nullptr, nullptr, 0, 4, 0, 0, nullptr, nullptr, nullptr) == PSPO_OK);
  CHECK(pspo_sample_cutoffs(nullptr, static_cast<int64_t*>(fake()), static_cast<int32_t*>(fake()), 1, 1, 0, 0,
                            static_cast<int32_t*>(fake()), nullptr, nullptr) == PSPO_ERR_INVALID_ARG);
  CHECK(pspo_sample_cutoffs(static_cast<double*>(fake()), static_cast<int64_t*>(fake()),
                            static_cast<int32_t*>(fake()), 1 << 16, 1 << 16, 0, 0, static_cast<int32_t*>(fake()),
                            nullptr, nullptr) == PSPO_ERR_INVALID_ARG);
  auto pack = [](int32_t P, int32_t K, int32_t cap, int32_t d, void* h) {
    return pspo_pack_prefixes(static_cast<int32_t*>(fake()), static_cast<int32_t*>(fake()),
                              static_cast<double*>(fake()), static_cast<int64_t*>(fake()), P, K, cap,
                              static_cast<int32_t*>(fake()), static_cast<float*>(fake()),
                              static_cast<uint16_t*>(fake()), d, static_cast<int32_t*>(fake()),
                              static_cast<int32_t*>(fake()), static_cast<int32_t*>(fake()),
                              static_cast<int32_t*>(fake()), static_cast<float*>(fake()),
                              static_cast<int32_t*>(fake()), static_cast<float*>(fake()),
                              static_cast<uint16_t*>(h), static_cast<int32_t*>(fake()), nullptr, nullptr);
  };
  CHECK(pack(2, 2, -1, 64, fake()) == PSPO_ERR_INVALID_ARG);
  CHECK(pack(2, 2, 16, 12, fake()) == PSPO_ERR_UNSUPPORTED);
  CHECK(pack(2, 2, 16, 64, fake(8)) == PSPO_ERR_INVALID_ARG);
  CHECK(pack(300, 300, 16, 64, fake()) == PSPO_ERR_UNSUPPORTED);
  CHECK(pack(std::numeric_limits<int32_t>::max(), 2, 16, 64, fake()) != PSPO_OK);
}

static int loss(int32_t N, int32_t d, int32_t V, uint32_t flags, float el, float eh, float scale, void* ws,
                size_t wsb) {
  return pspo_loss_fwd_bwd(static_cast<uint16_t*>(fake()), static_cast<uint16_t*>(fake()),
                           static_cast<int32_t*>(fake()), static_cast<float*>(fake()), static_cast<float*>(fake()),
                           static_cast<int32_t*>(fake()), static_cast<float*>(fake()), N, d, V, 4, el, eh, scale,
                           flags, static_cast<double*>(fake()), static_cast<float*>(fake()),
                           static_cast<float*>(fake()), nullptr, nullptr, nullptr, ws, wsb, nullptr);
}

static void loss_and_workspace() {
  const size_t ws = pspo_loss_workspace_bytes(100, 128, 1000, 0);
  CHECK(ws > 0);
  CHECK(loss(-1, 128, 1000, 0, 0.1f, 0.1f, 0.25f, fake(), ws) == PSPO_ERR_INVALID_ARG);
  CHECK(loss(100, 100, 1000, 0, 0.1f, 0.1f, 0.25f, fake(), ws) == PSPO_ERR_UNSUPPORTED);
  CHECK(loss(100, 128, 1000, 2, 0.1f, 0.1f, 0.25f, fake(), ws) == PSPO_ERR_INVALID_ARG);
  CHECK(loss(100, 128, 1000, 0, 1.0f, 0.1f, 0.25f, fake(), ws) == PSPO_ERR_INVALID_ARG);
  CHECK(loss(100, 128, 1000, 0, std::nanf(""), 0.1f, 0.25f, fake(), ws) == PSPO_ERR_INVALID_ARG);
  CHECK(loss(100, 128, 1000, 0, 0.1f, 0.1f, INFINITY, fake(), ws) == PSPO_ERR_INVALID_ARG);
  CHECK(loss(100, 128, 1000, 0, 0.1f, 0.1f, 0.25f, fake(16), ws) == PSPO_ERR_INVALID_ARG);
  CHECK(loss(100, 128, 1000, 0, 0.1f, 0.1f, 0.25f, fake(), 1024) == PSPO_ERR_WORKSPACE);
  // the workspace query at extreme sizes: no overflow, monotone in N
  const int32_t big = std::numeric_limits<int32_t>::max();
  for (uint32_t f : {0u, PSPO_KEEP_LOGITS}) {
    size_t prev = 0;
    for (int32_t n : {1, 1000, 1 << 20, 1 << 26, big}) {
      const size_t b = pspo_loss_workspace_bytes(n, 8192, 262144, f);
      CHECK(b >= prev);
      prev = b;
    }
    CHECK(pspo_loss_workspace_bytes(big, 8, big, f) > 0);
    CHECK(pspo_loss_workspace_bytes(-1, 8, 100, f) == 0);
  }
  CHECK(loss(big, 8192, 262144, 0, 0.1f, 0.1f, 0.25f, fake(), std::numeric_limits<size_t>::max()) != PSPO_OK);
  CHECK(pspo_score_proxy_workspace_bytes(big, 8192, big) > 0);
  CHECK(pspo_design_workspace_bytes(std::numeric_limits<int64_t>::max() / 64) > 0);
  CHECK(pspo_design_workspace_bytes(-1) == 0);
}

static void proxy_and_design() {
  const size_t ws = pspo_score_proxy_workspace_bytes(100, 128, 1000);
  auto prox = [&](int32_t N, int32_t d, void* w, size_t wsb) {
    return pspo_score_proxy(static_cast<uint16_t*>(fake()), static_cast<uint16_t*>(fake()),
                            static_cast<int32_t*>(fake()), N, d, 1000, static_cast<float*>(fake()), nullptr, nullptr,
                            nullptr, w, wsb, nullptr);
  };
  CHECK(prox(-1, 128, fake(), ws) == PSPO_ERR_INVALID_ARG);
  CHECK(prox(100, 100, fake(), ws) == PSPO_ERR_UNSUPPORTED);
  CHECK(prox(100, 128, nullptr, ws) == PSPO_ERR_INVALID_ARG);
  CHECK(prox(100, 128, fake(), 64) == PSPO_ERR_WORKSPACE);
  CHECK(pspo_design_weights(static_cast<float*>(fake()), static_cast<int32_t*>(fake()), static_cast<float*>(fake()),
                            16, static_cast<int32_t*>(fake()), static_cast<int32_t*>(fake()),
                            static_cast<float*>(fake()), static_cast<int64_t*>(fake()), 2, 65, 100,
                            static_cast<double*>(fake()), nullptr, nullptr, nullptr,
                            nullptr) == PSPO_ERR_UNSUPPORTED);
  CHECK(pspo_design_cutoffs(static_cast<double*>(fake()), static_cast<int64_t*>(fake()), 2, 100, std::nan(""), 0,
                            0.0, static_cast<double*>(fake()), fake(), pspo_design_workspace_bytes(100), nullptr,
                            nullptr) == PSPO_ERR_INVALID_ARG);
  CHECK(pspo_design_cutoffs(static_cast<double*>(fake()), static_cast<int64_t*>(fake()), 2, 100, 8.0, 7, 0.0,
                            static_cast<double*>(fake()), fake(), pspo_design_workspace_bytes(100), nullptr,
                            nullptr) == PSPO_ERR_INVALID_ARG);
  CHECK(pspo_mfma_loop(0, 4, static_cast<float*>(fake()), nullptr) == PSPO_ERR_INVALID_ARG);
  CHECK(std::strcmp(pspo_status_string(99), "PSPO_ERR_UNKNOWN") == 0);
}

int main() {
  xi_tables();
  sampler_and_packer();
  loss_and_workspace();
  proxy_and_design();
  std::printf(g_fail ? "abi_sanitize: FAILED\n" : "abi_sanitize: ok\n");
  return g_fail;
}
