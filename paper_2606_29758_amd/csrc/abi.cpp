// Status strings, thread-local error detail, device check, the check after
// every launch (with the PSPO_DEBUG mode), the per-product timing of the
// measurement mode and host-side validation of survival tables.
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

namespace pspo {

static thread_local std::string g_last_error;

void set_last_error(const std::string& msg) { g_last_error = msg; }
void clear_last_error() { g_last_error.clear(); }

int require_gfx950() {
  int dev = 0;
  PSPO_HIP_CHECK(hipGetDevice(&dev));
  // Architecture of each device, looked up once per device id.
  static std::once_flag once[64];
  static bool is_gfx950[64];
  if (dev < 0 || dev >= 64) return fail(PSPO_ERR_UNSUPPORTED, "device id out of range");
  hipError_t err = hipSuccess;
  std::call_once(once[dev], [&] {
    hipDeviceProp_t prop;
    err = hipGetDeviceProperties(&prop, dev);
    is_gfx950[dev] = (err == hipSuccess) && std::string(prop.gcnArchName).rfind("gfx950", 0) == 0;
  });
  if (err != hipSuccess) return fail(PSPO_ERR_HIP, std::string("hipGetDeviceProperties: ") + hipGetErrorString(err));
  if (!is_gfx950[dev]) return fail(PSPO_ERR_UNSUPPORTED, "libpspo kernels are built for gfx950 (MI355X) only");
  return PSPO_OK;
}

bool debug_mode() {
  const char* v = std::getenv("PSPO_DEBUG");
  return v != nullptr && v[0] != '\0' && std::strcmp(v, "0") != 0;
}

int after_launch(const char* kernel, hipStream_t stream) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(PSPO_ERR_HIP, std::string(kernel) + " (launch): " + hipGetErrorString(e));
  if (debug_mode()) {
    e = hipStreamSynchronize(stream);
    if (e == hipSuccess) e = hipGetLastError();
    if (e != hipSuccess) return fail(PSPO_ERR_HIP, std::string(kernel) + " (PSPO_DEBUG): " + hipGetErrorString(e));
  }
  return PSPO_OK;
}

// ---- per-product timing ------------------------------------------------------
namespace {
struct TimingState {
  bool on = false;
  int max = 0, used = 0;
  std::vector<hipEvent_t> ev;   // [max][2]: start, end of each record
  std::vector<int8_t> kind;     // [max]
  std::vector<int8_t> done;     // [max]: the end event was recorded
};
thread_local TimingState t_timing;

void destroy_events(TimingState& t) {
  for (hipEvent_t e : t.ev)
    if (e != nullptr) (void)hipEventDestroy(e);
  t.ev.clear();
  t.kind.clear();
  t.done.clear();
  t.on = false;
  t.max = t.used = 0;
}
}  // namespace

int ProductTimer::begin(int kind) {
  TimingState& t = t_timing;
  rec_ = -1;
  if (!t.on || t.used >= t.max) return PSPO_OK;
  const int r = t.used;
  PSPO_HIP_CHECK(hipEventRecord(t.ev[2 * r], stream_));
  t.kind[r] = static_cast<int8_t>(kind);
  t.done[r] = 0;
  t.used = r + 1;
  rec_ = r;
  return PSPO_OK;
}

int ProductTimer::end() {
  if (rec_ < 0) return PSPO_OK;
  TimingState& t = t_timing;
  const int r = rec_;
  rec_ = -1;
  PSPO_HIP_CHECK(hipEventRecord(t.ev[2 * r + 1], stream_));
  t.done[r] = 1;
  return PSPO_OK;
}

}  // namespace pspo

extern "C" {

int pspo_timing_start(int32_t max_records) {
  using namespace pspo;
  clear_last_error();
  TimingState& t = t_timing;
  PSPO_REQUIRE(!t.on, PSPO_ERR_INVALID_ARG, "timing is already started on this thread");
  PSPO_REQUIRE(max_records >= 1 && max_records <= (1 << 20), PSPO_ERR_INVALID_ARG,
               "max_records must lie in [1, 2^20]");
  t.ev.assign(2 * (size_t)max_records, nullptr);
  for (hipEvent_t& e : t.ev) {
    const hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) {
      e = nullptr;
      destroy_events(t);
      return fail(PSPO_ERR_HIP, std::string("hipEventCreate: ") + hipGetErrorString(err));
    }
  }
  t.kind.assign(max_records, 0);
  t.done.assign(max_records, 0);
  t.max = max_records;
  t.used = 0;
  t.on = true;
  return PSPO_OK;
}

int pspo_timing_stop(double* ms, int32_t* count) {
  using namespace pspo;
  clear_last_error();
  TimingState& t = t_timing;
  PSPO_REQUIRE(t.on, PSPO_ERR_INVALID_ARG, "timing is not started on this thread");
  if (ms == nullptr || count == nullptr) {
    destroy_events(t);
    return fail(PSPO_ERR_INVALID_ARG, "ms and count must not be NULL");
  }
  for (int k = 0; k < PSPO_TIMED_KINDS; ++k) {
    ms[k] = 0.0;
    count[k] = 0;
  }
  hipError_t first = hipSuccess;
  for (int r = 0; r < t.used; ++r) {
    if (!t.done[r]) continue;   // a call that failed between the two records
    hipError_t e = hipEventSynchronize(t.ev[2 * r + 1]);
    float x = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&x, t.ev[2 * r], t.ev[2 * r + 1]);
    if (e != hipSuccess) {
      if (first == hipSuccess) first = e;
      continue;
    }
    ms[t.kind[r]] += x;
    count[t.kind[r]] += 1;
  }
  destroy_events(t);
  if (first != hipSuccess) return fail(PSPO_ERR_HIP, std::string("timing events: ") + hipGetErrorString(first));
  return PSPO_OK;
}

const char* pspo_status_string(int status) {
  switch (status) {
    case PSPO_OK: return "PSPO_OK";
    case PSPO_ERR_INVALID_ARG: return "PSPO_ERR_INVALID_ARG";
    case PSPO_ERR_BAD_XI: return "PSPO_ERR_BAD_XI";
    case PSPO_ERR_WORKSPACE: return "PSPO_ERR_WORKSPACE";
    case PSPO_ERR_UNSUPPORTED: return "PSPO_ERR_UNSUPPORTED";
    case PSPO_ERR_HIP: return "PSPO_ERR_HIP";
    default: return "PSPO_ERR_UNKNOWN";
  }
}

const char* pspo_last_error(void) { return pspo::g_last_error.c_str(); }

int pspo_abi_version(void) { return 6; }

int pspo_validate_xi_host(const double* xi, const int64_t* xi_off, int32_t P) {
  using pspo::fail;
  pspo::clear_last_error();
  PSPO_REQUIRE(P >= 0, PSPO_ERR_INVALID_ARG, "P must be >= 0");
  if (P == 0) return PSPO_OK;
  PSPO_REQUIRE(xi_off != nullptr, PSPO_ERR_INVALID_ARG, "xi_off is NULL");
  PSPO_REQUIRE(xi_off[0] == 0, PSPO_ERR_INVALID_ARG, "xi_off[0] must be 0");
  for (int32_t p = 0; p < P; ++p)
    PSPO_REQUIRE(xi_off[p + 1] >= xi_off[p], PSPO_ERR_INVALID_ARG, "xi_off must be non-decreasing");
  PSPO_REQUIRE(xi != nullptr || xi_off[P] == 0, PSPO_ERR_INVALID_ARG, "xi is NULL");
  for (int32_t p = 0; p < P; ++p) {
    for (int64_t e = xi_off[p]; e < xi_off[p + 1]; ++e) {
      const double v = xi[e];
      if (!(v > 0.0 && v <= 1.0))
        return fail(PSPO_ERR_BAD_XI, "xi of prompt " + std::to_string(p) + " leaves (0, 1] at t = " +
                                         std::to_string(e - xi_off[p] + 1));
      if (e > xi_off[p] && v > xi[e - 1])
        return fail(PSPO_ERR_BAD_XI, "xi of prompt " + std::to_string(p) + " increases at t = " +
                                         std::to_string(e - xi_off[p] + 1));
    }
  }
  return PSPO_OK;
}

}  // extern "C"
