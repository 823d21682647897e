// Status strings, thread-local error detail, device check, the check after
// every launch (with the PSPO_DEBUG mode) and host-side validation of
// survival tables.
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>

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

}  // namespace pspo

extern "C" {

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

int pspo_abi_version(void) { return 5; }

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
