// Internal helpers of libpspo (host error reporting, device vector types).
#pragma once

#include <hip/hip_runtime.h>
#include <rocprofiler-sdk-roctx/roctx.h>

#include <cstdint>
#include <cstdio>
#include <string>

#include "pspo.h"

namespace pspo {

// ---- host-side error reporting -------------------------------------------
void set_last_error(const std::string& msg);
void clear_last_error();

// Returns `code` after recording `msg` as the thread's last error.
inline int fail(int code, const std::string& msg) {
  set_last_error(msg);
  return code;
}

#define PSPO_REQUIRE(cond, code, msg) \
  do {                                \
    if (!(cond)) return ::pspo::fail((code), (msg)); \
  } while (0)

#define PSPO_HIP_CHECK(expr)                                                     \
  do {                                                                           \
    hipError_t e_ = (expr);                                                      \
    if (e_ != hipSuccess)                                                        \
      return ::pspo::fail(PSPO_ERR_HIP, std::string(#expr ": ") + hipGetErrorString(e_)); \
  } while (0)

// The kernels are written for CDNA4 (gfx950) only; this checks the current device.
int require_gfx950();

// After every kernel launch: a launch error returns PSPO_ERR_HIP naming the
// kernel.  In the debug mode (the environment variable PSPO_DEBUG set to
// anything but "" or "0", read at every launch) the stream is also
// synchronised and an execution error is returned the same way, so a failing
// kernel is named where it happens; every call then runs synchronously.
bool debug_mode();
int after_launch(const char* kernel, hipStream_t stream);

// A roctx range named after the entry point, open while the call enqueues its
// work (rocprofv3 --marker-trace shows it next to the kernels it launched; it
// costs next to nothing with no tool attached).
struct TraceRange {
  explicit TraceRange(const char* name) { roctxRangePush(name); }
  ~TraceRange() { roctxRangePop(); }
  TraceRange(const TraceRange&) = delete;
  TraceRange& operator=(const TraceRange&) = delete;
};
#define PSPO_LAUNCHED(kernel, stream)                                   \
  do {                                                                  \
    if (int rc_ = ::pspo::after_launch((kernel), (stream))) return rc_; \
  } while (0)

// Per-product timing (the measurement mode of pspo_timing_start): begin()
// records the start event of a product of `kind` on the call's stream and
// end() its end event; both do nothing while timing is off on this thread or
// its records are used up.  They return PSPO_OK or PSPO_ERR_HIP.
class ProductTimer {
 public:
  explicit ProductTimer(hipStream_t stream) : stream_(stream) {}
  int begin(int kind);
  int end();

 private:
  hipStream_t stream_;
  int rec_ = -1;
};

inline bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// The K-blocked copies (layout.h) put an operand's 32-row blocks on the grid's
// y axis, which holds at most 65535 work-groups: token and vocabulary counts
// are supported up to this many rows after padding to whole tiles.
constexpr int64_t kMaxPaddedRows = 65535LL * 32;

// ---- device vector types ---------------------------------------------------
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// float -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

}  // namespace pspo
