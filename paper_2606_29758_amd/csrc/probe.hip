// Measurement helper: the sustained rate of the matrix cores on the MFMA form
// the products use (v_mfma_f32_16x16x32_bf16, tied accumulators), with no
// memory traffic.  It bounds what any schedule of the products can reach at the
// clock the chip holds under matrix-core load, next to the published peak.
#include "common.h"
#include "gemm.h"

namespace pspo {
namespace {

constexpr int kProbeChains = 16;   // independent accumulators per wave: covers the MFMA latency

// A bf16 in [-1, 1) from a 32-bit hash (random mantissa bits, like real operands).
__device__ __forceinline__ __bf16 probe_value(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return (__bf16)((float)(int32_t)x * (1.0f / 2147483648.0f));
}

__global__ __launch_bounds__(256) void mfma_loop_kernel(int iters, float* __restrict__ out) {
  const uint32_t tid = blockIdx.x * 256u + threadIdx.x;
  // two operand sets, alternated between consecutive MFMAs, so that the
  // operand bits toggle as they do in the products (power follows the data)
  bf16x8 a[2], b[2];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      a[s][e] = probe_value(tid * 32u + s * 16u + e);
      b[s][e] = probe_value(tid * 32u + s * 16u + 8u + e);
    }
  f32x4 acc[kProbeChains];
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kProbeChains; ++c) mfma_vgpr(acc[c], a[c & 1], b[c & 1]);
  }
  mfma_drain();
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  out[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace
}  // namespace pspo

extern "C" int pspo_mfma_loop(int32_t iters, int32_t blocks, float* out, hipStream_t stream) {
  using namespace pspo;
  clear_last_error();
  PSPO_REQUIRE(iters >= 1 && blocks >= 1, PSPO_ERR_INVALID_ARG, "iters and blocks must be >= 1");
  PSPO_REQUIRE(out != nullptr && aligned(out, 4), PSPO_ERR_INVALID_ARG, "out must be a non-NULL float pointer");
  if (int rc = require_gfx950()) return rc;
  hipLaunchKernelGGL(mfma_loop_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, iters, out);
  PSPO_LAUNCHED("mfma_loop_kernel", stream);
  return PSPO_OK;
}
