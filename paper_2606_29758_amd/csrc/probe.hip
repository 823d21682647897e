// Measurement helper: the sustained rate of the matrix cores on the MFMA form
// the products use (v_mfma_f32_16x16x32_bf16, tied accumulators), with no
// memory traffic.  It bounds what any schedule of the products can reach at the
// clock the chip holds under matrix-core load, next to the published peak.
#include "common.h"
#include "gemm.h"

namespace pspo {
namespace {

constexpr int kProbeChains = 16;   // independent accumulators per wave: covers the MFMA latency

__global__ __launch_bounds__(256) void mfma_loop_kernel(int iters, float* __restrict__ out) {
  const int tid = threadIdx.x;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(0.001f * (float)((tid + e) & 15));
    b[e] = (__bf16)(0.002f * (float)((tid * 3 + e) & 7));
  }
  f32x4 acc[kProbeChains];
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kProbeChains; ++c) mfma_vgpr(acc[c], a, b);
  }
  mfma_drain();
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  out[(int64_t)blockIdx.x * 256 + tid] = s;
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
  PSPO_HIP_CHECK(hipGetLastError());
  return PSPO_OK;
}
