// Per-row dot products of bf16 rows, one wave64 per row: the target logit
// z = W[target] . h of each token and, optionally, ||h||^2 in the same pass
// over the hidden row.  The exact bf16 products are summed in fp32, lane l
// taking the 8-element pieces l, l + 64, ... of the row, then a fixed butterfly
// over the lanes, so each result depends only on its two rows.
#pragma once

#include "common.h"

namespace pspo {
namespace {

// Rows t < n, n = min(N, *n_dev) (N alone when n_dev is NULL): hidden row
// idx[t] (t when idx is NULL, row stride d), target tgt[t].  zt[t] = W[tgt[t]]
// . h; a target outside [0, V) reads no W row and gives 0 (the callers flag
// such targets and never use the value).  sqnorm[t] = ||h||^2 when sqnorm is
// not NULL.  d % 8 == 0 and 16-byte aligned rows.  Grid ceil(rows / 4), 256
// threads.
__global__ __launch_bounds__(256) void row_dots_kernel(const uint16_t* __restrict__ hidden,
                                                       const uint16_t* __restrict__ w, int d, int V, int N,
                                                       const int32_t* __restrict__ idx,
                                                       const int32_t* __restrict__ tgt,
                                                       const int32_t* __restrict__ n_dev, float* __restrict__ zt,
                                                       float* __restrict__ sqnorm) {
  const int n = n_dev != nullptr ? min(N, *n_dev) : N;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= n) return;   // uniform over the wave
  const int o = tgt[t];
  const bool has_w = o >= 0 && o < V;
  const u32x4* hr = reinterpret_cast<const u32x4*>(hidden + (int64_t)(idx != nullptr ? idx[t] : t) * d);
  const u32x4* wr = reinterpret_cast<const u32x4*>(w + (int64_t)(has_w ? o : 0) * d);
  float dot = 0.f, sq = 0.f;
  for (int c = lane; c < d / 8; c += 64) {
    const u32x4 a = hr[c];
    const u32x4 b = has_w ? wr[c] : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float alo = __uint_as_float(a[e] << 16), ahi = __uint_as_float(a[e] & 0xFFFF0000u);
      dot = fmaf(alo, __uint_as_float(b[e] << 16), dot);
      dot = fmaf(ahi, __uint_as_float(b[e] & 0xFFFF0000u), dot);
      sq += alo * alo + ahi * ahi;
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    dot += __shfl_xor(dot, off);
    sq += __shfl_xor(sq, off);
  }
  if (lane == 0) {
    zt[t] = dot;
    if (sqnorm != nullptr) sqnorm[t] = sq;
  }
}

}  // namespace
}  // namespace pspo
