// Copies of bf16 matrices into the K-blocked operand layout of the matrix-core
// products: element (r, k) of an operand with R rows per K block sits at
// ((k / 32) * R + r) * 32 + k % 32.
#pragma once

#include "common.h"
#include "gemm.h"

namespace pspo {
namespace {

// K-blocked copy of (selected) bf16 rows: row t of dst is row idx[t] (or t) of
// the row-major `src` (cols columns, a multiple of 32) for t < n, where
// n = min(rows, *n_dev) (or rows), and zeros for n <= t.  With n_dev, rows at
// or past the next multiple of kTileLcm above n are not written (no product
// reads them).  Grid (cols / 32, rows_pad / 64), 256 threads: thread -> row
// blockIdx.y * 64 + tid / 4, 16-byte chunk tid % 4 of that row's K step.
__global__ __launch_bounds__(256) void kblock_rows_kernel(const uint16_t* __restrict__ src, int64_t ld_src, int rows,
                                                          const int32_t* __restrict__ idx,
                                                          const int32_t* __restrict__ n_dev,
                                                          uint16_t* __restrict__ dst, int64_t R) {
  int n = rows;
  const int t = blockIdx.y * 64 + (threadIdx.x >> 2);
  if (n_dev != nullptr) {
    n = min(n, *n_dev);
    if (t >= (n + kTileLcm - 1) / kTileLcm * kTileLcm) return;
  }
  const int ks = blockIdx.x, q = threadIdx.x & 3;
  u32x4 v = {0u, 0u, 0u, 0u};
  if (t < n) {
    const int64_t s = idx != nullptr ? idx[t] : t;
    v = *reinterpret_cast<const u32x4*>(src + s * ld_src + ks * kTileK + q * 8);
  }
  *reinterpret_cast<u32x4*>(dst + ((int64_t)ks * R + t) * kTileK + q * 8) = v;
}

// Transposed, zero-padded copy of a bf16 [rows x cols] matrix, in blocks of
// `chunk` source rows, each block K-blocked with R >= cols rows per K block:
// source row r, column c goes to
//   dst[(r / chunk) * R * chunk + (((r % chunk) / 32) * R + c) * 32 + r % 32]
// (0 for r >= rows), i.e. block b is the [cols x chunk] transpose of rows
// [b*chunk, (b+1)*chunk) with each 32-deep K step contiguous (rows cols..R-1
// of each K step are left unwritten).  64 x 64 tiles through LDS; cols, chunk
// and the padded row count are multiples of 64.
// Optionally, row r of the source is row rmap[r] of `src` and only the first
// min(rows, *n_dev) rows are present; 64-row blocks wholly past that count are
// not written (no product reads them).
__global__ __launch_bounds__(256) void transpose_pad_kernel(const uint16_t* __restrict__ src, int rows, int cols,
                                                            int64_t ld_src, uint16_t* __restrict__ dst, int64_t R,
                                                            int64_t chunk, const int32_t* __restrict__ rmap,
                                                            const int32_t* __restrict__ n_dev) {
  __shared__ uint16_t tile[64][66];
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  if (n_dev != nullptr) {
    rows = min(rows, *n_dev);
    if (r0 >= (rows + 63) / 64 * 64) return;
  }
  for (int rr = ty; rr < 64; rr += 4) {
    const int r = r0 + rr;
    tile[rr][tx] = (r < rows) ? src[(int64_t)(rmap ? rmap[r] : r) * ld_src + c0 + tx] : (uint16_t)0;
  }
  __syncthreads();
  const int64_t block = r0 / chunk, rin = r0 % chunk + tx;
  uint16_t* out = dst + block * R * chunk + ((rin / kTileK) * R) * kTileK + rin % kTileK;
  for (int cc = ty; cc < 64; cc += 4) out[(int64_t)(c0 + cc) * kTileK] = tile[tx][cc];
}

}  // namespace
}  // namespace pspo
