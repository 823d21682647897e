// Copies of bf16 matrices into the K-blocked operand layout of the matrix-core
// products: element (r, k) of an operand with R rows per K block sits at
// ((k / 32) * R + r) * 32 + k % 32.
#pragma once

#include "common.h"
#include "gemm.h"

namespace pspo {
namespace {

// K-blocked copies of (selected) bf16 rows, in one pass over the source.
// Row t of the copy is row idx[t] (or t) of the row-major `src` (row stride
// ld_src elements, `cols` columns, cols % 8 == 0) for t < n, where
// n = min(rows, *n_dev) (or rows), and zero for n <= t.  Columns cols ..
// round_up(cols, 64) - 1 of the copy are zero (the K padding the products
// need).  With n_dev, 32-row blocks at or past the next multiple of kTileLcm
// above n are not written (no product reads them).
//   dst_kb (if not NULL): the rows K-blocked with R_kb rows per K block:
//     element (t, c) at ((c / 32) * R_kb + t) * 32 + c % 32;
//   dst_t (if not NULL): their transpose, in blocks of `chunk` rows (a
//     multiple of 32), each K-blocked with R_t >= round_up(cols, 64) rows per
//     K block: element (t, c) at
//     (t / chunk) * R_t * chunk + (((t % chunk) / 32) * R_t + c) * 32 + t % 32
//     (rows round_up(cols, 64) .. R_t-1 of each K block are left unwritten).
// Grid (ceil(cols / 64), rows_pad / 32), 256 threads: a 32 x 64 tile, one
// 16-byte piece per thread in and out; the transposed pieces go through LDS
// and are written as whole 64-byte K rows (each output row of the tile is 32
// source rows).
__global__ __launch_bounds__(256) void kblock_rows_kernel(const uint16_t* __restrict__ src, int64_t ld_src, int cols,
                                                          int rows,
                                                          const int32_t* __restrict__ idx,
                                                          const int32_t* __restrict__ n_dev,
                                                          uint16_t* __restrict__ dst_kb, int64_t R_kb,
                                                          uint16_t* __restrict__ dst_t, int64_t R_t, int64_t chunk) {
  __shared__ uint16_t tile[32][64 + 8];   // padded rows: the column reads below hit distinct banks
  int n = rows;
  const int r0 = blockIdx.y * 32, c0 = blockIdx.x * 64;
  if (n_dev != nullptr) {
    n = min(n, *n_dev);
    if (r0 >= (n + kTileLcm - 1) / kTileLcm * kTileLcm) return;
  }
  const int tid = threadIdx.x;
  // in: row r0 + tid / 8, columns c0 + (tid % 8) * 8 .. +7
  {
    const int r = r0 + (tid >> 3), cp = (tid & 7) * 8;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (r < n && c0 + cp < cols) {   // an 8-column piece lies wholly inside or outside (cols % 8 == 0)
      const int64_t s = idx != nullptr ? idx[r] : r;
      v = *reinterpret_cast<const u32x4*>(src + s * ld_src + c0 + cp);
    }
    const int c = c0 + cp;
    if (dst_kb != nullptr)
      *reinterpret_cast<u32x4*>(dst_kb + ((int64_t)(c >> 5) * R_kb + r) * kTileK + (c & 31)) = v;
    if (dst_t != nullptr) *reinterpret_cast<u32x4*>(&tile[tid >> 3][cp]) = v;
  }
  if (dst_t == nullptr) return;
  __syncthreads();
  // out: column c0 + tid / 4 of source rows r0 + (tid % 4) * 8 .. +7
  {
    const int cl = tid >> 2, rp = (tid & 3) * 8;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = (uint32_t)tile[rp + 2 * e][cl] | ((uint32_t)tile[rp + 2 * e + 1][cl] << 16);
    u32x4 v = {w[0], w[1], w[2], w[3]};
    const int64_t blk = r0 / chunk, rin = r0 % chunk;   // 32-row blocks never straddle a chunk
    *reinterpret_cast<u32x4*>(dst_t + blk * R_t * chunk + ((rin >> 5) * R_t + c0 + cl) * kTileK + rp) = v;
  }
}

}  // namespace
}  // namespace pspo
