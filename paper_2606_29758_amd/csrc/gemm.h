// Tiled bf16 x bf16 -> fp32 matrix-core (MFMA) product for CDNA4 (gfx950),
// with a pluggable epilogue.  Every contraction of the LM-head loss is one of
// these "NT" products:
//
//   C[m][n] = sum_k A[m][k] * B[n][k],  A: [M x K], B: [N x K], both row-major
//   with K contiguous (row strides lda / ldb in elements), K % 64 == 0.
//
// Tiling: a 256-thread work-group (4 wave64s in a 2 x 2 arrangement) owns a
// 256 x 256 C tile; each wave owns 128 x 128 = 4 x 4 blocks of the
// v_mfma_f32_32x32x16_bf16 instruction, i.e. 256 fp32 accumulators per lane.
// K advances in steps of 64: A and B slices (256 rows x 128 bytes each) are
// loaded with 16-byte global loads into registers one step ahead and stored
// into a double-buffered LDS ring (2 x 64 KB), with an XOR swizzle of the
// 16-byte chunks so that the MFMA operand reads are bank-conflict free.
//
// Rows past M (or N) are clamped to the last valid row when loading; the
// epilogue masks them.  Work-group -> tile mapping is XCD-aware: work-groups
// are dispatched round-robin over the 8 XCDs, so consecutive tile ids are
// handed to the same XCD, in a grouped order that keeps 8 A-tiles resident
// while B-tiles stream (L2 reuse inside each XCD's private cache).
#pragma once

#include "common.h"

namespace pspo {

constexpr int kTileM = 256, kTileN = 256, kTileK = 64;
constexpr int kGemmThreads = 256;
constexpr int kNumXcd = 8;
constexpr int kGroupM = 8;

struct GemmShape {
  const uint16_t* A;
  int64_t lda;
  int M;
  const uint16_t* B;
  int64_t ldb;
  int N;
  int K;
  int tiles_m, tiles_n;
};

// Accumulator (i, j, r) of lane `lane` in wave (wm, wn) holds
//   C[row0 + wm*128 + i*32 + (r/4)*8 + (lane/32)*4 + r%4][col0 + wn*128 + j*32 + lane%32].
struct AccTile {
  f32x16 c[4][4];
};

__device__ __forceinline__ int acc_row(int wm, int i, int r, int lane) {
  return wm * 128 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
}
__device__ __forceinline__ int acc_col(int wn, int j, int lane) { return wn * 128 + j * 32 + (lane & 31); }

// Swizzled position of 16-byte chunk `c` (0..7) of LDS row `row` (row = 128 bytes).
__device__ __forceinline__ int lds_slot(int row, int c) { return row * 8 + (c ^ ((row ^ (row >> 3)) & 7)); }

__device__ __forceinline__ bool map_tile(const GemmShape& g, int& tm, int& tn) {
  const int bid = blockIdx.x;
  const int per_xcd = gridDim.x / kNumXcd;  // grid is padded to a multiple of 8
  const int t = (bid % kNumXcd) * per_xcd + bid / kNumXcd;
  if (t >= g.tiles_m * g.tiles_n) return false;
  const int width = kGroupM * g.tiles_n;
  const int first = (t / width) * kGroupM;
  const int gsize = min(g.tiles_m - first, kGroupM);
  const int rem = t % width;
  tm = first + rem % gsize;
  tn = rem / gsize;
  return true;
}

inline int gemm_grid(int tiles_m, int tiles_n) {
  const int n = tiles_m * tiles_n;
  return (n + kNumXcd - 1) / kNumXcd * kNumXcd;
}

// Epilogue interface: `Epi::apply(acc, tm, tn, wm, wn, lane, smem)`; smem is the
// (no longer needed) LDS ring, 128 KB, free for reductions after a barrier.
template <class Epi>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void gemm_nt_kernel(GemmShape g, Epi epi) {
  __shared__ u32x4 smem[2][2][kTileM * kTileK / 8];  // [buffer][A|B][256 rows x 8 chunks]

  int tm, tn;
  if (!map_tile(g, tm, tn)) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // global -> register staging: pass p covers rows p*32 + tid/8, chunk tid%8
  const int lrow = tid >> 3, lchunk = tid & 7;
  const u32x4* gA[8];
  const u32x4* gB[8];
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    const int ra = min(tm * kTileM + p * 32 + lrow, g.M - 1);
    const int rb = min(tn * kTileN + p * 32 + lrow, g.N - 1);
    gA[p] = reinterpret_cast<const u32x4*>(g.A + (int64_t)ra * g.lda) + lchunk;
    gB[p] = reinterpret_cast<const u32x4*>(g.B + (int64_t)rb * g.ldb) + lchunk;
  }
  u32x4 stA[8], stB[8];

  AccTile acc;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc.c[i][j] = f32x16{};

  const int nk = g.K / kTileK;

  auto load_global = [&](int kt) {
    const int koff = kt * (kTileK / 8);
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      stA[p] = gA[p][koff];
      stB[p] = gB[p][koff];
    }
  };
  auto store_lds = [&](int buf) {
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      const int row = p * 32 + lrow;
      smem[buf][0][lds_slot(row, lchunk)] = stA[p];
      smem[buf][1][lds_slot(row, lchunk)] = stB[p];
    }
  };

  load_global(0);
  store_lds(0);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_global(kt + 1);
    const u32x4* sA = smem[buf][0];
    const u32x4* sB = smem[buf][1];
#pragma unroll
    for (int kk = 0; kk < kTileK / 16; ++kk) {
      const int kc = kk * 2 + (lane >> 5);
      bf16x8 a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = wm * 128 + i * 32 + (lane & 31);
        a[i] = __builtin_bit_cast(bf16x8, sA[lds_slot(row, kc)]);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = wn * 128 + j * 32 + (lane & 31);
        b[j] = __builtin_bit_cast(bf16x8, sB[lds_slot(row, kc)]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc.c[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc.c[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) store_lds(buf ^ 1);
    __syncthreads();
  }

  epi.apply(acc, tm, tn, wm, wn, lane, reinterpret_cast<float*>(&smem[0][0][0]));
}

}  // namespace pspo
