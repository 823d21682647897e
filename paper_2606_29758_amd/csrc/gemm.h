// Tiled bf16 x bf16 -> fp32 matrix-core (MFMA) product for CDNA4 (gfx950),
// with a pluggable epilogue.  Every contraction of the LM-head loss is one of
// these "NT" products:
//
//   C[m][n] = sum_k A[m][k] * B[n][k],  A: [M x K], B: [N x K].
//
// Operands are K-blocked: element (r, k) of an operand with R rows per K block
// sits at ((k / 32) * R + r) * 32 + k % 32, so the 32-deep K step of a panel of
// consecutive rows is one contiguous block of 64-byte rows.  The A operand may
// instead be row-blocked: G rows per block (a multiple of the 384-row tile, so
// that a tile's rows lie in one block), each block its own K-blocked array of G
// rows, blocks `blk_stride_a` bytes apart, i.e. element (r, k) at
// (r / G) * blk_stride_a / 2 + ((k / 32) * G + r % G) * 32 + k % 32 (the
// layout a product writes when its output tiles are to sit in compact blocks,
// read back as the A operand of another).  The caller pads
// every operand: rows [0, tiles_m * 384) of A and [0, tiles_n * 256) of B must
// be readable (their content only reaches output rows / columns the epilogue
// masks), K % 32 == 0, and K-padding entries must be zero in both operands.
//
// Tiling: a 256-thread work-group (4 wave64s, 2 x 2) owns a 384 x 256 C tile;
// each wave owns 192 x 128 = 12 x 8 blocks of v_mfma_f32_16x16x32_bf16, i.e.
// 384 fp32 accumulators per lane: row blocks 0..7 in the 256 AGPRs, row blocks
// 8..11 in 128 VGPRs.  A 384 x 256 tile moves 40 KB of operands per 32-deep K
// step for 6.3 MFLOP (154 flop/byte, against 128 for a 256 x 256 tile): the
// products are bound by the rate at which the CU's load path delivers operand
// bytes while the matrix cores run, so fewer bytes per flop is what counts.
// On random bf16 operands this tile runs 5-20% faster than 256 x 256 on the
// loss call's shapes (measured on MI355X).
//
// Pipeline: K advances in steps of 32 (one MFMA depth) through a ring of
// kStages = 4 LDS stages of 40 KB, filled by global_load_lds_dwordx4 (no
// staging registers).  Step kt runs 12 groups of 8 MFMAs (row block g times
// the 8 column blocks), with one work-group barrier in the middle of the step
// (before group 6) that waits until step kt+1's stage has landed:
//   * groups 0..5 read this step's A blocks 6..11 (A operands are
//     single-buffered: a block's register is refilled only after its MFMAs)
//     and issue the 4 B-panel loads of step kt+3;
//   * groups 6..11 read step kt+1's A blocks 0..5 and its 8 B blocks (B is
//     double-buffered) and issue the 6 A-panel loads of step kt+4 into the
//     stage this step used (every read of it was done before the barrier).
// A stage is refilled half a step after its last read, so a load has 1.75 to
// 2.5 steps to land before the barrier that needs it (a barrier at the end of
// the step gives 1.1 to 1.9 with four stages); measured 3-5% faster.
// A group's LDS reads go out after its MFMAs (they feed later groups), except
// that the reads of groups 5 and 11 are issued by groups 4 and 10, ahead of
// their MFMAs: the two full LDS waits of a step (at the barrier, and before
// the next step's first MFMAs, which need all eight B blocks) then find their
// last reads sixteen MFMAs old instead of just issued (-1% per loss call).
// Each group is fenced with sched_barrier so the compiler keeps the interleave.
// LDS rows are 64 bytes; the four 16-byte chunks of row r are stored XOR-ed
// with ((r >> 1) ^ (r >> 2)) & 3 (bank-conflict free for the 16-row operand
// reads, period 16 rows).
//
// One dimension can be bounded by a count that lives in device memory (a
// product over a data-dependent subset of tokens needs no host round trip).
// Work-group -> tile mapping is XCD-aware: work-groups are dispatched
// round-robin over the 8 XCDs, so work-groups b, b + 8, b + 16, ... share an
// XCD; each XCD runs its share of a grouped order (4 A-tiles x 8 B-tiles
// resident per XCD round) for reuse inside its private L2, and the groups are
// dealt to the XCDs so that all eight read the same B panels at the same time
// (shared through the memory-side cache).
#pragma once

#include "common.h"

namespace pspo {

constexpr int kTileM = 384, kTileN = 256, kTileK = 32;
constexpr int kGemmThreads = 256;
constexpr int kNumXcd = 8;
constexpr int kGroupM = 4;
constexpr int kStages = 4;
constexpr int kLdsRow = kTileK * 2;                // 64 bytes
constexpr int kLdsA = kTileM * kLdsRow;            // 24 KB
constexpr int kLdsB = kTileN * kLdsRow;            // 16 KB
constexpr int kLdsStage = kLdsA + kLdsB;           // 40 KB
constexpr int kLdsBytes = kStages * kLdsStage;     // 160 KB
// both tile sizes divide this: padded token counts are multiples of it
constexpr int kTileLcm = 768;

// Accumulator layout: per wave 12 x 8 blocks of 16 x 16, four fp32 per lane each.
constexpr int kBlocksM = 12, kBlocksN = 8, kBlocksAgpr = 8;
constexpr int kWaveM = kBlocksM * 16, kWaveN = kBlocksN * 16;   // 192 x 128
constexpr int kAccPerBlock = 4;
constexpr int kLoadsA = kTileM / 4 / 16, kLoadsB = kTileN / 4 / 16;   // 6 + 4 per wave per step

// Which dimension of a product a device-resident bound applies to.
constexpr int kDynNone = 0, kDynM = 1, kDynN = 2, kDynK = 3;

struct GemmShape {
  const uint16_t* A;
  int64_t rows_a;            // rows per K block of A (>= tiles_m * kTileM)
  int M;
  const uint16_t* B;
  int64_t rows_b;            // rows per K block of B (>= tiles_n * kTileN)
  int N;
  int K;
  int tiles_m, tiles_n;      // grid extent (host-side upper bound)
  // Optional bound read from device memory when the kernel starts: limits M
  // (kDynM) or N (kDynN) to *dyn, or K (kDynK) to *dyn rounded up to kTileK.
  // Tiles outside the bound exit at once; a shorter K shortens the loop.
  const int32_t* dyn = nullptr;
  int dyn_dim = kDynNone;
  // Row tiles 0 .. spread_m-1 are placed evenly among the others in the
  // grouped order (and so spread over the XCDs and their rounds) instead of
  // first: for an epilogue that does extra work on those tiles only.
  int spread_m = 0;
  // Row-blocked A (0: plain K-blocked with rows_a rows per K block): rows per
  // block (a multiple of kTileM) and bytes between blocks.
  int blk_a = 0;
  int64_t blk_stride_a = 0;
};

// Accumulator (i, j, r) of lane `lane` in wave (wm, wn) holds
//   C[row0 + wm*192 + i*16 + (lane/16)*4 + r][col0 + wn*128 + j*16 + lane%16].
struct AccTile {
  f32x4 a[kBlocksAgpr][kBlocksN];              // row blocks 0..7
  f32x4 v[kBlocksM - kBlocksAgpr][kBlocksN];   // row blocks 8..11
};

// Element access with (after unrolling) constant indices.
__device__ __forceinline__ float acc_get(const AccTile& t, int i, int j, int r) {
  return i < kBlocksAgpr ? t.a[i][j][r] : t.v[i - kBlocksAgpr][j][r];
}
__device__ __forceinline__ void acc_set(AccTile& t, int i, int j, int r, float x) {
  if (i < kBlocksAgpr) t.a[i][j][r] = x;
  else t.v[i - kBlocksAgpr][j][r] = x;
}

__device__ __forceinline__ int acc_row(int wm, int i, int r, int lane) {
  return wm * kWaveM + i * 16 + (lane >> 4) * 4 + r;
}
__device__ __forceinline__ int acc_col(int wn, int j, int lane) { return wn * kWaveN + j * 16 + (lane & 15); }

constexpr float kLog2e = 1.4426950408889634f;

// max(a, b, c) in one instruction (v_max3_f32, IEEE maxNum semantics: a NaN
// operand is ignored, as with fmaxf); written as asm because the compiler's
// fmaxf on values of unknown origin first canonicalises each operand.
__device__ __forceinline__ float max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// The 384 x 256 fp32 tile of the accumulators as one contiguous block at
// `base`: [24 blocks of 16 rows][256 columns][16].  An accumulator block is 16
// rows x 16 columns and the lane's 4 rows of it one 16-byte piece, so each
// store instruction writes 1 KB of whole 128-byte lines (a store of half lines
// makes the L2 fetch the other half from memory); non-temporal stores.  AGPR
// blocks are read by explicit v_accvgpr_read: taken as one 4-register value,
// the compiler keeps a VGPR copy of the block live from the loop's end and
// spills accumulators to make room.
__device__ __forceinline__ void store_tile_rows16(const AccTile& acc, float* base, int wm, int wn, int lane) {
  unsigned char* zb = reinterpret_cast<unsigned char*>(base);
  const uint32_t lo = (uint32_t)(wm * (kWaveM / 16)) * (kTileN * 64u) + (uint32_t)(wn * kWaveN + (lane & 15)) * 64u +
                      (uint32_t)(lane >> 4) * 16u;
#pragma unroll
  for (int i = 0; i < kBlocksM; ++i) {
#pragma unroll
    for (int j = 0; j < kBlocksN; ++j) {
      f32x4 b;
      if (i < kBlocksAgpr) {
#pragma unroll
        for (int r = 0; r < kAccPerBlock; ++r) {
          float x;
          asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(x) : "a"(acc.a[i][j][r]));
          b[r] = x;
        }
      } else {
        b = acc.v[i - kBlocksAgpr][j];
      }
      __builtin_nontemporal_store(b, reinterpret_cast<f32x4*>(zb + (lo + (uint32_t)(i * kTileN * 64 + j * 1024))));
    }
    __builtin_amdgcn_sched_barrier(0);   // one row block's stores at a time
  }
}

__device__ __forceinline__ int chunk_swizzle(int row) { return ((row >> 1) ^ (row >> 2)) & 3; }

// Tile of work-group blockIdx.x among the tiles_m x tiles_n tiles that cover
// an M x N product (tiles_m/n: the launch's extents, possibly more than the
// product needs when M or N is bounded on the device).  The tile count is
// taken from the actual M and N so that the work spreads over all XCDs even
// when a device-side bound leaves only part of the launch with work.
// Row tile of launch-order position l when the first s of T row tiles are
// spread: position l holds one of them iff the count ceil((l + 1) s / T) of
// such slots up to l grows at l (slots evenly spaced, in increasing order);
// the other tiles keep their order.  A bijection on [0, T).
__host__ __device__ inline int spread_row_tile(int l, int s, int T) {
  const int c = ((l + 1) * s + T - 1) / T, cp = (l * s + T - 1) / T;
  return c > cp ? c - 1 : s + l - c;
}

// M, N, K of a product after its device-side bound.
__device__ __forceinline__ void bounded_dims(const GemmShape& g, int& M, int& N, int& K) {
  M = g.M;
  N = g.N;
  K = g.K;
  if (g.dyn != nullptr) {
    const int v = max(__builtin_amdgcn_readfirstlane(*g.dyn), 0);
    if (g.dyn_dim == kDynM) M = min(M, v);
    else if (g.dyn_dim == kDynN) N = min(N, v);
    else if (g.dyn_dim == kDynK) K = min(K, (v + kTileK - 1) / kTileK * kTileK);
  }
}

// The tiles of a product bounded to M x N (tiles_m/n: the launch's extents),
// and which positions of the grouped order each XCD runs: the whole groups
// (kGroupM row tiles x all column tiles) that divide evenly among the XCDs are
// dealt round-robin, group g to XCD g % 8, so that at any time every XCD works
// on the same column tiles (the memory-side cache then serves the column
// panels to all eight from one fetch); the positions left over are split into
// contiguous runs of per_rest.  Each XCD runs at most per_xcd positions.
struct TileGrid {
  int tiles_m, tiles_n, total, per_xcd;
  int width;       // positions per group
  int per_dealt;   // positions of the dealt groups per XCD
  int rest0;       // first position after the dealt groups
  int per_rest;    // positions of the remainder per XCD (the last run may be shorter)
};
__host__ __device__ inline TileGrid tile_grid(int tiles_m, int tiles_n, int M, int N) {
  TileGrid tg;
  tg.tiles_m = min(tiles_m, (M + kTileM - 1) / kTileM);
  tg.tiles_n = min(tiles_n, (N + kTileN - 1) / kTileN);
  tg.total = tg.tiles_m * tg.tiles_n;
  tg.width = kGroupM * tg.tiles_n;
  const int dealt = tg.tiles_m / kGroupM / kNumXcd * kNumXcd;
  tg.per_dealt = dealt / kNumXcd * tg.width;
  tg.rest0 = dealt * tg.width;
  tg.per_rest = (tg.total - tg.rest0 + kNumXcd - 1) / kNumXcd;
  tg.per_xcd = tg.per_dealt + tg.per_rest;   // = ceil(total / 8)
  return tg;
}
// Number of positions XCD x runs.
__host__ __device__ inline int xcd_count(const TileGrid& tg, int x) {
  return tg.per_dealt + min(max(tg.total - tg.rest0 - x * tg.per_rest, 0), tg.per_rest);
}
// Grouped-order position of XCD x's k-th tile (k < xcd_count(tg, x)).
__host__ __device__ inline int xcd_position(const TileGrid& tg, int x, int k) {
  if (k < tg.per_dealt) return ((k / tg.width) * kNumXcd + x) * tg.width + k % tg.width;
  return tg.rest0 + x * tg.per_rest + (k - tg.per_dealt);
}
// Tile (tm, tn) at position t of the grouped order (kGroupM row tiles x all
// column tiles per group).
__host__ __device__ inline void tile_at(const TileGrid& tg, int t, int spread_m, int& tm, int& tn) {
  const int width = kGroupM * tg.tiles_n;
  const int first = (t / width) * kGroupM;
  const int gsize = min(tg.tiles_m - first, kGroupM);
  const int rem = t % width;
  tm = first + rem % gsize;
  tn = rem / gsize;
  if (spread_m > 0) tm = spread_row_tile(tm, min(spread_m, tg.tiles_m), tg.tiles_m);
}

// How a launch covers the tiles.  An XCD's share of up to per_xcd positions on
// its 32 CUs that is no multiple of 32 ends in a partial round of whole tiles; a
// product with long tiles can instead run its whole rounds in one launch and
// the rest, split along K, in a second one whose parts fill the CUs.
enum : int {
  kLaunchWhole = 0,    // every position
  kLaunchRounds = 1,   // each XCD's first 32 floor(per_xcd / 32) positions
  kLaunchTail = 2,     // the rest, each tile in K parts (map_tail)
};
constexpr int kTailSlots = 64;   // work-groups per XCD of a tail launch (two rounds)

// Tile of work-group `bid` of a whole or whole-rounds launch.
__host__ __device__ inline bool map_tile_at(int bid, int tiles_m, int tiles_n, int M, int N, int& tm, int& tn,
                                            int spread_m, bool rounds_only) {
  const TileGrid tg = tile_grid(tiles_m, tiles_n, M, N);
  const int x = bid % kNumXcd, k = bid / kNumXcd;
  if (k >= xcd_count(tg, x)) return false;
  if (rounds_only && k >= tg.per_xcd / 32 * 32) return false;
  tile_at(tg, xcd_position(tg, x, k), spread_m, tm, tn);
  return true;
}
__device__ __forceinline__ bool map_tile(int tiles_m, int tiles_n, int M, int N, int& tm, int& tn,
                                         int spread_m = 0, bool rounds_only = false) {
  return map_tile_at(blockIdx.x, tiles_m, tiles_n, M, N, tm, tn, spread_m, rounds_only);
}

// K parts of each tail tile of an XCD with r tail tiles and nk K steps: the
// S <= min(64 / r, nk) with the fewest rounds per part, ceil(r S / 32) / S
// (the smaller S on ties).
__host__ __device__ inline int tail_parts(int r, int nk) {
  int best = 1, best_rounds = (r + 31) / 32;
  for (int s = 2; s * r <= kTailSlots && s <= nk; ++s) {
    const int rounds = (r * s + 31) / 32;
    if (rounds * best < best_rounds * s) {
      best = s;
      best_rounds = rounds;
    }
  }
  return best;
}

// Epilogue of a tail launch: the part's accumulators to slab `blockIdx.x`.
struct EpiSlab {
  float* slab;
  __device__ __forceinline__ void apply(const AccTile& acc, int, int, int wm, int wn, int lane, float*) const {
    store_tile_rows16(acc, slab + (int64_t)blockIdx.x * (kTileM * kTileN), wm, wn, lane);
  }
};

// Tail launch: work-group x + 8 k (x the XCD, k < 64) takes part k % S of the
// XCD's tail tile k / S, K steps [part nk / S, (part + 1) nk / S).  The tail
// tiles are the positions after the XCD's whole rounds.  Returns false for
// work-groups without a part.
__host__ __device__ inline bool map_tail(const TileGrid& tg, int bid, int nk, int& tm, int& tn, int& kb, int& ke,
                                         int* u_out = nullptr, int* parts_out = nullptr) {
  const int x = bid % kNumXcd, k = bid / kNumXcd;
  const int full = tg.per_xcd / 32 * 32;
  const int r = xcd_count(tg, x) - full;
  if (r <= 0 || k >= kTailSlots) return false;
  const int parts = tail_parts(r, nk);
  const int u = k / parts, part = k % parts;
  if (u >= r) return false;
  tile_at(tg, xcd_position(tg, x, full + u), 0, tm, tn);
  kb = part * nk / parts;
  ke = (part + 1) * nk / parts;
  if (u_out) *u_out = u;
  if (parts_out) *parts_out = parts;
  return true;
}

inline int gemm_grid(int tiles_m, int tiles_n) {
  const int n = tiles_m * tiles_n;
  return (n + kNumXcd - 1) / kNumXcd * kNumXcd;
}

template <int N>
struct Const {
  static constexpr int value = N;
};

typedef __attribute__((address_space(3))) void lds_void;

// c += a * b on one 16 x 16 x 32 bf16 block, accumulating in place (AGPRs or
// VGPRs).  Written as inline asm with the accumulator tied in/out: through the
// builtin, the register allocator is free to give the result a different
// register quadruple than the addend, and with every accumulator register live
// it then rotates accumulators through other registers with copies on every
// loop trip (each of which waits for the MFMA producing it).  The compiler's
// hazard tracking does not see inline asm as an MFMA, so the kernel pads the
// MFMA -> VALU hazard itself before its epilogue reads the accumulators
// (mfma_drain below); inside the loop no instruction reads or writes an
// accumulator register between the MFMAs that update it (the write-after-read
// hazard rules of the MFMA unit concern its accumulator input only).
__device__ __forceinline__ void mfma_agpr(f32x4& c, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}
__device__ __forceinline__ void mfma_vgpr(f32x4& c, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b));
}

// Enough independent wait states for any MFMA result to be readable by VALU,
// accvgpr reads or memory instructions (16-pass worst case plus margin).
__device__ __forceinline__ void mfma_drain() {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
}

// Work-group barrier for the LDS ring: waits until at most `Vm` of this wave's
// global->LDS loads are outstanding and all its LDS reads are done, then
// s_barrier.  (__syncthreads() would wait for every outstanding load, since its
// release fence covers loads that write LDS.)  The wait is the s_waitcnt
// builtin so the compiler's own wait-count tracking sees it; the barrier is
// inline asm with a "memory" clobber so no memory access moves across it.
template <int Vm>
__device__ __forceinline__ void stage_barrier() {
  static_assert(Vm >= 0 && Vm < 64, "vmcnt is a 6-bit field");
  // gfx9 s_waitcnt immediate: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14]
  constexpr int imm = (Vm & 0xF) | (0x7 << 4) | (0x0 << 8) | ((Vm >> 4) << 14);
  __builtin_amdgcn_s_waitcnt(imm);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// Epilogue interface: `Epi::apply(acc, tm, tn, wm, wn, lane, smem)` (acc may be
// overwritten); smem is the (no longer needed) LDS ring, 160 KB, free for
// reductions: every load into it has landed and all waves have passed a
// barrier before the call.
template <class Epi, int kLaunch = kLaunchWhole>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void gemm_nt_kernel(GemmShape g, Epi epi) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kLdsBytes];

  int M, N, K;
  bounded_dims(g, M, N, K);
  int tm, tn, kb = 0, nk = K / kTileK;
  if constexpr (kLaunch == kLaunchTail) {
    int ke;
    if (!map_tail(tile_grid(g.tiles_m, g.tiles_n, M, N), blockIdx.x, nk, tm, tn, kb, ke)) return;
    nk = ke - kb;
  } else {
    if (!map_tile(g.tiles_m, g.tiles_n, M, N, tm, tn, g.spread_m, kLaunch == kLaunchRounds)) return;
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  // Direct-to-LDS loads: a load instruction writes 16 rows (1 KB) of a stage;
  // lane l writes physical chunk l % 4 of row l / 4 and therefore fetches the
  // logical chunk (l % 4) ^ swizzle(row) of that row's 64-byte K slice.  Wave w
  // loads A rows w*96 + q*16 (q < 6) and B rows w*64 + q*16 (q < 4).
  const uint32_t lane_off = (uint32_t)((lane >> 2) * kLdsRow + (((lane & 3) ^ chunk_swizzle(lane >> 2)) << 4));
  // bytes per K step; the wave's A rows start at gA (the tile lies inside one
  // block of a row-blocked A)
  const int64_t kstep_a = (g.blk_a > 0 ? (int64_t)g.blk_a : g.rows_a) * kLdsRow, kstep_b = g.rows_b * kLdsRow;
  const int64_t ra = (int64_t)tm * kTileM + wave * (kTileM / 4);
  const unsigned char* gA = reinterpret_cast<const unsigned char*>(g.A) + (int64_t)kb * kstep_a +
                            (g.blk_a > 0 ? (ra / g.blk_a) * g.blk_stride_a + (ra % g.blk_a) * kLdsRow : ra * kLdsRow);
  const unsigned char* gB = reinterpret_cast<const unsigned char*>(g.B) +
                            ((int64_t)tn * kTileN + wave * (kTileN / 4)) * kLdsRow + (int64_t)kb * kstep_b;

  // MFMA operand reads: block i of A is rows wm*192 + i*16 + lane%16, K chunk
  // lane/16 (8 bf16 of the 32-deep step).  The swizzle of row r + 16 i equals
  // that of row r, so block i is the lane's base plus i * 16 rows.
  const int rdA = (wm * kWaveM + (lane & 15)) * kLdsRow + (((lane >> 4) ^ chunk_swizzle(lane & 15)) << 4);
  const int rdB = kLdsA + (wn * kWaveN + (lane & 15)) * kLdsRow + (((lane >> 4) ^ chunk_swizzle(lane & 15)) << 4);

  bf16x8 fa[kBlocksM], fb[2][kBlocksN];
  AccTile acc;
#pragma unroll
  for (int i = 0; i < kBlocksAgpr; ++i)
#pragma unroll
    for (int j = 0; j < kBlocksN; ++j) acc.a[i][j] = f32x4{};
#pragma unroll
  for (int i = 0; i < kBlocksM - kBlocksAgpr; ++i)
#pragma unroll
    for (int j = 0; j < kBlocksN; ++j) acc.v[i][j] = f32x4{};


  auto read_a = [&](int stage, int i) -> bf16x8 {
    return __builtin_bit_cast(bf16x8,
                              *reinterpret_cast<const u32x4*>(lds + stage * kLdsStage + rdA + i * 16 * kLdsRow));
  };
  auto read_b = [&](int stage, int j) -> bf16x8 {
    return __builtin_bit_cast(bf16x8,
                              *reinterpret_cast<const u32x4*>(lds + stage * kLdsStage + rdB + j * 16 * kLdsRow));
  };
  // Load q (0..9) of step kt into `stage`; steps past the last reload the last
  // one (in bounds, never consumed), so every step issues the same count.
  auto issue_load = [&](int kt, int stage, int q) {
    const int64_t kk = max(min(kt, nk - 1), 0);
    if (q < kLoadsA) {
      __builtin_amdgcn_global_load_lds(
          gA + kk * kstep_a + q * 16 * kLdsRow + lane_off,
          (lds_void*)(lds + stage * kLdsStage + (wave * (kTileM / 4) + q * 16) * kLdsRow), 16, 0, 0);
    } else {
      __builtin_amdgcn_global_load_lds(
          gB + kk * kstep_b + (q - kLoadsA) * 16 * kLdsRow + lane_off,
          (lds_void*)(lds + stage * kLdsStage + kLdsA + (wave * (kTileN / 4) + (q - kLoadsA) * 16) * kLdsRow), 16,
          0, 0);
    }
  };

  // Group g of step kt: (the mid-step barrier before group 6,) 8 MFMAs of row
  // block g on B slot s, then its LDS reads and global->LDS loads (groups 4
  // and 10: the reads of g and g + 1 first, then the MFMAs).  Loads of step s
  // go out in groups 6..11 of step s-4 (A) and 0..3 of step s-3 (B); at the
  // barrier of step kt, step kt+1's loads must have landed, and the 20 issued
  // after them (steps kt+2, kt+3) may still be in flight.
  auto group = [&](auto slot, int kt, int cur, int nxt, auto gq) {
    constexpr int s = decltype(slot)::value, gi = decltype(gq)::value;
    if constexpr (gi == kBlocksM / 2) stage_barrier<2 * (kLoadsA + kLoadsB)>();
    // the LDS reads that belong to group g (none feeds group g's own MFMAs):
    // groups 0..5 read this step's A blocks 6..11; groups 6..11 the next
    // step's A blocks 0..5 and its B blocks 2, 2, 1, 1, 1, 1
    auto reads = [&](auto gr) {
      constexpr int g = decltype(gr)::value;
      if constexpr (g < kBlocksM / 2) {
        fa[g + 6] = read_a(cur, g + 6);
      } else {
        fa[g - 6] = read_a(nxt, g - 6);
        if constexpr (g == 6) {
          fb[1 - s][0] = read_b(nxt, 0);
          fb[1 - s][1] = read_b(nxt, 1);
        } else if constexpr (g == 7) {
          fb[1 - s][2] = read_b(nxt, 2);
          fb[1 - s][3] = read_b(nxt, 3);
        } else {
          fb[1 - s][g - 4] = read_b(nxt, g - 4);
        }
      }
    };
    constexpr bool early = gi == kBlocksM / 2 - 2 || gi == kBlocksM - 2;   // groups 4 and 10
    constexpr bool none = gi == kBlocksM / 2 - 1 || gi == kBlocksM - 1;    // groups 5 and 11
    if constexpr (early) {
      reads(Const<gi>{});
      reads(Const<gi + 1>{});
    }
#pragma unroll
    for (int j = 0; j < kBlocksN; ++j) {
      if constexpr (gi < kBlocksAgpr) mfma_agpr(acc.a[gi][j], fa[gi], fb[s][j]);
      else mfma_vgpr(acc.v[gi - kBlocksAgpr][j], fa[gi], fb[s][j]);
    }
    if constexpr (!early && !none) reads(Const<gi>{});
    if constexpr (gi < kBlocksM / 2) {
      if constexpr (gi < kLoadsB) issue_load(kt + 3, (kt + 3) % kStages, kLoadsA + gi);
    } else {
      issue_load(kt + 4, cur, gi - 6);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  auto step = [&](auto slot, int kt) {
    const int cur = kt % kStages, nxt = (kt + 1) % kStages;
    group(slot, kt, cur, nxt, Const<0>{}); group(slot, kt, cur, nxt, Const<1>{});
    group(slot, kt, cur, nxt, Const<2>{}); group(slot, kt, cur, nxt, Const<3>{});
    group(slot, kt, cur, nxt, Const<4>{}); group(slot, kt, cur, nxt, Const<5>{});
    group(slot, kt, cur, nxt, Const<6>{}); group(slot, kt, cur, nxt, Const<7>{});
    group(slot, kt, cur, nxt, Const<8>{}); group(slot, kt, cur, nxt, Const<9>{});
    group(slot, kt, cur, nxt, Const<10>{}); group(slot, kt, cur, nxt, Const<11>{});
  };
  static_assert(kStages == 4 && kBlocksM == 12 && kBlocksN == 8 && kLoadsA == 6 && kLoadsB == 4,
                "the group schedule is written for this tile");

  // Prologue: steps 0..2 and the A part of step 3 in flight (its B part goes
  // out in groups 0..3 of step 0); wait for step 0; its A blocks 0..5 and B
  // blocks into registers (A blocks 6..11 are read in groups 0..5).  With
  // nk == 0 (a device-side K bound of 0) the loads and reads still happen, at
  // K offset 0, but no MFMA consumes them and the accumulators stay zero.
#pragma unroll
  for (int st = 0; st < kStages - 1; ++st)
#pragma unroll
    for (int q = 0; q < kLoadsA + kLoadsB; ++q) issue_load(st, st, q);
#pragma unroll
  for (int q = 0; q < kLoadsA; ++q) issue_load(kStages - 1, kStages - 1, q);
  stage_barrier<2 * (kLoadsA + kLoadsB) + kLoadsA>();
#pragma unroll
  for (int i = 0; i < kBlocksM / 2; ++i) fa[i] = read_a(0, i);
#pragma unroll
  for (int j = 0; j < kBlocksN; ++j) fb[0][j] = read_b(0, j);

  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    step(Const<0>{}, kt);
    step(Const<1>{}, kt + 1);
  }
  if (kt < nk) step(Const<0>{}, kt);

  // drain the (clamped, unused) loads still in flight before LDS is reused
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
  mfma_drain();
  __syncthreads();

  epi.apply(acc, tm, tn, wm, wn, lane, reinterpret_cast<float*>(lds));
}

}  // namespace pspo
