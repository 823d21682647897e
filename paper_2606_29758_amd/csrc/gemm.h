// Tiled bf16 x bf16 -> fp32 matrix-core (MFMA) product for CDNA4 (gfx950),
// with a pluggable epilogue.  Every contraction of the LM-head loss is one of
// these "NT" products:
//
//   C[m][n] = sum_k A[m][k] * B[n][k],  A: [M x K], B: [N x K], both row-major
//   with K contiguous (row strides lda / ldb in elements), K % 32 == 0, K > 0.
//
// Tiling: a 256-thread work-group (4 wave64s in a 2 x 2 arrangement) owns a
// 256 x 256 C tile; each wave owns 128 x 128 = 8 x 8 blocks of the
// v_mfma_f32_16x16x32_bf16 instruction, i.e. 256 fp32 accumulators per lane
// (the whole AGPR file).  On real (random) bf16 operands this instruction
// sustains a markedly higher rate than the 32x32x16 form at the same LDS
// traffic per flop (measured on MI355X: ~86% vs ~77% of peak in a pure MFMA
// loop), so it is the one used.
//
// Pipeline: K advances in steps of 32 (one MFMA depth) through a ring of
// kStages LDS stages (32 KB each: 256 rows x 64 bytes of A and of B).
// Operands go from global memory straight into LDS (global_load_lds_dwordx4:
// no staging registers, no LDS-write instructions); each wave loads 64 rows of
// A and 64 rows of B per step.  Step kt:
//   1. 64 MFMAs on the register slot holding step kt's operands, interleaved
//      with the 16 LDS reads of step kt+1's operands (into the other slot) and
//      the 8 loads of step kt+kStages-1 into the stage step kt-1 used;
//   2. wait until this wave's loads of step kt+2 have landed and its LDS reads
//      are done, then one work-group barrier: step kt+2 is visible to all and
//      every wave is done with the stage step kt used.
// A load therefore has kStages-3 whole steps (about 1000 MFMA cycles each) to
// land.  Each group of four MFMAs and its memory ops is fenced with
// sched_barrier so the compiler keeps the interleave.  LDS rows are 64 bytes;
// the four 16-byte chunks of row r are stored XOR-ed with ((r>>1) ^ (r>>2)) & 3,
// which is bank-conflict free for the 16-row operand reads and repeats every
// 16 rows, so all reads of a step use one per-lane base plus fixed offsets.
//
// Rows past M (or N) are clamped to the last valid row when loading; the
// epilogue masks them.  B rows can be gathered through an index map, and one
// dimension can be bounded by a count that lives in device memory (so a
// product over a data-dependent subset of tokens needs no host round trip).  Work-group -> tile mapping is XCD-aware: work-groups
// are dispatched round-robin over the 8 XCDs, so consecutive tile ids are
// handed to the same XCD, in a grouped order that keeps 8 A-tiles resident
// while B-tiles stream (L2 reuse inside each XCD's private cache).
#pragma once

#include "common.h"

namespace pspo {

constexpr int kTileM = 256, kTileN = 256, kTileK = 32;
constexpr int kGemmThreads = 256;
constexpr int kNumXcd = 8;
constexpr int kGroupM = 8;
constexpr int kStages = 5;
constexpr int kLdsRow = kTileK * 2;                // 64 bytes
constexpr int kLdsOperand = kTileM * kLdsRow;      // 16 KB
constexpr int kLdsStage = 2 * kLdsOperand;         // A + B: 32 KB
constexpr int kLdsBytes = kStages * kLdsStage;     // 160 KB

// Accumulator layout: per wave 8 x 8 blocks of 16 x 16, four fp32 per lane each.
constexpr int kBlocks = 8;
constexpr int kAccPerBlock = 4;

// Which dimension of a product a device-resident bound applies to.
constexpr int kDynNone = 0, kDynM = 1, kDynN = 2, kDynK = 3;

struct GemmShape {
  const uint16_t* A;
  int64_t lda;
  int M;
  const uint16_t* B;
  int64_t ldb;
  int N;
  int K;
  int tiles_m, tiles_n;      // grid extent (host-side upper bound)
  // Optional gather: row r of the B operand is row b_rows[r] of B.
  const int32_t* b_rows = nullptr;
  // Optional bound read from device memory when the kernel starts: limits M
  // (kDynM) or N (kDynN) to *dyn, or K (kDynK) to *dyn rounded up to kTileK.
  // Tiles outside the bound exit at once; a shorter K shortens the loop.
  const int32_t* dyn = nullptr;
  int dyn_dim = kDynNone;
  // K-blocked operands: element (r, k) of a K-blocked operand with row count
  // R lives at ((k / 32) * R + r) * 32 + k % 32, so each 32-deep K step of a
  // panel is one contiguous block; its lda / ldb is then R * 32 (elements from
  // one K step to the next) instead of the row stride.
  bool a_kb = false, b_kb = false;
};

// Accumulator (i, j, r) of lane `lane` in wave (wm, wn) holds
//   C[row0 + wm*128 + i*16 + (lane/16)*4 + r][col0 + wn*128 + j*16 + lane%16].
struct AccTile {
  f32x4 c[kBlocks][kBlocks];
};

__device__ __forceinline__ int acc_row(int wm, int i, int r, int lane) {
  return wm * 128 + i * 16 + (lane >> 4) * 4 + r;
}
__device__ __forceinline__ int acc_col(int wn, int j, int lane) { return wn * 128 + j * 16 + (lane & 15); }

// The accumulator of column block j that sits in row `rel` of this lane's rows
// (rel = row - (wm * 128 + (lane / 16) * 4); the lane holds rows i * 16 + r,
// i < 8, r < 4), picked with selects only (no divergent branch per value).
// Returns whether the lane holds that row.
__device__ __forceinline__ bool acc_pick(const AccTile& acc, int j, int rel, float& value) {
  float z = 0.f;
  bool has = false;
#pragma unroll
  for (int i = 0; i < kBlocks; ++i)
#pragma unroll
    for (int r = 0; r < kAccPerBlock; ++r) {
      const bool hit = rel == i * 16 + r;
      z = hit ? acc.c[i][j][r] : z;
      has = has || hit;
    }
  value = z;
  return has;
}

__device__ __forceinline__ int chunk_swizzle(int row) { return ((row >> 1) ^ (row >> 2)) & 3; }

// Tile of work-group blockIdx.x among the tiles_m x tiles_n tiles that cover
// an M x N product (tiles_m/n: the launch's extents, possibly more than the
// product needs when M or N is bounded on the device).  The tile count is
// taken from the actual M and N so that the work spreads over all XCDs even
// when a device-side bound leaves only part of the launch with work.
__device__ __forceinline__ bool map_tile(int tiles_m, int tiles_n, int M, int N, int& tm, int& tn) {
  tiles_m = min(tiles_m, (M + kTileM - 1) / kTileM);
  tiles_n = min(tiles_n, (N + kTileN - 1) / kTileN);
  const int total = tiles_m * tiles_n;
  const int per_xcd = (total + kNumXcd - 1) / kNumXcd;
  const int bid = blockIdx.x;
  if (bid / kNumXcd >= per_xcd) return false;
  const int t = (bid % kNumXcd) * per_xcd + bid / kNumXcd;
  if (t >= total) return false;
  const int width = kGroupM * tiles_n;
  const int first = (t / width) * kGroupM;
  const int gsize = min(tiles_m - first, kGroupM);
  const int rem = t % width;
  tm = first + rem % gsize;
  tn = rem / gsize;
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

// c += a * b on one 16 x 16 x 32 bf16 block, accumulating in place in AGPRs.
// Written as inline asm with the accumulator tied in/out: through the builtin,
// the register allocator is free to give the result a different AGPR quadruple
// than the addend, and with all 256 AGPRs live it then rotates accumulators
// through VGPRs with accvgpr read/write/mov copies on every loop trip (each of
// which waits for the MFMA producing it).  The compiler's hazard tracking does
// not see inline asm as an MFMA, so the kernel pads the MFMA -> VALU hazard
// itself before its epilogue reads the accumulators (mfma_drain below); inside
// the loop no instruction reads an accumulator within 64 MFMAs of its write.
__device__ __forceinline__ void mfma_16x16x32(f32x4& c, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
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
template <class Epi>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void gemm_nt_kernel(GemmShape g, Epi epi) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kLdsBytes];

  int M = g.M, N = g.N, K = g.K;
  if (g.dyn != nullptr) {
    const int v = max(__builtin_amdgcn_readfirstlane(*g.dyn), 0);
    if (g.dyn_dim == kDynM) M = min(M, v);
    else if (g.dyn_dim == kDynN) N = min(N, v);
    else if (g.dyn_dim == kDynK) K = min(K, (v + kTileK - 1) / kTileK * kTileK);
  }
  int tm, tn;
  if (!map_tile(g.tiles_m, g.tiles_n, M, N, tm, tn)) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  // Direct-to-LDS loads: instruction q (0..3) of operand o writes 1 KB = rows
  // wave*64 + q*16 + lane/4 of the stage, physical chunk lane%4, holding the
  // logical chunk (lane%4) ^ swizzle(row) of that row's 64-byte K slice.
  const unsigned char* src[2][4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int row = wave * 64 + q * 16 + (lane >> 2);
    const int chunk = (lane & 3) ^ chunk_swizzle(row);
    const int ra = min(tm * kTileM + row, M - 1);
    int rb = min(tn * kTileN + row, N - 1);
    if (g.b_rows != nullptr) rb = g.b_rows[rb];
    src[0][q] = reinterpret_cast<const unsigned char*>(g.A) + (int64_t)ra * (g.a_kb ? kTileK : g.lda) * 2 + chunk * 16;
    src[1][q] = reinterpret_cast<const unsigned char*>(g.B) + (int64_t)rb * (g.b_kb ? kTileK : g.ldb) * 2 + chunk * 16;
  }
  // bytes from one K step of an operand to the next
  const int64_t kstep_a = (g.a_kb ? g.lda : kTileK) * 2, kstep_b = (g.b_kb ? g.ldb : kTileK) * 2;
  const int wave_lds = wave * 64 * kLdsRow;

  // MFMA operand reads: block i of A is rows wm*128 + i*16 + lane%16, K chunk
  // lane/16 (8 bf16 of the 32-deep step).  The swizzle of row r + 16 i equals
  // that of row r, so block i is the lane's base plus i * 16 rows.
  const int ra0 = wm * 128 + (lane & 15), rb0 = wn * 128 + (lane & 15);
  const int rdA = ra0 * kLdsRow + (((lane >> 4) ^ chunk_swizzle(ra0)) << 4);
  const int rdB = kLdsOperand + rb0 * kLdsRow + (((lane >> 4) ^ chunk_swizzle(rb0)) << 4);

  bf16x8 fa[2][kBlocks], fb[2][kBlocks];
  AccTile acc;
#pragma unroll
  for (int i = 0; i < kBlocks; ++i)
#pragma unroll
    for (int j = 0; j < kBlocks; ++j) acc.c[i][j] = f32x4{};

  const int nk = K / kTileK;

  // Operand n (0..15) of a step, in the order the MFMAs consume them:
  // A0, B0..B7, A1..A7.
  auto read_frag = [&](int stage, auto slot, auto n) {
    constexpr int s = decltype(slot)::value, q = decltype(n)::value;
    const unsigned char* base = lds + stage * kLdsStage;
    if constexpr (q == 0) {
      fa[s][0] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(base + rdA));
    } else if constexpr (q <= 8) {
      fb[s][q - 1] =
          __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(base + rdB + (q - 1) * 16 * kLdsRow));
    } else {
      fa[s][q - 8] =
          __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(base + rdA + (q - 8) * 16 * kLdsRow));
    }
  };
  // MFMA group q (0..15): blocks (q/2, 4*(q%2) .. 4*(q%2)+3).
  auto mfma_group = [&](auto slot, auto q) {
    constexpr int s = decltype(slot)::value;
    constexpr int i = decltype(q)::value / 2, j = 4 * (decltype(q)::value % 2);
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      mfma_16x16x32(acc.c[i][j + jj], fa[s][i], fb[s][j + jj]);
  };
  // Load instruction q (0..7) of a step: operand q/4, 16-row group q%4.
  auto issue_load = [&](int kt, int stage, auto q) {
    constexpr int o = decltype(q)::value / 4, r = decltype(q)::value % 4;
    const int64_t koff = (int64_t)max(min(kt, nk - 1), 0) * (o == 0 ? kstep_a : kstep_b);
    __builtin_amdgcn_global_load_lds(src[o][r] + koff,
                                     (lds_void*)(lds + stage * kLdsStage + wave_lds + o * kLdsOperand +
                                                 r * 16 * kLdsRow),
                                     16, 0, 0);
  };
  auto issue_loads = [&](int kt, int stage) {
    issue_load(kt, stage, Const<0>{}); issue_load(kt, stage, Const<1>{});
    issue_load(kt, stage, Const<2>{}); issue_load(kt, stage, Const<3>{});
    issue_load(kt, stage, Const<4>{}); issue_load(kt, stage, Const<5>{});
    issue_load(kt, stage, Const<6>{}); issue_load(kt, stage, Const<7>{});
  };
  // Group q of a step: 4 MFMAs on `slot`; the next step's 16 operands are read
  // two per group in groups 0..7 (the last one 32 MFMAs before it is needed)
  // and the 8 loads of step kt+kStages-1 go one per group in groups 8..15.
  auto group = [&](auto slot, int next_stage, int kt_load, int refill, auto q) {
    constexpr int n = decltype(q)::value;
    constexpr int other = 1 - decltype(slot)::value;
    mfma_group(slot, q);
    if constexpr (n < 8) {
      read_frag(next_stage, Const<other>{}, Const<2 * n>{});
      read_frag(next_stage, Const<other>{}, Const<2 * n + 1>{});
    } else {
      issue_load(kt_load, refill, Const<n - 8>{});
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  auto step = [&](auto slot, int kt) {
    const int next_stage = (kt + 1) % kStages;
    const int refill = (kt + kStages - 1) % kStages;  // the stage step kt-1 used
    const int kl = kt + kStages - 1;
    group(slot, next_stage, kl, refill, Const<0>{}); group(slot, next_stage, kl, refill, Const<1>{});
    group(slot, next_stage, kl, refill, Const<2>{}); group(slot, next_stage, kl, refill, Const<3>{});
    group(slot, next_stage, kl, refill, Const<4>{}); group(slot, next_stage, kl, refill, Const<5>{});
    group(slot, next_stage, kl, refill, Const<6>{}); group(slot, next_stage, kl, refill, Const<7>{});
    group(slot, next_stage, kl, refill, Const<8>{}); group(slot, next_stage, kl, refill, Const<9>{});
    group(slot, next_stage, kl, refill, Const<10>{}); group(slot, next_stage, kl, refill, Const<11>{});
    group(slot, next_stage, kl, refill, Const<12>{}); group(slot, next_stage, kl, refill, Const<13>{});
    group(slot, next_stage, kl, refill, Const<14>{}); group(slot, next_stage, kl, refill, Const<15>{});
    stage_barrier<(kStages - 3) * 8>();
  };

  // prologue: steps 0 .. kStages-2 in flight; step 0 visible, its operands in
  // slot 0; then step 1 visible (read during step 0).  With nk == 0 (a
  // device-side K bound of 0) the loads and reads still happen, at K offset 0,
  // but no MFMA consumes them and the accumulators stay zero.
  for (int s = 0; s < kStages - 1; ++s) issue_loads(s, s);
  stage_barrier<(kStages - 2) * 8>();
  read_frag(0, Const<0>{}, Const<0>{}); read_frag(0, Const<0>{}, Const<1>{});
  read_frag(0, Const<0>{}, Const<2>{}); read_frag(0, Const<0>{}, Const<3>{});
  read_frag(0, Const<0>{}, Const<4>{}); read_frag(0, Const<0>{}, Const<5>{});
  read_frag(0, Const<0>{}, Const<6>{}); read_frag(0, Const<0>{}, Const<7>{});
  read_frag(0, Const<0>{}, Const<8>{}); read_frag(0, Const<0>{}, Const<9>{});
  read_frag(0, Const<0>{}, Const<10>{}); read_frag(0, Const<0>{}, Const<11>{});
  read_frag(0, Const<0>{}, Const<12>{}); read_frag(0, Const<0>{}, Const<13>{});
  read_frag(0, Const<0>{}, Const<14>{}); read_frag(0, Const<0>{}, Const<15>{});
  stage_barrier<(kStages - 3) * 8>();

  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    step(Const<0>{}, kt);
    step(Const<1>{}, kt + 1);
  }
  if (kt < nk) step(Const<0>{}, kt);

  // drain the (clamped, unused) loads still in flight before LDS is reused
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  mfma_drain();
  __syncthreads();

  epi.apply(acc, tm, tn, wm, wn, lane, reinterpret_cast<float*>(lds));
}

}  // namespace pspo
