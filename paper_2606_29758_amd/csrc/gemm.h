// Tiled bf16 x bf16 -> fp32 matrix-core (MFMA) product for CDNA4 (gfx950),
// with a pluggable epilogue.  Every contraction of the LM-head loss is one of
// these "NT" products:
//
//   C[m][n] = sum_k A[m][k] * B[n][k],  A: [M x K], B: [N x K], both row-major
//   with K contiguous (row strides lda / ldb in elements), K % 32 == 0.
//
// Tiling: a 256-thread work-group (4 wave64s in a 2 x 2 arrangement) owns a
// 256 x 256 C tile; each wave owns 128 x 128 = 4 x 4 blocks of the
// v_mfma_f32_32x32x16_bf16 instruction, i.e. 256 fp32 accumulators per lane
// (the whole AGPR file).
//
// Pipeline: K advances in steps of 32 through a ring of kStages LDS stages
// (32 KB each: 256 rows x 64 bytes of A and of B).  Operands go from global
// memory straight into LDS (global_load_lds_dwordx4: no staging registers, no
// LDS-write instructions); each wave loads 64 rows of A and 64 rows of B per
// step.  Step kt:
//   1. sub-step 0: 16 MFMAs on register slot 0 while the sub-step-1 operands
//      of stage kt are read into slot 1;
//   2. wait for this wave's loads of step kt+1, then one work-group barrier:
//      step kt+1 is now visible and every wave is done with step kt-1;
//   3. sub-step 1: 16 MFMAs on slot 1 while the loads of step kt+kStages-1 go
//      into the stage step kt-1 used and the sub-step-0 operands of step kt+1
//      are read into slot 0.
// A load therefore has kStages-2 steps (about 1000 MFMA cycles each) to land.
// Each phase is written as groups of two MFMAs and one or two memory ops,
// fenced with sched_barrier so the compiler keeps the interleave.
// LDS rows are 64 bytes; the four 16-byte chunks of row r are stored XOR-ed
// with ((r>>1) ^ (r>>2)) & 3, so the operand reads of consecutive rows hit
// distinct banks.
//
// Rows past M (or N) are clamped to the last valid row when loading; the
// epilogue masks them.  Work-group -> tile mapping is XCD-aware: work-groups
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

__device__ __forceinline__ int chunk_swizzle(int row) { return ((row >> 1) ^ (row >> 2)) & 3; }

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

template <int N>
struct Const {
  static constexpr int value = N;
};

// Scheduling-group masks of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedMfma = 0x008, kSchedVmemRead = 0x020, kSchedDsRead = 0x100;

typedef __attribute__((address_space(3))) void lds_void;

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
// overwritten); smem is the
// (no longer needed) LDS ring, 160 KB, free for reductions: every load into
// it has landed and all waves have passed a barrier before the call.
template <class Epi>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void gemm_nt_kernel(GemmShape g, Epi epi) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kLdsBytes];

  int tm, tn;
  if (!map_tile(g, tm, tn)) return;

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
    const int ra = min(tm * kTileM + row, g.M - 1);
    const int rb = min(tn * kTileN + row, g.N - 1);
    src[0][q] = reinterpret_cast<const unsigned char*>(g.A) + (int64_t)ra * g.lda * 2 + chunk * 16;
    src[1][q] = reinterpret_cast<const unsigned char*>(g.B) + (int64_t)rb * g.ldb * 2 + chunk * 16;
  }
  const int wave_lds = wave * 64 * kLdsRow;

  // MFMA operand reads: block i of A is row wm*128 + i*32 + lane%32; sub-step kk
  // reads logical chunk kk*2 + lane/32.
  int rdA[2][4], rdB[2][4];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ra = wm * 128 + i * 32 + (lane & 31);
      const int rb = wn * 128 + i * 32 + (lane & 31);
      const int c = kk * 2 + (lane >> 5);
      rdA[kk][i] = ra * kLdsRow + ((c ^ chunk_swizzle(ra)) << 4);
      rdB[kk][i] = kLdsOperand + rb * kLdsRow + ((c ^ chunk_swizzle(rb)) << 4);
    }

  bf16x8 fa[2][4], fb[2][4];
  AccTile acc;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc.c[i][j] = f32x16{};

  const int nk = g.K / kTileK;

  // Operand q (0..7) of a sub-step, in the order the MFMAs consume them:
  // A0, B0, B1, B2, B3, A1, A2, A3.
  auto read_frag = [&](int stage, auto kk, auto slot, auto q) {
    constexpr int k = decltype(kk)::value;
    constexpr int s = decltype(slot)::value;
    constexpr int n = decltype(q)::value;
    const unsigned char* base = lds + stage * kLdsStage;
    if constexpr (n == 0) {
      fa[s][0] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(base + rdA[k][0]));
    } else if constexpr (n <= 4) {
      fb[s][n - 1] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(base + rdB[k][n - 1]));
    } else {
      fa[s][n - 4] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(base + rdA[k][n - 4]));
    }
  };
  // MFMA pair q (0..7) of a sub-step: blocks (q/2, 2*(q%2)) and (q/2, 2*(q%2)+1).
  auto mfma_pair = [&](auto slot, auto q) {
    constexpr int s = decltype(slot)::value;
    constexpr int i = decltype(q)::value / 2, j = 2 * (decltype(q)::value % 2);
    acc.c[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s][i], fb[s][j], acc.c[i][j], 0, 0, 0);
    acc.c[i][j + 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s][i], fb[s][j + 1], acc.c[i][j + 1], 0, 0, 0);
  };
  // Load instruction q (0..7) of a step: operand q/4, 16-row group q%4.
  auto issue_load = [&](int kt, int stage, auto q) {
    constexpr int o = decltype(q)::value / 4, r = decltype(q)::value % 4;
    const int64_t koff = (int64_t)min(kt, nk - 1) * (kTileK * 2);
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
  auto read_all = [&](int stage, auto kk, auto slot) {
    read_frag(stage, kk, slot, Const<0>{}); read_frag(stage, kk, slot, Const<1>{});
    read_frag(stage, kk, slot, Const<2>{}); read_frag(stage, kk, slot, Const<3>{});
    read_frag(stage, kk, slot, Const<4>{}); read_frag(stage, kk, slot, Const<5>{});
    read_frag(stage, kk, slot, Const<6>{}); read_frag(stage, kk, slot, Const<7>{});
  };
  // Operand reads of one sub-step spread over MFMA groups 0..5 (two in groups
  // 0 and 1), so the last read is issued four MFMAs before the next sub-step
  // needs its operands.
  auto reads_of_group = [&](int stage, auto kk, auto slot, auto q) {
    constexpr int n = decltype(q)::value;
    if constexpr (n < 2) {
      read_frag(stage, kk, slot, Const<2 * n>{});
      read_frag(stage, kk, slot, Const<2 * n + 1>{});
    } else if constexpr (n < 6) {
      read_frag(stage, kk, slot, Const<n + 2>{});
    }
  };
  // Sub-step 0 of stage `cur` (operands in slot 0) while the slot-1 operands of
  // sub-step 1 are read: 8 groups of 2 MFMAs, fenced so the compiler keeps the
  // interleave.
  auto phase_a = [&](int cur, auto q) {
    mfma_pair(Const<0>{}, q);
    reads_of_group(cur, Const<1>{}, Const<1>{}, q);
    __builtin_amdgcn_sched_barrier(0);
  };
  // Sub-step 1 (slot 1) while step kt+kStages-1 is loaded and the slot-0
  // operands of the next stage are read: 8 groups of {2 MFMA, 1 load, reads}.
  auto phase_b = [&](int kt_load, int refill, int next, auto q) {
    mfma_pair(Const<1>{}, q);
    issue_load(kt_load, refill, q);
    reads_of_group(next, Const<0>{}, Const<0>{}, q);
    __builtin_amdgcn_sched_barrier(0);
  };

  auto run_phase_a = [&](int cur) {
    phase_a(cur, Const<0>{}); phase_a(cur, Const<1>{}); phase_a(cur, Const<2>{}); phase_a(cur, Const<3>{});
    phase_a(cur, Const<4>{}); phase_a(cur, Const<5>{}); phase_a(cur, Const<6>{}); phase_a(cur, Const<7>{});
    // this wave's loads of the next step have landed and its LDS reads are done;
    // after the barrier every wave's have (the loads of later steps stay in flight)
    stage_barrier<(kStages - 3) * 8>();
  };

  auto run_phase_b = [&](int kt) {
    const int next = (kt + 1) % kStages;
    const int refill = (kt + kStages - 1) % kStages;  // the stage step kt-1 used
    const int kl = kt + kStages - 1;
    phase_b(kl, refill, next, Const<0>{}); phase_b(kl, refill, next, Const<1>{});
    phase_b(kl, refill, next, Const<2>{}); phase_b(kl, refill, next, Const<3>{});
    phase_b(kl, refill, next, Const<4>{}); phase_b(kl, refill, next, Const<5>{});
    phase_b(kl, refill, next, Const<6>{}); phase_b(kl, refill, next, Const<7>{});
  };

  // prologue: steps 0 .. kStages-2 in flight, step 0 visible, sub-step 0 of step 0
  for (int s = 0; s < kStages - 1; ++s) issue_loads(s, s);
  stage_barrier<(kStages - 2) * 8>();
  read_all(0, Const<0>{}, Const<0>{});
  run_phase_a(0);

  // Iteration kt: sub-step 1 of step kt (loads of step kt+kStages-1 and the
  // slot-0 operands of step kt+1 issued alongside), then sub-step 0 of step kt+1.
  for (int kt = 0; kt + 1 < nk; ++kt) {
    run_phase_b(kt);
    run_phase_a((kt + 1) % kStages);
  }
  run_phase_b(nk - 1);
  // drain the (clamped, unused) loads still in flight before LDS is reused
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  epi.apply(acc, tm, tn, wm, wn, lane, reinterpret_cast<float*>(lds));
}

}  // namespace pspo
