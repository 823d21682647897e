// Fused LM-head + prefix-weighted PPO loss, forward and backward, on the
// matrix cores of gfx950.
//
// Per packed token i (PS-PPO Sec. 3.1 PPO objective, Sec. 3.2/3.3 truncated
// estimator, App. D LM-head score):
//   z_i = W h_i,  l_i = z_{i,o_i} - lse(z_i),  rho_i = exp(l_i - lold_i),
//   s_i = min(rho_i A, clip(rho_i) A),  loss = -scale * sum_i c_i s_i,
//   delta_i = -scale c_i mu_i rho_i A,  G_i = delta_i (e_{o_i} - softmax(z_i)),
//   dH_i = G_i W,  dW = sum_i G_i^T h_i.
//
// Schedule (the [N, V] logits never reach memory):
//   1. K-blocked bf16 copies of W (with, per vocabulary chunk, W[chunk]^T) and
//      of the hidden rows of the tokens whose logits are needed (the operand
//      layout of the matrix-core products);
//   2. forward product z^T = W H^T in 384 x 256 tiles; the epilogue reduces
//      each tile column (one token) to a partial (max, sum exp) over the tile's
//      384 vocabulary rows; the target logits come from a one-wave-per-row
//      dot product W[o] . h;
//   3. finalize: merge the partials into lse, then l, rho, the clip mask, delta
//      and a deterministic float64 loss reduction;
//   4. K-blocked copies of the backward tokens' hidden rows and of their
//      transpose H^T [d x Npad] (K-contiguous operands of the gradient
//      products);
//   5. per vocabulary chunk of Vc rows: the bf16 logit gradient without its
//      target entries, Delta_{i,v} = -delta_i exp(z_{i,v} - lse_i) for
//      v != o_i (0 at v = o_i), recomputed tile by tile on the matrix cores and
//      stored in both layouts ([Npad x Vc] and [Vc x Npad]); then
//      dW[chunk] = Delta^T H and dH += Delta W[chunk] as two more matrix-core
//      products.  With PSPO_KEEP_LOGITS the forward keeps the first chunk's
//      logits (fp16 offsets from each tile's per-column maximum) and a
//      memory-bound conversion replaces that chunk's recompute;
//   6. the target entries in float32, g_i = G_{i,o_i} = delta_i (1 - p_i(o_i))
//      = -delta_i expm1(l_i): dH_i += g_i W[o_i], and
//      dW[v] += sum_{i : o_i = v} g_i h_i with each row's terms summed in token
//      order (a stable bucketing of the backward tokens by target; no
//      floating-point atomics).  The target entry is the largest of its row
//      when the softmax is flat and the result of a cancellation when it is
//      peaked; carried in float32 it is rounded neither to 8 bits nor after a
//      cancellation.
#include <algorithm>
#include <cmath>

#include "common.h"
#include "gemm.h"
#include "layout.h"
#include "rowdot.h"

namespace pspo {
namespace {

constexpr float kNegInf = -INFINITY;

// ---------------------------------------------------------------------------
// Epilogues
// ---------------------------------------------------------------------------

// An off-target entry of the logit gradient delta (1[v = o] - exp(z - lse))
// (the objective of Sec. 3.1 differentiated through the log-softmax of App. D)
// is -delta exp(z - lse).  Its magnitude is computed as exp2(z log2(e) + c)
// with the per-column constant c = log2|delta| - lse log2(e): one fma and one
// exp per entry (c = -inf for a padding column, whose delta is 0, gives 0);
// its sign, that of -delta, is applied to packed bf16 pairs by XOR.  The
// target entries are then overwritten with 0 (zero_targets_kernel): they are
// added in float32 by the target-entry kernels.  The recomputing product and
// the kept-logit conversion both use these, so they produce the same bits.
__device__ __forceinline__ float grad_col_const(float lse, float delta) {
  return delta != 0.f ? fmaf(-lse, kLog2e, log2f(fabsf(delta))) : -INFINITY;
}
__device__ __forceinline__ uint32_t grad_sign_bits(float delta) { return delta > 0.f ? 0x80008000u : 0u; }
__device__ __forceinline__ float grad_mag(float z, float c) { return __builtin_amdgcn_exp2f(fmaf(z, kLog2e, c)); }

// Two floats as packed bf16 (round to nearest even): one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// Two floats as packed fp16 (round to nearest even), and one fp16 back.
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, f16x2));
}
__device__ __forceinline__ float f16_bits_to_f32(uint32_t bits) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(bits & 0xFFFFu));
}

// A forward tile's logits kept for the first backward chunk, as fp16 offsets
// from the tile's per-column maximum M (the value the forward writes to its
// partial maxima, taken here from the same two wave maxima in `red`):
// [24 blocks of 16 rows][256 columns][16 rows] fp16 at `base`.  The lane's 4
// rows of accumulator block (i, j) are one 8-byte piece, so each store
// instruction writes 512 contiguous bytes (whole 128-byte lines).  Every kept
// value is <= 0 and the large softmax entries sit near 0, where fp16 holds an
// offset to ~2^-11 relative: the logit gradient rebuilt from it stays far
// inside the bf16 rounding the gradient gets anyway, at half the bytes of the
// fp32 logits.
__device__ __forceinline__ void store_kept_f16(const AccTile& acc, const float* red, uint16_t* base, int wm, int wn,
                                               int lane) {
  unsigned char* zb = reinterpret_cast<unsigned char*>(base);
  float M[kBlocksN];
#pragma unroll
  for (int j = 0; j < kBlocksN; ++j) {
    const int cl = acc_col(wn, j, lane);
    M[j] = fmaxf(red[cl * 2], red[(kTileN + cl) * 2]);
  }
  const uint32_t lo = (uint32_t)(wm * (kWaveM / 16)) * (kTileN * 32u) + (uint32_t)(wn * kWaveN + (lane & 15)) * 32u +
                      (uint32_t)(lane >> 4) * 8u;
#pragma unroll
  for (int i = 0; i < kBlocksM; ++i) {
#pragma unroll
    for (int j = 0; j < kBlocksN; ++j) {
      float x[kAccPerBlock];
#pragma unroll
      for (int r = 0; r < kAccPerBlock; ++r) {
        if (i < kBlocksAgpr)
          asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(x[r]) : "a"(acc.a[i][j][r]));
        else
          x[r] = acc.v[i - kBlocksAgpr][j][r];
      }
      u32x2 h;
      h.x = pack_f16x2(x[0] - M[j], x[1] - M[j]);
      h.y = pack_f16x2(x[2] - M[j], x[3] - M[j]);
      __builtin_nontemporal_store(h, reinterpret_cast<u32x2*>(zb + (lo + (uint32_t)(i * kTileN * 32 + j * 512))));
    }
    __builtin_amdgcn_sched_barrier(0);   // one row block's stores at a time
  }
}

// Forward: rows = vocabulary (A = W), columns = the tokens whose logits are
// needed (B = their hidden rows, gathered; column t is token tok[t]); writes
// per-column softmax partials of each 384-row vocabulary tile.  (The target
// logits come from row_dots_kernel: picking one accumulator per column out
// of the 48 a lane holds costs a compare and a select for each of them.)
// kFull: every row of every tile is a token id (no per-row mask); otherwise
// the launch is the partial last vocabulary tile, tm0 its index (the product's
// row tile 0).  Two instantiations rather than a branch in one: with a branch
// the compiler spills accumulators.
template <bool kFull>
struct EpiForward {
  int V, N;
  int64_t ldp;  // stride between vocabulary tiles in the partial arrays (= Npad)
  int tm0;
  float* part_m;
  float* part_l;
  const int32_t* n_dev;
  uint16_t* zk;          // kept fp16 logit offsets of vocabulary tiles tm < kept_tiles, or NULL:
  int kept_tiles;        //   per tile (tm, tn) a block at (tm * kept_cols + tn) * 384 * 256
  int kept_cols;         //   (store_kept_f16)

  __device__ __forceinline__ void apply(const AccTile& acc, int tm_launch, int tn, int wm, int wn, int lane,
                                        float* smem) const {
    float* red = smem;  // [2 wave rows][256 columns][m, l]
    const int tm = kFull ? tm_launch : tm0 + tm_launch;
    const int n = min(N, __builtin_amdgcn_readfirstlane(*n_dev));
    const int vbase = tm * kTileM + acc_row(wm, 0, 0, lane);   // this lane's rows: vbase + i*16 + r
#pragma unroll
    for (int j = 0; j < kBlocksN; ++j) {
      const int cl = acc_col(wn, j, lane);
      // the lane's 48 values of column j (q = 4 i + r: row vbase + 16 i + r),
      // the AGPR ones read once into VGPRs for both passes below
      float xs[kBlocksM * kAccPerBlock];
#pragma unroll
      for (int q = 0; q < kBlocksM * kAccPerBlock; ++q) {
        if ((q >> 2) < kBlocksAgpr)
          asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(xs[q]) : "a"(acc.a[q >> 2][j][q & 3]));
        else
          xs[q] = acc.v[(q >> 2) - kBlocksAgpr][j][q & 3];
      }
      auto x = [&](int q) { return xs[q]; };
      float m, l;
      if constexpr (kFull) {
        // every row is a token id: three-input maxima (no per-value select),
        // exp2(z log2e - m log2e) as one fma + exp, four partial sums
        float mm[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) mm[k] = max3(x(k), x(k + 4), x(k + 8));
#pragma unroll
        for (int q = 12; q < kBlocksM * kAccPerBlock; q += 8)
#pragma unroll
          for (int k = 0; k < 4; ++k) mm[k] = max3(mm[k], x(q + k), x(q + k + 4));
        m = max3(mm[0], mm[1], max3(mm[2], mm[3], mm[3]));
        m = fmaxf(m, __shfl_xor(m, 16));
        m = fmaxf(m, __shfl_xor(m, 32));
        const float mb = m * kLog2e;
        float ls[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < kBlocksM * kAccPerBlock; ++q) ls[q & 3] += __builtin_amdgcn_exp2f(fmaf(x(q), kLog2e, -mb));
        l = (ls[0] + ls[1]) + (ls[2] + ls[3]);
      } else {
        m = kNegInf;
#pragma unroll
        for (int i = 0; i < kBlocksM; ++i)
#pragma unroll
          for (int r = 0; r < kAccPerBlock; ++r)
            if (vbase + i * 16 + r < V) m = fmaxf(m, x(i * kAccPerBlock + r));
        m = fmaxf(m, __shfl_xor(m, 16));
        m = fmaxf(m, __shfl_xor(m, 32));
        l = 0.f;
        if (m != kNegInf) {
          const float mb = m * kLog2e;
#pragma unroll
          for (int i = 0; i < kBlocksM; ++i)
#pragma unroll
            for (int r = 0; r < kAccPerBlock; ++r)
              if (vbase + i * 16 + r < V) l += __builtin_amdgcn_exp2f(fmaf(x(i * kAccPerBlock + r), kLog2e, -mb));
        }
      }
      l += __shfl_xor(l, 16);
      l += __shfl_xor(l, 32);
      if (lane < 16) {
        red[(wm * kTileN + cl) * 2 + 0] = m;
        red[(wm * kTileN + cl) * 2 + 1] = l;
      }
    }
    __syncthreads();
    const int c = threadIdx.x;
    const float m0 = red[c * 2], l0 = red[c * 2 + 1];
    const float m1 = red[(kTileN + c) * 2], l1 = red[(kTileN + c) * 2 + 1];
    const float M = fmaxf(m0, m1);
    float L = 0.f;
    if (m0 != kNegInf) L += l0 * __expf(m0 - M);
    if (m1 != kNegInf) L += l1 * __expf(m1 - M);
    const int t = tn * kTileN + c;
    if (t < n) {
      part_m[tm * ldp + t] = M;
      part_l[tm * ldp + t] = L;
    }
    if (zk != nullptr && tm < kept_tiles)   // the tile's logits, kept for the first backward chunk
      store_kept_f16(acc, red, zk + ((int64_t)tm * kept_cols + tn) * (kTileM * kTileN), wm, wn, lane);
  }
};

// Lane exchanges (all lanes active): DPP inside a quad (lane l ^ 1, l ^ 2) and
// inside a 16-lane row (the value of lane l + 4 / l - 4).  A lane whose source
// lies outside its row reads 0 (bound_ctrl), so no destination needs an
// initial value (with an explicit "old" operand of 0 the compiler zeroes a
// register before every move); callers use only lanes with a valid source.
__device__ __forceinline__ uint32_t quad_xor1(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, true);
}
__device__ __forceinline__ uint32_t quad_xor2(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, true);
}
__device__ __forceinline__ uint32_t row_from_plus4(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x104, 0xF, 0xF, true);   // row_shl:4
}
__device__ __forceinline__ uint32_t row_from_minus4(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x114, 0xF, 0xF, true);   // row_shr:4
}

// 4 x 4 transpose of bf16 pairs inside a quad of lanes: lane k holds rows 0..3 of
// token k as (r0 | r1 << 16, r2 | r3 << 16) and receives row k of tokens 0..3.
__device__ __forceinline__ u32x2 quad_transpose(u32x2 p, int k) {
  const bool lo2 = k < 2;
  const uint32_t r1 = quad_xor2(lo2 ? p.y : p.x);
  const uint32_t qa = lo2 ? p.x : r1, qb = lo2 ? r1 : p.y;   // tokens k%2 and k%2+2, rows 2(k/2), +1
  // 16-bit halves picked by lane parity with v_perm_b32 (byte selectors 0-3
  // take bytes of the second operand, 4-7 of the first): one instruction per
  // word instead of a select between two shift/mask pairs, which the compiler
  // turns into a divergent branch
  const bool even = (k & 1) == 0;
  const uint32_t r2 = quad_xor1(__builtin_amdgcn_perm(qb, qa, even ? 0x07060302u : 0x05040100u));
  u32x2 o;
  o.x = __builtin_amdgcn_perm(r2, qa, even ? 0x05040100u : 0x03020504u);
  o.y = __builtin_amdgcn_perm(r2, qb, even ? 0x07060100u : 0x03020706u);
  return o;
}

// Backward logit gradient (its target entries zeroed afterwards) for one vocabulary chunk:
// rows = vocabulary rows v0 + vl (A = W[v0:]), columns = the compacted tokens
// that carry gradient (column t < *n_dev).  Writes bf16 Delta in both K-blocked
// layouts (vocabulary rows for dW, token rows for dH); zero outside t < *n_dev,
// v < V.  Straight from registers, as 16-byte stores of which each instruction
// fills 16 whole 64-byte K rows (1 KB contiguous).  Blocks are taken two row
// blocks x two column blocks at a time:
//   * token-major: a lane's 4 rows of a block are 4 consecutive K entries of
//     its token; swapping 16-lane rows (v_permlane16_swap) between the two row
//     blocks gives each lane 8 consecutive K entries;
//   * vocabulary-major: a 4 x 4 transpose inside each quad of lanes gives a
//     lane 4 consecutive tokens of one row; exchanging with the quad 4 lanes
//     away (DPP row shift) between the two column blocks gives it 8.
// kFull: every row of every tile is a token id (no per-row mask; the only kind
// when V is a multiple of 384); otherwise the launch is the partial last
// vocabulary tile, tm0 its chunk row tile (the product's row tile 0).
template <bool kFull>
struct EpiDelta {
  int V, N, v0, tm0;
  // Both layouts row-blocked, so that each tile's values sit in a compact
  // region (the vocabulary-major one a contiguous 192 KB block):
  uint16_t* dT;          // [Vc/384][tkb][384][32]: rows = vocabulary entries (block = vocabulary tile), K = tokens
  int64_t tkb;           //   token K blocks per vocabulary block (Npad / 32)
  uint16_t* dN;          // [Npad/768][nkb][768][32]: rows = tokens (block = 3 token tiles), K = vocabulary entries
  int64_t nkb;           //   vocabulary K blocks per token block (Vc / 32)
  const float* clse;     // lse and delta of column t (columns t < *n_dev), in column order
  const float* cdelta;
  const int32_t* n_dev;

  __device__ __forceinline__ void apply(AccTile& acc, int tm_launch, int tn, int wm, int wn, int lane, float*) const {
    const int n = min(N, __builtin_amdgcn_readfirstlane(*n_dev));
    const int tm = kFull ? tm_launch : tm0 + tm_launch;
    const int vl0 = tm * kTileM + acc_row(wm, 0, 0, lane);   // chunk rows of this lane: vl0 + i*16 + r
    [[maybe_unused]] const int vbase = v0 + vl0;   // (rows past V of a partial last tile are masked)
    // per-column token data of the lane's 8 columns, fetched together (one
    // round trip: the arrays are in column order)
    float cc[kBlocksN];
    uint32_t sg[kBlocksN];
#pragma unroll
    for (int j = 0; j < kBlocksN; ++j) {
      const int t = tn * kTileN + acc_col(wn, j, lane);
      const float dl = t < n ? cdelta[t] : 0.f;
      cc[j] = grad_col_const(t < n ? clse[t] : 0.f, dl);
      sg[j] = grad_sign_bits(dl);
    }
    // Store addresses: a per-tile base (uniform) plus a 32-bit byte offset per
    // lane and block group.  The tile's 12 K blocks of the token-major layout
    // are 16 KB pieces 48 KB apart in token block tn / 3, its 8 K blocks of the
    // vocabulary-major layout consecutive 24 KB pieces of vocabulary block tm.
    const int k = lane & 3, q = (lane >> 2) & 3, g = lane >> 4;
    const bool qeven = (q & 1) == 0;
    unsigned char* nbase = reinterpret_cast<unsigned char*>(
        dN + (((int64_t)(tn / 3) * nkb + tm * (kTileM / kTileK)) * kTileLcm + (tn % 3) * kTileN) * kTileK);
    unsigned char* tbase = reinterpret_cast<unsigned char*>(
        dT + ((int64_t)tm * tkb + tn * (kTileN / kTileK)) * (kTileM * kTileK));
    const uint32_t kstepN = kTileLcm * (kTileK * 2), kstepT = kTileM * (kTileK * 2);
    // token-major: after the row swap the lane holds K entries
    // 16 (g % 2) + 8 (g / 2) .. +7 of its token wn*128 + j*16 + lane%16
    const uint32_t noff = (uint32_t)(wm * (kWaveM / kTileK)) * kstepN +
                          (uint32_t)(wn * kWaveN + (lane & 15)) * (kTileK * 2) +
                          (uint32_t)((g & 1) * 16 + (g >> 1) * 8) * 2;
    // vocabulary-major: after the exchanges the lane holds row wm*192 + i*16 +
    // 4g + k, tokens 16 (q % 2) + 8 (q / 2) .. +7 of the column-block pair
    const uint32_t toff = (uint32_t)(wn * (kWaveN / kTileK)) * kstepT +
                          (uint32_t)(wm * kWaveM + g * 4 + k) * (kTileK * 2) +
                          (uint32_t)((q & 1) * 16 + (q >> 1) * 8) * 2;
#pragma unroll
    for (int jp = 0; jp < kBlocksN / 2; ++jp) {
#pragma unroll
      for (int ip = 0; ip < kBlocksM / 2; ++ip) {
        // Delta of the four blocks, packed as bf16 pairs: blk[ii][jj] = rows
        // 0,1 | rows 2,3 of row block 2 ip + ii, column block 2 jp + jj
        // (columns past n have delta 0: no branch per value).
        u32x2 blk[2][2];
#pragma unroll
        for (int ii = 0; ii < 2; ++ii)
#pragma unroll
          for (int jj = 0; jj < 2; ++jj) {
            const int i = 2 * ip + ii, j = 2 * jp + jj;
            float x[kAccPerBlock];
#pragma unroll
            for (int r = 0; r < kAccPerBlock; ++r) {
              x[r] = grad_mag(acc_get(acc, i, j, r), cc[j]);
              if constexpr (!kFull) x[r] = (vbase + i * 16 + r < V) ? x[r] : 0.f;
            }
            blk[ii][jj].x = pack_bf16x2(x[0], x[1]) ^ sg[j];
            blk[ii][jj].y = pack_bf16x2(x[2], x[3]) ^ sg[j];
          }
        // vocabulary-major stores, one per row block
#pragma unroll
        for (int ii = 0; ii < 2; ++ii) {
          const u32x2 t0 = quad_transpose(blk[ii][0], k), t1 = quad_transpose(blk[ii][1], k);
          const u32x2 send = qeven ? t1 : t0;
          // both shifts in every lane, then a select: written as a select of
          // two lane exchanges, the compiler may branch on the condition, and
          // a DPP move reads nothing from lanes its EXEC mask has switched off
          uint32_t px = row_from_plus4(send.x), mx = row_from_minus4(send.x);
          uint32_t py = row_from_plus4(send.y), my = row_from_minus4(send.y);
          asm volatile("" : "+v"(px), "+v"(mx), "+v"(py), "+v"(my));
          u32x2 recv;
          recv.x = qeven ? px : mx;
          recv.y = qeven ? py : my;
          u32x4 o;
          o.x = qeven ? t0.x : recv.x;
          o.y = qeven ? t0.y : recv.y;
          o.z = qeven ? recv.x : t1.x;
          o.w = qeven ? recv.y : t1.y;
          *reinterpret_cast<u32x4*>(tbase + (toff + (uint32_t)jp * kstepT +
                                             (uint32_t)((2 * ip + ii) * 16 * kTileK * 2))) = o;
        }
        // token-major stores, one per column block (after the vocabulary-major
        // ones: the in-place row swaps then consume the packed values without copies)
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const auto sx = __builtin_amdgcn_permlane16_swap(blk[0][jj].x, blk[1][jj].x, false, false);
          const auto sy = __builtin_amdgcn_permlane16_swap(blk[0][jj].y, blk[1][jj].y, false, false);
          u32x4 o;
          o.x = sx[0];
          o.y = sy[0];
          o.z = sx[1];
          o.w = sy[1];
          *reinterpret_cast<u32x4*>(nbase + (noff + (uint32_t)ip * kstepN +
                                             (uint32_t)((2 * jp + jj) * 16 * kTileK * 2))) = o;
        }
        __builtin_amdgcn_sched_barrier(0);   // one group's values live at a time
      }
    }
  }
};

// The logit gradient of the first vocabulary chunk from the forward's kept
// fp16 logit offsets (zk: per 384 x 256 forward tile (tm, tn) a block at
// (tm * kept_cols + tn) * 384 * 256, [24 blocks of 16 rows][256 columns][16];
// the logit is M + offset with M the tile's per-column maximum in part_m)
// instead of a recomputing product: the values and layouts the logit-gradient
// epilogue writes for that chunk.  Backward column a < n = min(N, *n_dev) has
// the lse and delta clse[a], cdelta[a] and its logits sit in
// forward column afwd[a]; columns n <= a < round_up(n, 32) are written as the
// zero gradient of a padding column (the dW product reads whole 32-token K
// steps); rows v >= V are zero.
// Grid (Vc / 128, Npad / 32), 256 threads: 32 backward tokens x 128 vocabulary
// entries per block; thread tid takes token tid % 32's 32-byte piece (16 rows)
// of 16-row block tid / 32, so 32 consecutive threads read the pieces of 32
// consecutive backward tokens; the gradient goes through LDS and out in both
// layouts as 16-byte stores of whole 64-byte K rows.
__global__ __launch_bounds__(256) void logit_grad_kept_kernel(const uint16_t* __restrict__ zk,
                                                              const float* __restrict__ part_m, int64_t ldp,
                                                              int kept_cols, int Vc, int V, int N,
                                                              const int32_t* __restrict__ n_dev,
                                                              const int32_t* __restrict__ afwd,
                                                              const float* __restrict__ clse,
                                                              const float* __restrict__ cdelta,
                                                              uint16_t* __restrict__ dN, int64_t nkb,
                                                              uint16_t* __restrict__ dT, int64_t tkb) {
  __shared__ uint16_t tile[32][128 + 8];   // [token][entry]; padded rows: the column reads hit distinct banks
  const int n = min(N, *n_dev);
  const int a0 = blockIdx.y * 32, v0 = blockIdx.x * 128;   // Vc is a multiple of 128
  if (a0 >= n) return;
  const int tid = threadIdx.x;
  const int al = tid & 31, a = a0 + al;
  const int vl = (tid >> 5) * 16, v = v0 + vl;   // this thread's 16 rows
  uint32_t w[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};   // 16 bf16 (zero for padding columns)
  if (a < n) {
    const int f = afwd[a];
    const int vt = v / kTileM;
    const uint16_t* src = zk + ((int64_t)vt * kept_cols + (f >> 8)) * (kTileM * kTileN) +
                          (((v - vt * kTileM) >> 4) * kTileN + (f & (kTileN - 1))) * 16;
    const u32x4 h0 = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src));
    const u32x4 h1 = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + 8));
    const float M = part_m[vt * ldp + f];
    const float c = grad_col_const(clse[a], cdelta[a]);   // as the recomputing epilogue takes it
    const uint32_t sgn = grad_sign_bits(cdelta[a]);
#pragma unroll
    for (int e2 = 0; e2 < 8; ++e2) {
      const uint32_t hb = e2 < 4 ? h0[e2] : h1[e2 - 4];
      float x[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int e = 2 * e2 + u;
        x[u] = grad_mag(M + f16_bits_to_f32(hb >> (16 * u)), c);
        if (v + e >= V) x[u] = 0.f;
      }
      w[e2] = pack_bf16x2(x[0], x[1]) ^ sgn;
    }
  }
  *reinterpret_cast<u32x4*>(&tile[al][vl]) = u32x4{w[0], w[1], w[2], w[3]};
  *reinterpret_cast<u32x4*>(&tile[al][vl + 8]) = u32x4{w[4], w[5], w[6], w[7]};
  __syncthreads();
  // token-major: token a0 + tid / 8, entries v0 + (tid % 8) * 16 .. +15
  // (the row-blocked layout of the recomputing epilogue: blocks of 768 tokens)
  {
    const int tl = tid >> 3, ol = (tid & 7) * 16, ov = v0 + ol, at = a0 + tl;
    uint16_t* pn = dN + (((int64_t)(at / kTileLcm) * nkb + (ov >> 5)) * kTileLcm + at % kTileLcm) * kTileK + (ov & 31);
    *reinterpret_cast<u32x4*>(pn) = *reinterpret_cast<const u32x4*>(&tile[tl][ol]);
    *reinterpret_cast<u32x4*>(pn + 8) = *reinterpret_cast<const u32x4*>(&tile[tl][ol + 8]);
  }
  // vocabulary-major: entry v0 + tid / 2 of tokens a0 + (tid % 2) * 16 .. +15
  // (blocks of 384 vocabulary entries)
  {
    const int ol = tid >> 1, ap = (tid & 1) * 16, vv = v0 + ol;
    uint32_t q[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      q[e] = (uint32_t)tile[ap + 2 * e][ol] | ((uint32_t)tile[ap + 2 * e + 1][ol] << 16);
    uint16_t* pt = dT + (((int64_t)(vv / kTileM) * tkb + (a0 >> 5)) * kTileM + vv % kTileM) * kTileK + ap;
    *reinterpret_cast<u32x4*>(pt) = u32x4{q[0], q[1], q[2], q[3]};
    *reinterpret_cast<u32x4*>(pt + 8) = u32x4{q[4], q[5], q[6], q[7]};
  }
}

// The target entries of one chunk's logit-gradient layouts (the columns whose
// target lies in vocabulary rows [v0, v0 + vc)) set to 0: those entries are
// applied in float32 by the target-entry kernels.  Backward column a <
// min(N, *n_dev); the row-blocked layouts of EpiDelta (token blocks of 768,
// vocabulary blocks of 384).
__global__ __launch_bounds__(256) void zero_targets_kernel(int N, const int32_t* __restrict__ n_dev,
                                                           const int32_t* __restrict__ ctgt, int v0, int vc,
                                                           uint16_t* __restrict__ dN, int64_t nkb,
                                                           uint16_t* __restrict__ dT, int64_t tkb) {
  const int n = min(N, *n_dev);
  for (int a = blockIdx.x * 256 + threadIdx.x; a < n; a += gridDim.x * 256) {
    const int vl = ctgt[a] - v0;
    if (vl < 0 || vl >= vc) continue;
    dN[(((int64_t)(a / kTileLcm) * nkb + (vl >> 5)) * kTileLcm + a % kTileLcm) * kTileK + (vl & 31)] = 0;
    dT[(((int64_t)(vl / kTileM) * tkb + (a >> 5)) * kTileM + vl % kTileM) * kTileK + (a & 31)] = 0;
  }
}

// dW rows v0 + vl (A = Delta^T), columns = hidden features (B = H^T).
// Addresses are a per-tile base plus 32-bit byte offsets (a tile spans
// 384 rows of dW).  In accumulate mode each column block's 48 old values are
// loaded, added and stored before the next block's loads (a compiler memory
// fence between the blocks): hoisting every load of the tile would need 384
// more registers.
struct EpiDW {
  int V, d, v0;
  float* dW;
  bool accumulate;

  __device__ __forceinline__ void apply(const AccTile& acc, int tm, int tn, int wm, int wn, int lane, float*) const {
    const int row0 = v0 + tm * kTileM;                   // first dW row of the tile
    const int lr = acc_row(wm, 0, 0, lane);              // this lane's tile rows: lr + i*16 + r
    unsigned char* base = reinterpret_cast<unsigned char*>(dW + (int64_t)row0 * d + tn * kTileN);
    const uint32_t ld = (uint32_t)d * 4;
    const uint32_t loff = (uint32_t)lr * ld + (uint32_t)acc_col(wn, 0, lane) * 4;
    const int cb = tn * kTileN + acc_col(wn, 0, lane);   // this lane's columns: cb + j*16
#pragma unroll
    for (int j = 0; j < kBlocksN; ++j) {
      const bool cv = cb + j * 16 < d;
      float old[kBlocksM][kAccPerBlock];
#pragma unroll
      for (int i = 0; i < kBlocksM; ++i)
#pragma unroll
        for (int r = 0; r < kAccPerBlock; ++r) {
          const bool ok = accumulate && cv && row0 + lr + i * 16 + r < V;
          const uint32_t off = loff + (uint32_t)(i * 16 + r) * ld + (uint32_t)j * 64;
          old[i][r] = ok ? *reinterpret_cast<const float*>(base + off) : 0.f;
        }
#pragma unroll
      for (int i = 0; i < kBlocksM; ++i)
#pragma unroll
        for (int r = 0; r < kAccPerBlock; ++r) {
          const uint32_t off = loff + (uint32_t)(i * 16 + r) * ld + (uint32_t)j * 64;
          if (cv && row0 + lr + i * 16 + r < V)
            *reinterpret_cast<float*>(base + off) = old[i][r] + acc_get(acc, i, j, r);
        }
      asm volatile("" ::: "memory");
    }
  }
};

// dH rows = compacted tokens (A = Delta), columns = hidden features
// (B = W^T[:, v0:]); row t is written to d_hidden row tok[t], t < *n_dev.
// After the first vocabulary chunk each row block's old values are loaded,
// added and stored before the next block's loads (see EpiDW).
struct EpiDH {
  int N, d;
  float* dH;
  bool first;
  const int32_t* tok;
  const int32_t* n_dev;

  __device__ __forceinline__ void apply(const AccTile& acc, int tm, int tn, int wm, int wn, int lane, float*) const {
    const int n = min(N, __builtin_amdgcn_readfirstlane(*n_dev));
    const int cb = tn * kTileN + acc_col(wn, 0, lane);   // this lane's columns: cb + j*16
#pragma unroll
    for (int i = 0; i < kBlocksM; ++i) {
      float* rows[kAccPerBlock];
#pragma unroll
      for (int r = 0; r < kAccPerBlock; ++r) {
        const int t = tm * kTileM + acc_row(wm, i, r, lane);
        rows[r] = t < n ? dH + (int64_t)tok[t] * d : nullptr;
      }
      float old[kAccPerBlock][kBlocksN];
#pragma unroll
      for (int r = 0; r < kAccPerBlock; ++r)
#pragma unroll
        for (int j = 0; j < kBlocksN; ++j)
          old[r][j] = (!first && rows[r] != nullptr && cb + j * 16 < d) ? rows[r][cb + j * 16] : 0.f;
#pragma unroll
      for (int r = 0; r < kAccPerBlock; ++r)
#pragma unroll
        for (int j = 0; j < kBlocksN; ++j)
          if (rows[r] != nullptr && cb + j * 16 < d) rows[r][cb + j * 16] = old[r][j] + acc_get(acc, i, j, r);
      asm volatile("" ::: "memory");
    }
  }
};

// ---------------------------------------------------------------------------
// Small kernels
// ---------------------------------------------------------------------------

__global__ void fill_f32_kernel(float* __restrict__ p, int64_t n, float v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

__global__ void fill_i32_kernel(int32_t* __restrict__ p, int64_t n, int32_t v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

constexpr int kFinThreads = 256;
constexpr int kCompactThreads = 256, kCompactPer = 8, kCompactSpan = kCompactThreads * kCompactPer;

// Order-preserving compaction of the tokens t < N with keep(t) in two
// launches over blocks of kCompactSpan consecutive tokens: the first counts
// each block's kept tokens; the second adds the counts of the blocks before
// it and scatters: idx[0 .. count) are the kept indices in increasing order,
// pos[t] (if pos is not NULL) is t's place in idx or -1, mapped[p] (if mapped
// is not NULL) is map[idx[p]]; the last block writes the count (and stats[4],
// if asked).
template <class Keep>
__global__ __launch_bounds__(kCompactThreads) void compact_count_kernel(int N, Keep keep, int32_t* __restrict__ cnt) {
  __shared__ int sh[kCompactThreads];
  const int base = blockIdx.x * kCompactSpan;
  int c = 0;
#pragma unroll
  for (int e = 0; e < kCompactPer; ++e) {
    const int t = base + e * kCompactThreads + threadIdx.x;
    c += (t < N && keep(t)) ? 1 : 0;
  }
  sh[threadIdx.x] = c;
  __syncthreads();
  for (int s = kCompactThreads / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) sh[threadIdx.x] += sh[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) cnt[blockIdx.x] = sh[0];
}

template <class Keep>
__global__ __launch_bounds__(kCompactThreads) void compact_scatter_kernel(int N, Keep keep,
                                                                          const int32_t* __restrict__ cnt,
                                                                          int32_t* __restrict__ idx,
                                                                          int32_t* __restrict__ pos,
                                                                          const int32_t* __restrict__ map,
                                                                          int32_t* __restrict__ mapped,
                                                                          int32_t* __restrict__ count,
                                                                          double* __restrict__ stats) {
  __shared__ int sh[kCompactThreads];
  // this block's offset: the kept tokens of the blocks before it
  int o = 0;
  for (int k = threadIdx.x; k < (int)blockIdx.x; k += kCompactThreads) o += cnt[k];
  sh[threadIdx.x] = o;
  __syncthreads();
  for (int s = kCompactThreads / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) sh[threadIdx.x] += sh[threadIdx.x + s];
    __syncthreads();
  }
  o = sh[0];
  __syncthreads();
  // each thread owns kCompactPer consecutive tokens (the order of the output)
  const int t0 = blockIdx.x * kCompactSpan + threadIdx.x * kCompactPer;
  bool kept[kCompactPer];
  int c = 0;
#pragma unroll
  for (int e = 0; e < kCompactPer; ++e) {
    const int t = t0 + e;
    kept[e] = t < N && keep(t);
    c += kept[e] ? 1 : 0;
  }
  sh[threadIdx.x] = c;
  __syncthreads();
  for (int off = 1; off < kCompactThreads; off <<= 1) {
    const int v = threadIdx.x >= off ? sh[threadIdx.x - off] : 0;
    __syncthreads();
    sh[threadIdx.x] += v;
    __syncthreads();
  }
  int p = o + sh[threadIdx.x] - c;
#pragma unroll
  for (int e = 0; e < kCompactPer; ++e) {
    const int t = t0 + e;
    if (t < N) {
      if (kept[e]) {
        idx[p] = t;
        if (mapped) mapped[p] = map[t];
      }
      if (pos) pos[t] = kept[e] ? p : -1;
    }
    p += kept[e] ? 1 : 0;
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == kCompactThreads - 1) {
    *count = p;
    if (stats) stats[4] = (double)p;
  }
}

// Tokens whose logits the forward computes: all of them when every token's
// log-prob is wanted, else those of completions with A != 0 (a zero advantage
// makes the token's loss term and gradient exactly zero, so its logits are
// not needed; a token with an invalid completion id is left to finalize,
// which flags it).
struct KeepForward {
  int R, all;
  const int32_t* seq_id;
  const float* adv;
  __device__ bool operator()(int t) const {
    if (all) return true;
    const int s = seq_id[t];
    return s >= 0 && s < R && adv[s] != 0.f;
  }
};

// Tokens whose logit gradient is not identically zero (delta != 0): the
// backward products run over these only.
struct KeepActive {
  const float* delta;
  __device__ bool operator()(int t) const { return delta[t] != 0.f; }
};

template <class Keep>
int launch_compact(int N, const Keep& keep, int32_t* cnt, int32_t* idx, int32_t* pos, const int32_t* map,
                   int32_t* mapped, int32_t* count, double* stats, hipStream_t stream) {
  const unsigned nblk = (unsigned)((N + kCompactSpan - 1) / kCompactSpan);
  hipLaunchKernelGGL(compact_count_kernel<Keep>, dim3(nblk), dim3(kCompactThreads), 0, stream, N, keep, cnt);
  PSPO_LAUNCHED("compact_count_kernel", stream);
  hipLaunchKernelGGL(compact_scatter_kernel<Keep>, dim3(nblk), dim3(kCompactThreads), 0, stream, N, keep, cnt, idx,
                     pos, map, mapped, count, stats);
  PSPO_LAUNCHED("compact_scatter_kernel", stream);
  return PSPO_OK;
}

// d_hidden rows of tokens with delta == 0 are exactly zero.
__global__ __launch_bounds__(256) void zero_inactive_rows_kernel(int d, const float* __restrict__ delta,
                                                                 float* __restrict__ dH) {
  const int t = blockIdx.x;
  if (delta[t] != 0.f) return;
  f32x4* row = reinterpret_cast<f32x4*>(dH + (int64_t)t * d);
  for (int c = threadIdx.x; c < d / 4; c += blockDim.x) row[c] = f32x4{0.f, 0.f, 0.f, 0.f};
}

template <class T>
__device__ T block_sum(T v, T* sh) {
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int s = kFinThreads / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) sh[threadIdx.x] += sh[threadIdx.x + s];
    __syncthreads();
  }
  T r = sh[0];
  __syncthreads();
  return r;
}

__device__ float block_max(float v, float* sh) {
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int s = kFinThreads / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) sh[threadIdx.x] = fmaxf(sh[threadIdx.x], sh[threadIdx.x + s]);
    __syncthreads();
  }
  float r = sh[0];
  __syncthreads();
  return r;
}

// Per token: merge the vocabulary-tile partials into lse, then the PPO terms.
// Each block writes (sum c s, sum |c s|, #clipped, #A==0) and max c to blk[5*b].
__global__ __launch_bounds__(kFinThreads) void finalize_kernel(
    int N, int V, int R, int ntv, int64_t ldp, const float* __restrict__ part_m, const float* __restrict__ part_l,
    const float* __restrict__ zt, const int32_t* __restrict__ fwd_pos, const int32_t* __restrict__ target,
    const float* __restrict__ logp_old,
    const float* __restrict__ weight, const int32_t* __restrict__ seq_id, const float* __restrict__ adv,
    float eps_low, float eps_high, float loss_scale, float* __restrict__ lse_out, float* __restrict__ delta_out,
    float* __restrict__ logp_new, double* __restrict__ blk, int32_t* __restrict__ err_flag) {
  __shared__ double shd[kFinThreads];
  __shared__ float shf[kFinThreads];
  const int t = blockIdx.x * kFinThreads + threadIdx.x;
  double cs = 0.0, acs = 0.0, nclip = 0.0, nzero = 0.0;
  float maxw = 0.f;
  if (t < N) {
    // column of this token's forward partials; -1: its logits were not needed
    const int col = fwd_pos[t];
    float lse = NAN;
    if (col >= 0) {
      float M = kNegInf;
      for (int k = 0; k < ntv; ++k) M = fmaxf(M, part_m[k * ldp + col]);
      float L = 0.f;
      for (int k = 0; k < ntv; ++k) L += part_l[k * ldp + col] * __expf(part_m[k * ldp + col] - M);
      lse = M + logf(L);
    }
    const int tgt = target[t];
    const int seq = seq_id[t];
    const bool valid = tgt >= 0 && tgt < V && seq >= 0 && seq < R;
    const float A = valid ? adv[seq] : 0.f;
    const float c = weight[t];
    float l = NAN, s = 0.f, dl = 0.f;
    bool mu = false;
    if (valid && col >= 0) {
      l = zt[col] - lse;
      const float rho = expf(l - logp_old[t]);
      const float clipped = fminf(fmaxf(rho, 1.f - eps_low), 1.f + eps_high);
      s = fminf(rho * A, clipped * A);
      mu = (A > 0.f && rho <= 1.f + eps_high) || (A < 0.f && rho >= 1.f - eps_low);
      dl = mu ? -loss_scale * c * rho * A : 0.f;
      // a non-finite hidden row, head row, old log-prob or weight shows up in
      // lse, rho, the loss term or delta (and would spread into the gradients)
      if (err_flag && !(std::isfinite(lse) && std::isfinite(rho) && std::isfinite(c * s) && std::isfinite(dl)))
        atomicOr(err_flag, PSPO_DEVERR_NONFINITE);
    } else if (!valid && err_flag) {
      atomicOr(err_flag, (tgt >= 0 && tgt < V) ? PSPO_DEVERR_SEQ_ID : PSPO_DEVERR_TARGET);
    }
    // (a valid token without forward partials has A == 0: zero loss term and gradient)
    lse_out[t] = lse;
    delta_out[t] = dl;
    if (logp_new) logp_new[t] = l;
    cs = (double)c * (double)s;
    acs = fabs(cs);
    nclip = (A != 0.f && !mu) ? 1.0 : 0.0;
    nzero = (A == 0.f) ? 1.0 : 0.0;
    maxw = c;
  }
  cs = block_sum(cs, shd);
  acs = block_sum(acs, shd);
  nclip = block_sum(nclip, shd);
  nzero = block_sum(nzero, shd);
  maxw = block_max(maxw, shf);
  if (threadIdx.x == 0) {
    double* o = blk + 5 * (int64_t)blockIdx.x;
    o[0] = cs;
    o[1] = acs;
    o[2] = nclip;
    o[3] = nzero;
    o[4] = maxw;
  }
}

// One block: fixed-order reduction of the per-block sums (deterministic).
__global__ __launch_bounds__(kFinThreads) void reduce_loss_kernel(int nblk, const double* __restrict__ blk,
                                                                  float loss_scale, double* __restrict__ loss,
                                                                  double* __restrict__ stats) {
  __shared__ double shd[kFinThreads];
  double v[4] = {0, 0, 0, 0};
  double mx = 0.0;
  for (int b = threadIdx.x; b < nblk; b += kFinThreads) {
    for (int k = 0; k < 4; ++k) v[k] += blk[5 * (int64_t)b + k];
    mx = fmax(mx, blk[5 * (int64_t)b + 4]);
  }
  for (int k = 0; k < 4; ++k) v[k] = block_sum(v[k], shd);
  shd[threadIdx.x] = mx;
  __syncthreads();
  for (int s = kFinThreads / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) shd[threadIdx.x] = fmax(shd[threadIdx.x], shd[threadIdx.x + s]);
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    *loss = -(double)loss_scale * v[0];
    if (stats) {
      stats[0] = (double)loss_scale * v[1];
      stats[1] = v[2];
      stats[2] = v[3];
      stats[3] = shd[0];
      if (nblk == 0) stats[4] = 0.0;   // otherwise written by the backward-token compaction
    }
  }
}

// The tail tiles of a product launched as whole rounds plus a K-split tail
// (gemm_nt_kernel with kLaunchRounds, then kLaunchTail + EpiSlab): each tail
// tile's K parts are summed in order from the slabs of its work-groups
// x + 8 (u S + p) and handed to `out` row by row, 16 values at a time.
// Grid (24 blocks of 16 rows, 8 XCDs x 32 tail tiles), 256 threads.
template <class Out>
__global__ __launch_bounds__(256) void tail_reduce_kernel(GemmShape g, const float* __restrict__ slab, Out out) {
  __shared__ float rows[16][kTileN + 4];
  int M, N, K;
  bounded_dims(g, M, N, K);
  const TileGrid tg = tile_grid(g.tiles_m, g.tiles_n, M, N);
  const int x = blockIdx.y % kNumXcd, u = blockIdx.y / kNumXcd;
  const int full = tg.per_xcd / 32 * 32;
  const int r = xcd_count(tg, x) - full;
  if (u >= r) return;
  const int parts = tail_parts(r, K / kTileK);
  int tm, tn;
  tile_at(tg, xcd_position(tg, x, full + u), 0, tm, tn);
  const int rb = blockIdx.x, tid = threadIdx.x;
  // the slab layout [24 blocks of 16 rows][256 columns][16]: column tid of row
  // block rb is 16 consecutive floats
  f32x4 sum[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) sum[q] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int p = 0; p < parts; ++p) {
    const f32x4* src = reinterpret_cast<const f32x4*>(slab + (int64_t)(x + kNumXcd * (u * parts + p)) * (kTileM * kTileN) +
                                                      rb * (16 * kTileN) + tid * 16);
#pragma unroll
    for (int q = 0; q < 4; ++q) sum[q] += __builtin_nontemporal_load(src + q);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) rows[q * 4 + e][tid] = sum[q][e];
  __syncthreads();
  const int lr = tid >> 4, c0 = (tid & 15) * 16;
  out(tm * kTileM + rb * 16 + lr, tn * kTileN + c0, &rows[lr][c0]);
}

// dW rows v0 + row (< V), as EpiDW writes them: (accumulate ? old : 0) + sum.
struct TailDW {
  int V, d, v0;
  float* dW;
  bool accumulate;
  __device__ __forceinline__ void operator()(int row, int col0, const float* v) const {
    if (v0 + row >= V) return;
    float* o = dW + (int64_t)(v0 + row) * d;
#pragma unroll
    for (int e = 0; e < 16; ++e)
      if (col0 + e < d) o[col0 + e] = (accumulate ? o[col0 + e] : 0.f) + v[e];
  }
};

// d_hidden row tok[row] (row < n), as EpiDH writes it: (first ? 0 : old) + sum.
struct TailDH {
  int N, d;
  float* dH;
  bool first;
  const int32_t* tok;
  const int32_t* n_dev;
  __device__ __forceinline__ void operator()(int row, int col0, const float* v) const {
    if (row >= min(N, *n_dev)) return;
    float* o = dH + (int64_t)tok[row] * d;
#pragma unroll
    for (int e = 0; e < 16; ++e)
      if (col0 + e < d) o[col0 + e] = (first ? 0.f : o[col0 + e]) + v[e];
  }
};

// Per backward column a < min(N, *n_dev) (token act[a]): its forward column
// (where the kept logits sit), target, lse and delta, in column order, so the
// backward kernels fetch a column's data in one contiguous round trip; and the
// target entry of its logit-gradient row, G_{o} = delta (1 - p(o)), as
// -delta expm1(l) with l = z_o - lse the token's log-prob (no cancellation as
// p(o) -> 1).  A backward token has delta != 0, hence a forward column.
__global__ __launch_bounds__(256) void gather_backward_kernel(int N, const int32_t* __restrict__ n_dev,
                                                              const int32_t* __restrict__ act,
                                                              const int32_t* __restrict__ fpos,
                                                              const int32_t* __restrict__ target,
                                                              const float* __restrict__ lse,
                                                              const float* __restrict__ delta,
                                                              const float* __restrict__ zt,
                                                              int32_t* __restrict__ afwd, int32_t* __restrict__ ctgt,
                                                              float* __restrict__ clse, float* __restrict__ cdelta,
                                                              float* __restrict__ cg1) {
  const int n = min(N, *n_dev);
  for (int a = blockIdx.x * 256 + threadIdx.x; a < n; a += gridDim.x * 256) {
    const int t = act[a];
    const int f = fpos[t];
    afwd[a] = f;
    ctgt[a] = target[t];
    clse[a] = lse[t];
    cdelta[a] = delta[t];
    cg1[a] = -delta[t] * expm1f(zt[f] - lse[t]);
  }
}

// ---------------------------------------------------------------------------
// Target entries of the logit gradient, g_i = G_{i,o_i} = delta_i (1 - p_i(o_i)),
// in float32, after the chunked products that carried the other entries in bf16
// ---------------------------------------------------------------------------

// bf16 pair (one 32-bit word) to two floats, exactly.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// d_hidden[act[a]] += cg1[a] * W[ctgt[a]] for every backward column
// a < min(N, *n_dev) (App. D: the target entry of the head score's row, times
// that row of W).  One wave per column, 8 features per lane and step.
// d % 8 == 0.
// Grid ceil(N / 4), 256 threads.
__global__ __launch_bounds__(256) void onehot_dh_kernel(int N, int d, const int32_t* __restrict__ n_dev,
                                                        const int32_t* __restrict__ act,
                                                        const int32_t* __restrict__ ctgt,
                                                        const float* __restrict__ cg1,
                                                        const uint16_t* __restrict__ w, float* __restrict__ dH) {
  const int n = min(N, *n_dev);
  const int a = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (a >= n) return;   // uniform over the wave
  const float dl = cg1[a];
  const u32x4* wr = reinterpret_cast<const u32x4*>(w + (int64_t)ctgt[a] * d);
  f32x4* hr = reinterpret_cast<f32x4*>(dH + (int64_t)act[a] * d);
  for (int c = lane; c < d / 8; c += 64) {
    const u32x4 wv = wr[c];
    f32x4 lo = hr[2 * c], hi = hr[2 * c + 1];
    lo[0] = fmaf(dl, bf16_lo(wv[0]), lo[0]);
    lo[1] = fmaf(dl, bf16_hi(wv[0]), lo[1]);
    lo[2] = fmaf(dl, bf16_lo(wv[1]), lo[2]);
    lo[3] = fmaf(dl, bf16_hi(wv[1]), lo[3]);
    hi[0] = fmaf(dl, bf16_lo(wv[2]), hi[0]);
    hi[1] = fmaf(dl, bf16_hi(wv[2]), hi[1]);
    hi[2] = fmaf(dl, bf16_lo(wv[3]), hi[2]);
    hi[3] = fmaf(dl, bf16_hi(wv[3]), hi[3]);
    hr[2 * c] = lo;
    hr[2 * c + 1] = hi;
  }
}

// The dW side groups the backward columns by target id.  Stable bucketing,
// every result independent of scheduling:
//   count:  cnt[v] = #{a : ctgt[a] = v}                    (integer atomics)
//   scan:   start[v] = sum_{u < v} cnt[u]; cursor = start;   the non-empty ids
//           in increasing order in rows[0 .. *nrows)        (three launches)
//   fill:   each column takes a slot of its bucket           (arbitrary order)
//   rank:   column a goes to start[v] + #{b in bucket v : b < a} of `sorted`,
//           i.e. the bucket in increasing column order.
// The rank pass reads a column's whole bucket: O(sum_v cnt[v]^2) reads in all,
// from a bucket that the waves sharing it read together (a few microseconds
// for uniform targets; about a millisecond if every column had one target).
__global__ __launch_bounds__(256) void onehot_count_kernel(int N, const int32_t* __restrict__ n_dev,
                                                           const int32_t* __restrict__ ctgt,
                                                           int32_t* __restrict__ cnt) {
  const int n = min(N, *n_dev);
  for (int a = blockIdx.x * 256 + threadIdx.x; a < n; a += gridDim.x * 256) atomicAdd(&cnt[ctgt[a]], 1);
}

// The scan in three launches over blocks of kScanSpan ids (256 threads x 16
// consecutive ids each): per-block totals of cnt and of non-empty ids; their
// exclusive scan (one work-group, 256 blocks at a time); then each block's
// outputs from its offsets and a work-group scan of its threads' totals.
constexpr int kScanPer = 16, kScanSpan = 256 * kScanPer;

// Exclusive scan of one value per thread over a 256-thread work-group; also
// returns the work-group total.
__device__ int block_exclusive_scan(int v, int* sh, int& total) {
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const int a = threadIdx.x >= off ? sh[threadIdx.x - off] : 0;
    __syncthreads();
    sh[threadIdx.x] += a;
    __syncthreads();
  }
  total = sh[255];
  const int r = sh[threadIdx.x] - v;
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(256) void onehot_scan_totals_kernel(int V, const int32_t* __restrict__ cnt,
                                                                 int32_t* __restrict__ tot) {
  __shared__ int sh[256];
  const int v0 = blockIdx.x * kScanSpan + threadIdx.x * kScanPer;
  int c = 0, r = 0;
#pragma unroll
  for (int e = 0; e < kScanPer; ++e) {
    const int k = v0 + e < V ? cnt[v0 + e] : 0;
    c += k;
    r += k > 0 ? 1 : 0;
  }
  int tc, tr;
  block_exclusive_scan(c, sh, tc);
  block_exclusive_scan(r, sh, tr);
  if (threadIdx.x == 0) {
    tot[2 * blockIdx.x] = tc;
    tot[2 * blockIdx.x + 1] = tr;
  }
}

// One work-group: tot (a pair per block) -> exclusive offsets in place; the
// number of non-empty ids to *nrows.
__global__ __launch_bounds__(256) void onehot_scan_offsets_kernel(int nblk, int32_t* __restrict__ tot,
                                                                  int32_t* __restrict__ nrows) {
  __shared__ int sh[256];
  int base_c = 0, base_r = 0;
  for (int b0 = 0; b0 < nblk; b0 += 256) {
    const int b = b0 + threadIdx.x;
    const int c = b < nblk ? tot[2 * b] : 0, r = b < nblk ? tot[2 * b + 1] : 0;
    int tc, tr;
    const int ec = block_exclusive_scan(c, sh, tc);
    const int er = block_exclusive_scan(r, sh, tr);
    if (b < nblk) {
      tot[2 * b] = base_c + ec;
      tot[2 * b + 1] = base_r + er;
    }
    base_c += tc;
    base_r += tr;
  }
  if (threadIdx.x == 0) *nrows = base_r;
}

// start[v] = sum_{u < v} cnt[u]; cursor = start; the non-empty ids in
// increasing order in rows.
__global__ __launch_bounds__(256) void onehot_scan_write_kernel(int V, const int32_t* __restrict__ cnt,
                                                                const int32_t* __restrict__ off,
                                                                int32_t* __restrict__ start,
                                                                int32_t* __restrict__ cursor,
                                                                int32_t* __restrict__ rows) {
  __shared__ int sh[256];
  const int v0 = blockIdx.x * kScanSpan + threadIdx.x * kScanPer;
  int k[kScanPer];
  int c = 0, r = 0;
#pragma unroll
  for (int e = 0; e < kScanPer; ++e) {
    k[e] = v0 + e < V ? cnt[v0 + e] : 0;
    c += k[e];
    r += k[e] > 0 ? 1 : 0;
  }
  int tc, tr;
  c = off[2 * blockIdx.x] + block_exclusive_scan(c, sh, tc);
  r = off[2 * blockIdx.x + 1] + block_exclusive_scan(r, sh, tr);
#pragma unroll
  for (int e = 0; e < kScanPer; ++e) {
    if (v0 + e < V) {
      start[v0 + e] = c;
      cursor[v0 + e] = c;
      if (k[e] > 0) rows[r++] = v0 + e;
      c += k[e];
    }
  }
}

__global__ __launch_bounds__(256) void onehot_fill_kernel(int N, const int32_t* __restrict__ n_dev,
                                                          const int32_t* __restrict__ ctgt,
                                                          int32_t* __restrict__ cursor, int32_t* __restrict__ tmp) {
  const int n = min(N, *n_dev);
  for (int a = blockIdx.x * 256 + threadIdx.x; a < n; a += gridDim.x * 256) tmp[atomicAdd(&cursor[ctgt[a]], 1)] = a;
}

__global__ __launch_bounds__(256) void onehot_rank_kernel(int N, const int32_t* __restrict__ n_dev,
                                                          const int32_t* __restrict__ ctgt,
                                                          const int32_t* __restrict__ start,
                                                          const int32_t* __restrict__ cnt,
                                                          const int32_t* __restrict__ tmp,
                                                          int32_t* __restrict__ sorted) {
  const int n = min(N, *n_dev);
  for (int a = blockIdx.x * 256 + threadIdx.x; a < n; a += gridDim.x * 256) {
    const int v = ctgt[a], s = start[v], e = s + cnt[v];
    int rank = 0;
    for (int k = s; k < e; ++k) rank += tmp[k] < a ? 1 : 0;
    sorted[s + rank] = a;
  }
}

// dW[v] += sum over the bucket of v, in increasing column order, of
// cg1[a] * h[act[a]] (App. D: the target entries of the head scores), the sum
// accumulated in float32 and then added to the row.  One wave per non-empty
// id rows[k], k < *nrows (<= the launch's row bound); 8 features per lane and
// step, kOnehotSteps steps of the row per pass over the bucket.  d % 8 == 0.
// Grid ceil(bound / 4), 256 threads.
constexpr int kOnehotSteps = 8;   // 8 x 8 features per lane: 4096 of the row per pass over the bucket

__global__ __launch_bounds__(256) void onehot_dw_kernel(int bound, int d, const int32_t* __restrict__ nrows,
                                                        const int32_t* __restrict__ rows,
                                                        const int32_t* __restrict__ start,
                                                        const int32_t* __restrict__ cnt,
                                                        const int32_t* __restrict__ sorted,
                                                        const int32_t* __restrict__ act,
                                                        const float* __restrict__ cg1,
                                                        const uint16_t* __restrict__ hidden, float* __restrict__ dW) {
  const int k = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (k >= min(bound, *nrows)) return;   // uniform over the wave
  const int v = rows[k], s = start[v], e = s + cnt[v];
  const int d8 = d / 8;
  f32x4* out = reinterpret_cast<f32x4*>(dW + (int64_t)v * d);
  for (int c0 = 0; c0 < d8; c0 += 64 * kOnehotSteps) {
    f32x4 lo[kOnehotSteps], hi[kOnehotSteps];
#pragma unroll
    for (int q = 0; q < kOnehotSteps; ++q) lo[q] = hi[q] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int b = s; b < e; ++b) {
      const int a = sorted[b];
      const float dl = cg1[a];
      const u32x4* hr = reinterpret_cast<const u32x4*>(hidden + (int64_t)act[a] * d);
#pragma unroll
      for (int q = 0; q < kOnehotSteps; ++q) {
        const int c = c0 + q * 64 + lane;
        if (c < d8) {
          const u32x4 hv = hr[c];
          lo[q][0] = fmaf(dl, bf16_lo(hv[0]), lo[q][0]);
          lo[q][1] = fmaf(dl, bf16_hi(hv[0]), lo[q][1]);
          lo[q][2] = fmaf(dl, bf16_lo(hv[1]), lo[q][2]);
          lo[q][3] = fmaf(dl, bf16_hi(hv[1]), lo[q][3]);
          hi[q][0] = fmaf(dl, bf16_lo(hv[2]), hi[q][0]);
          hi[q][1] = fmaf(dl, bf16_hi(hv[2]), hi[q][1]);
          hi[q][2] = fmaf(dl, bf16_lo(hv[3]), hi[q][2]);
          hi[q][3] = fmaf(dl, bf16_hi(hv[3]), hi[q][3]);
        }
      }
    }
#pragma unroll
    for (int q = 0; q < kOnehotSteps; ++q) {
      const int c = c0 + q * 64 + lane;
      if (c < d8) {
        out[2 * c] += lo[q];
        out[2 * c + 1] += hi[q];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Workspace plan
// ---------------------------------------------------------------------------


struct Plan {
  int64_t Npad, Vpad, dpad, Vc, ntv, nfin;
  int64_t Dk;   // K of the products over the hidden features: d rounded up to 32 (zero padding)
  int64_t off_pm, off_pl, off_zt, off_lse, off_delta, off_fidx, off_fpos, off_nfwd, off_idx, off_nact, off_afwd,
      off_ctgt, off_clse, off_cdelta, off_cg1, off_ftgt, off_cnt, off_blk, off_wk, off_hk, off_ht, off_wt, off_dn, off_dt,
      off_slab, off_zk, off_oh_cnt, off_oh_start, off_oh_cursor, off_oh_rows, off_oh_nrows, off_oh_tot, off_oh_tmp,
      off_oh_sorted, total;
  bool keep;   // the forward keeps the first chunk's logits (fp16 offsets from the tile maxima)
};

Plan make_plan(int64_t N, int64_t d, int64_t V, bool keep) {
  Plan p{};
  p.Npad = round_up(N > 0 ? N : 1, kTileLcm);   // token rows: tiles of 256 (B side) and 384 (A side)
  p.Vpad = round_up(V, kTileM);
  p.dpad = round_up(d, kTileN);
  p.Dk = round_up(d, kTileK);
  const int64_t d64 = round_up(d, 64);   // columns the K-blocked copies write (64 per copy tile)
  // Vocabulary rows per backward chunk.  The base width is a multiple of
  // 384-row tiles for which the dW product of a chunk ((Vc / 384) x
  // ceil(d / 256) tiles of very long K) fills whole rounds of the 256 CUs
  // (d = 3584: 14 column tiles, 128 row tiles, exactly 7 rounds).  The
  // vocabulary is split evenly into as many chunks as it holds base widths,
  // plus one more only if the remainder exceeds a quarter of a base width: a
  // short last chunk would run its dH product at a short K, where the per-tile
  // read-modify-write and prologue costs dominate (V = 152064: three chunks of
  // 50688 rows instead of three of 49152 and one of 4608, -0.4% per call); the
  // K-split tails absorb the partial rounds.
  {
    int64_t a = p.dpad / kTileN, b = 256;
    while (b) {
      const int64_t r = a % b;
      a = b;
      b = r;
    }
    const int64_t rows = 256 / a * kTileM;
    const int64_t whole = p.Vpad / rows, rem = p.Vpad % rows;
    const int64_t nch = whole == 0 ? 1 : (rem * 4 <= rows ? whole : whole + 1);
    p.Vc = round_up((p.Vpad + nch - 1) / nch, kTileM);
  }
  p.ntv = p.Vpad / kTileM;
  p.nfin = (N + kFinThreads - 1) / kFinThreads;
  int64_t o = 0;
  auto take = [&](int64_t bytes) {
    const int64_t at = o;
    o = round_up(o + bytes, 256);
    return at;
  };
  p.off_pm = take(p.ntv * p.Npad * 4);
  p.off_pl = take(p.ntv * p.Npad * 4);
  p.off_zt = take(p.Npad * 4);
  p.off_lse = take(p.Npad * 4);
  p.off_delta = take(p.Npad * 4);
  p.off_fidx = take(p.Npad * 4);
  p.off_fpos = take(p.Npad * 4);
  p.off_nfwd = take(4);
  p.off_idx = take(p.Npad * 4);
  p.off_nact = take(4);
  p.off_afwd = take(p.Npad * 4);                                      // backward columns: forward column,
  p.off_ctgt = take(p.Npad * 4);                                      //   target, lse, delta
  p.off_clse = take(p.Npad * 4);
  p.off_cdelta = take(p.Npad * 4);
  p.off_cg1 = take(p.Npad * 4);                                       //   and target entry of the gradient row
  p.off_ftgt = take(p.Npad * 4);                                      // forward columns: target
  p.off_cnt = take((p.Npad + kCompactSpan - 1) / kCompactSpan * 4);   // per-block counts of a compaction
  p.off_blk = take((p.nfin > 0 ? p.nfin : 1) * 5 * 8);
  p.off_wk = take(d64 * p.Vpad * 2);                                  // W, K-blocked [d64/32][Vpad][32]
  p.off_hk = take(d64 * p.Npad * 2);                                  // gathered hidden rows [d64/32][Npad][32]
  p.off_ht = take(p.dpad * p.Npad * 2);                               // H[bwd]^T [Npad/32][dpad][32]
  p.off_wt = take(p.dpad * ((p.Vpad + p.Vc - 1) / p.Vc) * p.Vc * 2);  // per chunk: W^T [Vc/32][dpad][32]
  p.off_dn = take(p.Npad * p.Vc * 2);                                 // [Npad/768][Vc/32][768][32] (token blocks)
  p.off_dt = take(p.Vc * p.Npad * 2);                                 // [Vc/384][Npad/32][384][32] (vocabulary blocks)
  p.off_slab = take((int64_t)kNumXcd * kTailSlots * kTileM * kTileN * 4);   // K parts of tail tiles
  p.keep = keep;
  p.off_zk = take(keep ? p.Vc * p.Npad * 2 : 0);                      // kept fp16 logit offsets, one block per forward tile
  p.off_oh_cnt = take(V * 4);                                         // one-hot part: backward columns per target id,
  p.off_oh_start = take(V * 4);                                       //   bucket starts, fill cursors,
  p.off_oh_cursor = take(V * 4);
  p.off_oh_rows = take(V * 4);                                        //   non-empty ids and their count,
  p.off_oh_nrows = take(4);
  p.off_oh_tot = take((V + kScanSpan - 1) / kScanSpan * 8);           //   per-block totals of the scan
  p.off_oh_tmp = take(p.Npad * 4);                                    //   buckets unordered, then in column order
  p.off_oh_sorted = take(p.Npad * 4);
  p.total = o;
  return p;
}

template <class Epi>
int launch_gemm(const GemmShape& g, const Epi& epi, hipStream_t stream) {
  hipLaunchKernelGGL(gemm_nt_kernel<Epi>, dim3(gemm_grid(g.tiles_m, g.tiles_n)), dim3(kGemmThreads), 0, stream, g,
                     epi);
  PSPO_LAUNCHED(__PRETTY_FUNCTION__, stream);
  return PSPO_OK;
}

// A product with long tiles as whole rounds (epilogue `epi`), then the
// remaining tiles split along K into slabs, then their sums (written by `out`
// as `epi` would write them): the CUs stay busy through the last round.
template <class Epi, class Out>
int launch_gemm_split_tail(const GemmShape& g, const Epi& epi, const Out& out, float* slab, hipStream_t stream) {
  hipLaunchKernelGGL((gemm_nt_kernel<Epi, kLaunchRounds>), dim3(gemm_grid(g.tiles_m, g.tiles_n)), dim3(kGemmThreads),
                     0, stream, g, epi);
  PSPO_LAUNCHED("gemm_nt_kernel (whole rounds)", stream);
  hipLaunchKernelGGL((gemm_nt_kernel<EpiSlab, kLaunchTail>), dim3(kNumXcd * kTailSlots), dim3(kGemmThreads), 0,
                     stream, g, EpiSlab{slab});
  PSPO_LAUNCHED("gemm_nt_kernel (K-split tail)", stream);
  hipLaunchKernelGGL(tail_reduce_kernel<Out>, dim3(kTileM / 16, kNumXcd * 32), dim3(256), 0, stream, g,
                     (const float*)slab, out);
  PSPO_LAUNCHED("tail_reduce_kernel", stream);
  return PSPO_OK;
}

}  // namespace
}  // namespace pspo

extern "C" {

size_t pspo_loss_workspace_bytes(int32_t N, int32_t d, int32_t V, uint32_t flags) {
  if (N < 0 || d <= 0 || V <= 0) return 0;
  return (size_t)pspo::make_plan(N, d, V, (flags & PSPO_KEEP_LOGITS) != 0).total;
}

int pspo_loss_fwd_bwd(const uint16_t* hidden, const uint16_t* w_head, const int32_t* target, const float* logp_old,
                      const float* weight, const int32_t* seq_id, const float* advantage, int32_t N, int32_t d,
                      int32_t V, int32_t R, float eps_low, float eps_high, float loss_scale, uint32_t flags,
                      double* loss, float* d_hidden, float* d_w_head, float* logp_new, double* stats,
                      int32_t* err_flag, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  using namespace pspo;
  clear_last_error();
  TraceRange trace_range("pspo_loss_fwd_bwd");
  PSPO_REQUIRE(N >= 0 && R >= 0, PSPO_ERR_INVALID_ARG, "N and R must be >= 0");
  PSPO_REQUIRE(d > 0 && V > 0, PSPO_ERR_INVALID_ARG, "d and V must be > 0");
  PSPO_REQUIRE(d % 8 == 0, PSPO_ERR_UNSUPPORTED, "d must be a multiple of 8");
  PSPO_REQUIRE(N == 0 || R > 0, PSPO_ERR_INVALID_ARG, "R must be > 0 when N > 0");
  PSPO_REQUIRE((flags & ~(PSPO_ACCUMULATE_DW | PSPO_KEEP_LOGITS)) == 0, PSPO_ERR_INVALID_ARG,
               "unknown flag bits");
  PSPO_REQUIRE(std::isfinite(eps_low) && eps_low >= 0.f && eps_low < 1.f, PSPO_ERR_INVALID_ARG,
               "eps_low must lie in [0, 1)");
  PSPO_REQUIRE(std::isfinite(eps_high) && eps_high >= 0.f && eps_high < 1.f, PSPO_ERR_INVALID_ARG,
               "eps_high must lie in [0, 1)");
  PSPO_REQUIRE(std::isfinite(loss_scale), PSPO_ERR_INVALID_ARG, "loss_scale must be finite");
  PSPO_REQUIRE(loss && d_w_head, PSPO_ERR_INVALID_ARG, "loss and d_w_head must not be NULL");
  PSPO_REQUIRE(aligned(loss, 8) && aligned(d_w_head, 16), PSPO_ERR_INVALID_ARG, "misaligned output pointer");
  if (N > 0) {
    PSPO_REQUIRE(hidden && w_head && target && logp_old && weight && seq_id && advantage && d_hidden,
                 PSPO_ERR_INVALID_ARG, "null input pointer");
    PSPO_REQUIRE(aligned(hidden, 16) && aligned(w_head, 16) && aligned(d_hidden, 16), PSPO_ERR_INVALID_ARG,
                 "hidden, w_head and d_hidden must be 16-byte aligned");
    PSPO_REQUIRE(aligned(target, 4) && aligned(logp_old, 4) && aligned(weight, 4) && aligned(seq_id, 4) &&
                     aligned(advantage, 4) && aligned(logp_new, 4),
                 PSPO_ERR_INVALID_ARG, "misaligned per-token pointer");
    PSPO_REQUIRE(workspace != nullptr && aligned(workspace, 256), PSPO_ERR_INVALID_ARG,
                 "workspace must be non-NULL and 256-byte aligned");
  }
  if (stats) PSPO_REQUIRE(aligned(stats, 8), PSPO_ERR_INVALID_ARG, "misaligned stats");
  const Plan pl = make_plan(N, d, V, (flags & PSPO_KEEP_LOGITS) != 0);
  PSPO_REQUIRE(pl.Npad <= kMaxPaddedRows && pl.Vpad <= kMaxPaddedRows, PSPO_ERR_UNSUPPORTED,
               "N and V must each be at most " + std::to_string(kMaxPaddedRows) + " rows after padding");
  PSPO_REQUIRE(d <= kMaxPaddedRows, PSPO_ERR_UNSUPPORTED,
               "d must be at most " + std::to_string(kMaxPaddedRows));
  PSPO_REQUIRE(N == 0 || workspace_bytes >= (size_t)pl.total, PSPO_ERR_WORKSPACE,
               "workspace too small: need " + std::to_string(pl.total) + " bytes");
  if (int rc = require_gfx950()) return rc;

  const bool accumulate = (flags & PSPO_ACCUMULATE_DW) != 0;
  if (N == 0) {
    if (!accumulate) {
      hipLaunchKernelGGL(fill_f32_kernel, dim3(1024), dim3(256), 0, stream, d_w_head, (int64_t)V * d, 0.f);
      PSPO_LAUNCHED("fill_f32_kernel", stream);
    }
    hipLaunchKernelGGL(reduce_loss_kernel, dim3(1), dim3(kFinThreads), 0, stream, 0, nullptr, loss_scale, loss,
                       stats);
    PSPO_LAUNCHED("reduce_loss_kernel", stream);
    return PSPO_OK;
  }

  char* ws = static_cast<char*>(workspace);
  float* part_m = reinterpret_cast<float*>(ws + pl.off_pm);
  float* part_l = reinterpret_cast<float*>(ws + pl.off_pl);
  float* zt = reinterpret_cast<float*>(ws + pl.off_zt);
  float* lse = reinterpret_cast<float*>(ws + pl.off_lse);
  float* delta = reinterpret_cast<float*>(ws + pl.off_delta);
  int32_t* fwd_idx = reinterpret_cast<int32_t*>(ws + pl.off_fidx);
  int32_t* fwd_pos = reinterpret_cast<int32_t*>(ws + pl.off_fpos);
  int32_t* n_fwd = reinterpret_cast<int32_t*>(ws + pl.off_nfwd);
  int32_t* act_idx = reinterpret_cast<int32_t*>(ws + pl.off_idx);
  int32_t* n_act = reinterpret_cast<int32_t*>(ws + pl.off_nact);
  int32_t* cnt = reinterpret_cast<int32_t*>(ws + pl.off_cnt);
  int32_t* act_fwd = reinterpret_cast<int32_t*>(ws + pl.off_afwd);
  int32_t* act_tgt = reinterpret_cast<int32_t*>(ws + pl.off_ctgt);
  float* act_lse = reinterpret_cast<float*>(ws + pl.off_clse);
  float* act_delta = reinterpret_cast<float*>(ws + pl.off_cdelta);
  float* act_g1 = reinterpret_cast<float*>(ws + pl.off_cg1);
  int32_t* fwd_tgt = reinterpret_cast<int32_t*>(ws + pl.off_ftgt);
  double* blk = reinterpret_cast<double*>(ws + pl.off_blk);
  uint16_t* wk = reinterpret_cast<uint16_t*>(ws + pl.off_wk);
  uint16_t* hk = reinterpret_cast<uint16_t*>(ws + pl.off_hk);
  uint16_t* hT = reinterpret_cast<uint16_t*>(ws + pl.off_ht);
  uint16_t* wT = reinterpret_cast<uint16_t*>(ws + pl.off_wt);
  uint16_t* dN = reinterpret_cast<uint16_t*>(ws + pl.off_dn);
  uint16_t* dT = reinterpret_cast<uint16_t*>(ws + pl.off_dt);
  uint16_t* zk = pl.keep ? reinterpret_cast<uint16_t*>(ws + pl.off_zk) : nullptr;
  float* slab = reinterpret_cast<float*>(ws + pl.off_slab);
  int32_t* oh_cnt = reinterpret_cast<int32_t*>(ws + pl.off_oh_cnt);
  int32_t* oh_start = reinterpret_cast<int32_t*>(ws + pl.off_oh_start);
  int32_t* oh_cursor = reinterpret_cast<int32_t*>(ws + pl.off_oh_cursor);
  int32_t* oh_rows = reinterpret_cast<int32_t*>(ws + pl.off_oh_rows);
  int32_t* oh_nrows = reinterpret_cast<int32_t*>(ws + pl.off_oh_nrows);
  int32_t* oh_tot = reinterpret_cast<int32_t*>(ws + pl.off_oh_tot);
  int32_t* oh_tmp = reinterpret_cast<int32_t*>(ws + pl.off_oh_tmp);
  int32_t* oh_sorted = reinterpret_cast<int32_t*>(ws + pl.off_oh_sorted);
  const int Dk = (int)pl.Dk;

  const int tiles_tok_n = (int)(pl.Npad / kTileN);    // tokens on the B side
  const int tiles_tok_m = (int)(pl.Npad / kTileM);    // tokens on the A side
  const int tiles_voc = (int)pl.ntv;
  const int tiles_d = (int)(pl.dpad / kTileN);
  const unsigned ctiles64 = (unsigned)((d + 63) / 64);

  // 1. the tokens whose logits are needed (all of them if logp_new is wanted);
  //    W and their hidden rows as K-blocked operands
  if (int rc = launch_compact(N, KeepForward{R, logp_new != nullptr ? 1 : 0, seq_id, advantage}, cnt, fwd_idx,
                              fwd_pos, target, fwd_tgt, n_fwd, nullptr, stream))
    return rc;
  // W K-blocked (forward and logit-gradient products) and, per vocabulary
  // chunk, W[chunk]^T (dH product), in one pass over W
  hipLaunchKernelGGL(kblock_rows_kernel, dim3(ctiles64, (unsigned)(pl.Vpad / 32)), dim3(256), 0, stream, w_head,
                     (int64_t)d, d, V, nullptr, nullptr, wk, pl.Vpad, wT, pl.dpad, pl.Vc);
  PSPO_LAUNCHED("kblock_rows_kernel", stream);
  hipLaunchKernelGGL(kblock_rows_kernel, dim3(ctiles64, (unsigned)(pl.Npad / 32)), dim3(256), 0, stream, hidden,
                     (int64_t)d, d, N, fwd_idx, n_fwd, hk, pl.Npad, nullptr, (int64_t)0, (int64_t)kTileK);
  PSPO_LAUNCHED("kblock_rows_kernel", stream);
  // 2. forward logits -> per-tile softmax partials (target logits apart): the
  //    vocabulary tiles whose rows are all token ids, then a partial last one
  {
    ProductTimer timer(stream);
    if (int rc = timer.begin(PSPO_TIME_FORWARD)) return rc;
    const int tiles_full = V / kTileM, kept_tiles = zk != nullptr ? (int)(pl.Vc / kTileM) : 0;
    if (tiles_full > 0) {
      // the kept tiles' stores spread over the XCDs
      GemmShape g{wk, pl.Vpad, tiles_full * kTileM, hk, pl.Npad, N, Dk, tiles_full, tiles_tok_n, n_fwd, kDynN,
                  kept_tiles < tiles_full ? kept_tiles : tiles_full};
      EpiForward<true> e{V, N, pl.Npad, 0, part_m, part_l, n_fwd, zk, kept_tiles, tiles_tok_n};
      if (int rc = launch_gemm(g, e, stream)) return rc;
    }
    if (tiles_full < tiles_voc) {
      GemmShape g{wk + (int64_t)tiles_full * kTileM * kTileK, pl.Vpad, V - tiles_full * kTileM, hk, pl.Npad, N, Dk, 1,
                  tiles_tok_n, n_fwd, kDynN};
      EpiForward<false> e{V, N, pl.Npad, tiles_full, part_m, part_l, n_fwd, zk, kept_tiles, tiles_tok_n};
      if (int rc = launch_gemm(g, e, stream)) return rc;
    }
    if (int rc = timer.end()) return rc;
  }
  // the target logit of each forward column (the column's token row and target)
  hipLaunchKernelGGL(row_dots_kernel, dim3((unsigned)(pl.Npad / 4)), dim3(256), 0, stream, hidden, w_head, d, V, N,
                     fwd_idx, fwd_tgt, n_fwd, zt, nullptr);
  PSPO_LAUNCHED("row_dots_kernel", stream);
  // 3. lse, PPO terms, delta, loss
  hipLaunchKernelGGL(finalize_kernel, dim3((unsigned)pl.nfin), dim3(kFinThreads), 0, stream, N, V, R, tiles_voc,
                     pl.Npad, part_m, part_l, zt, fwd_pos, target, logp_old, weight, seq_id, advantage, eps_low,
                     eps_high, loss_scale, lse, delta, logp_new, blk, err_flag);
  PSPO_LAUNCHED("finalize_kernel", stream);
  hipLaunchKernelGGL(reduce_loss_kernel, dim3(1), dim3(kFinThreads), 0, stream, (int)pl.nfin, blk, loss_scale,
                     loss, stats);
  PSPO_LAUNCHED("reduce_loss_kernel", stream);
  // 4. the backward runs over the tokens with delta != 0 only (every other
  //    token has a zero logit-gradient row: zero d_hidden row, no dW term)
  if (int rc = launch_compact(N, KeepActive{delta}, cnt, act_idx, nullptr, nullptr, nullptr, n_act, stats, stream))
    return rc;
  hipLaunchKernelGGL(gather_backward_kernel, dim3((unsigned)((pl.Npad + 255) / 256)), dim3(256), 0, stream, N, n_act,
                     act_idx, fwd_pos, target, lse, delta, zt, act_fwd, act_tgt, act_lse, act_delta, act_g1);
  PSPO_LAUNCHED("gather_backward_kernel", stream);
  hipLaunchKernelGGL(zero_inactive_rows_kernel, dim3((unsigned)N), dim3(256), 0, stream, d, delta, d_hidden);
  PSPO_LAUNCHED("zero_inactive_rows_kernel", stream);
  // 5. operands of the gradient products: the backward tokens' hidden rows
  //    (K-blocked, in the forward's buffer) and their transpose H[bwd]^T
  //    [dpad x Npad], in one pass
  hipLaunchKernelGGL(kblock_rows_kernel, dim3(ctiles64, (unsigned)(pl.Npad / 32)), dim3(256), 0, stream, hidden,
                     (int64_t)d, d, N, act_idx, n_act, hk, pl.Npad, hT, pl.dpad, pl.Npad);
  PSPO_LAUNCHED("kblock_rows_kernel", stream);
  // 6. backward, one vocabulary chunk at a time; every product is bounded by
  //    the active-token count in device memory
  for (int64_t v0 = 0; v0 < pl.Vpad; v0 += pl.Vc) {
    const int64_t vc = (pl.Vpad - v0) < pl.Vc ? (pl.Vpad - v0) : pl.Vc;
    const int ctiles = (int)(vc / kTileM);
    ProductTimer t_grad(stream), t_dw(stream), t_dh(stream);
    if (int rc = t_grad.begin(PSPO_TIME_LOGIT_GRAD)) return rc;
    if (v0 == 0 && zk != nullptr) {
      hipLaunchKernelGGL(logit_grad_kept_kernel, dim3((unsigned)(pl.Vc / 128), (unsigned)(pl.Npad / 32)), dim3(256), 0,
                         stream, zk, part_m, pl.Npad, tiles_tok_n, (int)pl.Vc, V, N, n_act, act_fwd, act_lse,
                         act_delta, dN, pl.Vc / kTileK, dT, pl.Npad / kTileK);
      PSPO_LAUNCHED("logit_grad_kept_kernel", stream);
    } else {
      // the chunk's vocabulary tiles whose rows are all token ids, then a
      // partial last one (the last chunk's, when 384 does not divide V)
      const int64_t rows = (V - v0) < vc ? (V - v0) : vc;
      const int tfull = (int)(rows / kTileM);
      if (tfull > 0) {
        GemmShape g{wk + v0 * kTileK, pl.Vpad, tfull * kTileM, hk, pl.Npad, N, Dk, tfull, tiles_tok_n, n_act, kDynN};
        EpiDelta<true> e{V, N, (int)v0, 0, dT, pl.Npad / kTileK, dN, pl.Vc / kTileK, act_lse, act_delta, n_act};
        if (int rc = launch_gemm(g, e, stream)) return rc;
      }
      if (tfull < ctiles) {
        const int64_t vp = v0 + (int64_t)tfull * kTileM;   // first row of the partial tile
        GemmShape g{wk + vp * kTileK, pl.Vpad, (int)(V - vp), hk, pl.Npad, N, Dk, 1, tiles_tok_n, n_act, kDynN};
        EpiDelta<false> e{V, N, (int)v0, tfull, dT, pl.Npad / kTileK, dN, pl.Vc / kTileK, act_lse, act_delta,
                          n_act};
        if (int rc = launch_gemm(g, e, stream)) return rc;
      }
    }
    if (int rc = t_grad.end()) return rc;
    hipLaunchKernelGGL(zero_targets_kernel, dim3((unsigned)std::min<int64_t>((pl.Npad + 255) / 256, 1024)), dim3(256),
                       0, stream, N, n_act, act_tgt, (int)v0, (int)vc, dN, pl.Vc / kTileK, dT, pl.Npad / kTileK);
    PSPO_LAUNCHED("zero_targets_kernel", stream);
    {
      GemmShape g{dT, pl.Vc, (int)vc, hT, pl.dpad, d, (int)pl.Npad, ctiles, tiles_d, n_act, kDynK, 0,
                  kTileM, pl.Npad * kTileM * 2};
      EpiDW e{V, d, (int)v0, d_w_head, accumulate};
      if (int rc = t_dw.begin(PSPO_TIME_DW)) return rc;
      if (int rc = launch_gemm_split_tail(g, e, TailDW{V, d, (int)v0, d_w_head, accumulate}, slab, stream))
        return rc;
      if (int rc = t_dw.end()) return rc;
    }
    {
      GemmShape g{dN, pl.Npad, (int)pl.Npad, wT + (v0 / pl.Vc) * pl.dpad * pl.Vc, pl.dpad, d, (int)vc, tiles_tok_m,
                  tiles_d, n_act, kDynM, 0, kTileLcm, pl.Vc * kTileLcm * 2};
      EpiDH e{N, d, d_hidden, v0 == 0, act_idx, n_act};
      if (int rc = t_dh.begin(PSPO_TIME_DH)) return rc;
      if (int rc = launch_gemm_split_tail(g, e, TailDH{N, d, d_hidden, v0 == 0, act_idx, n_act}, slab, stream))
        return rc;
      if (int rc = t_dh.end()) return rc;
    }
  }
  // 7. the target entries of the logit gradient, in float32: the backward
  //    columns bucketed by target id in column order, then dW[v] += the sum
  //    of each bucket's g h rows and d_hidden += g W[o] row by row
  {
    const unsigned gcols = (unsigned)std::min<int64_t>((pl.Npad + 255) / 256, 1024);
    hipLaunchKernelGGL(fill_i32_kernel, dim3((unsigned)std::min<int64_t>((V + 255) / 256, 1024)), dim3(256), 0,
                       stream, oh_cnt, (int64_t)V, 0);
    PSPO_LAUNCHED("fill_i32_kernel", stream);
    hipLaunchKernelGGL(onehot_count_kernel, dim3(gcols), dim3(256), 0, stream, N, n_act, act_tgt, oh_cnt);
    PSPO_LAUNCHED("onehot_count_kernel", stream);
    const unsigned nscan = (unsigned)((V + kScanSpan - 1) / kScanSpan);
    hipLaunchKernelGGL(onehot_scan_totals_kernel, dim3(nscan), dim3(256), 0, stream, V, oh_cnt, oh_tot);
    PSPO_LAUNCHED("onehot_scan_totals_kernel", stream);
    hipLaunchKernelGGL(onehot_scan_offsets_kernel, dim3(1), dim3(256), 0, stream, (int)nscan, oh_tot, oh_nrows);
    PSPO_LAUNCHED("onehot_scan_offsets_kernel", stream);
    hipLaunchKernelGGL(onehot_scan_write_kernel, dim3(nscan), dim3(256), 0, stream, V, oh_cnt, oh_tot, oh_start,
                       oh_cursor, oh_rows);
    PSPO_LAUNCHED("onehot_scan_write_kernel", stream);
    hipLaunchKernelGGL(onehot_fill_kernel, dim3(gcols), dim3(256), 0, stream, N, n_act, act_tgt, oh_cursor, oh_tmp);
    PSPO_LAUNCHED("onehot_fill_kernel", stream);
    hipLaunchKernelGGL(onehot_rank_kernel, dim3(gcols), dim3(256), 0, stream, N, n_act, act_tgt, oh_start, oh_cnt,
                       oh_tmp, oh_sorted);
    PSPO_LAUNCHED("onehot_rank_kernel", stream);
    const int rows_bound = std::min(N, V);
    hipLaunchKernelGGL(onehot_dw_kernel, dim3((unsigned)((rows_bound + 3) / 4)), dim3(256), 0, stream, rows_bound, d,
                       oh_nrows, oh_rows, oh_start, oh_cnt, oh_sorted, act_idx, act_g1, hidden, d_w_head);
    PSPO_LAUNCHED("onehot_dw_kernel", stream);
    hipLaunchKernelGGL(onehot_dh_kernel, dim3((unsigned)((N + 3) / 4)), dim3(256), 0, stream, N, d, n_act, act_idx,
                       act_tgt, act_g1, w_head, d_hidden);
    PSPO_LAUNCHED("onehot_dh_kernel", stream);
  }
  return PSPO_OK;
}

}  // extern "C"
