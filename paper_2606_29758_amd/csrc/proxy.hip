// Output-head score proxy of the cutoff design, forward only (Sec. 3.3,
// Eq. gamma_proxy; App. D): for every completion token, under the old policy,
//
//   gamma = ||h||^2 * ||e_o - p||^2,   p = softmax(W h),  o = the generated token,
//
// the squared norm of the score of log p(o) with respect to the head W.  App. D
// evaluates ||e_o - p||^2 as 1 - 2 p(o) + ||p||^2 from two log-sum-exp
// reductions, lse(z) and lse(2z).  The kernels keep the same kind of second
// reduction but split off the target entry: per vocabulary tile, with the tile
// maximum m and e_v = exp(z_v - m),
//
//   S1 = sum_{v != o} e_v,   S2 = sum_{v != o} e_v^2,
//
// and after merging the tiles (with e_o = exp(z_o - M) at the common maximum M)
//
//   ||e_o - p||^2 = (1 - p(o))^2 + sum_{v != o} p_v^2 = (S1^2 + S2) / (S1 + e_o)^2,
//
// a sum of non-negative terms with no cancellation when p(o) -> 1 (where
// 1 - 2 p(o) + ||p||^2 in float32 would lose every digit).  ||p||^2 and
// log p(o) come out of the same sums.  The [N, V] logits are never stored.
#include <cmath>
#include <string>

#include "common.h"
#include "gemm.h"
#include "layout.h"
#include "rowdot.h"

namespace pspo {
namespace {

constexpr float kNegInf = -INFINITY;

// rows = vocabulary (A = W), columns = tokens (B = H).  Writes, per column and
// 384-row vocabulary tile, (m, S1, S2) over the tile's rows other than the
// column's target.  (The target logits come from row_dots_kernel: picking one
// accumulator per column out of the 48 a lane holds costs a compare and a
// select for each of them.)
// kFull: every row of every tile is a token id (no per-row mask); otherwise
// the launch is the partial last vocabulary tile, tm0 its index.  Two
// instantiations rather than a branch in one: with a branch the compiler
// spills accumulators.
template <bool kFull>
struct EpiProxy {
  int V, N;
  int64_t ldp;  // stride between vocabulary tiles in the partial arrays (= Npad)
  int tm0;
  const int32_t* target;
  float* part_m;
  float* part_s1;
  float* part_s2;

  __device__ __forceinline__ void apply(const AccTile& acc, int tm_launch, int tn, int wm, int wn, int,
                                        float* smem) const {
    float* red = smem;  // [2 wave rows][256 columns][m, S1, S2]
    // the lane index, recomputed here: otherwise the compiler keeps values
    // derived from the kernel's copy live across the product loop and spills one
    const int lane = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
    const int tm = kFull ? tm_launch : tm0 + tm_launch;
    const int vbase = tm * kTileM + acc_row(wm, 0, 0, lane);   // this lane's rows: vbase + i*16 + r
    // the targets of the lane's 8 columns, fetched together
    int tgts[kBlocksN];
#pragma unroll
    for (int j = 0; j < kBlocksN; ++j) {
      const int t = tn * kTileN + acc_col(wn, j, lane);
      tgts[j] = t < N ? target[t] : -1;
    }
#pragma unroll
    for (int j = 0; j < kBlocksN; ++j) asm volatile("" ::"v"(tgts[j]));   // keep the batch: no sinking
#pragma unroll
    for (int j = 0; j < kBlocksN; ++j) {
      const int cl = acc_col(wn, j, lane);
      const int tgt = tgts[j];
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
      float m, s1, s2;
      if constexpr (kFull) {
        // every row is a token id: three-input maxima, exp2(z log2e - m log2e)
        // as one fma + exp, the target's own entry selected away, four
        // partial sums of each kind
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
        float a1[4] = {0.f, 0.f, 0.f, 0.f}, a2[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < kBlocksM * kAccPerBlock; ++q) {
          float e = __builtin_amdgcn_exp2f(fmaf(x(q), kLog2e, -mb));
          e = vbase + (q >> 2) * 16 + (q & 3) != tgt ? e : 0.f;
          a1[q & 3] += e;
          a2[q & 3] = fmaf(e, e, a2[q & 3]);
        }
        s1 = (a1[0] + a1[1]) + (a1[2] + a1[3]);
        s2 = (a2[0] + a2[1]) + (a2[2] + a2[3]);
      } else {
        m = kNegInf;
#pragma unroll
        for (int i = 0; i < kBlocksM; ++i)
#pragma unroll
          for (int r = 0; r < kAccPerBlock; ++r)
            if (vbase + i * 16 + r < V) m = fmaxf(m, x(i * kAccPerBlock + r));
        m = fmaxf(m, __shfl_xor(m, 16));
        m = fmaxf(m, __shfl_xor(m, 32));
        s1 = 0.f;
        s2 = 0.f;
        if (m != kNegInf) {
#pragma unroll
          for (int i = 0; i < kBlocksM; ++i)
#pragma unroll
            for (int r = 0; r < kAccPerBlock; ++r) {
              const int v = vbase + i * 16 + r;
              // the target's own entry is left out (selected away, not subtracted)
              const float e = (v < V && v != tgt) ? __expf(x(i * kAccPerBlock + r) - m) : 0.f;
              s1 += e;
              s2 += e * e;
            }
        }
      }
      s1 += __shfl_xor(s1, 16);
      s1 += __shfl_xor(s1, 32);
      s2 += __shfl_xor(s2, 16);
      s2 += __shfl_xor(s2, 32);
      if (lane < 16) {
        float* o = red + (wm * kTileN + cl) * 3;
        o[0] = m;
        o[1] = s1;
        o[2] = s2;
      }
    }
    __syncthreads();
    const int c = threadIdx.x;
    const float* a = red + c * 3;
    const float* b = red + (kTileN + c) * 3;
    const float M = fmaxf(a[0], b[0]);
    float S1 = 0.f, S2 = 0.f;
    if (a[0] != kNegInf) {
      const float f = __expf(a[0] - M);
      S1 += a[1] * f;
      S2 += a[2] * f * f;
    }
    if (b[0] != kNegInf) {
      const float f = __expf(b[0] - M);
      S1 += b[1] * f;
      S2 += b[2] * f * f;
    }
    const int t = tn * kTileN + c;
    if (t < N) {
      part_m[tm * ldp + t] = M;
      part_s1[tm * ldp + t] = S1;
      part_s2[tm * ldp + t] = S2;
    }
  }
};

// Merge the vocabulary-tile partials of each token and form gamma, log p(o), ||p||^2.
__global__ __launch_bounds__(256) void proxy_finalize_kernel(int N, int V, int ntv, int64_t ldp,
                                                             const float* __restrict__ part_m,
                                                             const float* __restrict__ part_s1,
                                                             const float* __restrict__ part_s2,
                                                             const float* __restrict__ zt,
                                                             const float* __restrict__ hn,
                                                             const int32_t* __restrict__ target,
                                                             float* __restrict__ gamma, float* __restrict__ logp,
                                                             float* __restrict__ p_sq, int32_t* __restrict__ err_flag) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= N) return;
  const int tgt = target[t];
  if (tgt < 0 || tgt >= V) {
    gamma[t] = NAN;
    if (logp) logp[t] = NAN;
    if (p_sq) p_sq[t] = NAN;
    if (err_flag) atomicOr(err_flag, PSPO_DEVERR_TARGET);
    return;
  }
  float M = kNegInf;
  for (int k = 0; k < ntv; ++k) M = fmaxf(M, part_m[k * ldp + t]);
  float S1 = 0.f, S2 = 0.f;
  for (int k = 0; k < ntv; ++k) {
    const float m = part_m[k * ldp + t];
    if (m == kNegInf) continue;
    const float f = __expf(m - M);
    S1 += part_s1[k * ldp + t] * f;
    S2 += part_s2[k * ldp + t] * f * f;
  }
  const float et = expf(zt[t] - M);     // the target's entry (M >= z_o, so et <= 1)
  const float L = S1 + et;               // sum_v exp(z_v - M) >= 1
  const float inv = 1.f / L;
  gamma[t] = hn[t] * ((S1 * inv) * (S1 * inv) + S2 * inv * inv);
  if (logp) logp[t] = (zt[t] - M) - logf(L);
  if (p_sq) p_sq[t] = (S2 + et * et) * inv * inv;
}

struct ProxyPlan {
  int64_t Npad, Vpad, ntv;
  int64_t off_m, off_s1, off_s2, off_zt, off_hn, off_wk, off_hk, total;
};

ProxyPlan make_proxy_plan(int64_t N, int64_t d, int64_t V) {
  ProxyPlan p{};
  p.Npad = round_up(N > 0 ? N : 1, kTileN);
  p.Vpad = round_up(V, kTileM);
  p.ntv = p.Vpad / kTileM;
  int64_t o = 0;
  auto take = [&](int64_t bytes) {
    const int64_t at = o;
    o = round_up(o + bytes, 256);
    return at;
  };
  p.off_m = take(p.ntv * p.Npad * 4);
  p.off_s1 = take(p.ntv * p.Npad * 4);
  p.off_s2 = take(p.ntv * p.Npad * 4);
  p.off_zt = take(p.Npad * 4);
  p.off_hn = take(p.Npad * 4);
  const int64_t d64 = round_up(d, 64);   // columns the K-blocked copies write (zero past d)
  p.off_wk = take(d64 * p.Vpad * 2);     // W, K-blocked [d64/32][Vpad][32]
  p.off_hk = take(d64 * p.Npad * 2);     // hidden rows, K-blocked [d64/32][Npad][32]
  p.total = o;
  return p;
}

}  // namespace
}  // namespace pspo

extern "C" {

size_t pspo_score_proxy_workspace_bytes(int32_t N, int32_t d, int32_t V) {
  if (N < 0 || d <= 0 || V <= 0) return 0;
  return (size_t)pspo::make_proxy_plan(N, d, V).total;
}

int pspo_score_proxy(const uint16_t* hidden, const uint16_t* w_head, const int32_t* target, int32_t N, int32_t d,
                     int32_t V, float* gamma, float* logp, float* p_sq, int32_t* err_flag, void* workspace,
                     size_t workspace_bytes, hipStream_t stream) {
  using namespace pspo;
  clear_last_error();
  TraceRange trace_range("pspo_score_proxy");
  PSPO_REQUIRE(N >= 0, PSPO_ERR_INVALID_ARG, "N must be >= 0");
  PSPO_REQUIRE(d > 0 && V > 0, PSPO_ERR_INVALID_ARG, "d and V must be > 0");
  PSPO_REQUIRE(d % 8 == 0, PSPO_ERR_UNSUPPORTED, "d must be a multiple of 8");
  if (N == 0) return PSPO_OK;
  PSPO_REQUIRE(hidden && w_head && target && gamma, PSPO_ERR_INVALID_ARG, "null input or gamma pointer");
  PSPO_REQUIRE(aligned(hidden, 16) && aligned(w_head, 16), PSPO_ERR_INVALID_ARG,
               "hidden and w_head must be 16-byte aligned");
  PSPO_REQUIRE(aligned(target, 4) && aligned(gamma, 4) && aligned(logp, 4) && aligned(p_sq, 4),
               PSPO_ERR_INVALID_ARG, "misaligned per-token pointer");
  PSPO_REQUIRE(workspace != nullptr && aligned(workspace, 256), PSPO_ERR_INVALID_ARG,
               "workspace must be non-NULL and 256-byte aligned");
  const ProxyPlan pl = make_proxy_plan(N, d, V);
  PSPO_REQUIRE(pl.Npad <= kMaxPaddedRows && pl.Vpad <= kMaxPaddedRows && d <= kMaxPaddedRows,
               PSPO_ERR_UNSUPPORTED,
               "N, V and d must each be at most " + std::to_string(kMaxPaddedRows) + " rows after padding");
  PSPO_REQUIRE(workspace_bytes >= (size_t)pl.total, PSPO_ERR_WORKSPACE,
               "workspace too small: need " + std::to_string(pl.total) + " bytes");
  if (int rc = require_gfx950()) return rc;

  char* ws = static_cast<char*>(workspace);
  float* part_m = reinterpret_cast<float*>(ws + pl.off_m);
  float* part_s1 = reinterpret_cast<float*>(ws + pl.off_s1);
  float* part_s2 = reinterpret_cast<float*>(ws + pl.off_s2);
  float* zt = reinterpret_cast<float*>(ws + pl.off_zt);
  float* hn = reinterpret_cast<float*>(ws + pl.off_hn);
  uint16_t* wk = reinterpret_cast<uint16_t*>(ws + pl.off_wk);
  uint16_t* hk = reinterpret_cast<uint16_t*>(ws + pl.off_hk);

  const int tiles_tok = (int)(pl.Npad / kTileN);
  const int tiles_voc = (int)pl.ntv;
  const unsigned ctiles64 = (unsigned)((d + 63) / 64);
  const int Dk = (int)round_up(d, kTileK);   // K of the product: d with zero padding to whole K steps
  hipLaunchKernelGGL(kblock_rows_kernel, dim3(ctiles64, (unsigned)(pl.Vpad / 32)), dim3(256), 0, stream, w_head,
                     (int64_t)d, d, V, nullptr, nullptr, wk, pl.Vpad, nullptr, (int64_t)0, (int64_t)kTileK);
  PSPO_LAUNCHED("kblock_rows_kernel", stream);
  hipLaunchKernelGGL(kblock_rows_kernel, dim3(ctiles64, (unsigned)(pl.Npad / 32)), dim3(256), 0, stream, hidden,
                     (int64_t)d, d, N, nullptr, nullptr, hk, pl.Npad, nullptr, (int64_t)0, (int64_t)kTileK);
  PSPO_LAUNCHED("kblock_rows_kernel", stream);
  {
    // the vocabulary tiles whose rows are all token ids, then a partial last one
    ProductTimer timer(stream);
    if (int rc = timer.begin(PSPO_TIME_PROXY)) return rc;
    const int tiles_full = V / kTileM;
    if (tiles_full > 0) {
      GemmShape g{wk, pl.Vpad, tiles_full * kTileM, hk, pl.Npad, N, Dk, tiles_full, tiles_tok};
      EpiProxy<true> e{V, N, pl.Npad, 0, target, part_m, part_s1, part_s2};
      hipLaunchKernelGGL(gemm_nt_kernel<EpiProxy<true>>, dim3(gemm_grid(tiles_full, tiles_tok)), dim3(kGemmThreads),
                         0, stream, g, e);
      PSPO_LAUNCHED("gemm_nt_kernel (score proxy)", stream);
    }
    if (tiles_full < tiles_voc) {
      GemmShape g{wk + (int64_t)tiles_full * kTileM * kTileK, pl.Vpad, V - tiles_full * kTileM, hk, pl.Npad, N, Dk, 1,
                  tiles_tok};
      EpiProxy<false> e{V, N, pl.Npad, tiles_full, target, part_m, part_s1, part_s2};
      hipLaunchKernelGGL(gemm_nt_kernel<EpiProxy<false>>, dim3(gemm_grid(1, tiles_tok)), dim3(kGemmThreads), 0,
                         stream, g, e);
      PSPO_LAUNCHED("gemm_nt_kernel (score proxy)", stream);
    }
    if (int rc = timer.end()) return rc;
  }
  // the target logit and ||h||^2 of every token, one pass over its hidden row
  hipLaunchKernelGGL(row_dots_kernel, dim3((unsigned)((N + 3) / 4)), dim3(256), 0, stream, hidden, w_head, d, V, N,
                     nullptr, target, nullptr, zt, hn);
  PSPO_LAUNCHED("row_dots_kernel", stream);
  hipLaunchKernelGGL(proxy_finalize_kernel, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, stream, N, V,
                     tiles_voc, pl.Npad, part_m, part_s1, part_s2, zt, hn, target, gamma, logp, p_sq, err_flag);
  PSPO_LAUNCHED("proxy_finalize_kernel", stream);
  return PSPO_OK;
}

}  // extern "C"
