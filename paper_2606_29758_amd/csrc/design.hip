// Cutoff design of PS-PPO ("Computing xi" of Algorithm 1; Sec. 3.3, App. E, F).
//
// Weights.  For prompt p (completions r = pK .. pK+K-1, lengths T_r,
// T_p = max_r T_r) and step t = 1..T_p, over the n_t completions alive at t
// (T_r >= t):
//   gbar_t = (1/n_t) sum_r gamma_r(t)                 (output-head score proxy, App. D)
//   u_t    = 1/2 - 1/(2 n_t) || sum_{r in G_t} pi_r(.|t) - sum_{r in B_t} pi_r(.|t) ||_1
//            (reward-uncertainty proxy, App. E, with p = |G_t|/n_t; G_t / B_t the
//            successful / unsuccessful completions)
//   w_t    = gbar_t u_t.
// Each pi_r(.|t) is given by its top-k entries (token id, log-prob); the mass
// left outside them is one further coordinate shared by every completion.
//
// Design.  Per prompt, minimise sum_t w_t / xi_t subject to sum_t xi_t = B and
// 1 >= xi_1 >= ... >= xi_T > 0 (Eq. design_problem): Pooling Adjacent
// Violators builds contiguous blocks with non-increasing scores
// s_m = sqrt(W_m / L_m) (App. F); the optimum is xi = min(1, kappa s_m), the
// cap saturating a prefix of blocks and kappa spending the rest of the budget
// on the others.  Variants: Heuristic (the unconstrained closed form
// B sqrt(w_t) / sum_j sqrt(w_j), capped, then a running minimum), Uniform
// (H uniform on 1..T) and Time prior (xi_t = exp(-lambda (t-1))).  Every xi is
// floored at 2^-32, the resolution of the sampler's thresholds.
//
// Both kernels work in float64; their cost is small next to the proxy's
// forward pass (a few operations per completion token and per step; the
// design's sequential solve reads LDS-resident weights and block stack).
#include <cmath>
#include <mutex>
#include <string>

#include "common.h"

namespace pspo {
namespace {

constexpr int kDesignMaxEntries = 256;   // K * topk per step
constexpr double kXiFloor = 0x1p-32;

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// One wave per (prompt, step); 4 waves per block.
__global__ __launch_bounds__(256) void design_weights_kernel(
    const float* __restrict__ gamma, const int32_t* __restrict__ topk_ids, const float* __restrict__ topk_logp,
    int topk, const int32_t* __restrict__ lengths, const int32_t* __restrict__ full_off,
    const float* __restrict__ rewards, const int64_t* __restrict__ xi_off, int P, int K, int64_t total,
    double* __restrict__ w, double* __restrict__ gbar_out, double* __restrict__ u_out, int32_t* __restrict__ err_flag) {
  __shared__ int32_t sid[4][kDesignMaxEntries];
  __shared__ double sval[4][kDesignMaxEntries];
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t g = (int64_t)blockIdx.x * 4 + wv;
  const bool live = g < total;   // a wave past the end still takes part in the barrier
  // prompt of g: the last p with xi_off[p] <= g
  int lo = 0, hi = P - 1;
  while (live && lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (xi_off[mid] <= g) lo = mid;
    else hi = mid - 1;
  }
  const int p = lo;
  const int t = live ? (int)(g - xi_off[p]) + 1 : 0;

  // per-entry signed probabilities of the alive completions (0 for the others)
  const int ne = live ? K * topk : 0;
  for (int j = lane; j < ne; j += 64) {
    const int k = j / topk, r = p * K + k;
    int32_t id = -1;
    double v = 0.0;
    if (lengths[r] >= t) {
      const int64_t row = (int64_t)full_off[r] + t - 1;
      id = topk_ids[row * topk + (j - k * topk)];
      v = exp((double)topk_logp[row * topk + (j - k * topk)]) * (rewards[r] > 0.5f ? 1.0 : -1.0);
    }
    sid[wv][j] = id;
    sval[wv][j] = v;
  }
  __syncthreads();
  // each distinct token id is summed once, by the lane that holds its first occurrence
  double l1 = 0.0;
  for (int j = lane; j < ne; j += 64) {
    const int32_t id = sid[wv][j];
    if (id < 0) continue;
    bool first = true;
    for (int i = 0; i < j && first; ++i) first = sid[wv][i] != id;
    if (!first) continue;
    double s = 0.0;
    for (int i = j; i < ne; ++i)
      if (sid[wv][i] == id) s += sval[wv][i];
    l1 += fabs(s);
  }
  // per completion: the mass outside its top-k, and its gamma
  double rest = 0.0, gsum = 0.0, nalive = 0.0, nsucc = 0.0;
  if (live && lane < K) {
    const int r = p * K + lane;
    if (lengths[r] >= t) {
      const int64_t row = (int64_t)full_off[r] + t - 1;
      double mass = 0.0;
      for (int e = 0; e < topk; ++e) mass += exp((double)topk_logp[row * topk + e]);
      const bool ok = rewards[r] > 0.5f;
      rest = fmax(0.0, 1.0 - mass) * (ok ? 1.0 : -1.0);
      gsum = (double)gamma[row];
      nalive = 1.0;
      nsucc = ok ? 1.0 : 0.0;
    }
  }
  l1 = wave_sum(l1);
  rest = wave_sum(rest);
  gsum = wave_sum(gsum);
  nalive = wave_sum(nalive);
  nsucc = wave_sum(nsucc);
  if (live && lane == 0) {
    if (nalive == 0.0) {   // the table is longer than every completion of the prompt
      if (err_flag) atomicOr(err_flag, PSPO_DEVERR_BAD_XI);
      w[g] = NAN;
      return;
    }
    const double gb = gsum / nalive;
    // equal rewards among the alive completions: p is 0 or 1 and the norm is exactly 1,
    // so u = 0 (taken exactly); otherwise ||.||_1 <= 1 by the triangle inequality, so
    // u >= 0 and rounding below it is clamped
    const double u = (nsucc == 0.0 || nsucc == nalive) ? 0.0 : fmax(0.0, 0.5 - 0.5 * (l1 + fabs(rest)) / nalive);
    w[g] = gb * u;
    if (gbar_out) gbar_out[g] = gb;
    if (u_out) u_out[g] = u;
  }
}

// The budgeted monotone solve of one prompt (App. F) on the storage given: wr
// the weights, wv / ln the block stack (summed weight and length of each
// block), rest the suffix sums (it may alias wr: the weights are not read
// after the pooling).  Force-inlined at each call with pointers of one memory
// kind, so that LDS-resident data is read and written by LDS instructions
// rather than generic ones.  Called by all 64 lanes of the block's one wave:
// lane 0 pools, the lanes compute the block scores, lane 0 does the rest.
__device__ __forceinline__ void pav_solve(const double* wr, double* wv, int32_t* ln, double* rest, int T,
                                          double budget, double* xp) {
  const int lane = threadIdx.x;
  int M = 0;                       // blocks under the top, then all blocks
  if (lane == 0) {
    // Pooling Adjacent Violators: a stack of blocks (start, length, summed
    // weight); a new element pools with the block below it while that block's
    // score sqrt(W / L) is below its own.  Scores of positive lengths are in the
    // order of the mean weights, and tw / tl < W / L exactly when tw L < W tl, so
    // each step compares two products: no division or root per step (a product
    // rounds to 2^-53 relative, so the decision can differ from the exact one
    // only for blocks whose means agree to that; pooling or not such a pair
    // moves the table by the same relative amount).  The top block stays in
    // registers (the stack holds the blocks under it), so an element that does
    // not pool costs no stack access.
    // A block's start is not stored: the block under the top ends where the top
    // starts.
    int ts = 0, tl = 1;              // the top block
    double tw = wr[0];
    double w_next = T > 1 ? wr[1] : 0.0;   // each step's weight is read one step ahead
    for (int t = 1; t < T; ++t) {
      int s0 = t, L = 1;
      double W = w_next;
      if (t + 1 < T) w_next = wr[t + 1];
      bool top = true;
      while (top && tw * (double)L < W * (double)tl) {   // pool the top into the new block
        s0 = ts;
        L += tl;
        W = tw + W;
        if (M > 0) {
          --M;
          tl = ln[M];
          tw = wv[M];
          ts = s0 - tl;
        } else {
          top = false;
        }
      }
      if (top) {                     // the old top goes under the new block
        ln[M] = tl;
        wv[M] = tw;
        ++M;
      }
      ts = s0;
      tl = L;
      tw = W;
    }
    ln[M] = tl;
    wv[M] = tw;
    ++M;
  }
  M = __shfl(M, 0);
  __syncthreads();   // lane 0's stack is visible to every lane
  // the block scores sqrt(W_m / L_m), spread over the lanes
  for (int m = lane; m < M; m += 64) wv[m] = sqrt(wv[m] / (double)ln[m]);
  __syncthreads();
  if (lane != 0) return;
  // suffix sums of L_m s_m (accumulated from the last block)
  // first unsaturated block: kappa(m) = (B - sum_{j<m} L_j) / sum_{j>=m} L_j s_j, kappa(m) s_m <= 1
  double acc = 0.0;
  for (int m = M - 1; m >= 0; --m) {
    acc += (double)ln[m] * wv[m];
    rest[m] = acc;
  }
  int saturated = 0;
  double kappa = -1.0;   // < 0: only zero-weight blocks remain unsaturated
  for (int m = 0; m < M; ++m) {
    if (rest[m] == 0.0) {
      kappa = -1.0;
      break;
    }
    kappa = (budget - (double)saturated) / rest[m];
    if (kappa * wv[m] <= 1.0) break;
    saturated += ln[m];
  }
  for (int m = 0, start = 0; m < M; start += ln[m], ++m) {
    double v;
    if (kappa < 0.0) v = (start < saturated) ? 1.0 : (budget - (double)saturated) / (double)(T - saturated);
    else v = fmin(1.0, kappa * wv[m]);
    v = fmax(v, kXiFloor);
    for (int t = start; t < start + ln[m]; ++t) xp[t] = v;
  }
}

// LDS of one design block: the prompt's weights (8 bytes per step) and, when
// they fit as well, the PAV block stack (12 bytes per step: summed weight and
// length).
constexpr int kDesignLdsBytes = 160 * 1024;

// One block of 64 threads (one wave) per prompt: the lanes stage the prompt's
// weights in LDS, check them and sum their square roots; lane 0 then runs the
// sequential solve on LDS-resident data (the weights when T <= 20480, the
// block stack too when T <= 8192; otherwise from the workspace).
__global__ __launch_bounds__(64) void design_cutoffs_kernel(const double* __restrict__ w,
                                                            const int64_t* __restrict__ xi_off, double budget,
                                                            int variant, double lambda, double* __restrict__ xi,
                                                            int32_t* __restrict__ blen,
                                                            double* __restrict__ bval, int32_t* __restrict__ err_flag) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[kDesignLdsBytes];
  const int p = blockIdx.x;
  const int64_t a = xi_off[p];
  const int T = (int)(xi_off[p + 1] - a);
  const double* wp = w + a;
  double* xp = xi + a;
  if (variant == PSPO_DESIGN_UNIFORM) {
    for (int t = threadIdx.x; t < T; t += blockDim.x) xp[t] = (double)(T - t) / (double)T;
    return;
  }
  if (variant == PSPO_DESIGN_TIME_PRIOR) {
    for (int t = threadIdx.x; t < T; t += blockDim.x) xp[t] = fmax(exp(-lambda * (double)t), kXiFloor);
    return;
  }
  const bool w_in_lds = (int64_t)T * 8 <= kDesignLdsBytes;
  const bool stack_in_lds = (int64_t)T * 20 <= kDesignLdsBytes;
  double* wl = reinterpret_cast<double*>(lds);
  bool bad_lane = false;
  double part = 0.0;   // this lane's steps t = lane, lane + 64, ... in order
  for (int t = threadIdx.x; t < T; t += 64) {
    const double v = wp[t];
    if (w_in_lds) wl[t] = v;
    if (!(v >= 0.0) || isinf(v)) bad_lane = true;
    else part += sqrt(v);
  }
  const bool bad = __ballot(bad_lane) != 0;
  const double root_sum = wave_sum(part);   // the lanes' partial sums in a fixed butterfly order
  __syncthreads();
  const double* wr = w_in_lds ? wl : wp;
  const bool single = bad || budget >= (double)T || root_sum == 0.0 || variant == PSPO_DESIGN_HEURISTIC;
  if (single && threadIdx.x != 0) return;
  if (bad) {
    if (err_flag) atomicOr(err_flag, PSPO_DEVERR_BAD_XI);
    for (int t = 0; t < T; ++t) xp[t] = NAN;
    return;
  }
  if (budget >= (double)T) {
    for (int t = 0; t < T; ++t) xp[t] = 1.0;
    return;
  }
  if (root_sum == 0.0) {   // every weight zero: any feasible table is optimal
    for (int t = 0; t < T; ++t) xp[t] = budget / (double)T;
    return;
  }
  if (variant == PSPO_DESIGN_HEURISTIC) {
    double run = 1.0;
    for (int t = 0; t < T; ++t) {
      run = fmin(run, fmin(1.0, budget * sqrt(wr[t]) / root_sum));
      xp[t] = fmax(run, kXiFloor);
    }
    return;
  }
  // the solve, on LDS-resident weights and stack where they fit
  if (stack_in_lds)
    pav_solve(wl, reinterpret_cast<double*>(lds + (int64_t)T * 8), reinterpret_cast<int32_t*>(lds + (int64_t)T * 16),
              wl, T, budget, xp);
  else if (w_in_lds)
    pav_solve(wl, bval + a, blen + a, wl, T, budget, xp);
  else
    pav_solve(wp, bval + a, blen + a, xp, T, budget, xp);
}

// Argument checks shared by the design entry points (host only).
int check_design_args(const double* w, const int64_t* xi_off, int32_t P, int64_t total_T, double budget,
                      int32_t variant, double lambda, const double* xi) {
  PSPO_REQUIRE(P >= 1 && total_T >= 0, PSPO_ERR_INVALID_ARG, "need P >= 1 and total_T >= 0");
  PSPO_REQUIRE(variant >= PSPO_DESIGN_OPTIMIZED && variant <= PSPO_DESIGN_TIME_PRIOR, PSPO_ERR_INVALID_ARG,
               "unknown design variant");
  PSPO_REQUIRE(std::isfinite(budget) && budget > 0.0, PSPO_ERR_INVALID_ARG, "budget must be finite and > 0");
  PSPO_REQUIRE(std::isfinite(lambda) && lambda >= 0.0, PSPO_ERR_INVALID_ARG, "lambda must be finite and >= 0");
  if (total_T == 0) return PSPO_OK;
  PSPO_REQUIRE(w && xi_off && xi, PSPO_ERR_INVALID_ARG, "null pointer");
  PSPO_REQUIRE(aligned(w, 8) && aligned(xi_off, 8) && aligned(xi, 8), PSPO_ERR_INVALID_ARG,
               "misaligned pointer");
  return PSPO_OK;
}

// The PAV block stack of the prompts whose stack does not fit in LDS (length
// and summed weight per block, at most one block per step) carved from `ws`
// (pspo_design_workspace_bytes(total_T), whose first 4 bytes per step are
// spare), then the solve.  The kernel writes every stack entry before reading
// it, so the memory needs no clearing.
int launch_design(const double* w, const int64_t* xi_off, int32_t P, int64_t total_T, double budget, int32_t variant,
                  double lambda, double* xi, char* ws, int32_t* err_flag, hipStream_t stream) {
  int32_t* blen = reinterpret_cast<int32_t*>(ws + round_up(total_T * 4, 256));
  double* bval = reinterpret_cast<double*>(ws + 2 * round_up(total_T * 4, 256));
  hipLaunchKernelGGL(design_cutoffs_kernel, dim3((unsigned)P), dim3(64), 0, stream, w, xi_off, budget, variant,
                     lambda, xi, blen, bval, err_flag);
  PSPO_LAUNCHED("design_cutoffs_kernel", stream);
  return PSPO_OK;
}

}  // namespace

// Scratch of the no-allocation entry point: a file-scope device array, one copy
// per GPU, held until the process ends.  Host code never uses its name as an
// address (on the host it is a stand-in symbol): the device address comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t kNoAllocScratchBytes = size_t(8) << 20;   // total_T <= 2^19 steps
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch[kMaxDevices] = {};

// The current device's address of `scratch` (looked up on the first call on
// that device).
int scratch_address(char** out) {
  int dev = 0;
  PSPO_HIP_CHECK(hipGetDevice(&dev));
  PSPO_REQUIRE(dev >= 0 && dev < kMaxDevices, PSPO_ERR_UNSUPPORTED, "device id out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    PSPO_HIP_CHECK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    PSPO_REQUIRE(p != nullptr && aligned(p, 256), PSPO_ERR_HIP, "scratch has no usable device address");
    g_scratch[dev] = static_cast<char*>(p);
  }
  *out = g_scratch[dev];
  return PSPO_OK;
}

}  // namespace
}  // namespace pspo

extern "C" {

int pspo_design_weights(const float* gamma, const int32_t* topk_ids, const float* topk_logp, int32_t topk,
                        const int32_t* lengths, const int32_t* full_off, const float* rewards, const int64_t* xi_off,
                        int32_t P, int32_t K, int64_t total_T, double* w, double* gamma_bar, double* u,
                        int32_t* err_flag, hipStream_t stream) {
  using namespace pspo;
  clear_last_error();
  TraceRange trace_range("pspo_design_weights");
  PSPO_REQUIRE(P >= 1 && K >= 1 && total_T >= 0, PSPO_ERR_INVALID_ARG, "need P >= 1, K >= 1, total_T >= 0");
  PSPO_REQUIRE(K <= 64, PSPO_ERR_UNSUPPORTED, "K must be <= 64");
  PSPO_REQUIRE(topk >= 1 && (int64_t)K * topk <= kDesignMaxEntries, PSPO_ERR_UNSUPPORTED,
               "need topk >= 1 and K * topk <= 256");
  if (total_T == 0) return PSPO_OK;
  PSPO_REQUIRE(gamma && topk_ids && topk_logp && lengths && full_off && rewards && xi_off && w, PSPO_ERR_INVALID_ARG,
               "null pointer");
  PSPO_REQUIRE(aligned(w, 8) && aligned(gamma_bar, 8) && aligned(u, 8) && aligned(xi_off, 8), PSPO_ERR_INVALID_ARG,
               "misaligned float64 / int64 pointer");
  if (int rc = require_gfx950()) return rc;
  const int64_t blocks = (total_T + 3) / 4;
  PSPO_REQUIRE(blocks <= INT32_MAX, PSPO_ERR_UNSUPPORTED, "problem too large");
  hipLaunchKernelGGL(design_weights_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, gamma, topk_ids, topk_logp,
                     topk, lengths, full_off, rewards, xi_off, P, K, total_T, w, gamma_bar, u, err_flag);
  PSPO_LAUNCHED("design_weights_kernel", stream);
  return PSPO_OK;
}

size_t pspo_design_workspace_bytes(int64_t total_T) {
  using pspo::round_up;
  if (total_T < 0) return 0;
  return (size_t)(round_up(total_T * 4, 256) * 2 + round_up(total_T * 8, 256));
}

int pspo_design_cutoffs(const double* w, const int64_t* xi_off, int32_t P, int64_t total_T, double budget,
                        int32_t variant, double lambda, double* xi, void* workspace, size_t workspace_bytes,
                        int32_t* err_flag, hipStream_t stream) {
  using namespace pspo;
  clear_last_error();
  TraceRange trace_range("pspo_design_cutoffs");
  if (int rc = check_design_args(w, xi_off, P, total_T, budget, variant, lambda, xi)) return rc;
  if (total_T == 0) return PSPO_OK;
  PSPO_REQUIRE(workspace && aligned(workspace, 256), PSPO_ERR_INVALID_ARG,
               "workspace must be non-NULL and 256-byte aligned");
  PSPO_REQUIRE(workspace_bytes >= pspo_design_workspace_bytes(total_T), PSPO_ERR_WORKSPACE,
               "workspace too small: need " + std::to_string(pspo_design_workspace_bytes(total_T)) + " bytes");
  if (int rc = require_gfx950()) return rc;
  return launch_design(w, xi_off, P, total_T, budget, variant, lambda, xi, static_cast<char*>(workspace), err_flag,
                       stream);
}

int pspo_design_cutoffs_noalloc(const double* w, const int64_t* xi_off, int32_t P, int64_t total_T, double budget,
                                int32_t variant, double lambda, double* xi, int32_t* err_flag, hipStream_t stream) {
  using namespace pspo;
  clear_last_error();
  TraceRange trace_range("pspo_design_cutoffs_noalloc");
  if (int rc = check_design_args(w, xi_off, P, total_T, budget, variant, lambda, xi)) return rc;
  if (total_T == 0) return PSPO_OK;
  PSPO_REQUIRE(pspo_design_workspace_bytes(total_T) <= kNoAllocScratchBytes, PSPO_ERR_UNSUPPORTED,
               "total_T = " + std::to_string(total_T) + " needs " +
                   std::to_string(pspo_design_workspace_bytes(total_T)) + " bytes of scratch; the no-allocation "
                   "entry point has " + std::to_string(kNoAllocScratchBytes) + " (total_T <= 2^19)");
  if (int rc = require_gfx950()) return rc;
  char* ws = nullptr;
  if (int rc = scratch_address(&ws)) return rc;
  return launch_design(w, xi_off, P, total_T, budget, variant, lambda, xi, ws, err_flag, stream);
}

}  // extern "C"
