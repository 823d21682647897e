// Cutoff sampling and prefix packing (PS-PPO Sec. 3.2; Algorithm 1, the
// cutoff-sampling and prefix-reweighting steps of the update pass).
//
// Both are tiny next to the LM-head loss: one thread per completion draws its
// cutoff; packing is an exclusive scan over completions followed by a
// per-token fill and a 16-byte-vector gather of the kept hidden rows.
#include "common.h"

namespace pspo {
namespace {

constexpr double kTwo32 = 4294967296.0;

// Philox4x32-10 (Salmon et al., SC'11): ten rounds of two 32x32->64 multiplies
// with the Weyl key schedule.  Only output word 0 is needed.
__device__ __forceinline__ uint32_t philox_word0(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                 uint32_t k0, uint32_t k1) {
  constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  constexpr uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    if (round) {
      k0 += W0;
      k1 += W1;
    }
    const uint32_t hi0 = __umulhi(M0, c0), lo0 = M0 * c0;
    const uint32_t hi1 = __umulhi(M1, c2), lo1 = M1 * c2;
    const uint32_t n0 = hi1 ^ c1 ^ k0;
    const uint32_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return c0;
}

// Survival threshold q = max(1, floor(xi * 2^32)) (q = 2^32 for xi >= 1).
// xi * 2^32 is an exact power-of-two scaling; truncation of a value >= 1 is floor.
__device__ __forceinline__ uint64_t threshold(double xi) {
  const double s = xi * kTwo32;
  if (!(s >= 1.0)) return 1;               // also catches NaN (flagged by validation)
  if (s >= kTwo32) return 1ull << 32;
  return static_cast<uint64_t>(s);
}

// Flags tables that are not in (0,1] or increase along t.  grid.y = prompt.
__global__ void validate_xi_kernel(const double* __restrict__ xi, const int64_t* __restrict__ xi_off,
                                   int32_t* __restrict__ err_flag) {
  const int p = blockIdx.y;
  const int64_t b = xi_off[p], e = xi_off[p + 1];
  bool bad = false;
  for (int64_t i = b + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < e;
       i += (int64_t)gridDim.x * blockDim.x) {
    const double v = xi[i];
    bad |= !(v > 0.0 && v <= 1.0);
    if (i > b) bad |= v > xi[i - 1];
  }
  if (bad) atomicOr(err_flag, PSPO_DEVERR_BAD_XI);
}

// One thread per completion r = p*K + k: x_r = Philox word, then the largest
// t in [0, T_p] with x_r < q_{p,t} by binary search over the non-increasing
// thresholds (q_0 = 2^32 always admits t = 0), capped at the completion's length.
__global__ void sample_cutoffs_kernel(const double* __restrict__ xi, const int64_t* __restrict__ xi_off,
                                      const int32_t* __restrict__ lengths, int32_t R, int32_t K,
                                      uint32_t k0, uint32_t k1, uint32_t off_lo, uint32_t off_hi,
                                      int32_t* __restrict__ cutoffs) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= R) return;
  const int p = r / K;
  const int64_t base = xi_off[p];
  const int64_t Tp = xi_off[p + 1] - base;
  const uint64_t x = philox_word0((uint32_t)r, 0u, off_lo, off_hi, k0, k1);
  int64_t lo = 0, hi = Tp;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (x < threshold(xi[base + mid - 1])) lo = mid;
    else hi = mid - 1;
  }
  const int64_t Tr = lengths[r] > 0 ? lengths[r] : 0;
  cutoffs[r] = (int32_t)(lo < Tr ? lo : Tr);
}

// Exclusive scans of the cutoffs and of the lengths over all completions, in
// one work-group of 1024 threads walking the completions in chunks of 1024.
constexpr int kScanThreads = 1024;

__global__ __launch_bounds__(kScanThreads) void pack_scan_kernel(
    const int32_t* __restrict__ cutoffs, const int32_t* __restrict__ lengths, const int64_t* __restrict__ xi_off,
    int32_t R, int32_t K, int32_t capacity,
    int32_t* __restrict__ cu_seqlens, int32_t* __restrict__ full_off, int32_t* __restrict__ n_tokens,
    int32_t* __restrict__ err_flag) {
  __shared__ int64_t s_h[kScanThreads];
  __shared__ int64_t s_t[kScanThreads];
  int64_t carry_h = 0, carry_t = 0;
  const int tid = threadIdx.x;
  for (int base = 0; base < R; base += kScanThreads) {
    const int r = base + tid;
    int64_t T = 0, H = 0;
    if (r < R) {
      // a cutoff is capped at its completion's length and at its prompt's table horizon
      T = lengths[r] > 0 ? lengths[r] : 0;
      const int64_t Tp = xi_off[r / K + 1] - xi_off[r / K];
      const int64_t cap = T < Tp ? T : Tp;
      H = cutoffs[r] < 0 ? 0 : (cutoffs[r] > cap ? cap : cutoffs[r]);
    }
    s_h[tid] = H;
    s_t[tid] = T;
    __syncthreads();
    for (int off = 1; off < kScanThreads; off <<= 1) {  // Hillis-Steele inclusive scan
      int64_t ah = 0, at = 0;
      if (tid >= off) {
        ah = s_h[tid - off];
        at = s_t[tid - off];
      }
      __syncthreads();
      s_h[tid] += ah;
      s_t[tid] += at;
      __syncthreads();
    }
    if (r < R) {
      cu_seqlens[r + 1] = (int32_t)(carry_h + s_h[tid]);
      full_off[r + 1] = (int32_t)(carry_t + s_t[tid]);
    }
    carry_h += s_h[kScanThreads - 1];
    carry_t += s_t[kScanThreads - 1];
    __syncthreads();
  }
  if (tid == 0) {
    cu_seqlens[0] = 0;
    full_off[0] = 0;
    if (carry_h > capacity) {
      if (err_flag) atomicOr(err_flag, PSPO_DEVERR_CAPACITY);
      *n_tokens = capacity;
    } else {
      *n_tokens = (int32_t)carry_h;
    }
  }
}

// Per kept token: its source row, completion id, weight 2^32/q_{p,t} and the
// gathered target / old log-prob.  grid.y = completion, grid.x strides its tokens.
__global__ void pack_fill_kernel(const int32_t* __restrict__ cu_seqlens, const int32_t* __restrict__ full_off,
                                 const double* __restrict__ xi, const int64_t* __restrict__ xi_off,
                                 int32_t K, int32_t capacity, const int32_t* __restrict__ target_full,
                                 const float* __restrict__ logp_old_full, int32_t* __restrict__ src_row,
                                 int32_t* __restrict__ seq_id, float* __restrict__ weight,
                                 int32_t* __restrict__ target, float* __restrict__ logp_old) {
  const int r = blockIdx.y;
  const int p = r / K;
  const int32_t c0 = cu_seqlens[r], H = cu_seqlens[r + 1] - c0;
  const int32_t f0 = full_off[r];
  const int64_t xb = xi_off[p];
  for (int j = blockIdx.x * blockDim.x + threadIdx.x; j < H; j += gridDim.x * blockDim.x) {
    const int64_t i = (int64_t)c0 + j;
    if (i >= capacity) break;
    const int32_t src = f0 + j;
    src_row[i] = src;
    seq_id[i] = r;
    // 1/xi_t for timestep t = j+1, realised as float32(2^32 / double(q)) with an
    // IEEE (correctly rounded) float64 division.
    const double q = (double)threshold(xi[xb + j]);
    weight[i] = (float)(kTwo32 / q);
    if (target) target[i] = target_full[src];
    if (logp_old) logp_old[i] = logp_old_full[src];
  }
}

// Copies the kept hidden rows, one wave per row, 16 bytes per lane.
__global__ void pack_hidden_kernel(const int32_t* __restrict__ cu_seqlens, const int32_t* __restrict__ full_off,
                                   int32_t capacity, const u32x4* __restrict__ hidden_full,
                                   u32x4* __restrict__ hidden, int32_t vec_per_row) {
  const int r = blockIdx.y;
  const int32_t c0 = cu_seqlens[r], H = cu_seqlens[r + 1] - c0;
  const int32_t f0 = full_off[r];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int waves = blockDim.x >> 6;
  for (int j = blockIdx.x * waves + wave; j < H; j += gridDim.x * waves) {
    const int64_t i = (int64_t)c0 + j;
    if (i >= capacity) break;
    const u32x4* src = hidden_full + (int64_t)(f0 + j) * vec_per_row;
    u32x4* dst = hidden + i * vec_per_row;
    for (int c = lane; c < vec_per_row; c += 64) dst[c] = src[c];
  }
}

}  // namespace
}  // namespace pspo

extern "C" {

int pspo_sample_cutoffs(const double* xi, const int64_t* xi_off, const int32_t* lengths, int32_t P,
                        int32_t K, uint64_t seed, uint64_t offset, int32_t* cutoffs, int32_t* err_flag,
                        hipStream_t stream) {
  using namespace pspo;
  clear_last_error();
  TraceRange trace_range("pspo_sample_cutoffs");
  PSPO_REQUIRE(P >= 0 && K >= 0, PSPO_ERR_INVALID_ARG, "P and K must be >= 0");
  PSPO_REQUIRE((int64_t)P * K <= INT32_MAX, PSPO_ERR_INVALID_ARG, "P*K overflows int32");
  const int32_t R = P * K;
  if (R == 0) return PSPO_OK;
  PSPO_REQUIRE(xi && xi_off && lengths && cutoffs, PSPO_ERR_INVALID_ARG, "null pointer argument");
  PSPO_REQUIRE(aligned(xi, 8) && aligned(xi_off, 8) && aligned(lengths, 4) && aligned(cutoffs, 4),
               PSPO_ERR_INVALID_ARG, "misaligned pointer argument");
  if (int rc = require_gfx950()) return rc;
  if (err_flag) {
    hipLaunchKernelGGL(validate_xi_kernel, dim3(4, P), dim3(256), 0, stream, xi, xi_off, err_flag);
    PSPO_LAUNCHED("validate_xi_kernel", stream);
  }
  hipLaunchKernelGGL(sample_cutoffs_kernel, dim3((R + 255) / 256), dim3(256), 0, stream, xi, xi_off, lengths,
                     R, K, (uint32_t)seed, (uint32_t)(seed >> 32), (uint32_t)offset, (uint32_t)(offset >> 32),
                     cutoffs);
  PSPO_LAUNCHED("sample_cutoffs_kernel", stream);
  return PSPO_OK;
}

int pspo_pack_prefixes(const int32_t* cutoffs, const int32_t* lengths, const double* xi, const int64_t* xi_off,
                       int32_t P, int32_t K, int32_t capacity, const int32_t* target_full,
                       const float* logp_old_full, const uint16_t* hidden_full, int32_t d, int32_t* cu_seqlens,
                       int32_t* full_off, int32_t* src_row, int32_t* seq_id, float* weight, int32_t* target,
                       float* logp_old, uint16_t* hidden, int32_t* n_tokens, int32_t* err_flag,
                       hipStream_t stream) {
  using namespace pspo;
  clear_last_error();
  TraceRange trace_range("pspo_pack_prefixes");
  PSPO_REQUIRE(P >= 0 && K >= 0 && capacity >= 0, PSPO_ERR_INVALID_ARG, "P, K and capacity must be >= 0");
  PSPO_REQUIRE((int64_t)P * K <= 65535, PSPO_ERR_UNSUPPORTED, "packing supports at most 65535 completions");
  const int32_t R = P * K;
  PSPO_REQUIRE(cu_seqlens && full_off && n_tokens, PSPO_ERR_INVALID_ARG, "null output pointer");
  PSPO_REQUIRE((target_full == nullptr) == (target == nullptr), PSPO_ERR_INVALID_ARG,
               "target and target_full must be both given or both NULL");
  PSPO_REQUIRE((logp_old_full == nullptr) == (logp_old == nullptr), PSPO_ERR_INVALID_ARG,
               "logp_old and logp_old_full must be both given or both NULL");
  PSPO_REQUIRE((hidden_full == nullptr) == (hidden == nullptr), PSPO_ERR_INVALID_ARG,
               "hidden and hidden_full must be both given or both NULL");
  if (R > 0) {
    PSPO_REQUIRE(cutoffs && lengths && xi && xi_off, PSPO_ERR_INVALID_ARG, "null input pointer");
    PSPO_REQUIRE(capacity == 0 || (src_row && seq_id && weight), PSPO_ERR_INVALID_ARG, "null output pointer");
  }
  if (hidden_full) {
    PSPO_REQUIRE(d > 0 && d % 8 == 0, PSPO_ERR_UNSUPPORTED, "hidden gather needs d > 0 and d % 8 == 0");
    PSPO_REQUIRE(aligned(hidden_full, 16) && aligned(hidden, 16), PSPO_ERR_INVALID_ARG,
                 "hidden buffers must be 16-byte aligned");
  }
  if (int rc = require_gfx950()) return rc;
  hipLaunchKernelGGL(pack_scan_kernel, dim3(1), dim3(kScanThreads), 0, stream, cutoffs, lengths, xi_off, R, K,
                     capacity, cu_seqlens, full_off, n_tokens, err_flag);
  PSPO_LAUNCHED("pack_scan_kernel", stream);
  if (R == 0 || capacity == 0) return PSPO_OK;
  hipLaunchKernelGGL(pack_fill_kernel, dim3(16, R), dim3(256), 0, stream, cu_seqlens, full_off, xi, xi_off, K,
                     capacity, target_full, logp_old_full, src_row, seq_id, weight, target, logp_old);
  PSPO_LAUNCHED("pack_fill_kernel", stream);
  if (hidden_full) {
    hipLaunchKernelGGL(pack_hidden_kernel, dim3(64, R), dim3(256), 0, stream, cu_seqlens, full_off, capacity,
                       reinterpret_cast<const u32x4*>(hidden_full), reinterpret_cast<u32x4*>(hidden), d / 8);
    PSPO_LAUNCHED("pack_hidden_kernel", stream);
  }
  return PSPO_OK;
}

}  // extern "C"
