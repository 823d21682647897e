// One update pass of the PS-PPO hot path through libpspo's C ABI from C++
// alone: no Python, no torch.  Device buffers come from hipMalloc, the work
// runs on a stream of the program's own, and the library is linked like any
// shared library.  The program makes a small seeded batch (3 prompts x 4
// completions, d = 200, V = 3001: a width that is no multiple of 64 and a
// vocabulary that ends in a partial tile), samples the cutoffs, packs the
// prefixes, runs the loss with its gradients, and writes the inputs and the
// outputs as raw arrays into the directory given on the command line, where
// tests/test_gpu_abi_example.py checks them against the float64 oracle.
//
//   abi_example <output directory>
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "pspo.h"

#define HIP_CALL(x)                                                          \
  do {                                                                       \
    hipError_t e_ = (x);                                                     \
    if (e_ != hipSuccess) {                                                  \
      std::fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));           \
      return 2;                                                              \
    }                                                                        \
  } while (0)

#define PSPO_CALL(x)                                                                                  \
  do {                                                                                                \
    int s_ = (x);                                                                                     \
    if (s_ != PSPO_OK) {                                                                              \
      std::fprintf(stderr, "%s: %s: %s\n", #x, pspo_status_string(s_), pspo_last_error());            \
      return 3;                                                                                       \
    }                                                                                                 \
  } while (0)

namespace {

// A 64-bit linear congruential generator (Knuth's MMIX constants); inputs only.
struct Lcg {
  uint64_t s;
  uint32_t next() {
    s = s * 6364136223846793005ULL + 1442695040888963407ULL;
    return static_cast<uint32_t>(s >> 32);
  }
  double uniform() { return (next() + 0.5) / 4294967296.0; }           // (0, 1)
  double normal() {                                                     // Box-Muller
    const double u = uniform(), v = uniform();
    return std::sqrt(-2.0 * std::log(u)) * std::cos(6.283185307179586 * v);
  }
};

uint16_t to_bf16(float f) {   // round to nearest even (finite values)
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

template <class T>
bool save(const std::string& dir, const char* name, const T* data, size_t n) {
  FILE* f = std::fopen((dir + "/" + name).c_str(), "wb");
  if (!f) return false;
  const bool ok = std::fwrite(data, sizeof(T), n, f) == n;
  return std::fclose(f) == 0 && ok;
}

template <class T>
T* device_copy(const std::vector<T>& v, hipError_t* err) {
  T* p = nullptr;
  *err = hipMalloc(&p, v.size() * sizeof(T) + 16);
  if (*err == hipSuccess) *err = hipMemcpy(p, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice);
  return p;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 2) {
    std::fprintf(stderr, "usage: %s <output directory>\n", argv[0]);
    return 1;
  }
  const std::string dir = argv[1];
  const int P = 3, K = 4, R = P * K, d = 200, V = 3001;
  const uint64_t seed = 11, offset = 5;
  const float eps_low = 0.2f, eps_high = 0.28f, loss_scale = 1.0f / R;
  Lcg rng{2024};

  // batch: lengths, survival tables over each prompt's longest completion,
  // rewards -> group-centred advantages, hidden rows, head, targets, old log-probs
  std::vector<int32_t> lengths(R);
  for (int r = 0; r < R; ++r) lengths[r] = 20 + static_cast<int32_t>(rng.next() % 100);
  std::vector<int64_t> xi_off(P + 1, 0);
  std::vector<double> xi;
  for (int p = 0; p < P; ++p) {
    int T = 0;
    for (int k = 0; k < K; ++k) T = lengths[p * K + k] > T ? lengths[p * K + k] : T;
    for (int t = 1; t <= T; ++t) xi.push_back(1.0 - 0.9 * (t - 1) / T);   // in (0, 1], non-increasing
    xi_off[p + 1] = xi_off[p] + T;
  }
  std::vector<float> adv(R);
  for (int p = 0; p < P; ++p) {
    float rw[K], mean = 0.f;
    for (int k = 0; k < K; ++k) mean += (rw[k] = static_cast<float>(rng.next() & 1u)) / K;
    for (int k = 0; k < K; ++k) adv[p * K + k] = rw[k] - mean;
  }
  int32_t total = 0;
  for (int r = 0; r < R; ++r) total += lengths[r];
  std::vector<uint16_t> hidden(static_cast<size_t>(total) * d), w(static_cast<size_t>(V) * d);
  for (auto& x : hidden) x = to_bf16(static_cast<float>(rng.normal()));
  for (auto& x : w) x = to_bf16(static_cast<float>(0.05 * rng.normal()));
  std::vector<int32_t> target(total);
  std::vector<float> logp_old(total);
  for (int i = 0; i < total; ++i) {
    target[i] = static_cast<int32_t>(rng.next() % V);
    logp_old[i] = static_cast<float>(-std::log(static_cast<double>(V)) + 0.15 * rng.normal());
  }

  hipError_t err = hipSuccess;
  hipStream_t stream;
  HIP_CALL(hipStreamCreate(&stream));
  double* d_xi = device_copy(xi, &err);
  HIP_CALL(err);
  int64_t* d_xi_off = device_copy(xi_off, &err);
  HIP_CALL(err);
  int32_t* d_lengths = device_copy(lengths, &err);
  HIP_CALL(err);
  float* d_adv = device_copy(adv, &err);
  HIP_CALL(err);
  uint16_t* d_hidden_full = device_copy(hidden, &err);
  HIP_CALL(err);
  uint16_t* d_w = device_copy(w, &err);
  HIP_CALL(err);
  int32_t* d_target_full = device_copy(target, &err);
  HIP_CALL(err);
  float* d_logp_old_full = device_copy(logp_old, &err);
  HIP_CALL(err);

  int32_t *d_cutoffs, *d_cu, *d_full_off, *d_src, *d_seq, *d_tgt, *d_n, *d_err;
  float *d_weight, *d_lpo, *d_logp, *d_dh, *d_dw;
  uint16_t* d_hid;
  double *d_loss, *d_stats;
  HIP_CALL(hipMalloc(&d_cutoffs, R * 4));
  HIP_CALL(hipMalloc(&d_cu, (R + 1) * 4));
  HIP_CALL(hipMalloc(&d_full_off, (R + 1) * 4));
  HIP_CALL(hipMalloc(&d_src, total * 4));
  HIP_CALL(hipMalloc(&d_seq, total * 4));
  HIP_CALL(hipMalloc(&d_tgt, total * 4));
  HIP_CALL(hipMalloc(&d_weight, total * 4));
  HIP_CALL(hipMalloc(&d_lpo, total * 4));
  HIP_CALL(hipMalloc(&d_hid, static_cast<size_t>(total) * d * 2));
  HIP_CALL(hipMalloc(&d_n, 4));
  HIP_CALL(hipMalloc(&d_err, 4));
  HIP_CALL(hipMemset(d_err, 0, 4));

  // 1. cutoffs, 2. packing
  PSPO_CALL(pspo_sample_cutoffs(d_xi, d_xi_off, d_lengths, P, K, seed, offset, d_cutoffs, d_err, stream));
  PSPO_CALL(pspo_pack_prefixes(d_cutoffs, d_lengths, d_xi, d_xi_off, P, K, total, d_target_full,
                               d_logp_old_full, d_hidden_full, d, d_cu, d_full_off, d_src, d_seq, d_weight,
                               d_tgt, d_lpo, d_hid, d_n, d_err, stream));
  int32_t N = 0;
  HIP_CALL(hipMemcpyAsync(&N, d_n, 4, hipMemcpyDeviceToHost, stream));
  HIP_CALL(hipStreamSynchronize(stream));

  // 3. loss and gradients over the N packed tokens
  const size_t ws_bytes = pspo_loss_workspace_bytes(N, d, V, 0);
  void* d_ws = nullptr;
  HIP_CALL(hipMalloc(&d_ws, ws_bytes > 0 ? ws_bytes : 256));
  HIP_CALL(hipMalloc(&d_loss, 8));
  HIP_CALL(hipMalloc(&d_stats, 5 * 8));
  HIP_CALL(hipMalloc(&d_logp, (N > 0 ? N : 1) * 4));
  HIP_CALL(hipMalloc(&d_dh, static_cast<size_t>(N > 0 ? N : 1) * d * 4));
  HIP_CALL(hipMalloc(&d_dw, static_cast<size_t>(V) * d * 4));
  PSPO_CALL(pspo_loss_fwd_bwd(d_hid, d_w, d_tgt, d_lpo, d_weight, d_seq, d_adv, N, d, V, R, eps_low, eps_high,
                              loss_scale, 0, d_loss, d_dh, d_dw, d_logp, d_stats, d_err, d_ws, ws_bytes, stream));
  HIP_CALL(hipStreamSynchronize(stream));

  std::vector<int32_t> cutoffs(R);
  std::vector<float> logp(N), dh(static_cast<size_t>(N) * d), dw(static_cast<size_t>(V) * d);
  double loss = 0, stats[5];
  int32_t flag = 0;
  HIP_CALL(hipMemcpy(cutoffs.data(), d_cutoffs, R * 4, hipMemcpyDeviceToHost));
  HIP_CALL(hipMemcpy(logp.data(), d_logp, N * 4, hipMemcpyDeviceToHost));
  HIP_CALL(hipMemcpy(dh.data(), d_dh, dh.size() * 4, hipMemcpyDeviceToHost));
  HIP_CALL(hipMemcpy(dw.data(), d_dw, dw.size() * 4, hipMemcpyDeviceToHost));
  HIP_CALL(hipMemcpy(&loss, d_loss, 8, hipMemcpyDeviceToHost));
  HIP_CALL(hipMemcpy(stats, d_stats, 5 * 8, hipMemcpyDeviceToHost));
  HIP_CALL(hipMemcpy(&flag, d_err, 4, hipMemcpyDeviceToHost));

  bool ok = save(dir, "lengths.i32", lengths.data(), R) && save(dir, "xi.f64", xi.data(), xi.size()) &&
            save(dir, "xi_off.i64", xi_off.data(), xi_off.size()) && save(dir, "adv.f32", adv.data(), R) &&
            save(dir, "hidden.bf16", hidden.data(), hidden.size()) && save(dir, "w.bf16", w.data(), w.size()) &&
            save(dir, "target.i32", target.data(), target.size()) &&
            save(dir, "logp_old.f32", logp_old.data(), logp_old.size()) &&
            save(dir, "cutoffs.i32", cutoffs.data(), R) && save(dir, "logp.f32", logp.data(), logp.size()) &&
            save(dir, "dh.f32", dh.data(), dh.size()) && save(dir, "dw.f32", dw.data(), dw.size()) &&
            save(dir, "loss.f64", &loss, 1) && save(dir, "stats.f64", stats, 5);
  FILE* meta = std::fopen((dir + "/meta.txt").c_str(), "w");
  ok = ok && meta != nullptr;
  if (meta) {
    std::fprintf(meta, "%d %d %d %d %llu %llu %.9g %.9g %.9g %d %d\n", P, K, d, V,
                 static_cast<unsigned long long>(seed), static_cast<unsigned long long>(offset),
                 eps_low, eps_high, loss_scale, N, flag);
    ok = std::fclose(meta) == 0 && ok;
  }
  if (!ok) {
    std::fprintf(stderr, "could not write the results into %s\n", dir.c_str());
    return 4;
  }
  std::printf("abi_example: N=%d of %d tokens, loss=%.9g, err_flag=%d\n", N, total, loss, flag);
  return 0;
}
