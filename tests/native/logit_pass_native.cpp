// A native consumer of libcmsd: plain C++ on the HIP runtime and include/cmsd.h,
// no Python.  It generates a small seeded fp32 workload on the host (B = 6
// sequences, k_max = 5 drafts, V = 3001, rows of three spreads), uploads it, runs
// one decoding iteration three times on its own stream -- cmsd_confidence +
// cmsd_draft_len + cmsd_verify (dense layout), cmsd_logit_pass, and
// cmsd_logit_pass_fused on a zero-filled workspace -- checks that all three agree bit
// for bit (and that the fused call leaves its counters at zero), and writes inputs and
// outputs to the file named by argv[1] so the test suite can check them against the
// oracle.  Exit status 0 on success.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "cmsd.h"

namespace {

uint64_t g_state = 0x2545F4914F6CDD1Dull;  // xorshift64* (Vigna), fixed seed

uint64_t next_u64() {
  g_state ^= g_state >> 12;
  g_state ^= g_state << 25;
  g_state ^= g_state >> 27;
  return g_state * 0x2545F4914F6CDD1Dull;
}
double unit() { return (double)(next_u64() >> 11) * (1.0 / 9007199254740992.0); }  // [0, 1)
double normal() {                                                                   // Box-Muller
  const double u1 = 1.0 - unit(), u2 = unit();
  return std::sqrt(-2.0 * std::log(u1)) * std::cos(6.283185307179586 * u2);
}

#define HIP_OK(x)                                                            \
  do {                                                                       \
    if ((x) != hipSuccess) {                                                 \
      std::fprintf(stderr, "HIP error %s at line %d\n", #x, __LINE__);       \
      return 2;                                                              \
    }                                                                        \
  } while (0)
#define CMSD_OK_OR(x)                                                                          \
  do {                                                                                         \
    const cmsd_status s_ = (x);                                                                \
    if (s_ != CMSD_OK) {                                                                       \
      std::fprintf(stderr, "%s: %s\n", #x, cmsd_status_string(s_));                            \
      return 3;                                                                                \
    }                                                                                          \
  } while (0)

template <typename T>
T* dev_copy(const std::vector<T>& h) {
  T* d = nullptr;
  if (hipMalloc(&d, h.size() * sizeof(T)) != hipSuccess) return nullptr;
  if (hipMemcpy(d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice) != hipSuccess) return nullptr;
  return d;
}

template <typename T>
bool host_copy(std::vector<T>& h, const T* d) {
  return hipMemcpy(h.data(), d, h.size() * sizeof(T), hipMemcpyDeviceToHost) == hipSuccess;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 2) {
    std::fprintf(stderr, "usage: %s OUTPUT_FILE\n", argv[0]);
    return 2;
  }
  const int B = 6, K = 5, V = 3001;
  const int RD = B * K, RT = B * (K + 1);
  const double spread[3] = {0.5, 2.0, 8.0};
  std::vector<float> zd((size_t)RD * V), zt((size_t)RT * V), unif(RT);
  std::vector<int32_t> drafted(RD);
  for (int r = 0; r < RD; ++r) {
    const double s = spread[r % 3];
    for (int v = 0; v < V; ++v) zd[(size_t)r * V + v] = (float)(s * normal());
    // the drafted token: a Gumbel-max (exact softmax) sample of the drafter row
    double best = -INFINITY;
    for (int v = 0; v < V; ++v) {
      const double g = zd[(size_t)r * V + v] - std::log(-std::log(1.0 - unit()));
      if (g > best) {
        best = g;
        drafted[r] = v;
      }
    }
  }
  for (int b = 0; b < B; ++b)
    for (int i = 0; i <= K; ++i)
      for (int v = 0; v < V; ++v) {
        const size_t t = ((size_t)b * (K + 1) + i) * V + v;
        zt[t] = i < K ? (float)(zd[((size_t)b * K + i) * V + v] + 0.5 * normal()) : (float)(2.0 * normal());
      }
  for (int j = 0; j < RT; ++j) unif[j] = (float)(next_u64() >> 40) * (1.0f / 16777216.0f);  // k * 2^-24

  std::vector<int32_t> off_dense(B + 1), k_dense(B, K);
  for (int b = 0; b <= B; ++b) off_dense[b] = b * (K + 1);

  float* d_zd = dev_copy(zd);
  float* d_zt = dev_copy(zt);
  int32_t* d_drafted = dev_copy(drafted);
  float* d_unif = dev_copy(unif);
  int32_t* d_off_dense = dev_copy(off_dense);
  int32_t* d_k_dense = dev_copy(k_dense);
  if (!d_zd || !d_zt || !d_drafted || !d_unif || !d_off_dense || !d_k_dense) return 2;
  cmsd_row_stats *d_st1, *d_st2, *d_st3;
  cmsd_target_stats *d_ts1, *d_ts2, *d_ts3;
  int32_t *d_k1, *d_off1, *d_k2, *d_k3, *d_na1, *d_na2, *d_na3, *d_nx1, *d_nx2, *d_nx3;
  const size_t wsb = cmsd_verify_workspace_bytes(B, K, V);
  const size_t wsf = cmsd_logit_pass_fused_workspace_bytes(B, K, V);
  void *d_ws1, *d_ws2, *d_ws3;
  HIP_OK(hipMalloc(&d_st1, RD * sizeof(cmsd_row_stats)));
  HIP_OK(hipMalloc(&d_st2, RD * sizeof(cmsd_row_stats)));
  HIP_OK(hipMalloc(&d_ts1, RT * sizeof(cmsd_target_stats)));
  HIP_OK(hipMalloc(&d_ts2, RT * sizeof(cmsd_target_stats)));
  HIP_OK(hipMalloc(&d_k1, B * sizeof(int32_t)));
  HIP_OK(hipMalloc(&d_off1, (B + 1) * sizeof(int32_t)));
  HIP_OK(hipMalloc(&d_k2, B * sizeof(int32_t)));
  HIP_OK(hipMalloc(&d_na1, B * sizeof(int32_t)));
  HIP_OK(hipMalloc(&d_na2, B * sizeof(int32_t)));
  HIP_OK(hipMalloc(&d_nx1, B * sizeof(int32_t)));
  HIP_OK(hipMalloc(&d_nx2, B * sizeof(int32_t)));
  HIP_OK(hipMalloc(&d_ws1, wsb));
  HIP_OK(hipMalloc(&d_ws2, wsb));
  HIP_OK(hipMalloc(&d_st3, RD * sizeof(cmsd_row_stats)));
  HIP_OK(hipMalloc(&d_ts3, RT * sizeof(cmsd_target_stats)));
  HIP_OK(hipMalloc(&d_k3, B * sizeof(int32_t)));
  HIP_OK(hipMalloc(&d_na3, B * sizeof(int32_t)));
  HIP_OK(hipMalloc(&d_nx3, B * sizeof(int32_t)));
  HIP_OK(hipMalloc(&d_ws3, wsf));
  HIP_OK(hipMemset(d_ws3, 0, wsf));  // the fused call's counters start at zero
  hipStream_t st;
  HIP_OK(hipStreamCreate(&st));

  const cmsd_conf_params cp = {1.0f / 3, 1.0f / 3, 1.0f / 3, 1.0f};
  const cmsd_draft_params dp = {1, K, 1.0f};
  const cmsd_verify_params vp = {CMSD_MODE_CM, 3, 0.1f, 1.0f};
  // the three calls, dense layout (all K drafts verified)
  CMSD_OK_OR(cmsd_confidence(d_zd, CMSD_F32, RD, V, V, &cp, d_st1, st));
  CMSD_OK_OR(cmsd_draft_len(d_st1, B, &dp, d_k1, d_off1, st));
  CMSD_OK_OR(cmsd_verify(d_zd, V, d_st1, d_zt, V, RT, d_off_dense, d_k_dense, d_drafted, d_unif, CMSD_F32, B, K, V,
                         &vp, d_ts1, d_na1, d_nx1, d_ws1, wsb, st));
  // the same iteration in one call
  CMSD_OK_OR(cmsd_logit_pass(d_zd, V, d_zt, V, d_drafted, d_unif, CMSD_F32, B, K, V, &cp, &dp, &vp, 0, d_st2, d_k2,
                             d_ts2, d_na2, d_nx2, d_ws2, wsb, st));
  // and in one launch
  CMSD_OK_OR(cmsd_logit_pass_fused(d_zd, V, d_zt, V, d_drafted, d_unif, CMSD_F32, B, K, V, &cp, &dp, &vp, 0, d_st3,
                                   d_k3, d_ts3, d_na3, d_nx3, d_ws3, wsf, st));
  HIP_OK(hipStreamSynchronize(st));

  std::vector<cmsd_row_stats> st1(RD), st2(RD), st3(RD);
  std::vector<cmsd_target_stats> ts1(RT), ts2(RT), ts3(RT);
  std::vector<int32_t> k1(B), k2(B), k3(B), na1(B), na2(B), na3(B), nx1(B), nx2(B), nx3(B);
  std::vector<uint8_t> ws3(wsf);
  if (!host_copy(st1, d_st1) || !host_copy(st2, d_st2) || !host_copy(ts1, d_ts1) || !host_copy(ts2, d_ts2) ||
      !host_copy(k1, d_k1) || !host_copy(k2, d_k2) || !host_copy(na1, d_na1) || !host_copy(na2, d_na2) ||
      !host_copy(nx1, d_nx1) || !host_copy(nx2, d_nx2) || !host_copy(st3, d_st3) || !host_copy(ts3, d_ts3) ||
      !host_copy(k3, d_k3) || !host_copy(na3, d_na3) || !host_copy(nx3, d_nx3) ||
      !host_copy(ws3, static_cast<const uint8_t*>(d_ws3)))
    return 2;
  const bool same = std::memcmp(st1.data(), st2.data(), RD * sizeof(cmsd_row_stats)) == 0 &&
                    std::memcmp(ts1.data(), ts2.data(), RT * sizeof(cmsd_target_stats)) == 0 && k1 == k2 &&
                    na1 == na2 && nx1 == nx2;
  // the counters end the fused workspace and are zero again after the call
  bool counters_zero = true;
  for (size_t i = (wsf & ~(size_t)3) - 4 * (size_t)B; i < (wsf & ~(size_t)3); ++i) counters_zero &= ws3[i] == 0;
  const bool same_fused = std::memcmp(st2.data(), st3.data(), RD * sizeof(cmsd_row_stats)) == 0 &&
                          std::memcmp(ts2.data(), ts3.data(), RT * sizeof(cmsd_target_stats)) == 0 && k2 == k3 &&
                          na2 == na3 && nx2 == nx3 && counters_zero;

  // inputs and outputs for the oracle check: int32 B, K, V, then the arrays in order
  FILE* f = std::fopen(argv[1], "wb");
  if (!f) return 2;
  const int32_t hdr[3] = {B, K, V};
  std::fwrite(hdr, sizeof(hdr), 1, f);
  std::fwrite(zd.data(), sizeof(float), zd.size(), f);
  std::fwrite(zt.data(), sizeof(float), zt.size(), f);
  std::fwrite(drafted.data(), sizeof(int32_t), drafted.size(), f);
  std::fwrite(unif.data(), sizeof(float), unif.size(), f);
  std::fwrite(st1.data(), sizeof(cmsd_row_stats), st1.size(), f);
  std::fwrite(ts1.data(), sizeof(cmsd_target_stats), ts1.size(), f);
  std::fwrite(k1.data(), sizeof(int32_t), B, f);
  std::fwrite(na1.data(), sizeof(int32_t), B, f);
  std::fwrite(nx1.data(), sizeof(int32_t), B, f);
  std::fclose(f);

  for (void* p : {(void*)d_zd, (void*)d_zt, (void*)d_drafted, (void*)d_unif, (void*)d_off_dense, (void*)d_k_dense,
                  (void*)d_st1, (void*)d_st2, (void*)d_ts1, (void*)d_ts2, (void*)d_k1, (void*)d_off1, (void*)d_k2,
                  (void*)d_na1, (void*)d_na2, (void*)d_nx1, (void*)d_nx2, d_ws1, d_ws2, (void*)d_st3, (void*)d_ts3,
                  (void*)d_k3, (void*)d_na3, (void*)d_nx3, d_ws3})
    HIP_OK(hipFree(p));
  HIP_OK(hipStreamDestroy(st));
  std::printf("native logit pass: B=%d K=%d V=%d, one call %s the three calls, one launch %s the one call, "
              "n_accepted", B, K, V, same ? "bit-equal to" : "DIFFERS from", same_fused ? "bit-equal to" : "DIFFERS from");
  for (int b = 0; b < B; ++b) std::printf(" %d", na1[b]);
  std::printf("\n");
  return same && same_fused ? 0 : 1;
}
