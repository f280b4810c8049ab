// A C/C++ client of the SAEF library that uses nothing but include/saef.h and
// the HIP runtime: it builds a two-tensor layout, runs three SAEF iterations
// (double-way, K = 2) and one Top-K iteration on device buffers it owns, and
// checks the status codes and two invariants that hold for any input:
//   - every scale is >= 0 and the sign words have no bits past a tensor's end;
//   - with Top-K, exactly keep[l] bits are set per tensor and worker.
// Prints "abi client ok" and returns 0 on success.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>

#include <vector>

#include "saef.h"

#define CHECK_HIP(x)                                                        \
  do {                                                                      \
    hipError_t e_ = (x);                                                    \
    if (e_ != hipSuccess) {                                                 \
      printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
      return 1;                                                             \
    }                                                                       \
  } while (0)
#define CHECK_SAEF(x)                                    \
  do {                                                   \
    int r_ = (x);                                        \
    if (r_ != SAEF_OK) {                                 \
      printf("SAEF error %d at line %d\n", r_, __LINE__); \
      return 1;                                          \
    }                                                    \
  } while (0)

int main() {
  const int32_t L = 2, K = 2;
  const int64_t off[2] = {0, 1024};
  const int64_t n[2] = {1000, 77};
  const int64_t d_pad = 1152, W = d_pad / 64;  // 1024 + 77 rounded up to 64
  saef_layout* lay = nullptr;
  CHECK_SAEF(saef_layout_create(off, n, L, d_pad, K, &lay));
  float *g, *e, *es, *x, *xh, *scales, *sscales;
  uint64_t *signs, *ss;
  CHECK_HIP(hipMalloc(&g, K * d_pad * 4));
  CHECK_HIP(hipMalloc(&e, K * d_pad * 4));
  CHECK_HIP(hipMalloc(&es, d_pad * 4));
  CHECK_HIP(hipMalloc(&x, d_pad * 4));
  CHECK_HIP(hipMalloc(&xh, K * d_pad * 4));
  CHECK_HIP(hipMalloc(&scales, K * L * 4));
  CHECK_HIP(hipMalloc(&sscales, L * 4));
  CHECK_HIP(hipMalloc(&signs, K * W * 8));
  CHECK_HIP(hipMalloc(&ss, W * 8));
  std::vector<float> hg(K * d_pad);
  uint32_t s = 12345u;
  for (auto& v : hg) {
    s = s * 1664525u + 1013904223u;
    v = ((int32_t)(s >> 8) - (1 << 23)) * (1.0f / (1 << 23));  // uniform in [-1, 1)
  }
  CHECK_HIP(hipMemcpy(g, hg.data(), hg.size() * 4, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemset(e, 0, K * d_pad * 4));
  CHECK_HIP(hipMemset(es, 0, d_pad * 4));
  CHECK_HIP(hipMemset(x, 0, d_pad * 4));
  for (int64_t t = 0; t < 3; ++t)
    CHECK_SAEF(saef_round(lay, t, 2, K, 0.1f, SAEF_MODE_DC, g, e, es, x, xh, signs, scales, ss,
                          sscales, nullptr));
  CHECK_SAEF(saef_status(lay, nullptr));
  std::vector<float> hs(K * L);
  std::vector<uint64_t> hw(K * W);
  CHECK_HIP(hipMemcpy(hs.data(), scales, hs.size() * 4, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(hw.data(), signs, hw.size() * 8, hipMemcpyDeviceToHost));
  for (float v : hs)
    if (!(v >= 0.0f)) {
      printf("negative scale %g\n", v);
      return 1;
    }
  for (int k = 0; k < K; ++k)
    for (int l = 0; l < L; ++l) {
      const int64_t last = off[l] / 64 + (n[l] - 1) / 64;
      const int used = (int)(n[l] % 64);
      if (used != 0 && (hw[k * W + last] >> used) != 0) {
        printf("bits past the end of tensor %d\n", l);
        return 1;
      }
    }
  // one Top-K iteration on the same layout
  const int64_t keep[2] = {10, 1};
  saef_topk* tk = nullptr;
  CHECK_SAEF(saef_topk_create(lay, keep, &tk));
  int64_t total = 0;
  CHECK_SAEF(saef_topk_info(tk, &total));
  if (total != 11) {
    printf("total keep %lld\n", (long long)total);
    return 1;
  }
  uint32_t *rank, *srank;
  float *vals, *svals;
  CHECK_HIP(hipMalloc(&rank, K * W * 4));
  CHECK_HIP(hipMalloc(&srank, W * 4));
  CHECK_HIP(hipMalloc(&vals, K * total * 4));
  CHECK_HIP(hipMalloc(&svals, total * 4));
  CHECK_HIP(hipMemset(e, 0, K * d_pad * 4));
  CHECK_HIP(hipMemset(es, 0, d_pad * 4));
  CHECK_SAEF(saef_topk_round(tk, 0, 0, K, 0.1f, 0.0f, SAEF_MODE_DC, g, nullptr, e, es, x, xh,
                             signs, rank, vals, ss, srank, svals, nullptr));
  CHECK_SAEF(saef_status(lay, nullptr));
  CHECK_HIP(hipMemcpy(hw.data(), signs, hw.size() * 8, hipMemcpyDeviceToHost));
  for (int k = 0; k < K; ++k)
    for (int l = 0; l < L; ++l) {
      int64_t bits = 0;
      for (int64_t w = off[l] / 64; w <= off[l] / 64 + (n[l] - 1) / 64; ++w)
        bits += __builtin_popcountll(hw[k * W + w]);
      if (bits != keep[l]) {
        printf("worker %d tensor %d keeps %lld, not %lld\n", k, l, (long long)bits,
               (long long)keep[l]);
        return 1;
      }
    }
  // invalid arguments are rejected before anything is enqueued
  if (saef_round(lay, -1, 0, K, 0.1f, SAEF_MODE_DC, g, e, es, x, xh, signs, scales, ss, sscales,
                 nullptr) != SAEF_EINVAL) {
    printf("negative t accepted\n");
    return 1;
  }
  CHECK_SAEF(saef_topk_destroy(tk));
  CHECK_SAEF(saef_layout_destroy(lay));
  for (void* p : {(void*)g, (void*)e, (void*)es, (void*)x, (void*)xh, (void*)scales,
                  (void*)sscales, (void*)signs, (void*)ss, (void*)rank, (void*)srank, (void*)vals,
                  (void*)svals})
    CHECK_HIP(hipFree(p));
  printf("abi client ok\n");
  return 0;
}
