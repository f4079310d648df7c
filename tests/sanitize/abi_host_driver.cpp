// Host-side driver of the libmxq C ABI for the sanitizer build (test
// infrastructure).  Built host-only with AddressSanitizer and
// UndefinedBehaviorSanitizer and run on a machine without a GPU: every size
// query and every argument check runs for real; calls that pass validation
// reach a kernel launch, which the HIP runtime refuses without a device, so
// they must return MXQ_ERR_DEVICE.  Any out-of-bounds access, overflow or
// other undefined behaviour on these host paths aborts the run.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <vector>

#include "../../include/mxq.h"

static int failures = 0;
#define EXPECT(cond)                                                       \
  do {                                                                     \
    if (!(cond)) {                                                         \
      fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                          \
    }                                                                      \
  } while (0)

static mxq_fmt make_fmt(int64_t K, const std::vector<uint8_t> &w, int round = 0, int clamp = 0) {
  mxq_fmt f;
  f.K = K;
  f.block = 32;
  f.round = round;
  f.clamp = clamp;
  f.reserved = 0;
  f.widths = w.data();
  f.perm = nullptr;
  return f;
}

int main() {
  // width maps of every segment mix, including empty segments and 3-bit blocks
  const std::vector<std::vector<uint8_t>> maps = {
      {4}, {3}, {6}, {8}, {3, 4, 6, 8}, {4, 4, 4, 4, 4, 6, 8},
      {3, 3, 3, 3, 3, 6, 6, 8}, {8, 8, 8}, {6, 6, 6, 6, 6}, {4, 4, 4, 4, 4, 4, 4, 4, 4}};
  // a large, aligned, never dereferenced address stands in for device memory
  void *fake = (void *)(uintptr_t)(1u << 20);
  for (const auto &w : maps) {
    for (int clamp = 0; clamp < 2; ++clamp) {
      const mxq_fmt f = make_fmt(32 * (int64_t)w.size(), w, 0, clamp);
      const int64_t rb = mxq_act_packed_bytes(&f), erb = mxq_exp_row_bytes(&f);
      EXPECT(rb > 0 && rb % 16 == 0 && erb > 0 && erb % 16 == 0);
      for (int64_t M : {0, 1, 15, 16, 17, 255, 256, 257, 4096}) {
        EXPECT(mxq_act_bytes(&f, M) >= 0);
        EXPECT(mxq_act_exp_bytes(&f, M) >= 0);
        EXPECT(mxq_weight_bytes(&f, M) >= 0);
        EXPECT(mxq_weight_exp_bytes(&f, M) >= 0);
      }
      EXPECT(mxq_act_bytes(&f, -1) < 0);
      // validation failures: nothing is launched
      EXPECT(mxq_quantize_act(&f, (const uint16_t *)fake, 4, f.K - 1, (uint8_t *)fake,
                              (uint8_t *)fake, nullptr) == MXQ_ERR_SHAPE);
      EXPECT(mxq_gemm(&f, 4, 4, nullptr, (const uint8_t *)fake, (const uint8_t *)fake,
                      (const uint8_t *)fake, (float *)fake, 4, nullptr) == MXQ_ERR_NULL);
      EXPECT(mxq_gemm(&f, 4, 4, (const uint8_t *)fake, (const uint8_t *)fake,
                      (const uint8_t *)fake, (const uint8_t *)fake, (float *)fake, 3,
                      nullptr) == MXQ_ERR_SHAPE);
      // empty problems succeed without a launch
      EXPECT(mxq_gemm(&f, 0, 4, nullptr, nullptr, nullptr, nullptr, nullptr, 4, nullptr) ==
             MXQ_OK);
      EXPECT(mxq_quantize_act(&f, nullptr, 0, f.K, nullptr, nullptr, nullptr) == MXQ_OK);
      // valid calls reach a launch, which fails without a GPU
      for (int64_t M : {1, 16, 17, 300}) {
        EXPECT(mxq_quantize_act(&f, (const uint16_t *)fake, M, f.K, (uint8_t *)fake,
                                (uint8_t *)fake, nullptr) == MXQ_ERR_DEVICE);
        EXPECT(mxq_quantize_rows(&f, (const uint16_t *)fake, M, f.K, (uint8_t *)fake,
                                 (uint8_t *)fake, nullptr) == MXQ_ERR_DEVICE);
        EXPECT(mxq_gemm(&f, M, 40, (const uint8_t *)fake, (const uint8_t *)fake,
                        (const uint8_t *)fake, (const uint8_t *)fake, (float *)fake, 40,
                        nullptr) == MXQ_ERR_DEVICE);
      }
      EXPECT(mxq_pack_weights(&f, (const uint16_t *)fake, 300, f.K, (uint8_t *)fake,
                              (uint8_t *)fake, nullptr) == MXQ_ERR_DEVICE);
    }
  }
  // bad formats
  {
    const std::vector<uint8_t> bad = {4, 5};
    const mxq_fmt f = make_fmt(64, bad);
    EXPECT(mxq_act_packed_bytes(&f) == -MXQ_ERR_WIDTHS);
    const std::vector<uint8_t> unsorted = {8, 4};
    const mxq_fmt g = make_fmt(64, unsorted);
    EXPECT(mxq_weight_bytes(&g, 16) == -MXQ_ERR_WIDTHS);
    const mxq_fmt h = make_fmt(63, bad);
    EXPECT(mxq_act_bytes(&h, 4) == -MXQ_ERR_SHAPE);
    EXPECT(mxq_act_bytes(nullptr, 4) == -MXQ_ERR_NULL);
  }
  // a K so long that 32-bit kernel offsets would overflow is refused
  {
    const std::vector<uint8_t> w(131072, 8);
    const mxq_fmt f = make_fmt(32 * (int64_t)w.size(), w);
    EXPECT(mxq_gemm(&f, 64, 128, (const uint8_t *)fake, (const uint8_t *)fake,
                    (const uint8_t *)fake, (const uint8_t *)fake, (float *)fake, 128,
                    nullptr) == MXQ_ERR_SHAPE);
  }
  // calibration host functions
  {
    const int64_t d[3] = {4096, 4096, 14336};
    const double s[3] = {1.0, 2.0, 0.5};
    double R = 0.0;
    EXPECT(mxq_calib_ratio(3, d, s, 4.25, &R) == MXQ_OK);
    int32_t n4 = 0, n6 = 0, n8 = 0;
    EXPECT(mxq_calib_counts(4096, R, 1.0, 1, &n4, &n6, &n8) == MXQ_OK);
    EXPECT(n4 + n6 + n8 == 128);
    EXPECT(mxq_calib_counts(4096, 1e30, 1.0, 1, &n4, &n6, &n8) == MXQ_OK);
    EXPECT(n8 == 1 && n6 == 127 && n4 == 0);
    EXPECT(mxq_calib_counts(4096, -1e30, 1.0, 200, &n4, &n6, &n8) == MXQ_OK);
    EXPECT(n8 == 128 && n6 == 0 && n4 == 0);
    EXPECT(mxq_calib_ratio(0, d, s, 4.25, &R) == MXQ_ERR_SHAPE);
  }
  // attention: sizes, argument checks, and the static scratch limit
  {
    const std::vector<uint8_t> w = {4, 4, 6, 8};
    const mxq_fmt f = make_fmt(128, w);
    EXPECT(mxq_attn_work_bytes(&f, 2, 64, 8, 4096) > 0);
    EXPECT(mxq_attn_work_bytes(&f, 2, 64, 7, 4096) < 0);
    EXPECT(mxq_attn_decode_static(&f, (const uint16_t *)fake, 300, 64, 8, 64, 0.1f,
                                  (const uint8_t *)fake, (const uint8_t *)fake,
                                  (const uint8_t *)fake, (const uint8_t *)fake, (float *)fake,
                                  nullptr) == MXQ_ERR_SCRATCH);
    EXPECT(mxq_attn_decode(&f, (const uint16_t *)fake, 2, 64, 8, 100, 0.1f,
                           (const uint8_t *)fake, (const uint8_t *)fake, (const uint8_t *)fake,
                           (const uint8_t *)fake, (float *)fake, (float *)fake, 16,
                           nullptr) == MXQ_ERR_SHAPE);
  }
  for (int s = 0; s <= 9; ++s) EXPECT(mxq_status_str(s) != nullptr);
  if (failures) {
    fprintf(stderr, "%d expectation(s) failed\n", failures);
    return 1;
  }
  printf("abi host driver: ok\n");
  return 0;
}
