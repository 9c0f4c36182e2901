// Drives every entry point of include/cci.h through its validation and
// dispatch paths (valid calls reach the stub launchers, invalid ones must
// fail before them) in a build with AddressSanitizer and
// UndefinedBehaviorSanitizer.  Exit status 0 and "abi driver ok" on success.
#include <cmath>
#include <cstdio>
#include <cstring>

#include "../../include/cci.h"

extern int g_launches;

static int failures = 0;
#define EXPECT(cond)                                                   \
  do {                                                                 \
    if (!(cond)) {                                                     \
      std::fprintf(stderr, "FAILED line %d: %s\n", __LINE__, #cond);  \
      ++failures;                                                      \
    }                                                                  \
  } while (0)

alignas(16) static unsigned char buf[4][1 << 12];

int main() {
  void* A = buf[0];
  void* B = buf[1];
  void* C = buf[2];
  void* D = buf[3];
  void* mis = buf[0] + 8;
  size_t vb = 0, ib = 0;
  // sizes and host-only helpers
  EXPECT(cci_packed_sizes(256, 256, 8, 4, CCI_BF16, &vb, &ib) == CCI_OK && ib == 256 / 8 * 4 * 256 && vb == 2 * ib);
  EXPECT(cci_packed_sizes(12, 5, 8, 2, CCI_BF16, &vb, &ib) == CCI_EINVAL);
  EXPECT(cci_bbs_packed_sizes(8, 64, 4, 2, CCI_F32, &vb, &ib) == CCI_OK && vb == 4 * ib);
  EXPECT(cci_2of4_sizes(32, 128, &vb, &ib) == CCI_OK && vb == 32 * 128 && ib == 32 * 128 / 8);
  EXPECT(cci_index_stream_bytes(33, 3, &vb) == CCI_OK && vb == 16);
  for (int G = 1; G <= 256; ++G) {
    const int b = cci_index_width(G);
    EXPECT(b >= 1 && (1 << b) >= G && (b == 1 || (1 << (b - 1)) < G));
  }
  int32_t nt = 0;
  double p = 0.0;
  EXPECT(cci_td_schedule(50, 100, 8, 2, &nt, &p) == CCI_OK && nt == 6 && p == 0.5);
  EXPECT(cci_td_schedule(101, 100, 8, 2, &nt, &p) == CCI_EINVAL);
  EXPECT(cci_auto_algo(CCI_BF16, CCI_BF16, 4096, 4096, 4096, 4096, 16, 1) == CCI_ALGO_WIDE_TILE_MFMA);
  EXPECT(std::strlen(cci_status_str(CCI_EHIP)) > 0 && cci_version() >= 100);

  const int before = g_launches;
  // valid calls reach exactly one launcher each
  EXPECT(cci_pack((const float*)A, 64, 32, 8, 2, B, CCI_BF16, (uint8_t*)C, nullptr) == CCI_OK);
  EXPECT(cci_spmm(A, CCI_BF16, 16, 64, B, CCI_BF16, (const uint8_t*)C, 64, 8, 2, nullptr, D, CCI_BF16, nullptr) == CCI_OK);
  EXPECT(cci_spmm_algo(A, CCI_F32, 16, 64, B, CCI_F32, (const uint8_t*)C, 64, 8, 2, nullptr, D, CCI_F32,
                       CCI_ALGO_SPARSE_MAC, nullptr) == CCI_OK);
  EXPECT(cci_conv_im2col(A, CCI_BF16, 1, 8, 8, 32, 3, 3, 1, 1, 1, 1, B, CCI_BF16, (const uint8_t*)C, 64, 8, 2,
                         nullptr, D, CCI_BF16, nullptr) == CCI_OK);
  EXPECT(cci_bbs_pack((const float*)A, 8, 64, 4, 2, B, CCI_BF16, (uint8_t*)C, nullptr) == CCI_OK);
  EXPECT(cci_bbs_to_2of4(A, CCI_BF16, (const uint8_t*)B, 32, 128, 4, 2, C, (uint16_t*)D, nullptr) == CCI_OK);
  EXPECT(cci_to_2of4_transposed(A, CCI_BF16, (const uint8_t*)B, 128, 32, 16, 2, C, (uint16_t*)D, nullptr) == CCI_OK);
  cci_epilogue ep{(const float*)A, (const float*)B, nullptr, 1};
  EXPECT(cci_spmm_2of4(A, CCI_BF16, 5, 128, B, (const uint16_t*)C, 32, &ep, D, CCI_F32, nullptr) == CCI_OK);
  EXPECT(cci_td_mask((const float*)A, 16, 8, 8, 3, (const uint32_t*)B, 0.5, C, CCI_BF16, (uint8_t*)D, nullptr) == CCI_OK);
  EXPECT(cci_grad_packed(A, B, CCI_BF16, 4, 8, (const uint8_t*)C, 16, 8, 2, (float*)D, nullptr) == CCI_OK);
  EXPECT(cci_index_bits((const uint8_t*)A, 100, 3, (uint32_t*)B, nullptr) == CCI_OK);
  EXPECT(cci_spmm_bits(A, CCI_BF16, 4, 64, B, CCI_BF16, C, 4, 64, 16, 2, nullptr, D, CCI_BF16, nullptr) == CCI_OK);
  EXPECT(cci_maxpool2d_nhwc(A, CCI_BF16, 1, 8, 8, 16, 3, 2, 1, B, nullptr) == CCI_OK);
  EXPECT(cci_global_avgpool_nhwc(A, CCI_BF16, 1, 8, 8, 16, B, CCI_F32, nullptr) == CCI_OK);
  EXPECT(g_launches - before == 14);

  // invalid calls fail before any launch, with a message
  const int mid = g_launches;
  EXPECT(cci_pack((const float*)mis, 64, 32, 8, 2, B, CCI_BF16, (uint8_t*)C, nullptr) == CCI_EALIGN);
  EXPECT(cci_spmm(A, CCI_F32, 16, 64, B, CCI_BF16, (const uint8_t*)C, 64, 8, 2, nullptr, D, CCI_F32, nullptr) == CCI_EUNSUPPORTED);
  EXPECT(std::strlen(cci_last_error()) > 0);
  EXPECT(cci_spmm(A, CCI_BF16, -1, 64, B, CCI_BF16, (const uint8_t*)C, 64, 8, 2, nullptr, D, CCI_BF16, nullptr) == CCI_EINVAL);
  EXPECT(cci_spmm_algo(A, CCI_BF16, 16, 64, B, CCI_BF16, (const uint8_t*)C, 64, 8, 2, nullptr, D, CCI_BF16,
                       (cci_algo)10, nullptr) == CCI_EINVAL);
  EXPECT(cci_conv_im2col(A, CCI_BF16, 1, 2, 2, 32, 3, 3, 1, 1, 0, 0, B, CCI_BF16, (const uint8_t*)C, 64, 8, 2, nullptr,
                         D, CCI_BF16, nullptr) == CCI_EINVAL);
  EXPECT(cci_bbs_pack((const float*)A, 8, 62, 4, 2, B, CCI_BF16, (uint8_t*)C, nullptr) == CCI_EINVAL);
  EXPECT(cci_bbs_to_2of4(A, CCI_BF16, (const uint8_t*)B, 32, 128, 8, 3, C, (uint16_t*)D, nullptr) == CCI_EUNSUPPORTED);
  EXPECT(cci_spmm_2of4(A, CCI_BF16, 5, 96, B, (const uint16_t*)C, 32, nullptr, D, CCI_BF16, nullptr) == CCI_EUNSUPPORTED);
  EXPECT(cci_td_mask((const float*)A, 16, 8, 8, 9, (const uint32_t*)B, 0.5, C, CCI_BF16, (uint8_t*)D, nullptr) == CCI_EINVAL);
  EXPECT(cci_td_mask((const float*)A, 16, 8, 8, 3, (const uint32_t*)B, NAN, C, CCI_BF16, (uint8_t*)D, nullptr) == CCI_EINVAL);
  EXPECT(cci_grad_packed(A, B, CCI_BF16, 4, 8, (const uint8_t*)C, 16, 8, 9, (float*)D, nullptr) == CCI_EINVAL);
  EXPECT(cci_index_bits((const uint8_t*)A, 100, 9, (uint32_t*)B, nullptr) == CCI_EINVAL);
  EXPECT(cci_spmm_bits(A, CCI_BF16, 65, 64, B, CCI_BF16, C, 4, 64, 16, 2, nullptr, D, CCI_BF16, nullptr) == CCI_EUNSUPPORTED);
  EXPECT(cci_maxpool2d_nhwc(A, CCI_BF16, 1, 8, 8, 16, 3, 2, 2, B, nullptr) == CCI_EINVAL);
  // extreme sizes: rejected without overflow
  EXPECT(cci_spmm(A, CCI_BF16, INT64_MAX / 2, 64, B, CCI_BF16, (const uint8_t*)C, 64, 8, 2, nullptr, D, CCI_BF16, nullptr) == CCI_EINVAL);
  EXPECT(cci_packed_sizes(INT64_MAX / 4, INT64_MAX / 4, 8, 2, CCI_BF16, &vb, &ib) == CCI_EINVAL);
  EXPECT(cci_conv_im2col(A, CCI_BF16, INT64_MAX / 8, 1 << 20, 1 << 20, 1 << 24, 3, 3, 1, 1, 1, 1, B, CCI_BF16,
                         (const uint8_t*)C, 64, 8, 2, nullptr, D, CCI_BF16, nullptr) == CCI_EINVAL);
  EXPECT(cci_maxpool2d_nhwc(A, CCI_BF16, INT64_MAX / 4, INT64_MAX / 8, INT64_MAX / 8, 16, 3, 2, 1, B, nullptr) == CCI_EINVAL);
  EXPECT(cci_global_avgpool_nhwc(A, CCI_BF16, 3, int64_t(1) << 40, int64_t(1) << 40, 16, B, CCI_F32, nullptr) == CCI_EINVAL);
  EXPECT(cci_spmm_2of4(A, CCI_BF16, INT64_MAX / 2, 128, B, (const uint16_t*)C, 32, nullptr, D, CCI_BF16, nullptr) == CCI_EINVAL);
  EXPECT(g_launches == mid);
  // N = 0 is a no-op without pointers
  EXPECT(cci_spmm(nullptr, CCI_BF16, 0, 64, nullptr, CCI_BF16, nullptr, 64, 8, 2, nullptr, nullptr, CCI_BF16, nullptr) == CCI_OK);
  EXPECT(g_launches == mid);
  if (failures) return 1;
  std::printf("abi driver ok\n");
  return 0;
}
