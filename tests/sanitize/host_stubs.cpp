// Launcher stand-ins for a host-only build of the C-ABI layer (cci_api.cpp)
// under AddressSanitizer / UndefinedBehaviorSanitizer: every launcher
// records that it was reached and launches nothing, so the validation,
// dispatch and error paths run on the CPU.
#include <hip/hip_runtime.h>

#include "../../paper_1910_11971_amd/csrc/cci_launch.hpp"

int g_launches = 0;

namespace cci {

hipError_t launch_pack(const float*, int64_t, int64_t, int32_t, int32_t, void*, DType, uint8_t*, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}
bool sparse_mac_supports(const ProductArgs& a) { return a.G == 2 || a.G == 4 || a.G == 8 || a.G == 16 || a.G == 32; }
hipError_t launch_sparse_mac(const ProductArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
bool dense_tile_supports(const ProductArgs& a) { return a.x_t == DType::BF16 && 64 % a.G == 0; }
hipError_t launch_dense_tile(const ProductArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
bool wide_tile_supports(const ProductArgs& a) { return a.x_t == DType::BF16 && a.O % 256 == 0 && a.C % 64 == 0; }
hipError_t launch_wide_tile(const ProductArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
bool narrow_supports(const ProductArgs& a) { return a.x_t == DType::BF16 && a.C <= 256 && a.C % 8 == 0; }
hipError_t launch_narrow(const ProductArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
bool resident_supports(const ProductArgs& a) {
  return a.conv && a.x_t == DType::BF16 && a.geom.KH == 3 && a.geom.KW == 3 && a.geom.sh == 1 && a.geom.sw == 1 &&
         (a.geom.Cin == 32 || a.geom.Cin == 64) && (a.O == 32 || a.O == 64);
}
hipError_t launch_resident(const ProductArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
bool tap_tile_supports(const ProductArgs& a) {
  const int64_t cin = a.conv ? a.geom.Cin : a.C;
  return a.x_t == DType::BF16 && cin % 64 == 0 && 32 % a.G == 0 && (2 * a.K <= a.G || a.K == a.G) &&
         (a.O % 128 == 0 || (a.O % 64 == 0 && a.G <= 16));
}
hipError_t launch_tap_tile(const ProductArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
bool stream_tile_supports(const ProductArgs& a) {
  return a.x_t == DType::BF16 && a.C % 64 == 0 && a.C <= 256 && a.O % 64 == 0 && 32 % a.G == 0 &&
         (!a.conv || (a.geom.KH == 1 && a.geom.KW == 1 && a.geom.sh == 1 && a.geom.sw == 1 && a.geom.ph == 0 &&
                      a.geom.pw == 0));
}
hipError_t launch_stream_tile(const ProductArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
bool split_k_supports(const ProductArgs& a) {
  return a.x_t == DType::BF16 && a.val_t == DType::BF16 && a.C % 32 == 0 && a.O % 16 == 0 && a.K <= 4 &&
         (!a.conv || (a.geom.KH == 1 && a.geom.KW == 1 && a.geom.sh == 1 && a.geom.sw == 1 && a.geom.ph == 0 &&
                      a.geom.pw == 0));
}
hipError_t launch_split_k(const ProductArgs&, hipStream_t) { ++g_launches; return hipSuccess; }
hipError_t launch_bbs_pack(const float*, int64_t, int64_t, int32_t, int32_t, void*, DType, uint8_t*, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_to_2of4(bool, const void*, const uint8_t*, int64_t, int64_t, int32_t, int32_t, void*, uint16_t*,
                          hipStream_t) {
  ++g_launches;
  return hipSuccess;
}
bool spmm_2of4_fits(int64_t N, int64_t C, int64_t M, DType) { return N * C * 2 < (int64_t(1) << 31) && M * C < (int64_t(1) << 31); }
hipError_t launch_spmm_2of4(const void*, int64_t, int64_t, const void*, const uint16_t*, int64_t, const float*,
                            const float*, const void*, int32_t, void*, DType, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_td_mask(const float*, int64_t, int64_t, int32_t, int32_t, const uint32_t*, uint64_t, void*, DType,
                          uint8_t*, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_grad_packed(const void*, const void*, DType, int64_t, int64_t, const uint8_t*, int64_t, int32_t,
                              int32_t, float*, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}
int64_t index_stream_bytes(int64_t n, int32_t b) { return b == 8 ? n : (n * b + 31) / 32 * 4; }
hipError_t launch_index_bits(const uint8_t*, int64_t, int32_t, uint32_t*, hipStream_t) { ++g_launches; return hipSuccess; }
bool spmm_bits_supports(int64_t N, int64_t C, int64_t O, int32_t, int32_t) { return N <= 64 && C % 32 == 0 && O % 4 == 0; }
hipError_t launch_spmm_bits(const void*, int64_t, int64_t, const void*, const void*, int32_t, int64_t, int32_t, int32_t,
                            const float*, const float*, const void*, int32_t, void*, DType, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_maxpool(const void*, DType, int64_t, int64_t, int64_t, int64_t, int32_t, int32_t, int32_t, void*,
                          hipStream_t) {
  ++g_launches;
  return hipSuccess;
}
hipError_t launch_avgpool(const void*, DType, int64_t, int64_t, int64_t, int64_t, void*, DType, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}

}  // namespace cci
