// Host-side launcher interface between the C ABI layer (cci_api.cpp) and the
// kernel translation units.  Every launcher assumes validated arguments and
// returns the HIP status of its launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "cci_types.hpp"

namespace cci {

// Per-device set-up that a launcher needs once (a kernel's dynamic-LDS
// limit, an occupancy query).  Slot d holds the result for HIP device d,
// computed on the first launch with d current; a racing first launch on
// another thread computes the same value again, which is harmless.  These
// are the only values the library keeps between calls.
constexpr int kMaxDevices = 64;

inline int current_device() {
  int d = 0;
  if (hipGetDevice(&d) != hipSuccess || d < 0 || d >= kMaxDevices) return -1;
  return d;
}

// Raises `fn`'s dynamic-LDS limit to `bytes` once per device.
inline hipError_t set_lds_limit_once(std::atomic<int8_t> (&done)[kMaxDevices], const void* fn,
                                     int bytes) {
  const int d = current_device();
  if (d >= 0 && done[d].load(std::memory_order_acquire)) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess && d >= 0) done[d].store(1, std::memory_order_release);
  return e;
}

enum class DType { F32 = 0, BF16 = 1 };

struct ProductArgs {
  const void* X;
  DType x_t;
  int64_t N, C;          // GEMM rows / reduction length
  bool conv;
  int64_t B;             // conv: batch
  ConvGeom geom;         // conv only
  const void* vals;
  DType val_t;
  const uint8_t* idx;
  int64_t O;
  int32_t G, K;
  const float* scale;
  const float* bias;
  const void* residual;
  int32_t relu;
  void* Y;
  DType y_t;
};

hipError_t launch_pack(const float* W, int64_t O, int64_t C, int32_t G, int32_t K,
                       void* vals, DType val_t, uint8_t* idx, hipStream_t s);

// Alg. 1 dataflow on the vector ALUs (any dtype combination, G in {2,4,8,16,32}).
bool sparse_mac_supports(const ProductArgs& a);
hipError_t launch_sparse_mac(const ProductArgs& a, hipStream_t s);

// Packed groups expanded to dense bf16 tiles in LDS, bf16 MFMA.
bool dense_tile_supports(const ProductArgs& a);
hipError_t launch_dense_tile(const ProductArgs& a, hipStream_t s);

// The same expansion with 256 x 256 workgroup tiles and four waves of 128 x
// 128 accumulators (FC and stride-1 1x1 convolutions; bf16; C % 64 == 0,
// O % 256 == 0, 64 % G == 0).
bool wide_tile_supports(const ProductArgs& a);
hipError_t launch_wide_tile(const ProductArgs& a, hipStream_t s);

// Short reductions (C <= 256, C % 8 == 0): expanded weights of up to 80
// outputs per wave held in registers, pixels streamed through them (FC,
// stride-1 1x1 convolutions, and implicit-im2col convolutions with
// Cin % 8 == 0 or Cin == 4 and an even KW; bf16; O % 4 == 0).
bool narrow_supports(const ProductArgs& a);
hipError_t launch_narrow(const ProductArgs& a, hipStream_t s);

// k x k convolutions with unit stride and few outputs (3x3, Cin 32 or 64, O 32
// or 64; bf16): the expanded weights stay in registers for the whole launch,
// and each workgroup stages the input rows under its band of output rows in
// LDS once.
bool resident_supports(const ProductArgs& a);
hipError_t launch_resident(const ProductArgs& a, hipStream_t s);

// Convolutions of any geometry (implicit im2col) and FC products whose
// reduction splits into chunks of 64 channels under one tap (Cin % 64 == 0):
// 128 x 128 workgroup tiles, two workgroups per CU (bf16; O % 128 == 0,
// 32 % G == 0, KH * KW <= 32).
bool tap_tile_supports(const ProductArgs& a);
hipError_t launch_tap_tile(const ProductArgs& a, hipStream_t s);

// FC products and stride-1 1x1 convolutions with 64 <= C <= 256: a workgroup
// expands its 128 (or 64) outputs' weights over the whole reduction once and
// streams 128-row tiles of X past them (bf16 X/vals; C % 64 == 0,
// O % 64 == 0, 32 % G == 0).
bool stream_tile_supports(const ProductArgs& a);
hipError_t launch_stream_tile(const ProductArgs& a, hipStream_t s);

// Few row tiles over a long reduction: eight waves of a workgroup split the
// reduction of one 16 RF x 16 OF tile, each building its weight fragments in
// registers from the packed entries (bf16 X/vals; FC or stride-1 unpadded
// 1x1; C % 32 == 0, O % 16 == 0, K <= 4).
bool split_k_supports(const ProductArgs& a);
hipError_t launch_split_k(const ProductArgs& a, hipStream_t s);

// Balanced sparsity (groups of G inputs in one output row) and the 2:4
// sparse matrix-core product.
hipError_t launch_bbs_pack(const float* W, int64_t O, int64_t C, int32_t G, int32_t K, void* vals, DType val_t,
                           uint8_t* idx, hipStream_t s);
// Prepared 2:4 operand from a balanced packing (rows O, reduction C) or, with
// from_cci, from a CCI packing of W_hat [O][C] as the operand of W_hat^T
// (rows C, reduction O).  bf16 values; K <= 2, G % 4 == 0, reduction % 64 == 0,
// rows % 16 == 0.
hipError_t launch_to_2of4(bool from_cci, const void* vals, const uint8_t* idx, int64_t O, int64_t C, int32_t G,
                          int32_t K, void* av, uint16_t* ai, hipStream_t s);
bool spmm_2of4_fits(int64_t N, int64_t C, int64_t M, DType y_t);
hipError_t launch_spmm_2of4(const void* X, int64_t N, int64_t C, const void* av, const uint16_t* ai, int64_t M,
                            const float* scale, const float* bias, const void* residual, int32_t relu, void* Y,
                            DType y_t, hipStream_t s);

// Improved targeted dropout: candidate dropout of one step, and the gradient
// of the packed values of a CCI layer.
hipError_t launch_td_mask(const float* W, int64_t O, int64_t C, int32_t G, int32_t n_target, const uint32_t* bits,
                          uint64_t thr, void* We, DType w_t, uint8_t* keep, hipStream_t s);
hipError_t launch_grad_packed(const void* dY, const void* X, DType t, int64_t N, int64_t C, const uint8_t* idx,
                              int64_t O, int32_t G, int32_t K, float* dv, hipStream_t s);
// The same gradient on the matrix cores (bf16 dY and X, O % 8 == 0,
// C % 8 == 0, 128 % G == 0): dense 256 x 256 tiles of dY^T X, kept entries
// gathered.
bool grad_mfma_supports(const void* dY, const void* X, DType t, int64_t N, int64_t C, int64_t O, int32_t G);
hipError_t launch_grad_mfma(const void* dY, const void* X, int64_t N, int64_t C, const uint8_t* idx, int64_t O,
                            int32_t G, int32_t K, float* dv, hipStream_t s);

// Plain log2(G)-bit index streams and the few-row product that reads them.
int64_t index_stream_bytes(int64_t n, int32_t b);
hipError_t launch_index_bits(const uint8_t* idx, int64_t n, int32_t b, uint32_t* words, hipStream_t s);
bool spmm_bits_supports(int64_t N, int64_t C, int64_t O, int32_t G, int32_t K);
hipError_t launch_spmm_bits(const void* X, int64_t N, int64_t C, const void* vals, const void* idx, int32_t b,
                            int64_t O, int32_t G, int32_t K, const float* scale, const float* bias,
                            const void* residual, int32_t relu, void* Y, DType y_t, hipStream_t s);

hipError_t launch_maxpool(const void* X, DType t, int64_t B, int64_t H, int64_t W, int64_t C,
                          int32_t k, int32_t st, int32_t p, void* Y, hipStream_t s);
hipError_t launch_avgpool(const void* X, DType x_t, int64_t B, int64_t H, int64_t W, int64_t C,
                          void* Y, DType y_t, hipStream_t s);

}  // namespace cci
