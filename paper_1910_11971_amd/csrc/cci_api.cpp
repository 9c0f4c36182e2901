// C ABI of the CCI library: argument validation, kernel-family choice and
// error reporting.  Nothing here allocates, synchronises or keeps state other
// than the calling thread's last error message.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "../../include/cci.h"
#include "cci_launch.hpp"

namespace {

thread_local char g_last_error[512] = "";

cci_status fail(cci_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
  return s;
}

cci_status ok() {
  g_last_error[0] = '\0';
  return CCI_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// B * H * W * C < lim, checked without overflow (B >= 0; H, W, C >= 1).
bool fits_nhwc(int64_t B, int64_t H, int64_t W, int64_t C, int64_t lim) {
  if (W > lim || H > lim / W) return false;  // H * W <= lim
  const int64_t hw = H * W;
  if (C > lim / hw) return false;            // H * W * C <= lim
  return B <= (lim - 1) / (hw * C);          // B * H * W * C <= lim - 1
}

bool dtype_ok(cci_dtype t) { return t == CCI_F32 || t == CCI_BF16; }

cci::DType to_dt(cci_dtype t) { return t == CCI_F32 ? cci::DType::F32 : cci::DType::BF16; }

size_t dsize(cci_dtype t) { return t == CCI_F32 ? 4 : 2; }

cci_status check_groups(int64_t O, int64_t C, int32_t G, int32_t K) {
  if (G < 1 || G > 256) return fail(CCI_EINVAL, "G=%d outside [1, 256]", G);
  if (K < 1 || K > G) return fail(CCI_EINVAL, "K=%d outside [1, G=%d]", K, G);
  if (O < 1 || O % G != 0) return fail(CCI_EINVAL, "O=%lld is not a positive multiple of G=%d", (long long)O, G);
  if (C < 1) return fail(CCI_EINVAL, "C=%lld < 1", (long long)C);
  // packed arrays and grids are indexed with 64-bit offsets; keep element
  // counts well inside what the launch grids can cover
  if (O > (int64_t(1) << 31) || C > (int64_t(1) << 31) || O * C > (int64_t(1) << 40))
    return fail(CCI_EINVAL, "O*C too large");
  return CCI_OK;
}

cci_status check_types(cci_dtype x_t, cci_dtype val_t, cci_dtype y_t) {
  if (!dtype_ok(x_t) || !dtype_ok(val_t) || !dtype_ok(y_t))
    return fail(CCI_EINVAL, "unknown dtype code");
  const bool f32 = x_t == CCI_F32 && val_t == CCI_F32 && y_t == CCI_F32;
  const bool bf = x_t == CCI_BF16 && val_t == CCI_BF16;
  if (!f32 && !bf)
    return fail(CCI_EUNSUPPORTED, "dtype combination (x=%d, vals=%d, y=%d) not supported", x_t,
                val_t, y_t);
  return CCI_OK;
}

// The few-row product of cci_spmm_bits, reading the byte indices of
// cci_pack (8-bit entries): FC products and 1x1 convolutions whose rows are
// the pixels.
bool few_rows_ok(const cci::ProductArgs& a) {
  if (a.x_t != cci::DType::BF16 || a.val_t != cci::DType::BF16) return false;
  if (a.conv) {
    const cci::ConvGeom& g = a.geom;
    if (g.KH != 1 || g.KW != 1 || g.sh != 1 || g.sw != 1 || g.ph != 0 || g.pw != 0) return false;
  }
  return cci::spmm_bits_supports(a.N, a.C, a.O, a.G, a.K);
}

cci_status run_product(cci::ProductArgs& a, cci_algo algo, const cci_epilogue* ep,
                       void* stream) {
  a.scale = ep ? ep->scale : nullptr;
  a.bias = ep ? ep->bias : nullptr;
  a.residual = ep ? ep->residual : nullptr;
  a.relu = ep ? ep->relu : 0;
  if ((a.scale && !aligned16(a.scale)) || (a.bias && !aligned16(a.bias)) ||
      (a.residual && !aligned16(a.residual)))
    return fail(CCI_EALIGN, "epilogue pointer not 16-byte aligned");
  if (algo != CCI_ALGO_AUTO && algo != CCI_ALGO_SPARSE_MAC && algo != CCI_ALGO_DENSE_TILE_MFMA &&
      algo != CCI_ALGO_WIDE_TILE_MFMA && algo != CCI_ALGO_NARROW_MFMA && algo != CCI_ALGO_RESIDENT_MFMA &&
      algo != CCI_ALGO_FEW_ROWS_MFMA && algo != CCI_ALGO_TAP_TILE_MFMA && algo != CCI_ALGO_STREAM_TILE_MFMA &&
      algo != CCI_ALGO_SPLIT_K_MFMA)
    return fail(CCI_EINVAL, "unknown algo %d", (int)algo);
  if (a.N == 0) return ok();

  const bool mac_ok = cci::sparse_mac_supports(a);
  const bool tile_ok = cci::dense_tile_supports(a);
  cci_algo chosen = algo;
  if (algo == CCI_ALGO_AUTO) {
    const int64_t cin = a.conv ? a.geom.Cin : a.C;
    chosen = cci_auto_algo(a.x_t == cci::DType::F32 ? CCI_F32 : CCI_BF16,
                           a.val_t == cci::DType::F32 ? CCI_F32 : CCI_BF16, a.N, a.C, cin, a.O,
                           a.G, a.K);
  }
  // (the shape-only choice cannot see stride and padding)
  if (algo == CCI_ALGO_AUTO && chosen == CCI_ALGO_FEW_ROWS_MFMA && !few_rows_ok(a))
    chosen = tile_ok ? CCI_ALGO_DENSE_TILE_MFMA : CCI_ALGO_SPARSE_MAC;
  if (algo == CCI_ALGO_AUTO && chosen == CCI_ALGO_RESIDENT_MFMA && !cci::resident_supports(a))
    chosen = tile_ok ? CCI_ALGO_DENSE_TILE_MFMA : CCI_ALGO_SPARSE_MAC;
  if (algo == CCI_ALGO_AUTO && chosen == CCI_ALGO_WIDE_TILE_MFMA && !cci::wide_tile_supports(a))
    chosen = cci::tap_tile_supports(a) ? CCI_ALGO_TAP_TILE_MFMA : CCI_ALGO_DENSE_TILE_MFMA;
  if (algo == CCI_ALGO_AUTO && chosen == CCI_ALGO_NARROW_MFMA && !cci::narrow_supports(a))
    chosen = tile_ok ? CCI_ALGO_DENSE_TILE_MFMA : CCI_ALGO_SPARSE_MAC;
  if (algo == CCI_ALGO_AUTO && chosen == CCI_ALGO_TAP_TILE_MFMA && !cci::tap_tile_supports(a))
    chosen = tile_ok ? CCI_ALGO_DENSE_TILE_MFMA : CCI_ALGO_SPARSE_MAC;
  if (algo == CCI_ALGO_AUTO && chosen == CCI_ALGO_STREAM_TILE_MFMA && !cci::stream_tile_supports(a))
    chosen = cci::tap_tile_supports(a) ? CCI_ALGO_TAP_TILE_MFMA : tile_ok ? CCI_ALGO_DENSE_TILE_MFMA : CCI_ALGO_SPARSE_MAC;
  if (algo == CCI_ALGO_AUTO && chosen == CCI_ALGO_SPLIT_K_MFMA && !cci::split_k_supports(a))
    chosen = tile_ok ? CCI_ALGO_DENSE_TILE_MFMA : CCI_ALGO_SPARSE_MAC;
  if (chosen == CCI_ALGO_SPARSE_MAC && !mac_ok)
    return fail(CCI_EUNSUPPORTED, "sparse-MAC kernels need G in {2,4,8,16,32} (G=%d)", a.G);
  if (chosen == CCI_ALGO_DENSE_TILE_MFMA && !tile_ok)
    return fail(CCI_EUNSUPPORTED,
                "dense-tile MFMA kernels need bf16 X/vals, 64 %% G == 0 and C (conv: Cin) %% 32 == 0");
  if (chosen == CCI_ALGO_WIDE_TILE_MFMA && !cci::wide_tile_supports(a))
    return fail(CCI_EUNSUPPORTED,
                "wide-tile MFMA kernels need bf16 X/vals, an FC or stride-1 unpadded 1x1 product, "
                "C %% 64 == 0, O %% 256 == 0, 64 %% G == 0 and aligned pointers");
  if (chosen == CCI_ALGO_FEW_ROWS_MFMA && !few_rows_ok(a))
    return fail(CCI_EUNSUPPORTED,
                "few-row MFMA kernels need bf16 X/vals, an FC or stride-1 unpadded 1x1 product, N <= 64, "
                "C %% 32 == 0 and O %% 4 == 0");
  if (chosen == CCI_ALGO_RESIDENT_MFMA && !cci::resident_supports(a))
    return fail(CCI_EUNSUPPORTED,
                "resident MFMA kernels need bf16 X/vals, a 3x3 convolution with unit stride and padding "
                "below 3, Cin 32 or 64, O 32 or 64, aligned pointers and at most 5120 packed 8-column units");
  if (chosen == CCI_ALGO_NARROW_MFMA && !cci::narrow_supports(a))
    return fail(CCI_EUNSUPPORTED,
                "narrow MFMA kernels need bf16 X/vals, C <= 256, C %% 8 == 0, O %% 4 == 0, G <= 256, "
                "aligned pointers, and for a conv other than 1x1 stride 1 unpadded Cin %% 8 == 0 or "
                "Cin == 4 with an even KW");
  if (chosen == CCI_ALGO_TAP_TILE_MFMA && !cci::tap_tile_supports(a))
    return fail(CCI_EUNSUPPORTED,
                "tap-tile MFMA kernels need bf16 X/vals, Cin (FC: C) %% 64 == 0, O %% 128 == 0 with 32 %% G == 0 "
                "or O %% 64 == 0 with 16 %% G == 0, 2 K <= G or K == G, at most 32 filter taps and aligned "
                "pointers");
  if (chosen == CCI_ALGO_STREAM_TILE_MFMA && !cci::stream_tile_supports(a))
    return fail(CCI_EUNSUPPORTED,
                "stream-tile MFMA kernels need bf16 X/vals, an FC or stride-1 unpadded 1x1 product, "
                "C %% 64 == 0 with C <= 256, O %% 64 == 0, 32 %% G == 0 and aligned pointers");
  if (chosen == CCI_ALGO_SPLIT_K_MFMA && !cci::split_k_supports(a))
    return fail(CCI_EUNSUPPORTED,
                "split-K MFMA kernels need bf16 X/vals, an FC or stride-1 unpadded 1x1 product, "
                "C %% 32 == 0, O %% 16 == 0, K <= 4 and 16-byte aligned pointers");
  const hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = chosen == CCI_ALGO_SPARSE_MAC       ? cci::launch_sparse_mac(a, st)
                 : chosen == CCI_ALGO_SPLIT_K_MFMA   ? cci::launch_split_k(a, st)
                 : chosen == CCI_ALGO_STREAM_TILE_MFMA ? cci::launch_stream_tile(a, st)
                 : chosen == CCI_ALGO_TAP_TILE_MFMA  ? cci::launch_tap_tile(a, st)
                 : chosen == CCI_ALGO_WIDE_TILE_MFMA ? cci::launch_wide_tile(a, st)
                 : chosen == CCI_ALGO_RESIDENT_MFMA  ? cci::launch_resident(a, st)
                 : chosen == CCI_ALGO_FEW_ROWS_MFMA
                     ? cci::launch_spmm_bits(a.X, a.N, a.C, a.vals, a.idx, 8, a.O, a.G, a.K, a.scale, a.bias,
                                             a.residual, a.relu, a.Y, a.y_t, st)
                 : chosen == CCI_ALGO_NARROW_MFMA    ? cci::launch_narrow(a, st)
                                                     : cci::launch_dense_tile(a, st);
  if (e != hipSuccess) return fail(CCI_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

// ---------------------------------------------------------------------------
// Balanced sparsity and the 2:4 sparse matrix-core product.

cci_status check_bbs_groups(int64_t O, int64_t C, int32_t G, int32_t K) {
  if (G < 1 || G > 256) return fail(CCI_EINVAL, "G=%d outside [1, 256]", G);
  if (K < 1 || K > G) return fail(CCI_EINVAL, "K=%d outside [1, G=%d]", K, G);
  if (O < 1) return fail(CCI_EINVAL, "O=%lld < 1", (long long)O);
  if (C < 1 || C % G != 0) return fail(CCI_EINVAL, "C=%lld is not a positive multiple of G=%d", (long long)C, G);
  if (O > (int64_t(1) << 31) || C > (int64_t(1) << 31) || O * C > (int64_t(1) << 40))
    return fail(CCI_EINVAL, "O*C too large");
  return CCI_OK;
}

cci_status check_2of4(int64_t M, int64_t R) {
  if (M < 16 || M % 16 != 0) return fail(CCI_EUNSUPPORTED, "2:4 operand rows M=%lld must be a positive multiple of 16", (long long)M);
  if (R < 64 || R % 64 != 0)
    return fail(CCI_EUNSUPPORTED, "2:4 operand reduction length %lld must be a positive multiple of 64", (long long)R);
  if (M * R >= (int64_t(1) << 31)) return fail(CCI_EINVAL, "2:4 operand too large");
  return CCI_OK;
}

cci_status to_2of4(bool from_cci, const void* vals, cci_dtype val_t, const uint8_t* idx, int64_t O, int64_t C,
                   int32_t G, int32_t K, void* a_vals, uint16_t* a_idx, void* stream) {
  if (cci_status s = from_cci ? check_groups(O, C, G, K) : check_bbs_groups(O, C, G, K)) return s;
  if (!dtype_ok(val_t)) return fail(CCI_EINVAL, "unknown dtype code");
  if (val_t != CCI_BF16) return fail(CCI_EUNSUPPORTED, "the 2:4 operand holds bf16 values");
  if (G % 4 != 0 || K > 2)
    return fail(CCI_EUNSUPPORTED,
                "a 2:4 operand needs at most 2 kept weights in every aligned run of 4: G %% 4 == 0 and K <= 2 "
                "(G=%d, K=%d)", G, K);
  if (cci_status s = from_cci ? check_2of4(C, O) : check_2of4(O, C)) return s;
  if (!vals || !idx || !a_vals || !a_idx) return fail(CCI_EINVAL, "null pointer");
  if (!aligned16(vals) || !aligned16(idx) || !aligned16(a_vals) || !aligned16(a_idx))
    return fail(CCI_EALIGN, "pointer not 16-byte aligned");
  hipError_t e = cci::launch_to_2of4(from_cci, vals, idx, O, C, G, K, a_vals, a_idx, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(CCI_EHIP, "2:4 conversion launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

int32_t cci_version(void) { return 100; }

const char* cci_status_str(cci_status s) {
  switch (s) {
    case CCI_OK: return "CCI_OK";
    case CCI_EINVAL: return "CCI_EINVAL: invalid argument";
    case CCI_EUNSUPPORTED: return "CCI_EUNSUPPORTED: not supported by this build";
    case CCI_EALIGN: return "CCI_EALIGN: pointer not 16-byte aligned";
    case CCI_EHIP: return "CCI_EHIP: HIP runtime error";
  }
  return "unknown cci_status";
}

const char* cci_last_error(void) { return g_last_error; }

cci_status cci_packed_sizes(int64_t O, int64_t C, int32_t G, int32_t K, cci_dtype val_t,
                            size_t* val_bytes, size_t* idx_bytes) {
  if (cci_status s = check_groups(O, C, G, K)) return s;
  if (!dtype_ok(val_t)) return fail(CCI_EINVAL, "unknown dtype code");
  if (!val_bytes || !idx_bytes) return fail(CCI_EINVAL, "null output pointer");
  const size_t n = static_cast<size_t>(O / G) * static_cast<size_t>(K) * static_cast<size_t>(C);
  *val_bytes = n * dsize(val_t);
  *idx_bytes = n;
  return ok();
}

cci_status cci_pack(const float* W, int64_t O, int64_t C, int32_t G, int32_t K, void* vals,
                    cci_dtype val_t, uint8_t* idx, void* stream) {
  if (cci_status s = check_groups(O, C, G, K)) return s;
  if (!dtype_ok(val_t)) return fail(CCI_EINVAL, "unknown dtype code");
  if (!W || !vals || !idx) return fail(CCI_EINVAL, "null pointer");
  if (!aligned16(W) || !aligned16(vals) || !aligned16(idx))
    return fail(CCI_EALIGN, "pointer not 16-byte aligned");
  hipError_t e = cci::launch_pack(W, O, C, G, K, vals, to_dt(val_t), idx,
                                  static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(CCI_EHIP, "pack launch failed: %s", hipGetErrorString(e));
  return ok();
}

cci_algo cci_auto_algo(cci_dtype x_t, cci_dtype val_t, int64_t N, int64_t C, int64_t cin,
                       int64_t O, int32_t G, int32_t K) {
  // The matrix cores multiply the expanded tile at 2516.6 dense bf16 TFLOP/s;
  // the vector ALUs multiply only kept weights at 78.6 fp32 TFLOP/s (no
  // packed fp32).  Expanded work is G/K times the kept work, so the tile
  // path wins whenever K/G > 78.6/2516.6 (about 1/32).
  const bool bf = x_t == CCI_BF16 && val_t == CCI_BF16 && G >= 1 && 64 % G == 0;
  // Up to 64 rows every packed weight feeds at most 64 multiply-adds: the
  // packed bytes set the time, and the few-row kernel (one expanded 16 x 32
  // tile per k-step and wave, read once) takes 7-24 us on a 4096 x 4096
  // layer where the tile kernels need 55-70 us.
  // (A ragged last tile, O % 16 != 0, stays on the tile kernels: ResNet-50's
  // 64 x 2048 -> 1000 classifier inside the forward, its 6 MB of weights
  // cold, takes 35.5 us here against 27.1 us on the dense-tile kernel; 18.9
  // us here with the weights warm in cache.)
  if (x_t == CCI_BF16 && val_t == CCI_BF16 && C == cin && N <= 64 && C % 32 == 0 && O % 16 == 0)
    return CCI_ALGO_FEW_ROWS_MFMA;
  // 3x3 convolutions over 32 or 64 channels into 32 or 64 outputs: their
  // whole expanded tile fits in registers, so it is expanded once per
  // workgroup and only activations stream (measured 2-3x the dense-tile
  // kernel on a 32 x 56 x 56 x 64 -> 64 layer).  Only unit stride is taken:
  // other strides run on the dense-tile kernels.
  if (x_t == CCI_BF16 && val_t == CCI_BF16 && (cin == 32 || cin == 64) && C == 9 * cin && (O == 32 || O == 64) &&
      O % G == 0)
    return CCI_ALGO_RESIDENT_MFMA;
  const bool mac_g = G == 2 || G == 4 || G == 8 || G == 16 || G == 32;
  const bool narrow_shape = x_t == CCI_BF16 && val_t == CCI_BF16 && C <= 256 && C % 8 == 0 && O % 4 == 0 &&
                            (cin == 4 || cin % 8 == 0);
  // The tap-chunk kernels (128 x 128 or 128 x 64 tiles, reduction in
  // 64-channel chunks under one filter tap): every k x k convolution over a
  // multiple of 64 channels into a multiple of 128 outputs, strided 1x1
  // layers, and FC / 1x1 products the wide-tile kernels do not fill the chip
  // with.  Measured on ResNet-50's layers at batch 64 against the previous
  // choice: 3x3 stride 2 28.9 vs 112.6 us (Cin 128), 31.5 vs 109.1 us (Cin
  // 256), 45 vs 99 us (Cin 512); 3x3 stride 1 28.6 vs 38.4 us (Cin 128);
  // strided 1x1 26-36 vs 37-45 us; 12544 x 1024 x 256 18.5 vs 23.3 us; the
  // bottleneck 1x1 layers with their residual add 52 vs 64 us (64 -> 256,
  // 200 704 pixels) and 35 vs 39 us (128 -> 512, 50 176 pixels).
  // A reduction of one 64-channel chunk leaves their pipeline empty: such
  // products never go to them (MobileNetV2's 12544 x 64 -> 384: 9.4 us
  // there, 8.0 us on the dense-tile kernels; from 100 K rows on, the
  // streaming kernels below take them).
  const bool tap_fits = x_t == CCI_BF16 && val_t == CCI_BF16 && G >= 1 && 32 % G == 0 && (2 * K <= G || K == G) &&
                        cin % 64 == 0 && O % 128 == 0 && C / cin <= 32;
  const bool tap_shape = tap_fits && C >= 128;
  // Short reductions the tile kernels cannot take (Cin % 32 != 0) stream
  // through register-resident weights (narrow kernels): 1x1 layers and FC
  // products with C % 8 == 0, and convolutions over 4 input channels (an
  // even KW) or a multiple of 8.  Large 1x1 / FC products with C <= 128 do
  // too (8-20% ahead of the dense-tile kernels at 50 K - 800 K rows) unless
  // the streaming (C = 64) or tap-chunk (C = 128, O % 128 == 0) kernels
  // take them.
  const bool narrow_large = C == cin && C <= 128 && N >= 100000;
  // One 64-channel chunk over >= 100 K rows: the streaming kernels (the
  // expanded tile expanded once per workgroup, 128-row tiles streamed past
  // it): 64 -> 256 at 200 704 rows 37 vs 41-48 us (with a residual 47 vs
  // 53 us), 64 -> 64 17 vs 19-22 us.
  if (x_t == CCI_BF16 && val_t == CCI_BF16 && C == 64 && cin == 64 && N >= 100000 && O % 64 == 0 && G >= 1 &&
      32 % G == 0)
    return CCI_ALGO_STREAM_TILE_MFMA;
  if (tap_fits && narrow_large) return CCI_ALGO_TAP_TILE_MFMA;
  if (narrow_shape && (cin % 32 != 0 || narrow_large)) return CCI_ALGO_NARROW_MFMA;
  // Long reductions over few row tiles (the late projecting 1x1 layers of
  // MobileNetV2 at batch 64, 3 136 rows): the tile kernels walk 9-15
  // 64-channel chunks one memory round trip at a time on a fraction of the
  // CUs.  When 64 x 32 tiles fill at most one round of the chip, the
  // split-reduction kernels take them (576 -> 160: 8.0 vs 13.4 us; 960 ->
  // 160: 10.8 vs 19.5 us; 512 x 512 -> 320: 4.9 vs 7.9 us; 256 x 1024 ->
  // 160: 6.1 vs 12.0 us); else, with O % 64 == 0, the tap-chunk kernels'
  // 64-output tiles (960 -> 320: 13.6 us vs 15.4 split, 20.8 dense-tile).
  // From 12 544 rows on the dense-tile kernels stay ahead (576 -> 96: 14.6
  // vs 20.2 us; 384 -> 64: 8.7 vs 9.1 tap, 9.5 split).  O % 128 == 0 keeps
  // the routes below (tap-chunk or wide-tile), measured on ResNet-50.
  if (x_t == CCI_BF16 && val_t == CCI_BF16 && C == cin && C >= 512 && C <= 1024 && C % 32 == 0 && O % 16 == 0 &&
      O % 128 != 0) {
    // (at C = 512 two k-steps per wave: half a round at most; 4096 x 512 ->
    // 96 is 9.0 us split, 8.3 us dense-tile)
    const int64_t t64x32 = (N + 63) / 64 * ((O + 31) / 32);
    if (t64x32 <= (C >= 576 ? 256 : 128) && K <= 4) return CCI_ALGO_SPLIT_K_MFMA;
    if (O % 64 == 0 && G <= 16 && 16 % G == 0 && (2 * K <= G || K == G)) return CCI_ALGO_TAP_TILE_MFMA;
  }
  // FC and 1x1 products with a reduction of >= 256 that fill the chip with
  // 256 x 256 tiles (>= 128 of them) run on the wide-tile kernels: 2.2-2.4x
  // the dense-tile kernel on 4096^3, and level with the tap-chunk kernels on
  // ResNet-50's 1x1 layers with 196 such tiles.
  const int64_t tiles256 = (N + 255) / 256 * (O / 256);
  if (bf && C == cin && C % 64 == 0 && C >= 256 && O % 256 == 0 && tiles256 >= 128) return CCI_ALGO_WIDE_TILE_MFMA;
  if (tap_shape) return CCI_ALGO_TAP_TILE_MFMA;
  const bool tile_shape = bf && cin % 32 == 0;
  if (tile_shape && (32 * static_cast<int64_t>(K) > G || !mac_g)) return CCI_ALGO_DENSE_TILE_MFMA;
  return CCI_ALGO_SPARSE_MAC;
}

cci_status cci_spmm_algo(const void* X, cci_dtype x_t, int64_t N, int64_t C, const void* vals,
                         cci_dtype val_t, const uint8_t* idx, int64_t O, int32_t G, int32_t K,
                         const cci_epilogue* ep, void* Y, cci_dtype y_t, cci_algo algo, void* stream) {
  if (cci_status s = check_groups(O, C, G, K)) return s;
  if (N < 0) return fail(CCI_EINVAL, "N=%lld < 0", (long long)N);
  if (cci_status s = check_types(x_t, val_t, y_t)) return s;
  if (N > 0 && (!X || !vals || !idx || !Y)) return fail(CCI_EINVAL, "null pointer");
  if (N > (int64_t(1) << 40) / (C > O ? C : O)) return fail(CCI_EINVAL, "N too large");
  if (N > 0 && (!aligned16(X) || !aligned16(vals) || !aligned16(idx) || !aligned16(Y)))
    return fail(CCI_EALIGN, "pointer not 16-byte aligned");
  cci::ProductArgs a{};
  a.X = X;
  a.x_t = to_dt(x_t);
  a.N = N;
  a.C = C;
  a.conv = false;
  a.vals = vals;
  a.val_t = to_dt(val_t);
  a.idx = idx;
  a.O = O;
  a.G = G;
  a.K = K;
  a.Y = Y;
  a.y_t = to_dt(y_t);
  return run_product(a, algo, ep, stream);
}

cci_status cci_conv_im2col_algo(const void* X, cci_dtype x_t, int64_t B, int64_t H, int64_t W,
                                int64_t Cin, int32_t KH, int32_t KW, int32_t stride_h,
                                int32_t stride_w, int32_t pad_h, int32_t pad_w, const void* vals,
                                cci_dtype val_t, const uint8_t* idx, int64_t O, int32_t G,
                                int32_t K, const cci_epilogue* ep, void* Y, cci_dtype y_t,
                                cci_algo algo, void* stream) {
  if (B < 0 || H < 1 || W < 1 || Cin < 1 || KH < 1 || KW < 1 || stride_h < 1 || stride_w < 1 ||
      pad_h < 0 || pad_w < 0)
    return fail(CCI_EINVAL, "bad convolution geometry");
  if (H > (1 << 20) || W > (1 << 20) || Cin > (1 << 24) || KH > 64 || KW > 64 ||
      pad_h > 64 || pad_w > 64 || stride_h > 64 || stride_w > 64)
    return fail(CCI_EINVAL, "convolution geometry out of range");
  if (H + 2 * pad_h < KH || W + 2 * pad_w < KW) return fail(CCI_EINVAL, "kernel larger than padded input");
  const int64_t C = static_cast<int64_t>(KH) * KW * Cin;
  if (cci_status s = check_groups(O, C, G, K)) return s;
  if (cci_status s = check_types(x_t, val_t, y_t)) return s;
  const int64_t Ho = (H + 2 * pad_h - KH) / stride_h + 1;
  const int64_t Wo = (W + 2 * pad_w - KW) / stride_w + 1;
  if (!fits_nhwc(B, H, W, Cin, int64_t(1) << 31)) return fail(CCI_EINVAL, "input tensor too large");
  const int64_t N = B * Ho * Wo;  // B * H * W < 2^31 and Ho, Wo <= H, W + 128: no overflow
  if (N > (int64_t(1) << 40) / (C > O ? C : O)) return fail(CCI_EINVAL, "output too large");
  if (N > 0 && (!X || !vals || !idx || !Y)) return fail(CCI_EINVAL, "null pointer");
  if (N > 0 && (!aligned16(X) || !aligned16(vals) || !aligned16(idx) || !aligned16(Y)))
    return fail(CCI_EALIGN, "pointer not 16-byte aligned");
  cci::ProductArgs a{};
  a.X = X;
  a.x_t = to_dt(x_t);
  a.N = N;
  a.C = C;
  a.conv = true;
  a.B = B;
  a.geom = cci::ConvGeom{static_cast<int32_t>(H), static_cast<int32_t>(W),
                         static_cast<int32_t>(Cin), KH, KW, stride_h, stride_w, pad_h, pad_w,
                         static_cast<int32_t>(Ho), static_cast<int32_t>(Wo)};
  a.vals = vals;
  a.val_t = to_dt(val_t);
  a.idx = idx;
  a.O = O;
  a.G = G;
  a.K = K;
  a.Y = Y;
  a.y_t = to_dt(y_t);
  return run_product(a, algo, ep, stream);
}

cci_status cci_spmm(const void* X, cci_dtype x_t, int64_t N, int64_t C, const void* vals,
                    cci_dtype val_t, const uint8_t* idx, int64_t O, int32_t G, int32_t K,
                    const cci_epilogue* ep, void* Y, cci_dtype y_t, void* stream) {
  return cci_spmm_algo(X, x_t, N, C, vals, val_t, idx, O, G, K, ep, Y, y_t, CCI_ALGO_AUTO, stream);
}

cci_status cci_conv_im2col(const void* X, cci_dtype x_t, int64_t B, int64_t H, int64_t W,
                           int64_t Cin, int32_t KH, int32_t KW, int32_t stride_h, int32_t stride_w,
                           int32_t pad_h, int32_t pad_w, const void* vals, cci_dtype val_t,
                           const uint8_t* idx, int64_t O, int32_t G, int32_t K,
                           const cci_epilogue* ep, void* Y, cci_dtype y_t, void* stream) {
  return cci_conv_im2col_algo(X, x_t, B, H, W, Cin, KH, KW, stride_h, stride_w, pad_h, pad_w, vals,
                              val_t, idx, O, G, K, ep, Y, y_t, CCI_ALGO_AUTO, stream);
}

cci_status cci_bbs_packed_sizes(int64_t O, int64_t C, int32_t G, int32_t K, cci_dtype val_t,
                                size_t* val_bytes, size_t* idx_bytes) {
  if (cci_status s = check_bbs_groups(O, C, G, K)) return s;
  if (!dtype_ok(val_t)) return fail(CCI_EINVAL, "unknown dtype code");
  if (!val_bytes || !idx_bytes) return fail(CCI_EINVAL, "null output pointer");
  const size_t n = static_cast<size_t>(O) * static_cast<size_t>(C / G) * static_cast<size_t>(K);
  *val_bytes = n * dsize(val_t);
  *idx_bytes = n;
  return ok();
}

cci_status cci_bbs_pack(const float* W, int64_t O, int64_t C, int32_t G, int32_t K, void* vals,
                        cci_dtype val_t, uint8_t* idx, void* stream) {
  if (cci_status s = check_bbs_groups(O, C, G, K)) return s;
  if (!dtype_ok(val_t)) return fail(CCI_EINVAL, "unknown dtype code");
  if (!W || !vals || !idx) return fail(CCI_EINVAL, "null pointer");
  if (!aligned16(W) || !aligned16(vals) || !aligned16(idx)) return fail(CCI_EALIGN, "pointer not 16-byte aligned");
  hipError_t e = cci::launch_bbs_pack(W, O, C, G, K, vals, to_dt(val_t), idx, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(CCI_EHIP, "bbs pack launch failed: %s", hipGetErrorString(e));
  return ok();
}

cci_status cci_2of4_sizes(int64_t M, int64_t R, size_t* val_bytes, size_t* idx_bytes) {
  if (cci_status s = check_2of4(M, R)) return s;
  if (!val_bytes || !idx_bytes) return fail(CCI_EINVAL, "null output pointer");
  *val_bytes = static_cast<size_t>(M) * static_cast<size_t>(R);      // M x R/2 bf16
  *idx_bytes = static_cast<size_t>(M) * static_cast<size_t>(R) / 8;  // M x R/16 uint16
  return ok();
}

cci_status cci_bbs_to_2of4(const void* vals, cci_dtype val_t, const uint8_t* idx, int64_t O, int64_t C,
                           int32_t G, int32_t K, void* a_vals, uint16_t* a_idx, void* stream) {
  return to_2of4(false, vals, val_t, idx, O, C, G, K, a_vals, a_idx, stream);
}

cci_status cci_to_2of4_transposed(const void* vals, cci_dtype val_t, const uint8_t* idx, int64_t O, int64_t C,
                                  int32_t G, int32_t K, void* a_vals, uint16_t* a_idx, void* stream) {
  return to_2of4(true, vals, val_t, idx, O, C, G, K, a_vals, a_idx, stream);
}

cci_status cci_spmm_2of4(const void* X, cci_dtype x_t, int64_t N, int64_t R, const void* a_vals,
                         const uint16_t* a_idx, int64_t M, const cci_epilogue* ep, void* Y, cci_dtype y_t,
                         void* stream) {
  if (!dtype_ok(x_t) || !dtype_ok(y_t)) return fail(CCI_EINVAL, "unknown dtype code");
  if (x_t != CCI_BF16) return fail(CCI_EUNSUPPORTED, "the 2:4 product takes bf16 X");
  if (N < 0 || N >= (int64_t(1) << 31)) return fail(CCI_EINVAL, "N=%lld outside [0, 2^31)", (long long)N);
  if (cci_status s = check_2of4(M, R)) return s;
  if (!cci::spmm_2of4_fits(N, R, M, to_dt(y_t))) return fail(CCI_EINVAL, "product too large");
  const float* scale = ep ? ep->scale : nullptr;
  const float* bias = ep ? ep->bias : nullptr;
  const void* residual = ep ? ep->residual : nullptr;
  if ((scale && !aligned16(scale)) || (bias && !aligned16(bias)) || (residual && !aligned16(residual)))
    return fail(CCI_EALIGN, "epilogue pointer not 16-byte aligned");
  if (N == 0) return ok();
  if (!X || !a_vals || !a_idx || !Y) return fail(CCI_EINVAL, "null pointer");
  if (!aligned16(X) || !aligned16(a_vals) || !aligned16(a_idx) || !aligned16(Y))
    return fail(CCI_EALIGN, "pointer not 16-byte aligned");
  hipError_t e = cci::launch_spmm_2of4(X, N, R, a_vals, a_idx, M, scale, bias, residual, ep ? ep->relu : 0, Y,
                                       to_dt(y_t), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(CCI_EHIP, "2:4 product launch failed: %s", hipGetErrorString(e));
  return ok();
}

cci_status cci_td_schedule(int64_t step, int64_t total, int32_t G, int32_t K, int32_t* n_target,
                           double* drop_rate) {
  if (total < 1 || step < 0 || step > total) return fail(CCI_EINVAL, "step %lld outside [0, %lld]", (long long)step, (long long)total);
  if (G < 1 || G > 256 || K < 1 || K > G) return fail(CCI_EINVAL, "G=%d, K=%d out of range", G, K);
  if (!n_target || !drop_rate) return fail(CCI_EINVAL, "null output pointer");
  // first half: candidates ramp 0 -> G-K at dropout 1/2; second half: dropout 1/2 -> 1
  const double f = static_cast<double>(step) / static_cast<double>(total);
  const double ramp = f >= 0.5 ? 1.0 : 2.0 * f;
  *n_target = static_cast<int32_t>(std::floor(static_cast<double>(G - K) * ramp + 0.5));
  *drop_rate = f < 0.5 ? 0.5 : f;
  return ok();
}

cci_status cci_td_mask(const float* W, int64_t O, int64_t C, int32_t G, int32_t n_target, const uint32_t* bits,
                       double drop_rate, void* W_eff, cci_dtype w_t, uint8_t* keep, void* stream) {
  if (cci_status s = check_groups(O, C, G, 1)) return s;
  if (n_target < 0 || n_target > G) return fail(CCI_EINVAL, "n_target=%d outside [0, G=%d]", n_target, G);
  if (!(drop_rate >= 0.0 && drop_rate <= 1.0)) return fail(CCI_EINVAL, "drop_rate outside [0, 1]");
  if (!dtype_ok(w_t)) return fail(CCI_EINVAL, "unknown dtype code");
  if (!W || !bits || !W_eff || !keep) return fail(CCI_EINVAL, "null pointer");
  if (!aligned16(W) || !aligned16(bits) || !aligned16(W_eff) || !aligned16(keep))
    return fail(CCI_EALIGN, "pointer not 16-byte aligned");
  const uint64_t thr = static_cast<uint64_t>(std::floor(drop_rate * 4294967296.0));
  hipError_t e = cci::launch_td_mask(W, O, C, G, n_target, bits, thr, W_eff, to_dt(w_t), keep,
                                     static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(CCI_EHIP, "td mask launch failed: %s", hipGetErrorString(e));
  return ok();
}

cci_status cci_grad_packed(const void* dY, const void* X, cci_dtype t, int64_t N, int64_t C, const uint8_t* idx,
                           int64_t O, int32_t G, int32_t K, float* dvals, void* stream) {
  if (cci_status s = check_groups(O, C, G, K)) return s;
  if (!dtype_ok(t)) return fail(CCI_EINVAL, "unknown dtype code");
  if (N < 0) return fail(CCI_EINVAL, "N=%lld < 0", (long long)N);
  if (N > (int64_t(1) << 40) / (C > O ? C : O)) return fail(CCI_EINVAL, "N too large");
  if (!idx || !dvals) return fail(CCI_EINVAL, "null pointer");
  if (N > 0 && (!dY || !X)) return fail(CCI_EINVAL, "null pointer");
  if ((N > 0 && (!aligned16(dY) || !aligned16(X))) || !aligned16(idx) || !aligned16(dvals))
    return fail(CCI_EALIGN, "pointer not 16-byte aligned");
  hipError_t e = cci::launch_grad_packed(dY, X, to_dt(t), N, C, idx, O, G, K, dvals, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(CCI_EHIP, "packed-gradient launch failed: %s", hipGetErrorString(e));
  return ok();
}

int32_t cci_index_width(int32_t G) {
  if (G < 1 || G > 256) return -1;
  int32_t b = 1;
  while ((1 << b) < G) ++b;
  return b;
}

cci_status cci_index_stream_bytes(int64_t n, int32_t bits, size_t* bytes) {
  if (n < 0 || bits < 1 || bits > 8) return fail(CCI_EINVAL, "n=%lld or bits=%d out of range", (long long)n, bits);
  if (!bytes) return fail(CCI_EINVAL, "null output pointer");
  *bytes = static_cast<size_t>((n * bits + 31) / 32 * 4);
  return ok();
}

cci_status cci_index_bits(const uint8_t* idx, int64_t n, int32_t bits, uint32_t* words, void* stream) {
  if (n < 0 || n >= (int64_t(1) << 36) || bits < 1 || bits > 8)
    return fail(CCI_EINVAL, "n=%lld or bits=%d out of range", (long long)n, bits);
  if (n == 0) return ok();
  if (!idx || !words) return fail(CCI_EINVAL, "null pointer");
  if (!aligned16(idx) || !aligned16(words)) return fail(CCI_EALIGN, "pointer not 16-byte aligned");
  hipError_t e = cci::launch_index_bits(idx, n, bits, words, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(CCI_EHIP, "index-bits launch failed: %s", hipGetErrorString(e));
  return ok();
}

cci_status cci_spmm_bits(const void* X, cci_dtype x_t, int64_t N, int64_t C, const void* vals, cci_dtype val_t,
                         const void* idx, int32_t idx_bits, int64_t O, int32_t G, int32_t K, const cci_epilogue* ep,
                         void* Y, cci_dtype y_t, void* stream) {
  if (cci_status s = check_groups(O, C, G, K)) return s;
  if (cci_status s = check_types(x_t, val_t, y_t)) return s;
  if (N < 0) return fail(CCI_EINVAL, "N=%lld < 0", (long long)N);
  if (idx_bits < cci_index_width(G) || idx_bits > 8)
    return fail(CCI_EINVAL, "idx_bits=%d outside [%d, 8] for G=%d", idx_bits, cci_index_width(G), G);
  if (x_t != CCI_BF16) return fail(CCI_EUNSUPPORTED, "the bit-index product takes bf16 X and values");
  if (!cci::spmm_bits_supports(N, C, O, G, K))
    return fail(CCI_EUNSUPPORTED, "the bit-index product is for N <= 64 rows, C %% 32 == 0 and O %% 4 == 0");
  const float* scale = ep ? ep->scale : nullptr;
  const float* bias = ep ? ep->bias : nullptr;
  const void* residual = ep ? ep->residual : nullptr;
  if ((scale && !aligned16(scale)) || (bias && !aligned16(bias)) || (residual && !aligned16(residual)))
    return fail(CCI_EALIGN, "epilogue pointer not 16-byte aligned");
  if (N == 0) return ok();
  if (!X || !vals || !idx || !Y) return fail(CCI_EINVAL, "null pointer");
  if (!aligned16(X) || !aligned16(vals) || !aligned16(idx) || !aligned16(Y))
    return fail(CCI_EALIGN, "pointer not 16-byte aligned");
  hipError_t e = cci::launch_spmm_bits(X, N, C, vals, idx, idx_bits, O, G, K, scale, bias, residual, ep ? ep->relu : 0,
                                       Y, to_dt(y_t), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(CCI_EHIP, "bit-index product launch failed: %s", hipGetErrorString(e));
  return ok();
}

cci_status cci_maxpool2d_nhwc(const void* X, cci_dtype t, int64_t B, int64_t H, int64_t W,
                              int64_t C, int32_t k, int32_t s, int32_t p, void* Y, void* stream) {
  if (!dtype_ok(t)) return fail(CCI_EINVAL, "unknown dtype code");
  if (B < 0 || H < 1 || W < 1 || C < 1 || k < 1 || s < 1 || p < 0 || 2 * p > k ||
      H + 2 * p < k || W + 2 * p < k)
    return fail(CCI_EINVAL, "bad pooling geometry");
  if (!fits_nhwc(B, H, W, C, int64_t(1) << 40)) return fail(CCI_EINVAL, "tensor too large");
  if (B == 0) return ok();
  if (!X || !Y) return fail(CCI_EINVAL, "null pointer");
  if (!aligned16(X) || !aligned16(Y)) return fail(CCI_EALIGN, "pointer not 16-byte aligned");
  hipError_t e = cci::launch_maxpool(X, to_dt(t), B, H, W, C, k, s, p, Y,
                                     static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(CCI_EHIP, "maxpool launch failed: %s", hipGetErrorString(e));
  return ok();
}

cci_status cci_global_avgpool_nhwc(const void* X, cci_dtype x_t, int64_t B, int64_t H, int64_t W,
                                   int64_t C, void* Y, cci_dtype y_t, void* stream) {
  if (!dtype_ok(x_t) || !dtype_ok(y_t)) return fail(CCI_EINVAL, "unknown dtype code");
  if (B < 0 || H < 1 || W < 1 || C < 1) return fail(CCI_EINVAL, "bad pooling geometry");
  if (!fits_nhwc(B, H, W, C, int64_t(1) << 40)) return fail(CCI_EINVAL, "tensor too large");
  if (B == 0) return ok();
  if (!X || !Y) return fail(CCI_EINVAL, "null pointer");
  if (!aligned16(X) || !aligned16(Y)) return fail(CCI_EALIGN, "pointer not 16-byte aligned");
  hipError_t e = cci::launch_avgpool(X, to_dt(x_t), B, H, W, C, Y, to_dt(y_t),
                                     static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(CCI_EHIP, "avgpool launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"
