// CCI-sparse products with a short reduction (C <= 256): the 1x1 layers of
// narrow networks (MobileNetV2's expanding and projecting convolutions,
// Sec. 6), small FC layers, and convolutions with few input channels (a
// CNN's first layer: Cin = 4, or Cin % 8 == 0) read through implicit im2col
// (Sec. 3.2's lowering, never materialised).
//
// The method is the one of the tile kernels (Alg. 1's row G g + idx[g][k][c]
// receives vals[g][k][c]; the expanded product runs on the bf16 matrix
// cores), with a split for reductions too short to fill a channel pipeline:
//
//   - a slice of up to TM output tiles (16 outputs each) belongs to one wave,
//     which expands the packed groups of its slice once, straight from HBM
//     into MFMA operand fragments held in registers for the wave's lifetime
//     (output 16 t + lane % 16, channels 32 s + 8 (lane / 16) .. +7);
//   - the wave then streams groups of P 16-pixel blocks through them: the
//     activations of the next group are loaded (16 bytes per lane, rows
//     zero-padded past C and N by the buffer's range check) while the MFMAs
//     and the fused epilogue of the current one run.  For a convolution the
//     8 columns of a lane are one tap's 8 channels (Cin % 8 == 0) or two
//     horizontally adjacent taps' 4 channels (Cin == 4, KW even), so they
//     are one 16-byte (or two 8-byte) reads of the NHWC input, zero outside
//     the image;
//   - the accumulators leave the matrix cores with 4 consecutive outputs of
//     one pixel per lane; scale / bias (staged in LDS), residual (requested
//     with the group's MFMAs) and ReLU are applied in fp32 and each lane
//     stores 8 (bf16) or 16 (fp32) bytes.
//
// The slices of one pixel group are consecutive waves, so with 1, 2 or 4
// slices they share a workgroup and the group's activations come from HBM
// once (with 3 slices a workgroup holds parts of two groups: about 1.5x);
// the packed weights are read once per wave and every output is written
// once.  The layers this serves are bound by HBM bandwidth: their MFMA work
// is small next to their bytes.
#include "cci_device.hpp"
#include "cci_launch.hpp"

namespace cci {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kMaxC = 256;                // reduction length covered (8 k-steps of 32)
constexpr int kSliceOut = 80;             // outputs of the largest slice (TM <= 5)
constexpr int kWavesTarget = 3072;        // resident waves if the runtime cannot say
constexpr uint32_t kOOB = 0x80000000u;    // buffer offset that reads as zero / drops a store
constexpr int kRsrcWord3 = 0x00020000;    // raw buffer descriptor word 3 (gfx9 family)

struct NParams {
  const uint16_t* X;
  const uint16_t* vals;
  const uint8_t* idx;
  const float* scale;
  const float* bias;
  const void* residual;
  void* Y;
  uint32_t x_bytes, y_bytes;
  int32_t N, C, O, G, K, relu;
  int32_t H, W, Cin, KW, sh, sw, ph, pw, Ho, Wo;  // convolutions (implicit im2col)
  int32_t tpw;      // output tiles per slice
  int32_t nslices;  // slices covering the O / 16 (rounded up) output tiles
  int32_t npg;      // pixel groups of 16 P pixels
  int32_t wps;      // waves per slice (set at launch)
};

// Per k-step count S (= ceil(C / 32)): P 16-pixel blocks per step, at most TM
// output tiles per slice.  Registers: weights 4 TM S, accumulators 4 TM P,
// activations 2 x 4 P S (current and next group).
template <int S>
struct Shape {
  static constexpr int P = S == 1 ? 4 : (S == 2 ? 2 : 1);
  static constexpr int TM = S == 1 ? 4 : (S <= 3 ? 5 : (S == 4 ? 4 : (S <= 6 ? 3 : 2)));
  static_assert(16 * TM <= kSliceOut, "slice staging");
};

__device__ __forceinline__ float relu_f(float y) { return y > 0.0f ? y : (y != y ? y : 0.0f); }

// CM: 0 rows of X are the GEMM rows (FC, 1x1 stride-1 unpadded conv);
// 4 a convolution over 4 input channels; 8 a convolution over Cin % 8 == 0.
// RES: a residual is added (its reads are issued with the group's MFMAs).
template <typename YT, int S, int CM, bool RES>
__device__ __forceinline__ void narrow_body(const NParams& p, float* sb) {
  constexpr int P = Shape<S>::P, TM = Shape<S>::TM;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int gw = static_cast<int>(blockIdx.x) * (kThreads / 64) + w;
  if (gw >= p.nslices * p.wps) return;  // whole wave: no barriers below
  const int slice = gw % p.nslices;
  const int wv = gw / p.nslices;
  const int t0 = slice * p.tpw;                           // first output tile of the slice
  const int tw = min(p.tpw, (p.O + 15) / 16 - t0);        // tiles of this slice
  const int ol = lane & 15, kq = lane >> 4;

  // ---- pixel groups: the first group's activations are loaded before the
  // weights are expanded, so the two latencies overlap ----------------------
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.X), (short)0, static_cast<int>(p.x_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t yr =
      __builtin_amdgcn_make_buffer_rsrc(p.Y, (short)0, static_cast<int>(p.y_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(p.residual), (short)0, p.residual ? static_cast<int>(p.y_bytes) : 0, kRsrcWord3);
  const uint32_t N = static_cast<uint32_t>(p.N), C = static_cast<uint32_t>(p.C), O = static_cast<uint32_t>(p.O);
  // B fragment of block b, k-step s: pixel 16 b + ol of the group, columns
  // 32 s + 8 kq .. +7 (zero past C or N, and outside the image)
  int tkh[S], tkw[S], tci[S];  // conv: tap row, tap column, channel of the lane's columns
  bool sok[S];
#pragma unroll
  for (int s = 0; s < S; ++s) {
    const int c = 32 * s + 8 * kq;
    sok[s] = c < p.C;
    if constexpr (CM != 0) {
      const int t = c / p.Cin;
      tci[s] = c - t * p.Cin;
      tkh[s] = t / p.KW;
      tkw[s] = t - tkh[s] * p.KW;
    }
  }
  auto load_group = [&](int pg, bf16x8_t (&xf)[P][S]) {
#pragma unroll
    for (int b = 0; b < P; ++b) {
      const uint32_t n = static_cast<uint32_t>(pg) * (16u * P) + 16u * b + static_cast<uint32_t>(ol);
      if constexpr (CM == 0) {
#pragma unroll
        for (int s = 0; s < S; ++s) {
          const uint32_t c = 32u * s + 8u * static_cast<uint32_t>(kq);
          const uint32_t off = (n < N && c < C) ? (n * C + c) * 2u : kOOB;
          xf[b][s] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
        }
      } else {
        // output pixel n = (image, oh, ow) -> top-left input position
        const uint32_t hw = static_cast<uint32_t>(p.Ho * p.Wo);
        const uint32_t img = n / hw;
        const uint32_t rem = n - img * hw;
        const uint32_t oh = rem / static_cast<uint32_t>(p.Wo);
        const uint32_t ow = rem - oh * static_cast<uint32_t>(p.Wo);
        const int ih0 = static_cast<int>(oh) * p.sh - p.ph, iw0 = static_cast<int>(ow) * p.sw - p.pw;
        const bool nok = n < N;
#pragma unroll
        for (int s = 0; s < S; ++s) {
          const int ih = ih0 + tkh[s], iw = iw0 + tkw[s];
          const bool rok = nok && sok[s] && static_cast<uint32_t>(ih) < static_cast<uint32_t>(p.H);
          const uint32_t pos = (img * static_cast<uint32_t>(p.H) + static_cast<uint32_t>(ih)) *
                                   static_cast<uint32_t>(p.W) + static_cast<uint32_t>(iw);
          if constexpr (CM == 8) {
            const bool ok = rok && static_cast<uint32_t>(iw) < static_cast<uint32_t>(p.W);
            const uint32_t off = ok ? (pos * static_cast<uint32_t>(p.Cin) + static_cast<uint32_t>(tci[s])) * 2u : kOOB;
            xf[b][s] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
          } else {  // taps (kh, kw) and (kh, kw + 1), 4 channels (8 bytes) each
            const bool ok0 = rok && static_cast<uint32_t>(iw) < static_cast<uint32_t>(p.W);
            const bool ok1 = rok && static_cast<uint32_t>(iw + 1) < static_cast<uint32_t>(p.W);
            const uint32_t off0 = ok0 ? pos * 8u : kOOB;
            const uint32_t off1 = ok1 ? pos * 8u + 8u : kOOB;
            const u32x2_t lo = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(xr, off0, 0, 0));
            const u32x2_t hi = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(xr, off1, 0, 0));
            xf[b][s] = __builtin_bit_cast(bf16x8_t, u32x4_t{lo[0], lo[1], hi[0], hi[1]});
          }
        }
      }
    }
  };

  int pg = wv;
  if (pg >= p.npg) return;
  bf16x8_t xc[P][S], xn[P][S];
  load_group(pg, xc);

  // ---- scale / bias of the slice's outputs, staged in this wave's LDS ------
  float* ss = sb + w * 2 * kSliceOut;
  for (int i = lane; i < 16 * tw; i += 64) {
    const int o = 16 * t0 + i;
    ss[i] = (p.scale && o < p.O) ? p.scale[o] : 1.0f;
    ss[kSliceOut + i] = (p.bias && o < p.O) ? p.bias[o] : 0.0f;
  }

  // ---- expanded weights: fragment (t, s) of output 16 (t0 + t) + ol --------
  // Each (group, channel) keeps K entries with distinct rows, so at most one
  // slot matches a row; slots and channels past the slice or C stay zero.
  // The loads of up to 8 fragments are issued together, slot by slot
  // (ceil(TM / TC) K rounds of memory latency rather than TM S K, with a
  // bounded number of registers in flight).
  constexpr int TC = 8 / S >= TM ? TM : (8 / S < 1 ? 1 : 8 / S);
  int64_t ebase[TM];
  uint32_t rrow[TM];
  bool tok[TM];
#pragma unroll
  for (int t = 0; t < TM; ++t) {
    const int o = 16 * (t0 + t) + ol;
    tok[t] = t < tw && o < p.O;
    const int g = tok[t] ? o / p.G : 0;
    rrow[t] = static_cast<uint32_t>(tok[t] ? o - g * p.G : 0);
    ebase[t] = static_cast<int64_t>(g) * p.K * p.C;
  }
  u32x4_t wacc[TM][S];
#pragma unroll
  for (int t = 0; t < TM; ++t)
#pragma unroll
    for (int s = 0; s < S; ++s) wacc[t][s] = u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
  for (int tc = 0; tc < TM; tc += TC) {
    for (int kk = 0; kk < p.K; ++kk) {
      u32x4_t v[TC][S];
      u32x2_t ix[TC][S];
#pragma unroll
      for (int u = 0; u < TC; ++u)
#pragma unroll
        for (int s = 0; s < S; ++s) {
          const int t = tc + u < TM ? tc + u : TM - 1;
          const int c = 32 * s + 8 * kq;
          const bool ok = tc + u < TM && tok[t] && c < p.C;
          const int64_t e = ebase[t] + static_cast<int64_t>(kk) * p.C + c;
          v[u][s] = ok ? *reinterpret_cast<const u32x4_t*>(p.vals + e) : u32x4_t{0u, 0u, 0u, 0u};
          ix[u][s] = ok ? *reinterpret_cast<const u32x2_t*>(p.idx + e) : u32x2_t{0xffffffffu, 0xffffffffu};
        }
#pragma unroll
      for (int u = 0; u < TC; ++u) {
        if (tc + u >= TM) continue;
#pragma unroll
        for (int s = 0; s < S; ++s)
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const uint32_t row = (ix[u][s][j >> 2] >> (8 * (j & 3))) & 0xffu;
            const uint32_t half = (j & 1) ? 0xffff0000u : 0x0000ffffu;
            wacc[tc + u][s][j >> 1] |= row == rrow[tc + u] ? (v[u][s][j >> 1] & half) : 0u;
          }
      }
    }
  }
  bf16x8_t wf[TM][S];
#pragma unroll
  for (int t = 0; t < TM; ++t)
#pragma unroll
    for (int s = 0; s < S; ++s) wf[t][s] = __builtin_bit_cast(bf16x8_t, wacc[t][s]);

  constexpr uint32_t ysz = sizeof(YT);
  using RV = std::conditional_t<ysz == 2, u32x2_t, f32x4_t>;  // a lane's 4 residual values
  // Y / residual offset of (block b, tile t) of group g
  auto yoff = [&](int g, int b, int t) {
    const uint32_t n = static_cast<uint32_t>(g) * (16u * P) + 16u * b + static_cast<uint32_t>(ol);
    const uint32_t o = static_cast<uint32_t>(16 * (t0 + t) + 4 * kq);
    return (n < N && o < O) ? (n * O + o) * ysz : kOOB;
  };
  while (true) {
    const int pn = pg + p.wps;
    load_group(pn, xn);  // past the last group: every offset is out of range
    RV res[P][TM];
    if constexpr (RES) {  // this group's residual, requested before its MFMAs
#pragma unroll
      for (int b = 0; b < P; ++b)
#pragma unroll
        for (int t = 0; t < TM; ++t) {
          if (t >= tw) continue;
          if constexpr (ysz == 2)
            res[b][t] = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(rr, yoff(pg, b, t), 0, 0));
          else
            res[b][t] = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rr, yoff(pg, b, t), 0, 0));
        }
    }
    f32x4_t acc[P][TM];
#pragma unroll
    for (int b = 0; b < P; ++b)
#pragma unroll
      for (int t = 0; t < TM; ++t) {
        acc[b][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        if (t < tw) {
#pragma unroll
          for (int s = 0; s < S; ++s)
            acc[b][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[t][s], xc[b][s], acc[b][t], 0, 0, 0);
        }
      }
    // epilogue: lane holds outputs 16 (t0 + t) + 4 kq .. +3 of pixel 16 b + ol
#pragma unroll
    for (int b = 0; b < P; ++b) {
      u32x2_t pk[TM];  // bf16 output: the rounded values of each tile
#pragma unroll
      for (int t = 0; t < TM; ++t) {
        if (t >= tw) continue;
        const int oi = 16 * t + 4 * kq;  // within the slice
        const uint32_t off = yoff(pg, b, t);
        const f32x4_t sc = *reinterpret_cast<const f32x4_t*>(ss + oi);
        const f32x4_t bi = *reinterpret_cast<const f32x4_t*>(ss + kSliceOut + oi);
        f32x4_t y = acc[b][t] * sc + bi;
        if constexpr (RES) {
          if constexpr (ysz == 2) {
            const u32x2_t q = res[b][t];
            y[0] += __uint_as_float(q[0] << 16);
            y[1] += __uint_as_float(q[0] & 0xffff0000u);
            y[2] += __uint_as_float(q[1] << 16);
            y[3] += __uint_as_float(q[1] & 0xffff0000u);
          } else {
            y += res[b][t];
          }
        }
        if (p.relu) {
#pragma unroll
          for (int e = 0; e < 4; ++e) y[e] = relu_f(y[e]);
        }
        if constexpr (ysz == 2) {
          // v_cvt_pk_bf16_f32: round to nearest even
          pk[t] = u32x2_t{__builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y[0], y[1]}), bf16x2_t)),
                          __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y[2], y[3]}), bf16x2_t))};
        } else {
          __builtin_amdgcn_raw_buffer_store_b128(
              __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(yr, 0, 0, 0)), y), yr, off, 0, 0);
        }
      }
      if constexpr (ysz == 2 && S < 4) {
#pragma unroll
        for (int t = 0; t < TM; ++t) {
          if (t >= tw) continue;
          __builtin_amdgcn_raw_buffer_store_b64(
              __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b64(yr, 0, 0, 0)), pk[t]), yr,
              yoff(pg, b, t), 0, 0);
        }
      } else if constexpr (ysz == 2) {
        // With four or more k-steps (the 7x7 stem) tiles t, t + 1 both inside
        // O leave as 16-byte stores (8-byte ones cost about 1.6x as much store
        // time; with fewer k-steps the extra exchange costs more than it
        // saves): lanes l and l ^ 16 (q = kq and its partner) swap halves so
        // that the even one holds outputs 8 (kq / 2) .. +7 of tile t and the
        // odd one those of tile t + 1 (ds_swizzle in bit mode, xor 16 within
        // each 32-lane half).  A last unpaired tile keeps its 8-byte store.
        const bool odd = kq & 1;
#pragma unroll
        for (int t = 0; t < TM; t += 2) {
          if (t >= tw) continue;
          if (t + 1 < tw && t + 1 < TM && 16 * (t0 + t + 2) <= O) {
            const u32x2_t snd = odd ? pk[t] : pk[t + 1 < TM ? t + 1 : t];
            const uint32_t r0 = static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(static_cast<int>(snd[0]), 0x401F));
            const uint32_t r1 = static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(static_cast<int>(snd[1]), 0x401F));
            const u32x2_t mine = odd ? pk[t + 1 < TM ? t + 1 : t] : pk[t];
            const u32x4_t v = odd ? u32x4_t{r0, r1, mine[0], mine[1]} : u32x4_t{mine[0], mine[1], r0, r1};
            const uint32_t n = static_cast<uint32_t>(pg) * (16u * P) + 16u * b + static_cast<uint32_t>(ol);
            const uint32_t o = static_cast<uint32_t>(16 * (t0 + t) + (odd ? 16 : 0) + 8 * (kq >> 1));
            const uint32_t off = n < N ? (n * O + o) * ysz : kOOB;
            __builtin_amdgcn_raw_buffer_store_b128(
                __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(yr, 0, 0, 0)), v), yr, off, 0, 0);
          } else {
            __builtin_amdgcn_raw_buffer_store_b64(
                __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b64(yr, 0, 0, 0)), pk[t]), yr, yoff(pg, b, t),
                0, 0);
            if (t + 1 < tw && t + 1 < TM)
              __builtin_amdgcn_raw_buffer_store_b64(
                  __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b64(yr, 0, 0, 0)), pk[t + 1 < TM ? t + 1 : t]),
                  yr, yoff(pg, b, t + 1 < TM ? t + 1 : t), 0, 0);
          }
        }
      }
    }
    if (pn >= p.npg) break;
    pg = pn;
#pragma unroll
    for (int b = 0; b < P; ++b)
#pragma unroll
      for (int s = 0; s < S; ++s) xc[b][s] = xn[b][s];
  }
}

// (The body is a device function: with it inside the kernel template, the
// host pass of this compiler emitted no launch stubs for the kernels.)
template <typename YT, int S, int CM, bool RES>
__global__ __launch_bounds__(kThreads) void narrow_kernel(NParams p) {
  __shared__ __attribute__((aligned(16))) float sb[(kThreads / 64) * 2 * kSliceOut];
  narrow_body<YT, S, CM, RES>(p, sb);
}

// Waves of narrow_kernel<YT, S> that fit on the current device at once
// (queried once per device).
template <typename YT, int S, int CM, bool RES>
int64_t resident_waves() {
  static std::atomic<int64_t> cached[kMaxDevices];
  const int dev = current_device();
  if (dev >= 0) {
    const int64_t w = cached[dev].load(std::memory_order_acquire);
    if (w > 0) return w;
  }
  int cus = 0, blocks = 0;
  int64_t waves = static_cast<int64_t>(kWavesTarget);
  if (dev >= 0 && hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, reinterpret_cast<const void*>(&narrow_kernel<YT, S, CM, RES>),
                                                   kThreads, 0) == hipSuccess &&
      cus >= 1 && blocks >= 1) {
    waves = static_cast<int64_t>(cus) * blocks * (kThreads / 64);
    cached[dev].store(waves, std::memory_order_release);
  }
  return waves;
}

// One wave per (slice, pixel group) when that fits on the device at once;
// otherwise as many waves as are resident, each streaming several groups.
template <typename YT, int S, int CM, bool RES>
hipError_t launch_k(NParams p, hipStream_t s) {
  const int64_t per_slice = std::max<int64_t>(1, resident_waves<YT, S, CM, RES>() / p.nslices);
  p.wps = static_cast<int32_t>(std::min<int64_t>(p.npg, per_slice));
  const int64_t waves = static_cast<int64_t>(p.nslices) * p.wps;
  const uint32_t grid = static_cast<uint32_t>((waves + 3) / 4);
  hipLaunchKernelGGL((narrow_kernel<YT, S, CM, RES>), dim3(grid), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

template <typename YT, int CM>
hipError_t launch_s(const NParams& p, int S, hipStream_t s) {
  switch (S) {
    case 1: return p.residual ? launch_k<YT, 1, CM, true>(p, s) : launch_k<YT, 1, CM, false>(p, s);
    case 2: return p.residual ? launch_k<YT, 2, CM, true>(p, s) : launch_k<YT, 2, CM, false>(p, s);
    case 3: return p.residual ? launch_k<YT, 3, CM, true>(p, s) : launch_k<YT, 3, CM, false>(p, s);
    case 4: return p.residual ? launch_k<YT, 4, CM, true>(p, s) : launch_k<YT, 4, CM, false>(p, s);
    case 5: return p.residual ? launch_k<YT, 5, CM, true>(p, s) : launch_k<YT, 5, CM, false>(p, s);
    case 6: return p.residual ? launch_k<YT, 6, CM, true>(p, s) : launch_k<YT, 6, CM, false>(p, s);
    case 7: return p.residual ? launch_k<YT, 7, CM, true>(p, s) : launch_k<YT, 7, CM, false>(p, s);
    case 8: return p.residual ? launch_k<YT, 8, CM, true>(p, s) : launch_k<YT, 8, CM, false>(p, s);
    default: return hipErrorInvalidConfiguration;
  }
}

// 0: rows; 4 / 8: implicit-im2col convolution over 4 / a multiple of 8 input channels
int conv_mode(const ProductArgs& a) {
  if (!a.conv) return 0;
  const ConvGeom& g = a.geom;
  if (g.KH == 1 && g.KW == 1 && g.sh == 1 && g.sw == 1 && g.ph == 0 && g.pw == 0) return 0;
  if (g.Cin % 8 == 0) return 8;
  if (g.Cin == 4 && g.KW % 2 == 0) return 4;
  return -1;
}

int max_tiles(int S) {
  switch (S) {
    case 1: return Shape<1>::TM;
    case 2: return Shape<2>::TM;
    case 3: return Shape<3>::TM;
    case 4: return Shape<4>::TM;
    case 5: return Shape<5>::TM;
    case 6: return Shape<6>::TM;
    case 7: return Shape<7>::TM;
    default: return Shape<8>::TM;
  }
}
int pixel_blocks(int S) { return S == 1 ? Shape<1>::P : (S == 2 ? Shape<2>::P : 1); }

}  // namespace

bool narrow_supports(const ProductArgs& a) {
  if (a.x_t != DType::BF16 || a.val_t != DType::BF16) return false;
  if (conv_mode(a) < 0) return false;
  if (a.G < 1 || a.G > 256 || a.K < 1 || a.K > a.G || a.O % a.G != 0) return false;
  if (a.C < 1 || a.C > kMaxC || a.C % 8 != 0 || a.O % 4 != 0 || a.N < 1) return false;
  const auto al = [](const void* q, uintptr_t m) { return (reinterpret_cast<uintptr_t>(q) & (m - 1)) == 0; };
  const uintptr_t ya = a.y_t == DType::F32 ? 16 : 8;
  if (!al(a.X, 16) || !al(a.vals, 16) || !al(a.idx, 8) || !al(a.Y, ya)) return false;
  if ((a.scale && !al(a.scale, 4)) || (a.bias && !al(a.bias, 4)) || (a.residual && !al(a.residual, ya)))
    return false;
  // every buffer offset is 32-bit and stays below the out-of-range marker
  const int64_t lim = static_cast<int64_t>(kOOB);
  const int64_t x_elems = a.conv ? a.B * static_cast<int64_t>(a.geom.H) * a.geom.W * a.geom.Cin : a.N * a.C;
  if (x_elems * 2 >= lim || a.N * a.C * 2 >= lim || a.N * a.O * (a.y_t == DType::F32 ? 4 : 2) >= lim) return false;
  return true;
}

hipError_t launch_narrow(const ProductArgs& a, hipStream_t s) {
  if (!narrow_supports(a)) return hipErrorInvalidConfiguration;
  NParams p{};
  p.X = static_cast<const uint16_t*>(a.X);
  p.vals = static_cast<const uint16_t*>(a.vals);
  p.idx = a.idx;
  p.scale = a.scale;
  p.bias = a.bias;
  p.residual = a.residual;
  p.Y = a.Y;
  const int cm = conv_mode(a);
  p.x_bytes = static_cast<uint32_t>(
      (cm == 0 ? a.N * a.C : a.B * static_cast<int64_t>(a.geom.H) * a.geom.W * a.geom.Cin) * 2);
  if (cm != 0) {
    const ConvGeom& g = a.geom;
    p.H = g.H;
    p.W = g.W;
    p.Cin = g.Cin;
    p.KW = g.KW;
    p.sh = g.sh;
    p.sw = g.sw;
    p.ph = g.ph;
    p.pw = g.pw;
    p.Ho = g.Ho;
    p.Wo = g.Wo;
  }
  p.y_bytes = static_cast<uint32_t>(a.N * a.O * (a.y_t == DType::F32 ? 4 : 2));
  p.N = static_cast<int32_t>(a.N);
  p.C = static_cast<int32_t>(a.C);
  p.O = static_cast<int32_t>(a.O);
  p.G = a.G;
  p.K = a.K;
  p.relu = a.relu;
  const int S = static_cast<int>((a.C + 31) / 32);
  const int tiles = static_cast<int>((a.O + 15) / 16);
  const int tm = max_tiles(S);
  p.nslices = (tiles + tm - 1) / tm;
  p.tpw = (tiles + p.nslices - 1) / p.nslices;  // balanced slices
  p.nslices = (tiles + p.tpw - 1) / p.tpw;
  const int64_t gp = 16 * static_cast<int64_t>(pixel_blocks(S));
  p.npg = static_cast<int32_t>((a.N + gp - 1) / gp);
  if (a.y_t == DType::F32)
    return cm == 0 ? launch_s<float, 0>(p, S, s) : cm == 4 ? launch_s<float, 4>(p, S, s) : launch_s<float, 8>(p, S, s);
  return cm == 0 ? launch_s<uint16_t, 0>(p, S, s)
                 : cm == 4 ? launch_s<uint16_t, 4>(p, S, s) : launch_s<uint16_t, 8>(p, S, s);
}

}  // namespace cci
