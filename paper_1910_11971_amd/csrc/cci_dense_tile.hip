// CCI-sparse product on the matrix cores (implicit GEMM).
//
// The packed groups of an output block are expanded into a dense bf16 weight
// tile in LDS -- a zero fill, then every kept weight is written to row
// G*g + idx of its column, the target row of Alg. 1 (Sec. 3.2) -- and the
// tile is multiplied on v_mfma_f32_16x16x32_bf16 against activations that
// are also staged in LDS.
//
// Why expand instead of multiplying only kept weights: CCI keeps K of G
// entries along the *output* dimension for each reduction index.  Dense MFMA
// cannot skip those zeros and gfx950's 2:4 sparse MFMA sparsifies the
// *reduction* dimension, so neither fits.  The vector ALUs can do only the
// kept work, but at 78.6 fp32 TFLOP/s (no packed fp32) against 2516.6 dense
// bf16 TFLOP/s on the matrix cores, so for K/G > 1/32 the expanded tile is
// faster.  The packed form still cuts the weight bytes read by G/K x 2/3.
//
// Work decomposition.  A workgroup (4 waves) owns WO 64-output blocks and
// a set of output pixels; the waves are arranged WO (output blocks) x WP
// (pixel groups).  Each wave accumulates up to MT 16-pixel tiles x 64
// outputs in registers.  The reduction runs over channel chunks of CINB
// channels x all KH*KW taps:
//   - the activation patch of the chunk (every input pixel any tap of the
//     workgroup's outputs touches, CINB channels) is DMA'd from HBM straight
//     into LDS with buffer_load...lds; out-of-image pixels read as zero
//     because their buffer offsets are out of range (this *is* the conv
//     padding); 16-byte chunks are XOR-swizzled per pixel so the MFMA operand
//     reads are bank-conflict free;
//   - the expanded weight tile of the chunk is built in LDS;
//   - with two buffers, chunk j+1 is in flight while chunk j is multiplied.
// Patch geometry: "rect" mode (k x k convolutions) stages the input rows and
// columns under a band of RH output rows; "rows" mode (FC and 1x1
// convolutions, any stride) stages one input pixel per output pixel.
// Workgroup ids are mapped so that the output blocks of one pixel range sit
// on the same XCD (they read the same activations through its L2).
#include "cci_launch.hpp"

namespace cci {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kBN = 64;          // outputs per wave
constexpr int kKS = 32;          // reduction columns per MFMA k-step
constexpr int kMT = 8;           // max 16-pixel tiles per wave
constexpr int kBPad = 8;         // weight-tile row padding (bf16 elements)
constexpr int kXcds = 8;
constexpr int kLdsMax = 160 * 1024;
constexpr uint32_t kOOB = 0x80000000u;  // buffer offset that reads as zero

struct Plan {
  int32_t rect;        // 1: k x k patch; 0: one patch pixel per output pixel
  int32_t WO, WP;      // wave arrangement (WO * WP == 4)
  int32_t nob;         // output super-blocks of WO*64 outputs
  int64_t parts;       // pixel partitions (multiple of kXcds)
  int64_t part_len;    // rows mode: output pixels per partition; rect: output rows (RH)
  int32_t row_parts;   // rect: partitions per image
  int32_t cinb;        // channels per chunk (power of two, multiple of 32)
  int32_t nchunks;
  int32_t taps;
  int32_t patch_cols;  // rect: staged input columns
  int32_t patch_pix;   // staged pixels per chunk
  int32_t b_pitch;     // bf16 elements per weight-tile row
  int32_t b_bytes;     // bytes of one weight tile (WO*64 rows)
  int32_t buf_bytes;   // weight tile + patch
  int32_t nbuf;        // 1 or 2
};

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t v) { return __builtin_bit_cast(bf16x8_t, v); }

// 16-byte chunk c of patch pixel q lives in slot q*cpp + swz(q, c).
__device__ __forceinline__ int swz(int q, int c, int cpp) {
  return cpp >= 8 ? (c ^ (q & 7)) : (c ^ ((q >> 1) & 3));
}

template <typename YT>
__global__ __launch_bounds__(kThreads) void dense_tile_kernel(
    const uint16_t* __restrict__ X, uint32_t x_bytes, int64_t N, int64_t C, ConvGeom g, int32_t Bimg,
    const uint16_t* __restrict__ vals, const uint8_t* __restrict__ idx, int64_t O, int32_t G,
    int32_t K, Epilogue<YT> ep, YT* __restrict__ Y, Plan pl) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];

  // ---- workgroup -> (pixel partition, output super-block), XCD-aware ----
  const int64_t id = blockIdx.x;
  const int64_t j = id / kXcds;
  const int32_t ob = static_cast<int32_t>(j % pl.nob);
  const int64_t part = (j / pl.nob) * kXcds + id % kXcds;
  if (part >= pl.parts) return;

  // Pixel set of this workgroup.
  int32_t npix;            // output pixels owned
  int64_t P0 = 0;          // rows mode: first output pixel
  int32_t b_img = 0, oh0 = 0;  // rect mode
  if (pl.rect) {
    b_img = static_cast<int32_t>(part / pl.row_parts);
    if (b_img >= Bimg) return;
    oh0 = static_cast<int32_t>((part % pl.row_parts) * pl.part_len);
    const int32_t rh = g.Ho - oh0 < pl.part_len ? g.Ho - oh0 : static_cast<int32_t>(pl.part_len);
    npix = rh * g.Wo;
  } else {
    P0 = part * pl.part_len;
    if (P0 >= N) return;
    npix = static_cast<int32_t>(N - P0 < pl.part_len ? N - P0 : pl.part_len);
  }
  const int32_t ntiles = (npix + 15) / 16;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wo = wave % pl.WO;
  const int wp = wave / pl.WO;
  const int lrow = lane & 15;
  const int lk = lane >> 4;
  const int cpp = pl.cinb / 8;                   // 16-byte chunks per patch pixel
  const int64_t o_wave = (static_cast<int64_t>(ob) * pl.WO + wo) * kBN;
  const int32_t my_tiles = ntiles > wp ? (ntiles - wp + pl.WP - 1) / pl.WP : 0;  // tiles wp, wp+WP, ...

  __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(X), (short)0,
                                                                static_cast<int>(x_bytes), 0x00020000);

  // Per-lane geometry of each owned tile: patch pixel of tap (0,0).
  int32_t qbase[kMT];
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) {
    int32_t p = (wp + mt * pl.WP) * 16 + lrow;
    p = p < npix ? p : 0;                        // idle lanes read pixel 0 (never stored)
    if (pl.rect) {
      const int32_t r = p / g.Wo;
      const int32_t ow = p - r * g.Wo;
      qbase[mt] = r * g.sh * pl.patch_cols + ow * g.sw;
    } else {
      qbase[mt] = p;
    }
  }

  // Input geometry of the staged patch.
  const int32_t ih_base = oh0 * g.sh - g.ph;     // rect: first staged input row
  const int32_t iw_base = -g.pw;                 // rect: first staged input column

  // Issue the DMA of chunk `ch`'s activation patch into buffer `buf`.
  auto issue_patch = [&](int ch, int buf) {
    uint8_t* pbase = lds + buf * pl.buf_bytes + pl.b_bytes;
    const int32_t slots = pl.patch_pix * cpp;
    const int32_t ci0 = ch * pl.cinb;
    for (int32_t s0 = wave * 64; s0 < slots; s0 += kWaves * 64) {
      const int32_t s = s0 + lane;
      const int32_t q = s / cpp;
      const int32_t phys = s - q * cpp;
      const int32_t c = swz(q, phys, cpp);       // XOR swizzle is its own inverse
      uint32_t off = kOOB;
      if (s < slots) {
        if (pl.rect) {
          const int32_t pr = q / pl.patch_cols;
          const int32_t pc = q - pr * pl.patch_cols;
          const int32_t ih = ih_base + pr;
          const int32_t iw = iw_base + pc;
          if (ih >= 0 && ih < g.H && iw >= 0 && iw < g.W)
            off = static_cast<uint32_t>(((static_cast<int64_t>(b_img) * g.H + ih) * g.W + iw) * g.Cin +
                                        ci0 + 8 * c) * 2u;
        } else if (q < npix) {
          const int64_t n = P0 + q;
          int64_t pix = n;                       // FC / 1x1 stride 1: row n
          if (g.sh != 1 || g.sw != 1) {          // 1x1 strided: gather input pixel
            const int64_t hw = static_cast<int64_t>(g.Ho) * g.Wo;
            const int64_t b = n / hw;
            const int64_t rem = n - b * hw;
            const int64_t oh = rem / g.Wo;
            const int64_t ow = rem - oh * g.Wo;
            pix = (b * g.H + oh * g.sh) * g.W + ow * g.sw;
          }
          off = static_cast<uint32_t>((pix * g.Cin + ci0 + 8 * c) * 2);
        }
      }
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t*)(pbase + s0 * 16), 16, off, 0, 0, 0);
    }
  };

  // Expand chunk `ch`'s packed weights into buffer `buf` (zero fill first).
  auto zero_weights = [&](int buf) {
    u32x4_t* b4 = reinterpret_cast<u32x4_t*>(lds + buf * pl.buf_bytes);
    const int n16 = pl.b_bytes / 16;
    for (int e = threadIdx.x; e < n16; e += kThreads) b4[e] = u32x4_t{0u, 0u, 0u, 0u};
  };
  auto scatter_weights = [&](int ch, int buf) {
    uint16_t* bs = reinterpret_cast<uint16_t*>(lds + buf * pl.buf_bytes);
    const int c8n = pl.cinb / 8;
    const int gpb = (pl.WO * kBN) / G;           // groups per super-block
    const int64_t g0 = static_cast<int64_t>(ob) * gpb;
    const int64_t ngroups = O / G;
    const int per_group = K * pl.taps * c8n;
    const int items = gpb * per_group;
    const int32_t ci0 = ch * pl.cinb;
    for (int it = threadIdx.x; it < items; it += kThreads) {
      const int gl = it / per_group;
      int rem = it - gl * per_group;
      const int k = rem / (pl.taps * c8n);
      rem -= k * (pl.taps * c8n);
      const int tap = rem / c8n;
      const int c8 = rem - tap * c8n;
      const int64_t gg = g0 + gl;
      if (gg >= ngroups) continue;
      const int64_t src = (gg * K + k) * C + static_cast<int64_t>(tap) * g.Cin + ci0 + 8 * c8;
      const u32x4_t v = *reinterpret_cast<const u32x4_t*>(vals + src);
      const uint2 ix = *reinterpret_cast<const uint2*>(idx + src);
      uint16_t* dst = bs + static_cast<int64_t>(gl) * G * pl.b_pitch + tap * pl.cinb + 8 * c8;
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        const uint32_t r = ((jj < 4 ? ix.x : ix.y) >> (8 * (jj & 3))) & 0xffu;
        const uint16_t w = static_cast<uint16_t>(v[jj >> 1] >> (16 * (jj & 1)));
        if (r < static_cast<uint32_t>(G)) dst[r * pl.b_pitch + jj] = w;
      }
    }
  };

  f32x4_t acc[kMT][4];
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
    for (int ot = 0; ot < 4; ++ot) acc[mt][ot] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

  // Multiply the chunk held in buffer `buf`.  Reduction steps of 32 columns
  // run tap-major; the operand fragments of step s+1 are read from LDS while
  // the MFMAs of step s issue (two register sets, statically alternated).
  struct Frags {
    bf16x8_t w[4];
    bf16x8_t x[kMT];
  };
  auto compute = [&](int buf) {
    const uint16_t* bs = reinterpret_cast<const uint16_t*>(lds + buf * pl.buf_bytes) +
                         static_cast<int64_t>(wo) * kBN * pl.b_pitch + lrow * pl.b_pitch + 8 * lk;
    const uint8_t* patch = lds + buf * pl.buf_bytes + pl.b_bytes;
    const int ksteps = pl.cinb / kKS;
    const int nsteps = pl.taps * ksteps;
    auto load = [&](int st, Frags& f) {
      const int tap = st / ksteps;
      const int kb = st - tap * ksteps;
      const int kh = tap / g.KW;
      const int kw = tap - kh * g.KW;
      const int32_t dq = pl.rect ? kh * pl.patch_cols + kw : 0;
      const int col = tap * pl.cinb + kb * kKS;
#pragma unroll
      for (int ot = 0; ot < 4; ++ot)
        f.w[ot] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(bs + ot * 16 * pl.b_pitch + col));
      const int c = kb * 4 + lk;
#pragma unroll
      for (int mt = 0; mt < kMT; ++mt) {
        // unconditional (idle tiles read a clamped, valid pixel) so the
        // compiler can count outstanding LDS reads exactly
        const int32_t q = qbase[mt] + dq;
        f.x[mt] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(patch + (q * cpp + swz(q, c, cpp)) * 16));
      }
    };
    auto mma = [&](const Frags& f) {
#pragma unroll
      for (int mt = 0; mt < kMT; ++mt) {
        if (mt < my_tiles) {
#pragma unroll
          for (int ot = 0; ot < 4; ++ot)
            acc[mt][ot] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.w[ot], f.x[mt], acc[mt][ot], 0, 0, 0);
        }
      }
    };
    // Loads past the last step re-read the last step (clamped) so that every
    // load is unconditional and the compiler can count outstanding reads.
    Frags f0, f1;
    load(0, f0);
    for (int st = 0; st < nsteps; st += 2) {
      load(st + 1 < nsteps ? st + 1 : nsteps - 1, f1);
      mma(f0);
      load(st + 2 < nsteps ? st + 2 : nsteps - 1, f0);
      if (st + 1 < nsteps) mma(f1);
    }
  };

  // ---- chunk pipeline -----------------------------------------------------
  issue_patch(0, 0);
  zero_weights(0);
  __syncthreads();
  scatter_weights(0, 0);
  __builtin_amdgcn_s_waitcnt(0);  // patch DMA of chunk 0 landed (vm and lgkm counters drained)
  __syncthreads();
  for (int ch = 0; ch < pl.nchunks; ++ch) {
    const int buf = pl.nbuf == 2 ? (ch & 1) : 0;
    const bool more = ch + 1 < pl.nchunks;
    if (pl.nbuf == 2) {
      if (more) {
        issue_patch(ch + 1, buf ^ 1);
        zero_weights(buf ^ 1);
      }
      compute(buf);
      if (more) {
        __syncthreads();                         // zero fill of the next tile complete
        scatter_weights(ch + 1, buf ^ 1);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
      }
    } else {
      compute(buf);
      if (more) {
        __syncthreads();                         // all waves done with the buffer
        issue_patch(ch + 1, 0);
        zero_weights(0);
        __syncthreads();
        scatter_weights(ch + 1, 0);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
      }
    }
  }

  // ---- fused epilogue: lane holds outputs o+4lk+[0..3] of one pixel ----
  const bool vec_ok = (O % 4) == 0;
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) {
    if (mt >= my_tiles) break;
    const int32_t p = (wp + mt * pl.WP) * 16 + lrow;
    if (p >= npix) continue;
    int64_t n;
    if (pl.rect) {
      const int32_t r = p / g.Wo;
      const int32_t ow = p - r * g.Wo;
      n = (static_cast<int64_t>(b_img) * g.Ho + oh0 + r) * g.Wo + ow;
    } else {
      n = P0 + p;
    }
#pragma unroll
    for (int ot = 0; ot < 4; ++ot) {
      const int64_t o = o_wave + ot * 16 + 4 * lk;
      if (o >= O) continue;
      const int64_t yo = n * O + o;
      if (vec_ok) {
        float y[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) y[jj] = apply_epilogue<YT>(acc[mt][ot][jj], o + jj, yo + jj, ep);
        if constexpr (sizeof(YT) == 2) {
          uint2 pk;
          pk.x = f32_to_bf16_rne(y[0]) | (static_cast<uint32_t>(f32_to_bf16_rne(y[1])) << 16);
          pk.y = f32_to_bf16_rne(y[2]) | (static_cast<uint32_t>(f32_to_bf16_rne(y[3])) << 16);
          *reinterpret_cast<uint2*>(Y + yo) = pk;
        } else {
          *reinterpret_cast<float4*>(Y + yo) = make_float4(y[0], y[1], y[2], y[3]);
        }
      } else {
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          if (o + jj < O) io<YT>::store(Y, yo + jj, apply_epilogue<YT>(acc[mt][ot][jj], o + jj, yo + jj, ep));
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Host-side planning.

bool is_rows_mode(const ProductArgs& a) {
  return !a.conv || (a.geom.KH == 1 && a.geom.KW == 1 && a.geom.ph == 0 && a.geom.pw == 0);
}

// Fill the LDS layout for a given chunk width; false if it does not fit.
bool layout(Plan& pl, int32_t cinb, int32_t Cin, int32_t nbuf) {
  pl.cinb = cinb;
  pl.nchunks = Cin / cinb;
  pl.b_pitch = pl.taps * cinb + kBPad;
  pl.b_bytes = pl.WO * kBN * pl.b_pitch * 2;
  // the DMA writes whole 64-slot (1 KiB) blocks: round the patch up so the
  // tail of its last block stays inside this buffer
  const int64_t patch_bytes = (static_cast<int64_t>(pl.patch_pix) * cinb * 2 + 1023) / 1024 * 1024;
  const int64_t buf = pl.b_bytes + patch_bytes;
  if (buf * nbuf > kLdsMax) return false;
  pl.buf_bytes = static_cast<int32_t>(buf);
  pl.nbuf = nbuf;
  return true;
}

// Choose the wave arrangement, pixel partition and channel chunk.  The cost
// model counts MFMA tile-steps on the busiest CU (one workgroup per CU at a
// time) plus a charge for re-reading activations once per output block.
bool make_plan(const ProductArgs& a, Plan& best) {
  const int32_t Cin = a.conv ? a.geom.Cin : static_cast<int32_t>(a.C);
  const bool rows = is_rows_mode(a);
  const int32_t taps = a.conv ? a.geom.KH * a.geom.KW : 1;
  double best_cost = 1e300;
  bool found = false;
  for (int WO = 1; WO <= 4; WO *= 2) {
    if (WO > 1 && (a.O + kBN - 1) / kBN < WO) break;
    const int WP = kWaves / WO;
    const int64_t max_pix = static_cast<int64_t>(WP) * kMT * 16;
    Plan pl{};
    pl.rect = rows ? 0 : 1;
    pl.WO = WO;
    pl.WP = WP;
    pl.taps = taps;
    pl.nob = static_cast<int32_t>((a.O + WO * kBN - 1) / (WO * kBN));
    // candidate partition sizes
    for (int64_t len = 1; len <= (rows ? max_pix / 16 : 64); ++len) {
      int64_t parts, pix_per_part;
      if (rows) {
        pix_per_part = len * 16;
        parts = (a.N + pix_per_part - 1) / pix_per_part;
        pl.part_len = pix_per_part;
        pl.patch_pix = static_cast<int32_t>(pix_per_part);
      } else {
        const int64_t RH = len;
        if (RH > a.geom.Ho) break;
        pix_per_part = RH * a.geom.Wo;
        if (pix_per_part > max_pix) break;
        pl.row_parts = static_cast<int32_t>((a.geom.Ho + RH - 1) / RH);
        parts = a.B * pl.row_parts;
        pl.part_len = RH;
        pl.patch_cols = (a.geom.Wo - 1) * a.geom.sw + a.geom.KW;
        const int32_t prow = static_cast<int32_t>((RH - 1) * a.geom.sh + a.geom.KH);
        pl.patch_pix = prow * pl.patch_cols;
      }
      // channel chunk and buffering: pick the cheapest that fits.  Costs are
      // in MFMA issue slots (16 cycles); an exposed patch load costs its
      // bytes at one CU's share of HBM bandwidth (~13 B/clk).
      double cbest = 1e300;
      Plan pbest{};
      for (int32_t cinb = 512; cinb >= kKS; cinb /= 2) {
        if (Cin % cinb) continue;
        for (int32_t nbuf = 1; nbuf <= 2; ++nbuf) {
          Plan t = pl;
          if (nbuf == 2 && Cin / cinb < 2) continue;
          if (!layout(t, cinb, Cin, nbuf)) continue;
          const double load = t.patch_pix * static_cast<double>(cinb) * 2.0 / 208.0;
          const double exposed = nbuf == 2 ? load : load * t.nchunks;
          const double expand = t.nchunks * (t.b_bytes / 2048.0 + 8.0);
          const double c = exposed + expand;
          if (c < cbest) {
            cbest = c;
            pbest = t;
          }
        }
      }
      if (cbest >= 1e299) continue;
      pl = pbest;
      const int64_t wgs = parts * pl.nob;
      const int64_t per_cu = (wgs + 255) / 256;
      const int64_t tiles = (pix_per_part + 15) / 16;
      const int64_t tiles_per_wave = (tiles + WP - 1) / WP;
      const double mfma = static_cast<double>(tiles_per_wave) * taps * (Cin / kKS) * 4.0;
      const double reread = (pl.nob - 1) * static_cast<double>(pix_per_part) * taps * Cin * 2.0 / 4096.0 / 16.0;
      const double cost = static_cast<double>(per_cu) * (mfma + cbest + reread);
      if (cost < best_cost) {
        best_cost = cost;
        best = pl;
        best.parts = (parts + kXcds - 1) / kXcds * kXcds;
        found = true;
      }
    }
  }
  return found;
}

template <typename YT>
hipError_t launch_y(const ProductArgs& a, const Plan& pl, hipStream_t s) {
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&dense_tile_kernel<YT>), hipFuncAttributeMaxDynamicSharedMemorySize,
      kLdsMax);
  if (attr != hipSuccess) return attr;
  const size_t lds = static_cast<size_t>(pl.buf_bytes) * pl.nbuf;
  const dim3 grid(static_cast<uint32_t>(pl.parts * pl.nob));
  Epilogue<YT> ep{a.scale, a.bias, static_cast<const YT*>(a.residual), a.relu};
  ConvGeom g = a.geom;
  int32_t Bimg = static_cast<int32_t>(a.B);
  int64_t x_elems;
  if (!a.conv) {  // FC: rows of X are "pixels" of a 1x1 convolution
    g = ConvGeom{1, 1, static_cast<int32_t>(a.C), 1, 1, 1, 1, 0, 0, 1, 1};
    Bimg = 1;
    x_elems = a.N * a.C;
  } else {
    x_elems = a.B * static_cast<int64_t>(a.geom.H) * a.geom.W * a.geom.Cin;
  }
  hipLaunchKernelGGL((dense_tile_kernel<YT>), grid, dim3(kThreads), lds, s,
                     static_cast<const uint16_t*>(a.X), static_cast<uint32_t>(x_elems * 2), a.N, a.C, g, Bimg,
                     static_cast<const uint16_t*>(a.vals), a.idx, a.O, a.G, a.K, ep, static_cast<YT*>(a.Y), pl);
  return hipGetLastError();
}

}  // namespace

bool dense_tile_supports(const ProductArgs& a) {
  if (a.x_t != DType::BF16 || a.val_t != DType::BF16) return false;
  if (a.G < 1 || kBN % a.G != 0) return false;
  const int64_t Cin = a.conv ? a.geom.Cin : a.C;
  if (Cin % kKS != 0) return false;
  const int64_t x_elems = a.conv ? a.B * static_cast<int64_t>(a.geom.H) * a.geom.W * a.geom.Cin : a.N * a.C;
  if (x_elems * 2 >= static_cast<int64_t>(kOOB)) return false;  // 32-bit buffer offsets
  Plan pl;
  return make_plan(a, pl);
}

hipError_t launch_dense_tile(const ProductArgs& a, hipStream_t s) {
  Plan pl;
  if (!make_plan(a, pl)) return hipErrorInvalidConfiguration;
  if (a.y_t == DType::BF16) return launch_y<bf16_t>(a, pl, s);
  return launch_y<float>(a, pl, s);
}

}  // namespace cci
