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
// Work decomposition.  A workgroup (8 waves, two per SIMD) owns WO 64-output
// blocks and a set of output pixels; the waves are arranged WO (output
// blocks) x WP (pixel groups).  Each wave accumulates up to MT 16-pixel tiles
// x 64 outputs in registers.  The reduction runs over channel chunks of CINB
// channels x all KH*KW taps:
//   - the activation patch of the chunk (every input pixel any tap of the
//     workgroup's outputs touches, CINB channels) is DMA'd from HBM straight
//     into LDS with buffer_load...lds; out-of-image pixels read as zero
//     because their buffer offsets are out of range (this *is* the conv
//     padding); each pixel's 16-byte chunks are followed by one pad slot so
//     the MFMA operand reads are bank-conflict free;
//   - the expanded weight tile of the chunk is built in LDS while the patch
//     streams in (the packed rows are loaded into registers first);
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
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kThreads = 512;
constexpr int kWaves = 8;          // two per SIMD: one wave's stalls are the other's MFMA slots
constexpr int kLoadWaves = 4;      // waves 0..3 stream activations; waves 4..7 expand weights
constexpr int kRoleThreads = kLoadWaves * 64;
constexpr int kBN = 64;            // outputs per wave
constexpr int kKS = 32;            // reduction columns per MFMA k-step
constexpr int kMT = 4;             // max 16-pixel tiles per wave
constexpr int kBPad = 8;           // weight-tile row padding (bf16 elements)
constexpr int kXcds = 8;
constexpr int kLdsMax = 160 * 1024;
constexpr int kDmaMax = 20;        // patch DMA instructions per loader thread per chunk
constexpr int kDmaEarly = 2;       // of those, issued before the expanders' loads are queued
constexpr int kRowMax = 8;         // packed-row segments per expander thread per expansion
constexpr int kUnitMax = 4;        // ring: staged scatter units per expander thread
constexpr int kPkMax = 4;          // ring: staging DMA instructions (value, index) per loader thread
constexpr int kStPitch = kBN * 4 + 16;   // epilogue staging: bytes per pixel row (padded)
constexpr uint32_t kOOB = 0x80000000u;   // buffer offset that reads as zero / drops a store
constexpr int kRsrcWord3 = 0x00020000;   // raw buffer descriptor word 3 (gfx9 family)

// Division by a launch-constant divisor d >= 1: floor(n / d) = umulhi(n, m)
// with m = floor(2^32 / d) + 1, exact for n * d < 2^32.  d == 1 has m = 0 and
// an all-ones `one` mask that passes n through, so there is no branch.
struct FastDiv {
  uint32_t m, one;
};
__host__ __device__ inline FastDiv make_fastdiv(uint32_t d) {
  return FastDiv{d > 1 ? static_cast<uint32_t>((uint64_t(1) << 32) / d + 1) : 0u, d > 1 ? 0u : ~0u};
}
__device__ __forceinline__ uint32_t fdiv(uint32_t n, FastDiv f) { return __umulhi(n, f.m) + (n & f.one); }

// Everything a launch needs, as 32-bit values computed on the host (every
// extent is checked to stay below 2^31 bytes before a launch is planned).
struct Params {
  const uint16_t* X;
  const uint16_t* vals;
  const uint8_t* idx;
  const float* scale;
  const float* bias;
  const void* residual;
  void* Y;
  uint32_t x_bytes, y_bytes, packed_n;  // buffer extents: bytes, bytes, packed elements
  int32_t N, C, O, G, K, relu;
  // convolution geometry; FC runs as a 1x1 convolution over N "pixels"
  int32_t H, W, Cin, KW, sh, sw, ph, pw, Ho, Wo, Bimg;
  int32_t strided;      // rows mode: 1x1 convolution with stride (input pixels are gathered)
  // plan: work split
  int32_t WO, WP;       // wave arrangement (WO * WP == 8)
  int32_t nob;          // output super-blocks of WO*64 outputs
  int32_t part_len;     // rows mode: output pixels per partition; rect: output rows (RH)
  int32_t row_parts;    // rect: partitions per image
  // plan: reduction chunks and LDS layout
  int32_t cinb;         // channels per chunk (power of two, multiple of 32)
  int32_t lg_cpp;       // log2(cinb / 8): 16-byte data chunks per patch pixel
  int32_t lg_ksteps;    // log2(cinb / 32)
  int32_t nchunks, taps;
  int32_t wres;         // 1: one weight tile holds every chunk (expanded once); 0: ring of three
  int32_t nwb;          // weight tiles in LDS (1, or 3 for the ring)
  int32_t npb;          // patch buffers in LDS (ring; chunk j uses buffer j % npb)
  int32_t patch_cols;   // rect: staged input columns
  int32_t patch_pix;    // staged pixels per chunk
  int32_t slots;        // 16-byte patch slots per chunk (patch_pix * (cpp + 1))
  int32_t b_pitch;      // bf16 elements per weight-tile row
  int32_t w_bytes;      // bytes of one weight tile (WO*64 rows)
  int32_t p_bytes;      // bytes of one patch buffer
  int32_t s_bytes;      // ring: bytes of one packed-row staging buffer (0: resident)
  int32_t s_vslots;     // ring: 16-byte value slots of one staging buffer (the index slots follow
                        // at a 1 KiB boundary, s_vblk64 * 64 slots in)
  int32_t s_islots;     // ring: 16-byte index slots
  int32_t s_vblk64;     // ring: value slots rounded up to 64
  int32_t ncols8;       // 8-column blocks of one expansion (whole tile or one chunk)
  int32_t nu;           // expansion units (group x 8-column block) per expander thread
  int32_t nus;          // ring: staged scatter units (packed row x 8-column block) per expander thread
  int32_t nrows;        // packed rows of one output super-block
  int32_t mt;           // 16-pixel tiles per wave (compile-time instantiation)
  uint32_t kw_mul;      // tap / KW == (tap * kw_mul) >> 20 for tap < 4096
  // loader slot walk: each step advances 256 slots = dq pixels + dc slots;
  // rect: dq pixels = dpr patch rows + diw patch columns
  int32_t dq, dc, dpr, diw;
  FastDiv fd_nob, fd_rparts, fd_wo, fd_pcols, fd_pps, fd_k, fd_ncols8, fd_tc, fd_howo;
  FastDiv fd_taps, fd_v8, fd_v16;  // ring staging: taps, cinb/8, cinb/16
};

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t v) { return __builtin_bit_cast(bf16x8_t, v); }

// Workgroup barrier for LDS traffic only.  __syncthreads() also waits for
// every outstanding vector-memory operation (the patch DMA counts as one),
// which would serialise the activation stream with the weight expansion.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Wait until at most N vector-memory operations of this wave are in flight
// (loads complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
// Patch layout: pixel q occupies cpp + 1 consecutive 16-byte slots (cpp
// data chunks and one pad slot).  The odd slot pitch spreads 8 consecutive
// pixels reading the same chunk over all 32 banks, and makes the operand
// address of any tap a single add.
template <typename YT, bool RECT, int MT>
__global__ __launch_bounds__(kThreads) void dense_tile_kernel(Params p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  constexpr uint32_t ysz = sizeof(YT);

  // ---- workgroup -> (pixel partition, output super-block), XCD-aware ----
  const uint32_t id = blockIdx.x;
  const uint32_t jid = id / kXcds;
  const uint32_t jq = fdiv(jid, p.fd_nob);
  const int32_t ob = static_cast<int32_t>(jid - jq * static_cast<uint32_t>(p.nob));
  const uint32_t part = jq * kXcds + id % kXcds;

  int32_t npix, P0 = 0, b_img = 0, oh0 = 0;
  if constexpr (RECT) {
    b_img = static_cast<int32_t>(fdiv(part, p.fd_rparts));
    if (b_img >= p.Bimg) return;
    oh0 = static_cast<int32_t>(part - static_cast<uint32_t>(b_img * p.row_parts)) * p.part_len;
    const int32_t rh = p.Ho - oh0 < p.part_len ? p.Ho - oh0 : p.part_len;
    npix = rh * p.Wo;
  } else {
    P0 = static_cast<int32_t>(part) * p.part_len;
    if (P0 >= p.N) return;
    npix = p.N - P0 < p.part_len ? p.N - P0 : p.part_len;
  }

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool loader = wave < kLoadWaves;  // wave-uniform role
  const int rt = threadIdx.x - (loader ? 0 : kRoleThreads);  // thread index within the role
  const int cpp = 1 << p.lg_cpp;
  const int pps = cpp + 1;
  const int32_t wofs_patch = p.nwb * p.w_bytes;  // LDS offset of patch buffer 0

  // ---- expanders: weight-tile build -----------------------------------------
  // Unit u = (group gl, 8-column block col8) of one expansion (the whole tile,
  // or one chunk): its G tile rows x 8 columns are zero-filled and receive
  // the 8 columns of the group's K packed rows, all by one thread (program
  // order is the only synchronisation).  Thread rt owns units rt + 256 j
  // (j < nu); its packed-row segments ("slots", unit-major, K per unit) are
  // loaded kRowMax at a time.  The tile column of col8 is 8 * col8, its
  // source column tap * Cin + (chunk) * cinb + 8 * c8.
  const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.vals), (short)0, static_cast<int>(p.packed_n * 2u), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t ir = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(p.idx), (short)0, static_cast<int>(p.packed_n), kRsrcWord3);
  const int gpb = (p.WO * kBN) / p.G;
  // groups that exist (the last super-block may be partial)
  const int glim = p.O / p.G - ob * gpb < gpb ? p.O / p.G - ob * gpb : gpb;
  const int nslots = p.nu * p.K;
  const uint32_t gmask = static_cast<uint32_t>(p.G - 1);
  struct Packed {
    u32x4_t v[kRowMax];
    u32x2_t ix[kRowMax];
    int32_t dst[kRowMax];  // tile element offset of the unit's first row (< 0: none); bit 30: first slot
  };
  constexpr int32_t kFirst = 1 << 30;
  Packed P;
  // load slots s0 .. s0+kRowMax-1 of the expansion of chunk ch
  auto load_slots = [&](int ch, int s0) {
#pragma unroll
    for (int i = 0; i < kRowMax; ++i) {
      const int sl = s0 + i;
      const int j = static_cast<int>(fdiv(sl, p.fd_k));
      const int k = sl - j * p.K;
      const int u = rt + kRoleThreads * j;
      const int gl = static_cast<int>(fdiv(u, p.fd_ncols8));
      const int col8 = u - gl * p.ncols8;
      const bool ok = sl < nslots && gl < glim;
      const int chl = static_cast<int>(fdiv(col8, p.fd_tc));
      const int rem = col8 - chl * (p.taps << p.lg_cpp);
      const uint32_t e = static_cast<uint32_t>(((ob * gpb + gl) * p.K + k) * p.C + (rem >> p.lg_cpp) * p.Cin +
                                               (chl + ch) * p.cinb + 8 * (rem & (cpp - 1)));
      P.v[i] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(vr, ok ? e * 2u : kOOB, 0, 0));
      P.ix[i] = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(ir, ok ? e : kOOB, 0, 0));
      P.dst[i] = ok ? (gl * p.G * p.b_pitch + 8 * col8) | (k == 0 ? kFirst : 0) : -1;
    }
  };
  // write the loaded slots into weight tile wb: a unit's first slot zero-fills
  // its G rows; every kept weight goes to row G*g + idx (Alg. 1's target row)
  auto scatter_slots = [&](int wb) {
    uint16_t* bs = reinterpret_cast<uint16_t*>(lds + wb * p.w_bytes);
#pragma unroll
    for (int i = 0; i < kRowMax; ++i) {
      if (P.dst[i] >= 0) {
        uint16_t* dst = bs + (P.dst[i] & (kFirst - 1));
        if (P.dst[i] & kFirst) {
          for (int r = 0; r < p.G; ++r)
            *reinterpret_cast<u32x4_t*>(dst + r * p.b_pitch) = u32x4_t{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          // idx: row in the group (< G, a power of two on this path; the
          // mask keeps a corrupt index inside its own group)
          const uint32_t row = (P.ix[i][jj >> 2] >> (8 * (jj & 3))) & gmask;
          const uint16_t w = static_cast<uint16_t>(P.v[i][jj >> 1] >> (16 * (jj & 1)));
          dst[row * p.b_pitch + jj] = w;
        }
      }
    }
  };
  // whole expansion of chunk ch into tile wb; the first kRowMax slots may
  // already be loaded (prefetched)
  auto expand = [&](int ch, int wb, bool prefetched) {
    for (int s0 = 0; s0 < nslots; s0 += kRowMax) {
      if (s0 > 0 || !prefetched) load_slots(ch, s0);
      scatter_slots(wb);
    }
  };
  if (!loader) load_slots(0, 0);

  // ---- loaders: patch DMA -------------------------------------------------
  // Loader thread rt owns slots rt + 256 i (i < nd); consecutive slots of one
  // pixel are its 16-byte channel chunks (the last one is the pad slot).  The
  // offsets of chunk 0 are walked incrementally (the first kDmaEarly DMAs
  // are issued as soon as their offsets are known, the rest after the
  // expanders' packed-row loads are queued); chunk j reuses them plus
  // j*cinb*2.
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.X), (short)0, static_cast<int>(p.x_bytes), kRsrcWord3);
  const int32_t nd = p.slots > wave * 64 ? (p.slots - wave * 64 + kRoleThreads - 1) / kRoleThreads : 0;
  uint32_t doff[kDmaMax];
  auto dma = [&](uint32_t pofs, int i, uint32_t off) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t*)(lds + pofs + (wave + kLoadWaves * i) * 1024), 16, off,
                                             0, 0, 0);
  };
  if (loader) {
    const int32_t cin2 = p.Cin * 2;
    int32_t s = rt;
    int32_t q = static_cast<int32_t>(fdiv(static_cast<uint32_t>(s), p.fd_pps));
    int32_t c = s - q * pps;
    if constexpr (RECT) {
      int32_t pr = static_cast<int32_t>(fdiv(static_cast<uint32_t>(q), p.fd_pcols));
      int32_t iw = q - pr * p.patch_cols;  // patch column
      const int32_t ih0 = oh0 * p.sh - p.ph;
      // the pixel index may be negative (padding): then the slot is invalid
      int32_t off = ((b_img * p.H + ih0 + pr) * p.W + iw - p.pw) * cin2 + 16 * c;
      const int32_t d_base = (p.dpr * p.W + p.diw) * cin2 + 16 * p.dc;
      const int32_t d_carry = cin2 - 16 * pps;
      const int32_t d_wrap = (p.W - p.patch_cols) * cin2;
#pragma unroll
      for (int i = 0; i < kDmaMax; ++i) {
        if (i < nd) {
          const int32_t ih = ih0 + pr, iwi = iw - p.pw;
          const bool ok = s < p.slots && c < cpp && static_cast<uint32_t>(ih) < static_cast<uint32_t>(p.H) &&
                          static_cast<uint32_t>(iwi) < static_cast<uint32_t>(p.W);
          doff[i] = ok ? static_cast<uint32_t>(off) : kOOB;
          if (i < kDmaEarly) dma(static_cast<uint32_t>(wofs_patch), i, doff[i]);
          s += kRoleThreads;
          c += p.dc;
          const bool carry = c >= pps;
          c -= carry ? pps : 0;
          iw += p.diw + (carry ? 1 : 0);
          const bool wrap = iw >= p.patch_cols;
          iw -= wrap ? p.patch_cols : 0;
          pr += p.dpr + (wrap ? 1 : 0);
          off += d_base + (carry ? d_carry : 0) + (wrap ? d_wrap : 0);
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < kDmaMax; ++i) {
        if (i < nd) {
          const bool ok = s < p.slots && c < cpp && q < npix;
          uint32_t nn = static_cast<uint32_t>(P0 + (q < npix ? q : 0));
          if (p.strided) {  // strided 1x1 (uniform branch): gather the input pixel
            const uint32_t b = fdiv(nn, p.fd_howo);
            const uint32_t rem = nn - b * static_cast<uint32_t>(p.Ho * p.Wo);
            const uint32_t oh = fdiv(rem, p.fd_wo);
            nn = (b * p.H + oh * p.sh) * p.W + (rem - oh * p.Wo) * p.sw;
          }
          doff[i] = ok ? nn * static_cast<uint32_t>(cin2) + 16u * static_cast<uint32_t>(c) : kOOB;
          if (i < kDmaEarly) dma(static_cast<uint32_t>(wofs_patch), i, doff[i]);
          s += kRoleThreads;
          c += p.dc;
          const bool carry = c >= pps;
          c -= carry ? pps : 0;
          q += p.diw + (carry ? 1 : 0);
        }
      }
    }
  }
  auto issue_patch = [&](int ch, uint32_t pofs) {
    const uint32_t add = static_cast<uint32_t>(ch * p.cinb) * 2u;
#pragma unroll
    for (int i = 0; i < kDmaMax; ++i) {
      if (i < nd) dma(pofs, i, doff[i] + add);  // wave-uniform
    }
  };

  // ---- per-lane tile geometry: patch pixel of tap (0,0), output byte offset ----
  const int wo = wave % p.WO;
  const int wp = wave / p.WO;
  const int lrow = lane & 15;
  const int lk = lane >> 4;
  const int32_t o_wave = (ob * p.WO + wo) * kBN;
  // Tiles wp, wp+WP, ... belong to this wave; only the last of its MT tile
  // slots can be empty (then its MFMAs are skipped).
  const bool last_tile = (wp + (MT - 1) * p.WP) * 16 < npix;
  uint32_t abase[MT];  // A-fragment LDS byte offset of each tile at tap (0,0), k-step 0
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int32_t px = (wp + mt * p.WP) * 16 + lrow;
    const int32_t pc = px < npix ? px : 0;  // idle lanes read pixel 0 and store nothing
    int32_t qb;
    if constexpr (RECT) {
      const int32_t r = static_cast<int32_t>(fdiv(pc, p.fd_wo));
      qb = r * p.sh * p.patch_cols + (pc - r * p.Wo) * p.sw;
    } else {
      qb = pc;
    }
    abase[mt] = static_cast<uint32_t>((qb * pps + lk) * 16);
  }
  const uint32_t bbase = static_cast<uint32_t>(((wo * kBN + lrow) * p.b_pitch + 8 * lk) * 2);

  f32x4_t acc[MT][4];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int ot = 0; ot < 4; ++ot) acc[mt][ot] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

  // ---- multiply one chunk: weights at LDS offset wofs (+ column col0), patch at pofs ----
  // Reduction steps of 32 columns run tap-major; the operand fragments of
  // step s+1 are read from LDS while the MFMAs of step s issue (two register
  // sets, statically alternated; every read is unconditional so the
  // compiler can count outstanding LDS reads exactly).
  struct Frags {
    bf16x8_t w[4];
    bf16x8_t x[MT];
  };
  // Loaders first issue the next chunk's patch DMA (chunk `dch` into LDS at
  // `dofs`; dch < 0: none).  While a loader waits for room in the memory
  // queue, the expander wave sharing its SIMD keeps the matrix core busy.
  auto compute = [&](uint32_t wofs, uint32_t pofs, int dch, uint32_t dofs) {
    const uint8_t* wb = lds + wofs + bbase;
    const uint8_t* pb = lds + pofs;
    if (loader && dch >= 0) issue_patch(dch, dofs);
    const int nsteps = p.taps << p.lg_ksteps;
    auto addr = [&](int st, uint32_t& aoff, uint32_t& boff) {
      // step -> (tap, kb) -> (kh, kw): shifts and one multiply, all scalar
      const int tap = st >> p.lg_ksteps;
      const int kb = st & ((1 << p.lg_ksteps) - 1);
      const int kh = static_cast<int>((static_cast<uint32_t>(tap) * p.kw_mul) >> 20);
      const int kw = tap - kh * p.KW;
      const int32_t dq = RECT ? kh * p.patch_cols + kw : 0;
      aoff = static_cast<uint32_t>(dq * pps * 16 + kb * 64);
      boff = static_cast<uint32_t>((tap * p.cinb + kb * kKS) * 2);
    };
    auto load_w = [&](uint32_t boff, Frags& f) {
#pragma unroll
      for (int ot = 0; ot < 4; ++ot)
        f.w[ot] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(wb + boff + ot * 16 * p.b_pitch * 2));
    };
    auto load_x = [&](uint32_t aoff, int mt, Frags& f) {
      f.x[mt] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(pb + abase[mt] + aoff));
    };
    // One reduction step on `cur` while the fragments of step `nst` stream
    // into `nxt`: each tile's 4 MFMAs are followed by one LDS read, so every
    // read is issued about one step ahead of its use and at most ~12 reads
    // are outstanding (the LDS counter tracks 15).
    auto step = [&](const Frags& cur, Frags& nxt, int nst) {
      uint32_t aoff, boff;
      addr(nst, aoff, boff);
      load_w(boff, nxt);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        if (mt < MT - 1 || last_tile) {
#pragma unroll
          for (int ot = 0; ot < 4; ++ot)
            acc[mt][ot] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur.w[ot], cur.x[mt], acc[mt][ot], 0, 0, 0);
        }
        load_x(aoff, mt, nxt);
      }
    };
    Frags f0, f1;
    {
      uint32_t aoff, boff;
      addr(0, aoff, boff);
      load_w(boff, f0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) load_x(aoff, mt, f0);
    }
    // Steps past the end re-read the last step (clamped): every read is
    // unconditional, so the compiler can count outstanding reads exactly.
    for (int st = 0; st < nsteps; st += 2) {
      step(f0, f1, st + 1 < nsteps ? st + 1 : nsteps - 1);
      if (st + 1 < nsteps) step(f1, f0, st + 2 < nsteps ? st + 2 : nsteps - 1);
    }
  };

  // ---- ring mode: packed rows staged in LDS by the loaders ----------------
  // Chunk j's packed rows (value segments, then index segments, each 16-byte
  // slot-linear: [row][tap][channel]) are DMA'd two chunks ahead into one of
  // two staging buffers; the expanders build chunk j's tile from there while
  // chunk j-1 is multiplied.
  const int32_t sofs = wofs_patch + p.npb * p.p_bytes;  // LDS offset of staging buffer 0
  // loader thread rt's staging slots: value slot rt + 256 i and index slot
  // rt + 256 i, element offsets at chunk 0 (kOOB: none)
  uint32_t pk_v[kPkMax], pk_i[kPkMax];
  if (loader && !p.wres) {
    const int32_t rowbase = ob * gpb * p.K;
    const int32_t rlim = glim * p.K;
#pragma unroll
    for (int i = 0; i < kPkMax; ++i) {
      const int32_t sl = rt + kRoleThreads * i;
      {
        const int32_t r = static_cast<int32_t>(fdiv(static_cast<uint32_t>(sl), p.fd_v8));  // (row, tap) pair
        const int32_t j = sl - r * cpp;
        const int32_t row = static_cast<int32_t>(fdiv(static_cast<uint32_t>(r), p.fd_taps));
        const int32_t tap = r - row * p.taps;
        pk_v[i] = sl < p.s_vslots && row < rlim
                      ? static_cast<uint32_t>((rowbase + row) * p.C + tap * p.Cin + 8 * j) : kOOB;
      }
      {
        const int32_t r = static_cast<int32_t>(fdiv(static_cast<uint32_t>(sl), p.fd_v16));  // (row, tap) pair
        const int32_t j = sl - r * (cpp >> 1);
        const int32_t row = static_cast<int32_t>(fdiv(static_cast<uint32_t>(r), p.fd_taps));
        const int32_t tap = r - row * p.taps;
        pk_i[i] = sl < p.s_islots && row < rlim
                      ? static_cast<uint32_t>((rowbase + row) * p.C + tap * p.Cin + 16 * j) : kOOB;
      }
    }
  }
  const int npv = p.s_vslots > wave * 64 ? (p.s_vslots - wave * 64 + kRoleThreads - 1) / kRoleThreads : 0;
  const int npi = p.s_islots > wave * 64 ? (p.s_islots - wave * 64 + kRoleThreads - 1) / kRoleThreads : 0;
  auto issue_packed = [&](int ch, int sb) {
    const uint32_t stg = static_cast<uint32_t>(sofs + sb * p.s_bytes);
    const uint32_t istg = stg + static_cast<uint32_t>(p.s_vblk64) * 16u;
    const uint32_t add = static_cast<uint32_t>(ch * p.cinb);
#pragma unroll
    for (int i = 0; i < kPkMax; ++i) {
      if (i < npv)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_void_t*)(lds + stg + (wave + kLoadWaves * i) * 1024), 16,
                                                 pk_v[i] == kOOB ? kOOB : (pk_v[i] + add) * 2u, 0, 0, 0);
      if (i < npi)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ir, (lds_void_t*)(lds + istg + (wave + kLoadWaves * i) * 1024), 16,
                                                 pk_i[i] == kOOB ? kOOB : pk_i[i] + add, 0, 0, 0);
    }
  };
  // Scatter one chunk's staged packed rows into weight tile wb, which was
  // zero-filled a chunk earlier.  Unit = (packed row, 8-column block), so the
  // work spreads over K times more threads than whole groups would.  With
  // K == G every row is kept in ascending order: a row is copied whole.
  // per-thread scatter units of the staged path, decoded once:
  // staged byte offset of the unit's value segment, tile element offset
  int32_t su_src[kUnitMax], su_dst[kUnitMax];
  if (!loader && !p.wres) {
    const int rowpitch = 8 * p.ncols8;  // staged elements per packed row
    const int rlim = glim * p.K;
#pragma unroll
    for (int j = 0; j < kUnitMax; ++j) {
      const int u = rt + kRoleThreads * j;
      const int r = static_cast<int>(fdiv(u, p.fd_ncols8));
      const int col8 = u - r * p.ncols8;
      const int gl = static_cast<int>(fdiv(r, p.fd_k));
      const bool ok = j < p.nus && r < rlim;
      su_src[j] = ok ? (r * rowpitch + 8 * col8) : -1;
      su_dst[j] = gl * p.G * p.b_pitch + 8 * col8 + (p.K == p.G ? (r - gl * p.K) * p.b_pitch : 0);
    }
  }
  auto scatter_staged = [&](int wb, int sb) {
    const uint8_t* stg = lds + sofs + sb * p.s_bytes;
    uint16_t* bs = reinterpret_cast<uint16_t*>(lds + wb * p.w_bytes);
#pragma unroll
    for (int j = 0; j < kUnitMax; ++j) {
      if (su_src[j] < 0) continue;
      uint16_t* dst = bs + su_dst[j];
      const u32x4_t v = *reinterpret_cast<const u32x4_t*>(stg + su_src[j] * 2);
      if (p.K == p.G) {  // every row kept, in order: the row is copied whole
        *reinterpret_cast<u32x4_t*>(dst) = v;
        continue;
      }
      const u32x2_t ix = *reinterpret_cast<const u32x2_t*>(stg + p.s_vblk64 * 16 + su_src[j]);
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        const uint32_t rr = (ix[jj >> 2] >> (8 * (jj & 3))) & gmask;  // idx: row in the group
        const uint16_t w = static_cast<uint16_t>(v[jj >> 1] >> (16 * (jj & 1)));
        dst[rr * p.b_pitch + jj] = w;
      }
    }
  };
  // zero fill of weight tile wb by the loaders (not needed when K == G): DMA
  // with an out-of-range source offset writes zeros into LDS without reading
  // memory, so a loader never waits on the LDS queue for it (a tile is a
  // whole number of KiB)
  auto zero_tile = [&](int wb) {
    if (p.K == p.G) return;
    const int nblk = p.w_bytes / 1024;
    for (int b = wave; b < nblk; b += kLoadWaves)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t*)(lds + wb * p.w_bytes + b * 1024), 16, kOOB, 0, 0, 0);
  };

  // ---- chunk pipeline -----------------------------------------------------
  // Loaders stream patches through npb (1 or 2) buffers: chunk 0 from the
  // first instructions, chunk j+1 during chunk j's MFMAs.  Expanders build
  // the weight tile: once (resident), or (ring) chunk 0 from registers and
  // chunk j+1 from its staged packed rows while chunk j is multiplied, into
  // the other of two tiles.  A loader's MFMAs fill the SIMD its partner
  // expander shares while that one builds.  One barrier per chunk; one call
  // site for compute() keeps the accumulators in place.
  // The packed-row loads go into the memory queue ahead of the bulk of the
  // patch DMA, which would otherwise hold them up.
  lds_barrier();
  const bool ring = !p.wres;
  if (loader) {
#pragma unroll
    for (int i = kDmaEarly; i < kDmaMax; ++i)
      if (i < nd) dma(static_cast<uint32_t>(wofs_patch), i, doff[i]);
    if (ring && p.nchunks > 1) {
      issue_packed(1, 1);
      zero_tile(1);
    }
    wait_vm<0>();  // chunk 0 (and chunk 1's packed rows) landed
  } else {
    expand(0, 0, true);
  }
  lds_barrier();
  int pb = 0;
  for (int ch = 0; ch < p.nchunks; ++ch) {
    const int wcur = ch % 3;  // ring tile of chunk ch
    const uint32_t wofs = p.wres ? static_cast<uint32_t>(ch * p.taps * p.cinb * 2) : static_cast<uint32_t>(wcur * p.w_bytes);
    const int nb = p.npb == 2 ? pb ^ 1 : 0;
    if (ring && ch + 1 < p.nchunks) {
      const int wnext = wcur == 2 ? 0 : wcur + 1;
      if (loader) {
        if (ch + 2 < p.nchunks) {
          issue_packed(ch + 2, ch & 1);
          zero_tile(wnext == 2 ? 0 : wnext + 1);  // the tile of chunk ch+2 (last read by chunk ch-1)
        }
      } else {
        scatter_staged(wnext, (ch + 1) & 1);
      }
    }
    // with two patch buffers the next chunk streams in during this one
    const int dch = p.npb == 2 && ch + 1 < p.nchunks ? ch + 1 : -1;
    compute(wofs, static_cast<uint32_t>(wofs_patch + pb * p.p_bytes), dch, static_cast<uint32_t>(wofs_patch + nb * p.p_bytes));
    if (ch + 1 < p.nchunks) {
      if (p.npb == 1) {
        lds_barrier();  // every wave is done with the patch buffer
        if (loader) issue_patch(ch + 1, static_cast<uint32_t>(wofs_patch));
      }
      if (loader) wait_vm<0>();  // chunk ch+1's patch (and chunk ch+2's packed rows) landed
      lds_barrier();
      pb = nb;
    }
  }

  // ---- fused epilogue, staged through LDS ---------------------------------
  // A lane's accumulators are 4 consecutive outputs of one pixel per (tile,
  // 16-output block).  Each wave parks its fp32 block (MT*16 pixels x 64
  // outputs) in LDS and reads it back transposed: a lane then owns 8
  // consecutive outputs of one pixel, applies scale/bias/residual/ReLU,
  // rounds once and writes them with one store, so 8 lanes write a pixel's
  // whole run of 64 outputs.
  lds_barrier();  // every wave is done with the operand buffers
  uint8_t* stg = lds + wave * (MT * 16 * kStPitch);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int ot = 0; ot < 4; ++ot)
      *reinterpret_cast<f32x4_t*>(stg + (mt * 16 + lrow) * kStPitch + (ot * 16 + 4 * lk) * 4) = acc[mt][ot];
  const __amdgpu_buffer_rsrc_t yr =
      __builtin_amdgcn_make_buffer_rsrc(p.Y, (short)0, static_cast<int>(p.y_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(p.residual), (short)0, p.residual ? static_cast<int>(p.y_bytes) : 0, kRsrcWord3);
  const int c8 = lane & 7;                 // 8-output block of the wave's 64
  const int32_t o = o_wave + 8 * c8;
  // O % 4 == 0: a block holds 8, 4 (the last one) or no valid outputs
  const int nvalid = o + 8 <= p.O ? 8 : (o < p.O ? 4 : 0);
  f32x4_t sc0{1.f, 1.f, 1.f, 1.f}, sc1{1.f, 1.f, 1.f, 1.f}, bi0{0.f, 0.f, 0.f, 0.f}, bi1{0.f, 0.f, 0.f, 0.f};
  if (p.scale && nvalid) sc0 = *reinterpret_cast<const f32x4_t*>(p.scale + o);
  if (p.scale && nvalid == 8) sc1 = *reinterpret_cast<const f32x4_t*>(p.scale + o + 4);
  if (p.bias && nvalid) bi0 = *reinterpret_cast<const f32x4_t*>(p.bias + o);
  if (p.bias && nvalid == 8) bi1 = *reinterpret_cast<const f32x4_t*>(p.bias + o + 4);
#pragma unroll
  for (int r = 0; r < MT * 2; ++r) {  // 8 pixels per pass
    const int lp = r * 8 + (lane >> 3);  // wave-local staged pixel
    const int mt = r >> 1;
    if (mt == MT - 1 && !last_tile) break;  // wave-uniform: empty tile slot
    const int32_t px = (wp + mt * p.WP) * 16 + (lp & 15);
    const f32x4_t a0 = *reinterpret_cast<const f32x4_t*>(stg + lp * kStPitch + c8 * 32);
    const f32x4_t a1 = *reinterpret_cast<const f32x4_t*>(stg + lp * kStPitch + c8 * 32 + 16);
    uint32_t n;
    if constexpr (RECT) {
      const int32_t orow = static_cast<int32_t>(fdiv(px, p.fd_wo));
      n = static_cast<uint32_t>((b_img * p.Ho + oh0 + orow) * p.Wo + (px - orow * p.Wo));
    } else {
      n = static_cast<uint32_t>(P0 + px);
    }
    const bool ok = px < npix && nvalid > 0;
    const uint32_t off = ok ? (n * static_cast<uint32_t>(p.O) + static_cast<uint32_t>(o)) * ysz : kOOB;
    const uint32_t off_hi = ok && nvalid == 8 ? off + 4 * ysz : kOOB;  // outputs o+4..o+7
    f32x4_t y0, y1;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      y0[jj] = __builtin_fmaf(a0[jj], sc0[jj], bi0[jj]);
      y1[jj] = __builtin_fmaf(a1[jj], sc1[jj], bi1[jj]);
    }
    if (p.residual) {
      if constexpr (ysz == 2) {
        const u32x2_t r0 = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(rr, off, 0, 0));
        const u32x2_t r1 = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(rr, off_hi, 0, 0));
        y0[0] += __uint_as_float(r0[0] << 16);
        y0[1] += __uint_as_float(r0[0] & 0xffff0000u);
        y0[2] += __uint_as_float(r0[1] << 16);
        y0[3] += __uint_as_float(r0[1] & 0xffff0000u);
        y1[0] += __uint_as_float(r1[0] << 16);
        y1[1] += __uint_as_float(r1[0] & 0xffff0000u);
        y1[2] += __uint_as_float(r1[1] << 16);
        y1[3] += __uint_as_float(r1[1] & 0xffff0000u);
      } else {
        y0 += __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, 0));
        y1 += __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rr, off_hi, 0, 0));
      }
    }
    if (p.relu) {
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        y0[jj] = y0[jj] > 0.0f ? y0[jj] : (y0[jj] != y0[jj] ? y0[jj] : 0.0f);
        y1[jj] = y1[jj] > 0.0f ? y1[jj] : (y1[jj] != y1[jj] ? y1[jj] : 0.0f);
      }
    }
    if constexpr (ysz == 2) {
      // v_cvt_pk_bf16_f32: round to nearest even
      const u32x4_t pk = {__builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y0[0], y0[1]}), bf16x2_t)),
                          __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y0[2], y0[3]}), bf16x2_t)),
                          __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y1[0], y1[1]}), bf16x2_t)),
                          __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y1[2], y1[3]}), bf16x2_t))};
      if (nvalid == 8 || !ok) {
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(yr, 0, 0, 0)), pk), yr, off, 0, 0);
      } else {  // last block of 4
        const u32x2_t lo = {pk[0], pk[1]};
        __builtin_amdgcn_raw_buffer_store_b64(
            __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b64(yr, 0, 0, 0)), lo), yr, off, 0, 0);
      }
    } else {
      __builtin_amdgcn_raw_buffer_store_b128(
          __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(yr, 0, 0, 0)), y0), yr, off, 0, 0);
      __builtin_amdgcn_raw_buffer_store_b128(
          __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(yr, 0, 0, 0)), y1), yr, off_hi, 0, 0);
    }
  }
}

// ---------------------------------------------------------------------------
// Host-side planning.

bool is_rows_mode(const ProductArgs& a) {
  return !a.conv || (a.geom.KH == 1 && a.geom.KW == 1 && a.geom.ph == 0 && a.geom.pw == 0);
}

int ilog2(int v) {
  int l = 0;
  while ((1 << l) < v) ++l;
  return l;
}

// Fill the chunk and LDS layout; false if it does not fit the LDS, the
// per-thread DMA budget or the per-thread expansion budget.
bool layout(Params& pl, int32_t cinb, int32_t Cin, int32_t wres, int32_t npb, int32_t G, int32_t K) {
  pl.cinb = cinb;
  pl.lg_cpp = ilog2(cinb / 8);
  pl.lg_ksteps = ilog2(cinb / kKS);
  pl.nchunks = Cin / cinb;
  if (!wres && pl.nchunks < 2) return false;
  if (npb < 1 || npb > pl.nchunks) return false;
  const int32_t cpp = cinb / 8, pps = cpp + 1;
  const int64_t slots = static_cast<int64_t>(pl.patch_pix) * pps;
  if (slots > static_cast<int64_t>(kDmaMax) * kRoleThreads) return false;
  pl.slots = static_cast<int32_t>(slots);
  const int32_t tc = pl.taps * cpp;
  pl.wres = wres;
  pl.ncols8 = wres ? pl.nchunks * tc : tc;
  pl.b_pitch = pl.ncols8 * 8 + kBPad;
  pl.w_bytes = pl.WO * kBN * pl.b_pitch * 2;
  pl.nrows = (pl.WO * kBN / G) * K;
  pl.nu = ((pl.WO * kBN / G) * pl.ncols8 + kRoleThreads - 1) / kRoleThreads;
  pl.nus = (pl.nrows * pl.ncols8 + kRoleThreads - 1) / kRoleThreads;
  if (!wres && pl.nus > kUnitMax) return false;
  if (pl.nu * K > 4 * kRowMax) return false;  // at most four load rounds per expansion
  pl.nwb = wres ? 1 : 3;
  // the DMA writes whole 64-slot (1 KiB) blocks: round the patch up so the
  // tail of its last block stays inside its buffer
  pl.p_bytes = static_cast<int32_t>((slots * 16 + 1023) / 1024 * 1024);
  pl.npb = npb;
  pl.s_bytes = pl.s_vslots = pl.s_islots = pl.s_vblk64 = 0;
  if (!wres) {  // packed-row staging: nrows x taps x (cinb/8 value + cinb/16 index) slots
    pl.s_vslots = pl.nrows * pl.taps * (cinb / 8);
    pl.s_islots = pl.nrows * pl.taps * (cinb / 16);
    pl.s_vblk64 = (pl.s_vslots + 63) / 64 * 64;
    pl.s_bytes = (pl.s_vblk64 + (pl.s_islots + 63) / 64 * 64) * 16;
    if (pl.s_vslots > kPkMax * kRoleThreads || pl.s_islots > kPkMax * kRoleThreads) return false;
  }
  if (static_cast<int64_t>(pl.nwb) * pl.w_bytes + static_cast<int64_t>(npb) * pl.p_bytes +
          2 * static_cast<int64_t>(pl.s_bytes) > kLdsMax)
    return false;
  pl.fd_taps = make_fastdiv(pl.taps);
  pl.fd_v8 = make_fastdiv(cinb / 8);
  pl.fd_v16 = make_fastdiv(cinb / 16);
  pl.dq = kRoleThreads / pps;
  pl.dc = kRoleThreads % pps;
  // rect: dq pixels = dpr patch rows + diw patch columns; rows: diw = dq pixels
  pl.dpr = pl.patch_cols > 0 ? pl.dq / pl.patch_cols : 0;
  pl.diw = pl.patch_cols > 0 ? pl.dq % pl.patch_cols : pl.dq;
  pl.fd_pps = make_fastdiv(pps);
  pl.fd_k = make_fastdiv(K);
  pl.fd_ncols8 = make_fastdiv(pl.ncols8);
  pl.fd_tc = make_fastdiv(tc);
  return true;
}

// Modelled duration (cycles) of one workgroup: a chunk's patch streams at
// one CU's share of HBM bandwidth (~13 B/clk) once its buffer is free (two
// buffers: from the start of the previous chunk's MFMAs); its MFMAs start
// when it has arrived, its weights are expanded and the previous chunk is
// done.
double model_cycles(const Params& t, double mfma_chunk, double store, int K) {
  const double load = t.patch_pix * static_cast<double>(t.cinb) * 2.0 / 13.0;
  // expansion by the 256 expander threads: zero fill (b128 writes) and
  // K packed-row segments per unit
  const double build = t.w_bytes / 16.0 / kRoleThreads * 8.0 + t.nu * K * 120.0;
  const double latency = 1500.0, barrier = 150.0, setup = 1500.0;
  const double e_first = setup + latency + build * (t.wres ? 1 : 2);
  double arrive = setup / 2 + latency + load, done = 0.0, start = 0.0;
  double done2 = 0.0;  // done time of chunk c-2
  const int n = t.nchunks;
  for (int c = 0; c < n; ++c) {
    if (c > 0) {
      const double issue = t.npb == 2 ? start : done + barrier;
      arrive = (issue > arrive ? issue : arrive) + load;
    }
    double ready_w = e_first;
    // ring: chunk c is scattered during chunk c-1's MFMAs by the expander half
    if (!t.wres && c >= 1) ready_w = (c >= 2 ? done2 : e_first) + barrier + t.nus * 8.0 * 16.0;
    double st = c == 0 ? 0.0 : done + barrier;
    st = st > arrive ? st : arrive;
    st = st > ready_w ? st : ready_w;
    start = st;
    done2 = done;
    done = st + mfma_chunk;
  }
  return done + store;
}

// Choose the wave arrangement, pixel partition, channel chunk and LDS plan
// with the smallest modelled time on the busiest CU (one workgroup per CU at
// a time).
bool make_plan(const ProductArgs& a, Params& best, uint32_t& grid) {
  const int32_t Cin = a.conv ? a.geom.Cin : static_cast<int32_t>(a.C);
  const bool rows = is_rows_mode(a);
  const int32_t taps = a.conv ? a.geom.KH * a.geom.KW : 1;
  const int64_t ysz = a.y_t == DType::F32 ? 4 : 2;
  double best_cost = 1e300;
  bool found = false;
  for (int WO = 1; WO <= 8; WO *= 2) {
    if (WO > 1 && (a.O + kBN - 1) / kBN < WO) break;
    if ((WO * kBN) % a.G != 0) continue;
    const int WP = kWaves / WO;
    const int64_t max_pix = static_cast<int64_t>(WP) * kMT * 16;
    Params pl{};
    pl.WO = WO;
    pl.WP = WP;
    pl.taps = taps;
    pl.nob = static_cast<int32_t>((a.O + WO * kBN - 1) / (WO * kBN));
    for (int64_t len = 1; len <= (rows ? max_pix / 16 : 64); ++len) {
      int64_t parts, pix_per_part;
      if (rows) {
        pix_per_part = len * 16;
        parts = (a.N + pix_per_part - 1) / pix_per_part;
        pl.part_len = static_cast<int32_t>(pix_per_part);
        pl.patch_pix = static_cast<int32_t>(pix_per_part);
        pl.patch_cols = 0;
      } else {
        const int64_t RH = len;
        if (RH > a.geom.Ho) break;
        pix_per_part = RH * a.geom.Wo;
        if (pix_per_part > max_pix) break;
        pl.row_parts = static_cast<int32_t>((a.geom.Ho + RH - 1) / RH);
        parts = a.B * pl.row_parts;
        pl.part_len = static_cast<int32_t>(RH);
        pl.patch_cols = (a.geom.Wo - 1) * a.geom.sw + a.geom.KW;
        const int32_t prow = static_cast<int32_t>((RH - 1) * a.geom.sh + a.geom.KH);
        pl.patch_pix = prow * pl.patch_cols;
      }
      const int64_t wgs = parts * pl.nob;
      const int64_t per_cu = (wgs + 255) / 256;
      const int64_t tiles = (pix_per_part + 15) / 16;
      const int64_t tiles_per_wave = (tiles + WP - 1) / WP;  // instantiated: 1..4
      // MFMA load of the busiest SIMD: waves w and w+4 share one SIMD
      int64_t simd_tiles = 0;
      for (int w = 0; w < kWaves / 2; ++w) {
        int64_t t2 = 0;
        for (int ww = w; ww < kWaves; ww += kWaves / 2) {
          const int64_t wpp = ww / WO;
          t2 += tiles > wpp ? (tiles - wpp + WP - 1) / WP : 0;
        }
        simd_tiles = t2 > simd_tiles ? t2 : simd_tiles;
      }
      const double store = static_cast<double>(pix_per_part) * WO * kBN * ysz / 13.0;
      for (int32_t cinb = 512; cinb >= kKS; cinb /= 2) {
        if (Cin % cinb) continue;
        const double mfma_chunk = static_cast<double>(simd_tiles) * taps * (cinb / kKS) * 4.0 * 16.0;
        for (int32_t wres = 1; wres >= 0; --wres) {
          for (int32_t npb = 1; npb <= 2; ++npb) {
            Params t = pl;
            if (!layout(t, cinb, Cin, wres, npb, a.G, a.K)) continue;
            const double cost = static_cast<double>(per_cu) * model_cycles(t, mfma_chunk, store, a.K);
            if (cost < best_cost) {
              best_cost = cost;
              best = t;
              const int64_t parts8 = (parts + kXcds - 1) / kXcds * kXcds;
              best.fd_nob = make_fastdiv(static_cast<uint32_t>(best.nob));
              best.mt = static_cast<int32_t>(tiles_per_wave);
              grid = static_cast<uint32_t>(parts8 * best.nob);
              found = true;
            }
          }
        }
      }
    }
  }
  return found;
}

// Pointers, extents and geometry of one call (the plan fields are already set).
void fill_params(const ProductArgs& a, Params& p) {
  p.X = static_cast<const uint16_t*>(a.X);
  p.vals = static_cast<const uint16_t*>(a.vals);
  p.idx = a.idx;
  p.scale = a.scale;
  p.bias = a.bias;
  p.residual = a.residual;
  p.Y = a.Y;
  const int64_t ysz = a.y_t == DType::F32 ? 4 : 2;
  p.y_bytes = static_cast<uint32_t>(a.N * a.O * ysz);
  p.packed_n = static_cast<uint32_t>((a.O / a.G) * a.K * a.C);
  p.N = static_cast<int32_t>(a.N);
  p.C = static_cast<int32_t>(a.C);
  p.O = static_cast<int32_t>(a.O);
  p.G = a.G;
  p.K = a.K;
  p.relu = a.relu;
  ConvGeom g = a.geom;
  int64_t x_elems, bimg = a.B;
  if (!a.conv) {  // FC: rows of X are the "pixels" of a 1x1 convolution
    g = ConvGeom{1, 1, static_cast<int32_t>(a.C), 1, 1, 1, 1, 0, 0, 1, 1};
    bimg = 1;
    x_elems = a.N * a.C;
  } else {
    x_elems = a.B * static_cast<int64_t>(a.geom.H) * a.geom.W * a.geom.Cin;
  }
  p.x_bytes = static_cast<uint32_t>(x_elems * 2);
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
  p.Bimg = static_cast<int32_t>(bimg);
  p.strided = (g.sh != 1 || g.sw != 1) ? 1 : 0;
  p.fd_rparts = make_fastdiv(static_cast<uint32_t>(p.row_parts > 0 ? p.row_parts : 1));
  p.fd_wo = make_fastdiv(static_cast<uint32_t>(g.Wo));
  p.fd_pcols = make_fastdiv(static_cast<uint32_t>(p.patch_cols > 0 ? p.patch_cols : 1));
  p.fd_howo = make_fastdiv(static_cast<uint32_t>(g.Ho * g.Wo));
  p.kw_mul = static_cast<uint32_t>((1u << 20) / static_cast<uint32_t>(g.KW) + 1);
}

template <typename YT, bool RECT, int MT>
hipError_t launch_yrm(const Params& p, uint32_t grid, hipStream_t s) {
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&dense_tile_kernel<YT, RECT, MT>), hipFuncAttributeMaxDynamicSharedMemorySize,
      kLdsMax);
  if (attr != hipSuccess) return attr;
  size_t lds = static_cast<size_t>(p.nwb) * p.w_bytes + static_cast<size_t>(p.npb) * p.p_bytes +
               2 * static_cast<size_t>(p.s_bytes);
  const size_t staging = static_cast<size_t>(kWaves) * MT * 16 * kStPitch;  // epilogue reuses the LDS
  if (lds < staging) lds = staging;
  hipLaunchKernelGGL((dense_tile_kernel<YT, RECT, MT>), dim3(grid), dim3(kThreads), lds, s, p);
  return hipGetLastError();
}

template <typename YT, bool RECT>
hipError_t launch_yr(const Params& p, uint32_t grid, hipStream_t s) {
  switch (p.mt) {
    case 1: return launch_yrm<YT, RECT, 1>(p, grid, s);
    case 2: return launch_yrm<YT, RECT, 2>(p, grid, s);
    case 3: return launch_yrm<YT, RECT, 3>(p, grid, s);
    default: return launch_yrm<YT, RECT, 4>(p, grid, s);
  }
}

}  // namespace

bool dense_tile_supports(const ProductArgs& a) {
  if (a.x_t != DType::BF16 || a.val_t != DType::BF16) return false;
  if (a.G < 1 || kBN % a.G != 0 || a.O % 4 != 0) return false;
  const int64_t Cin = a.conv ? a.geom.Cin : a.C;
  if (Cin % kKS != 0) return false;
  // every buffer offset and index is 32-bit and must stay below the
  // out-of-range marker
  const int64_t x_elems = a.conv ? a.B * static_cast<int64_t>(a.geom.H) * a.geom.W * a.geom.Cin : a.N * a.C;
  const int64_t y_bytes = a.N * a.O * (a.y_t == DType::F32 ? 4 : 2);
  const int64_t p_bytes = (a.O / a.G) * a.K * a.C * 2;
  const int64_t lim = static_cast<int64_t>(kOOB);
  // (the loaders walk signed byte offsets that may pass the last image by
  // a few rows of padding: keep X well below the limit)
  if (x_elems * 2 >= lim / 2 || y_bytes >= lim || p_bytes >= lim) return false;
  Params pl;
  uint32_t grid;
  return make_plan(a, pl, grid);
}

hipError_t launch_dense_tile(const ProductArgs& a, hipStream_t s) {
  Params p{};
  uint32_t grid = 0;
  if (!make_plan(a, p, grid)) return hipErrorInvalidConfiguration;
  fill_params(a, p);
  const bool rect = !is_rows_mode(a);
  if (a.y_t == DType::BF16)
    return rect ? launch_yr<bf16_t, true>(p, grid, s) : launch_yr<bf16_t, false>(p, grid, s);
  return rect ? launch_yr<float, true>(p, grid, s) : launch_yr<float, false>(p, grid, s);
}

}  // namespace cci
