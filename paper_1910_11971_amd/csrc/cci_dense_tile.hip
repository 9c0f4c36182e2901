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
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kThreads = 512;
constexpr int kWaves = 8;          // two per SIMD: one wave's stalls are the other's MFMA slots
constexpr int kBN = 64;          // outputs per wave
constexpr int kKS = 32;          // reduction columns per MFMA k-step
constexpr int kMT = 4;           // max 16-pixel tiles per wave
constexpr int kBPad = 8;         // weight-tile row padding (bf16 elements)
constexpr int kXcds = 8;
constexpr int kLdsMax = 160 * 1024;
constexpr int kDmaMax = 10;      // patch DMA instructions per thread per chunk
constexpr int kRowMax = 4;       // packed rows per thread per chunk (expansion)
constexpr uint32_t kOOB = 0x80000000u;  // buffer offset that reads as zero / drops a store
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer descriptor word 3 (gfx9 family)

// Division by a launch-constant divisor d >= 1: floor(n / d) = umulhi(n, m)
// with m = floor(2^32 / d) + 1, exact for n * d < 2^32 (d == 1: n itself).
struct FastDiv {
  uint32_t d, m;
};
__host__ __device__ inline FastDiv make_fastdiv(uint32_t d) {
  return FastDiv{d, d > 1 ? static_cast<uint32_t>((uint64_t(1) << 32) / d + 1) : 0u};
}
__device__ __forceinline__ uint32_t fdiv(uint32_t n, FastDiv f) {
  return f.d == 1 ? n : __umulhi(n, f.m);
}

struct Plan {
  int32_t rect;        // 1: k x k patch; 0: one patch pixel per output pixel
  int32_t WO, WP;      // wave arrangement (WO * WP == 8)
  int32_t nob;         // output super-blocks of WO*64 outputs
  int64_t parts;       // pixel partitions (multiple of kXcds)
  int64_t part_len;    // rows mode: output pixels per partition; rect: output rows (RH)
  int32_t row_parts;   // rect: partitions per image
  int32_t cinb;        // channels per chunk (power of two, multiple of 32)
  int32_t lg_cpp;      // log2(cinb / 8): 16-byte data chunks per patch pixel
  int32_t lg_ksteps;   // log2(cinb / 32)
  int32_t nchunks;
  int32_t taps;
  int32_t patch_cols;  // rect: staged input columns
  int32_t patch_pix;   // staged pixels per chunk
  int32_t b_pitch;     // bf16 elements per weight-tile row
  int32_t b_bytes;     // bytes of one weight tile (WO*64 rows)
  int32_t buf_bytes;   // weight tile + patch
  int32_t nbuf;        // 1 or 2
  int32_t mt;          // 16-pixel tiles per wave (compile-time instantiation)
  FastDiv fd_wo;       // output width (rect)
  FastDiv fd_pcols;    // patch columns (rect)
  FastDiv fd_pps;      // 16-byte slots per patch pixel (cpp + 1: one pad slot)
  FastDiv fd_k;        // K
  FastDiv fd_ncols8;   // 8-column blocks per weight-tile row
  FastDiv fd_kw;       // KW
};

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t v) { return __builtin_bit_cast(bf16x8_t, v); }


// Patch layout: pixel q occupies cpp + 1 consecutive 16-byte slots (cpp
// data chunks and one pad slot).  The odd slot pitch spreads 8 consecutive
// pixels reading the same chunk over all 32 banks, and makes the operand
// address of any tap a single add.
template <typename YT, bool RECT, int MT>
__global__ __launch_bounds__(kThreads) void dense_tile_kernel(
    const uint16_t* __restrict__ X, uint32_t x_bytes, int64_t N, int64_t C, ConvGeom g, int32_t Bimg,
    const uint16_t* __restrict__ vals, const uint8_t* __restrict__ idx, uint32_t packed_n, int64_t O,
    int32_t G, int32_t K, Epilogue<YT> ep, YT* __restrict__ Y, Plan pl) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  constexpr uint32_t ysz = sizeof(YT);

  // ---- workgroup -> (pixel partition, output super-block), XCD-aware ----
  const int64_t id = blockIdx.x;
  const int64_t jid = id / kXcds;
  const int32_t ob = static_cast<int32_t>(jid % pl.nob);
  const int64_t part = (jid / pl.nob) * kXcds + id % kXcds;

  int32_t npix;
  int64_t P0 = 0;
  int32_t b_img = 0, oh0 = 0;
  if constexpr (RECT) {
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

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wo = wave % pl.WO;
  const int wp = wave / pl.WO;
  const int lrow = lane & 15;
  const int lk = lane >> 4;
  const int cpp = 1 << pl.lg_cpp;
  const int pps = cpp + 1;
  const int64_t o_wave = (static_cast<int64_t>(ob) * pl.WO + wo) * kBN;
  // Tiles wp, wp+WP, ... belong to this wave; only the last of its MT tile
  // slots can be empty (then its MFMAs are skipped).
  const bool last_tile = (wp + (MT - 1) * pl.WP) * 16 < npix;

  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(X), (short)0, static_cast<int>(x_bytes), kRsrcWord3);
  const uint32_t y_bytes = static_cast<uint32_t>(N * O) * ysz;
  const __amdgpu_buffer_rsrc_t yr =
      __builtin_amdgcn_make_buffer_rsrc(Y, (short)0, static_cast<int>(y_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<YT*>(ep.residual), (short)0, ep.residual ? static_cast<int>(y_bytes) : 0, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(vals), (short)0, static_cast<int>(packed_n * 2u), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t ir = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(idx), (short)0, static_cast<int>(packed_n), kRsrcWord3);

  // ---- per-lane tile geometry: patch pixel of tap (0,0), output byte offset ----
  int32_t qbase[MT];
  uint32_t yoff[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int32_t p = (wp + mt * pl.WP) * 16 + lrow;
    const bool valid = p < npix;
    const int32_t pc = valid ? p : 0;  // idle lanes read pixel 0 and store nothing
    int64_t n;
    if constexpr (RECT) {
      const int32_t r = static_cast<int32_t>(fdiv(pc, pl.fd_wo));
      const int32_t ow = pc - r * g.Wo;
      qbase[mt] = r * g.sh * pl.patch_cols + ow * g.sw;
      n = (static_cast<int64_t>(b_img) * g.Ho + oh0 + r) * g.Wo + ow;
    } else {
      qbase[mt] = pc;
      n = P0 + pc;
    }
    // an invalid pixel's offset is >= 2^31, so adding an output offset keeps
    // it out of range (the store is dropped)
    yoff[mt] = valid ? static_cast<uint32_t>(n) * static_cast<uint32_t>(O) * ysz : kOOB;
  }

  // ---- per-lane patch DMA offsets for channel chunk 0 (branch-free) ----
  const int32_t slots = pl.patch_pix * pps;
  const int32_t ndma = slots > wave * 64 ? (slots - wave * 64 + kWaves * 64 - 1) / (kWaves * 64) : 0;
  uint32_t doff[kDmaMax];
  {
    const int32_t ih_base = oh0 * g.sh - g.ph;
    const int32_t iw_base = -g.pw;
    const uint32_t img = static_cast<uint32_t>(b_img) * static_cast<uint32_t>(g.H);
    const bool strided = g.sh != 1 || g.sw != 1;
#pragma unroll
    for (int i = 0; i < kDmaMax; ++i) {
      const int32_t s = (wave + kWaves * i) * 64 + lane;
      const int32_t q = static_cast<int32_t>(fdiv(static_cast<uint32_t>(s), pl.fd_pps));
      const int32_t c = s - q * pps;  // c == cpp: pad slot
      const bool slot_ok = s < slots && c < cpp;
      uint32_t pix;
      bool ok;
      if constexpr (RECT) {
        const int32_t pr = static_cast<int32_t>(fdiv(static_cast<uint32_t>(q), pl.fd_pcols));
        const int32_t ih = ih_base + pr;
        const int32_t iw = iw_base + (q - pr * pl.patch_cols);
        ok = slot_ok && static_cast<uint32_t>(ih) < static_cast<uint32_t>(g.H) &&
             static_cast<uint32_t>(iw) < static_cast<uint32_t>(g.W);
        pix = (img + static_cast<uint32_t>(ih)) * static_cast<uint32_t>(g.W) + static_cast<uint32_t>(iw);
      } else {
        ok = slot_ok && q < npix;
        const int64_t nn = P0 + (q < npix ? q : 0);
        int64_t pp = nn;  // FC / 1x1 stride 1: row n
        if (strided) {    // strided 1x1 (wave-uniform branch): gather the input pixel
          const int64_t hw = static_cast<int64_t>(g.Ho) * g.Wo;
          const int64_t b = nn / hw;
          const int64_t rem = nn - b * hw;
          const int64_t oh = rem / g.Wo;
          pp = (b * g.H + oh * g.sh) * g.W + (rem - oh * g.Wo) * g.sw;
        }
        pix = static_cast<uint32_t>(pp);
      }
      doff[i] = ok ? (pix * static_cast<uint32_t>(g.Cin) + 8u * static_cast<uint32_t>(c)) * 2u : kOOB;
    }
  }
  auto issue_patch = [&](int ch, int buf) {
    uint8_t* pbase = lds + buf * pl.buf_bytes + pl.b_bytes;
    const uint32_t add = static_cast<uint32_t>(ch * pl.cinb) * 2u;
#pragma unroll
    for (int i = 0; i < kDmaMax; ++i) {
      if (i < ndma)  // wave-uniform
        __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t*)(pbase + (wave + kWaves * i) * 1024), 16,
                                                 doff[i] + add, 0, 0, 0);
    }
  };

  // ---- weight-tile expansion: thread -> one 8-column block, several rows ----
  const int c8n = pl.cinb / 8;
  const int ncols8 = pl.taps * c8n;
  const int rstep = kThreads / ncols8;
  const int r0 = static_cast<int>(fdiv(threadIdx.x, pl.fd_ncols8));
  const int col8 = threadIdx.x - r0 * ncols8;
  const int tap_e = col8 >> (pl.lg_cpp);  // c8n == cpp
  const int c8 = col8 - tap_e * c8n;
  const int gpb = (pl.WO * kBN) / G;
  const int nrows = gpb * K;
  uint32_t psrc[kRowMax];   // element offset of the packed row at chunk 0 (kOOB: none)
  int32_t drow[kRowMax];    // bf16 element offset of the group's first tile row
#pragma unroll
  for (int jr = 0; jr < kRowMax; ++jr) {
    const int r = r0 + jr * rstep;
    const int gl = static_cast<int>(fdiv(r, pl.fd_k));
    const int64_t gg = static_cast<int64_t>(ob) * gpb + gl;
    const bool ok = r0 < rstep && r < nrows && gg * G < O;
    psrc[jr] = ok ? static_cast<uint32_t>((gg * K + (r - gl * K)) * C + static_cast<int64_t>(tap_e) * g.Cin + 8 * c8)
                  : kOOB;
    drow[jr] = ok ? gl * G * pl.b_pitch + tap_e * pl.cinb + 8 * c8 : -1;
  }
  auto zero_weights = [&](int buf) {
    u32x4_t* b4 = reinterpret_cast<u32x4_t*>(lds + buf * pl.buf_bytes);
    const int n16 = pl.b_bytes / 16;
    for (int e = threadIdx.x; e < n16; e += kThreads) b4[e] = u32x4_t{0u, 0u, 0u, 0u};
  };
  auto scatter_weights = [&](int ch, int buf) {
    uint16_t* bs = reinterpret_cast<uint16_t*>(lds + buf * pl.buf_bytes);
    const uint32_t add = static_cast<uint32_t>(ch * pl.cinb);
    u32x4_t v[kRowMax];
    u32x2_t ix[kRowMax];
#pragma unroll
    for (int jr = 0; jr < kRowMax; ++jr) {  // all loads first: one exposed latency
      const uint32_t e = psrc[jr] == kOOB ? kOOB : psrc[jr] + add;
      v[jr] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(vr, e == kOOB ? kOOB : e * 2u, 0, 0));
      ix[jr] = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(ir, e, 0, 0));
    }
#pragma unroll
    for (int jr = 0; jr < kRowMax; ++jr) {
      if (drow[jr] < 0) continue;
      uint16_t* dst = bs + drow[jr];
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        const uint32_t r = (ix[jr][jj >> 2] >> (8 * (jj & 3))) & 0xffu;
        const uint16_t w = static_cast<uint16_t>(v[jr][jj >> 1] >> (16 * (jj & 1)));
        if (r < static_cast<uint32_t>(G)) dst[r * pl.b_pitch + jj] = w;
      }
    }
  };

  f32x4_t acc[MT][4];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int ot = 0; ot < 4; ++ot) acc[mt][ot] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

  // ---- multiply the chunk held in buffer `buf` ----
  // Reduction steps of 32 columns run tap-major; the operand fragments of
  // step s+1 are read from LDS while the MFMAs of step s issue (two register
  // sets, statically alternated; every read is unconditional so the
  // compiler can count outstanding LDS reads exactly).
  struct Frags {
    bf16x8_t w[4];
    bf16x8_t x[MT];
  };
  // A-fragment LDS byte offset of each tile at tap (0,0), k-step 0.
  uint32_t abase[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
    abase[mt] = static_cast<uint32_t>(pl.b_bytes + (qbase[mt] * pps + lk) * 16);
  const uint32_t bbase = static_cast<uint32_t>(((wo * kBN + lrow) * pl.b_pitch + 8 * lk) * 2);
  const uint32_t kw_mul = static_cast<uint32_t>((1u << 20) / g.KW + 1);  // tap / KW for tap < 4096

  auto compute = [&](int buf) {
    const uint8_t* base = lds + buf * pl.buf_bytes;
    const int nsteps = pl.taps << pl.lg_ksteps;
    auto addr = [&](int st, uint32_t& aoff, uint32_t& boff) {
      // step -> (tap, kb) -> (kh, kw): shifts and one multiply, all scalar
      const int tap = st >> pl.lg_ksteps;
      const int kb = st & ((1 << pl.lg_ksteps) - 1);
      const int kh = static_cast<int>((static_cast<uint32_t>(tap) * kw_mul) >> 20);
      const int kw = tap - kh * g.KW;
      const int32_t dq = RECT ? kh * pl.patch_cols + kw : 0;
      aoff = static_cast<uint32_t>(dq * pps * 16 + kb * 64);
      boff = static_cast<uint32_t>((tap * pl.cinb + kb * kKS) * 2);
    };
    auto load_w = [&](uint32_t boff, Frags& f) {
#pragma unroll
      for (int ot = 0; ot < 4; ++ot)
        f.w[ot] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(base + bbase + boff + ot * 16 * pl.b_pitch * 2));
    };
    auto load_x = [&](uint32_t aoff, int mt, Frags& f) {
      f.x[mt] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(base + abase[mt] + aoff));
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

  // ---- chunk pipeline -----------------------------------------------------
  // One call site for compute() keeps the accumulators in place (no copies
  // at control-flow joins).
  issue_patch(0, 0);
  zero_weights(0);
  __syncthreads();
  scatter_weights(0, 0);
  __builtin_amdgcn_s_waitcnt(0);  // this thread's patch DMA and LDS writes landed
  __syncthreads();
  for (int ch = 0; ch < pl.nchunks; ++ch) {
    const bool dbl = pl.nbuf == 2;
    const int buf = dbl ? (ch & 1) : 0;
    const bool more = ch + 1 < pl.nchunks;
    if (dbl && more) {
      issue_patch(ch + 1, buf ^ 1);
      zero_weights(buf ^ 1);
    }
    compute(buf);
    if (more) {
      __syncthreads();  // double: zero fill done; single: buffer free
      if (!dbl) {
        issue_patch(ch + 1, 0);
        zero_weights(0);
        __syncthreads();
      }
      scatter_weights(ch + 1, dbl ? buf ^ 1 : 0);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
    }
  }

  // ---- fused epilogue: lane holds outputs o..o+3 (o = o_wave+16ot+4lk) of one pixel ----
  f32x4_t sc[4], bi[4];
  uint32_t ooff[4];
#pragma unroll
  for (int ot = 0; ot < 4; ++ot) {
    const int64_t o = o_wave + ot * 16 + 4 * lk;
    const bool ok = o < O;
    ooff[ot] = ok ? static_cast<uint32_t>(o) * ysz : kOOB;
    sc[ot] = (ep.scale && ok) ? *reinterpret_cast<const f32x4_t*>(ep.scale + o) : f32x4_t{1.f, 1.f, 1.f, 1.f};
    bi[ot] = (ep.bias && ok) ? *reinterpret_cast<const f32x4_t*>(ep.bias + o) : f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {  // padding tiles have out-of-range offsets
#pragma unroll
    for (int ot = 0; ot < 4; ++ot) {
      const uint32_t off = yoff[mt] + ooff[ot];  // >= 2^31 if either is out of range
      f32x4_t y;
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) y[jj] = __builtin_fmaf(acc[mt][ot][jj], sc[ot][jj], bi[ot][jj]);
      if constexpr (ysz == 2) {
        if (ep.residual) {
          const u32x2_t rv = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(rr, off, 0, 0));
          y[0] += __uint_as_float(rv[0] << 16);
          y[1] += __uint_as_float(rv[0] & 0xffff0000u);
          y[2] += __uint_as_float(rv[1] << 16);
          y[3] += __uint_as_float(rv[1] & 0xffff0000u);
        }
        if (ep.relu) {
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) y[jj] = y[jj] > 0.0f ? y[jj] : (y[jj] != y[jj] ? y[jj] : 0.0f);
        }
        // v_cvt_pk_bf16_f32: round to nearest even
        const bf16x2_t lo = __builtin_convertvector((f32x2_t{y[0], y[1]}), bf16x2_t);
        const bf16x2_t hi = __builtin_convertvector((f32x2_t{y[2], y[3]}), bf16x2_t);
        const u32x2_t pk = {__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
        __builtin_amdgcn_raw_buffer_store_b64(
            __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b64(yr, 0, 0, 0)), pk), yr, off, 0, 0);
      } else {
        if (ep.residual) {
          const f32x4_t rv = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, 0));
          y += rv;
        }
        if (ep.relu) {
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) y[jj] = y[jj] > 0.0f ? y[jj] : (y[jj] != y[jj] ? y[jj] : 0.0f);
        }
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(yr, 0, 0, 0)), y), yr, off, 0, 0);
      }
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

// Fill the LDS layout for a channel chunk; false if it does not fit the LDS,
// the per-thread DMA budget or the per-thread expansion budget.
bool layout(Plan& pl, int32_t cinb, int32_t Cin, int32_t nbuf, int32_t G, int32_t K) {
  pl.cinb = cinb;
  pl.lg_cpp = ilog2(cinb / 8);
  pl.lg_ksteps = ilog2(cinb / kKS);
  pl.nchunks = Cin / cinb;
  pl.b_pitch = pl.taps * cinb + kBPad;
  pl.b_bytes = pl.WO * kBN * pl.b_pitch * 2;
  const int64_t slots = static_cast<int64_t>(pl.patch_pix) * (cinb / 8 + 1);
  if (slots > static_cast<int64_t>(kDmaMax) * kThreads) return false;
  const int ncols8 = pl.taps * (cinb / 8);
  if (ncols8 > kThreads) return false;
  const int rstep = kThreads / ncols8;
  const int nrows = (pl.WO * kBN / G) * K;
  if ((nrows + rstep - 1) / rstep > kRowMax) return false;
  // the DMA writes whole 64-slot (1 KiB) blocks: round the patch up so the
  // tail of its last block stays inside this buffer
  const int64_t patch_bytes = (slots * 16 + 1023) / 1024 * 1024;
  const int64_t buf = pl.b_bytes + patch_bytes;
  if (buf * nbuf > kLdsMax) return false;
  pl.buf_bytes = static_cast<int32_t>(buf);
  pl.nbuf = nbuf;
  pl.fd_pps = make_fastdiv(cinb / 8 + 1);
  pl.fd_k = make_fastdiv(K);
  pl.fd_ncols8 = make_fastdiv(ncols8);
  return true;
}

// Choose the wave arrangement, pixel partition and channel chunk.  Costs are
// in MFMA issue slots (16 cycles) on the busiest CU (one workgroup per CU at
// a time): the MFMAs of its busiest wave, the exposed patch loads (bytes at
// one CU's share of HBM bandwidth, ~13 B/clk), the weight-tile expansion and
// a charge for re-reading activations once per extra output super-block.
bool make_plan(const ProductArgs& a, Plan& best) {
  const int32_t Cin = a.conv ? a.geom.Cin : static_cast<int32_t>(a.C);
  const bool rows = is_rows_mode(a);
  const int32_t taps = a.conv ? a.geom.KH * a.geom.KW : 1;
  double best_cost = 1e300;
  bool found = false;
  for (int WO = 1; WO <= 8; WO *= 2) {
    if (WO > 1 && (a.O + kBN - 1) / kBN < WO) break;
    if ((WO * kBN) % a.G != 0) continue;
    const int WP = kWaves / WO;
    const int64_t max_pix = static_cast<int64_t>(WP) * kMT * 16;
    Plan pl{};
    pl.rect = rows ? 0 : 1;
    pl.WO = WO;
    pl.WP = WP;
    pl.taps = taps;
    pl.fd_kw = make_fastdiv(a.conv ? a.geom.KW : 1);
    pl.fd_wo = make_fastdiv(a.conv ? a.geom.Wo : 1);
    pl.nob = static_cast<int32_t>((a.O + WO * kBN - 1) / (WO * kBN));
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
        pl.fd_pcols = make_fastdiv(pl.patch_cols);
        const int32_t prow = static_cast<int32_t>((RH - 1) * a.geom.sh + a.geom.KH);
        pl.patch_pix = prow * pl.patch_cols;
      }
      double cbest = 1e300;
      Plan pbest{};
      for (int32_t cinb = 512; cinb >= kKS; cinb /= 2) {
        if (Cin % cinb) continue;
        for (int32_t nbuf = 1; nbuf <= 2; ++nbuf) {
          Plan t = pl;
          if (nbuf == 2 && Cin / cinb < 2) continue;
          if (!layout(t, cinb, Cin, nbuf, a.G, a.K)) continue;
          const double load = t.patch_pix * static_cast<double>(cinb) * 2.0 / 208.0;
          const double exposed = nbuf == 2 ? load : load * t.nchunks;
          const double expand = t.nchunks * (t.b_bytes / 2048.0 + 16.0);
          const double c = exposed + expand;
          if (c < cbest) {
            cbest = c;
            pbest = t;
          }
        }
      }
      if (cbest >= 1e299) continue;
      const int64_t wgs = parts * pbest.nob;
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
      const double mfma = static_cast<double>(simd_tiles) * taps * (Cin / kKS) * 4.0;
      const double reread = (pbest.nob - 1) * static_cast<double>(pix_per_part) * taps * Cin * 2.0 / 4096.0 / 16.0;
      const double cost = static_cast<double>(per_cu) * (mfma + cbest + reread);
      if (cost < best_cost) {
        best_cost = cost;
        best = pbest;
        best.parts = (parts + kXcds - 1) / kXcds * kXcds;
        best.mt = static_cast<int32_t>(tiles_per_wave);
        found = true;
      }
    }
  }
  return found;
}

template <typename YT, bool RECT, int MT>
hipError_t launch_yrm(const ProductArgs& a, const Plan& pl, hipStream_t s) {
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&dense_tile_kernel<YT, RECT, MT>), hipFuncAttributeMaxDynamicSharedMemorySize,
      kLdsMax);
  if (attr != hipSuccess) return attr;
  const size_t lds = static_cast<size_t>(pl.buf_bytes) * pl.nbuf;
  const dim3 grid(static_cast<uint32_t>(pl.parts * pl.nob));
  Epilogue<YT> ep{a.scale, a.bias, static_cast<const YT*>(a.residual), a.relu};
  ConvGeom g = a.geom;
  int32_t Bimg = static_cast<int32_t>(a.B);
  int64_t x_elems;
  if (!a.conv) {  // FC: rows of X are the "pixels" of a 1x1 convolution
    g = ConvGeom{1, 1, static_cast<int32_t>(a.C), 1, 1, 1, 1, 0, 0, 1, 1};
    Bimg = 1;
    x_elems = a.N * a.C;
  } else {
    x_elems = a.B * static_cast<int64_t>(a.geom.H) * a.geom.W * a.geom.Cin;
  }
  const uint32_t packed_n = static_cast<uint32_t>((a.O / a.G) * a.K * a.C);
  hipLaunchKernelGGL((dense_tile_kernel<YT, RECT, MT>), grid, dim3(kThreads), lds, s,
                     static_cast<const uint16_t*>(a.X), static_cast<uint32_t>(x_elems * 2), a.N, a.C, g, Bimg,
                     static_cast<const uint16_t*>(a.vals), a.idx, packed_n, a.O, a.G, a.K, ep,
                     static_cast<YT*>(a.Y), pl);
  return hipGetLastError();
}

template <typename YT, bool RECT>
hipError_t launch_yr(const ProductArgs& a, const Plan& pl, hipStream_t s) {
  switch (pl.mt) {
    case 1: return launch_yrm<YT, RECT, 1>(a, pl, s);
    case 2: return launch_yrm<YT, RECT, 2>(a, pl, s);
    case 3: return launch_yrm<YT, RECT, 3>(a, pl, s);
    default: return launch_yrm<YT, RECT, 4>(a, pl, s);
  }
}

template <typename YT>
hipError_t launch_y(const ProductArgs& a, const Plan& pl, hipStream_t s) {
  return pl.rect ? launch_yr<YT, true>(a, pl, s) : launch_yr<YT, false>(a, pl, s);
}

}  // namespace

bool dense_tile_supports(const ProductArgs& a) {
  if (a.x_t != DType::BF16 || a.val_t != DType::BF16) return false;
  if (a.G < 1 || kBN % a.G != 0 || a.O % 4 != 0) return false;
  const int64_t Cin = a.conv ? a.geom.Cin : a.C;
  if (Cin % kKS != 0) return false;
  // every buffer offset is 32-bit and must stay below the out-of-range marker
  const int64_t x_elems = a.conv ? a.B * static_cast<int64_t>(a.geom.H) * a.geom.W * a.geom.Cin : a.N * a.C;
  const int64_t y_bytes = a.N * a.O * (a.y_t == DType::F32 ? 4 : 2);
  const int64_t p_bytes = (a.O / a.G) * a.K * a.C * 2;
  const int64_t lim = static_cast<int64_t>(kOOB);
  if (x_elems * 2 >= lim || y_bytes >= lim || p_bytes >= lim) return false;
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
