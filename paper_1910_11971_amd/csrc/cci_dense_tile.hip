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
constexpr int kBN = 64;            // outputs per wave
constexpr int kKS = 32;            // reduction columns per MFMA k-step
constexpr int kMT = 4;             // max 16-pixel tiles per wave
constexpr int kBPad = 8;           // weight-tile row padding (bf16 elements)
constexpr int kXcds = 8;
constexpr int kLdsMax = 160 * 1024;
constexpr int kDmaMax = 10;        // patch DMA instructions per thread per chunk
constexpr int kRowMax = 4;         // packed rows per thread per chunk (expansion)
constexpr int kPackedOps = 2 * kRowMax;  // vector loads of one chunk's packed rows
constexpr uint32_t kOOB = 0x80000000u;   // buffer offset that reads as zero / drops a store
constexpr int kRsrcWord3 = 0x00020000;   // raw buffer descriptor word 3 (gfx9 family)

// Division by a launch-constant divisor d >= 1: floor(n / d) = umulhi(n, m)
// with m = floor(2^32 / d) + 1, exact for n * d < 2^32.  d == 1 has m = 0 and
// an all-ones `one` mask that passes n through, so there is no branch.
struct FastDiv {
  uint32_t d, m, one;
};
__host__ __device__ inline FastDiv make_fastdiv(uint32_t d) {
  return FastDiv{d, d > 1 ? static_cast<uint32_t>((uint64_t(1) << 32) / d + 1) : 0u, d > 1 ? 0u : ~0u};
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
  // plan
  int32_t WO, WP;       // wave arrangement (WO * WP == 8)
  int32_t nob;          // output super-blocks of WO*64 outputs
  int32_t part_len;     // rows mode: output pixels per partition; rect: output rows (RH)
  int32_t row_parts;    // rect: partitions per image
  int32_t cinb;         // channels per chunk (power of two, multiple of 32)
  int32_t lg_cpp;       // log2(cinb / 8): 16-byte data chunks per patch pixel
  int32_t lg_ksteps;    // log2(cinb / 32)
  int32_t nchunks, taps;
  int32_t patch_cols;   // rect: staged input columns
  int32_t patch_pix;    // staged pixels per chunk
  int32_t b_pitch;      // bf16 elements per weight-tile row
  int32_t b_bytes;      // bytes of one weight tile (WO*64 rows)
  int32_t buf_bytes;    // weight tile + patch region
  int32_t nbuf;         // 1 or 2
  int32_t ncols8;       // 8-column blocks per weight-tile row
  int32_t rstep;        // expansion: packed rows apart between one thread's rows
  int32_t nrows;        // packed rows of one output super-block
  int32_t mt;           // 16-pixel tiles per wave (compile-time instantiation)
  FastDiv fd_nob, fd_rparts, fd_wo, fd_pcols, fd_pps, fd_k, fd_ncols8, fd_howo;
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
  const int wo = wave % p.WO;
  const int wp = wave / p.WO;
  const int lrow = lane & 15;
  const int lk = lane >> 4;
  const int cpp = 1 << p.lg_cpp;
  const int pps = cpp + 1;
  const int32_t o_wave = (ob * p.WO + wo) * kBN;
  // Tiles wp, wp+WP, ... belong to this wave; only the last of its MT tile
  // slots can be empty (then its MFMAs are skipped).
  const bool last_tile = (wp + (MT - 1) * p.WP) * 16 < npix;

  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.X), (short)0, static_cast<int>(p.x_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.vals), (short)0, static_cast<int>(p.packed_n * 2u), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t ir = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(p.idx), (short)0, static_cast<int>(p.packed_n), kRsrcWord3);

  // ---- weight-tile expansion: thread -> one 8-column block, several packed rows ----
  const int r0 = static_cast<int>(fdiv(threadIdx.x, p.fd_ncols8));
  const int col8 = threadIdx.x - r0 * p.ncols8;
  const int tap_e = col8 >> p.lg_cpp;  // 8-column blocks per tap == cpp
  const int c8 = col8 - (tap_e << p.lg_cpp);
  const int gpb = (p.WO * kBN) / p.G;
  uint32_t psrc[kRowMax];   // element offset of the packed row at chunk 0 (kOOB: none)
  int32_t drow[kRowMax];    // bf16 element offset of the row's group in the tile (-1: none)
#pragma unroll
  for (int jr = 0; jr < kRowMax; ++jr) {
    const int r = r0 + jr * p.rstep;
    const int gl = static_cast<int>(fdiv(r, p.fd_k));
    const int32_t gg = ob * gpb + gl;
    const bool ok = r0 < p.rstep && r < p.nrows && gg * p.G < p.O;
    psrc[jr] = ok ? static_cast<uint32_t>((gg * p.K + (r - gl * p.K)) * p.C + tap_e * p.Cin + 8 * c8) : kOOB;
    drow[jr] = ok ? gl * p.G * p.b_pitch + tap_e * p.cinb + 8 * c8 : -1;
  }
  struct Packed {
    u32x4_t v[kRowMax];
    u32x2_t ix[kRowMax];
  };
  // kPackedOps loads, always issued (absent rows read zeros out of range)
  auto load_packed = [&](int ch, Packed& P) {
    const uint32_t add = static_cast<uint32_t>(ch * p.cinb);
#pragma unroll
    for (int jr = 0; jr < kRowMax; ++jr) {
      const uint32_t e = psrc[jr] == kOOB ? kOOB : psrc[jr] + add;
      P.v[jr] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(vr, e == kOOB ? kOOB : e * 2u, 0, 0));
      P.ix[jr] = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(ir, e, 0, 0));
    }
  };
  auto zero_weights = [&](int buf) {
    u32x4_t* b4 = reinterpret_cast<u32x4_t*>(lds + buf * p.buf_bytes);
    const int n16 = p.b_bytes / 16;
    for (int e = threadIdx.x; e < n16; e += kThreads) b4[e] = u32x4_t{0u, 0u, 0u, 0u};
  };
  // every kept weight goes to row G*g + idx of its column (Alg. 1's target row)
  auto scatter_weights = [&](int buf, const Packed& P) {
    uint16_t* bs = reinterpret_cast<uint16_t*>(lds + buf * p.buf_bytes);
#pragma unroll
    for (int jr = 0; jr < kRowMax; ++jr) {
      if (drow[jr] < 0) continue;
      uint16_t* dst = bs + drow[jr];
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        const uint32_t r = (P.ix[jr][jj >> 2] >> (8 * (jj & 3))) & 0xffu;
        const uint16_t w = static_cast<uint16_t>(P.v[jr][jj >> 1] >> (16 * (jj & 1)));
        if (r < static_cast<uint32_t>(p.G)) dst[r * p.b_pitch + jj] = w;
      }
    }
  };

  // ---- per-lane patch DMA offsets for channel chunk 0 ----
  // Every thread issues exactly kDmaMax DMA instructions so that the
  // compiler's (and our) counts of outstanding vector-memory operations are
  // exact: slots past the wave's last one repeat that slot, rewriting the
  // same bytes with the same data.  A wave with no slot at all writes zeros
  // to its own first block, which the planner keeps inside the patch region.
  const int32_t slots = p.patch_pix * pps;
  const int32_t nd = slots > wave * 64 ? (slots - wave * 64 + kWaves * 64 - 1) / (kWaves * 64) : 0;
  const int32_t ilast = nd > 0 ? nd - 1 : 0;
  uint32_t doff[kDmaMax];
  {
    const int32_t ih_base = oh0 * p.sh - p.ph;
    const uint32_t img = static_cast<uint32_t>(b_img * p.H);
#pragma unroll
    for (int i = 0; i < kDmaMax; ++i) {
      const int32_t ie = i < ilast ? i : ilast;  // wave-uniform
      const int32_t s = (wave + kWaves * ie) * 64 + lane;
      const int32_t q = static_cast<int32_t>(fdiv(static_cast<uint32_t>(s), p.fd_pps));
      const int32_t c = s - q * pps;  // c == cpp: pad slot
      const bool slot_ok = s < slots && c < cpp;
      uint32_t pix;
      bool ok;
      if constexpr (RECT) {
        const int32_t pr = static_cast<int32_t>(fdiv(static_cast<uint32_t>(q), p.fd_pcols));
        const int32_t ih = ih_base + pr;
        const int32_t iw = q - pr * p.patch_cols - p.pw;
        ok = slot_ok && static_cast<uint32_t>(ih) < static_cast<uint32_t>(p.H) &&
             static_cast<uint32_t>(iw) < static_cast<uint32_t>(p.W);
        pix = (img + static_cast<uint32_t>(ih)) * static_cast<uint32_t>(p.W) + static_cast<uint32_t>(iw);
      } else {
        ok = slot_ok && q < npix;
        uint32_t nn = static_cast<uint32_t>(P0 + (q < npix ? q : 0));
        if (p.strided) {  // strided 1x1 (uniform branch): gather the input pixel
          const uint32_t b = fdiv(nn, p.fd_howo);
          const uint32_t rem = nn - b * static_cast<uint32_t>(p.Ho * p.Wo);
          const uint32_t oh = fdiv(rem, p.fd_wo);
          nn = (b * p.H + oh * p.sh) * p.W + (rem - oh * p.Wo) * p.sw;
        }
        pix = nn;
      }
      doff[i] = ok ? (pix * static_cast<uint32_t>(p.Cin) + 8u * static_cast<uint32_t>(c)) * 2u : kOOB;
    }
  }
  auto issue_patch = [&](int ch, int buf) {
    uint8_t* pbase = lds + buf * p.buf_bytes + p.b_bytes;
    const uint32_t add = static_cast<uint32_t>(ch * p.cinb) * 2u;
#pragma unroll
    for (int i = 0; i < kDmaMax; ++i) {
      const int32_t ie = i < ilast ? i : ilast;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t*)(pbase + (wave + kWaves * ie) * 1024), 16,
                                               doff[i] + add, 0, 0, 0);
    }
  };

  // ---- per-lane tile geometry: patch pixel of tap (0,0), output byte offset ----
  int32_t qbase[MT];
  uint32_t yoff[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int32_t px = (wp + mt * p.WP) * 16 + lrow;
    const bool valid = px < npix;
    const int32_t pc = valid ? px : 0;  // idle lanes read pixel 0 and store nothing
    uint32_t n;
    if constexpr (RECT) {
      const int32_t r = static_cast<int32_t>(fdiv(pc, p.fd_wo));
      const int32_t ow = pc - r * p.Wo;
      qbase[mt] = r * p.sh * p.patch_cols + ow * p.sw;
      n = static_cast<uint32_t>((b_img * p.Ho + oh0 + r) * p.Wo + ow);
    } else {
      qbase[mt] = pc;
      n = static_cast<uint32_t>(P0 + pc);
    }
    // an invalid pixel's offset is >= 2^31, so adding an output offset keeps
    // it out of range (the store is dropped)
    yoff[mt] = valid ? n * static_cast<uint32_t>(p.O) * ysz : kOOB;
  }

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
    abase[mt] = static_cast<uint32_t>(p.b_bytes + (qbase[mt] * pps + lk) * 16);
  const uint32_t bbase = static_cast<uint32_t>(((wo * kBN + lrow) * p.b_pitch + 8 * lk) * 2);
  const uint32_t kw_mul = static_cast<uint32_t>((1u << 20) / p.KW + 1);  // tap / KW for tap < 4096

  auto compute = [&](int buf) {
    const uint8_t* base = lds + buf * p.buf_bytes;
    const int nsteps = p.taps << p.lg_ksteps;
    auto addr = [&](int st, uint32_t& aoff, uint32_t& boff) {
      // step -> (tap, kb) -> (kh, kw): shifts and one multiply, all scalar
      const int tap = st >> p.lg_ksteps;
      const int kb = st & ((1 << p.lg_ksteps) - 1);
      const int kh = static_cast<int>((static_cast<uint32_t>(tap) * kw_mul) >> 20);
      const int kw = tap - kh * p.KW;
      const int32_t dq = RECT ? kh * p.patch_cols + kw : 0;
      aoff = static_cast<uint32_t>(dq * pps * 16 + kb * 64);
      boff = static_cast<uint32_t>((tap * p.cinb + kb * kKS) * 2);
    };
    auto load_w = [&](uint32_t boff, Frags& f) {
#pragma unroll
      for (int ot = 0; ot < 4; ++ot)
        f.w[ot] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(base + bbase + boff + ot * 16 * p.b_pitch * 2));
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
  // Chunk j's packed rows are loaded into registers before its patch DMA is
  // issued, so the expansion waits only for them (the DMA keeps streaming);
  // the DMA of chunk j is waited for just before chunk j is multiplied.
  // With two buffers, chunk j+1's loads, DMA and zero fill are issued before
  // chunk j is multiplied.  One call site for compute() keeps the
  // accumulators in place (no copies at control-flow joins).
  const bool dbl = p.nbuf == 2;
  Packed P;
  load_packed(0, P);
  issue_patch(0, 0);
  zero_weights(0);
  lds_barrier();             // zero fill visible to every wave
  scatter_weights(0, P);     // waits for the packed loads only
  if (dbl && p.nchunks > 1) {
    load_packed(1, P);
    issue_patch(1, 1);
    zero_weights(1);
    wait_vm<kPackedOps + kDmaMax>();  // chunk 0's patch landed
  } else {
    wait_vm<0>();
  }
  lds_barrier();
  for (int ch = 0; ch < p.nchunks; ++ch) {
    const int buf = dbl ? (ch & 1) : 0;
    compute(buf);
    if (ch + 1 < p.nchunks) {
      lds_barrier();  // every wave is done with `buf`; a pending zero fill is visible
      if (!dbl) {
        load_packed(ch + 1, P);
        issue_patch(ch + 1, 0);
        zero_weights(0);
        lds_barrier();
        scatter_weights(0, P);
        wait_vm<0>();
      } else {
        scatter_weights(buf ^ 1, P);
        if (ch + 2 < p.nchunks) {
          load_packed(ch + 2, P);
          issue_patch(ch + 2, buf);
          zero_weights(buf);
          wait_vm<kPackedOps + kDmaMax>();  // chunk ch+1's patch landed
        } else {
          wait_vm<0>();
        }
      }
      lds_barrier();
    }
  }

  // ---- fused epilogue: lane holds outputs o..o+3 (o = o_wave+16ot+4lk) of one pixel ----
  const __amdgpu_buffer_rsrc_t yr =
      __builtin_amdgcn_make_buffer_rsrc(p.Y, (short)0, static_cast<int>(p.y_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(p.residual), (short)0, p.residual ? static_cast<int>(p.y_bytes) : 0, kRsrcWord3);
  f32x4_t sc[4], bi[4];
  uint32_t ooff[4];
#pragma unroll
  for (int ot = 0; ot < 4; ++ot) {
    const int32_t o = o_wave + ot * 16 + 4 * lk;
    const bool ok = o < p.O;
    ooff[ot] = ok ? static_cast<uint32_t>(o) * ysz : kOOB;
    sc[ot] = (p.scale && ok) ? *reinterpret_cast<const f32x4_t*>(p.scale + o) : f32x4_t{1.f, 1.f, 1.f, 1.f};
    bi[ot] = (p.bias && ok) ? *reinterpret_cast<const f32x4_t*>(p.bias + o) : f32x4_t{0.f, 0.f, 0.f, 0.f};
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
        if (p.residual) {
          const u32x2_t rv = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(rr, off, 0, 0));
          y[0] += __uint_as_float(rv[0] << 16);
          y[1] += __uint_as_float(rv[0] & 0xffff0000u);
          y[2] += __uint_as_float(rv[1] << 16);
          y[3] += __uint_as_float(rv[1] & 0xffff0000u);
        }
        if (p.relu) {
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
        if (p.residual) {
          const f32x4_t rv = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, 0));
          y += rv;
        }
        if (p.relu) {
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
bool layout(Params& pl, int32_t cinb, int32_t Cin, int32_t nbuf, int32_t G, int32_t K) {
  pl.cinb = cinb;
  pl.lg_cpp = ilog2(cinb / 8);
  pl.lg_ksteps = ilog2(cinb / kKS);
  pl.nchunks = Cin / cinb;
  pl.b_pitch = pl.taps * cinb + kBPad;
  pl.b_bytes = pl.WO * kBN * pl.b_pitch * 2;
  const int64_t slots = static_cast<int64_t>(pl.patch_pix) * (cinb / 8 + 1);
  if (slots > static_cast<int64_t>(kDmaMax) * kThreads) return false;
  pl.ncols8 = pl.taps * (cinb / 8);
  if (pl.ncols8 > kThreads) return false;
  pl.rstep = kThreads / pl.ncols8;
  pl.nrows = (pl.WO * kBN / G) * K;
  if ((pl.nrows + pl.rstep - 1) / pl.rstep > kRowMax) return false;
  // The DMA writes whole 64-slot (1 KiB) blocks: round the patch up so the
  // tail of its last block stays inside this buffer, and keep at least one
  // block per wave (a wave without a slot writes its first block).
  int64_t patch_bytes = (slots * 16 + 1023) / 1024 * 1024;
  if (patch_bytes < kWaves * 1024) patch_bytes = kWaves * 1024;
  const int64_t buf = pl.b_bytes + patch_bytes;
  if (buf * nbuf > kLdsMax) return false;
  pl.buf_bytes = static_cast<int32_t>(buf);
  pl.nbuf = nbuf;
  pl.fd_pps = make_fastdiv(cinb / 8 + 1);
  pl.fd_k = make_fastdiv(K);
  pl.fd_ncols8 = make_fastdiv(pl.ncols8);
  return true;
}

// Choose the wave arrangement, pixel partition and channel chunk.  Costs are
// in MFMA issue slots (16 cycles) on the busiest CU (one workgroup per CU at
// a time): the MFMAs of its busiest wave, the exposed patch loads (bytes at
// one CU's share of HBM bandwidth, ~13 B/clk), the weight-tile expansion and
// a charge for re-reading activations once per extra output super-block.
bool make_plan(const ProductArgs& a, Params& best, uint32_t& grid) {
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
      double cbest = 1e300;
      Params pbest{};
      for (int32_t cinb = 512; cinb >= kKS; cinb /= 2) {
        if (Cin % cinb) continue;
        for (int32_t nbuf = 1; nbuf <= 2; ++nbuf) {
          Params t = pl;
          if (nbuf == 2 && Cin / cinb < 2) continue;
          if (!layout(t, cinb, Cin, nbuf, a.G, a.K)) continue;
          // the first chunk's patch streams under its expansion; with two
          // buffers later patches stream under the MFMAs
          const double load = t.patch_pix * static_cast<double>(cinb) * 2.0 / 208.0;
          const double expand = t.b_bytes / 2048.0 + 16.0;
          const double first = load > expand ? load : expand;
          const double rest = (t.nchunks - 1) * (nbuf == 2 ? expand * 0.5 : load + expand);
          const double c = first + rest + 8.0 * (t.nchunks - 1);
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
        const int64_t parts8 = (parts + kXcds - 1) / kXcds * kXcds;
        best.fd_nob = make_fastdiv(static_cast<uint32_t>(best.nob));
        best.mt = static_cast<int32_t>(tiles_per_wave);
        grid = static_cast<uint32_t>(parts8 * best.nob);
        found = true;
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
}

template <typename YT, bool RECT, int MT>
hipError_t launch_yrm(const Params& p, uint32_t grid, hipStream_t s) {
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&dense_tile_kernel<YT, RECT, MT>), hipFuncAttributeMaxDynamicSharedMemorySize,
      kLdsMax);
  if (attr != hipSuccess) return attr;
  const size_t lds = static_cast<size_t>(p.buf_bytes) * p.nbuf;
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
  if (x_elems * 2 >= lim || y_bytes >= lim || p_bytes >= lim) return false;
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
