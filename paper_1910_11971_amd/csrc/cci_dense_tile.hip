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
//     padding); patch and weight tile use the layouts described below, so
//     that the operand reads are (nearly) bank-conflict free;
//   - the expanded weight tile is built in LDS while the patch streams in
//     (the packed rows are staged in LDS by DMA first);
//   - with two buffers, chunk j+1 is in flight while chunk j is multiplied.
// Patch geometry: "rect" mode (k x k convolutions) stages the input rows and
// columns under a band of RH output rows; "rows" mode (FC and 1x1
// convolutions, any stride) stages one input pixel per output pixel.
// Workgroup ids are mapped so that the output blocks of one pixel range sit
// on the same XCD (they read the same activations through its L2).
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
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kThreads = 512;
constexpr int kWaves = 8;          // two per SIMD: one wave's stalls are the other's MFMA slots
constexpr int kLoadWaves = 4;      // waves 0..3 stream activations; waves 4..7 expand weights
constexpr int kRoleThreads = kLoadWaves * 64;
constexpr int kBN = 64;            // outputs per wave
constexpr int kKS = 32;            // reduction columns per MFMA k-step
constexpr int kMT = 4;             // max 16-pixel tiles per wave
constexpr int kXcds = 8;
constexpr int kLdsMax = 160 * 1024;
constexpr int kDmaMax = 20;        // patch DMA instructions per loader thread per chunk
constexpr int kDmaEarly = 2;       // of those, issued before the expanders' staging DMAs are queued
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
  int32_t ngroups;      // O / G
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
  int32_t slots;        // 16-byte patch slots per chunk
  int32_t pp;           // rect: slot pitch of a patch pixel (cpp + 1, odd)
  // rect loader walk: 16^-1 mod pp; a step of 256 slots moves dcs chunks
  // (mod pp) and dqs pixels (16 more when the chunk wraps)
  int32_t inv16, dcs, dqs;
  int32_t nkb;          // bytes of one 16-row block of a weight tile (1 KiB per 32-column k-step)
  int32_t w_bytes;      // bytes of one weight tile (WO*64 rows)
  int32_t p_bytes;      // bytes of one patch buffer
  int32_t s_bytes;      // ring: bytes of one packed-row staging buffer (0: resident)
  int32_t s_vslots;     // ring: 16-byte value slots of one staging buffer (the index slots follow
                        // at a 1 KiB boundary, s_vblk64 * 64 slots in)
  int32_t s_islots;     // ring: 16-byte index slots
  int32_t s_vblk64;     // ring: value slots rounded up to 64
  int32_t fofs;         // LDS offset of the first tile's packed-row staging
  int32_t f_vblk64;     // its value slots rounded up to 64 (the index slots follow)
  int32_t lds_bytes;    // LDS used by the operand pipeline
  int32_t ncols8;       // 8-column blocks of one expansion (whole tile or one chunk)
  int32_t nu;           // first-tile expansion units per expander lane (bound over the waves)
  int32_t lg_gpb;       // log2(groups per output super-block)
  int32_t epg;          // first tile: groups per expander wave (max(1, 16 WO / G))
  int32_t nus;          // ring: staged scatter units (packed row x 8-column block) per expander thread
  int32_t nrows;        // packed rows of one output super-block
  int32_t mt;           // 16-pixel tiles per wave (compile-time instantiation)
  uint32_t kw_mul;      // tap / KW == (tap * kw_mul) >> 20 for tap < 4096
  FastDiv fd_nob, fd_rparts, fd_wo, fd_pcols, fd_k, fd_howo;
  FastDiv fd_ncols8, fd_nc2, fd_cin8;  // staging: ncols8, ncols8 / 2; Cin / 8
  FastDiv fd_erows;     // first tile: packed rows per expander wave
  FastDiv fd_pp, fd_taps;
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
// Touch every 64-byte line of the launch arguments with one batch of
// scalar loads and a single wait.  Arguments reach a wave through the
// scalar cache, which starts each launch cold; the compiler loads them
// lazily, as values are needed, so without this each first touch of a line
// would stall the wave for its own round trip.
__device__ __forceinline__ void prefetch_args() {
  static_assert(sizeof(Params) > 6 * 64 && sizeof(Params) <= 7 * 64, "the arguments span seven lines");
  const auto ka = __builtin_amdgcn_kernarg_segment_ptr();
  uint32_t k0, k1, k2, k3, k4, k5, k6;
  asm volatile(
      "s_load_dword %0, %7, 0x0\n\ts_load_dword %1, %7, 0x40\n\ts_load_dword %2, %7, 0x80\n\t"
      "s_load_dword %3, %7, 0xc0\n\ts_load_dword %4, %7, 0x100\n\ts_load_dword %5, %7, 0x140\n\t"
      "s_load_dword %6, %7, 0x180\n\ts_waitcnt lgkmcnt(0)"
      : "=s"(k0), "=s"(k1), "=s"(k2), "=s"(k3), "=s"(k4), "=s"(k5), "=s"(k6)
      : "s"(ka)
      : "memory");
}

// LDS layouts.  A wave's 16-byte LDS read runs without bank conflicts when,
// in each half of the wave, the 32 addresses fall into distinct 16-byte
// slots modulo 512 bytes (measured on gfx950; a row pitch of an odd number
// of slots is not enough).  An MFMA operand fragment is read by lanes
// (row = lane % 16, k-chunk = lane / 16), so:
//   - weight tile: element (o, k) at byte
//       ((o / 16) * NK + k / 32) * 1024 + (k / 8 % 4) * 256 + (o % 16) * 16 + (k % 8) * 2
//     (NK = 32-column k-steps of the tile): a fragment is 1 KiB, lane l reads
//     bytes 16 l .. 16 l + 15;
//   - rows-mode patch (FC, 1x1): pixel q, 16-byte channel chunk c at slot
//       ((q / 16) * cpp + c) * 16 + q % 16
//     (cpp = chunks per pixel, even): a tile's 16 pixels of one chunk are
//     256 contiguous bytes;
//   - rect-mode patch (k x k): slot (cpp + 1) q + 16 c.  The address is
//     linear in the pixel, so every tap reads at a uniform offset from the
//     tap-(0,0) address; with an odd pixel pitch and chunks 16 slots apart
//     the 16 pixels x 2 chunks of a half-wave land in distinct slots
//     modulo 512 bytes (only tiles that straddle an output row can see a
//     two-way conflict).  A DMA instruction still fetches runs of a few
//     neighbouring pixels (its rate falls with the number of distinct
//     cache lines it touches); one slot in cpp + 1 is a hole.
template <typename YT, bool RECT, int MT>
__global__ __launch_bounds__(kThreads) void dense_tile_kernel(Params p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  prefetch_args();
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
  const int32_t wofs_patch = p.nwb * p.w_bytes;  // LDS offset of patch buffer 0
  // weight-tile byte offsets of row o and of 8-column block col8 (they add)
  auto rowaddr = [&](int o) { return (o >> 4) * p.nkb + (o & 15) * 16; };
  auto coladdr = [](int col8) { return (col8 >> 2) * 1024 + (col8 & 3) * 256; };
  const int32_t nkbm = p.nkb - 256;  // rowaddr(r) == 16 r + (r >> 4) * nkbm

  // ---- expanders: first weight tile ---------------------------------------
  // Packed rows are staged in LDS row-major: value slot r * ncols8 + j holds
  // the 8 values of packed row r in column block j of the expansion, index
  // slot r * ncols8 / 2 + j / 2 the 16 indices of blocks j and j + 1 (ncols8
  // is even).  The ring stages one chunk in tile order (block j is tile
  // column block j); the first tile is staged in memory order (block j is
  // source columns 8 j .. 8 j + 7), so each packed row is one contiguous
  // copy.
  // The resident tile (every chunk), or the ring's chunk-0 tile, is built by
  // the four expander waves from a staging area at fofs.  Expander wave e
  // owns groups [e * epg, (e + 1) * epg) -- tile rows [16 WO e, 16 WO (e + 1))
  // when G <= 16 WO, else one group (waves past the last group idle) --
  // i.e. whole groups and a contiguous run of packed rows: it DMAs those
  // rows, zero-fills its rows' fragments, then writes every kept weight of
  // them; program order alone puts its zero fill before its writes, and no
  // other wave touches them.
  // Rolled loops keep this code short: it runs once per workgroup, from a
  // cold instruction cache.
  const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.vals), (short)0, static_cast<int>(p.packed_n * 2u), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t ir = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(p.idx), (short)0, static_cast<int>(p.packed_n), kRsrcWord3);
  const int gpb = 1 << p.lg_gpb;  // groups per output super-block
  // groups that exist (the last super-block may be partial)
  const int glim = p.ngroups - ob * gpb < gpb ? p.ngroups - ob * gpb : gpb;
  const int rlim = glim * p.K;               // packed rows that exist
  const int32_t rowbase = ob * gpb * p.K;    // first packed row of the super-block
  const uint32_t gmask = static_cast<uint32_t>(p.G - 1);
  const int ewave = wave - kLoadWaves;       // expander index (negative on loaders)
  // packed rows of this expander wave (none on waves past the last group)
  const int erows = ewave * p.epg < gpb ? p.epg * p.K : 0;
  const int er0 = ewave * p.epg * p.K;       // its first packed row
  // tile column block of first-tile staged block j (memory order)
  auto first_col8 = [&](int j) {
    const int tap = static_cast<int>(fdiv(j, p.fd_cin8));
    const int cin8 = j - tap * (p.Cin >> 3);
    return ((cin8 >> p.lg_cpp) * p.taps + tap) * cpp + (cin8 & (cpp - 1));
  };
  // write staged packed-row segment (row r, tile column block col8) into the
  // tile at tb: every kept weight goes to row G*g + idx (Alg. 1's target
  // row); with K == G every row is kept in ascending order and the segment
  // is copied whole.  sv / si: byte offsets of its value and index slots.
  auto scatter_unit = [&](uint8_t* tb, const uint8_t* stg, int sv, int si, int col8, int r) {
    const int gl = static_cast<int>(fdiv(r, p.fd_k));
    uint8_t* dst = tb + rowaddr(gl * p.G) + coladdr(col8);
    const u32x4_t v = *reinterpret_cast<const u32x4_t*>(stg + sv);
    if (p.K == p.G) {
      *reinterpret_cast<u32x4_t*>(dst + rowaddr(r - gl * p.K)) = v;
      return;
    }
    const u32x2_t ix = *reinterpret_cast<const u32x2_t*>(stg + si);
    // The upper half-wave writes the segment's elements in the order
    // 4..7, 0..3 (element t ^ 4 at step t): two half-waves then hit
    // different bank words with each store.
    const bool hi = lane >= 32;
    const u32x4_t vr = hi ? u32x4_t{v[2], v[3], v[0], v[1]} : v;
    const u32x2_t ixr = hi ? u32x2_t{ix[1], ix[0]} : ix;
    uint8_t* const d_lo = dst + (hi ? 8 : 0);  // steps 0..3: byte 2 (t ^ 4 h)
    uint8_t* const d_hi = dst - (hi ? 8 : 0);  // steps 4..7
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      // idx: row in the group (< G, a power of two on this path; the mask
      // keeps a corrupt index inside its own group)
      const int32_t rr = static_cast<int32_t>((ixr[t >> 2] >> (8 * (t & 3))) & gmask);
      const uint16_t w = static_cast<uint16_t>(vr[t >> 1] >> (16 * (t & 1)));
      *reinterpret_cast<uint16_t*>((t < 4 ? d_lo : d_hi) + (rr << 4) + (rr >> 4) * nkbm + 2 * t) = w;
    }
  };
  // source element of staged block j of packed row r, chunk ch (ring: tile
  // order; the resident first tile uses memory order, see stage_first)
  auto ring_src = [&](int r, int j, int ch) -> uint32_t {
    return __umul24(rowbase + r, p.C) + __umul24(j >> p.lg_cpp, p.Cin) + ch * p.cinb + 8 * (j & (cpp - 1));
  };
  // this wave's staging DMAs (lanes past the end of its range stay idle).
  // Resident: its packed rows are one contiguous run of memory, copied as
  // is; ring: the chunk-0 columns of each row.
  auto stage_first = [&]() {
    const int nv = erows * p.ncols8;
    const int32_t rows_ok = rlim - er0;  // rows of this wave that exist
    uint8_t* const vdst = lds + p.fofs + er0 * p.ncols8 * 16;
    uint8_t* const idst = lds + p.fofs + (p.f_vblk64 + (er0 * p.ncols8 >> 1)) * 16;
    if (p.wres) {  // one contiguous run: byte offsets step by 16 per slot
      const int nok = rows_ok * p.ncols8;  // value slots of rows that exist
      const uint32_t v0 = static_cast<uint32_t>(__umul24(rowbase + er0, p.C)) * 2u + 16u * lane;
      const uint32_t i0 = static_cast<uint32_t>(__umul24(rowbase + er0, p.C)) + 16u * lane;
#pragma unroll 1
      for (int b = 0; b < nv; b += 64)
        if (b + lane < nv)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_void_t*)(vdst + b * 16), 16,
                                                   b + lane < nok ? v0 + 16u * b : kOOB, 0, 0, 0);
#pragma unroll 1
      for (int b = 0; b < (nv >> 1); b += 64)
        if (b + lane < (nv >> 1))
          __builtin_amdgcn_raw_ptr_buffer_load_lds(ir, (lds_void_t*)(idst + b * 16), 16,
                                                   b + lane < (nok >> 1) ? i0 + 16u * b : kOOB, 0, 0, 0);
      return;
    }
#pragma unroll 1
    for (int b = 0; b < nv; b += 64) {
      const int sl = b + lane;
      const int rl = static_cast<int>(fdiv(sl, p.fd_ncols8));
      const uint32_t off = rl < rows_ok ? ring_src(er0 + rl, sl - rl * p.ncols8, 0) * 2u : kOOB;
      if (sl < nv) __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_void_t*)(vdst + b * 16), 16, off, 0, 0, 0);
    }
#pragma unroll 1
    for (int b = 0; b < (nv >> 1); b += 64) {
      const int sl = b + lane;
      const int rl = static_cast<int>(fdiv(sl, p.fd_nc2));
      const uint32_t off = rl < rows_ok ? ring_src(er0 + rl, 2 * (sl - rl * (p.ncols8 >> 1)), 0) : kOOB;
      if (sl < (nv >> 1)) __builtin_amdgcn_raw_ptr_buffer_load_lds(ir, (lds_void_t*)(idst + b * 16), 16, off, 0, 0, 0);
    }
  };
  // zero fill of this wave's tile rows (not needed when K == G: every
  // element is written), then the scatter once its staging DMAs have landed
  auto expand_first = [&]() {
    if (p.K != p.G && erows > 0) {
      // tile rows [e * epg * G, (e + 1) * epg * G): whole 16-row blocks
      const int z1 = ((ewave + 1) * p.epg * p.G >> 4) * (p.nkb >> 4);
#pragma unroll 1
      for (int z = (ewave * p.epg * p.G >> 4) * (p.nkb >> 4) + lane; z < z1; z += 64)
        *reinterpret_cast<u32x4_t*>(lds + z * 16) = u32x4_t{0u, 0u, 0u, 0u};
    }
    wait_vm<0>();
    // units row-fastest: a wave's lanes span all its groups
    const int n = erows * p.ncols8;
    const int rows_ok = rlim - er0;  // rows of this wave that exist
#pragma unroll 1
    for (int u = lane; u < n; u += 64) {
      const int j = static_cast<int>(fdiv(u, p.fd_erows)), rl = u - j * erows;
      if (rl < rows_ok) {
        const int sl = (er0 + rl) * p.ncols8 + j;  // value slot
        scatter_unit(lds, lds + p.fofs, sl * 16, (p.f_vblk64 + (sl >> 1)) * 16 + (j & 1) * 8,
                     p.wres ? first_col8(j) : j, er0 + rl);
      }
    }
  };
  if (!loader) stage_first();

  // ---- loaders: patch DMA -------------------------------------------------
  // Loader thread rt owns slots rt + 256 i (i < nd).  Rect mode: slot s
  // holds chunk s % (cpp + 1) of patch pixel s / (cpp + 1) (the last one is
  // a pad slot); rows mode: chunk (s / 16) % cpp of pixel
  // 16 * (s / (16 cpp)) + s % 16.  The source offsets of chunk 0 are
  // computed once; chunk j reuses them plus j*cinb*2.
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.X), (short)0, static_cast<int>(p.x_bytes), kRsrcWord3);
  const int32_t nd = p.slots > wave * 64 ? (p.slots - wave * 64 + kRoleThreads - 1) / kRoleThreads : 0;
  uint32_t doff[kDmaMax];
  auto dma = [&](uint32_t pofs, int i, uint32_t off) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t*)(lds + pofs + (wave + kLoadWaves * i) * 1024), 16, off,
                                             0, 0, 0);
  };
  if (loader) {
    const uint32_t cin2 = static_cast<uint32_t>(p.Cin * 2);
    // rect: slot s = pp q + 16 c.  The walk state of s = rt + 256 i --
    // chunk c = s / 16 mod pp and patch pixel q = (s - 16 c) / pp -- steps
    // by dcs chunks and dqs pixels (16 more when c wraps)
    int32_t c = 0, q = 0;
    const int32_t ih0 = oh0 * p.sh - p.ph;
    if constexpr (RECT) {
      const int32_t t = rt * p.inv16;
      c = t - static_cast<int32_t>(fdiv(static_cast<uint32_t>(t), p.fd_pp)) * p.pp;
      q = (rt - 16 * c) / p.pp;  // exact; negative before the first pixel of chunk c
    }
#pragma unroll
    for (int i = 0; i < kDmaMax; ++i) {
      if (i < nd) {
        const int32_t s = rt + kRoleThreads * i;
        bool ok;
        uint32_t off;
        if constexpr (RECT) {
          const int32_t qq = q > 0 ? q : 0;
          const int32_t pr = static_cast<int32_t>(fdiv(static_cast<uint32_t>(qq), p.fd_pcols));
          const int32_t ih = ih0 + pr, iw = qq - pr * p.patch_cols - p.pw;
          // holes (c >= cpp), pixels past the patch and out-of-image pixels
          // (the padding) read as zero
          ok = c < cpp && q >= 0 && q < p.patch_pix && static_cast<uint32_t>(ih) < static_cast<uint32_t>(p.H) &&
               static_cast<uint32_t>(iw) < static_cast<uint32_t>(p.W);
          off = __umul24(__umul24(b_img * p.H + ih, p.W) + iw, cin2) + 16 * c;
          c += p.dcs;
          const bool wrap = c >= p.pp;
          c -= wrap ? p.pp : 0;
          q += p.dqs + (wrap ? 16 : 0);
        } else {
          const int32_t q = ((s >> (4 + p.lg_cpp)) << 4) | (s & 15);  // patch pixel
          const int32_t c = (s >> 4) & (cpp - 1);                       // 16-byte chunk
          ok = s < p.slots && q < npix;
          uint32_t nn = static_cast<uint32_t>(P0 + (q < npix ? q : 0));
          if (p.strided) {  // strided 1x1 (uniform branch): gather the input pixel
            const uint32_t b = fdiv(nn, p.fd_howo);
            const uint32_t rem = nn - b * static_cast<uint32_t>(p.Ho * p.Wo);
            const uint32_t oh = fdiv(rem, p.fd_wo);
            nn = (b * p.H + oh * p.sh) * p.W + (rem - oh * p.Wo) * p.sw;
          }
          off = __umul24(nn, cin2) + 16 * c;
        }
        doff[i] = ok ? off : kOOB;
        if (i < kDmaEarly) dma(static_cast<uint32_t>(wofs_patch), i, doff[i]);
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
  // Activation operand of tile mt at tap (0,0), chunk lk of k-step 0: patch
  // pixel qb of the lane's output pixel; every later step adds a uniform
  // offset.
  uint32_t abase[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int32_t px = (wp + mt * p.WP) * 16 + lrow;
    const int32_t pc = px < npix ? px : 0;  // idle lanes read pixel 0 and store nothing
    if constexpr (RECT) {
      const int32_t r = static_cast<int32_t>(fdiv(pc, p.fd_wo));
      const int32_t qb = r * p.sh * p.patch_cols + (pc - r * p.Wo) * p.sw;
      abase[mt] = static_cast<uint32_t>((qb * p.pp + 16 * lk) * 16);
    } else {
      abase[mt] = static_cast<uint32_t>(((pc & ~15) << (4 + p.lg_cpp)) + ((pc & 15) << 4) + lk * 256);
    }
  }
  // weight operand: 16-row block 4 wo + ot, lane-linear inside the fragment
  const uint32_t bbase = static_cast<uint32_t>(wo * 4 * p.nkb + lane * 16);

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
    // step st = tap * ksteps + kb: weight k-step st of the chunk; patch
    // pixel shift dq of the tap and chunks 4 kb .. 4 kb + 3 (uniform offset)
    auto addr = [&](int st) {
      // step -> (tap, kb) -> (kh, kw): shifts and one multiply, all scalar
      const int tap = st >> p.lg_ksteps;
      const int kb = st & ((1 << p.lg_ksteps) - 1);
      if constexpr (RECT) {
        const int kh = static_cast<int>((static_cast<uint32_t>(tap) * p.kw_mul) >> 20);
        const int kw = tap - kh * p.KW;
        return static_cast<uint32_t>(((kh * p.patch_cols + kw) * p.pp + kb * 64) * 16);
      } else {
        return static_cast<uint32_t>(kb * 1024);
      }
    };
    auto load_w = [&](int st, Frags& f) {
#pragma unroll
      for (int ot = 0; ot < 4; ++ot)
        f.w[ot] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(wb + st * 1024 + ot * p.nkb));
    };
    auto load_x = [&](uint32_t aoff, int mt, Frags& f) {
      f.x[mt] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(pb + abase[mt] + aoff));
    };
    // One reduction step on `cur` while the fragments of step `nst` stream
    // into `nxt`: each tile's 4 MFMAs are followed by one LDS read, so every
    // read is issued about one step ahead of its use and at most ~12 reads
    // are outstanding (the LDS counter tracks 15).
    auto step = [&](const Frags& cur, Frags& nxt, int nst) {
      const uint32_t aoff = addr(nst);
      load_w(nst, nxt);
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
      const uint32_t aoff = addr(0);
      load_w(0, f0);
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
  // Chunk j's packed rows are DMA'd two chunks ahead into one of two staging
  // buffers (row-major, tile order); the expanders build chunk j's tile from
  // there while chunk j-1 is multiplied.
  const int32_t sofs = wofs_patch + p.npb * p.p_bytes;  // LDS offset of staging buffer 0
  // loader thread rt's staging slots: value slot rt + 256 i and index slot
  // rt + 256 i, element offsets at chunk 0 (kOOB: none)
  uint32_t pk_v[kPkMax], pk_i[kPkMax];
  if (loader && !p.wres) {
#pragma unroll
    for (int i = 0; i < kPkMax; ++i) {
      const int32_t sl = rt + kRoleThreads * i;
      const int32_t rv = static_cast<int32_t>(fdiv(static_cast<uint32_t>(sl), p.fd_ncols8));
      pk_v[i] = sl < p.s_vslots && rv < rlim ? ring_src(rv, sl - rv * p.ncols8, 0) : kOOB;
      const int32_t ri = static_cast<int32_t>(fdiv(static_cast<uint32_t>(sl), p.fd_nc2));
      pk_i[i] = sl < p.s_islots && ri < rlim ? ring_src(ri, 2 * (sl - ri * (p.ncols8 >> 1)), 0) : kOOB;
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
  // zero-filled a chunk earlier.  Unit u = (packed row u / ncols8, column
  // block u % ncols8) is staged value slot u, so the work spreads over K
  // times more threads than whole groups would.  With K == G every row is
  // kept in ascending order: a row segment is copied whole.
  // per-thread scatter units, decoded once: staged byte offsets of the
  // values and indices, tile byte offset (< 0 in su_src: none)
  int32_t su_src[kUnitMax], su_idx[kUnitMax], su_dst[kUnitMax];
  if (!loader && !p.wres) {
#pragma unroll
    for (int j = 0; j < kUnitMax; ++j) {
      const int u = rt + kRoleThreads * j;
      const int r = static_cast<int>(fdiv(u, p.fd_ncols8));
      const int col8 = u - r * p.ncols8;
      const int gl = static_cast<int>(fdiv(r, p.fd_k));
      const bool ok = j < p.nus && r < rlim;
      su_src[j] = ok ? u * 16 : -1;
      su_idx[j] = (p.s_vblk64 + (u >> 1)) * 16 + (col8 & 1) * 8;
      su_dst[j] = rowaddr(gl * p.G) + coladdr(col8) + (p.K == p.G ? rowaddr(r - gl * p.K) : 0);
    }
  }
  auto scatter_staged = [&](int wb, int sb) {
    const uint8_t* stg = lds + sofs + sb * p.s_bytes;
    uint8_t* bs = lds + wb * p.w_bytes;
#pragma unroll
    for (int j = 0; j < kUnitMax; ++j) {
      if (su_src[j] < 0) continue;
      uint8_t* dst = bs + su_dst[j];
      const u32x4_t v = *reinterpret_cast<const u32x4_t*>(stg + su_src[j]);
      if (p.K == p.G) {  // every row kept, in order: the row is copied whole
        *reinterpret_cast<u32x4_t*>(dst) = v;
        continue;
      }
      const u32x2_t ix = *reinterpret_cast<const u32x2_t*>(stg + su_idx[j]);
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        const int32_t rr = static_cast<int32_t>((ix[jj >> 2] >> (8 * (jj & 3))) & gmask);  // idx: row in the group
        const uint16_t w = static_cast<uint16_t>(v[jj >> 1] >> (16 * (jj & 1)));
        *reinterpret_cast<uint16_t*>(dst + (rr << 4) + (rr >> 4) * nkbm + 2 * jj) = w;
      }
    }
  };
  // zero fill of weight tile wb (not needed when K == G).  In the prologue
  // the loaders zero a tile with DMA from an out-of-range source offset,
  // which writes zeros into LDS without reading memory (a tile is a whole
  // number of KiB); in the loop the expanders zero a tile with plain LDS
  // stores, keeping the loaders' memory queue for the patch and staging.
  auto zero_tile = [&](int wb) {
    if (p.K == p.G) return;
    const int nblk = p.w_bytes / 1024;
    for (int b = wave; b < nblk; b += kLoadWaves)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t*)(lds + wb * p.w_bytes + b * 1024), 16, kOOB, 0, 0, 0);
  };
  auto zero_tile_lds = [&](int wb) {
    if (p.K == p.G) return;
    u32x4_t* t4 = reinterpret_cast<u32x4_t*>(lds + wb * p.w_bytes);
#pragma unroll 1
    for (int z = rt; z < (p.w_bytes >> 4); z += kRoleThreads) t4[z] = u32x4_t{0u, 0u, 0u, 0u};
  };

  // ---- chunk pipeline -----------------------------------------------------
  // Loaders stream patches through npb (1 or 2) buffers: chunk 0 from the
  // first instructions, chunk j+1 during chunk j's MFMAs.  Expanders build
  // the weight tile: once (resident), or (ring) chunk 0 from registers and
  // chunk j+1 from its staged packed rows while chunk j is multiplied, into
  // the other of two tiles.  A loader's MFMAs fill the SIMD its partner
  // expander shares while that one builds.  One barrier per chunk; one call
  // site for compute() keeps the accumulators in place.
  // The loaders issue the first kDmaEarly patch DMAs as soon as their
  // offsets are known and the rest after this barrier, by which the
  // expanders' staging DMAs are queued: issued behind the bulk of the
  // patch they would hold up the weight expansion.
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
    expand_first();
  }
  lds_barrier();
  int pb = 0;
  for (int ch = 0; ch < p.nchunks; ++ch) {
    const int wcur = ch % 3;  // ring tile of chunk ch
    const uint32_t wofs = p.wres ? static_cast<uint32_t>((ch * p.taps << p.lg_ksteps) * 1024)
                                 : static_cast<uint32_t>(wcur * p.w_bytes);
    const int nb = p.npb == 2 ? pb ^ 1 : 0;
    if (ring && ch + 1 < p.nchunks) {
      const int wnext = wcur == 2 ? 0 : wcur + 1;
      if (loader) {
        if (ch + 2 < p.nchunks) issue_packed(ch + 2, ch & 1);
      } else {
        if (ch + 2 < p.nchunks) zero_tile_lds(wnext == 2 ? 0 : wnext + 1);  // chunk ch+2's tile (last read by chunk ch-1)
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
  const int32_t cpp = cinb / 8;
  // rect: pixel-major, cpp chunks and a pad slot per pixel, rounded up to
  // the 64 slots one DMA instruction writes; rows: whole blocks of 16 pixels
  pl.pp = cpp + 1;
  pl.inv16 = 1;
  while ((16 * pl.inv16) % pl.pp != 1 % pl.pp) ++pl.inv16;
  pl.dcs = (kRoleThreads * pl.inv16) % pl.pp;
  pl.dqs = (kRoleThreads - 16 * pl.dcs) / pl.pp;  // exact
  const int64_t slots = pl.patch_cols > 0 ? (static_cast<int64_t>(pl.patch_pix - 1) * pl.pp + 16 * (cpp - 1) + 64) / 64 * 64
                                          : static_cast<int64_t>((pl.patch_pix + 15) / 16) * 16 * cpp;
  if (slots > static_cast<int64_t>(kDmaMax) * kRoleThreads) return false;
  pl.slots = static_cast<int32_t>(slots);
  const int32_t tc = pl.taps * cpp;
  pl.wres = wres;
  pl.ncols8 = wres ? pl.nchunks * tc : tc;
  pl.nkb = pl.ncols8 / 4 * 1024;
  pl.w_bytes = pl.WO * 4 * pl.nkb;
  pl.nrows = (pl.WO * kBN / G) * K;
  pl.lg_gpb = ilog2(pl.WO * kBN / G);
  // first tile: each expander wave owns epg groups, i.e. epg*K packed
  // rows x ncols8 units
  pl.epg = pl.WO * 16 >= G ? pl.WO * 16 / G : 1;
  pl.nu = (pl.epg * K * pl.ncols8 + 63) / 64;
  pl.nus = (pl.nrows * pl.ncols8 + kRoleThreads - 1) / kRoleThreads;
  if (!wres && pl.nus > kUnitMax) return false;
  pl.nwb = wres ? 1 : 3;
  pl.p_bytes = static_cast<int32_t>(slots * 16);
  pl.npb = npb;
  pl.s_bytes = pl.s_vslots = pl.s_islots = pl.s_vblk64 = 0;
  if (!wres) {  // packed-row staging: nrows x ncols8 value slots + half as many index slots
    pl.s_vslots = pl.nrows * pl.ncols8;
    pl.s_islots = pl.nrows * pl.ncols8 / 2;
    pl.s_vblk64 = (pl.s_vslots + 63) / 64 * 64;
    pl.s_bytes = (pl.s_vblk64 + (pl.s_islots + 63) / 64 * 64) * 16;
    if (pl.s_vslots > kPkMax * kRoleThreads || pl.s_islots > kPkMax * kRoleThreads) return false;
  }
  if (static_cast<int64_t>(pl.nwb) * pl.w_bytes + static_cast<int64_t>(npb) * pl.p_bytes +
          2 * static_cast<int64_t>(pl.s_bytes) > kLdsMax)
    return false;
  // first-tile staging: ring staging buffer 0; resident: the second patch
  // buffer (not in use before chunk 1 streams in) when it is large enough,
  // else the space after the patch buffers
  pl.f_vblk64 = (pl.nrows * pl.ncols8 + 63) / 64 * 64;
  const int64_t f_bytes = (pl.f_vblk64 + (pl.nrows * pl.ncols8 / 2 + 63) / 64 * 64) * 16;
  const int64_t after = static_cast<int64_t>(pl.nwb) * pl.w_bytes + static_cast<int64_t>(npb) * pl.p_bytes;
  if (!wres) {
    pl.fofs = static_cast<int32_t>(after);
  } else if (npb == 2 && f_bytes <= pl.p_bytes) {
    pl.fofs = pl.nwb * pl.w_bytes + pl.p_bytes;
  } else {
    if (after + f_bytes > kLdsMax) return false;
    pl.fofs = static_cast<int32_t>(after);
  }
  pl.lds_bytes = static_cast<int32_t>(after + 2 * static_cast<int64_t>(pl.s_bytes));
  if (pl.fofs + f_bytes > pl.lds_bytes) pl.lds_bytes = static_cast<int32_t>(pl.fofs + f_bytes);
  pl.fd_ncols8 = make_fastdiv(pl.ncols8);
  pl.fd_erows = make_fastdiv(pl.epg * K);
  pl.fd_nc2 = make_fastdiv(pl.ncols8 / 2);
  pl.fd_cin8 = make_fastdiv(Cin / 8);
  pl.fd_k = make_fastdiv(K);
  pl.fd_pp = make_fastdiv(pl.pp);
  pl.fd_taps = make_fastdiv(pl.taps);
  return true;
}

// Modelled duration (cycles) of one workgroup: a chunk's patch streams at
// kPatchBpc bytes per cycle once its buffer is free (two buffers: from the
// start of the previous chunk's MFMAs); its MFMAs start when it has
// arrived, its weights are expanded and the previous chunk is done.  The
// constants were fitted to measured times of every legal plan of 24 layer
// shapes (ResNet-50's and MobileNetV2's, the 3x3 / 1x1 / FC benchmark
// layers): the plan the model picks is on average within 5% of the fastest
// measured one (within 25% for every shape; it was 2x off for some shapes
// with the previous hand-set constants).
constexpr double kPatchBpc = 20.0;      // patch / output bytes per cycle per CU
constexpr double kUnitCycles = 400.0;   // one expansion unit (packed row segment) per expander lane
constexpr double kMfmaCycles = 20.0;    // one 16x16x32 MFMA with its operand reads
double model_cycles(const Params& t, double mfma_chunk, double store, int K) {
  const double load = t.patch_pix * static_cast<double>(t.cinb) * 2.0 / kPatchBpc;
  // expansion by the 256 expander threads: zero fill (b128 writes) and
  // K packed-row segments per unit
  const double build = t.w_bytes / 16.0 / kRoleThreads * 8.0 + t.nu * K * kUnitCycles;
  // (chunk_latency: ResNet-50's 3x3 layers' chunks were measured at 6.5-10 K
  // cycles almost independently of the part's pixel count)
  const double latency = 5633.0, barrier = 100.0, setup = 1813.0, chunk_latency = 1873.0;
  const double e_first = setup + latency + build * (t.wres ? 1 : 2);
  double arrive = setup / 2 + latency + load, done = 0.0, start = 0.0;
  double done2 = 0.0;  // done time of chunk c-2
  const int n = t.nchunks;
  for (int c = 0; c < n; ++c) {
    if (c > 0) {
      // every chunk's patch request pays a memory latency; with two patch
      // buffers it is issued when the previous chunk starts, so it hides
      // behind that chunk's MFMAs when they are long enough
      const double issue = t.npb == 2 ? start : done + barrier;
      arrive = (issue > arrive ? issue : arrive) + chunk_latency + load;
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
      const double store = static_cast<double>(pix_per_part) * WO * kBN * ysz / kPatchBpc;
      for (int32_t cinb = 512; cinb >= kKS; cinb /= 2) {
        if (Cin % cinb) continue;
        const double mfma_chunk = static_cast<double>(simd_tiles) * taps * (cinb / kKS) * 4.0 * kMfmaCycles;
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
  p.ngroups = static_cast<int32_t>(a.O / a.G);
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
  static std::atomic<int8_t> lds_set[kMaxDevices];
  const hipError_t attr =
      set_lds_limit_once(lds_set, reinterpret_cast<const void*>(&dense_tile_kernel<YT, RECT, MT>), kLdsMax);
  if (attr != hipSuccess) return attr;
  size_t lds = static_cast<size_t>(p.lds_bytes);
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
