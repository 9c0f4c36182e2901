// CCI-sparse product on the matrix cores: wide-tile plan for large FC and
// stride-1 1x1 products (implicit GEMM with X rows = pixels).
//
// The method is the dense-tile one -- each chunk of packed groups becomes a
// dense bf16 weight tile in LDS (zero fill, then every kept weight written
// to row G*g + idx of its column: the routing of Alg. 1, Sec. 3.2) that is
// multiplied on v_mfma_f32_16x16x32_bf16 -- with a work split sized for
// products large enough to fill the chip with 256 x 256 output tiles:
//   - a workgroup is four waves, one per SIMD, and owns 256 pixels x 256
//     outputs; each wave accumulates 128 pixels x 128 outputs (256 fp32 per
//     lane, in the accumulation registers), so every fragment read from LDS
//     feeds eight MFMAs, and each expanded weight tile serves 256 pixels;
//   - the reduction runs over chunks of 64 channels.  The activations of
//     chunk j+3 are DMA'd into LDS during chunk j (three buffers, each
//     refilled as soon as the chunk that used it is done); the packed
//     weights of chunk j+2 are loaded into registers during chunk j and
//     written into the second weight tile during chunk j+1; the barrier of
//     a chunk sits in its middle, after which no wave reads that chunk's
//     buffers (every fragment is already in registers), so the next chunk's
//     fragments stream in behind the remaining MFMAs;
//   - one wave per SIMD issues in order, so the loads and tile writes are
//     placed between single MFMAs;
//   - workgroup ids are remapped so that each XCD holds a patch of tiles of
//     a few pixel blocks x many output blocks (tiles that share activations
//     or packed rows sit behind one L2): 4 pixel blocks, or 2 when the
//     packed rows of an output block are under a quarter of a pixel block's
//     activations (K / G < 1/6), so that the XCD's share of the larger
//     operand is fetched fewer times.
//
// LDS layouts (bytes):
//   activation buffer: pixel q at q * 128; its 16-byte column c holds
//     channels 8 * (c ^ sw(q)) .. +7 of the chunk, sw(q) = (q >> 1) % 8.
//     The DMA still reads each pixel's 128 contiguous bytes (one cache line
//     per 8 lanes); with the swizzle a fragment read (16 pixels, one or two
//     8-channel columns per 16 / 32 lanes) touches distinct 16-byte bank
//     slots within every 16 and every 32 lanes.
//   weight tile: 16-row block b, k-step s at (2 b + s) * 1024, inside it
//     (k / 8 % 4) * 256 + (o % 16) * 16 + (k % 8) * 2: the fragment a lane
//     reads is its 16 contiguous bytes at lane * 16.
#include <type_traits>

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

constexpr int kThreads = 256;                   // four waves, one per SIMD
constexpr int kTile = 256;                      // pixels and outputs of a workgroup
constexpr int kCK = 64;                         // channels per chunk (two k-steps)
constexpr int kXBytes = kTile * kCK * 2;        // one activation buffer
constexpr int kWBytes = kTile * kCK * 2;        // one weight tile
constexpr int kWOfs = 3 * kXBytes;              // weight tiles follow the three activation buffers
constexpr int kLds = kWOfs + 2 * kWBytes;       // 160 KiB
constexpr int kEpPitch = 128 * 4 + 16;          // epilogue staging: bytes per pixel row
constexpr uint32_t kOOB = 0x80000000u;          // buffer offset that reads as zero / drops a store
constexpr int kRsrcWord3 = 0x00020000;          // raw buffer descriptor word 3 (gfx9 family)
static_assert(kLds <= 160 * 1024, "LDS budget");
static_assert(4 * 64 * kEpPitch <= kLds, "epilogue staging reuses the operand buffers");

struct WParams {
  const uint16_t* X;
  const uint16_t* vals;
  const uint8_t* idx;
  const float* scale;
  const float* bias;
  const void* residual;
  void* Y;
  uint32_t x_bytes, v_bytes, i_bytes, y_bytes;
  int32_t N, C, O, G, K, relu;
  int32_t npb, nob, nch;  // pixel blocks, output blocks (of 256), channel chunks
  int32_t rows_w;         // packed rows behind 64 outputs: 64 K / G
  int32_t grid8;          // grid / 8 when the grid is a multiple of 8, else 0
  int32_t pgr;            // pixel blocks per run of the XCD tile order (2 or 4)
};

__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Wait until at most N vector-memory operations of this wave are in flight
// (loads complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

template <bool B>
struct BoolC {
  static constexpr bool value = B;
};

// acc += A * B on the matrix cores, with the accumulator pinned to the
// accumulation registers: all 256 of them hold the wave's 128 x 128 tile,
// and the builtin lets the register allocator shuttle accumulators through
// the vector registers.  Dependent uses of acc by vector instructions are
// separated from the last MFMA by mfma_drain().
// (volatile: kept in program order with the other volatile statements below)
__device__ __forceinline__ void mfma_acc(f32x4_t& acc, const bf16x8_t a, const bf16x8_t b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// Longer than any dependency between a vector write of an accumulation
// register and an MFMA reading it, or an MFMA result and a vector read.
__device__ __forceinline__ void mfma_drain() { asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 15\n\ts_nop 15" ::: "memory"); }
// Pin acc's current value in the accumulation registers at this point of
// the volatile sequence (no code).
__device__ __forceinline__ void acc_fence(f32x4_t& acc) { asm volatile("" : "+a"(acc)); }

// Packed-weight loads into registers, issued as plain instructions.  The
// compiler does not track them as pending loads (it cannot count the LDS DMAs
// issued after them and would wait for every outstanding load); the kernel
// waits for them itself with wait_vm<> before any use.
__device__ __forceinline__ u32x4_t sdesc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const auto rfl = [](uint32_t x) { return static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(x))); };
  return u32x4_t{rfl(static_cast<uint32_t>(a)), rfl(static_cast<uint32_t>(a >> 32) & 0xffffu), rfl(bytes),
                 static_cast<uint32_t>(kRsrcWord3)};
}
__device__ __forceinline__ u32x4_t load_x4(const u32x4_t d, uint32_t off) {
  u32x4_t v;
  asm volatile("buffer_load_dwordx4 %0, %1, %2, 0 offen" : "=v"(v) : "v"(off), "s"(d) : "memory");
  return v;
}
__device__ __forceinline__ u32x2_t load_x2(const u32x4_t d, uint32_t off) {
  u32x2_t v;
  asm volatile("buffer_load_dwordx2 %0, %1, %2, 0 offen" : "=v"(v) : "v"(off), "s"(d) : "memory");
  return v;
}
__device__ __forceinline__ uint32_t load_x1(const u32x4_t d, uint32_t off) {
  uint32_t v;
  asm volatile("buffer_load_dword %0, %1, %2, 0 offen" : "=v"(v) : "v"(off), "s"(d) : "memory");
  return v;
}

// Geometry of a workgroup tile of PT 16-pixel tiles per wave (namespace
// scope: the kernel's lambdas must not capture constants of the template).
template <int PT>
struct Geo {
  static constexpr int TP = PT * 32;        // pixels of the workgroup's tile
  static constexpr int XB = TP * kCK * 2;   // one activation buffer
  static constexpr int WOFS = 3 * XB;       // weight tiles follow the three activation buffers
  static constexpr int WPX = PT * 2048;     // bytes of one wave's pixel half of a buffer
};

// Word k of a unit's packed indices.
__device__ __forceinline__ uint32_t iword(const u32x2_t v, int k) { return v[k]; }
__device__ __forceinline__ uint32_t iword(uint32_t v, int) { return v; }

// Byte offset of tile row o (< 256) in the weight tile, k-column 0.
__device__ __forceinline__ uint32_t trow(uint32_t o) { return ((o >> 4) << 11) | ((o & 15) << 4); }

// A unit is UE (8 or 4) consecutive channels of one packed row; UPL units
// per lane per chunk; MASK: the units outnumber the packed rows' (some lanes
// idle), else every lane's units exist and the checks compile away.  FULL: K == G (every entry kept, indices ascending, so
// a unit is one row's 16 bytes).  BIGG: G > 16 (a group spans 16-row
// blocks of the tile).
template <typename YT, int PT, int UPL, int UE, bool FULL, bool BIGG, bool MASK>
__device__ __forceinline__ void wide_tile_body(const WParams& p, uint8_t* lds) {
  constexpr int NW = FULL ? UPL : 2 * UPL;  // vector-memory operations of one packed-chunk load
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wp = w >> 1, wo = w & 1;  // pixel half, output half of this wave

  // ---- tile of this workgroup ------------------------------------------------
  // Dispatch places workgroup b on XCD b % 8; L numbers the workgroups of
  // one XCD consecutively, and runs of pgr * nob consecutive L cover pgr
  // pixel blocks x every output block, output-block-major.
  const uint32_t bid = blockIdx.x;
  const uint32_t L = p.grid8 ? (bid & 7u) * static_cast<uint32_t>(p.grid8) + (bid >> 3) : bid;
  const uint32_t pgr = static_cast<uint32_t>(p.pgr);
  const uint32_t per = pgr * static_cast<uint32_t>(p.nob);
  const uint32_t pg = L / per;
  const uint32_t pgs = min(pgr, static_cast<uint32_t>(p.npb) - pgr * pg);
  const uint32_t within = L - pg * per;
  const uint32_t ob = within / pgs;
  const uint32_t pb = pgr * pg + (within - ob * pgs);

  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.X), (short)0, static_cast<int>(p.x_bytes), kRsrcWord3);
  const u32x4_t vd = sdesc(p.vals, p.v_bytes), id = sdesc(p.idx, p.i_bytes);

  // ---- activation DMA --------------------------------------------------------
  // DMA instruction i of wave w fills pixels (8w + i) * 8 .. +8 of a buffer:
  // lane l writes the 16 bytes at (8w + i) * 1024 + 16 l, i.e. pixel
  // q = (8w + i) * 8 + l / 8, column l % 8, which holds channel block
  // (l % 8) ^ sw(q).  Pixels past N read as zero.
  uint32_t xoff[PT];
#pragma unroll
  for (int i = 0; i < PT; ++i) {
    const uint32_t q = static_cast<uint32_t>((PT * w + i) * 8 + (lane >> 3));
    const uint32_t px = pb * Geo<PT>::TP + q;
    const uint32_t k8 = static_cast<uint32_t>(lane & 7) ^ ((q >> 1) & 7u);
    xoff[i] = px < static_cast<uint32_t>(p.N) ? px * static_cast<uint32_t>(p.C) * 2u + k8 * 16u : kOOB;
  }
  auto issue_x_one = [&](int ch, int buf, int i) {
    lds_void_t* d = (lds_void_t*)(lds + buf * Geo<PT>::XB + w * (PT * 1024) + i * 1024);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, d, 16, xoff[i] + static_cast<uint32_t>(ch) * (kCK * 2), 0, 0, 0);
  };
  auto issue_x = [&](int ch, int buf) {
    uint8_t* dst = lds + buf * Geo<PT>::XB + w * (PT * 1024);
    const uint32_t co = static_cast<uint32_t>(ch) * (kCK * 2);
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      lds_void_t* d = (lds_void_t*)(dst + i * 1024);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, d, 16, xoff[i] + co, 0, 0, 0);
    }
  };

  // ---- packed weights ---------------------------------------------------------
  // Wave w expands tile rows [64 w, 64 w + 64): 64 / G groups, rows_w packed
  // rows.  Unit u of a lane is packed row r = (lane + 64 u) * UE / 64 of
  // them, channels c .. c + UE - 1 of the chunk, c = (lane * UE) % 64 (the
  // lanes of a row read its 64 channels contiguously).
  uint32_t voff[UPL], ioff[UPL], ubase[UPL];
  bool uok[UPL];
#pragma unroll
  for (int u = 0; u < UPL; ++u) {
    const int v = lane + 64 * u;
    const int r = UE == 8 ? v >> 3 : v >> 4;
    const int c = UE == 8 ? (v & 7) * 8 : (v & 15) * 4;
    uok[u] = !MASK || r < p.rows_w;  // (MASK: some lanes have no unit)
    const uint32_t prow = (ob * 4u + static_cast<uint32_t>(w)) * static_cast<uint32_t>(p.rows_w) + static_cast<uint32_t>(r);
    voff[u] = uok[u] ? (prow * static_cast<uint32_t>(p.C) + static_cast<uint32_t>(c)) * 2u : kOOB;
    ioff[u] = uok[u] ? prow * static_cast<uint32_t>(p.C) + static_cast<uint32_t>(c) : kOOB;
    // first tile row of the unit's group (FULL: the unit's own row)
    const int o0 = 64 * w + (FULL ? r : (r / p.K) * p.G);
    const int cb = c >> 3;
    ubase[u] = trow(static_cast<uint32_t>(uok[u] ? o0 : 0)) +
               static_cast<uint32_t>((cb >> 2) * 1024 + (cb & 3) * 256 + (c & 7) * 2);
  }
  // a unit's values and indices, in registers of exactly their size (an
  // asm load result is never copied before its wait)
  using PV = std::conditional_t<UE == 8, u32x4_t, u32x2_t>;
  using PI = std::conditional_t<UE == 8, u32x2_t, uint32_t>;
  PV pv[UPL];
  PI pi[UPL];
  auto load_w = [&](int ch) {
#pragma unroll
    for (int u = 0; u < UPL; ++u) {
      if constexpr (UE == 8) {
        pv[u] = load_x4(vd, voff[u] + static_cast<uint32_t>(ch) * (kCK * 2));
        if constexpr (!FULL) pi[u] = load_x2(id, ioff[u] + static_cast<uint32_t>(ch) * kCK);
      } else {
        pv[u] = load_x2(vd, voff[u] + static_cast<uint32_t>(ch) * (kCK * 2));
        pi[u] = load_x1(id, ioff[u] + static_cast<uint32_t>(ch) * kCK);
      }
    }
  };
  // tile offset of row rr of a group, relative to its first row
  auto grow = [](uint32_t rr) { return BIGG ? trow(rr) : rr << 4; };
  // Building a tile.  The two tiles are zeroed once.  K == G: a build
  // overwrites every entry.  Four entries per lane (UNSC): a build first
  // clears only the entries the build two chunks earlier (same tile) wrote,
  // then writes its own.  Otherwise it zeroes its rows (cheaper from eight
  // entries per lane up), then writes.  All clears of a
  // build are issued before its writes, so across lanes a clear never lands
  // after a write.  Wave w owns tile rows [64 w, 64 w + 64) in every step.
  constexpr bool UNSC = !FULL && UPL * UE <= 4;
  PI pold1[UPL], pold2[UPL];  // indices of the last two builds (UNSC)
#pragma unroll
  for (int u = 0; u < UPL; ++u) pold1[u] = pold2[u] = PI{};
  auto w_fence = [&]() {  // the loaded values are used only after this point
#pragma unroll
    for (int u = 0; u < UPL; ++u) {
      asm volatile("" : "+v"(pv[u]));
      if constexpr (!FULL) asm volatile("" : "+v"(pi[u]));
    }
  };
  auto zero_piece = [&](uint8_t* tb, int i) {
    *reinterpret_cast<u32x4_t*>(tb + w * 8192 + (i * 64 + lane) * 16) = u32x4_t{0u, 0u, 0u, 0u};
  };
  auto zero_rows = [&](uint8_t* tb) {
#pragma unroll
    for (int i = 0; i < 8; ++i) zero_piece(tb, i);
  };
  auto unscatter_e = [&](uint8_t* tb, int u, int e) {  // element e of unscatter(tb, u)
    if (!uok[u]) return;
    const uint32_t rr = (iword(pold2[u], e >> 2) >> (8 * (e & 3))) & 0xffu;
    *reinterpret_cast<uint16_t*>(tb + ubase[u] + grow(rr) + 2 * e) = 0;
  };
  // Element order of the in-loop writes of 8-channel units (PERM): lane l
  // writes element e ^ 2 m2 at step e, m2 = (l / 2) % 4.  Lanes of one
  // half-wave hit random rows of the same 16-byte column, so in plain order
  // they collide on the same banks; XOR-ing the column per lane spreads them
  // over 4x as many.  permute_unit reorders a unit's registers once so that
  // step e reads its value and index at fixed positions.
  constexpr bool PERM = UE == 8 && !FULL && !UNSC;
  const uint32_t m2 = (static_cast<uint32_t>(lane) >> 1) & 3u;
  uint32_t eoff[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) eoff[e] = PERM ? 2u * (static_cast<uint32_t>(e) ^ (2u * m2)) : 2u * e;
  auto permute_unit = [&](int u) {
    if constexpr (PERM) {
      const bool s1 = (m2 & 1u) != 0, s2 = (m2 & 2u) != 0;
      const u32x4_t v = pv[u];
      const u32x4_t t = s1 ? u32x4_t{v[1], v[0], v[3], v[2]} : v;  // element XOR 2: dwords XOR 1
      pv[u] = s2 ? u32x4_t{t[2], t[3], t[0], t[1]} : t;              // element XOR 4: dwords XOR 2
      const u32x2_t x = pi[u];
      const u32x2_t y = s2 ? u32x2_t{x[1], x[0]} : x;               // index bytes XOR 4: dword swap
      const uint32_t hs = 16u * (m2 & 1u);                           // index bytes XOR 2: half swap
      pi[u] = u32x2_t{__builtin_amdgcn_alignbit(y[0], y[0], hs), __builtin_amdgcn_alignbit(y[1], y[1], hs)};
    }
  };
  auto scatter_e = [&](uint8_t* tb, int u, int e) {  // element e of scatter(tb, u), K < G
    if (!uok[u]) return;
    const uint32_t rr = (iword(pi[u], e >> 2) >> (8 * (e & 3))) & 0xffu;
    *reinterpret_cast<uint16_t*>(tb + ubase[u] + grow(rr) + eoff[e]) = static_cast<uint16_t>(pv[u][e >> 1] >> (16 * (e & 1)));
  };
  auto scatter_full = [&](uint8_t* tb, int u) {  // K == G: the unit's 16 bytes
    if constexpr (UE == 8) {
      if (uok[u]) *reinterpret_cast<u32x4_t*>(tb + ubase[u]) = pv[u];
    }
  };
  auto scatter = [&](uint8_t* tb, int u) {
    if (!uok[u]) return;
    if constexpr (FULL && UE == 8) {
      *reinterpret_cast<u32x4_t*>(tb + ubase[u]) = pv[u];
    } else {
#pragma unroll
      for (int e = 0; e < UE; ++e) {
        const uint32_t rr = (iword(pi[u], e >> 2) >> (8 * (e & 3))) & 0xffu;  // row within the group
        *reinterpret_cast<uint16_t*>(tb + ubase[u] + grow(rr) + 2 * e) =
            static_cast<uint16_t>(pv[u][e >> 1] >> (16 * (e & 1)));
      }
    }
  };
  auto rotate_idx = [&]() {
    if constexpr (UNSC) {
#pragma unroll
      for (int u = 0; u < UPL; ++u) {
        pold2[u] = pold1[u];
        pold1[u] = pi[u];
      }
    }
  };

  // ---- MFMAs --------------------------------------------------------------------
  // acc[pt][ot]: 16 pixels (tile pt of the wave's 128) x 16 outputs (tile ot
  // of its 128).  A lane holds outputs 4 (lane / 16) .. +3 of pixel lane % 16.
  f32x4_t acc[PT][8];
#pragma unroll
  for (int pt = 0; pt < PT; ++pt)
#pragma unroll
    for (int ot = 0; ot < 8; ++ot) acc[pt][ot] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int pt = 0; pt < PT; ++pt)
#pragma unroll
    for (int ot = 0; ot < 8; ++ot) acc_fence(acc[pt][ot]);
  mfma_drain();  // the zero writes land before the first MFMA reads them
  // B fragment (activations): pixel lane % 16, channels 8 * (4 s + lane / 16) ..
  const uint32_t xl = static_cast<uint32_t>(lane & 15), xk = static_cast<uint32_t>(lane >> 4);
  const uint32_t sw = (xl >> 1) & 7u;
  const uint32_t boff0 = xl * 128u + ((xk ^ sw) << 4);
  const uint32_t boff1 = xl * 128u + (((4u + xk) ^ sw) << 4);
  auto ld = [](const uint8_t* q) { return *reinterpret_cast<const bf16x8_t*>(q); };

  // ---- pipeline -------------------------------------------------------------------
  // A wave's vector-memory operations are issued in the order X(0) W(0) X(1)
  // W(1) X(2), then per chunk j: W(j+2) (group 7) and X(j+3) (groups 8-11,
  // into the buffer chunk j has just released).  Loads complete in issue
  // order, so "X(c) has landed" is "at most <ops issued after it> in flight".
  const int nch = p.nch;
  issue_x(0, 0);
  load_w(0);
  if (nch > 1) issue_x(1, 1);
  if (nch > 1) wait_vm<PT>(); else wait_vm<0>();  // W(0)
  w_fence();
  zero_rows(lds + Geo<PT>::WOFS);
  zero_rows(lds + Geo<PT>::WOFS + kWBytes);
#pragma unroll
  for (int u = 0; u < UPL; ++u) scatter(lds + Geo<PT>::WOFS, u);
  rotate_idx();
  if (nch > 1) load_w(1);
  if (nch > 2) issue_x(2, 2);
  if (nch > 2) wait_vm<PT>(); else wait_vm<0>();  // X(0), X(1), W(1)
  w_fence();
  lds_barrier();

  // Chunk j is 16 groups of 8 MFMAs: group g multiplies k-step g / 8 by
  // output tile g % 8 against the wave's 8 pixel tiles.  Fragments sit in
  // registers well before use: af[g] holds the weight fragment of group g,
  // b0 / b1 the activation fragments of k-step 0 / 1.  The barrier of chunk
  // j sits between groups 7 and 8; the instruction order is fixed with
  // scheduling barriers:
  //   groups 0-7: read b1[g] and af[g + 8] (the rest of chunk j, so after
  //     the barrier no wave reads chunk j's buffers); build tile j+1: clear
  //     (groups 0-3), write W(j+1) (groups 4-7); then load W(j+2);
  //   barrier: X(j+1) has landed and tile j+1 is complete in every wave;
  //   groups 8-15: DMA X(j+3) into chunk j's buffer (two per group, groups
  //     8-11), read chunk j+1's b0 (two per group, groups 8-11) and
  //     af[g - 8] from the new buffers.
  // Every fragment read is issued at least four groups (~500 cycles of
  // MFMAs) before its use.  M1 / M2 / M3: chunks j+1 / j+2 / j+3 exist
  // (compile-time, so the steady-state body has no branches).
  bf16x8_t b0[PT], b1[PT], af[16];
  auto read_first = [&](int j) {  // chunk j's k-step-0 fragments
    const uint8_t* xb = lds + (j % 3) * Geo<PT>::XB + wp * Geo<PT>::WPX;
    const uint8_t* wb = lds + Geo<PT>::WOFS + (j & 1) * kWBytes + wo * 16384 + lane * 16;
#pragma unroll
    for (int pt = 0; pt < PT; ++pt) b0[pt] = ld(xb + pt * 2048 + boff0);
#pragma unroll
    for (int g = 0; g < 8; ++g) af[g] = ld(wb + g * 2048);
  };
  constexpr int kUPG = (UPL + 3) / 4;  // packed units per group (groups 0-3 clear, 4-7 write)
  // xbuf = j % 3 and tbit = j % 2 select the buffers; the unrolled steady
  // state passes them as literals, so every LDS address of a chunk (the DMA
  // targets in M0 included) is a constant offset from the wave's base.
  auto chunk = [&](int j, int xbuf, int tbit, auto m1, auto m2, auto m3) __attribute__((always_inline)) {
    constexpr bool more1 = decltype(m1)::value, more2 = decltype(m2)::value, more3 = decltype(m3)::value;
    const uint8_t* xb = lds + xbuf * Geo<PT>::XB + wp * Geo<PT>::WPX;
    const uint8_t* wb = lds + Geo<PT>::WOFS + tbit * kWBytes + wo * 16384 + lane * 16;
    const int xnb = xbuf == 2 ? 0 : xbuf + 1;
    const uint8_t* xn = lds + xnb * Geo<PT>::XB + wp * Geo<PT>::WPX;  // chunk j+1
    const uint8_t* wn = lds + Geo<PT>::WOFS + (tbit ^ 1) * kWBytes + wo * 16384 + lane * 16;
    uint8_t* tb = lds + Geo<PT>::WOFS + (tbit ^ 1) * kWBytes;  // tile j+1, built here
#pragma unroll
    for (int g = 0; g < 16; ++g) {
      if constexpr (more1) {
        if (g == 8) {
          if constexpr (more2) wait_vm<PT + 2 * NW>(); else wait_vm<0>();  // X(j+1)
          lds_barrier();
        }
      }
      // One wave per SIMD issues in order, so other work overlaps an MFMA
      // only when it sits between two of them: slot i follows MFMA i.
#pragma unroll
      for (int i = 0; i < PT; ++i) {
        mfma_acc(acc[i][g & 7], af[g], g < 8 ? b0[i] : b1[i]);
        __builtin_amdgcn_sched_barrier(0);
        if (g < 8) {
          if (i == 0 && g < PT) b1[g % PT] = ld(xb + g * 2048 + boff1);
          if (i == 1) af[g + 8] = ld(wb + (g * 2 + 1) * 1024);
          if constexpr (more1) {
            if constexpr (PERM) {
#pragma unroll
              for (int u = i; u < UPL; u += PT)
                if (g == 3) permute_unit(u);  // W(j+1) is in registers since chunk j-1 ended
            }
            if constexpr (FULL) {
              if (g >= 4 && i >= 2 && i < 2 + kUPG) scatter_full(tb, (g - 4) * kUPG + (i - 2));
            } else {
              if constexpr (!UNSC) {
                if (g < 4 && (i == 2 || i == 3)) zero_piece(tb, 2 * g + (i - 2));
              }
#pragma unroll
              for (int k = 0; k < kUPG; ++k) {
                const int u = (g & 3) * kUPG + k;
#pragma unroll
                for (int e = i; e < UE; e += PT) {  // element e of unit u, at slot e % PT
                  if (u < UPL) {
                    if (g < 4) {
                      if constexpr (UNSC) unscatter_e(tb, u, e);
                    } else {
                      scatter_e(tb, u, e);
                    }
                  }
                }
              }
            }
            if (g == 7 && i == PT - 1) {
              rotate_idx();
              if constexpr (more2) load_w(j + 2);
            }
          }
        } else if constexpr (more1) {
          if (g < 8 + PT / 2) {
            if constexpr (more3) {
              if (i == 0) {
                issue_x_one(j + 3, xbuf, 2 * (g - 8));
                issue_x_one(j + 3, xbuf, 2 * (g - 8) + 1);
              }
            }
            if (i == 1) b0[(2 * (g - 8)) % PT] = ld(xn + (2 * (g - 8)) * 2048 + boff0);
            if (i == 2) b0[(2 * (g - 8) + 1) % PT] = ld(xn + (2 * (g - 8) + 1) * 2048 + boff0);
          }
          if (i == 3) af[g - 8] = ld(wn + (g - 8) * 2048);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // W(j+2) is in registers before the loop carries it on (copies of it
    // may be made at the loop head)
    if constexpr (more2) {
      if constexpr (more3) wait_vm<PT>(); else wait_vm<0>();
      w_fence();
    }
  };
  read_first(0);
  int j = 0;
  const BoolC<true> T{};
  const BoolC<false> F{};
  // (with four or eight packed units per lane the six copies no longer fit
  // the registers: those variants keep the one-chunk loop)
  if constexpr (FULL || UPL <= 2) {
#pragma unroll 1
    for (; j + 8 < nch; j += 6) {  // six chunks: both rotations return to their start
      chunk(j, 0, 0, T, T, T);
      chunk(j + 1, 1, 1, T, T, T);
      chunk(j + 2, 2, 0, T, T, T);
      chunk(j + 3, 0, 1, T, T, T);
      chunk(j + 4, 1, 0, T, T, T);
      chunk(j + 5, 2, 1, T, T, T);
    }
  }
#pragma unroll 1
  for (; j + 3 < nch; ++j) chunk(j, j % 3, j & 1, T, T, T);
  if (j + 2 < nch) {
    chunk(j, j % 3, j & 1, T, T, F);
    ++j;
  }
  if (j + 1 < nch) {
    chunk(j, j % 3, j & 1, T, F, F);
    ++j;
  }
  chunk(j, j % 3, j & 1, F, F, F);

  // ---- fused epilogue -----------------------------------------------------------
  // Each wave parks 64 pixels x 128 outputs (fp32) at a time in its own LDS
  // region (pitch 528 bytes: the read-back below is conflict-free) and
  // reads them back by pixel rows: a lane then owns 8 consecutive outputs
  // of one pixel (16 lanes cover the wave's 128), applies scale / bias /
  // residual / ReLU in fp32, rounds once and stores 16 (bf16) or 32 bytes.
  mfma_drain();    // the last MFMAs have written acc
#pragma unroll
  for (int pt = 0; pt < PT; ++pt)
#pragma unroll
    for (int ot = 0; ot < 8; ++ot) acc_fence(acc[pt][ot]);
  lds_barrier();  // every wave is done with the operand buffers
  constexpr uint32_t ysz = sizeof(YT);
  const __amdgpu_buffer_rsrc_t yr =
      __builtin_amdgcn_make_buffer_rsrc(p.Y, (short)0, static_cast<int>(p.y_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rsr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(p.residual), (short)0, p.residual ? static_cast<int>(p.y_bytes) : 0, kRsrcWord3);
  const int c8 = lane & 15;  // 8-output block of the wave's 128
  const uint32_t o = ob * kTile + static_cast<uint32_t>(wo * 128 + 8 * c8);
  f32x4_t sc0{1.f, 1.f, 1.f, 1.f}, sc1{1.f, 1.f, 1.f, 1.f}, bi0{0.f, 0.f, 0.f, 0.f}, bi1{0.f, 0.f, 0.f, 0.f};
  if (p.scale) {
    sc0 = *reinterpret_cast<const f32x4_t*>(p.scale + o);
    sc1 = *reinterpret_cast<const f32x4_t*>(p.scale + o + 4);
  }
  if (p.bias) {
    bi0 = *reinterpret_cast<const f32x4_t*>(p.bias + o);
    bi1 = *reinterpret_cast<const f32x4_t*>(p.bias + o + 4);
  }
  uint8_t* stg = lds + w * 64 * kEpPitch;
  const auto row_off = [&](int h, int rr) {  // Y / residual byte offset of the lane's row rr of pass h
    const uint32_t px = pb * Geo<PT>::TP + static_cast<uint32_t>(wp * (PT * 16) + h * 64 + 4 * rr + (lane >> 4));
    return px < static_cast<uint32_t>(p.N) ? (px * static_cast<uint32_t>(p.O) + o) * ysz : kOOB;
  };
#pragma unroll
  for (int h = 0; h < PT / 4; ++h) {
    // bf16 residual: all 16 rows' 16-byte pieces are requested before the
    // rows are processed (one load latency per pass, not one per row)
    u32x4_t rres[16];
    if constexpr (ysz == 2) {
      if (p.residual) {
#pragma unroll
        for (int rr = 0; rr < 16; ++rr)
          rres[rr] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rsr, row_off(h, rr), 0, 0));
      }
    }
#pragma unroll
    for (int pt = 0; pt < 4; ++pt)
#pragma unroll
      for (int ot = 0; ot < 8; ++ot)
        *reinterpret_cast<f32x4_t*>(stg + (pt * 16 + (lane & 15)) * kEpPitch + (ot * 16 + 4 * (lane >> 4)) * 4) =
            acc[4 * h + pt][ot];
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      const int row = 4 * rr + (lane >> 4);
      const uint8_t* src = stg + row * kEpPitch + c8 * 32;
      f32x4_t y0 = *reinterpret_cast<const f32x4_t*>(src);
      f32x4_t y1 = *reinterpret_cast<const f32x4_t*>(src + 16);
      const uint32_t off = row_off(h, rr);
      y0 = y0 * sc0 + bi0;
      y1 = y1 * sc1 + bi1;
      if (p.residual) {
        if constexpr (ysz == 2) {
          const u32x4_t r = rres[rr];
          y0[0] += __uint_as_float(r[0] << 16);
          y0[1] += __uint_as_float(r[0] & 0xffff0000u);
          y0[2] += __uint_as_float(r[1] << 16);
          y0[3] += __uint_as_float(r[1] & 0xffff0000u);
          y1[0] += __uint_as_float(r[2] << 16);
          y1[1] += __uint_as_float(r[2] & 0xffff0000u);
          y1[2] += __uint_as_float(r[3] << 16);
          y1[3] += __uint_as_float(r[3] & 0xffff0000u);
        } else {
          y0 += __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rsr, off, 0, 0));
          y1 += __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rsr, off + 16, 0, 0));
        }
      }
      if (p.relu) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          y0[e] = y0[e] > 0.0f ? y0[e] : (y0[e] != y0[e] ? y0[e] : 0.0f);
          y1[e] = y1[e] > 0.0f ? y1[e] : (y1[e] != y1[e] ? y1[e] : 0.0f);
        }
      }
      if constexpr (ysz == 2) {
        // v_cvt_pk_bf16_f32: round to nearest even
        const u32x4_t pk = {__builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y0[0], y0[1]}), bf16x2_t)),
                            __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y0[2], y0[3]}), bf16x2_t)),
                            __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y1[0], y1[1]}), bf16x2_t)),
                            __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y1[2], y1[3]}), bf16x2_t))};
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(yr, 0, 0, 0)), pk), yr, off, 0, 0);
      } else {
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(yr, 0, 0, 0)), y0), yr, off, 0, 0);
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(yr, 0, 0, 0)), y1), yr, off + 16, 0, 0);
      }
    }
  }
}

// (The body is a device function: with it inside the kernel template, the
// host pass of this compiler emitted no launch stubs for the kernels.)
template <typename YT, int PT, int UPL, int UE, bool FULL, bool BIGG, bool MASK>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void wide_tile_kernel(WParams p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  wide_tile_body<YT, PT, UPL, UE, FULL, BIGG, MASK>(p, lds);
}

// Rows of X are pixels: FC, or a 1x1 convolution with unit stride and no
// padding over NHWC activations.
bool plain_rows(const ProductArgs& a) {
  if (!a.conv) return true;
  const ConvGeom& g = a.geom;
  return g.KH == 1 && g.KW == 1 && g.sh == 1 && g.sw == 1 && g.ph == 0 && g.pw == 0;
}

template <typename YT, int PT, int UPL, int UE, bool FULL, bool BIGG, bool MASK>
hipError_t launch_wu(const WParams& p, uint32_t grid, hipStream_t s) {
  static std::atomic<int8_t> lds_set[kMaxDevices];
  const hipError_t attr = set_lds_limit_once(
      lds_set, reinterpret_cast<const void*>(&wide_tile_kernel<YT, PT, UPL, UE, FULL, BIGG, MASK>), kLds);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((wide_tile_kernel<YT, PT, UPL, UE, FULL, BIGG, MASK>), dim3(grid), dim3(kThreads), kLds, s, p);
  return hipGetLastError();
}

template <typename YT, int PT, bool BIGG, int UPL>
hipError_t launch_wm(const WParams& p, uint32_t grid, hipStream_t s) {
  return p.rows_w == 8 * UPL ? launch_wu<YT, PT, UPL, 8, false, BIGG, false>(p, grid, s)
                             : launch_wu<YT, PT, UPL, 8, false, BIGG, true>(p, grid, s);
}

template <typename YT, int PT, bool BIGG>
hipError_t launch_wg(const WParams& p, uint32_t grid, hipStream_t s) {
  // packed elements per lane per chunk: rows_w (= 64 K / G)
  if (p.rows_w == 4) return launch_wu<YT, PT, 1, 4, false, BIGG, false>(p, grid, s);
  if (p.rows_w <= 8) return launch_wm<YT, PT, BIGG, 1>(p, grid, s);
  if (p.rows_w <= 16) return launch_wm<YT, PT, BIGG, 2>(p, grid, s);
  if (p.rows_w <= 32) return launch_wm<YT, PT, BIGG, 4>(p, grid, s);
  return launch_wu<YT, PT, 8, 8, false, BIGG, true>(p, grid, s);
}

template <typename YT, int PT>
hipError_t launch_wp(const WParams& p, uint32_t grid, hipStream_t s) {
  if (p.K == p.G) return launch_wu<YT, PT, 8, 8, true, false, false>(p, grid, s);
  return p.G > 16 ? launch_wg<YT, PT, true>(p, grid, s) : launch_wg<YT, PT, false>(p, grid, s);
}

// Pixels per workgroup tile: 256, or 128 when 256-pixel tiles would leave
// more than half of the CUs idle.
int tile_pixels(int64_t N, int64_t O) { return (N + 255) / 256 * (O / kTile) >= 128 ? 256 : 128; }

}  // namespace

bool wide_tile_supports(const ProductArgs& a) {
  if (a.x_t != DType::BF16 || a.val_t != DType::BF16) return false;
  if (!plain_rows(a)) return false;
  if (a.G < 1 || a.G > 64 || 64 % a.G != 0 || a.K < 1 || a.K > a.G) return false;
  if (a.C % kCK != 0 || a.O % kTile != 0 || a.N < 1) return false;
  const auto al = [](const void* q, uintptr_t m) { return (reinterpret_cast<uintptr_t>(q) & (m - 1)) == 0; };
  if (!al(a.X, 16) || !al(a.vals, 16) || !al(a.idx, 8) || !al(a.Y, 16)) return false;
  if ((a.scale && !al(a.scale, 16)) || (a.bias && !al(a.bias, 16)) || (a.residual && !al(a.residual, 16)))
    return false;
  // every buffer offset is 32-bit and stays below the out-of-range marker
  const int64_t lim = static_cast<int64_t>(kOOB);
  const int64_t packed = (a.O / a.G) * a.K * a.C;
  if (a.N * a.C * 2 >= lim || packed * 2 >= lim || a.N * a.O * (a.y_t == DType::F32 ? 4 : 2) >= lim) return false;
  return true;
}

hipError_t launch_wide_tile(const ProductArgs& a, hipStream_t s) {
  if (!wide_tile_supports(a)) return hipErrorInvalidConfiguration;
  WParams p{};
  p.X = static_cast<const uint16_t*>(a.X);
  p.vals = static_cast<const uint16_t*>(a.vals);
  p.idx = a.idx;
  p.scale = a.scale;
  p.bias = a.bias;
  p.residual = a.residual;
  p.Y = a.Y;
  const int64_t ysz = a.y_t == DType::F32 ? 4 : 2;
  const int64_t packed = (a.O / a.G) * a.K * a.C;
  p.x_bytes = static_cast<uint32_t>(a.N * a.C * 2);
  p.v_bytes = static_cast<uint32_t>(packed * 2);
  p.i_bytes = static_cast<uint32_t>(packed);
  p.y_bytes = static_cast<uint32_t>(a.N * a.O * ysz);
  p.N = static_cast<int32_t>(a.N);
  p.C = static_cast<int32_t>(a.C);
  p.O = static_cast<int32_t>(a.O);
  p.G = a.G;
  p.K = a.K;
  p.relu = a.relu;
  const int tp = tile_pixels(a.N, a.O);
  p.npb = static_cast<int32_t>((a.N + tp - 1) / tp);
  p.nob = static_cast<int32_t>(a.O / kTile);
  p.nch = static_cast<int32_t>(a.C / kCK);
  p.rows_w = 64 * a.K / a.G;
  const int64_t grid = static_cast<int64_t>(p.npb) * p.nob;
  if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
  p.grid8 = grid % 8 == 0 ? static_cast<int32_t>(grid / 8) : 0;
  // An XCD running P pixel blocks x (32 / P) output blocks fetches P blocks
  // of X (256 C bf16 each) and 32 / P blocks of packed rows (256 C K / G
  // values and indices, 3 bytes each): 2 beats 4 when 8 K / G < 4 / 3.
  p.pgr = 6 * a.K < a.G ? 2 : 4;
  const uint32_t g = static_cast<uint32_t>(grid);
  if (tp == 256) return a.y_t == DType::BF16 ? launch_wp<bf16_t, 8>(p, g, s) : launch_wp<float, 8>(p, g, s);
  return a.y_t == DType::BF16 ? launch_wp<bf16_t, 4>(p, g, s) : launch_wp<float, 4>(p, g, s);
}

}  // namespace cci
