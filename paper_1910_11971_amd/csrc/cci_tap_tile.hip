// CCI-sparse product on the matrix cores, tap-chunk plan: convolutions of
// any geometry through implicit im2col, and FC products, whose reduction
// splits into chunks of 64 input channels under one filter tap.
//
// Chunk j of the reduction is packed columns 64 j .. 64 j + 63, i.e. tap
// t = j / (Cin / 64) (kh = t / KW, kw = t % KW) and input channels
// 64 (j % (Cin / 64)) .. +63: the columns of W [O][KH][KW][Cin] in order.  Per
// chunk:
//   - the packed groups of the workgroup's 128 outputs are expanded to a
//     dense 128 x 64 bf16 tile in LDS (zero fill, then every kept weight
//     written to row G*g + idx of its column: the routing of Alg. 1,
//     Sec. 3.2);
//   - the 128 output pixels' input pixels under tap t are DMA'd to LDS, 128
//     contiguous bytes each; a tap that falls into the padding reads zero
//     through the buffer's range check (its offset has bit 31 set);
//   - the tile is multiplied on v_mfma_f32_16x16x32_bf16.
// Work split: a workgroup is four waves and owns 128 pixels x 128 outputs;
// wave (wp, wo) accumulates pixels 64 wp .. +63 x outputs 64 wo .. +63 in
// sixteen 16 x 16 accumulators.  A workgroup takes 80 KiB of LDS (three
// activation buffers, two weight tiles), so two share a CU and the tile
// builds, barriers and epilogue of one overlap the other's MFMAs.  This
// serves the products with long reductions and few output tiles (k x k
// convolutions over 128-512 channels, 1x1 layers of 10^4 pixels) that leave
// most CUs idle under 256 x 256 tiles.
//
// LDS layouts (bytes):
//   activation buffer: pixel q at q * 128; its 16-byte column c holds
//     channels 8 * (c ^ sw(q)) .. +7 of the chunk, sw(q) = (q >> 1) % 8 (a
//     fragment read of 16 pixels touches distinct bank slots per 16 lanes).
//   weight tile: 16-row block b, k-step s at (2 b + s) * 1024, inside it
//     (k / 8 % 4) * 256 + (o % 16) * 16 + (k % 8) * 2: the fragment a lane
//     reads is its 16 contiguous bytes at lane * 16.
#include <type_traits>
#include <utility>

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

constexpr int kThreads = 256;             // four waves
constexpr int kTP = 128;                  // pixels of a workgroup tile
constexpr int kCK = 64;                   // reduction columns per chunk (two k-steps)
constexpr int kXB = kTP * kCK * 2;        // one activation buffer
// NX activation buffers, then the two weight tiles: 80 KiB with three
// buffers (two workgroups per CU), 96 KiB with four (one per CU, one chunk
// more of prefetch)
// TO outputs per workgroup tile (128, or 64 for grids that would leave CUs
// idle): one weight tile is TO x 64 bf16
constexpr int wb_bytes(int to) { return to * kCK * 2; }
constexpr int lds_bytes(int nx, int to) { return nx * kXB + 2 * wb_bytes(to); }
// epilogue staging: bytes per pixel row of a wave's 64 x TO/2 fp32 block
constexpr int ep_pitch(int to) { return to / 2 * 4 + 16; }
constexpr int kMaxTaps = 32;              // taps of one filter (one validity bit each)
constexpr uint32_t kDeepGrid = 257;       // grids below this run one workgroup per CU
constexpr int64_t kSmallGrid = 128;       // fewer 128-output tiles than this (half the CUs): 64-output tiles
constexpr uint32_t kOOB = 0x80000000u;    // buffer offset that reads as zero / drops a store
constexpr int kRsrcWord3 = 0x00020000;    // raw buffer descriptor word 3 (gfx9 family)
static_assert(4 * 64 * ep_pitch(128) <= lds_bytes(3, 128) && 4 * 64 * ep_pitch(64) <= lds_bytes(3, 64),
              "epilogue staging reuses the operand buffers");

struct TParams {
  const uint16_t* X;
  const uint16_t* vals;
  const uint8_t* idx;
  const float* scale;
  const float* bias;
  const void* residual;
  void* Y;
  uint32_t x_bytes, v_bytes, i_bytes, y_bytes;
  int32_t N, C, O, G, K, relu;
  int32_t npb, nob, nch;  // pixel blocks (of 128), output blocks (of TO), chunks
  int32_t cpt;            // chunks per tap: Cin / 64
  int32_t rows_w;         // packed rows behind one wave's TO / 4 tile rows: TO / 4 * K / G
  int32_t grid8;          // launched workgroups / 8 (the tile count rounded up to a multiple of 8)
  int32_t ntiles;         // npb * nob
  // input geometry (an FC product is B = N images of 1 x 1 pixel)
  int32_t H, W, Cin, KH, KW, sh, sw, ph, pw, HoWo, Wo;
};

__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Wait until at most N vector-memory operations of this wave are in flight
// (loads complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Packed-weight loads into registers, issued as plain instructions that the
// compiler does not count (it would otherwise wait for the LDS DMAs issued
// after them); the kernel waits for them with wait_vm<> before any use.
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

// f(integral_constant<int, K>) for K in the sequence, in order.
template <int... K, typename F>
__device__ __forceinline__ void for_k(std::integer_sequence<int, K...>, F&& f) {
  (f(std::integral_constant<int, K>{}), ...);
}

// acc += A * B on the matrix cores, with the accumulator pinned to the
// accumulation registers (the builtin lets the register allocator move the
// 64 accumulators between register files every chunk).  Dependent uses of
// acc by vector instructions are separated from the last MFMA by
// mfma_drain().  (volatile: kept in program order with the other volatile
// statements.)
__device__ __forceinline__ void mfma_acc(f32x4_t& acc, const bf16x8_t a, const bf16x8_t b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// Longer than any dependency between a vector write of an accumulation
// register and an MFMA reading it, or an MFMA result and a vector read.
__device__ __forceinline__ void mfma_drain() { asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 15\n\ts_nop 15" ::: "memory"); }
// Pin acc's current value in the accumulation registers at this point of
// the volatile sequence (no code).
__device__ __forceinline__ void acc_fence(f32x4_t& acc) { asm volatile("" : "+a"(acc)); }

// Ring stage K's packed units are used only after this point (after the
// wait that covers their loads).
template <int K, bool FULL, int RW, int UPL>
__device__ __forceinline__ void fence_stage(u32x4_t (&pv)[RW][UPL], u32x2_t (&pi)[RW][UPL]) {
#pragma unroll
  for (int u = 0; u < UPL; ++u) {
    asm volatile("" : "+v"(pv[K][u]));
    if constexpr (!FULL) asm volatile("" : "+v"(pi[K][u]));
  }
}

// Byte offset of tile row o (< 128) in the weight tile, k-column 0.
__device__ __forceinline__ uint32_t trow(uint32_t o) { return ((o >> 4) << 11) | ((o & 15) << 4); }

// UPL: 8-channel packed units per lane per chunk.  FULL: K == G (every
// entry kept, indices ascending, so a unit is one tile row's 16 bytes).
// BIGG: G == 32 (a group spans two 16-row blocks).  MASK: some lanes have no
// unit (else the checks compile away).
template <typename YT, int UPL, bool FULL, bool BIGG, bool MASK, int NX, int TO>
__device__ __forceinline__ void tap_tile_body(const TParams& p, uint8_t* lds) {
  constexpr int RW = NX - 1;         // packed-unit ring stages: W(m) is issued with X(m)
  constexpr int OT = TO / 32;        // 16-output tiles per wave
  constexpr int RPW = TO / 4;        // weight-tile rows a wave builds
  constexpr int WB = wb_bytes(TO);   // one weight tile
  constexpr int PITCH = ep_pitch(TO);
  constexpr int NMF = 4 * OT;        // MFMAs of one k-step
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wp = w >> 1, wo = w & 1;  // pixel half, output half (TO / 2 outputs) of this wave

  // ---- tile of this workgroup ---------------------------------------------
  // Dispatch places workgroup b on XCD b % 8; L numbers the workgroups of one
  // XCD consecutively, output block fastest, so the tiles that read the same
  // activations run behind one L2.  (The grid is rounded up to a multiple
  // of 8; the workgroups past the last tile leave at once.)
  const uint32_t bid = blockIdx.x;
  const uint32_t L = (bid & 7u) * static_cast<uint32_t>(p.grid8) + (bid >> 3);
  if (L >= static_cast<uint32_t>(p.ntiles)) return;
  const uint32_t pb = L / static_cast<uint32_t>(p.nob);
  const uint32_t ob = L - pb * static_cast<uint32_t>(p.nob);

  // ---- activation DMA ---------------------------------------------------------
  // DMA instruction i of wave w fills pixels (4 w + i) * 8 .. +7 of a buffer:
  // lane l writes the 16 bytes at (4 w + i) * 1024 + 16 l, i.e. pixel
  // q = (4 w + i) * 8 + l / 8, column l % 8, which holds channel block
  // (l % 8) ^ sw(q).  xbase: byte offset of that block of the input pixel
  // under tap (0, 0) (negative in the padding); xinv bit t: tap t of the
  // pixel falls into the padding, or the pixel is past N.
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.X), (short)0, static_cast<int>(p.x_bytes), kRsrcWord3);
  int32_t xbase[4];
  uint32_t xinv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int q = (4 * w + i) * 8 + (lane >> 3);
    const int px = static_cast<int>(pb) * kTP + q;
    const int k8 = (lane & 7) ^ ((q >> 1) & 7);
    xbase[i] = 0;
    xinv[i] = ~0u;
    if (px < p.N) {
      const int img = px / p.HoWo;
      const int rem = px - img * p.HoWo;
      const int oh = rem / p.Wo;
      const int ow = rem - oh * p.Wo;
      const int ih0 = oh * p.sh - p.ph, iw0 = ow * p.sw - p.pw;
      xbase[i] = ((img * p.H + ih0) * p.W + iw0) * p.Cin * 2 + k8 * 16;
      uint32_t inv = 0;
      int t = 0;
      for (int kh = 0; kh < p.KH; ++kh) {
        const bool hok = static_cast<unsigned>(ih0 + kh) < static_cast<unsigned>(p.H);
        for (int kw = 0; kw < p.KW; ++kw, ++t) {
          const bool ok = hok && static_cast<unsigned>(iw0 + kw) < static_cast<unsigned>(p.W);
          inv |= (ok ? 0u : 1u) << t;
        }
      }
      xinv[i] = inv;
    }
  }
  // Tap cursor of the next chunk to DMA: t = tap, cb = channel block,
  // kw = column of the tap, off = byte offset of (tap, block) from the
  // pixel's tap-(0, 0) block.  The next block of a tap, and the first block
  // of the next tap in the row, are both 128 bytes further.
  int cur_t = 0, cur_cb = 0, cur_kw = 0;
  int32_t cur_off = 0;
  const int32_t row_skip = (p.W - p.KW) * p.Cin * 2;
  auto issue_x = [&](int buf) {
    uint8_t* dst = lds + buf * kXB + w * 4096;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t off = static_cast<uint32_t>(xbase[i] + cur_off) | (((xinv[i] >> cur_t) & 1u) << 31);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t*)(dst + i * 1024), 16, off, 0, 0, 0);
    }
    cur_off += 128;
    if (++cur_cb == p.cpt) {
      cur_cb = 0;
      ++cur_t;
      if (++cur_kw == p.KW) {
        cur_kw = 0;
        cur_off += row_skip;
      }
    }
  };

  // ---- packed weights ---------------------------------------------------------
  // Wave w expands tile rows [RPW w, RPW w + RPW): RPW / G groups, rows_w
  // packed rows.  Unit u of a lane is packed row r = (lane + 64 u) / 8 of them,
  // channels 8 c8 .. +7 of the chunk, c8 = (lane + 64 u) % 8.
  const u32x4_t vd = sdesc(p.vals, p.v_bytes), id = sdesc(p.idx, p.i_bytes);
  // The lanes of one packed row write neighbouring column blocks whose
  // 16-byte row segments all start on the same bank, so at step e lane l
  // writes element e ^ m, m = l % 8, of its unit: one instruction's two-byte
  // stores spread over four times as many banks.  A unit's values and
  // indices are permuted once (permute_unit) so that step e reads them at
  // fixed positions.
  const uint32_t m = static_cast<uint32_t>(lane & 7);
  const uint32_t bsel = 0x03020100u ^ ((m & 3u) * 0x01010101u);  // byte j <- byte j ^ (m % 4)
  uint32_t voff[UPL], ioff[UPL], ubase[UPL];
  bool uok[UPL];
#pragma unroll
  for (int u = 0; u < UPL; ++u) {
    const int v = lane + 64 * u;
    const int r = v >> 3, c8 = v & 7;
    uok[u] = !MASK || r < p.rows_w;
    const uint32_t prow = (ob * static_cast<uint32_t>(TO / p.G) + static_cast<uint32_t>(w * (RPW / p.G))) *
                              static_cast<uint32_t>(p.K) +
                          static_cast<uint32_t>(r);
    voff[u] = uok[u] ? (prow * static_cast<uint32_t>(p.C) + static_cast<uint32_t>(c8 * 8)) * 2u : kOOB;
    ioff[u] = uok[u] ? prow * static_cast<uint32_t>(p.C) + static_cast<uint32_t>(c8 * 8) : kOOB;
    const int o0 = RPW * w + (FULL ? r : (r / p.K) * p.G);  // first tile row of the unit's group
    // (non-FULL: bits 1..3 carry 2 m, the byte offset of element m)
    ubase[u] = trow(static_cast<uint32_t>(uok[u] ? o0 : 0)) +
               static_cast<uint32_t>((c8 >> 2) * 1024 + (c8 & 3) * 256) + (FULL ? 0u : 2u * m);
  }
  // Register ring of RW stages: stage k holds the packed units of the
  // chunks j with j % RW == k (the index is always a compile-time constant).
  u32x4_t pv[RW][UPL];
  u32x2_t pi[RW][UPL];
  auto load_w = [&](int ch, auto kc) {
    constexpr int k = decltype(kc)::value;
#pragma unroll
    for (int u = 0; u < UPL; ++u) {
      pv[k][u] = load_x4(vd, voff[u] + static_cast<uint32_t>(ch) * (kCK * 2));
      if constexpr (!FULL) pi[k][u] = load_x2(id, ioff[u] + static_cast<uint32_t>(ch) * kCK);
    }
  };
  auto w_fence = [&](auto kc) { fence_stage<decltype(kc)::value, FULL>(pv, pi); };
  auto permute_unit = [&](auto kc, int u) {  // element e of the unit moves to position e ^ m
    constexpr int k = decltype(kc)::value;
    if constexpr (!FULL) {
      u32x4_t d = pv[k][u];
      u32x2_t x = pi[k][u];
      if (m & 4u) {
        d = u32x4_t{d[2], d[3], d[0], d[1]};
        x = u32x2_t{x[1], x[0]};
      }
      if (m & 2u) d = u32x4_t{d[1], d[0], d[3], d[2]};
      const uint32_t hs = 16u * (m & 1u);
      pv[k][u] = u32x4_t{__builtin_amdgcn_alignbit(d[0], d[0], hs), __builtin_amdgcn_alignbit(d[1], d[1], hs),
                         __builtin_amdgcn_alignbit(d[2], d[2], hs), __builtin_amdgcn_alignbit(d[3], d[3], hs)};
      pi[k][u] = u32x2_t{__builtin_amdgcn_perm(x[0], x[0], bsel), __builtin_amdgcn_perm(x[1], x[1], bsel)};
    }
  };
  // tile offset of row rr of a group, relative to its first row
  auto grow = [](uint32_t rr) { return BIGG ? trow(rr) : rr << 4; };
  // Building a tile: wave w zeroes its RPW rows (RPW / 16 blocks of 16 rows,
  // both k-steps: RPW * 128 bytes at w * RPW * 128), then
  // writes its kept weights; LDS operations of one wave complete in order.
  auto zero_piece = [&](uint8_t* tb, int i) {
    *reinterpret_cast<u32x4_t*>(tb + w * (RPW * 128) + i * 1024 + lane * 16) = u32x4_t{0u, 0u, 0u, 0u};
  };
  auto scatter_e = [&](uint8_t* tb, auto kc, int u, int e) {  // step e of unit u (element e ^ m)
    constexpr int k = decltype(kc)::value;
    if (!uok[u]) return;
    if constexpr (FULL) {
      if (e == 0) *reinterpret_cast<u32x4_t*>(tb + ubase[u]) = pv[k][u];
    } else {
      // row within the group (masked to the group's span: a bad index byte
      // cannot address past the tile)
      const uint32_t rr = (pi[k][u][e >> 2] >> (8 * (e & 3))) & (BIGG ? 31u : 15u);
      *reinterpret_cast<uint16_t*>(tb + ((ubase[u] + grow(rr)) ^ (2u * static_cast<uint32_t>(e)))) =
          static_cast<uint16_t>(pv[k][u][e >> 1] >> (16 * (e & 1)));
    }
  };

  // ---- MFMAs ------------------------------------------------------------------
  // acc[pt][ot]: 16 pixels (tile pt of the wave's 64) x 16 outputs (tile ot
  // of its TO / 2).  A lane holds outputs 4 (lane / 16) .. +3 of pixel
  // lane % 16.
  f32x4_t acc[4][OT];
#pragma unroll
  for (int pt = 0; pt < 4; ++pt)
#pragma unroll
    for (int ot = 0; ot < OT; ++ot) acc[pt][ot] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int pt = 0; pt < 4; ++pt)
#pragma unroll
    for (int ot = 0; ot < OT; ++ot) acc_fence(acc[pt][ot]);
  mfma_drain();  // the zero writes land before the first MFMA reads them
  // B fragment (activations): pixel lane % 16, channels 8 (4 s + lane / 16) ..
  const uint32_t xl = static_cast<uint32_t>(lane & 15), xk = static_cast<uint32_t>(lane >> 4);
  const uint32_t swz = (xl >> 1) & 7u;
  const uint32_t boff0 = xl * 128u + ((xk ^ swz) << 4), boff1 = xl * 128u + (((4u + xk) ^ swz) << 4);
  auto ld = [](const uint8_t* q) { return *reinterpret_cast<const bf16x8_t*>(q); };

  // ---- pipeline -----------------------------------------------------------------
  // A wave's vector-memory operations are issued in pairs W(m), X(m) (packed
  // units into ring stage m % RW, activations into buffer m % NX), m = 0 ..
  // RW - 1 before the loop, then m = j + RW during chunk j: into the stage
  // and the buffer that chunk j-1 released.  Tile j+1 is built during chunk j
  // from stage (j+1) % RW.  Loads complete in issue order, so "X(j+1) has
  // landed" (and W(j+1) with it) is "at most the pairs issued after it are in
  // flight".
  constexpr int kPair = (FULL ? 1 : 2) * UPL + 4;  // vector-memory operations of one pair
  const int nch = p.nch;
  auto wait_pairs = [](int n) {  // at most n pairs in flight (n < RW)
    switch (n) {
      case 0: wait_vm<0>(); break;
      case 1: wait_vm<kPair>(); break;
      case 2: wait_vm<(RW > 2 ? 2 : 0) * kPair>(); break;
      case 3: wait_vm<(RW > 3 ? 3 : 0) * kPair>(); break;
      default: wait_vm<(RW > 4 ? 4 : 0) * kPair>(); break;
    }
  };
  static_assert(RW <= 5 && (RW - 1) * kPair < 64, "vmcnt range");
  for_k(std::make_integer_sequence<int, RW>{}, [&](auto kc) {
    if (decltype(kc)::value < nch) {
      load_w(decltype(kc)::value, kc);
      issue_x(decltype(kc)::value % NX);
    }
  });
  wait_pairs(min(RW, nch) - 1);  // W(0), X(0)
  w_fence(std::integral_constant<int, 0>{});
  for (int u = 0; u < UPL; ++u) permute_unit(std::integral_constant<int, 0>{}, u);
  if constexpr (!FULL)
    for (int i = 0; i < RPW / 8; ++i) zero_piece(lds + NX * kXB, i);
  for (int u = 0; u < UPL; ++u)
    for (int e = 0; e < 8; ++e) scatter_e(lds + NX * kXB, std::integral_constant<int, 0>{}, u, e);
  lds_barrier();

  // Chunk j with j % RW == k.  Its 32 MFMAs (k-step 0, then 1) are issued
  // one by one with the other work of the chunk placed between them (one
  // wave per SIMD issues in order):
  //   k-step 0: the k-step-1 fragments (slots 0-7), the zero fill of tile
  //     j+1 (slots 8-11), the pair W(j+RW), X(j+RW) (slots 12-15);
  //   then wait for W(j+1) and X(j+1);
  //   k-step 1: the kept weights of tile j+1 (8 UPL two-byte stores spread
  //     over the 16 slots);
  //   barrier: tile j+1 and X(j+1) are complete in every wave.
  // ST: the pair and tile j+1 exist and the wait is the steady-state one.
  auto step = [&](int j, auto kc, auto st) {
    constexpr int k = decltype(kc)::value;
    constexpr int k1 = (k + 1) % RW;
    constexpr bool ST = decltype(st)::value;
    const bool issue = ST || j + RW < nch;
    const bool next = ST || j + 1 < nch;
    const uint8_t* xb = lds + (j % NX) * kXB + wp * 8192;
    const uint8_t* wb = lds + NX * kXB + (j & 1) * WB + wo * (OT * 2048) + lane * 16;
    uint8_t* tb = lds + NX * kXB + ((j + 1) & 1) * WB;
    bf16x8_t fa[OT], fb[4], ga[OT], gb[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) fb[q] = ld(xb + q * 2048 + boff0);
#pragma unroll
    for (int q = 0; q < OT; ++q) fa[q] = ld(wb + (2 * q) * 1024);
#pragma unroll
    for (int i = 0; i < NMF; ++i) {
      mfma_acc(acc[i / OT][i % OT], fa[i % OT], fb[i / OT]);
      __builtin_amdgcn_sched_barrier(0);
      if (i < OT) ga[i] = ld(wb + (2 * i + 1) * 1024);
      if (i >= OT && i < OT + 4) gb[i - OT] = ld(xb + (i - OT) * 2048 + boff1);
      if constexpr (!FULL) {
        if (i >= NMF / 2 && i < NMF / 2 + RPW / 8 && next) zero_piece(tb, i - NMF / 2);
      }
      if (i == NMF - 4 && issue) load_w(j + RW, kc);
      if (i == NMF - 3 && issue) issue_x((j + RW) % NX);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (next) {
      if constexpr (ST) {
        wait_vm<(RW - 1) * kPair>();
      } else {
        wait_pairs(min(j + RW, nch - 1) - (j + 1));
      }
      w_fence(std::integral_constant<int, k1>{});
#pragma unroll
      for (int u = 0; u < UPL; ++u) permute_unit(std::integral_constant<int, k1>{}, u);
    }
#pragma unroll
    for (int i = 0; i < NMF; ++i) {
      mfma_acc(acc[i / OT][i % OT], ga[i % OT], gb[i / OT]);
      __builtin_amdgcn_sched_barrier(0);
      if (next) {
        // step q of the 8 UPL stores goes to slot q * NMF / (8 UPL)
#pragma unroll
        for (int q = 0; q < 8 * UPL; ++q)
          if ((q * NMF) / (8 * UPL) == i) scatter_e(tb, std::integral_constant<int, k1>{}, q >> 3, q & 7);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    lds_barrier();
  };
  // RW chunks per iteration of the steady state, so every ring stage index
  // is a constant; the tail (fewer than 2 RW chunks) starts again at stage 0.
  int j = 0;
#pragma unroll 1
  for (; j + 2 * RW - 1 < nch; j += RW)
    for_k(std::make_integer_sequence<int, RW>{},
          [&](auto kc) { step(j + decltype(kc)::value, kc, std::integral_constant<bool, true>{}); });
  for_k(std::make_integer_sequence<int, 2 * RW - 1>{}, [&](auto qc) {
    constexpr int q = decltype(qc)::value;
    if (j + q < nch) step(j + q, std::integral_constant<int, q % RW>{}, std::integral_constant<bool, false>{});
  });

  // ---- fused epilogue -----------------------------------------------------------
  // Each wave parks its 64 pixels x TO/2 outputs (fp32) in its own LDS region
  // (pitch TO/2 * 4 + 16 bytes: conflict-free both ways) and reads them back
  // by pixel rows: a lane then owns 8 consecutive outputs of one pixel (LPR
  // lanes cover the wave's TO/2), applies scale / bias / residual / ReLU in
  // fp32, rounds once and stores 16 (bf16) or 32 bytes.  (The loop's last
  // barrier has released the operand buffers.)
  constexpr int LPR = TO / 16;   // lanes per pixel row
  constexpr int RPP = 64 / LPR;  // rows per pass (LPR passes)
  mfma_drain();  // the last MFMAs have written acc
#pragma unroll
  for (int pt = 0; pt < 4; ++pt)
#pragma unroll
    for (int ot = 0; ot < OT; ++ot) acc_fence(acc[pt][ot]);
  constexpr uint32_t ysz = sizeof(YT);
  uint8_t* stg = lds + w * 64 * PITCH;
  const __amdgpu_buffer_rsrc_t yr =
      __builtin_amdgcn_make_buffer_rsrc(p.Y, (short)0, static_cast<int>(p.y_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rsr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(p.residual), (short)0, p.residual ? static_cast<int>(p.y_bytes) : 0, kRsrcWord3);
  const int c8 = lane % LPR;  // 8-output block of the wave's TO/2
  const uint32_t o = ob * TO + static_cast<uint32_t>(wo * (TO / 2) + 8 * c8);
  const auto row_off = [&](int rr) {  // Y / residual byte offset of the lane's row rr
    const uint32_t px = pb * kTP + static_cast<uint32_t>(wp * 64 + RPP * rr + lane / LPR);
    return px < static_cast<uint32_t>(p.N) ? (px * static_cast<uint32_t>(p.O) + o) * ysz : kOOB;
  };
  // bf16 residual: all rows' 16-byte pieces are requested before the
  // accumulators are parked (one load latency, not one per row)
  u32x4_t rres[LPR];
  if constexpr (ysz == 2) {
    if (p.residual) {
#pragma unroll
      for (int rr = 0; rr < LPR; ++rr)
        rres[rr] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rsr, row_off(rr), 0, 0));
    }
  }
#pragma unroll
  for (int pt = 0; pt < 4; ++pt)
#pragma unroll
    for (int ot = 0; ot < OT; ++ot)
      *reinterpret_cast<f32x4_t*>(stg + (pt * 16 + (lane & 15)) * PITCH + (ot * 16 + 4 * (lane >> 4)) * 4) =
          acc[pt][ot];
  f32x4_t sc0{1.f, 1.f, 1.f, 1.f}, sc1{1.f, 1.f, 1.f, 1.f}, bi0{0.f, 0.f, 0.f, 0.f}, bi1{0.f, 0.f, 0.f, 0.f};
  if (p.scale) {
    sc0 = *reinterpret_cast<const f32x4_t*>(p.scale + o);
    sc1 = *reinterpret_cast<const f32x4_t*>(p.scale + o + 4);
  }
  if (p.bias) {
    bi0 = *reinterpret_cast<const f32x4_t*>(p.bias + o);
    bi1 = *reinterpret_cast<const f32x4_t*>(p.bias + o + 4);
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this wave's staging writes have landed
#pragma unroll
  for (int rr = 0; rr < LPR; ++rr) {
    const int row = RPP * rr + lane / LPR;
    const uint8_t* src = stg + row * PITCH + c8 * 32;
    f32x4_t y0 = *reinterpret_cast<const f32x4_t*>(src);
    f32x4_t y1 = *reinterpret_cast<const f32x4_t*>(src + 16);
    const uint32_t off = row_off(rr);
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

template <typename YT, int UPL, bool FULL, bool BIGG, bool MASK, int NX, int TO>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(NX == 3 ? 2 : 1, NX == 3 ? 2 : 1)))
void tap_tile_kernel(TParams p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  tap_tile_body<YT, UPL, FULL, BIGG, MASK, NX, TO>(p, lds);
}

template <typename YT, int UPL, bool FULL, bool BIGG, bool MASK, int NX, int TO>
hipError_t launch_tn(const TParams& p, hipStream_t s) {
  static std::atomic<int8_t> lds_set[kMaxDevices];
  const hipError_t attr = set_lds_limit_once(
      lds_set, reinterpret_cast<const void*>(&tap_tile_kernel<YT, UPL, FULL, BIGG, MASK, NX, TO>), lds_bytes(NX, TO));
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((tap_tile_kernel<YT, UPL, FULL, BIGG, MASK, NX, TO>), dim3(8u * static_cast<uint32_t>(p.grid8)),
                     dim3(kThreads), lds_bytes(NX, TO), s, p);
  return hipGetLastError();
}

// Two workgroups per CU once the grid covers every CU twice; below that,
// one per CU with the deeper prefetch.
template <typename YT, int UPL, bool FULL, bool BIGG, bool MASK, int TO>
hipError_t launch_tu(const TParams& p, hipStream_t s) {
  return static_cast<uint32_t>(p.ntiles) >= kDeepGrid ? launch_tn<YT, UPL, FULL, BIGG, MASK, 3, TO>(p, s)
                                                       : launch_tn<YT, UPL, FULL, BIGG, MASK, 4, TO>(p, s);
}

template <typename YT, bool BIGG, int TO>
hipError_t launch_tg(const TParams& p, hipStream_t s) {
  // units per wave: 8 rows_w; per lane: rows_w / 8, rounded up (rows_w <= 16:
  // at most half of a group kept)
  if (p.rows_w < 8) return launch_tu<YT, 1, false, BIGG, true, TO>(p, s);
  if (p.rows_w == 8) return launch_tu<YT, 1, false, BIGG, false, TO>(p, s);
  if constexpr (TO == 128) {
    if (p.rows_w < 16) return launch_tu<YT, 2, false, BIGG, true, TO>(p, s);
    return launch_tu<YT, 2, false, BIGG, false, TO>(p, s);
  }
  return hipErrorInvalidConfiguration;  // (TO = 64: rows_w <= 8)
}

template <typename YT>
hipError_t launch_ty(const TParams& p, hipStream_t s, int to) {
  if (to == 64) {
    if (p.K == p.G) return launch_tu<YT, 2, true, false, false, 64>(p, s);
    return launch_tg<YT, false, 64>(p, s);
  }
  if (p.K == p.G) return launch_tu<YT, 4, true, false, false, 128>(p, s);
  return p.G == 32 ? launch_tg<YT, true, 128>(p, s) : launch_tg<YT, false, 128>(p, s);
}

}  // namespace

bool tap_tile_supports(const ProductArgs& a) {
  if (a.x_t != DType::BF16 || a.val_t != DType::BF16) return false;
  if (a.G < 1 || a.G > 32 || 32 % a.G != 0 || a.K < 1 || a.K > a.G) return false;
  // at most half of each group kept, or all of it (dense control): above
  // that the packed units no longer fit the registers beside the rings
  if (2 * a.K > a.G && a.K != a.G) return false;
  // O % 128 (tiles of 128 outputs), or O % 64 with G <= 16 (tiles of 64: a
  // group must fit one wave's 16 rows)
  if (a.N < 1 || a.O % 64 != 0 || (a.O % 128 != 0 && a.G > 16)) return false;
  const int64_t cin = a.conv ? a.geom.Cin : a.C;
  if (cin % kCK != 0) return false;
  if (a.conv && a.geom.KH * a.geom.KW > kMaxTaps) return false;
  const auto al = [](const void* q, uintptr_t m) { return (reinterpret_cast<uintptr_t>(q) & (m - 1)) == 0; };
  if (!al(a.X, 16) || !al(a.vals, 16) || !al(a.idx, 8) || !al(a.Y, 16)) return false;
  if ((a.scale && !al(a.scale, 16)) || (a.bias && !al(a.bias, 16)) || (a.residual && !al(a.residual, 16)))
    return false;
  // every buffer offset is 32-bit and stays below the out-of-range marker
  const int64_t lim = static_cast<int64_t>(kOOB);
  const int64_t x_elems = a.conv ? a.B * a.geom.H * a.geom.W * a.geom.Cin : a.N * a.C;
  const int64_t packed = (a.O / a.G) * a.K * a.C;
  if (x_elems * 2 >= lim || packed * 2 >= lim || a.N * a.O * (a.y_t == DType::F32 ? 4 : 2) >= lim) return false;
  return true;
}

hipError_t launch_tap_tile(const ProductArgs& a, hipStream_t s) {
  if (!tap_tile_supports(a)) return hipErrorInvalidConfiguration;
  TParams p{};
  p.X = static_cast<const uint16_t*>(a.X);
  p.vals = static_cast<const uint16_t*>(a.vals);
  p.idx = a.idx;
  p.scale = a.scale;
  p.bias = a.bias;
  p.residual = a.residual;
  p.Y = a.Y;
  const int64_t ysz = a.y_t == DType::F32 ? 4 : 2;
  const int64_t packed = (a.O / a.G) * a.K * a.C;
  if (a.conv) {
    const ConvGeom& g = a.geom;
    p.x_bytes = static_cast<uint32_t>(a.B * g.H * g.W * g.Cin * 2);
    p.H = g.H;
    p.W = g.W;
    p.Cin = g.Cin;
    p.KH = g.KH;
    p.KW = g.KW;
    p.sh = g.sh;
    p.sw = g.sw;
    p.ph = g.ph;
    p.pw = g.pw;
    p.HoWo = g.Ho * g.Wo;
    p.Wo = g.Wo;
  } else {  // N images of one pixel
    p.x_bytes = static_cast<uint32_t>(a.N * a.C * 2);
    p.H = p.W = 1;
    p.Cin = static_cast<int32_t>(a.C);
    p.KH = p.KW = 1;
    p.sh = p.sw = 1;
    p.ph = p.pw = 0;
    p.HoWo = p.Wo = 1;
  }
  p.v_bytes = static_cast<uint32_t>(packed * 2);
  p.i_bytes = static_cast<uint32_t>(packed);
  p.y_bytes = static_cast<uint32_t>(a.N * a.O * ysz);
  p.N = static_cast<int32_t>(a.N);
  p.C = static_cast<int32_t>(a.C);
  p.O = static_cast<int32_t>(a.O);
  p.G = a.G;
  p.K = a.K;
  p.relu = a.relu;
  p.npb = static_cast<int32_t>((a.N + kTP - 1) / kTP);
  // 128-output tiles, unless O is not a multiple of 128 or they would leave
  // more than half of the CUs idle and 64-output ones are possible (measured:
  // 3136 x 4608 x 512, 100 tiles, 51 -> 44 us; at 196 tiles the 64-output
  // plan is 10-15% slower)
  const int64_t grid128 = a.O % 128 == 0 ? static_cast<int64_t>(p.npb) * (a.O / 128) : 0;
  const int to = a.O % 128 == 0 && (grid128 >= kSmallGrid || a.G > 16) ? 128 : 64;
  p.nob = static_cast<int32_t>(a.O / to);
  p.nch = static_cast<int32_t>(a.C / kCK);
  p.cpt = p.Cin / kCK;
  p.rows_w = to / 4 * a.K / a.G;
  const int64_t grid = static_cast<int64_t>(p.npb) * p.nob;
  if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
  p.ntiles = static_cast<int32_t>(grid);
  p.grid8 = static_cast<int32_t>((grid + 7) / 8);
  return a.y_t == DType::BF16 ? launch_ty<bf16_t>(p, s, to) : launch_ty<float>(p, s, to);
}

}  // namespace cci
