// CCI-sparse product on the matrix cores, streaming plan: FC products and
// stride-1 1x1 convolutions with a short reduction (64 <= C <= 256) over
// many rows.
//
// A workgroup owns one tile of TO outputs (128, or 64 when O % 128 != 0)
// for the whole launch.  It expands the packed groups of those outputs over
// the whole reduction once (zero fill, then every kept weight written to row
// G*g + idx of its column: the routing of Alg. 1, Sec. 3.2) into a dense
// TO x C bf16 tile that stays in LDS, then streams a strided sequence of
// TP-row tiles of X past it.  Each 64-channel chunk of a row tile is one
// step: its activations are DMA'd into a ring of NR LDS buffers NR - 1 steps
// ahead and multiplied on v_mfma_f32_16x16x32_bf16; after a row tile's last
// chunk its outputs are finished in the accumulator layout (scale, bias,
// residual, ReLU, one rounding), staged through a few LDS rows per wave and
// stored as whole 128-byte lines while the next tile's chunks are already in
// flight.  The expansion and the launch are paid once per workgroup instead
// of once per tile, and no tile waits for its own activations.
// Work split: four waves, TP / 64 along the rows and the rest along the
// outputs; a wave accumulates 64 rows x its outputs in 16 x 16 accumulators
// (a lane holds outputs 4 (lane / 16) .. +3 of row lane % 16).
//
// LDS layouts (bytes):
//   weight tile, chunk c at c * TO * 128: 16-row block b, k-step s at
//     (2 b + s) * 1024, inside it (k / 8 % 4) * 256 + (o % 16) * 16 +
//     (k % 8) * 2, so the fragment a lane reads is its 16 bytes at lane * 16;
//   NR activation buffers of TP * 128 bytes after the weight tile: row q at
//     q * 128, its 16-byte column c holding channels 8 (c ^ ((q >> 1) % 8))
//     .. +7 of the chunk (a fragment read of 16 rows touches distinct bank
//     slots per 16 lanes);
//   scale and bias of the TO outputs (fp32);
//   per wave, 16 staged output rows at a pitch of their bytes + 16.
#include <algorithm>

#include "cci_device.hpp"
#include "cci_launch.hpp"

namespace cci {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kThreads = 256;           // four waves
constexpr int kCK = 64;                 // reduction columns per chunk (two k-steps)
constexpr int xb_bytes(int tp) { return tp * kCK * 2; }  // one activation buffer
constexpr int kMaxC = 256;              // the whole expanded tile stays in LDS
constexpr int kLdsMax = 160 * 1024;     // LDS of a CU
constexpr uint32_t kOOB = 0x80000000u;  // buffer offset that reads as zero / drops a store
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer descriptor word 3 (gfx9 family)
constexpr int wch_bytes(int to) { return to * kCK * 2; }
// one wave's epilogue staging: 16 rows of its TO / WO outputs in Y's type
// (ysz bytes each), padded by 16 bytes per row
constexpr int stage_pitch(int tp, int to, int ysz) { return to / (4 / (tp / 64)) * ysz + 16; }
// the weight tile, the ring of nr activation buffers, scale and bias of the
// TO outputs, then the four waves' staging rows
constexpr int lds_bytes(int nch, int tp, int to, int nr, int ysz) {
  return nch * wch_bytes(to) + nr * xb_bytes(tp) + 2 * to * 4 + 4 * 16 * stage_pitch(tp, to, ysz);
}

struct SParams {
  const uint16_t* X;
  const uint16_t* vals;
  const uint8_t* idx;
  const float* scale;
  const float* bias;
  const void* residual;
  void* Y;
  uint32_t x_bytes, y_bytes;
  int32_t N, C, O, G, K, relu;
  int32_t nch;  // C / 64
  int32_t npt;  // row tiles of TP
  int32_t nob;  // output tiles of TO
  int32_t s8;   // row-tile streams per XCD (each run by nob workgroups)
};

__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Wait until at most N vector-memory operations of this wave are in flight
// (they complete in issue order, loads and stores alike).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
// The same for a wave-uniform count n (a multiple of 4; above 60 it waits
// for 60, which is only stricter).
__device__ __forceinline__ void wait_vm_n(int n) {
  switch (min(n, 60) >> 2) {
    case 0: wait_vm<0>(); break;
    case 1: wait_vm<4>(); break;
    case 2: wait_vm<8>(); break;
    case 3: wait_vm<12>(); break;
    case 4: wait_vm<16>(); break;
    case 5: wait_vm<20>(); break;
    case 6: wait_vm<24>(); break;
    case 7: wait_vm<28>(); break;
    case 8: wait_vm<32>(); break;
    case 9: wait_vm<36>(); break;
    case 10: wait_vm<40>(); break;
    case 11: wait_vm<44>(); break;
    case 12: wait_vm<48>(); break;
    case 13: wait_vm<52>(); break;
    case 14: wait_vm<56>(); break;
    default: wait_vm<60>(); break;
  }
}

// acc = A * B (first k-step of a row tile) or acc += A * B, with the
// accumulator pinned to the accumulation registers.  Vector reads of acc are
// separated from the last MFMA by mfma_drain().
__device__ __forceinline__ void mfma_first(f32x4_t& acc, const bf16x8_t a, const bf16x8_t b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=a"(acc) : "v"(a), "v"(b));
}
__device__ __forceinline__ void mfma_acc(f32x4_t& acc, const bf16x8_t a, const bf16x8_t b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
__device__ __forceinline__ void mfma_drain() { asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 15\n\ts_nop 15" ::: "memory"); }
__device__ __forceinline__ void acc_fence(f32x4_t& acc) { asm volatile("" : "+a"(acc)); }

// Byte offset of tile row o in a weight-tile chunk, k-column 0.
__device__ __forceinline__ uint32_t trow(uint32_t o) { return ((o >> 4) << 11) | ((o & 15) << 4); }

template <typename YT, int TP, int TO, int NR>
__device__ __forceinline__ void stream_body(const SParams& p, uint8_t* lds) {
  // (64-row tiles with four waves along 256 outputs were measured no faster
  // and are not instantiated)
  static_assert(TP == 128, "row tiles of 128 rows");
  constexpr int D = NR - 1;             // prefetch distance in steps
  constexpr int WP = TP / 64;           // waves along the rows (64 each)
  constexpr int WO = 4 / WP;            // waves along the outputs
  constexpr int OT = TO / (16 * WO);    // 16-output tiles per wave
  constexpr int XB = xb_bytes(TP);
  constexpr int NDI = TP / 32;          // DMA instructions of one chunk per wave
  constexpr int WCH = wch_bytes(TO);    // one chunk of the weight tile
  constexpr uint32_t ysz = sizeof(YT);
  static_assert(OT % 2 == 0, "residual loads take output tiles in pairs");
  constexpr int NRS = (ysz == 2 ? 2 : 4) * OT;  // residual loads (16 bytes) per wave and row tile
  constexpr int SP = stage_pitch(TP, TO, ysz);
  constexpr int LPR = (TO / WO) * ysz / 16;  // lanes per staged row (16 bytes each)
  constexpr int RPP = 64 / LPR;         // staged rows per pass
  constexpr int NST = 4 * (16 / RPP);   // stores per wave and row tile
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wp = w / WO, wo = w % WO;

  // ---- work of this workgroup ------------------------------------------------
  // Dispatch places workgroup b on XCD b % 8.  The nob workgroups of one
  // stream (one per output tile) are on one XCD and read the same row tiles
  // st, st + NS, ... at about the same time, so X comes from HBM once.
  const uint32_t bid = blockIdx.x;
  const uint32_t xcd = bid & 7u, slot = bid >> 3;
  const uint32_t nob = static_cast<uint32_t>(p.nob);
  const uint32_t ob = slot % nob;
  const uint32_t ns = 8u * static_cast<uint32_t>(p.s8);
  const uint32_t st = xcd * static_cast<uint32_t>(p.s8) + slot / nob;
  const uint32_t npt = static_cast<uint32_t>(p.npt);
  if (st >= npt) return;
  const int nt = static_cast<int>((npt - st + ns - 1) / ns);  // row tiles of this workgroup
  const int nch = p.nch;
  const int S = nt * nch;  // steps

  uint8_t* wt = lds;
  uint8_t* xring = lds + nch * WCH;
  float* sbs = reinterpret_cast<float*>(xring + NR * XB);  // scale [TO], bias [TO]
  uint8_t* stg = reinterpret_cast<uint8_t*>(sbs + 2 * TO) + w * 16 * SP;  // this wave's staging

  // ---- activation DMA ---------------------------------------------------------
  // Instruction i of wave w fills rows (4 w + i) * 8 .. +7 of a buffer: lane l
  // writes the 16 bytes at (4 w + i) * 1024 + 16 l, i.e. row q = (4 w + i) * 8
  // + l / 8, column l % 8, holding channel block (l % 8) ^ ((q >> 1) % 8).
  // Rows past N read as zero.
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.X), (short)0, static_cast<int>(p.x_bytes), kRsrcWord3);
  uint32_t xq[NDI], xk[NDI];
#pragma unroll
  for (int i = 0; i < NDI; ++i) {
    const uint32_t q = static_cast<uint32_t>((NDI * w + i) * 8 + (lane >> 3));
    xq[i] = q;
    xk[i] = (static_cast<uint32_t>(lane & 7) ^ ((q >> 1) & 7u)) * 16u;
  }
  int dma_k = 0, dma_c = 0, dma_b = 0;  // row tile (of this workgroup), chunk and buffer of the next DMA
  auto issue_x = [&]() {
    const uint32_t pt = st + static_cast<uint32_t>(dma_k) * ns;
    uint8_t* dst = xring + dma_b * XB + w * (NDI * 1024);
#pragma unroll
    for (int i = 0; i < NDI; ++i) {
      const uint32_t px = pt * TP + xq[i];
      const uint32_t off = px < static_cast<uint32_t>(p.N)
                               ? px * static_cast<uint32_t>(p.C) * 2u + static_cast<uint32_t>(dma_c) * 128u + xk[i]
                               : kOOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t*)(dst + i * 1024), 16, off, 0, 0, 0);
    }
    if (++dma_c == nch) {
      dma_c = 0;
      ++dma_k;
    }
    dma_b = dma_b == NR - 1 ? 0 : dma_b + 1;
  };

  // ---- prologue: first D chunks in flight, epilogue constants, the tile ----
  for (int m = 0; m < D && m < S; ++m) issue_x();
  __builtin_amdgcn_sched_barrier(0);
  // outputs of the lane's accumulator rows: obase + 16 ot + 0..3
  const uint32_t ocol = static_cast<uint32_t>(wo * (TO / WO) + 4 * (lane >> 4));  // in the tile
  const uint32_t obase = ob * TO + ocol;
  if (threadIdx.x < TO) {
    const uint32_t o = ob * TO + threadIdx.x;
    sbs[threadIdx.x] = p.scale ? p.scale[o] : 1.0f;
    sbs[TO + threadIdx.x] = p.bias ? p.bias[o] : 0.0f;
  }
  // Zero the expanded tile, then write every kept weight of the workgroup's
  // TO / G groups: thread t takes column t of each packed row.
  for (int b = static_cast<int>(threadIdx.x) * 16; b < nch * WCH; b += kThreads * 16)
    *reinterpret_cast<u32x4_t*>(wt + b) = u32x4_t{0u, 0u, 0u, 0u};
  lds_barrier();
  {
    const int c = static_cast<int>(threadIdx.x);
    const int rows = (TO / p.G) * p.K;
    if (c < p.C) {
      const uint32_t kk = static_cast<uint32_t>(c & 63);
      const uint32_t cpos = static_cast<uint32_t>(c >> 6) * WCH + (kk >> 5) * 1024u + ((kk >> 3) & 3u) * 256u + (kk & 7u) * 2u;
      const int64_t prow0 = static_cast<int64_t>(ob) * rows;
      const uint32_t gm = static_cast<uint32_t>(p.G - 1);
#pragma unroll 4
      for (int r = 0; r < rows; ++r) {
        const int64_t e = (prow0 + r) * p.C + c;
        const uint16_t v = p.vals[e];
        const uint32_t o = static_cast<uint32_t>((r / p.K) * p.G) + (static_cast<uint32_t>(p.idx[e]) & gm);
        *reinterpret_cast<uint16_t*>(wt + cpos + trow(o)) = v;
      }
    }
  }
  wait_vm<0>();  // this wave's first DMAs (and every prologue load) have landed
  lds_barrier();

  // ---- steps --------------------------------------------------------------------
  const __amdgpu_buffer_rsrc_t yr =
      __builtin_amdgcn_make_buffer_rsrc(p.Y, (short)0, static_cast<int>(p.y_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rsr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(p.residual), (short)0, p.residual ? static_cast<int>(p.y_bytes) : 0, kRsrcWord3);
  const bool has_res = p.residual != nullptr;
  // Y / residual byte offset of the lane's accumulator row pt, output tile ot
  // in row tile k
  auto y_off = [&](int k, int pt, int ot) {
    const uint32_t px = (st + static_cast<uint32_t>(k) * ns) * TP +
                        static_cast<uint32_t>(wp * 64 + pt * 16 + (lane & 15));
    return px < static_cast<uint32_t>(p.N) ? (px * static_cast<uint32_t>(p.O) + obase + 16u * ot) * ysz : kOOB;
  };
  // residual: for bf16, lane l loads the 16 bytes of outputs 8 (q / 2) .. +7
  // of tile ot + (q odd) for each tile pair (q = lane / 16); its partner
  // l ^ 16 holds the other halves (exchanged in the epilogue); for fp32 the
  // lane's own 4 outputs per tile
  u32x4_t res[4][OT];
  const bool qodd = (lane >> 4) & 1;
  auto r_off = [&](int k, int pt, int otp) {  // bf16: byte offset of the lane's 16 residual bytes
    const uint32_t px = (st + static_cast<uint32_t>(k) * ns) * TP +
                        static_cast<uint32_t>(wp * 64 + pt * 16 + (lane & 15));
    const uint32_t o = ob * TO + static_cast<uint32_t>(wo * (TO / WO) + 16 * otp + (qodd ? 16 : 0) + 8 * (lane >> 5));
    return px < static_cast<uint32_t>(p.N) ? (px * static_cast<uint32_t>(p.O) + o) * ysz : kOOB;
  };

  f32x4_t acc[4][OT];
  const uint32_t xl = static_cast<uint32_t>(lane & 15), xkq = static_cast<uint32_t>(lane >> 4);
  const uint32_t swz = (xl >> 1) & 7u;
  const uint32_t boff0 = xl * 128u + ((xkq ^ swz) << 4), boff1 = xl * 128u + (((4u + xkq) ^ swz) << 4);
  auto ld = [](const uint8_t* q) { return *reinterpret_cast<const bf16x8_t*>(q); };

  // Vector-memory operations each step issues after its top wait, in this
  // order: the residual loads of a row tile (NRS, in the step before the
  // tile's last, or in the last when a tile is one chunk), the DMA of step
  // s + D (NDI, while there is one), and after the last chunk of a tile its
  // stores (NST).  The top wait of step s needs the DMA of step s, issued
  // in step s - D: at most the operations issued after it may be in flight.
  auto res_step = [&](int s) {  // does step s load a row tile's residual?
    if (!has_res) return false;
    const int c = s % nch;
    return nch == 1 || c == nch - 2;
  };
  auto ops_pre = [&](int s) { return res_step(s) ? NRS : 0; };
  auto ops_x = [&](int s) { return s + D < S ? NDI : 0; };
  auto ops_post = [&](int s) { return s % nch == nch - 1 ? NST : 0; };

  int cc = 0, kt = 0, buf = 0;  // chunk, row tile (of this workgroup), activation buffer of step s
#pragma unroll 1
  for (int s = 0; s < S; ++s) {
    if (s >= D) {
      int n = ops_post(s - D);
      for (int j = s - D + 1; j < s; ++j) n += ops_pre(j) + ops_x(j) + ops_post(j);
      wait_vm_n(n);
    }
    lds_barrier();  // the chunk is in LDS for every wave; step s-1's buffer is free
    __builtin_amdgcn_sched_barrier(0);
    if (res_step(s)) {
#pragma unroll
      for (int pt = 0; pt < 4; ++pt)
#pragma unroll
        for (int ot = 0; ot < OT; ot += 2) {
          if constexpr (ysz == 2) {
            res[pt][ot] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rsr, r_off(kt, pt, ot), 0, 0));
          } else {
            res[pt][ot] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rsr, y_off(kt, pt, ot), 0, 0));
            res[pt][ot + 1] =
                __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rsr, y_off(kt, pt, ot + 1), 0, 0));
          }
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    if (s + D < S) issue_x();
    __builtin_amdgcn_sched_barrier(0);

    const uint8_t* xb = xring + buf * XB + wp * 8192;
    const uint8_t* wb = wt + cc * WCH + wo * (OT * 2048) + lane * 16;
    bf16x8_t fa[OT], fb[4], ga[OT], gb[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) fb[q] = ld(xb + q * 2048 + boff0);
#pragma unroll
    for (int q = 0; q < OT; ++q) fa[q] = ld(wb + (2 * q) * 1024);
#pragma unroll
    for (int q = 0; q < OT; ++q) ga[q] = ld(wb + (2 * q + 1) * 1024);
#pragma unroll
    for (int q = 0; q < 4; ++q) gb[q] = ld(xb + q * 2048 + boff1);
    if (cc == 0) {
#pragma unroll
      for (int i = 0; i < 4 * OT; ++i) mfma_first(acc[i / OT][i % OT], fa[i % OT], fb[i / OT]);
    } else {
#pragma unroll
      for (int i = 0; i < 4 * OT; ++i) mfma_acc(acc[i / OT][i % OT], fa[i % OT], fb[i / OT]);
    }
#pragma unroll
    for (int i = 0; i < 4 * OT; ++i) mfma_acc(acc[i / OT][i % OT], ga[i % OT], gb[i / OT]);
    __builtin_amdgcn_sched_barrier(0);

    if (cc == nch - 1) {
      // ---- fused epilogue of row tile kt, in the accumulator layout ----------
      mfma_drain();
#pragma unroll
      for (int pt = 0; pt < 4; ++pt)
#pragma unroll
        for (int ot = 0; ot < OT; ++ot) acc_fence(acc[pt][ot]);
      // Each 16-row slab is finished in the accumulator layout, rounded,
      // staged in this wave's LDS rows and stored as 16-byte pieces, LPR
      // lanes per row (whole 128-byte lines of Y).  (A wave's LDS operations
      // complete in order, so the next slab's writes follow this slab's
      // reads.)
      const uint32_t row0 = (st + static_cast<uint32_t>(kt) * ns) * TP + static_cast<uint32_t>(wp * 64);
      const uint32_t col_b = (ob * TO + static_cast<uint32_t>(wo * (TO / WO))) * ysz + static_cast<uint32_t>(lane % LPR) * 16u;
#pragma unroll
      for (int pt = 0; pt < 4; ++pt) {
        u32x2_t rl[OT];  // bf16 residual of the lane's 4 outputs per tile
        if constexpr (ysz == 2) {
          if (has_res) {
            // even lane: loaded tile ot's 0..7 (of its 16-output group) and
            // keeps 0..3, sends 4..7, receives the partner's tile ot+1 0..3;
            // odd lane: loaded tile ot+1's, keeps 4..7 (ds_swizzle xor 16)
#pragma unroll
            for (int ot = 0; ot < OT; ot += 2) {
              const u32x4_t L = res[pt][ot];
              const uint32_t s0 = qodd ? L[0] : L[2], s1 = qodd ? L[1] : L[3];
              const uint32_t r0 = static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(static_cast<int>(s0), 0x401F));
              const uint32_t r1 = static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(static_cast<int>(s1), 0x401F));
              rl[ot] = qodd ? u32x2_t{r0, r1} : u32x2_t{L[0], L[1]};
              rl[ot + 1] = qodd ? u32x2_t{L[2], L[3]} : u32x2_t{r0, r1};
            }
          }
        }
#pragma unroll
        for (int ot = 0; ot < OT; ++ot) {
          const f32x4_t sc = *reinterpret_cast<const f32x4_t*>(sbs + ocol + 16 * ot);
          const f32x4_t bi = *reinterpret_cast<const f32x4_t*>(sbs + TO + ocol + 16 * ot);
          f32x4_t y = acc[pt][ot] * sc + bi;
          if (has_res) {
            if constexpr (ysz == 2) {
              const u32x2_t r = rl[ot];
              y[0] += __uint_as_float(r[0] << 16);
              y[1] += __uint_as_float(r[0] & 0xffff0000u);
              y[2] += __uint_as_float(r[1] << 16);
              y[3] += __uint_as_float(r[1] & 0xffff0000u);
            } else {
              y += __builtin_bit_cast(f32x4_t, res[pt][ot]);
            }
          }
          if (p.relu) {
#pragma unroll
            for (int e = 0; e < 4; ++e) y[e] = y[e] > 0.0f ? y[e] : (y[e] != y[e] ? y[e] : 0.0f);
          }
          uint8_t* sp = stg + (lane & 15) * SP + (ot * 16 + 4 * (lane >> 4)) * ysz;
          if constexpr (ysz == 2) {
            // v_cvt_pk_bf16_f32: round to nearest even
            *reinterpret_cast<u32x2_t*>(sp) =
                u32x2_t{__builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y[0], y[1]}), bf16x2_t)),
                        __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y[2], y[3]}), bf16x2_t))};
          } else {
            *reinterpret_cast<f32x4_t*>(sp) = y;
          }
        }
#pragma unroll
        for (int ps = 0; ps < 16 / RPP; ++ps) {
          const int row = ps * RPP + lane / LPR;
          const u32x4_t v = *reinterpret_cast<const u32x4_t*>(stg + row * SP + (lane % LPR) * 16);
          const uint32_t px = row0 + static_cast<uint32_t>(pt * 16 + row);
          const uint32_t off = px < static_cast<uint32_t>(p.N) ? px * static_cast<uint32_t>(p.O) * ysz + col_b : kOOB;
          __builtin_amdgcn_raw_buffer_store_b128(
              __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(yr, 0, 0, 0)), v), yr, off, 0, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (++cc == nch) {
      cc = 0;
      ++kt;
    }
    buf = buf == NR - 1 ? 0 : buf + 1;
  }
}

template <typename YT, int TP, int TO, bool TWO>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(TWO ? 2 : 1, TWO ? 2 : 1)))
void stream_tile_kernel(SParams p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  stream_body<YT, TP, TO, 3>(p, lds);
}

int device_cus() {
  static std::atomic<int> cached[kMaxDevices];
  const int dev = current_device();
  if (dev >= 0) {
    const int c = cached[dev].load(std::memory_order_acquire);
    if (c > 0) return c;
  }
  int cus = 0;
  if (dev >= 0 && hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus >= 1) {
    cached[dev].store(cus, std::memory_order_release);
    return cus;
  }
  return 256;
}

template <typename YT, int TP, int TO, bool TWO>
hipError_t launch_st(SParams p, hipStream_t s) {
  static std::atomic<int8_t> lds_set[kMaxDevices];
  const int lds = lds_bytes(p.nch, TP, TO, 3, sizeof(YT));
  const hipError_t attr = set_lds_limit_once(
      lds_set, reinterpret_cast<const void*>(&stream_tile_kernel<YT, TP, TO, TWO>),
      std::min(lds_bytes(kMaxC / kCK, TP, TO, 3, sizeof(YT)), kLdsMax));
  if (attr != hipSuccess) return attr;
  // workgroups resident at once: two per CU when their LDS fits twice
  const int64_t slots = static_cast<int64_t>(device_cus()) * (TWO ? 2 : 1);
  const int64_t per_xcd = std::max<int64_t>(1, slots / (8 * static_cast<int64_t>(p.nob)));
  p.s8 = static_cast<int32_t>(std::min<int64_t>(per_xcd, (static_cast<int64_t>(p.npt) + 7) / 8));
  const uint32_t grid = 8u * static_cast<uint32_t>(p.nob) * static_cast<uint32_t>(p.s8);
  hipLaunchKernelGGL((stream_tile_kernel<YT, TP, TO, TWO>), dim3(grid), dim3(kThreads), lds, s, p);
  return hipGetLastError();
}

template <typename YT, int TP, int TO>
hipError_t launch_sr(SParams p, int64_t N, hipStream_t s) {
  p.npt = static_cast<int32_t>((N + TP - 1) / TP);
  p.nob = p.O / TO;
  return 2 * lds_bytes(p.nch, TP, TO, 3, sizeof(YT)) <= kLdsMax ? launch_st<YT, TP, TO, true>(p, s)
                                                       : launch_st<YT, TP, TO, false>(p, s);
}

template <typename YT>
hipError_t launch_sy(const SParams& p, int64_t N, hipStream_t s) {
  if (p.O % 128 == 0) return launch_sr<YT, 128, 128>(p, N, s);
  return launch_sr<YT, 128, 64>(p, N, s);
}

}  // namespace

bool stream_tile_supports(const ProductArgs& a) {
  if (a.x_t != DType::BF16 || a.val_t != DType::BF16) return false;
  if (a.G < 1 || a.G > 32 || 32 % a.G != 0 || a.K < 1 || a.K > a.G) return false;
  if (a.conv) {
    const ConvGeom& g = a.geom;
    if (g.KH != 1 || g.KW != 1 || g.sh != 1 || g.sw != 1 || g.ph != 0 || g.pw != 0) return false;
  }
  if (a.N < 1 || a.C % kCK != 0 || a.C > kMaxC || a.O % 64 != 0) return false;
  const auto al = [](const void* q, uintptr_t m) { return (reinterpret_cast<uintptr_t>(q) & (m - 1)) == 0; };
  const uintptr_t ya = a.y_t == DType::F32 ? 16 : 8;
  if (!al(a.X, 16) || !al(a.Y, ya) || (a.residual && !al(a.residual, ya))) return false;
  if ((a.scale && !al(a.scale, 16)) || (a.bias && !al(a.bias, 16))) return false;
  // every buffer offset is 32-bit and stays below the out-of-range marker
  const int64_t lim = static_cast<int64_t>(kOOB);
  if (a.N * a.C * 2 >= lim || a.N * a.O * (a.y_t == DType::F32 ? 4 : 2) >= lim) return false;
  return true;
}

hipError_t launch_stream_tile(const ProductArgs& a, hipStream_t s) {
  if (!stream_tile_supports(a)) return hipErrorInvalidConfiguration;
  SParams p{};
  p.X = static_cast<const uint16_t*>(a.X);
  p.vals = static_cast<const uint16_t*>(a.vals);
  p.idx = a.idx;
  p.scale = a.scale;
  p.bias = a.bias;
  p.residual = a.residual;
  p.Y = a.Y;
  p.x_bytes = static_cast<uint32_t>(a.N * a.C * 2);
  p.y_bytes = static_cast<uint32_t>(a.N * a.O * (a.y_t == DType::F32 ? 4 : 2));
  p.N = static_cast<int32_t>(a.N);
  p.C = static_cast<int32_t>(a.C);
  p.O = static_cast<int32_t>(a.O);
  p.G = a.G;
  p.K = a.K;
  p.relu = a.relu;
  p.nch = static_cast<int32_t>(a.C / kCK);
  return a.y_t == DType::BF16 ? launch_sy<bf16_t>(p, a.N, s) : launch_sy<float>(p, a.N, s);
}

}  // namespace cci
