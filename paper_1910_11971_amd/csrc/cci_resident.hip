// CCI-sparse k x k convolutions with unit stride and few outputs -- the 3x3
// layers of a CNN's first stage (Cin 32 or 64, 32 or 64 outputs) -- on the
// matrix cores, with the expanded weights resident in registers.
//
// The method is that of the other matrix-core kernels: Alg. 1's target row
// G g + idx[g][k][c] receives vals[g][k][c] (Sec. 3.2), i.e. the packed groups
// expand into the dense masked weight tile, and the tile is multiplied on
// v_mfma_f32_16x16x32_bf16 against activations read through implicit im2col
// (the convolution lowered to a product, Sec. 3.2, never materialised).
// What differs is the schedule.  A layer this small has an expanded tile of at
// most 64 x 576 bf16 (72 KiB): one copy fits in the registers of the two
// waves that share a SIMD, so it is expanded once per workgroup and never
// again, and nothing but activations moves during the product:
//
//   - prologue: the packed groups are loaded into registers before any
//     activation traffic is queued (so they do not wait behind it), scattered
//     into a zero-filled LDS tile in MFMA fragment order, and each wave reads
//     its fragments: wave w holds outputs 32 (w / streams) .. +31 over the
//     whole reduction (2 x S fragments, S = KH*KW*Cin / 32);
//   - a workgroup owns a band of R output rows of one image.  At the start
//     every input row under the band -- R + KH - 1 rows, each with the
//     padding columns, padding rows and columns reading as zero -- is DMA'd
//     from HBM into LDS (buffer_load ... lds), so each activation is read from
//     HBM once per band;
//   - the band's 16-pixel tiles are dealt to the pixel streams (four when two
//     waves split 64 outputs, eight for 32 outputs), which run without
//     further synchronisation once the staged rows have landed;
//   - each lane's B fragment is 8 channels of one input pixel; an input row
//     stores pixel q's 16-byte channel chunk c at slot
//         q * cpp + (c ^ ((q * cpp / 16) mod cpp))        (cpp = Cin / 8)
//     which keeps a DMA instruction on 1 KiB of contiguous activations and
//     gives every quarter-wave and half-wave of a fragment read distinct
//     16-byte slots modulo 256 and 512 bytes (no bank conflicts) whenever its
//     16 pixels sit in one output row;
//   - the fused epilogue (scale and bias staged in LDS, residual, ReLU, one
//     round-to-nearest-even) writes each lane's 4 consecutive outputs of one
//     pixel.
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

constexpr int kThreads = 512;        // 8 waves, two per SIMD
constexpr int kWaves = 8;
constexpr int kUnitsMax = 10;        // packed 8-column units per thread (64 x 640 dense)
constexpr int kEpiBytes = 1024;      // LDS: scale[64], bias[64], a dummy word at the end
constexpr int kLdsMax = 160 * 1024;
constexpr int kXcds = 8;
constexpr uint32_t kOOB = 0x80000000u;  // buffer offset that reads as zero / drops a store
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer descriptor word 3 (gfx9 family)

struct RParams {
  const uint16_t* X;
  const uint16_t* vals;
  const uint8_t* idx;
  const float* scale;
  const float* bias;
  const void* residual;
  void* Y;
  uint32_t x_bytes, y_bytes, p_elems;  // buffer extents: bytes, bytes, packed elements
  int32_t O, G, K, relu;
  int32_t H, W, Ho, Wo, ph, pw;
  int32_t R;          // output rows per band
  int32_t bpi;        // bands per image
  int32_t grid8;      // bands / 8 when that divides (neighbouring bands on one XCD), else 0
  int32_t streams;    // pixel streams: 8 / (O / 32)
  int32_t pcols;      // staged input columns: Wo + KW - 1
  int32_t row_bytes;  // LDS bytes of one staged input row (the kernel's RP: 8 or 16 KiB)
  uint32_t wo_mul;    // n / Wo == umulhi(n, wo_mul) + (n & wo_one) for the band's pixels:
  uint32_t wo_one;    //   floor(2^32 / Wo) + 1 and 0, or 0 and all ones when Wo == 1
  int32_t dpr;        // DMA instructions per staged row (1 KiB each, covering its used part)
  int32_t wt_bytes;   // LDS bytes of the expanded tile: O * C * 2
  int32_t ring_bytes; // LDS bytes of the staged rows: (R + KH - 1) * row_bytes
  int32_t nunits;     // packed 8-column units: (O / G) * K * C / 8
  int32_t rows_a;     // output rows of phase A (its tiles start before the band's later rows land)
};

// Wait until at most N vector-memory operations of this wave are in flight
// (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
// The same with a wave-uniform run-time bound; bounds above 31 wait for 31
// (waiting for more operations than needed is always safe).
__device__ __forceinline__ void wait_vm_dyn(int n) {
  n = n < 0 ? 0 : (n > 31 ? 31 : n);
  switch (n) {
#define CCI_WAIT_CASE(k) \
  case k: wait_vm<k>(); break;
    CCI_WAIT_CASE(0) CCI_WAIT_CASE(1) CCI_WAIT_CASE(2) CCI_WAIT_CASE(3) CCI_WAIT_CASE(4) CCI_WAIT_CASE(5)
    CCI_WAIT_CASE(6) CCI_WAIT_CASE(7) CCI_WAIT_CASE(8) CCI_WAIT_CASE(9) CCI_WAIT_CASE(10) CCI_WAIT_CASE(11)
    CCI_WAIT_CASE(12) CCI_WAIT_CASE(13) CCI_WAIT_CASE(14) CCI_WAIT_CASE(15) CCI_WAIT_CASE(16) CCI_WAIT_CASE(17)
    CCI_WAIT_CASE(18) CCI_WAIT_CASE(19) CCI_WAIT_CASE(20) CCI_WAIT_CASE(21) CCI_WAIT_CASE(22) CCI_WAIT_CASE(23)
    CCI_WAIT_CASE(24) CCI_WAIT_CASE(25) CCI_WAIT_CASE(26) CCI_WAIT_CASE(27) CCI_WAIT_CASE(28) CCI_WAIT_CASE(29)
    CCI_WAIT_CASE(30)
#undef CCI_WAIT_CASE
    default: wait_vm<31>(); break;
  }
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
__device__ __forceinline__ void barrier_only() { asm volatile("s_barrier" ::: "memory"); }

// Packed-weight and epilogue-operand loads, issued as plain instructions: the
// compiler does not track them as pending (it would otherwise wait for every
// activation DMA issued after them before their first use); the kernel waits
// for them itself with wait_vm<> before any use.
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

__device__ __forceinline__ float relu_f(float y) { return y > 0.0f ? y : (y != y ? y : 0.0f); }

// KH x KW taps over CPP 16-byte chunks (8 channels each) per input pixel.
template <typename YT, int KH, int KW, int CPP, int RP, bool RES>
__device__ __forceinline__ void resident_body(const RParams& p, uint8_t* lds) {
  constexpr int C = KH * KW * CPP * 8;  // reduction length
  constexpr int C8 = C / 8;             // 8-column units per packed row
  constexpr int S = C / 32;             // k-steps of 32 columns
  constexpr int CB = CPP / 4;           // k-steps per tap
  constexpr uint32_t ysz = sizeof(YT);
  static_assert(CPP == 4 || CPP == 8, "Cin 32 or 64");

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int streams = p.streams;
  const int slice = wave / streams;  // outputs 32 slice .. 32 slice + 31
  const int stream = wave - slice * streams;

  // ---- the band: R output rows of one image (neighbouring bands on one XCD
  // share their halo rows through its L2) ----------------------------------
  const uint32_t id = blockIdx.x;
  const int band = p.grid8 ? static_cast<int>((id % kXcds) * static_cast<uint32_t>(p.grid8) + id / kXcds)
                           : static_cast<int>(id);
  const int img = band / p.bpi;
  const int oh0 = (band - img * p.bpi) * p.R;
  const int rows = min(p.R, p.Ho - oh0);
  const int npix = rows * p.Wo;
  const int nrows = rows + KH - 1;  // staged input rows
  const int ih0 = oh0 - p.ph;       // input row of staged row 0
  uint8_t* const ring = lds + p.wt_bytes;  // staged row r at ring + r * RP
  float* const epi = reinterpret_cast<float*>(lds + p.wt_bytes + p.ring_bytes);

  // ---- packed groups and epilogue operands into registers -----------------
  // Unit u = packed elements 8 u .. 8 u + 7 (row u / C8, columns 8 (u % C8) ..).
  const u32x4_t vd = sdesc(p.vals, p.p_elems * 2u), idd = sdesc(p.idx, p.p_elems);
  u32x4_t pv[kUnitsMax];
  u32x2_t pi[kUnitsMax];
  // (a wave issues only the loads of units some lane of it has)
  const auto wave_has = [&](int u) { return u * kThreads + wave * 64 < p.nunits; };
#pragma unroll
  for (int u = 0; u < kUnitsMax; ++u) {
    if (wave_has(u)) {
      const uint32_t unit = threadIdx.x + static_cast<uint32_t>(u * kThreads);
      const bool ok = unit < static_cast<uint32_t>(p.nunits);
      pv[u] = load_x4(vd, ok ? unit * 16u : kOOB);
      pi[u] = load_x2(idd, ok ? unit * 8u : kOOB);
    }
  }
  // thread t < O / 4 stages scale and bias of outputs 4 t .. 4 t + 3
  const bool epi_t = static_cast<int>(threadIdx.x) * 4 < p.O;
  const u32x4_t sd = sdesc(p.scale, p.scale ? static_cast<uint32_t>(p.O) * 4u : 0u);
  const u32x4_t bd = sdesc(p.bias, p.bias ? static_cast<uint32_t>(p.O) * 4u : 0u);
  const uint32_t eoff = epi_t ? threadIdx.x * 16u : kOOB;
  const u32x4_t sc_raw = load_x4(sd, eoff);  // (absent scale / bias: a zero-length buffer, reads 0)
  const u32x4_t bi_raw = load_x4(bd, eoff);

  // ---- activation DMA, in row order ----------------------------------------
  // Wave w issues instructions f = w, w + 8, ... of the (row, j) sequence of a
  // batch of rows; instruction (r, j) fills slots 64 j .. 64 j + 63 of staged
  // row r.  The first batch -- the rows the first tiles read -- is queued
  // now, the rest once the weights are expanded.
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.X), (short)0, static_cast<int>(p.x_bytes), kRsrcWord3);
  const auto dma_rows = [&](int r0, int r1) {  // returns this wave's instruction count
    int n = 0;
    for (int f = r0 * p.dpr + wave; f < r1 * p.dpr; f += kWaves) {
      const int r = f / p.dpr;
      const int j = f - r * p.dpr;
      const uint32_t s = static_cast<uint32_t>(j * 64 + lane);
      const uint32_t q = s / CPP;                                  // staged column
      const uint32_t c = (s & (CPP - 1)) ^ ((s >> 4) & (CPP - 1));  // channel chunk held by slot s
      const int iw = static_cast<int>(q) - p.pw;
      const int ih = ih0 + r;
      const bool ok = q < static_cast<uint32_t>(p.pcols) && ih >= 0 && ih < p.H && iw >= 0 && iw < p.W;
      const uint32_t off =
          ok ? ((static_cast<uint32_t>(img * p.H + ih) * static_cast<uint32_t>(p.W) + static_cast<uint32_t>(iw)) *
                    static_cast<uint32_t>(CPP * 8) + c * 8u) * 2u
             : kOOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t*)(ring + r * RP + j * 1024), 16, off, 0, 0, 0);
      ++n;
    }
    return n;
  };
  // phase A: the tiles whose rows all lie in the first r1 staged rows
  const int r1 = min(nrows, p.rows_a + KH - 1);
  const int tiles_a = min((npix + 15) >> 4, (p.rows_a * p.Wo) >> 4);
  const int ndma_a = dma_rows(0, r1);

  // ---- expand the packed groups into the LDS tile (fragment order) -------
  // Fragment (o / 16, s) of 16 outputs x 32 columns is 1 KiB at
  // ((o / 16) * S + s) * 1024; element (o % 16, kk) of it at
  // ((kk / 8) * 16 + o % 16) * 16 + (kk % 8) * 2: lane l reads bytes 16 l ..
  for (int i = static_cast<int>(threadIdx.x); i < p.wt_bytes / 16; i += kThreads)
    *reinterpret_cast<u32x4_t*>(lds + 16 * i) = u32x4_t{0u, 0u, 0u, 0u};
  wait_vm_dyn(ndma_a);  // the packed units and epilogue operands (issued before the DMAs)
  if (epi_t) {
    const f32x4_t one = {1.0f, 1.0f, 1.0f, 1.0f};
    *reinterpret_cast<f32x4_t*>(epi + 4 * threadIdx.x) = p.scale ? __builtin_bit_cast(f32x4_t, sc_raw) : one;
    *reinterpret_cast<f32x4_t*>(epi + 64 + 4 * threadIdx.x) = __builtin_bit_cast(f32x4_t, bi_raw);
  }
  lds_barrier();  // zero fill done everywhere
  // Element e of a unit goes to tile row o = G g + idx (an index >= G, which
  // the format rules out, is clamped into the group), column c0 + e.  A
  // write's LDS bank is set by o % 16 and e; the lanes of a wave hold
  // neighbouring column blocks of one packed row, whose kept rows repeat, so
  // at step e lane l writes element e ^ (l % 8) of its block instead of e:
  // one instruction's two-byte stores then spread over four times as many
  // banks.  (The lane's values and indices are permuted once per unit.)
  const uint32_t m = static_cast<uint32_t>(lane & 7);
  const uint32_t bsel = 0x03020100u ^ ((m & 3u) * 0x01010101u);  // byte j <- byte j ^ (m % 4)
#pragma unroll
  for (int u = 0; u < kUnitsMax; ++u) {
    if (wave_has(u)) {
      const int unit = static_cast<int>(threadIdx.x) + u * kThreads;
      if (unit < p.nunits) {
        const int prow = unit / C8;
        const int c0 = (unit - prow * C8) * 8;
        const int gG = (prow / p.K) * p.G;  // the group's first row
        const uint32_t ubase = static_cast<uint32_t>((c0 >> 5) * 1024 + ((c0 & 31) >> 3) * 256);
        // element e of (d, ix) below is element e ^ m of the unit
        uint32_t d[4] = {pv[u][0], pv[u][1], pv[u][2], pv[u][3]};
        uint32_t iw[2] = {pi[u][0], pi[u][1]};
        if (m & 4u) {
          const uint32_t t0 = d[0], t1 = d[1];
          d[0] = d[2]; d[1] = d[3]; d[2] = t0; d[3] = t1;
          const uint32_t ti = iw[0];
          iw[0] = iw[1]; iw[1] = ti;
        }
        if (m & 2u) {
          const uint32_t t0 = d[0], t2 = d[2];
          d[0] = d[1]; d[1] = t0; d[2] = d[3]; d[3] = t2;
        }
        if (m & 1u) {
#pragma unroll
          for (int j = 0; j < 4; ++j) d[j] = __builtin_amdgcn_alignbit(d[j], d[j], 16);
        }
        iw[0] = __builtin_amdgcn_perm(iw[0], iw[0], bsel);
        iw[1] = __builtin_amdgcn_perm(iw[1], iw[1], bsel);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t ix = min((iw[e >> 2] >> (8 * (e & 3))) & 0xffu, static_cast<uint32_t>(p.G - 1));
          const uint32_t o = static_cast<uint32_t>(gG) + ix;
          const uint32_t a = (o >> 4) * (S * 1024) + (o & 15) * 16 + ubase + 2u * (static_cast<uint32_t>(e) ^ m);
          *reinterpret_cast<uint16_t*>(lds + a) = static_cast<uint16_t>(d[e >> 1] >> (16 * (e & 1)));
        }
      }
    }
  }
  lds_barrier();  // tile complete
  bf16x8_t wf[2][S];
  {
    const uint8_t* ws = lds + (2 * slice) * (S * 1024) + lane * 16;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int s = 0; s < S; ++s) wf[b][s] = *reinterpret_cast<const bf16x8_t*>(ws + (b * S + s) * 1024);
  }
  const int obase = 32 * slice + 4 * (lane >> 4);  // this lane's first output of block 0

  // ---- tiles ---------------------------------------------------------------
  const __amdgpu_buffer_rsrc_t yr =
      __builtin_amdgcn_make_buffer_rsrc(p.Y, (short)0, static_cast<int>(p.y_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(p.residual), (short)0, RES ? static_cast<int>(p.y_bytes) : 0, kRsrcWord3);
  const int tiles = (npix + 15) >> 4;
  const uint32_t lq = static_cast<uint32_t>(lane >> 4);
  const uint32_t pix0 = static_cast<uint32_t>((img * p.Ho + oh0) * p.Wo);  // the band's first output pixel
  const int ndma_b = dma_rows(r1, nrows);
  wait_vm_dyn(ndma_b);  // this wave's phase-A rows
  barrier_only();       // everyone's
  const auto tile = [&](int t) __attribute__((always_inline)) {
    const int pl = t * 16 + (lane & 15);
    const bool valid = pl < npix;
    const int plc = valid ? pl : npix - 1;  // past the band: read a staged pixel, store nothing
    const int ohl = static_cast<int>(__umulhi(static_cast<uint32_t>(plc), p.wo_mul) + (static_cast<uint32_t>(plc) & p.wo_one));
    const int ow = plc - ohl * p.Wo;
    // B fragment of k-step s: tap (kh, kw) = (s / CB) / KW, (s / CB) % KW,
    // channels 32 (s % CB) + 8 lq .. +7 of staged pixel (ohl + kh, ow + kw),
    // at z[kw][cb] + kh * RP + kw * CPP * 16 (the last two an instruction
    // offset): z holds the lane's pixel and the chunk swizzle of its column.
    // Reads run D k-steps ahead of the MFMAs (sched_barrier keeps the order:
    // left alone, the compiler waits for each pair of reads right after
    // issuing it).
    uint32_t z[KW][CB];
    {
      const uint32_t a0 = static_cast<uint32_t>(p.wt_bytes) + static_cast<uint32_t>(ohl) * RP +
                          static_cast<uint32_t>(ow) * (CPP * 16);
#pragma unroll
      for (int kw = 0; kw < KW; ++kw) {
        const uint32_t f = ((static_cast<uint32_t>(ow + kw) * CPP) >> 4) & (CPP - 1);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) z[kw][cb] = a0 + (((static_cast<uint32_t>(cb * 4) + lq) ^ f) * 16);
      }
    }
    const auto xread = [&](int s) {
      const int tap = s / CB, cb = s - (s / CB) * CB;
      const int kh = tap / KW, kw = tap - (tap / KW) * KW;
      return *reinterpret_cast<const bf16x8_t*>(lds + z[kw][cb] + (kh * RP + kw * CPP * 16));
    };
    constexpr int D = 8;
    bf16x8_t xb[S];
#pragma unroll
    for (int s = 0; s < D && s < S; ++s) xb[s] = xread(s);
    f32x4_t acc0 = {0.0f, 0.0f, 0.0f, 0.0f}, acc1 = acc0;
#pragma unroll
    for (int s = 0; s < S; ++s) {
      __builtin_amdgcn_sched_barrier(0);
      acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[0][s], xb[s], acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[1][s], xb[s], acc1, 0, 0, 0);
      if (s + D < S) xb[s + D] = xread(s + D);
    }
    __builtin_amdgcn_sched_barrier(0);
    // epilogue: lane holds outputs o .. o + 3 (o = obase + 16 b) of pixel pl
    const uint32_t opix = pix0 + static_cast<uint32_t>(pl);
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int o = obase + 16 * b;
      f32x4_t y = b ? acc1 : acc0;
      const f32x4_t sc = *reinterpret_cast<const f32x4_t*>(epi + o);
      const f32x4_t bi = *reinterpret_cast<const f32x4_t*>(epi + 64 + o);
      y = y * sc + bi;
      const uint32_t off = valid ? (opix * static_cast<uint32_t>(p.O) + static_cast<uint32_t>(o)) * ysz : kOOB;
      if constexpr (RES) {
        if constexpr (ysz == 2) {
          const u32x2_t rv = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(rr, off, 0, 0));
          y[0] += __uint_as_float(rv[0] << 16);
          y[1] += __uint_as_float(rv[0] & 0xffff0000u);
          y[2] += __uint_as_float(rv[1] << 16);
          y[3] += __uint_as_float(rv[1] & 0xffff0000u);
        } else {
          y += __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, 0));
        }
      }
      if (p.relu) {
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = relu_f(y[e]);
      }
      if constexpr (ysz == 2) {
        // v_cvt_pk_bf16_f32: round to nearest even
        const u32x2_t pk = {__builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y[0], y[1]}), bf16x2_t)),
                            __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{y[2], y[3]}), bf16x2_t))};
        __builtin_amdgcn_raw_buffer_store_b64(
            __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b64(yr, 0, 0, 0)), pk), yr, off, 0, 0);
      } else {
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(yr, 0, 0, 0)), y), yr, off, 0, 0);
      }
    }
  };
  // phase A, then (one barrier for every wave) phase B
  int t = stream;
  for (; t < tiles_a; t += streams) tile(t);
  wait_vm<0>();  // this wave's DMAs (and its phase-A stores)
  barrier_only();
  for (; t < tiles; t += streams) tile(t);
}

template <typename YT, int KH, int KW, int CPP, int RP, bool RES>
__global__ __launch_bounds__(kThreads) void resident_kernel(RParams p) {
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];
  resident_body<YT, KH, KW, CPP, RP, RES>(p, lds);
}

// Shapes this family takes: bf16 X and vals, a KH x KW convolution with unit
// stride whose (KH, KW, Cin) has an instantiation, 32 or 64 outputs.
bool shape_ok(const ProductArgs& a) {
  if (!a.conv || a.x_t != DType::BF16 || a.val_t != DType::BF16) return false;
  const ConvGeom& g = a.geom;
  if (g.sh != 1 || g.sw != 1 || g.KH != 3 || g.KW != 3) return false;
  if (g.Cin != 32 && g.Cin != 64) return false;
  if (a.O != 32 && a.O != 64) return false;
  if (a.G < 1 || a.O % a.G != 0 || a.K < 1 || a.K > a.G) return false;
  if (g.pw < 0 || g.ph < 0 || g.pw >= g.KW || g.ph >= g.KH || g.Ho < 1 || g.Wo < 1) return false;
  return true;
}

// Bytes of a staged input row: 8 or 16 KiB (a compile-time pitch, so that
// the kernel's tap offsets are instruction offsets); 0 if a row needs more.
int rows_bytes(const ProductArgs& a) {
  const int cpp = a.geom.Cin / 8;
  const int pcols = a.geom.Wo + a.geom.KW - 1;
  const int need = pcols * cpp * 16;
  return need <= 8192 ? 8192 : (need <= 16384 ? 16384 : 0);
}

// Band height: the number of output rows per workgroup that minimises
// (waves of workgroups) x (prologue + rounds), the prologue counted as three
// rounds; LDS must hold the expanded tile and the band's input rows.
int plan_rows(const ProductArgs& a, int cus) {
  const ConvGeom& g = a.geom;
  const int64_t wt = a.O * a.C * 2;
  const int rb = rows_bytes(a);
  if (rb == 0) return 0;
  const int streams = 8 / static_cast<int>(a.O / 32);
  int best = 0;
  int64_t best_cost = 0;
  for (int R = 1; R <= g.Ho; ++R) {
    if (wt + static_cast<int64_t>(R + g.KH - 1) * rb + kEpiBytes > kLdsMax) break;
    const int64_t bands = a.B * ((g.Ho + R - 1) / R);
    const int64_t waves = (bands + cus - 1) / cus;
    const int64_t rounds = (static_cast<int64_t>(R) * g.Wo + 16 * streams - 1) / (16 * streams);
    const int64_t cost = waves * (3 + rounds);
    if (best == 0 || cost < best_cost) {
      best = R;
      best_cost = cost;
    }
  }
  return best;
}

template <typename YT, int KH, int KW, int CPP, int RP, bool RES>
hipError_t launch_k(const RParams& p, uint32_t grid, int lds, hipStream_t s) {
  static std::atomic<int8_t> lds_set[kMaxDevices];
  const hipError_t attr = set_lds_limit_once(
      lds_set, reinterpret_cast<const void*>(&resident_kernel<YT, KH, KW, CPP, RP, RES>), kLdsMax);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((resident_kernel<YT, KH, KW, CPP, RP, RES>), dim3(grid), dim3(kThreads), lds, s, p);
  return hipGetLastError();
}

template <typename YT, int CPP, int RP>
hipError_t launch_r(const RParams& p, bool res, uint32_t grid, int lds, hipStream_t s) {
  return res ? launch_k<YT, 3, 3, CPP, RP, true>(p, grid, lds, s) : launch_k<YT, 3, 3, CPP, RP, false>(p, grid, lds, s);
}

template <typename YT, int CPP>
hipError_t launch_y(const RParams& p, bool res, uint32_t grid, int lds, hipStream_t s) {
  return p.row_bytes == 8192 ? launch_r<YT, CPP, 8192>(p, res, grid, lds, s)
                             : launch_r<YT, CPP, 16384>(p, res, grid, lds, s);
}

constexpr int kCus = 256;  // MI355X compute units (the plan's target; any device count is correct)

}  // namespace

bool resident_supports(const ProductArgs& a) {
  if (!shape_ok(a)) return false;
  const auto al = [](const void* q, uintptr_t m) { return (reinterpret_cast<uintptr_t>(q) & (m - 1)) == 0; };
  if (!al(a.X, 16) || !al(a.vals, 16) || !al(a.idx, 8) || !al(a.Y, 16)) return false;
  if ((a.scale && !al(a.scale, 16)) || (a.bias && !al(a.bias, 16)) || (a.residual && !al(a.residual, 16)))
    return false;
  const int64_t units = (a.O / a.G) * a.K * a.C / 8;
  if (units > static_cast<int64_t>(kUnitsMax) * kThreads) return false;
  // every buffer offset is 32-bit and stays below the out-of-range marker
  const int64_t lim = static_cast<int64_t>(kOOB);
  const ConvGeom& g = a.geom;
  const int64_t x_bytes = a.B * static_cast<int64_t>(g.H) * g.W * g.Cin * 2;
  const int64_t y_bytes = a.N * a.O * (a.y_t == DType::F32 ? 4 : 2);
  if (x_bytes >= lim || y_bytes >= lim || (a.O / a.G) * a.K * a.C * 2 >= lim) return false;
  if (a.B * static_cast<int64_t>(g.Ho) >= (int64_t(1) << 30)) return false;
  return plan_rows(a, kCus) > 0;
}

hipError_t launch_resident(const ProductArgs& a, hipStream_t s) {
  if (!resident_supports(a)) return hipErrorInvalidConfiguration;
  const ConvGeom& g = a.geom;
  RParams p{};
  p.X = static_cast<const uint16_t*>(a.X);
  p.vals = static_cast<const uint16_t*>(a.vals);
  p.idx = a.idx;
  p.scale = a.scale;
  p.bias = a.bias;
  p.residual = a.residual;
  p.Y = a.Y;
  p.x_bytes = static_cast<uint32_t>(a.B * static_cast<int64_t>(g.H) * g.W * g.Cin * 2);
  p.y_bytes = static_cast<uint32_t>(a.N * a.O * (a.y_t == DType::F32 ? 4 : 2));
  p.p_elems = static_cast<uint32_t>((a.O / a.G) * a.K * a.C);
  p.O = static_cast<int32_t>(a.O);
  p.G = a.G;
  p.K = a.K;
  p.relu = a.relu;
  p.H = g.H;
  p.W = g.W;
  p.Ho = g.Ho;
  p.Wo = g.Wo;
  p.ph = g.ph;
  p.pw = g.pw;
  p.R = plan_rows(a, kCus);
  p.bpi = (g.Ho + p.R - 1) / p.R;
  const int64_t bands = a.B * p.bpi;
  if (bands > 0x7fffffff) return hipErrorInvalidConfiguration;
  p.grid8 = bands % kXcds == 0 ? static_cast<int32_t>(bands / kXcds) : 0;
  p.streams = 8 / static_cast<int32_t>(a.O / 32);
  p.pcols = g.Wo + g.KW - 1;
  p.row_bytes = rows_bytes(a);
  p.dpr = ((g.Wo + g.KW - 1) * (g.Cin / 8) * 16 + 1023) / 1024;  // only the used part of a row
  p.wo_mul = g.Wo > 1 ? static_cast<uint32_t>((uint64_t(1) << 32) / static_cast<uint64_t>(g.Wo) + 1) : 0u;
  p.wo_one = g.Wo > 1 ? 0u : ~0u;
  p.wt_bytes = static_cast<int32_t>(a.O * a.C * 2);
  p.ring_bytes = (p.R + g.KH - 1) * p.row_bytes;
  p.nunits = static_cast<int32_t>((a.O / a.G) * a.K * a.C / 8);
  p.rows_a = (p.R + 1) / 2;
  const int lds = p.wt_bytes + p.ring_bytes + kEpiBytes;
  const uint32_t grid = static_cast<uint32_t>(bands);
  const bool res = a.residual != nullptr;
  if (a.y_t == DType::BF16)
    return g.Cin == 64 ? launch_y<bf16_t, 8>(p, res, grid, lds, s) : launch_y<bf16_t, 4>(p, res, grid, lds, s);
  return g.Cin == 64 ? launch_y<float, 8>(p, res, grid, lds, s) : launch_y<float, 4>(p, res, grid, lds, s);
}

}  // namespace cci
