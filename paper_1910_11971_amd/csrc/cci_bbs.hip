// Balanced sparsity -- the paper's comparison structure (Sec. 2.4, Sec. 3.3,
// Fig. 2b) -- and the 2:4 sparse matrix-core product it maps onto.
//
// Balanced groups are G contiguous weights of one output row (weights of
// different inputs); each keeps its K largest |w| and the index of a kept
// weight names the input it multiplies.  Along the reduction that is exactly
// the sparsity gfx950's sparse MFMA skips: v_smfmac_f32_16x16x64_bf16 takes
// an A operand in which every aligned run of 4 reduction positions holds at
// most 2 nonzeros, stored as 2 values plus 2-bit positions.  A balanced
// packing with K <= 2 and G % 4 == 0 (so no run of 4 inputs holds more than
// 2 kept weights) is re-expressed in that form, and so is the transpose of a
// CCI packing (its groups run along the output channels, the reduction of
// the backward product dX = dY . W_hat).
//
// Lane layout of v_smfmac_f32_16x16x64_bf16 (measured on gfx950 with an
// in-bounds probe of the builtin): lane l = i + 16 b holds
//   A: row i, dense reduction columns 16 b .. 16 b + 15 as 4 runs of 4; its
//      element e (0..7) is at column 16 b + 4 (e / 2) + z_e, z_e = bits
//      2e .. 2e+1 of the index operand (abid 0);
//   B: column i, reduction rows 8 b .. 8 b + 7 in elements 0..7 and
//      32 + 8 b .. 32 + 8 b + 7 in elements 8..15;
//   D: rows 4 b .. 4 b + 3 of column i.
//
// Prepared 2:4 operand of an M x C matrix A (M % 16 == 0, C % 64 == 0):
//   vals bf16 [C/64][M/16][64 lanes][8], idx uint16 [C/64][M/16][64 lanes]:
// fragment (k-step s, row block mb) is 1 KiB of values and 128 B of indices,
// and the fragments of one k-step are contiguous, so a product kernel stages
// a k-step of 256 rows with 16 + 2 contiguous 1 KiB copies.
#include <type_traits>

#include "cci_device.hpp"
#include "cci_launch.hpp"

namespace cci {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint16_t u16x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr uint32_t kOOB = 0x80000000u;   // buffer offset that reads as zero
constexpr int kRsrcWord3 = 0x00020000;   // raw buffer descriptor word 3 (gfx9 family)

// ---------------------------------------------------------------------------
// Balanced-sparsity projection: one lane per (row o, group j).  The lanes of
// a wave take consecutive groups of one row, so the row is read contiguously.

constexpr int kPackThreads = 256;

__device__ __forceinline__ uint32_t abs_bits(float w) { return __float_as_uint(w) & 0x7fffffffu; }

template <typename VT> __device__ __forceinline__ void put(VT* p, int64_t i, float w);
template <> __device__ __forceinline__ void put<float>(float* p, int64_t i, float w) { p[i] = w; }
template <> __device__ __forceinline__ void put<bf16_t>(bf16_t* p, int64_t i, float w) {
  p[i].bits = f32_to_bf16_rne(w);
}

template <int G, typename VT>
__global__ __launch_bounds__(kPackThreads) void bbs_pack_fixed(const float* __restrict__ W, int64_t C,
                                                               int64_t total, int32_t K,
                                                               VT* __restrict__ vals,
                                                               uint8_t* __restrict__ idx) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * kPackThreads + threadIdx.x;  // o * (C / G) + j
  if (t >= total) return;
  const float* w = W + t * G;  // group j of row o starts at o * C + j * G = t * G
  float v[G];
  uint32_t key[G];
#pragma unroll
  for (int r = 0; r < G; ++r) {
    v[r] = w[r];
    key[r] = abs_bits(v[r]);
  }
  int slot = 0;
#pragma unroll
  for (int r = 0; r < G; ++r) {
    int rank = 0;
#pragma unroll
    for (int q = 0; q < G; ++q) rank += (key[q] > key[r]) || (key[q] == key[r] && q < r);
    if (rank < K) {
      put<VT>(vals, t * K + slot, v[r]);
      idx[t * K + slot] = static_cast<uint8_t>(r);
      ++slot;
    }
  }
}

template <typename VT>
__global__ __launch_bounds__(kPackThreads) void bbs_pack_generic(const float* __restrict__ W, int64_t total,
                                                                 int32_t G, int32_t K, VT* __restrict__ vals,
                                                                 uint8_t* __restrict__ idx) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * kPackThreads + threadIdx.x;
  if (t >= total) return;
  const float* w = W + t * G;
  int slot = 0;
  for (int r = 0; r < G && slot < K; ++r) {
    const uint32_t kr = abs_bits(w[r]);
    int rank = 0;
    for (int q = 0; q < G; ++q) {
      const uint32_t kq = abs_bits(w[q]);
      rank += (kq > kr) || (kq == kr && q < r);
    }
    if (rank < K) {
      put<VT>(vals, t * K + slot, w[r]);
      idx[t * K + slot] = static_cast<uint8_t>(r);
      ++slot;
    }
  }
}

template <typename VT>
hipError_t bbs_pack_typed(const float* W, int64_t O, int64_t C, int32_t G, int32_t K, VT* vals,
                          uint8_t* idx, hipStream_t s) {
  const int64_t total = O * (C / G);
  const dim3 grid(static_cast<uint32_t>((total + kPackThreads - 1) / kPackThreads));
  const dim3 block(kPackThreads);
  switch (G) {
    case 2: hipLaunchKernelGGL((bbs_pack_fixed<2, VT>), grid, block, 0, s, W, C, total, K, vals, idx); break;
    case 4: hipLaunchKernelGGL((bbs_pack_fixed<4, VT>), grid, block, 0, s, W, C, total, K, vals, idx); break;
    case 8: hipLaunchKernelGGL((bbs_pack_fixed<8, VT>), grid, block, 0, s, W, C, total, K, vals, idx); break;
    case 16: hipLaunchKernelGGL((bbs_pack_fixed<16, VT>), grid, block, 0, s, W, C, total, K, vals, idx); break;
    default: hipLaunchKernelGGL((bbs_pack_generic<VT>), grid, block, 0, s, W, total, G, K, vals, idx);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Preparing the 2:4 operand.  One lane per (k-step s, row block mb, fragment
// lane l): it collects the kept entries of row 16 mb + l % 16 that fall in
// the 16 reduction columns c0 = 64 s + 16 (l / 16) .. c0 + 15, in ascending
// column order, and places each in slot 2 q + (1 if an earlier entry of the
// same run q = (column - c0) / 4 took slot 2 q).  Unused slots hold 0 at a
// position different from the run's other slot.  The caller guarantees at
// most 2 kept entries per run (K <= 2, G % 4 == 0).

struct Slots24 {
  uint16_t v[8];
  uint32_t z[8];
  uint32_t used;  // bit 2q + r: slot r of run q taken
};

__device__ __forceinline__ void slots_init(Slots24& S) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    S.v[e] = 0;
    S.z[e] = 0;
  }
  S.used = 0;
}

// Entry at column offset p (0..15) with value bits vb.
__device__ __forceinline__ void slots_add(Slots24& S, uint32_t p, uint16_t vb) {
  const uint32_t q = p >> 2;
  const uint32_t r = (S.used >> (2 * q)) & 1u;  // slot 0 taken -> slot 1
  const uint32_t e = 2 * q + r;
  S.used |= 1u << e;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    S.v[k] = (static_cast<uint32_t>(k) == e) ? vb : S.v[k];
    S.z[k] = (static_cast<uint32_t>(k) == e) ? (p & 3u) : S.z[k];
  }
}

// Index word and value vector of the lane; an empty slot gets a position
// distinct from its partner's.
__device__ __forceinline__ void slots_emit(const Slots24& S, uint16_t* vout, uint16_t* iout) {
  uint32_t word = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const bool u0 = (S.used >> (2 * q)) & 1u, u1 = (S.used >> (2 * q + 1)) & 1u;
    const uint32_t z0 = u0 ? S.z[2 * q] : (u1 ? (S.z[2 * q + 1] + 1u) & 3u : 0u);
    const uint32_t z1 = u1 ? S.z[2 * q + 1] : (z0 + 1u) & 3u;
    word |= (z0 << (4 * q)) | (z1 << (4 * q + 2));
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) vout[e] = S.v[e];
  *iout = static_cast<uint16_t>(word);
}

// From a balanced packing vals/idx [M][C/G][K] (rows M = O).
__global__ __launch_bounds__(256) void bbs_to_24_kernel(const uint16_t* __restrict__ vals,
                                                        const uint8_t* __restrict__ idx, int64_t M,
                                                        int64_t C, int32_t G, int32_t K,
                                                        uint16_t* __restrict__ av, uint16_t* __restrict__ ai) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;  // ((s * M/16) + mb) * 64 + l
  const int64_t total = (C / 64) * (M / 16) * 64;
  if (t >= total) return;
  const int l = static_cast<int>(t & 63);
  const int64_t frag = t >> 6;
  const int64_t mb = frag % (M / 16), s = frag / (M / 16);
  const int64_t m = mb * 16 + (l & 15);
  const int64_t c0 = s * 64 + 16 * (l >> 4);
  const int64_t ng = C / G;
  Slots24 S;
  slots_init(S);
  for (int64_t j = c0 / G; j <= (c0 + 15) / G; ++j)
    for (int k = 0; k < K; ++k) {
      const int64_t e = (m * ng + j) * K + k;
      const int64_t p = j * G + idx[e] - c0;
      if (p >= 0 && p < 16) slots_add(S, static_cast<uint32_t>(p), vals[e]);
    }
  slots_emit(S, av + t * 8, ai + t);
}

// From a CCI packing vals/idx [O/G][K][C] of W_hat [O][C]: the operand of
// W_hat^T (rows M = C, reduction O), whose runs of G reduction positions are
// the CCI groups.
__global__ __launch_bounds__(256) void cci_t_to_24_kernel(const uint16_t* __restrict__ vals,
                                                          const uint8_t* __restrict__ idx, int64_t O,
                                                          int64_t C, int32_t G, int32_t K,
                                                          uint16_t* __restrict__ av, uint16_t* __restrict__ ai) {
  const int64_t M = C, R = O;  // rows and reduction length of the operand
  const int64_t t = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t total = (R / 64) * (M / 16) * 64;
  if (t >= total) return;
  const int l = static_cast<int>(t & 63);
  const int64_t frag = t >> 6;
  const int64_t mb = frag % (M / 16), s = frag / (M / 16);
  const int64_t c = mb * 16 + (l & 15);        // row of the operand = input column of W_hat
  const int64_t o0 = s * 64 + 16 * (l >> 4);  // its reduction columns = output channels
  Slots24 S;
  slots_init(S);
  for (int64_t g = o0 / G; g <= (o0 + 15) / G; ++g)
    for (int k = 0; k < K; ++k) {
      const int64_t e = (g * K + k) * C + c;
      const int64_t p = g * G + idx[e] - o0;
      if (p >= 0 && p < 16) slots_add(S, static_cast<uint32_t>(p), vals[e]);
    }
  slots_emit(S, av + t * 8, ai + t);
}

// ---------------------------------------------------------------------------
// 2:4 product Y[n][m] = epilogue(sum_c A[m][c] X[n][c]) on the sparse matrix
// cores.  A workgroup of eight waves (two per SIMD) owns 256 rows of A x 256
// rows of X; wave w accumulates A rows 128 (w % 2) .. +128 (8 fragments) x
// X rows 64 (w / 2) .. +64 (4 fragments): 32 sparse MFMAs per 64-column
// k-step, 128 fp32 accumulators per lane.  Each k-step's operands (A: 16 KiB
// of values, 2 KiB of indices; X: 256 rows x 128 B) are DMA'd into one of
// three LDS stages two k-steps ahead (buffer_load ... lds, 16 B per lane);
// one barrier per k-step.  A bf16 output tile leaves through LDS as whole
// row segments.
//
// X stage layout: row r at r * 128, its 16-byte unit u (channels 8u .. 8u+7
// of the k-step) at (u ^ ((r >> 1) & 7)) * 16: a DMA instruction reads 8
// rows x 128 contiguous bytes, and the B-fragment reads (16 rows, units q
// and 4 + q) hit distinct 16-byte bank slots within each quarter- and
// half-wave.

constexpr int kS4Threads = 512;
constexpr int kS4Tile = 256;                           // A rows and X rows of a workgroup
constexpr int kS4AV = 16384;                           // A values of a stage
constexpr int kS4AI = 2048;                            // A indices of a stage
constexpr int kS4X = kS4Tile * 128;                    // X rows of a stage
constexpr int kS4Stage = kS4AV + kS4AI + kS4X;         // 51200
constexpr int kS4Lds = 3 * kS4Stage;                   // 153600
static_assert(kS4Lds <= 160 * 1024, "LDS budget");
static_assert(8 * 64 * 272 <= kS4Lds, "the output staging reuses the operand stages");

struct S4Params {
  const uint16_t* X;
  const uint16_t* av;
  const uint16_t* ai;
  const float* scale;
  const float* bias;
  const void* residual;
  void* Y;
  uint32_t x_bytes, av_bytes, ai_bytes;
  int32_t N, C, M, relu;
  int32_t nmt, nnt;  // tiles of 256 A rows, of 256 X rows
  int32_t grid8;     // grid / 8 when the grid is a multiple of 8, else 0
};

__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

template <typename YT>
__global__ __launch_bounds__(kS4Threads) void spmm24_kernel(S4Params p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w & 1, wn = w >> 1;

  // ---- tile: the workgroups of one XCD (dispatch puts workgroup b on XCD
  // b % 8) cover groups of 4 A-row tiles x consecutive X-row tiles.
  const uint32_t bid = blockIdx.x;
  const uint32_t L = p.grid8 ? (bid & 7u) * static_cast<uint32_t>(p.grid8) + (bid >> 3) : bid;
  const uint32_t per = 4u * static_cast<uint32_t>(p.nnt);
  const uint32_t grp = L / per;
  const uint32_t gm = min(4u, static_cast<uint32_t>(p.nmt) - 4u * grp);
  const uint32_t within = L - grp * per;
  const uint32_t nt = within / gm;
  const uint32_t mt = 4u * grp + (within - nt * gm);
  const int32_t m0 = static_cast<int32_t>(mt) * kS4Tile, n0 = static_cast<int32_t>(nt) * kS4Tile;
  const int32_t mblocks = p.M / 16;

  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.X), (short)0, static_cast<int>(p.x_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t vr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.av), (short)0, static_cast<int>(p.av_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t ir =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.ai), (short)0, static_cast<int>(p.ai_bytes), kRsrcWord3);

  // ---- DMA offsets (k-step 0; a k-step adds a constant) ---------------------
  // X: instruction i of wave w fills rows 32 w + 8 i .. +8: lane l writes
  // row r = 32 w + 8 i + l / 8, slot l % 8, which holds unit (l % 8) ^ sw(r).
  uint32_t xoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t r = static_cast<uint32_t>(32 * w + 8 * i + (lane >> 3));
    const uint32_t u = static_cast<uint32_t>(lane & 7) ^ ((r >> 1) & 7u);
    const uint32_t n = static_cast<uint32_t>(n0) + r;
    xoff[i] = n < static_cast<uint32_t>(p.N) ? n * static_cast<uint32_t>(p.C) * 2u + u * 16u : kOOB;
  }
  // A values: instruction i of wave w fills fragment 2 w + i (1 KiB contiguous).
  uint32_t voff[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int32_t mb = m0 / 16 + 2 * w + i;
    voff[i] = mb < mblocks ? static_cast<uint32_t>(mb) * 1024u + static_cast<uint32_t>(lane) * 16u : kOOB;
  }
  // A indices: waves 0 and 1 fill fragments 8 w .. 8 w + 7 (128 B each).
  uint32_t ioff = kOOB;
  if (w < 2) {
    const int32_t mb = m0 / 16 + 8 * w + (lane >> 3);
    ioff = mb < mblocks ? static_cast<uint32_t>(mb) * 128u + static_cast<uint32_t>(lane & 7) * 16u : kOOB;
  }
  const uint32_t vstep = static_cast<uint32_t>(mblocks) * 1024u, istep = static_cast<uint32_t>(mblocks) * 128u;

  auto issue = [&](int ks, int buf) {
    uint8_t* st = lds + buf * kS4Stage;
    const uint32_t xo = static_cast<uint32_t>(ks) * 128u;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t o = xoff[i] == kOOB ? kOOB : xoff[i] + xo;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t*)(st + kS4AV + kS4AI + (32 * w + 8 * i) * 128), 16, o,
                                               0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint32_t o = voff[i] == kOOB ? kOOB : voff[i] + static_cast<uint32_t>(ks) * vstep;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_void_t*)(st + (2 * w + i) * 1024), 16, o, 0, 0, 0);
    }
    if (w < 2) {
      const uint32_t o = ioff == kOOB ? kOOB : ioff + static_cast<uint32_t>(ks) * istep;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ir, (lds_void_t*)(st + kS4AV + 8 * w * 128), 16, o, 0, 0, 0);
    }
  };

  f32x4_t acc[8][4];
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[a][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nk = p.C / 64;
  issue(0, 0);
  if (nk > 1) issue(1, 1);
  // B-fragment addresses inside a stage's X rows: lane (i, q) reads row
  // 64 wn + 16 t + i, units q and 4 + q.
  const int bi = lane & 15, bq = lane >> 4;
  uint32_t boff[4][2];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const uint32_t r = static_cast<uint32_t>(64 * wn + 16 * t + bi);
    const uint32_t sw = (r >> 1) & 7u;
    boff[t][0] = r * 128u + ((static_cast<uint32_t>(bq) ^ sw) * 16u);
    boff[t][1] = r * 128u + (((4u + static_cast<uint32_t>(bq)) ^ sw) * 16u);
  }

  for (int j = 0; j < nk; ++j) {
    // this wave's DMAs of k-step j are done when at most those of k-step j+1 remain
    if (j + 1 < nk) {
      if (w < 2) wait_vm<7>(); else wait_vm<6>();
    } else {
      wait_vm<0>();
    }
    lds_barrier();
    if (j + 2 < nk) issue(j + 2, (j + 2) % 3);
    const uint8_t* st = lds + (j % 3) * kS4Stage;
    bf16x8_t av[8];
    int ai[8];
#pragma unroll
    for (int a = 0; a < 8; ++a) {
      av[a] = *reinterpret_cast<const bf16x8_t*>(st + (8 * wm + a) * 1024 + lane * 16);
      ai[a] = *reinterpret_cast<const uint16_t*>(st + kS4AV + (8 * wm + a) * 128 + lane * 2);
    }
    const uint8_t* xs = st + kS4AV + kS4AI;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const bf16x8_t lo = *reinterpret_cast<const bf16x8_t*>(xs + boff[t][0]);
      const bf16x8_t hi = *reinterpret_cast<const bf16x8_t*>(xs + boff[t][1]);
      const bf16x16_t b = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
#pragma unroll
      for (int a = 0; a < 8; ++a)
        acc[a][t] = __builtin_amdgcn_smfmac_f32_16x16x64_bf16(av[a], b, acc[a][t], ai[a], 0, 0);
    }
  }

  // ---- epilogue: lane holds rows 4 (lane / 16) .. +3 of A (outputs) for X
  // row lane % 16 of each 16 x 16 block.  Scale, bias, residual and ReLU in
  // fp32, one rounding.  A bf16 result is staged per wave in LDS (64 X rows x
  // 128 outputs, rows padded to 272 B) and written back as whole 256-byte row
  // segments; fp32 results are stored from the registers.
  const bool yf32 = std::is_same<YT, float>::value;
  constexpr int kStPitch = 272;
  uint8_t* stg = lds + w * (64 * kStPitch);
  if (!yf32) lds_barrier();  // every wave is done with the operand stages
#pragma unroll
  for (int a = 0; a < 8; ++a) {
    const int32_t mbase = m0 + 16 * (8 * wm + a);
    if (mbase >= p.M) continue;
    const int32_t m = mbase + 4 * (lane >> 4);
    f32x4_t sc = {1.f, 1.f, 1.f, 1.f}, bs = {0.f, 0.f, 0.f, 0.f};
    if (p.scale) sc = *reinterpret_cast<const f32x4_t*>(p.scale + m);
    if (p.bias) bs = *reinterpret_cast<const f32x4_t*>(p.bias + m);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int32_t nl = 16 * t + (lane & 15);
      const int32_t n = n0 + 64 * wn + nl;
      const int64_t yo = static_cast<int64_t>(n) * p.M + m;
      float y[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) y[r] = acc[a][t][r] * sc[r] + bs[r];
      if (p.residual && n < p.N) {
        if (yf32) {
          const f32x4_t rv = *reinterpret_cast<const f32x4_t*>(static_cast<const float*>(p.residual) + yo);
#pragma unroll
          for (int r = 0; r < 4; ++r) y[r] += rv[r];
        } else {
          const u16x4_t rv = *reinterpret_cast<const u16x4_t*>(static_cast<const uint16_t*>(p.residual) + yo);
#pragma unroll
          for (int r = 0; r < 4; ++r) y[r] += bf16_to_f32(rv[r]);
        }
      }
      if (p.relu) {
#pragma unroll
        for (int r = 0; r < 4; ++r) y[r] = y[r] > 0.0f ? y[r] : (y[r] != y[r] ? y[r] : 0.0f);
      }
      if (yf32) {
        if (n < p.N) *reinterpret_cast<f32x4_t*>(static_cast<float*>(p.Y) + yo) = f32x4_t{y[0], y[1], y[2], y[3]};
      } else {
        *reinterpret_cast<u16x4_t*>(stg + nl * kStPitch + (16 * a + 4 * (lane >> 4)) * 2) =
            u16x4_t{f32_to_bf16_rne(y[0]), f32_to_bf16_rne(y[1]), f32_to_bf16_rne(y[2]), f32_to_bf16_rne(y[3])};
      }
    }
  }
  if (!yf32) {
    // (each wave reads back only what it wrote: program order suffices)
    const int32_t mw = m0 + 128 * wm + 8 * (lane & 15);  // this lane's 8 outputs
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      const int32_t nl = 4 * rr + (lane >> 4);
      const int32_t n = n0 + 64 * wn + nl;
      const u32x4_t v = *reinterpret_cast<const u32x4_t*>(stg + nl * kStPitch + (lane & 15) * 16);
      if (n < p.N && mw < p.M)
        *reinterpret_cast<u32x4_t*>(static_cast<uint16_t*>(p.Y) + static_cast<int64_t>(n) * p.M + mw) = v;
    }
  }
}

template <typename YT>
hipError_t launch_s4(const S4Params& p, uint32_t grid, hipStream_t s) {
  static std::atomic<int8_t> lds_set[kMaxDevices];
  const hipError_t attr = set_lds_limit_once(lds_set, reinterpret_cast<const void*>(&spmm24_kernel<YT>), kS4Lds);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((spmm24_kernel<YT>), dim3(grid), dim3(kS4Threads), kS4Lds, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bbs_pack(const float* W, int64_t O, int64_t C, int32_t G, int32_t K, void* vals, DType val_t,
                           uint8_t* idx, hipStream_t s) {
  if (val_t == DType::F32) return bbs_pack_typed<float>(W, O, C, G, K, static_cast<float*>(vals), idx, s);
  return bbs_pack_typed<bf16_t>(W, O, C, G, K, static_cast<bf16_t*>(vals), idx, s);
}

hipError_t launch_to_2of4(bool from_cci, const void* vals, const uint8_t* idx, int64_t O, int64_t C, int32_t G,
                          int32_t K, void* av, uint16_t* ai, hipStream_t s) {
  const int64_t M = from_cci ? C : O, R = from_cci ? O : C;
  const int64_t total = (R / 64) * (M / 16) * 64;
  if (total == 0) return hipSuccess;
  const dim3 grid(static_cast<uint32_t>((total + 255) / 256));
  if (from_cci)
    hipLaunchKernelGGL(cci_t_to_24_kernel, grid, dim3(256), 0, s, static_cast<const uint16_t*>(vals), idx, O, C, G,
                       K, static_cast<uint16_t*>(av), ai);
  else
    hipLaunchKernelGGL(bbs_to_24_kernel, grid, dim3(256), 0, s, static_cast<const uint16_t*>(vals), idx, O, C, G, K,
                       static_cast<uint16_t*>(av), ai);
  return hipGetLastError();
}

bool spmm_2of4_fits(int64_t N, int64_t C, int64_t M, DType y_t) {
  const int64_t lim = static_cast<int64_t>(kOOB);
  return N * C * 2 < lim && M * C < lim && N * M * (y_t == DType::F32 ? 4 : 2) < (int64_t(1) << 40);
}

hipError_t launch_spmm_2of4(const void* X, int64_t N, int64_t C, const void* av, const uint16_t* ai, int64_t M,
                            const float* scale, const float* bias, const void* residual, int32_t relu, void* Y,
                            DType y_t, hipStream_t s) {
  S4Params p{};
  p.X = static_cast<const uint16_t*>(X);
  p.av = static_cast<const uint16_t*>(av);
  p.ai = ai;
  p.scale = scale;
  p.bias = bias;
  p.residual = residual;
  p.Y = Y;
  p.x_bytes = static_cast<uint32_t>(N * C * 2);
  p.av_bytes = static_cast<uint32_t>(M * C);        // M x C/2 bf16 values
  p.ai_bytes = static_cast<uint32_t>(M * C / 8);    // (C/64) x (M/16) fragments x 64 lanes x 2 B
  p.N = static_cast<int32_t>(N);
  p.C = static_cast<int32_t>(C);
  p.M = static_cast<int32_t>(M);
  p.relu = relu;
  p.nmt = static_cast<int32_t>((M + kS4Tile - 1) / kS4Tile);
  p.nnt = static_cast<int32_t>((N + kS4Tile - 1) / kS4Tile);
  const uint32_t grid = static_cast<uint32_t>(p.nmt) * static_cast<uint32_t>(p.nnt);
  p.grid8 = grid % 8 == 0 ? static_cast<int32_t>(grid / 8) : 0;
  return y_t == DType::F32 ? launch_s4<float>(p, grid, s) : launch_s4<bf16_t>(p, grid, s);
}

}  // namespace cci
