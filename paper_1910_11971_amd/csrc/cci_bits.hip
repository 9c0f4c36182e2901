// Plain log2(G)-bit indices (Sec. 3.1) and the product that reads them where
// weight bytes bind: few rows.
//
// Index stream: with b = ceil(log2 G) bits per kept weight, entry e of an
// index array sits at bits e*b .. e*b+b-1 of a little-endian stream of
// 32-bit words (stream bit t = bit t % 32 of word t / 32).  b = 8 is the byte
// array cci_pack writes.
//
// Few-row product (N <= 64).  With few rows every packed weight is used by
// at most N multiply-adds, so the packed bytes (2 per value + b/8 per index)
// set the time.  A workgroup of eight waves owns 16 output channels (the
// last one fewer when O % 16 != 0: its missing rows stay zero and are not
// stored); wave w
// takes the 32-column k-steps w, w+8, ... of the reduction.  Per k-step a wave
//   - clears its 16 x 32 bf16 tile in LDS (one 16-byte store per lane),
//   - reads the kept entries of the groups covering its 16 rows (lanes over
//     the 32 columns, so values and index bits are read contiguously),
//     decodes each index from the stream, and writes every value whose row
//     falls in the tile to (row, column) -- Alg. 1's routing to row gG+idx,
//   - reads the tile back as the A fragment of v_mfma_f32_16x16x32_bf16 and
//     multiplies it with up to four 16-row fragments of X.
// The eight waves' partial sums are added in LDS; the fused epilogue and one
// rounding follow.  The tile stores unit u (8 columns) of row i at
// (u ^ ((i >> 2) & 3)) * 16 + i * 64, so a fragment read touches distinct
// 16-byte bank slots within every quarter-wave.
#include <algorithm>
#include <type_traits>

#include "cci_device.hpp"
#include "cci_launch.hpp"

namespace cci {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint16_t u16x4_t __attribute__((ext_vector_type(4)));

constexpr int kRsrcWord3 = 0x00020000;  // raw buffer descriptor word 3 (gfx9 family)

// ---------------------------------------------------------------------------
// Index stream: one lane per 32-bit output word.

__global__ __launch_bounds__(256) void index_bits_kernel(const uint8_t* __restrict__ idx, int64_t n, int32_t b,
                                                         uint32_t* __restrict__ words, int64_t nw) {
  const int64_t w = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (w >= nw) return;
  const int64_t t0 = w * 32;
  const int64_t e0 = t0 / b, e1 = (t0 + 31) / b;  // entries touching this word
  uint32_t word = 0;
  for (int64_t e = e0; e <= e1 && e < n; ++e) {
    const int64_t sh = e * b - t0;                 // -b < sh < 32
    const uint32_t v = idx[e] & ((1u << b) - 1u);
    word |= sh >= 0 ? (v << sh) : (v >> -sh);
  }
  words[w] = word;
}

// ---------------------------------------------------------------------------

constexpr int kFThreads = 512;  // eight waves
constexpr int kFWaves = 8;

struct FParams {
  const uint16_t* X;
  const uint16_t* vals;
  const void* idx;
  const float* scale;
  const float* bias;
  const void* residual;
  void* Y;
  uint32_t x_bytes, i_bytes, v_bytes;
  int32_t N, C, O, G, K, b, relu;
};

// Loads of one k-step: up to PL kept entries per lane (index word(s) and
// value) and the lane's X fragments.
template <int PL, int NB>
struct Fetch {
  uint32_t lo[PL > 0 ? PL : 1], hi[PL > 0 ? PL : 1];
  uint16_t v[PL > 0 ? PL : 1];
  u32x4_t x[NB];
};

template <int NB, int PL, typename YT>
__global__ __launch_bounds__(kFThreads) void spmm_bits_kernel(FParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t tiles[kFWaves][1024];
  __shared__ __attribute__((aligned(16))) f32x4_t red[kFWaves][NB][64];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int32_t o0 = static_cast<int32_t>(blockIdx.x) * 16;
  const int32_t g_lo = o0 / p.G, g_hi = min((o0 + 15) / p.G, p.O / p.G - 1);
  // (group, slot) pairs cover the k-step's 32 columns: lanes 0..31 take the
  // even pairs, lanes 32..63 the odd ones, lane & 31 the column; entry u of
  // a lane is pair pk + 2u, at packed offset base[u] + 32 s in k-step s
  const int32_t npairs = (g_hi - g_lo + 1) * p.K;
  const int32_t pk = lane >> 5, cj = lane & 31;
  constexpr int PA = PL > 0 ? PL : 1;
  int64_t base[PA];
  int32_t row0[PA];
  bool on[PA];
#pragma unroll
  for (int u = 0; u < PL; ++u) {
    const int32_t q = pk + 2 * u;
    on[u] = q < npairs;
    const int32_t gl = on[u] ? q / p.K : 0, k = on[u] ? q - gl * p.K : 0;
    base[u] = (static_cast<int64_t>(g_lo + gl) * p.K + k) * p.C + cj;
    row0[u] = (g_lo + gl) * p.G - o0;
  }

  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.X), (short)0, static_cast<int>(p.x_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t ir =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p.idx), (short)0, static_cast<int>(p.i_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t vr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.vals), (short)0, static_cast<int>(p.v_bytes), kRsrcWord3);
  const uint32_t mask = (1u << p.b) - 1u;
  uint8_t* tile = tiles[w];
  const int ti = lane & 15, tq = lane >> 4;
  const uint8_t* frag = tile + ti * 64 + ((tq ^ ((ti >> 2) & 3)) * 16);

  auto fetch = [&](int32_t s, Fetch<PL, NB>& f) {
    const int32_t c0 = s * 32;
#pragma unroll
    for (int u = 0; u < PL; ++u) {
      const int64_t e = base[u] + c0;
      const uint32_t voff = on[u] ? static_cast<uint32_t>(e) * 2u : 0x80000000u;
      f.v[u] = __builtin_amdgcn_raw_buffer_load_b16(vr, voff, 0, 0);
      if (p.b == 8) {
        f.lo[u] = __builtin_amdgcn_raw_buffer_load_b8(ir, on[u] ? static_cast<uint32_t>(e) : 0x80000000u, 0, 0);
        f.hi[u] = 0;
      } else {
        const uint32_t off = on[u] ? static_cast<uint32_t>((e * p.b) >> 5) * 4u : 0x80000000u;
        f.lo[u] = __builtin_amdgcn_raw_buffer_load_b32(ir, off, 0, 0);
        f.hi[u] = __builtin_amdgcn_raw_buffer_load_b32(ir, on[u] ? off + 4u : 0x80000000u, 0, 0);
      }
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const uint32_t n = static_cast<uint32_t>(16 * nb + ti);
      const uint32_t off = n < static_cast<uint32_t>(p.N)
                               ? (n * static_cast<uint32_t>(p.C) + static_cast<uint32_t>(c0 + 8 * tq)) * 2u
                               : 0x80000000u;
      f.x[nb] = __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0);
    }
  };

  f32x4_t acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int32_t nks = p.C / 32;
  if constexpr (PL == 0) {
    // many entries per lane (large G x K): walk the pairs with loads inline
    const int32_t gl0 = pk / p.K, k0 = pk - gl0 * p.K;
    for (int32_t s = w; s < nks; s += kFWaves) {
      const int32_t c0 = s * 32;
      *reinterpret_cast<u32x4_t*>(tile + lane * 16) = u32x4_t{0u, 0u, 0u, 0u};
      int32_t gl = gl0, k = k0;
      for (int32_t q = pk; q < npairs; q += 2) {
        const int64_t e = (static_cast<int64_t>(g_lo + gl) * p.K + k) * p.C + c0 + cj;
        uint32_t r;
        if (p.b == 8) {
          r = __builtin_amdgcn_raw_buffer_load_b8(ir, static_cast<uint32_t>(e), 0, 0);
        } else {
          const uint32_t off = static_cast<uint32_t>((e * p.b) >> 5) * 4u;
          const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b32(ir, off, 0, 0);
          const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b32(ir, off + 4u, 0, 0);
          r = __builtin_amdgcn_alignbit(hi, lo, static_cast<uint32_t>((e * p.b) & 31)) & mask;
        }
        const int32_t row = (g_lo + gl) * p.G + static_cast<int32_t>(r) - o0;
        if (row >= 0 && row < 16)
          *reinterpret_cast<uint16_t*>(tile + row * 64 + (((cj >> 3) ^ ((row >> 2) & 3)) * 16) + (cj & 7) * 2) =
              p.vals[e];
        k += 2;
        while (k >= p.K) {
          k -= p.K;
          ++gl;
        }
      }
      const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(frag);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const uint32_t n = static_cast<uint32_t>(16 * nb + ti);
        const uint32_t off = n < static_cast<uint32_t>(p.N)
                                 ? (n * static_cast<uint32_t>(p.C) + static_cast<uint32_t>(c0 + 8 * tq)) * 2u
                                 : 0x80000000u;
        const u32x4_t xv = __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8_t, xv), acc[nb], 0, 0, 0);
      }
    }
  } else {
  Fetch<PL, NB> cur, nxt;
  if (w < nks) fetch(w, cur);
  for (int32_t s = w; s < nks; s += kFWaves) {
    if (s + kFWaves < nks) fetch(s + kFWaves, nxt);
    const int32_t c0 = s * 32;
    *reinterpret_cast<u32x4_t*>(tile + lane * 16) = u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
    for (int u = 0; u < PL; ++u) {
      const int64_t e = base[u] + c0;
      const uint32_t r = p.b == 8 ? cur.lo[u] : __builtin_amdgcn_alignbit(cur.hi[u], cur.lo[u],
                                                                          static_cast<uint32_t>((e * p.b) & 31)) & mask;
      const int32_t row = row0[u] + static_cast<int32_t>(r);
      if (on[u] && row >= 0 && row < 16)
        *reinterpret_cast<uint16_t*>(tile + row * 64 + (((cj >> 3) ^ ((row >> 2) & 3)) * 16) + (cj & 7) * 2) = cur.v[u];
    }
    const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(frag);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8_t, cur.x[nb]), acc[nb], 0, 0, 0);
    cur = nxt;
  }
  }

  // ---- sum the eight waves' partials; wave nb finishes X rows 16 nb .. +16
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) red[w][nb][lane] = acc[nb];
  __syncthreads();
  if (w >= NB) return;
  f32x4_t sum = red[0][w][lane];
#pragma unroll
  for (int v = 1; v < kFWaves; ++v) sum += red[v][w][lane];
  const int32_t n = 16 * w + ti;
  const int32_t o = o0 + 4 * tq;  // lane holds outputs o .. o+3 of row n
  if (n >= p.N || o >= p.O) return;  // (O % 4 == 0: a lane's 4 outputs are all inside or all past O)
  const bool yf32 = std::is_same<YT, float>::value;
  const int64_t yo = static_cast<int64_t>(n) * p.O + o;
  float y[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    y[r] = sum[r];
    if (p.scale) y[r] *= p.scale[o + r];
    if (p.bias) y[r] += p.bias[o + r];
  }
  if (p.residual) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      y[r] += yf32 ? static_cast<const float*>(p.residual)[yo + r]
                   : bf16_to_f32(static_cast<const uint16_t*>(p.residual)[yo + r]);
  }
  if (p.relu) {
#pragma unroll
    for (int r = 0; r < 4; ++r) y[r] = y[r] > 0.0f ? y[r] : (y[r] != y[r] ? y[r] : 0.0f);
  }
  if (yf32) {
    *reinterpret_cast<f32x4_t*>(static_cast<float*>(p.Y) + yo) = f32x4_t{y[0], y[1], y[2], y[3]};
  } else {
    *reinterpret_cast<u16x4_t*>(static_cast<uint16_t*>(p.Y) + yo) =
        u16x4_t{f32_to_bf16_rne(y[0]), f32_to_bf16_rne(y[1]), f32_to_bf16_rne(y[2]), f32_to_bf16_rne(y[3])};
  }
}

template <int NB, int PL>
hipError_t launch_fp(const FParams& p, DType y_t, hipStream_t s) {
  const dim3 grid(static_cast<uint32_t>((p.O + 15) / 16));
  if (y_t == DType::F32)
    hipLaunchKernelGGL((spmm_bits_kernel<NB, PL, float>), grid, dim3(kFThreads), 0, s, p);
  else
    hipLaunchKernelGGL((spmm_bits_kernel<NB, PL, bf16_t>), grid, dim3(kFThreads), 0, s, p);
  return hipGetLastError();
}

// PL: kept entries a lane reads per k-step, ceil(pairs / 2), where pairs =
// (groups that 16 consecutive rows starting at a multiple of 16 can touch) x K.
// Up to 8 they are loaded a k-step ahead; beyond, the generic walk.
template <int NB>
hipError_t launch_f(const FParams& p, DType y_t, hipStream_t s) {
  const int32_t groups = 16 % p.G == 0 ? 16 / p.G : (p.G % 16 == 0 ? 1 : 15 / p.G + 2);
  const int32_t pl = (groups * p.K + 1) / 2;
  if (pl <= 1) return launch_fp<NB, 1>(p, y_t, s);
  if (pl <= 2) return launch_fp<NB, 2>(p, y_t, s);
  if (pl <= 4) return launch_fp<NB, 4>(p, y_t, s);
  if (pl <= 8) return launch_fp<NB, 8>(p, y_t, s);
  return launch_fp<NB, 0>(p, y_t, s);
}

}  // namespace

int64_t index_stream_bytes(int64_t n, int32_t b) { return b == 8 ? n : (n * b + 31) / 32 * 4; }

hipError_t launch_index_bits(const uint8_t* idx, int64_t n, int32_t b, uint32_t* words, hipStream_t s) {
  const int64_t nw = (n * b + 31) / 32;
  if (nw == 0) return hipSuccess;
  hipLaunchKernelGGL(index_bits_kernel, dim3(static_cast<uint32_t>((nw + 255) / 256)), dim3(256), 0, s, idx, n, b,
                     words, nw);
  return hipGetLastError();
}

bool spmm_bits_supports(int64_t N, int64_t C, int64_t O, int32_t G, int32_t K) {
  return N >= 0 && N <= 64 && C % 32 == 0 && O % 4 == 0 && N * C * 2 < (int64_t(1) << 31) &&
         (O / G) * K * C < (int64_t(1) << 30);
}

hipError_t launch_spmm_bits(const void* X, int64_t N, int64_t C, const void* vals, const void* idx, int32_t b,
                            int64_t O, int32_t G, int32_t K, const float* scale, const float* bias,
                            const void* residual, int32_t relu, void* Y, DType y_t, hipStream_t s) {
  FParams p{};
  p.X = static_cast<const uint16_t*>(X);
  p.vals = static_cast<const uint16_t*>(vals);
  p.idx = idx;
  p.scale = scale;
  p.bias = bias;
  p.residual = residual;
  p.Y = Y;
  p.x_bytes = static_cast<uint32_t>(N * C * 2);
  p.i_bytes = static_cast<uint32_t>(index_stream_bytes((O / G) * K * C, b));
  p.v_bytes = static_cast<uint32_t>((O / G) * K * C * 2);
  p.N = static_cast<int32_t>(N);
  p.C = static_cast<int32_t>(C);
  p.O = static_cast<int32_t>(O);
  p.G = G;
  p.K = K;
  p.b = b;
  p.relu = relu;
  if (N <= 16) return launch_f<1>(p, y_t, s);
  if (N <= 32) return launch_f<2>(p, y_t, s);
  return launch_f<4>(p, y_t, s);
}

}  // namespace cci
