// Split-reduction MFMA kernel for products with few row tiles and a long
// reduction (Sec. 3.2's Y = X . W_hat^T with W_hat kept as CCI groups,
// Sec. 3.1): e.g. 3 136 x 960 -> 160, where a tile kernel that walks the
// reduction serially spends one memory round trip per chunk and leaves most
// CUs idle.
//
// A workgroup of eight waves owns a tile of 16 RF rows x 16 OF outputs and
// splits the reduction between its waves: wave w takes the 32-column k-steps
// w, w + 8, w + 16, ...  A wave issues the loads of up to U of its k-steps at
// once, so one memory latency covers its share of the reduction, then
// multiplies them on v_mfma_f32_16x16x32_bf16.  When the packed rows of the
// tile's groups fit in LDS beside the partial tiles (WL), the workgroup
// copies them there once, while its first X loads are in flight, and the
// waves load only X per k-step; otherwise each lane also loads its own
// group's packed entries.  The eight partial tiles are added through LDS in
// two rounds, and the fused epilogue (scale, bias, residual, ReLU; one
// rounding) writes 8 outputs per thread.
//
// Weight fragments are built in registers, never in memory.  The A operand
// of the MFMA gives lane l output row r = l % 16 and columns c0 .. c0 + 7
// (c0 = 32 s + 8 (l / 16)).  Output o = gG + rr lies in group g at slot rr;
// each of the group's K kept entries of column c holds a value and a slot
// index (Alg. 1), so entry k of column c lands in row r exactly when its
// index equals rr.  A lane reads its group's K value rows (16 bytes) and
// index rows (8 bytes) for its 8 columns, compares each index byte with rr
// (a bytewise zero test of idx ^ rr, widened to a 16-bit mask per column)
// and keeps the matching values.  Distinct kept entries of one column have
// distinct slots, so at most one value survives per element.
#include <type_traits>

#include "cci_device.hpp"
#include "cci_launch.hpp"

namespace cci {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kThreads = 512;  // eight waves
constexpr int kWaves = 8;
constexpr int kXcds = 8;

struct KParams {
  const uint16_t* X;
  const uint16_t* vals;
  const uint8_t* idx;
  const float* scale;
  const float* bias;
  const void* residual;
  void* Y;
  int32_t N, C, O, G, relu;
  int32_t nob;    // output blocks (O / (16 OF))
  int32_t tiles;  // row blocks x output blocks
  int32_t tpx;    // tiles per XCD (ceil(tiles / 8))
};

// k-steps whose loads a wave keeps in flight together: as many as fit about
// 128 registers of operands.
// (With the packed rows staged in LDS only X is loaded per k-step; 128-row
// tiles then keep 96 registers of it beside their 64 accumulators.)
constexpr int batch_budget(int rf, bool wl) { return wl && rf == 8 ? 96 : 128; }
constexpr int batch_steps(int rf, int of, int k, bool wl) {
  return batch_budget(rf, wl) / (4 * rf + (wl ? 0 : 6 * of * k)) < 1
             ? 1
             : (batch_budget(rf, wl) / (4 * rf + (wl ? 0 : 6 * of * k)) > 4
                    ? 4
                    : batch_budget(rf, wl) / (4 * rf + (wl ? 0 : 6 * of * k)));
}

// 64 x 64 tiles hold 64 accumulator registers: only K = 1 leaves room for
// its operands without spilling.
constexpr bool tile_fits(int rf, int of, int k) { return !(rf == 4 && of == 4) || k == 1; }

// Bytes of idx that equal the lane's slot become 0xffff masks over the
// matching bf16 values: m[d] covers columns 2d, 2d + 1.
__device__ __forceinline__ void slot_masks(uint32_t i0, uint32_t i1, uint32_t rrx, uint32_t m[4]) {
  uint32_t b[2] = {i0 ^ rrx, i1 ^ rrx};
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t x = b[h];
    // bit 7 of every byte: set where the byte is nonzero (no carries cross bytes)
    const uint32_t t = ((x & 0x7f7f7f7fu) + 0x7f7f7f7fu) | x;
    const uint32_t zb = ~t & 0x80808080u;
    b[h] = zb | (zb - (zb >> 7));  // 0xff in every zero byte
  }
  m[0] = __builtin_amdgcn_perm(b[0], b[0], 0x01010000u);
  m[1] = __builtin_amdgcn_perm(b[0], b[0], 0x03030202u);
  m[2] = __builtin_amdgcn_perm(b[1], b[1], 0x01010000u);
  m[3] = __builtin_amdgcn_perm(b[1], b[1], 0x03030202u);
}

template <int RF, int OF, int K>
struct Step {
  u32x4_t x[RF];
  u32x4_t v[OF][K];
  u32x2_t i[OF][K];
};

template <int RF, int OF, int K, bool WL, typename YT>
__global__ __launch_bounds__(kThreads) void split_k_kernel(KParams p) {
  constexpr int TR = 16 * RF, TO = 16 * OF, PITCH = TO + 4;
  constexpr int U = batch_steps(RF, OF, K, WL);
  __shared__ __attribute__((aligned(16))) float red[4][TR][PITCH];
  __shared__ __attribute__((aligned(16))) float sb[2][TO];  // the tile's scale and bias
  // WL: the packed rows of the tile's groups, values then indices
  extern __shared__ __attribute__((aligned(16))) uint8_t wlds[];

  // workgroup b runs on XCD b % 8: each XCD takes a contiguous run of tiles,
  // so the output blocks of one row block share that XCD's L2 copy of X
  const int32_t b = static_cast<int32_t>(blockIdx.x);
  const int32_t t = (b % kXcds) * p.tpx + b / kXcds;
  if (t >= p.tiles) return;  // whole workgroup: before any barrier
  const int32_t rb = t / p.nob, ob = t - rb * p.nob;
  const int32_t w = static_cast<int32_t>(threadIdx.x) / 64, lane = static_cast<int32_t>(threadIdx.x) % 64;
  const int32_t lr = lane % 16, lq = lane / 16;
  const int32_t n0 = rb * TR, o0 = ob * TO;

  // per output fragment: the lane's group row base (in the packed arrays, or
  // in the staged copy of groups g_lo ..) and slot
  const int32_t g_lo = o0 / p.G;
  int64_t gbase[OF];
  uint32_t rrx[OF];
#pragma unroll
  for (int f = 0; f < OF; ++f) {
    const int32_t o = o0 + 16 * f + lr;
    const int32_t g = o / p.G;
    rrx[f] = static_cast<uint32_t>(o - g * p.G) * 0x01010101u;
    gbase[f] = static_cast<int64_t>(WL ? g - g_lo : g) * K * p.C;
  }
  // X rows past N read row N - 1 (their sums are never stored)
  const uint16_t* xrow[RF];
#pragma unroll
  for (int r = 0; r < RF; ++r) {
    const int32_t n = min(n0 + 16 * r + lr, p.N - 1);
    xrow[r] = p.X + static_cast<int64_t>(n) * p.C + 8 * lq;
  }

  f32x4_t acc[RF][OF];
#pragma unroll
  for (int r = 0; r < RF; ++r)
#pragma unroll
    for (int f = 0; f < OF; ++f) acc[r][f] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int32_t nks = p.C / 32;
  Step<RF, OF, K> st[U];
  const auto load_batch = [&](int32_t s0) {
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int32_t s = s0 + kWaves * j;
      if (s < nks) {
#pragma unroll
        for (int r = 0; r < RF; ++r) st[j].x[r] = *reinterpret_cast<const u32x4_t*>(xrow[r] + 32 * s);
        if (!WL) {
          const int32_t c0 = 32 * s + 8 * lq;
#pragma unroll
          for (int f = 0; f < OF; ++f)
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const int64_t e = gbase[f] + static_cast<int64_t>(k) * p.C + c0;
              st[j].v[f][k] = *reinterpret_cast<const u32x4_t*>(p.vals + e);
              st[j].i[f][k] = *reinterpret_cast<const u32x2_t*>(p.idx + e);
            }
        }
      }
    }
  };
  int32_t s0 = w;
  load_batch(s0);
  // scale and bias of the tile's outputs to LDS now, not one round trip after
  // the reduction (the barriers below publish them)
  {
    const int32_t tid = static_cast<int32_t>(threadIdx.x);
    if (p.scale && tid < TO / 4)
      *reinterpret_cast<f32x4_t*>(&sb[0][4 * tid]) = *reinterpret_cast<const f32x4_t*>(p.scale + o0 + 4 * tid);
    if (p.bias && tid >= TO / 4 && tid < TO / 2)
      *reinterpret_cast<f32x4_t*>(&sb[1][4 * tid - TO]) =
          *reinterpret_cast<const f32x4_t*>(p.bias + o0 + 4 * tid - TO);
  }
  // WL: copy the packed rows of groups g_lo .. g_hi (contiguous in both
  // arrays) while the first X batch is in flight
  const int32_t nel = WL ? ((min(o0 + TO, p.O) - 1) / p.G - g_lo + 1) * K * p.C : 0;
  if (WL) {
    const int64_t e0 = static_cast<int64_t>(g_lo) * K * p.C;
    const int32_t tid = static_cast<int32_t>(threadIdx.x);
    for (int32_t q = tid; q < nel / 8; q += kThreads)
      *reinterpret_cast<u32x4_t*>(wlds + 16 * q) = *reinterpret_cast<const u32x4_t*>(p.vals + e0 + 8 * q);
    for (int32_t q = tid; q < nel / 16; q += kThreads)
      *reinterpret_cast<u32x4_t*>(wlds + 2 * nel + 16 * q) = *reinterpret_cast<const u32x4_t*>(p.idx + e0 + 16 * q);
    __syncthreads();
  }
  while (true) {
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int32_t s = s0 + kWaves * j;
      if (s < nks) {
        const int32_t c0 = 32 * s + 8 * lq;
#pragma unroll
        for (int f = 0; f < OF; ++f) {
          u32x4_t a = u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
          for (int k = 0; k < K; ++k) {
            u32x4_t v;
            u32x2_t ix;
            if (WL) {
              const int32_t le = static_cast<int32_t>(gbase[f]) + k * p.C + c0;
              v = *reinterpret_cast<const u32x4_t*>(wlds + 2 * le);
              ix = *reinterpret_cast<const u32x2_t*>(wlds + 2 * nel + le);
            } else {
              v = st[j].v[f][k];
              ix = st[j].i[f][k];
            }
            uint32_t m[4];
            slot_masks(ix[0], ix[1], rrx[f], m);
#pragma unroll
            for (int d = 0; d < 4; ++d) a[d] |= v[d] & m[d];
          }
          const bf16x8_t av = __builtin_bit_cast(bf16x8_t, a);
#pragma unroll
          for (int r = 0; r < RF; ++r)
            acc[r][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8_t, st[j].x[r]),
                                                                acc[r][f], 0, 0, 0);
        }
      }
    }
    s0 += kWaves * U;
    if (s0 >= nks) break;
    load_batch(s0);
  }

  // ---- add the eight partial tiles: waves 4..7 into 0..3, then 0..3 in LDS.
  // Lane l holds outputs 4 (l / 16) .. +3 of tile row l % 16.
  const auto put = [&](int slot) {
#pragma unroll
    for (int r = 0; r < RF; ++r)
#pragma unroll
      for (int f = 0; f < OF; ++f)
        *reinterpret_cast<f32x4_t*>(&red[slot][16 * r + lr][16 * f + 4 * lq]) = acc[r][f];
  };
  if (w >= 4) put(w - 4);
  __syncthreads();
  if (w < 4) {
#pragma unroll
    for (int r = 0; r < RF; ++r)
#pragma unroll
      for (int f = 0; f < OF; ++f) acc[r][f] += *reinterpret_cast<const f32x4_t*>(&red[w][16 * r + lr][16 * f + 4 * lq]);
  }
  __syncthreads();
  if (w < 4) put(w);
  __syncthreads();

  // ---- epilogue: thread -> (row, 8 consecutive outputs)
  constexpr int kPerRow = TO / 8;
  const int32_t tid = static_cast<int32_t>(threadIdx.x);
  if (tid >= TR * kPerRow) return;
  const int32_t nl = tid / kPerRow, ol = (tid % kPerRow) * 8;
  const int32_t n = n0 + nl, o = o0 + ol;
  if (n >= p.N) return;
  float y[8];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    f32x4_t sum = *reinterpret_cast<const f32x4_t*>(&red[0][nl][ol + 4 * h]);
#pragma unroll
    for (int v = 1; v < 4; ++v) sum += *reinterpret_cast<const f32x4_t*>(&red[v][nl][ol + 4 * h]);
#pragma unroll
    for (int e = 0; e < 4; ++e) y[4 * h + e] = sum[e];
  }
  if (p.scale) {
    const f32x4_t sc0 = *reinterpret_cast<const f32x4_t*>(&sb[0][ol]);
    const f32x4_t sc1 = *reinterpret_cast<const f32x4_t*>(&sb[0][ol + 4]);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      y[e] *= sc0[e];
      y[4 + e] *= sc1[e];
    }
  }
  if (p.bias) {
    const f32x4_t b0 = *reinterpret_cast<const f32x4_t*>(&sb[1][ol]);
    const f32x4_t b1 = *reinterpret_cast<const f32x4_t*>(&sb[1][ol + 4]);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      y[e] += b0[e];
      y[4 + e] += b1[e];
    }
  }
  const bool yf32 = std::is_same<YT, float>::value;
  const int64_t yo = static_cast<int64_t>(n) * p.O + o;
  if (p.residual) {
    if (yf32) {
      const float* rp = static_cast<const float*>(p.residual) + yo;
      const f32x4_t r0 = *reinterpret_cast<const f32x4_t*>(rp);
      const f32x4_t r1 = *reinterpret_cast<const f32x4_t*>(rp + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        y[e] += r0[e];
        y[4 + e] += r1[e];
      }
    } else {
      const u32x4_t rv = *reinterpret_cast<const u32x4_t*>(static_cast<const uint16_t*>(p.residual) + yo);
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        y[2 * d] += __uint_as_float(rv[d] << 16);
        y[2 * d + 1] += __uint_as_float(rv[d] & 0xffff0000u);
      }
    }
  }
  if (p.relu) {
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = y[e] > 0.0f ? y[e] : (y[e] != y[e] ? y[e] : 0.0f);
  }
  if (yf32) {
    float* yp = static_cast<float*>(p.Y) + yo;
    *reinterpret_cast<f32x4_t*>(yp) = f32x4_t{y[0], y[1], y[2], y[3]};
    *reinterpret_cast<f32x4_t*>(yp + 4) = f32x4_t{y[4], y[5], y[6], y[7]};
  } else {
    u32x4_t out;
#pragma unroll
    for (int d = 0; d < 4; ++d)
      out[d] = static_cast<uint32_t>(f32_to_bf16_rne(y[2 * d])) |
               (static_cast<uint32_t>(f32_to_bf16_rne(y[2 * d + 1])) << 16);
    *reinterpret_cast<u32x4_t*>(static_cast<uint16_t*>(p.Y) + yo) = out;
  }
}

constexpr int64_t kLdsMax = 160 * 1024;

// Static LDS of a tile shape: the partial tiles and the scale / bias rows.
constexpr int64_t red_bytes(int rf, int of) { return 4 * (16 * rf) * (16 * of + 4) * 4 + 2 * (16 * of) * 4; }

// Groups one output block of TO outputs touches, at most: TO / G when G
// divides TO, one when TO divides G, else every alignment's worst case.
int64_t block_groups(int64_t TO, int64_t G) {
  if (TO % G == 0) return TO / G;
  if (G % TO == 0) return 1;
  return (TO + G - 2) / G + 1;
}

// Bytes of the staged packed rows (values and indices) of one output block.
int64_t staged_bytes(int of, int64_t C, int32_t G, int32_t K) { return 3 * block_groups(16 * of, G) * K * C; }

template <int RF, int OF, int K, bool WL>
hipError_t launch_rokw(const KParams& p, int64_t dyn, DType y_t, hipStream_t s) {
  const uint32_t grid = static_cast<uint32_t>(p.tpx) * kXcds;
  static std::atomic<int8_t> lds_set[2][kMaxDevices];
  const auto kf = &split_k_kernel<RF, OF, K, WL, float>;
  const auto kb = &split_k_kernel<RF, OF, K, WL, bf16_t>;
  if (WL) {
    const int limit = static_cast<int>(kLdsMax - red_bytes(RF, OF));
    const hipError_t e = y_t == DType::F32 ? set_lds_limit_once(lds_set[0], reinterpret_cast<const void*>(kf), limit)
                                           : set_lds_limit_once(lds_set[1], reinterpret_cast<const void*>(kb), limit);
    if (e != hipSuccess) return e;
  }
  if (y_t == DType::F32)
    hipLaunchKernelGGL(kf, dim3(grid), dim3(kThreads), static_cast<uint32_t>(dyn), s, p);
  else
    hipLaunchKernelGGL(kb, dim3(grid), dim3(kThreads), static_cast<uint32_t>(dyn), s, p);
  return hipGetLastError();
}

template <int RF, int OF, int K>
hipError_t launch_rok(const KParams& p, bool wl, int64_t dyn, DType y_t, hipStream_t s) {
  if constexpr (!tile_fits(RF, OF, K)) {
    return hipErrorInvalidConfiguration;
  } else {
    return wl ? launch_rokw<RF, OF, K, true>(p, dyn, y_t, s) : launch_rokw<RF, OF, K, false>(p, 0, y_t, s);
  }
}

template <int RF, int OF>
hipError_t launch_ro(const KParams& p, int32_t K, bool wl, int64_t dyn, DType y_t, hipStream_t s) {
  switch (K) {
    case 1: return launch_rok<RF, OF, 1>(p, wl, dyn, y_t, s);
    case 2: return launch_rok<RF, OF, 2>(p, wl, dyn, y_t, s);
    case 3: return launch_rok<RF, OF, 3>(p, wl, dyn, y_t, s);
    case 4: return launch_rok<RF, OF, 4>(p, wl, dyn, y_t, s);
    default: return hipErrorInvalidConfiguration;
  }
}

}  // namespace

// Tile shape: the candidate with the least modelled time.  Each workgroup
// pays one memory round trip (~1.5 us) per batch of its waves' loads and one
// for its epilogue, and streams its operands at ~150 GB/s per CU; at one
// workgroup per CU (two waves per SIMD) the grid runs in ceil(tiles / 256)
// rounds; X is re-read once per output block from L2 (~20 TB/s over the
// chip).
static void split_k_tile(int64_t N, int64_t C, int64_t O, int32_t G, int32_t K, int32_t& rf, int32_t& of) {
  static const int32_t cand[6][2] = {{8, 2}, {4, 4}, {2, 4}, {4, 2}, {2, 2}, {2, 1}};
  double best = 1e300;
  rf = 2;
  of = 1;
  const int64_t per_wave = (C / 32 + kWaves - 1) / kWaves;
  for (const auto& c : cand) {
    if (O % (16 * c[1]) != 0 || !tile_fits(c[0], c[1], K)) continue;
    const int64_t nob = O / (16 * c[1]);
    const int64_t tiles = (N + 16 * c[0] - 1) / (16 * c[0]) * nob;
    const bool wl = red_bytes(c[0], c[1]) + staged_bytes(c[1], C, G, K) <= kLdsMax;
    const int64_t u = batch_steps(c[0], c[1], K, wl);
    const int64_t batches = (per_wave + u - 1) / u;
    const double rounds = static_cast<double>((tiles + 255) / 256);
    const double wg_bytes = static_cast<double>(16 * c[0]) * C * 2 + static_cast<double>(16 * c[1]) * C * K * 3 / 2;
    const double t = rounds * (static_cast<double>(batches + 1) * 1.5 + wg_bytes / 150e3) +
                     static_cast<double>(N) * C * 2 * nob / 20e6;
    if (t < best) {
      best = t;
      rf = c[0];
      of = c[1];
    }
  }
}

bool split_k_supports(const ProductArgs& a) {
  if (a.x_t != DType::BF16 || a.val_t != DType::BF16) return false;
  if (a.G < 1 || a.G > 256 || a.K < 1 || a.K > 4 || a.K > a.G) return false;
  if (a.conv) {
    const ConvGeom& g = a.geom;
    if (g.KH != 1 || g.KW != 1 || g.sh != 1 || g.sw != 1 || g.ph != 0 || g.pw != 0) return false;
  }
  if (a.N < 1 || a.C < 32 || a.C % 32 != 0 || a.O % 16 != 0) return false;
  const auto al = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
  if (!al(a.X) || !al(a.vals) || !al(a.idx) || !al(a.Y) || (a.residual && !al(a.residual))) return false;
  if ((a.scale && !al(a.scale)) || (a.bias && !al(a.bias))) return false;
  // tile and group indices stay in 32 bits
  if (a.N > (int64_t(1) << 30) || a.O > (int64_t(1) << 24) || a.C > (int64_t(1) << 24)) return false;
  return true;
}

hipError_t launch_split_k(const ProductArgs& a, hipStream_t s) {
  if (!split_k_supports(a)) return hipErrorInvalidConfiguration;
  int32_t rf, of;
  split_k_tile(a.N, a.C, a.O, a.G, a.K, rf, of);
  KParams p{};
  p.X = static_cast<const uint16_t*>(a.X);
  p.vals = static_cast<const uint16_t*>(a.vals);
  p.idx = a.idx;
  p.scale = a.scale;
  p.bias = a.bias;
  p.residual = a.residual;
  p.Y = a.Y;
  p.N = static_cast<int32_t>(a.N);
  p.C = static_cast<int32_t>(a.C);
  p.O = static_cast<int32_t>(a.O);
  p.G = a.G;
  p.relu = a.relu;
  p.nob = static_cast<int32_t>(a.O / (16 * of));
  const int64_t tiles = (a.N + 16 * rf - 1) / (16 * rf) * p.nob;
  if (tiles > (int64_t(1) << 30)) return hipErrorInvalidConfiguration;
  p.tiles = static_cast<int32_t>(tiles);
  p.tpx = static_cast<int32_t>((tiles + kXcds - 1) / kXcds);
  // the packed rows of a block go to LDS when they fit beside the partial tiles
  const int64_t dyn = staged_bytes(of, a.C, a.G, a.K);
  const bool wl = red_bytes(rf, of) + dyn <= kLdsMax;
  if (rf == 8 && of == 2) return launch_ro<8, 2>(p, a.K, wl, dyn, a.y_t, s);
  if (rf == 4 && of == 4) return launch_ro<4, 4>(p, a.K, wl, dyn, a.y_t, s);
  if (rf == 4 && of == 2) return launch_ro<4, 2>(p, a.K, wl, dyn, a.y_t, s);
  if (rf == 2 && of == 4) return launch_ro<2, 4>(p, a.K, wl, dyn, a.y_t, s);
  if (rf == 2 && of == 2) return launch_ro<2, 2>(p, a.K, wl, dyn, a.y_t, s);
  return launch_ro<2, 1>(p, a.K, wl, dyn, a.y_t, s);
}

}  // namespace cci
