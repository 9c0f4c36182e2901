// CCI-sparse product with the dataflow of the paper's Alg. 1 (Sec. 3.2),
// on the vector ALUs: only the K kept weights of each group are multiplied,
// and the G outputs of a group stay in registers ("output stationary",
// Sec. 3.3) until the whole reduction is done.
//
// Mapping (wave64):
//   - lanes run over rows n of X (samples, or output pixels of a conv); each
//     lane owns R rows (lane + 64 i), so one packed weight feeds R FMAs;
//   - each wave owns GPW consecutive groups (GPW*G = 16 outputs for G <= 16),
//     so the packed stream (value, index) it reads is the same for every lane:
//     it is fetched once per wave and made wave-uniform with readfirstlane,
//     and the index selects an accumulator through a uniform branch tree --
//     no per-lane dynamic register indexing;
//   - the 4 waves of a workgroup share one X tile staged in LDS as fp32
//     (each activation read from HBM once per workgroup, converted once);
//   - each wave stages its groups' packed stream for the same columns in LDS
//     (coalesced loads), so the per-slot reads in the inner loop are LDS
//     broadcasts instead of dependent global loads.
//
// General path: any dtype combination, any C, conv through implicit im2col.
#include "cci_device.hpp"
#include "cci_launch.hpp"

namespace cci {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kCB = 32;  // reduction columns per LDS chunk
constexpr int kSlotRows = 32;  // packed rows (group x slot) per wave: GPW*K <= 32

// acc[r][i] += v * x[i] for the uniform row r, via a binary tree of uniform
// branches over [LO, HI).
template <int LO, int HI, int G, int R>
struct RowDispatch {
  __device__ static __forceinline__ void run(float (&acc)[G][R], int r, float v,
                                             const float (&x)[R]) {
    constexpr int MID = (LO + HI) / 2;
    if (r < MID)
      RowDispatch<LO, MID, G, R>::run(acc, r, v, x);
    else
      RowDispatch<MID, HI, G, R>::run(acc, r, v, x);
  }
};
template <int LO, int G, int R>
struct RowDispatch<LO, LO + 1, G, R> {
  __device__ static __forceinline__ void run(float (&acc)[G][R], int, float v,
                                             const float (&x)[R]) {
#pragma unroll
    for (int i = 0; i < R; ++i) acc[LO][i] = __builtin_fmaf(v, x[i], acc[LO][i]);
    // A leaf-specific marker keeps the compiler from merging the G leaves
    // into one dynamically indexed update (which would demote acc to scratch).
    asm volatile("; cci row %0" ::"n"(LO));
  }
};

__device__ __forceinline__ int uniform_i(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ float uniform_f(float v) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}

template <int G, int R, typename XT, typename VT, typename YT, bool CONV>
__global__ __launch_bounds__(kThreads) void sparse_mac_kernel(
    const XT* __restrict__ X, int64_t N, int64_t C, ConvGeom geom,
    const VT* __restrict__ vals, const uint8_t* __restrict__ idx, int64_t O, int32_t K,
    Epilogue<YT> ep, YT* __restrict__ Y, int64_t row_blocks) {
  constexpr int GPW = G >= 16 ? 1 : 16 / G;
  constexpr int ROWS = 64 * R;
  constexpr int PITCH = kCB + 1;  // odd pitch: lanes hit distinct banks
  __shared__ float xs[ROWS * PITCH];
  __shared__ int32_t pix_b[CONV ? ROWS : 1], pix_h[CONV ? ROWS : 1], pix_w[CONV ? ROWS : 1];
  __shared__ float pv[kWaves][kSlotRows][kCB];    // packed values of this chunk (fp32)
  __shared__ uint8_t pi[kWaves][kSlotRows][kCB];  // their intra-group row indices

  const int lane = threadIdx.x & 63;
  const int wave = uniform_i(threadIdx.x >> 6);
  const int64_t rb = blockIdx.x % row_blocks;
  const int64_t gb = blockIdx.x / row_blocks;
  const int64_t row0 = rb * ROWS;
  const int64_t ngroups = O / G;
  const int64_t g0 = (gb * kWaves + wave) * GPW;  // wave-uniform

  if constexpr (CONV) {
    for (int r = threadIdx.x; r < ROWS; r += kThreads) {
      const int64_t n = row0 + r;
      if (n < N) {
        const int64_t hw = static_cast<int64_t>(geom.Ho) * geom.Wo;
        const int64_t b = n / hw;
        const int64_t rem = n - b * hw;
        const int64_t oh = rem / geom.Wo;
        const int64_t ow = rem - oh * geom.Wo;
        pix_b[r] = static_cast<int32_t>(b);
        pix_h[r] = static_cast<int32_t>(oh * geom.sh - geom.ph);
        pix_w[r] = static_cast<int32_t>(ow * geom.sw - geom.pw);
      } else {
        pix_b[r] = -1;
        pix_h[r] = 0;
        pix_w[r] = 0;
      }
    }
  }

  float acc[GPW][G][R];
#pragma unroll
  for (int gi = 0; gi < GPW; ++gi)
#pragma unroll
    for (int r = 0; r < G; ++r)
#pragma unroll
      for (int i = 0; i < R; ++i) acc[gi][r][i] = 0.0f;

  for (int64_t c0 = 0; c0 < C; c0 += kCB) {
    __syncthreads();  // previous tile consumed; pixel decode visible
    {
      const int col = threadIdx.x % kCB;
      const int64_t c = c0 + col;
      int kh = 0, kw = 0;
      int64_t cin = 0;
      if constexpr (CONV) {
        if (c < C) {
          const int64_t tap = c / geom.Cin;
          cin = c - tap * geom.Cin;
          kh = static_cast<int>(tap / geom.KW);
          kw = static_cast<int>(tap - static_cast<int64_t>(kh) * geom.KW);
        }
      }
      for (int r = threadIdx.x / kCB; r < ROWS; r += kThreads / kCB) {
        const int64_t n = row0 + r;
        float v = 0.0f;
        if (c < C && n < N) {
          if constexpr (CONV) {
            const int b = pix_b[r];
            const int ih = pix_h[r] + kh;
            const int iw = pix_w[r] + kw;
            if (ih >= 0 && ih < geom.H && iw >= 0 && iw < geom.W)
              v = io<XT>::load(X, ((static_cast<int64_t>(b) * geom.H + ih) * geom.W + iw) * geom.Cin + cin);
          } else {
            v = io<XT>::load(X, n * C + c);
          }
        }
        xs[r * PITCH + col] = v;
      }
    }
    {  // this wave's packed rows (gi, k) for columns c0 .. c0+31
      const int col = lane & (kCB - 1);
      const int64_t c = c0 + col;
      const int nrow = GPW * K;
      for (int rr = lane >> 5; rr < nrow; rr += 2) {
        const int gi = rr / K;
        const int k = rr - gi * K;
        const int64_t g = g0 + gi;
        float v = 0.0f;
        uint8_t ix = 0xff;  // no row: never matches
        if (g < ngroups && c < C) {
          const int64_t off = (g * K + k) * C + c;
          v = io<VT>::load(vals, off);
          ix = idx[off];
        }
        pv[wave][rr][col] = v;
        pi[wave][rr][col] = ix;
      }
    }
    __syncthreads();

    const int cmax = static_cast<int>(C - c0 < kCB ? C - c0 : kCB);
    if (K == G) {
      // every row of a group is kept and the kept rows are stored in
      // ascending order, so slot k targets row k: no dispatch needed
      for (int cc = 0; cc < cmax; ++cc) {
        float x[R];
#pragma unroll
        for (int i = 0; i < R; ++i) x[i] = xs[(lane + 64 * i) * PITCH + cc];
#pragma unroll
        for (int gi = 0; gi < GPW; ++gi) {
#pragma unroll
          for (int k = 0; k < G; ++k) {
            const float v = uniform_f(pv[wave][gi * G + k][cc]);
#pragma unroll
            for (int i = 0; i < R; ++i) acc[gi][k][i] = __builtin_fmaf(v, x[i], acc[gi][k][i]);
          }
        }
      }
    } else {
#pragma unroll 2
      for (int cc = 0; cc < cmax; ++cc) {
        float x[R];
#pragma unroll
        for (int i = 0; i < R; ++i) x[i] = xs[(lane + 64 * i) * PITCH + cc];
#pragma unroll
        for (int gi = 0; gi < GPW; ++gi) {
          // slots in batches of 4: the LDS reads of a batch are issued
          // together, then dispatched (absent slots carry row 0xff)
          for (int k0 = 0; k0 < K; k0 += 4) {
            int r[4];
            float v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int k = k0 + j < K ? k0 + j : K - 1;
              r[j] = k0 + j < K ? uniform_i(pi[wave][gi * K + k][cc]) : 0xff;
              v[j] = uniform_f(pv[wave][gi * K + k][cc]);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j)
              if (r[j] < G) RowDispatch<0, G, G, R>::run(acc[gi], r[j], v[j], x);
          }
        }
      }
    }
  }

#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int64_t n = row0 + lane + 64 * i;
    if (n >= N) continue;
#pragma unroll
    for (int gi = 0; gi < GPW; ++gi) {
      const int64_t g = g0 + gi;
      if (g >= ngroups) break;
#pragma unroll
      for (int r = 0; r < G; ++r) {
        const int64_t o = g * G + r;
        const int64_t yo = n * O + o;
        io<YT>::store(Y, yo, apply_epilogue<YT>(acc[gi][r][i], o, yo, ep));
      }
    }
  }
}

template <int G, int R, typename XT, typename VT, typename YT>
hipError_t launch_g(const ProductArgs& a, hipStream_t s) {
  constexpr int GPW = G >= 16 ? 1 : 16 / G;
  const int64_t rows_per_block = 64 * R;
  const int64_t row_blocks = (a.N + rows_per_block - 1) / rows_per_block;
  const int64_t ngroups = a.O / G;
  const int64_t group_blocks = (ngroups + GPW * kWaves - 1) / (GPW * kWaves);
  const dim3 grid(static_cast<uint32_t>(row_blocks * group_blocks));
  Epilogue<YT> ep{a.scale, a.bias, static_cast<const YT*>(a.residual), a.relu};
  const XT* X = static_cast<const XT*>(a.X);
  const VT* vals = static_cast<const VT*>(a.vals);
  YT* Y = static_cast<YT*>(a.Y);
  if (a.conv)
    hipLaunchKernelGGL((sparse_mac_kernel<G, R, XT, VT, YT, true>), grid, dim3(kThreads), 0, s, X,
                       a.N, a.C, a.geom, vals, a.idx, a.O, a.K, ep, Y, row_blocks);
  else
    hipLaunchKernelGGL((sparse_mac_kernel<G, R, XT, VT, YT, false>), grid, dim3(kThreads), 0, s,
                       X, a.N, a.C, a.geom, vals, a.idx, a.O, a.K, ep, Y, row_blocks);
  return hipGetLastError();
}

template <int R, typename XT, typename VT, typename YT>
hipError_t launch_r(const ProductArgs& a, hipStream_t s) {
  switch (a.G) {
    case 2: return launch_g<2, R, XT, VT, YT>(a, s);
    case 4: return launch_g<4, R, XT, VT, YT>(a, s);
    case 8: return launch_g<8, R, XT, VT, YT>(a, s);
    case 16: return launch_g<16, R, XT, VT, YT>(a, s);
    case 32: return launch_g<32, (R > 2 ? 2 : R), XT, VT, YT>(a, s);
    default: return hipErrorInvalidValue;
  }
}

// Few rows (N <= kSmallRows, FC / plain rows): the row-tiled kernel would
// launch a handful of workgroups.  Instead one wave computes the G outputs
// of one group for one row n (Alg. 1's output-stationary registers): its
// lanes run over the columns c (coalesced reads of X[n][.] and of the packed
// stream), each adds vals * x of every kept slot to the accumulator of the
// slot's row, and a wave reduction sums the lanes' partial sums.
constexpr int64_t kSmallRows = 256;

template <int G, typename XT, typename VT, typename YT>
__global__ __launch_bounds__(kThreads) void sparse_mac_rows_kernel(const XT* __restrict__ X, int64_t N, int64_t C,
                                                                   const VT* __restrict__ vals,
                                                                   const uint8_t* __restrict__ idx, int64_t O,
                                                                   int32_t K, Epilogue<YT> ep, YT* __restrict__ Y) {
  const int lane = threadIdx.x & 63;
  const int64_t ngroups = O / G;
  const int64_t wv = static_cast<int64_t>(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6);
  if (wv >= N * ngroups) return;  // whole wave
  const int64_t n = wv / ngroups, g = wv - n * ngroups;
  float acc[G];
#pragma unroll
  for (int r = 0; r < G; ++r) acc[r] = 0.0f;
  for (int64_t c = lane; c < C; c += 64) {
    const float x = io<XT>::load(X, n * C + c);
#pragma unroll 4
    for (int32_t k = 0; k < K; ++k) {
      const int64_t q = (g * K + k) * C + c;
      const uint32_t i = idx[q];
      const float v = io<VT>::load(vals, q) * x;
#pragma unroll
      for (int r = 0; r < G; ++r) acc[r] += i == static_cast<uint32_t>(r) ? v : 0.0f;
    }
  }
#pragma unroll
  for (int r = 0; r < G; ++r)
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc[r] += __shfl_xor(acc[r], off, 64);
  if (lane < G) {
    float y = acc[0];
#pragma unroll
    for (int r = 1; r < G; ++r) y = lane == r ? acc[r] : y;
    const int64_t o = g * G + lane;
    io<YT>::store(Y, n * O + o, apply_epilogue<YT>(y, o, n * O + o, ep));
  }
}

template <typename XT, typename VT, typename YT>
hipError_t launch_rows(const ProductArgs& a, hipStream_t s) {
  const int64_t waves = a.N * (a.O / a.G);
  const dim3 grid(static_cast<uint32_t>((waves + kThreads / 64 - 1) / (kThreads / 64)));
  Epilogue<YT> ep{a.scale, a.bias, static_cast<const YT*>(a.residual), a.relu};
  const auto X = static_cast<const XT*>(a.X);
  const auto V = static_cast<const VT*>(a.vals);
  const auto Y = static_cast<YT*>(a.Y);
  switch (a.G) {
    case 2: hipLaunchKernelGGL((sparse_mac_rows_kernel<2, XT, VT, YT>), grid, dim3(kThreads), 0, s, X, a.N, a.C, V, a.idx, a.O, a.K, ep, Y); break;
    case 4: hipLaunchKernelGGL((sparse_mac_rows_kernel<4, XT, VT, YT>), grid, dim3(kThreads), 0, s, X, a.N, a.C, V, a.idx, a.O, a.K, ep, Y); break;
    case 8: hipLaunchKernelGGL((sparse_mac_rows_kernel<8, XT, VT, YT>), grid, dim3(kThreads), 0, s, X, a.N, a.C, V, a.idx, a.O, a.K, ep, Y); break;
    case 16: hipLaunchKernelGGL((sparse_mac_rows_kernel<16, XT, VT, YT>), grid, dim3(kThreads), 0, s, X, a.N, a.C, V, a.idx, a.O, a.K, ep, Y); break;
    case 32: hipLaunchKernelGGL((sparse_mac_rows_kernel<32, XT, VT, YT>), grid, dim3(kThreads), 0, s, X, a.N, a.C, V, a.idx, a.O, a.K, ep, Y); break;
    default: return hipErrorInvalidConfiguration;
  }
  return hipGetLastError();
}

template <typename XT, typename VT, typename YT>
hipError_t launch_t(const ProductArgs& a, hipStream_t s) {
  if (!a.conv && a.N <= kSmallRows) return launch_rows<XT, VT, YT>(a, s);
  // Small row counts: one row per lane keeps more workgroups in flight.
  if (a.N <= 4096) return launch_r<1, XT, VT, YT>(a, s);
  return launch_r<4, XT, VT, YT>(a, s);
}

}  // namespace

bool sparse_mac_supports(const ProductArgs& a) {
  const bool g_ok = a.G == 2 || a.G == 4 || a.G == 8 || a.G == 16 || a.G == 32;
  const bool t_ok = (a.x_t == DType::F32 && a.val_t == DType::F32 && a.y_t == DType::F32) ||
                    (a.x_t == DType::BF16 && a.val_t == DType::BF16);
  return g_ok && t_ok;
}

hipError_t launch_sparse_mac(const ProductArgs& a, hipStream_t s) {
  if (a.x_t == DType::F32) return launch_t<float, float, float>(a, s);
  if (a.y_t == DType::BF16) return launch_t<bf16_t, bf16_t, bf16_t>(a, s);
  return launch_t<bf16_t, bf16_t, float>(a, s);
}

}  // namespace cci
