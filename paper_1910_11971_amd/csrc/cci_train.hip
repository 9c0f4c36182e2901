// Training-step kernels of improved targeted dropout (Sec. 5.1; schedule of
// Sec. 6) for a CCI layer.
//
// cci_td_mask: candidate dropout of one step.  One lane per (group g,
// column c), as in the projection: the lane ranks the G weights of its group
// by magnitude (larger |w| first, ties to the lower row), marks the n_target
// lowest as candidates, and drops a candidate when the caller's random word
// for it is below floor(drop_rate * 2^32).  HBM-bound: reads W and the random
// words, writes W_eff and the keep mask, all coalesced along c.
//
// cci_grad_packed: gradient of the packed values once the mask is fixed,
//   dvals[g][k][c] = sum_n dY[n][gG + idx[g][k][c]] * X[n][c].
// (bf16 operands in the shapes it takes run on the matrix cores instead:
// cci_grad.hip.  This kernel serves fp32, short reductions and other shapes.)
// A workgroup owns four consecutive groups and 256 columns (a lane per
// column, its indices in registers); per pass of up to 32 rows the rows of dY
// restricted to those groups' outputs and of X restricted to the columns are
// staged in LDS with every load in flight, then each lane gathers the
// entries its indices name (one LDS read and one FMA per kept weight and row).
// Only kept weights are touched: N * nnz multiply-adds on the vector ALUs.
#include <algorithm>
#include <type_traits>

#include "cci_device.hpp"
#include "cci_launch.hpp"

namespace cci {
namespace {

constexpr int kMaskThreads = 256;

__device__ __forceinline__ uint32_t abs_bits(float w) { return __float_as_uint(w) & 0x7fffffffu; }

template <typename WT> __device__ __forceinline__ void put(WT* p, int64_t i, float w);
template <> __device__ __forceinline__ void put<float>(float* p, int64_t i, float w) { p[i] = w; }
template <> __device__ __forceinline__ void put<bf16_t>(bf16_t* p, int64_t i, float w) {
  p[i].bits = f32_to_bf16_rne(w);
}

template <int G, typename WT>
__global__ __launch_bounds__(kMaskThreads) void td_mask_fixed(const float* __restrict__ W, const uint32_t* __restrict__ bits,
                                                              int64_t C, int64_t cblocks, int32_t n_target, uint64_t thr,
                                                              WT* __restrict__ We, uint8_t* __restrict__ keep) {
  const int64_t blk = blockIdx.x;
  const int64_t g = blk / cblocks;
  const int64_t c = (blk % cblocks) * kMaskThreads + threadIdx.x;
  if (c >= C) return;
  float w[G];
  uint32_t key[G];
#pragma unroll
  for (int r = 0; r < G; ++r) {
    w[r] = W[(g * G + r) * C + c];
    key[r] = abs_bits(w[r]);
  }
#pragma unroll
  for (int r = 0; r < G; ++r) {
    int rank = 0;
#pragma unroll
    for (int q = 0; q < G; ++q) rank += (key[q] > key[r]) || (key[q] == key[r] && q < r);
    const int64_t o = (g * G + r) * C + c;
    const bool drop = rank >= G - n_target && static_cast<uint64_t>(bits[o]) < thr;
    put<WT>(We, o, drop ? 0.0f : w[r]);
    keep[o] = drop ? 0 : 1;
  }
}

template <typename WT>
__global__ __launch_bounds__(kMaskThreads) void td_mask_generic(const float* __restrict__ W, const uint32_t* __restrict__ bits,
                                                                int64_t C, int64_t cblocks, int32_t G, int32_t n_target,
                                                                uint64_t thr, WT* __restrict__ We,
                                                                uint8_t* __restrict__ keep) {
  const int64_t blk = blockIdx.x;
  const int64_t g = blk / cblocks;
  const int64_t c = (blk % cblocks) * kMaskThreads + threadIdx.x;
  if (c >= C) return;
  const float* col = W + g * G * C + c;
  for (int r = 0; r < G; ++r) {
    const float wr = col[r * C];
    const uint32_t kr = abs_bits(wr);
    int rank = 0;
    for (int q = 0; q < G; ++q) {
      const uint32_t kq = abs_bits(col[q * C]);
      rank += (kq > kr) || (kq == kr && q < r);
    }
    const int64_t o = (g * G + r) * C + c;
    const bool drop = rank >= G - n_target && static_cast<uint64_t>(bits[o]) < thr;
    put<WT>(We, o, drop ? 0.0f : wr);
    keep[o] = drop ? 0 : 1;
  }
}

template <typename WT>
hipError_t td_mask_typed(const float* W, int64_t O, int64_t C, int32_t G, int32_t n_target, const uint32_t* bits,
                         uint64_t thr, WT* We, uint8_t* keep, hipStream_t s) {
  const int64_t cblocks = (C + kMaskThreads - 1) / kMaskThreads;
  const dim3 grid(static_cast<uint32_t>((O / G) * cblocks));
  const dim3 block(kMaskThreads);
  switch (G) {
    case 2: hipLaunchKernelGGL((td_mask_fixed<2, WT>), grid, block, 0, s, W, bits, C, cblocks, n_target, thr, We, keep); break;
    case 4: hipLaunchKernelGGL((td_mask_fixed<4, WT>), grid, block, 0, s, W, bits, C, cblocks, n_target, thr, We, keep); break;
    case 8: hipLaunchKernelGGL((td_mask_fixed<8, WT>), grid, block, 0, s, W, bits, C, cblocks, n_target, thr, We, keep); break;
    case 16: hipLaunchKernelGGL((td_mask_fixed<16, WT>), grid, block, 0, s, W, bits, C, cblocks, n_target, thr, We, keep); break;
    case 32: hipLaunchKernelGGL((td_mask_fixed<32, WT>), grid, block, 0, s, W, bits, C, cblocks, n_target, thr, We, keep); break;
    default:
      hipLaunchKernelGGL((td_mask_generic<WT>), grid, block, 0, s, W, bits, C, cblocks, G, n_target, thr, We, keep);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Gradient of the packed values.  A workgroup owns GB consecutive groups and
// 256 columns (a lane per column); per pass over the rows it takes KB slots
// of every group, so one staged X[n][c] feeds GB * KB multiply-adds.

constexpr int kGradThreads = 256;     // columns of a workgroup
constexpr int kGradLdsFloats = 8192;  // dY staging (32 KiB): rows per pass = min(32, 8192 / (GB * G))

template <typename T> __device__ __forceinline__ float ld(const T* p, int64_t i);
template <> __device__ __forceinline__ float ld<float>(const float* p, int64_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld<bf16_t>(const bf16_t* p, int64_t i) { return bf16_to_f32(p[i].bits); }

template <typename T, int GB, int KB>
__global__ __launch_bounds__(kGradThreads) void grad_packed_kernel(const T* __restrict__ dY, const T* __restrict__ X,
                                                                   const uint8_t* __restrict__ idx,
                                                                   float* __restrict__ dv, int64_t N, int64_t C,
                                                                   int64_t O, int32_t G, int32_t K, int64_t cblocks,
                                                                   int32_t R) {
  extern __shared__ __attribute__((aligned(16))) float lds_f[];
  float* Xs = lds_f;                       // R rows x 256 columns of X
  float* dYs = lds_f + R * kGradThreads;   // R rows x (GB * G) outputs of dY
  const int64_t ngroups = O / G;
  const int64_t g0 = (blockIdx.x / cblocks) * GB;
  const int32_t gcount = static_cast<int32_t>(ngroups - g0 < GB ? ngroups - g0 : GB);
  const int64_t c = (blockIdx.x % cblocks) * kGradThreads + threadIdx.x;
  const bool live = c < C;
  const int32_t width = gcount * G;  // dY columns staged per row
  for (int32_t k0 = 0; k0 < K; k0 += KB) {
    int off[GB][KB];  // LDS offset of the entry each slot gathers, inside a staged row
    float acc[GB][KB];
#pragma unroll
    for (int gi = 0; gi < GB; ++gi)
#pragma unroll
      for (int k = 0; k < KB; ++k) {
        const bool on = live && gi < gcount && k0 + k < K;
        const int ix = on ? idx[((g0 + gi) * K + k0 + k) * C + c] : 0;
        off[gi][k] = gi * G + (ix < G ? ix : G - 1);  // (a packing from cci_pack always has idx < G)
        acc[gi][k] = 0.0f;
      }
    for (int64_t n0 = 0; n0 < N; n0 += R) {
      const int rows = static_cast<int>(N - n0 < R ? N - n0 : R);
      __syncthreads();  // the previous pass's readers are done with dYs / Xs
      // stage the pass's dY rows (restricted to the groups) and X rows
      // (restricted to the columns): every load in flight at once
      for (int t = threadIdx.x; t < rows * width; t += kGradThreads) {
        const int n = t / width, q = t - n * width;
        dYs[t] = ld<T>(dY, (n0 + n) * O + g0 * G + q);
      }
      for (int n = 0; n < rows; ++n) Xs[n * kGradThreads + threadIdx.x] = live ? ld<T>(X, (n0 + n) * C + c) : 0.0f;
      __syncthreads();
      if (live) {
        for (int n = 0; n < rows; ++n) {
          const float x = Xs[n * kGradThreads + threadIdx.x];
          const float* row = dYs + n * width;
#pragma unroll
          for (int gi = 0; gi < GB; ++gi)
#pragma unroll
            for (int k = 0; k < KB; ++k) acc[gi][k] = __builtin_fmaf(row[off[gi][k]], x, acc[gi][k]);
        }
      }
    }
    if (live) {
#pragma unroll
      for (int gi = 0; gi < GB; ++gi)
#pragma unroll
        for (int k = 0; k < KB; ++k)
          if (gi < gcount && k0 + k < K) dv[((g0 + gi) * K + k0 + k) * C + c] = acc[gi][k];
    }
  }
}

template <typename T, int GB, int KB>
hipError_t grad_launch(const T* dY, const T* X, int64_t N, int64_t C, const uint8_t* idx, int64_t O, int32_t G,
                       int32_t K, float* dv, hipStream_t s) {
  const int64_t cblocks = (C + kGradThreads - 1) / kGradThreads;
  const int64_t gblocks = (O / G + GB - 1) / GB;
  const dim3 grid(static_cast<uint32_t>(gblocks * cblocks));
  const int32_t R = static_cast<int32_t>(std::max<int64_t>(1, std::min<int64_t>(32, kGradLdsFloats / (GB * G))));
  const size_t lds = static_cast<size_t>(R) * (GB * G + kGradThreads) * sizeof(float);
  hipLaunchKernelGGL((grad_packed_kernel<T, GB, KB>), grid, dim3(kGradThreads), lds, s, dY, X, idx, dv, N, C, O, G, K,
                     cblocks, R);
  return hipGetLastError();
}

template <typename T>
hipError_t grad_typed(const T* dY, const T* X, int64_t N, int64_t C, const uint8_t* idx, int64_t O, int32_t G,
                      int32_t K, float* dv, hipStream_t s) {
  // four groups per workgroup (X read once per four groups; enough
  // workgroups to fill the chip), up to eight slots of each per pass
  if (K == 1) return grad_launch<T, 4, 1>(dY, X, N, C, idx, O, G, K, dv, s);
  if (K == 2) return grad_launch<T, 4, 2>(dY, X, N, C, idx, O, G, K, dv, s);
  if (K <= 4) return grad_launch<T, 4, 4>(dY, X, N, C, idx, O, G, K, dv, s);
  return grad_launch<T, 4, 8>(dY, X, N, C, idx, O, G, K, dv, s);
}

}  // namespace

hipError_t launch_td_mask(const float* W, int64_t O, int64_t C, int32_t G, int32_t n_target, const uint32_t* bits,
                          uint64_t thr, void* We, DType w_t, uint8_t* keep, hipStream_t s) {
  if (w_t == DType::F32) return td_mask_typed<float>(W, O, C, G, n_target, bits, thr, static_cast<float*>(We), keep, s);
  return td_mask_typed<bf16_t>(W, O, C, G, n_target, bits, thr, static_cast<bf16_t*>(We), keep, s);
}

hipError_t launch_grad_packed(const void* dY, const void* X, DType t, int64_t N, int64_t C, const uint8_t* idx,
                              int64_t O, int32_t G, int32_t K, float* dv, hipStream_t s) {
  // bf16 operands of at least one reduction step go to the matrix cores
  if (N >= 32 && grad_mfma_supports(dY, X, t, N, C, O, G)) return launch_grad_mfma(dY, X, N, C, idx, O, G, K, dv, s);
  if (t == DType::F32)
    return grad_typed<float>(static_cast<const float*>(dY), static_cast<const float*>(X), N, C, idx, O, G, K, dv, s);
  return grad_typed<bf16_t>(static_cast<const bf16_t*>(dY), static_cast<const bf16_t*>(X), N, C, idx, O, G, K, dv, s);
}

}  // namespace cci
