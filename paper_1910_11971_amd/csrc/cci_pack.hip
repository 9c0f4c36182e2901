// Magnitude projection onto CCI sparsity (paper Sec. 5.1 with the group
// constraint of Sec. 3.1): one lane per (group g, column c).
//
// HBM-bound: reads the G weights of its group column (consecutive lanes read
// consecutive columns, so each of the G row reads is coalesced), ranks them by
// |w| and writes the K survivors (value + intra-group row) in ascending row
// order, one coalesced store per slot.
#include "cci_device.hpp"
#include "cci_launch.hpp"

namespace cci {
namespace {

constexpr int kPackThreads = 256;

__device__ __forceinline__ uint32_t abs_bits(float w) { return __float_as_uint(w) & 0x7fffffffu; }

template <typename VT> __device__ __forceinline__ void put(VT* p, int64_t i, float w);
template <> __device__ __forceinline__ void put<float>(float* p, int64_t i, float w) { p[i] = w; }
template <> __device__ __forceinline__ void put<bf16_t>(bf16_t* p, int64_t i, float w) {
  p[i].bits = f32_to_bf16_rne(w);
}

// Register-resident group (G known at compile time).  The rank of row r is
// the number of rows that beat it (larger |w|, or equal |w| and a lower
// row); each pair of rows is compared once and credits one of the two.  (For
// K < (G - 1) / 2 the K winners are taken one at a time instead: the same
// set, in fewer operations; the ranking is vector-ALU work comparable to
// the kernel's HBM time.)
// The kept rows form a bit mask; slot k then takes the k-th lowest kept row,
// so each slot is one store of consecutive columns (coalesced), its value
// re-read from the cache lines just loaded.  With K = G every row is kept in
// order (the dense control): a copy.
template <int G, typename VT>
__global__ __launch_bounds__(kPackThreads) void pack_fixed(const float* __restrict__ W, int64_t C,
                                                           int64_t cblocks, int32_t K,
                                                           VT* __restrict__ vals,
                                                           uint8_t* __restrict__ idx) {
  const int64_t blk = blockIdx.x;
  const int64_t g = blk / cblocks;
  const int64_t c = (blk % cblocks) * kPackThreads + threadIdx.x;
  if (c >= C) return;
  const float* col = W + g * G * C + c;
  if (K == G) {
#pragma unroll
    for (int r = 0; r < G; ++r) {
      const int64_t o = (g * K + r) * C + c;
      put<VT>(vals, o, col[r * C]);
      idx[o] = static_cast<uint8_t>(r);
    }
    return;
  }
  uint32_t key[G];
#pragma unroll
  for (int r = 0; r < G; ++r) key[r] = abs_bits(col[r * C]);
  uint32_t kept = 0;
  if (2 * K + 1 < G) {
    // Few kept rows: take the largest remaining |w| K times (a strict
    // comparison scanning up from row 0 keeps the lower row on a tie; a
    // taken row's key drops below every |w|): 3 G K operations against the
    // 3 G (G - 1) / 2 of the pairwise rank.
    int32_t sk[G];
#pragma unroll
    for (int r = 0; r < G; ++r) sk[r] = static_cast<int32_t>(key[r]);
    for (int32_t k = 0; k < K; ++k) {
      int32_t best = sk[0];
      int br = 0;
#pragma unroll
      for (int r = 1; r < G; ++r) {
        const bool gt = sk[r] > best;
        best = gt ? sk[r] : best;
        br = gt ? r : br;
      }
      kept |= 1u << br;
#pragma unroll
      for (int r = 0; r < G; ++r) sk[r] = r == br ? -1 : sk[r];
    }
  } else {
    int rank[G];
#pragma unroll
    for (int r = 0; r < G; ++r) rank[r] = 0;
#pragma unroll
    for (int r = 1; r < G; ++r)
#pragma unroll
      for (int q = 0; q < r; ++q) {
        const bool q_wins = key[q] >= key[r];  // q < r: a tie goes to q
        rank[r] += q_wins ? 1 : 0;
        rank[q] += q_wins ? 0 : 1;
      }
#pragma unroll
    for (int r = 0; r < G; ++r) kept |= (rank[r] < K ? 1u : 0u) << r;
  }
  for (int32_t k = 0; k < K; ++k) {
    const int r = __builtin_ctz(kept);
    kept &= kept - 1u;
    const int64_t o = (g * K + k) * C + c;
    put<VT>(vals, o, col[static_cast<int64_t>(r) * C]);
    idx[o] = static_cast<uint8_t>(r);
  }
}

// Any G <= 256: the group column is re-read from cache for each rank count.
template <typename VT>
__global__ __launch_bounds__(kPackThreads) void pack_generic(const float* __restrict__ W, int64_t C,
                                                             int64_t cblocks, int32_t G, int32_t K,
                                                             VT* __restrict__ vals,
                                                             uint8_t* __restrict__ idx) {
  const int64_t blk = blockIdx.x;
  const int64_t g = blk / cblocks;
  const int64_t c = (blk % cblocks) * kPackThreads + threadIdx.x;
  if (c >= C) return;
  const float* col = W + g * G * C + c;
  int slot = 0;
  for (int r = 0; r < G && slot < K; ++r) {
    const float wr = col[r * C];
    const uint32_t kr = abs_bits(wr);
    int rank = 0;
    for (int q = 0; q < G; ++q) {
      const uint32_t kq = abs_bits(col[q * C]);
      rank += (kq > kr) || (kq == kr && q < r);
    }
    if (rank < K) {
      const int64_t o = (g * K + slot) * C + c;
      put<VT>(vals, o, wr);
      idx[o] = static_cast<uint8_t>(r);
      ++slot;
    }
  }
}

template <typename VT>
hipError_t launch_typed(const float* W, int64_t O, int64_t C, int32_t G, int32_t K, VT* vals,
                        uint8_t* idx, hipStream_t s) {
  const int64_t cblocks = (C + kPackThreads - 1) / kPackThreads;
  const dim3 grid(static_cast<uint32_t>((O / G) * cblocks));
  const dim3 block(kPackThreads);
  switch (G) {
    case 2: hipLaunchKernelGGL((pack_fixed<2, VT>), grid, block, 0, s, W, C, cblocks, K, vals, idx); break;
    case 4: hipLaunchKernelGGL((pack_fixed<4, VT>), grid, block, 0, s, W, C, cblocks, K, vals, idx); break;
    case 8: hipLaunchKernelGGL((pack_fixed<8, VT>), grid, block, 0, s, W, C, cblocks, K, vals, idx); break;
    case 16: hipLaunchKernelGGL((pack_fixed<16, VT>), grid, block, 0, s, W, C, cblocks, K, vals, idx); break;
    case 32: hipLaunchKernelGGL((pack_fixed<32, VT>), grid, block, 0, s, W, C, cblocks, K, vals, idx); break;
    default:
      hipLaunchKernelGGL((pack_generic<VT>), grid, block, 0, s, W, C, cblocks, G, K, vals, idx);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_pack(const float* W, int64_t O, int64_t C, int32_t G, int32_t K, void* vals,
                       DType val_t, uint8_t* idx, hipStream_t s) {
  if (val_t == DType::F32)
    return launch_typed<float>(W, O, C, G, K, static_cast<float*>(vals), idx, s);
  return launch_typed<bf16_t>(W, O, C, G, K, static_cast<bf16_t*>(vals), idx, s);
}

}  // namespace cci
