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

// Register-resident group (G known at compile time, a power of two).
//
// The order is |w| descending, then row ascending.  Each key gets its row in
// its low log2(G) bits, (|w| with those bits cleared) | (G - 1 - r): the keys
// are then distinct, and they order the rows exactly as |w| does wherever
// two |w| differ above those bits.  With distinct keys the next largest key
// below p is p - 1 - min_r(p - 1 - key_r) in unsigned arithmetic (keys below
// p give p - 1 - key_r < p; the others wrap past 2^31), two operations per
// row and round; the next smallest above p likewise.  min(K, G - K) + 1
// rounds find the boundary of the kept set from the nearer end, and the kept
// set is the exact one unless the last kept and the first dropped key agree
// above the row bits: such columns (ties, or |w| closer than 2^-19 relative)
// are ranked exactly, each pair of rows compared once.
// The kept rows form a bit mask; slot k then takes the k-th lowest kept row,
// so each slot is one store of consecutive columns (coalesced), its value
// re-read from the cache lines just loaded (four slots' loads in flight at
// once).  With K = G every row is kept in order (the dense control): a copy.
template <int G> struct RowBits {
  static constexpr int value = G == 2 ? 1 : G == 4 ? 2 : G == 8 ? 3 : G == 16 ? 4 : 5;
};

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
  constexpr int kRB = RowBits<G>::value;
  constexpr uint32_t kRM = (1u << kRB) - 1u;
  static_assert((1 << kRB) == G, "G must be a power of two up to 32");
  uint32_t key[G];
#pragma unroll
  for (int r = 0; r < G; ++r) key[r] = (abs_bits(col[r * C]) & ~kRM) | (kRM - r);
  uint32_t kept = 0;
  bool exact;
  if (2 * K <= G) {
    // Largest keys: K rounds, then one more for the first dropped key.
    uint32_t p = 0x80000000u, last = 0;
    for (int32_t k = 0; k <= K; ++k) {
      uint32_t m = 0xffffffffu;
#pragma unroll
      for (int r = 0; r < G; ++r) m = min(m, p - 1u - key[r]);
      last = p;
      p = p - 1u - m;
      if (k < K) kept |= 1u << (kRM - (p & kRM));
    }
    exact = (last >> kRB) != (p >> kRB);
  } else {
    // Smallest keys: the G - K dropped rows, then the first kept key.
    const int32_t D = G - K;
    uint32_t p = 0xffffffffu, last = 0, dropped = 0;
    for (int32_t k = 0; k <= D; ++k) {
      uint32_t m = 0xffffffffu;
#pragma unroll
      for (int r = 0; r < G; ++r) m = min(m, key[r] - p - 1u);
      last = p;
      p = p + 1u + m;
      if (k < D) dropped |= 1u << (kRM - (p & kRM));
    }
    constexpr uint32_t kAll = G == 32 ? 0xffffffffu : (1u << (G & 31)) - 1u;
    kept = ~dropped & kAll;
    exact = (last >> kRB) != (p >> kRB);
  }
  if (__builtin_expect(!exact, 0)) {
    uint32_t full[G];
#pragma unroll
    for (int r = 0; r < G; ++r) full[r] = abs_bits(col[r * C]);
    int rank[G];
#pragma unroll
    for (int r = 0; r < G; ++r) rank[r] = 0;
#pragma unroll
    for (int r = 1; r < G; ++r)
#pragma unroll
      for (int q = 0; q < r; ++q) {
        const bool q_wins = full[q] >= full[r];  // q < r: a tie goes to q
        rank[r] += q_wins ? 1 : 0;
        rank[q] += q_wins ? 0 : 1;
      }
    kept = 0;
#pragma unroll
    for (int r = 0; r < G; ++r) kept |= (rank[r] < K ? 1u : 0u) << r;
  }
  for (int32_t k0 = 0; k0 < K; k0 += 4) {
    int rr[4];
    float v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      rr[j] = __builtin_ctz(kept | 0x80000000u);
      kept &= kept - 1u;
      if (k0 + j < K) v[j] = col[static_cast<int64_t>(rr[j]) * C];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (k0 + j < K) {
        const int64_t o = (g * K + k0 + j) * C + c;
        put<VT>(vals, o, v[j]);
        idx[o] = static_cast<uint8_t>(rr[j]);
      }
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
