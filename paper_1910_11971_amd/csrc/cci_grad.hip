// Gradient of the packed values of a CCI layer on the matrix cores (the
// training step of improved targeted dropout, Sec. 5.1 / Sec. 6, once the
// mask is fixed):
//   dvals[g][k][c] = sum_n dY[n][gG + idx[g][k][c]] * X[n][c],
// the kept entries of the weight gradient dY^T X.  A vector-ALU kernel that
// multiplies only kept entries does K/G of the dense work, but at 1/32 of
// the matrix cores' rate; so for bf16 operands the dense tile of dY^T X is
// computed on v_mfma_f32_16x16x32_bf16 and only its kept entries are
// written.
//
// Work split: a workgroup (four waves, one per SIMD) owns 256 outputs x 256
// columns; wave w accumulates outputs 128 (w % 2) .. +127 x columns
// 128 (w / 2) .. +127 in its 256 accumulation registers.  The reduction
// runs over samples in steps of 32:
//   - both operands are sample-major ([N][O] and [N][C]); each step's 32 rows
//     of the workgroup's dY and X columns are DMA'd into LDS row by row
//     (buffer_load ... lds; three buffers, two steps ahead), 16-byte chunk c
//     of row r at chunk c ^ f(r), f(r) = 2 ((r % 4) + 4 ((r / 8) % 2));
//   - the MFMA operands need 8 consecutive samples per lane: they are read
//     with ds_read_b64_tr_b16, which hands each lane of a 16-lane group one
//     column of the 4 x 16 block its lanes address (two reads per fragment).
//     With the swizzle every such read touches each 32-byte bank slot at
//     most twice (512 bytes in two LDS cycles);
//   - a step's fragments are read while the previous step's MFMAs issue;
//   - after the last step each wave parks 128 outputs x 32 columns of its
//     accumulators in LDS at a time and gathers the entries the packed
//     indices name: row gG + idx of column c goes to dvals[g][k][c].
// bf16 inputs widen exactly; products and sums are fp32.
#include "cci_device.hpp"
#include "cci_launch.hpp"

namespace cci {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4_t;
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kThreads = 256;  // four waves, one per SIMD
constexpr int kTile = 256;     // workgroup tile: 256 outputs x 256 columns
constexpr int kRows = 32;      // samples per reduction step
constexpr int kOpBytes = kRows * kTile * 2;  // one operand of one step (16 KiB)
constexpr int kStage = 2 * kOpBytes;         // dY then X
constexpr int kBufs = 3;
constexpr int kLds = kBufs * kStage;         // 96 KiB
constexpr int kEpPitch = 136;                // epilogue staging: floats per parked column (128 + 8)
constexpr int kXcds = 8;
constexpr uint32_t kOOB = 0x80000000u;  // buffer offset that reads as zero
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer descriptor word 3 (gfx9 family)
static_assert(4 * 32 * kEpPitch * 4 <= kLds, "epilogue staging reuses the operand buffers");

struct GParams {
  const uint16_t* dY;
  const uint16_t* X;
  const uint8_t* idx;
  float* dv;
  uint32_t dy_bytes, x_bytes;
  int32_t N, C, O, G, K;
  int32_t nob, ncb, nsteps;  // output blocks, column blocks (of 256), reduction steps
  int32_t grid8;             // grid / 8 when the grid is a multiple of 8, else 0
};

__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
// acc += A * B with the accumulator pinned to the accumulation registers (all
// 256 of them hold the wave's 128 x 128 block).  Vector accesses of an
// accumulator are separated from MFMAs that write it by mfma_drain().
__device__ __forceinline__ void mfma_acc(f32x4_t& acc, const bf16x8_t a, const bf16x8_t b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
__device__ __forceinline__ void mfma_drain() { asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 15\n\ts_nop 15" ::: "memory"); }

// XOR of the 16-byte chunk index in staged row r (even: a 32-byte pair stays a pair).
__device__ __forceinline__ uint32_t swz(uint32_t r) { return 2u * ((r & 3u) | (((r >> 3) & 1u) << 2)); }

// One MFMA operand fragment (8 samples x 16 columns, transposed to a lane per
// column) from the tile at byte `a`: two transposing reads, samples 0-3 and 4-7.
__device__ __forceinline__ bf16x8_t frag(const uint8_t* lds, uint32_t a) {
  const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(lds + a));
  const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(lds + a + 4 * kTile * 2));
  const u32x2_t l2 = __builtin_bit_cast(u32x2_t, lo), h2 = __builtin_bit_cast(u32x2_t, hi);
  return __builtin_bit_cast(bf16x8_t, u32x4_t{l2[0], l2[1], h2[0], h2[1]});
}

__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void grad_mfma_kernel(GParams p) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wo = w & 1, wc = w >> 1;

  // ---- tile of this workgroup (dispatch places workgroup b on XCD b % 8) ----
  const uint32_t bid = blockIdx.x;
  const uint32_t L = p.grid8 ? (bid & 7u) * static_cast<uint32_t>(p.grid8) + (bid >> 3) : bid;
  const int ob = static_cast<int>(L / static_cast<uint32_t>(p.ncb));
  const int cb = static_cast<int>(L - static_cast<uint32_t>(ob * p.ncb));
  const int o0 = ob * kTile, c0 = cb * kTile;

  // ---- DMA: instruction j (0..31) of a step fills slots 64 j .. 64 j + 63 of
  // the stage: j < 16 the dY rows, else the X rows.  Wave w issues j = w + 4 i.
  const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.dY), (short)0, static_cast<int>(p.dy_bytes), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.X), (short)0, static_cast<int>(p.x_bytes), kRsrcWord3);
  uint32_t soff[8];  // source byte offset at step 0 (kOOB: a column past the operand)
  uint32_t srow[8];  // the slot's staged row
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int j = w + 4 * i;
    const uint32_t s = static_cast<uint32_t>(((j & 15) << 6) + lane);  // slot within the operand
    const uint32_t r = s >> 5;                                          // 32 chunks per row
    const uint32_t cc = (s & 31u) ^ swz(r);                             // logical chunk held by the slot
    const bool isx = j >= 16;
    const uint32_t width = static_cast<uint32_t>(isx ? p.C : p.O);
    const uint32_t col = static_cast<uint32_t>(isx ? c0 : o0) + 8u * cc;
    srow[i] = r;
    soff[i] = col < width ? (r * width + col) * 2u : kOOB;
  }
  const auto issue = [&](int step, int buf) {
    const uint32_t n0 = static_cast<uint32_t>(step * kRows);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int j = w + 4 * i;
      const bool isx = i >= 4;  // (j >= 16 exactly when i >= 4)
      const uint32_t width = static_cast<uint32_t>(isx ? p.C : p.O);
      const bool ok = soff[i] != kOOB && n0 + srow[i] < static_cast<uint32_t>(p.N);
      const uint32_t off = ok ? soff[i] + n0 * width * 2u : kOOB;
      lds_void_t* d = (lds_void_t*)(lds + buf * kStage + j * 1024);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(isx ? xr : yr, d, 16, off, 0, 0, 0);
    }
  };

  // ---- fragment addresses (within an operand tile) ----------------------------
  // Lane l of 16-lane group q addresses row 8 q + (l % 16) / 4, columns
  // 16 m + 4 (l % 4) .. +3 of block m: chunk 2 m + (l % 4) / 2 (swizzled),
  // half (l % 4) % 2.
  const uint32_t q = static_cast<uint32_t>(lane >> 4), li = static_cast<uint32_t>(lane & 15);
  const uint32_t fr = 8u * q + (li >> 2);
  const uint32_t fh = swz(fr) >> 1;  // in [0, 8)
  const uint32_t fbase = fr * (kTile * 2) + 16u * ((li & 3u) >> 1) + 8u * (li & 1u);
  uint32_t aoff[8], boff[8];
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    aoff[m] = fbase + 32u * (static_cast<uint32_t>(m) ^ fh) + static_cast<uint32_t>(wo * 256);
    boff[m] = kOpBytes + fbase + 32u * (static_cast<uint32_t>(m) ^ fh) + static_cast<uint32_t>(wc * 256);
  }

  f32x4_t acc[8][8];
#pragma unroll
  for (int m = 0; m < 8; ++m)
#pragma unroll
    for (int n = 0; n < 8; ++n) acc[m][n] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  mfma_drain();

  // Step s's fragments are read during step s - 1's MFMAs: at iteration s the
  // wave waits for step s + 1's rows, meets the others at the barrier (after
  // which nobody reads buffer s % 3 any more: its fragments are in registers),
  // queues step s + 3 into that buffer, reads step s + 1's fragments and
  // issues step s's MFMAs.
  const int nsteps = p.nsteps;
  issue(0, 0);
  if (nsteps > 1) issue(1, 1);
  if (nsteps > 2) issue(2, 2);
  if (nsteps > 2) wait_vm<16>(); else if (nsteps > 1) wait_vm<8>(); else wait_vm<0>();
  lds_barrier();
  bf16x8_t a[8], b[8];
#pragma unroll
  for (int m = 0; m < 8; ++m) a[m] = frag(lds, aoff[m]);
#pragma unroll
  for (int n = 0; n < 8; ++n) b[n] = frag(lds, boff[n]);
  for (int s = 0; s < nsteps; ++s) {
    bf16x8_t an[8], bn[8];
    if (s + 1 < nsteps) {
      if (s + 2 < nsteps) wait_vm<8>(); else wait_vm<0>();  // this wave's DMAs of step s + 1
      lds_barrier();
      if (s + 3 < nsteps) issue(s + 3, s % 3);
      const uint32_t sb = static_cast<uint32_t>(((s + 1) % 3) * kStage);
#pragma unroll
      for (int m = 0; m < 8; ++m) an[m] = frag(lds, sb + aoff[m]);
#pragma unroll
      for (int n = 0; n < 8; ++n) bn[n] = frag(lds, sb + boff[n]);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int m = 0; m < 8; ++m)
#pragma unroll
      for (int n = 0; n < 8; ++n) mfma_acc(acc[m][n], a[m], b[n]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      a[m] = an[m];
      b[m] = bn[m];
    }
  }
  mfma_drain();
  lds_barrier();  // every wave is done with the operand buffers

  // ---- gather the kept entries ---------------------------------------------------
  // Lane (q, li) holds D[16 m + 4 q + j][16 n + li] of block (m, n); per pass
  // of 32 columns (blocks n = 2 t, 2 t + 1) the wave parks them column-major
  // (pitch kEpPitch floats) and reads back row gG + idx of each column: lane l
  // takes columns 4 (l % 8) .. +3 of packed rows l / 8 + 8 x (one 4-byte index
  // load and one 16-byte store per row), its index loads issued together.
  float* stg = reinterpret_cast<float*>(lds) + w * 32 * kEpPitch;
  const int ow0 = o0 + 128 * wo;   // the wave's first output
  const int gw0 = ow0 / p.G;       // its first group (G divides 128)
  const int ngw = 128 / p.G;       // its groups
  const int ngroups = p.O / p.G;
  const int nrow = ngw * p.K;      // packed rows (g, k) of its groups
  const int cq = lane & 7, r0 = lane >> 3;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
#pragma unroll
    for (int m = 0; m < 8; ++m)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        *reinterpret_cast<f32x4_t*>(stg + (16 * h + li) * kEpPitch + 16 * m + 4 * q) = acc[m][2 * t + h];
    const int c = c0 + 128 * wc + 32 * t + 4 * cq;  // the lane's first column
    const bool cok = c < p.C;
#pragma unroll 1
    for (int x0 = 0; 8 * x0 < nrow; x0 += 4) {
      uint32_t iv[4];
      int64_t e[4];
      bool ok[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const int r = r0 + 8 * (x0 + x);
        const int gi = r / p.K, k = r - gi * p.K;
        ok[x] = cok && r < nrow && gw0 + gi < ngroups;
        e[x] = (static_cast<int64_t>(gw0 + gi) * p.K + k) * p.C + c;
        iv[x] = ok[x] ? *reinterpret_cast<const uint32_t*>(p.idx + e[x]) : 0u;
      }
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        if (ok[x]) {
          const int r = r0 + 8 * (x0 + x);
          const int gbase = (r / p.K) * p.G;  // the group's first row within the wave
          f32x4_t v;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            uint32_t ix = (iv[x] >> (8 * j)) & 0xffu;
            ix = ix < static_cast<uint32_t>(p.G) ? ix : static_cast<uint32_t>(p.G - 1);
            v[j] = stg[(4 * cq + j) * kEpPitch + gbase + static_cast<int>(ix)];
          }
          *reinterpret_cast<f32x4_t*>(p.dv + e[x]) = v;
        }
      }
    }
  }
}

}  // namespace

bool grad_mfma_supports(const void* dY, const void* X, DType t, int64_t N, int64_t C, int64_t O, int32_t G) {
  if (t != DType::BF16 || N < 1) return false;
  if (O % 8 != 0 || C % 8 != 0 || G < 1 || 128 % G != 0) return false;
  const auto al = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
  if (!al(dY) || !al(X)) return false;
  const int64_t lim = static_cast<int64_t>(kOOB);
  return N * O * 2 < lim && N * C * 2 < lim;
}

hipError_t launch_grad_mfma(const void* dY, const void* X, int64_t N, int64_t C, const uint8_t* idx, int64_t O,
                            int32_t G, int32_t K, float* dv, hipStream_t s) {
  GParams p{};
  p.dY = static_cast<const uint16_t*>(dY);
  p.X = static_cast<const uint16_t*>(X);
  p.idx = idx;
  p.dv = dv;
  p.dy_bytes = static_cast<uint32_t>(N * O * 2);
  p.x_bytes = static_cast<uint32_t>(N * C * 2);
  p.N = static_cast<int32_t>(N);
  p.C = static_cast<int32_t>(C);
  p.O = static_cast<int32_t>(O);
  p.G = G;
  p.K = K;
  p.nob = static_cast<int32_t>((O + kTile - 1) / kTile);
  p.ncb = static_cast<int32_t>((C + kTile - 1) / kTile);
  p.nsteps = static_cast<int32_t>((N + kRows - 1) / kRows);
  const int64_t grid = static_cast<int64_t>(p.nob) * p.ncb;
  if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
  p.grid8 = grid % kXcds == 0 ? static_cast<int32_t>(grid / kXcds) : 0;
  static std::atomic<int8_t> lds_set[kMaxDevices];
  const hipError_t attr = set_lds_limit_once(lds_set, reinterpret_cast<const void*>(&grad_mfma_kernel), kLds);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(grad_mfma_kernel, dim3(static_cast<uint32_t>(grid)), dim3(kThreads), kLds, s, p);
  return hipGetLastError();
}

}  // namespace cci
