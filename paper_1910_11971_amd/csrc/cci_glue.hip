// CNN glue for the ResNet-shaped forward: NHWC max pooling and global average
// pooling.  Memory-bound elementwise/reduction kernels, consecutive lanes on
// consecutive channels (coalesced): bf16 max pooling with C % 8 == 0 gives a
// lane 8 channels of one output pixel (16-byte reads and writes, 32-bit
// index arithmetic); otherwise one lane per output element.
#include "cci_device.hpp"
#include "cci_launch.hpp"

namespace cci {
namespace {

constexpr int kThreads = 256;

template <typename T>
__global__ __launch_bounds__(kThreads) void maxpool_kernel(const T* __restrict__ X, int64_t B,
                                                           int64_t H, int64_t W, int64_t C,
                                                           int32_t k, int32_t st, int32_t p,
                                                           int64_t Ho, int64_t Wo,
                                                           T* __restrict__ Y) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
  const int64_t total = B * Ho * Wo * C;
  if (e >= total) return;
  const int64_t c = e % C;
  const int64_t pix = e / C;
  const int64_t ow = pix % Wo;
  const int64_t oh = (pix / Wo) % Ho;
  const int64_t b = pix / (Wo * Ho);
  float m = -__builtin_inff();
  for (int32_t i = 0; i < k; ++i) {
    const int64_t ih = oh * st - p + i;
    if (ih < 0 || ih >= H) continue;
    for (int32_t jj = 0; jj < k; ++jj) {
      const int64_t iw = ow * st - p + jj;
      if (iw < 0 || iw >= W) continue;
      const float v = io<T>::load(X, ((b * H + ih) * W + iw) * C + c);
      m = v > m ? v : m;
    }
  }
  io<T>::store(Y, e, m);  // exact: m is one of the inputs
}

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// bf16, C % 8 == 0: lane e owns channels 8 (e % C8) .. +7 of output pixel
// e / C8.  The window is scanned in the same order with the same comparison
// as maxpool_kernel, so the result is the same input value.
__global__ __launch_bounds__(kThreads) void maxpool_bf16x8_kernel(const u32x4_t* __restrict__ X, uint32_t H,
                                                                  uint32_t W, uint32_t C8, int32_t k, int32_t st,
                                                                  int32_t p, uint32_t Ho, uint32_t Wo,
                                                                  uint32_t total, u32x4_t* __restrict__ Y) {
  const uint32_t e = blockIdx.x * kThreads + threadIdx.x;
  if (e >= total) return;
  const uint32_t c8 = e % C8;
  const uint32_t pix = e / C8;
  const uint32_t ow = pix % Wo;
  const uint32_t t = pix / Wo;
  const uint32_t oh = t % Ho;
  const uint32_t b = t / Ho;
  float m[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) m[j] = -__builtin_inff();
  for (int32_t i = 0; i < k; ++i) {
    const int32_t ih = static_cast<int32_t>(oh) * st - p + i;
    if (ih < 0 || ih >= static_cast<int32_t>(H)) continue;
    for (int32_t jj = 0; jj < k; ++jj) {
      const int32_t iw = static_cast<int32_t>(ow) * st - p + jj;
      if (iw < 0 || iw >= static_cast<int32_t>(W)) continue;
      const u32x4_t v = X[((b * H + static_cast<uint32_t>(ih)) * W + static_cast<uint32_t>(iw)) * C8 + c8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float f = __uint_as_float((j & 1) ? (v[j >> 1] & 0xffff0000u) : (v[j >> 1] << 16));
        m[j] = f > m[j] ? f : m[j];
      }
    }
  }
  u32x4_t out;
#pragma unroll
  for (int j = 0; j < 4; ++j)  // exact: every m is an input value (or -inf), its top 16 bits
    out[j] = (__float_as_uint(m[2 * j]) >> 16) | (__float_as_uint(m[2 * j + 1]) & 0xffff0000u);
  Y[e] = out;
}

template <typename XT, typename YT>
__global__ __launch_bounds__(kThreads) void avgpool_kernel(const XT* __restrict__ X, int64_t B,
                                                           int64_t HW, int64_t C,
                                                           YT* __restrict__ Y) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
  if (e >= B * C) return;
  const int64_t c = e % C;
  const int64_t b = e / C;
  float acc = 0.0f;
  for (int64_t i = 0; i < HW; ++i) acc += io<XT>::load(X, (b * HW + i) * C + c);
  io<YT>::store(Y, e, acc / static_cast<float>(HW));
}

}  // namespace

hipError_t launch_maxpool(const void* X, DType t, int64_t B, int64_t H, int64_t W, int64_t C,
                          int32_t k, int32_t st, int32_t p, void* Y, hipStream_t s) {
  const int64_t Ho = (H + 2 * p - k) / st + 1;
  const int64_t Wo = (W + 2 * p - k) / st + 1;
  const int64_t total = B * Ho * Wo * C;
  const auto al16 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15u) == 0; };
  if (t == DType::BF16 && C % 8 == 0 && al16(X) && al16(Y) && B * H * W * C < (int64_t{1} << 31) &&
      total < (int64_t{1} << 31)) {
    const uint32_t vt = static_cast<uint32_t>(total / 8);
    hipLaunchKernelGGL(maxpool_bf16x8_kernel, dim3((vt + kThreads - 1) / kThreads), dim3(kThreads), 0, s,
                       static_cast<const u32x4_t*>(X), static_cast<uint32_t>(H), static_cast<uint32_t>(W),
                       static_cast<uint32_t>(C / 8), k, st, p, static_cast<uint32_t>(Ho), static_cast<uint32_t>(Wo),
                       vt, static_cast<u32x4_t*>(Y));
    return hipGetLastError();
  }
  const dim3 grid(static_cast<uint32_t>((total + kThreads - 1) / kThreads));
  if (t == DType::F32)
    hipLaunchKernelGGL((maxpool_kernel<float>), grid, dim3(kThreads), 0, s,
                       static_cast<const float*>(X), B, H, W, C, k, st, p, Ho, Wo,
                       static_cast<float*>(Y));
  else
    hipLaunchKernelGGL((maxpool_kernel<bf16_t>), grid, dim3(kThreads), 0, s,
                       static_cast<const bf16_t*>(X), B, H, W, C, k, st, p, Ho, Wo,
                       static_cast<bf16_t*>(Y));
  return hipGetLastError();
}

hipError_t launch_avgpool(const void* X, DType x_t, int64_t B, int64_t H, int64_t W, int64_t C,
                          void* Y, DType y_t, hipStream_t s) {
  const dim3 grid(static_cast<uint32_t>((B * C + kThreads - 1) / kThreads));
  const int64_t HW = H * W;
  if (x_t == DType::F32 && y_t == DType::F32)
    hipLaunchKernelGGL((avgpool_kernel<float, float>), grid, dim3(kThreads), 0, s,
                       static_cast<const float*>(X), B, HW, C, static_cast<float*>(Y));
  else if (x_t == DType::BF16 && y_t == DType::F32)
    hipLaunchKernelGGL((avgpool_kernel<bf16_t, float>), grid, dim3(kThreads), 0, s,
                       static_cast<const bf16_t*>(X), B, HW, C, static_cast<float*>(Y));
  else if (x_t == DType::BF16 && y_t == DType::BF16)
    hipLaunchKernelGGL((avgpool_kernel<bf16_t, bf16_t>), grid, dim3(kThreads), 0, s,
                       static_cast<const bf16_t*>(X), B, HW, C, static_cast<bf16_t*>(Y));
  else
    hipLaunchKernelGGL((avgpool_kernel<float, bf16_t>), grid, dim3(kThreads), 0, s,
                       static_cast<const float*>(X), B, HW, C, static_cast<bf16_t*>(Y));
  return hipGetLastError();
}

}  // namespace cci
