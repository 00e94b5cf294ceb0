// Euler step of the rectified-flow sampler, x_out = x - dsigma * v, for the
// latent handed from one denoising stage to the next (the Step of the
// wavefront algorithm).  Each element is evaluated in float64 as one product
// and one difference and rounded once to the storage type (bf16 through a
// round-to-odd float32, nearest even).  HBM-bound: 16-byte vectors, a grid
// of 4 vectors per thread.

#include <hip/hip_runtime.h>

#include "ff_internal.h"
#include "ff_numeric.h"

namespace ff {
namespace {

constexpr int kThreads = 256;
constexpr int kVecPerThread = 4;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline double step(double x, double v, double dsigma) {
  // no contraction into an fma: the product is rounded before the difference
#pragma clang fp contract(off)
  const double p = dsigma * v;
  return x - p;
}

__global__ __launch_bounds__(kThreads) void euler_bf16_kernel(const u32x4* x,
                                                              const u32x4* __restrict__ v,
                                                              u32x4* y, int64_t n_vec,
                                                              double dsigma) {
  const int64_t base = (int64_t(blockIdx.x) * kVecPerThread) * kThreads + threadIdx.x;
#pragma unroll
  for (int u = 0; u < kVecPerThread; ++u) {
    const int64_t i = base + int64_t(u) * kThreads;
    if (i >= n_vec) break;
    const u32x4 a = x[i], b = v[i];
    u32x4 r;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const double lo = step(bf16_lo(a[j]), bf16_lo(b[j]), dsigma);
      const double hi = step(bf16_hi(a[j]), bf16_hi(b[j]), dsigma);
      r[j] = pack_bf16_rne(round_to_odd_f32(lo), round_to_odd_f32(hi));
    }
    y[i] = r;
  }
}

__global__ __launch_bounds__(kThreads) void euler_f32_kernel(const float4* x,
                                                             const float4* __restrict__ v,
                                                             float4* y, int64_t n_vec,
                                                             double dsigma) {
  const int64_t base = (int64_t(blockIdx.x) * kVecPerThread) * kThreads + threadIdx.x;
#pragma unroll
  for (int u = 0; u < kVecPerThread; ++u) {
    const int64_t i = base + int64_t(u) * kThreads;
    if (i >= n_vec) break;
    const float4 a = x[i], b = v[i];
    float4 r;
    r.x = float(step(a.x, b.x, dsigma));
    r.y = float(step(a.y, b.y, dsigma));
    r.z = float(step(a.z, b.z, dsigma));
    r.w = float(step(a.w, b.w, dsigma));
    y[i] = r;
  }
}

// elements past the last whole vector
__global__ void euler_tail_kernel(const void* x, const void* v, void* y, int64_t first, int64_t n,
                                  double dsigma, int is_bf16) {
  const int64_t i = first + threadIdx.x;
  if (i >= n) return;
  if (is_bf16) {
    const uint16_t a = static_cast<const uint16_t*>(x)[i], b = static_cast<const uint16_t*>(v)[i];
    const double r = step(__uint_as_float(uint32_t(a) << 16), __uint_as_float(uint32_t(b) << 16),
                          dsigma);
    static_cast<uint16_t*>(y)[i] = uint16_t(pack_bf16_rne(round_to_odd_f32(r), 0.0f) & 0xffffu);
  } else {
    static_cast<float*>(y)[i] =
        float(step(static_cast<const float*>(x)[i], static_cast<const float*>(v)[i], dsigma));
  }
}

}  // namespace

hipError_t launch_euler(const void* x, const void* v, void* y, int64_t n, double dsigma,
                        int dtype, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int per_vec = dtype == FF_DT_BF16 ? 8 : 4;
  const int64_t n_vec = n / per_vec;
  if (n_vec > 0) {
    const int64_t per_block = int64_t(kThreads) * kVecPerThread;
    const dim3 grid(unsigned((n_vec + per_block - 1) / per_block));
    if (dtype == FF_DT_BF16)
      hipLaunchKernelGGL(euler_bf16_kernel, grid, dim3(kThreads), 0, stream,
                         static_cast<const u32x4*>(x), static_cast<const u32x4*>(v),
                         static_cast<u32x4*>(y), n_vec, dsigma);
    else
      hipLaunchKernelGGL(euler_f32_kernel, grid, dim3(kThreads), 0, stream,
                         static_cast<const float4*>(x), static_cast<const float4*>(v),
                         static_cast<float4*>(y), n_vec, dsigma);
  }
  const int64_t first = n_vec * per_vec;
  if (first < n)
    hipLaunchKernelGGL(euler_tail_kernel, dim3(1), dim3(8), 0, stream, x, v, y, first, n, dsigma,
                       dtype == FF_DT_BF16 ? 1 : 0);
  return hipGetLastError();
}

}  // namespace ff
