// Fused non-GEMM operators of the interaction modules, for gfx950.
//
// §IV-D fuses every run of neighbouring non-GEMM operators of a model's
// interaction modules into one kernel whose threads fill the output element
// by element with contiguous reads and writes.  After each GEMM of a DCNv2
// cross layer the run is  x_next = x0 * (y + b) + x  (a broadcast add, a
// multiply, an add); after each GEMM of the MLP it is  h = max(0, z + c).
// Both are one pass over [B, n] with 16-byte accesses when the row length
// allows.  A one-thread marker kernel records the device wall clock, to time
// when each module's first operator starts (Algorithm 2's measurement, §V).
#include "dpi_internal.h"

namespace dpi {
namespace {

typedef float float4_t __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kBlockThreads) void cross_fuse_kernel(const float* __restrict__ x0,
                                                                   const float* __restrict__ y,
                                                                   const float* __restrict__ bias,
                                                                   const float* __restrict__ x, float* __restrict__ out,
                                                                   int64_t rows, int32_t n, int32_t vec) {
  const int64_t per_row = vec ? n / 4 : n;
  const int64_t total = rows * per_row;
  for (int64_t i = (int64_t)blockIdx.x * kBlockThreads + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kBlockThreads) {
    const int64_t r = i / per_row, c = i - r * per_row;
    if (vec) {
      const int64_t o = r * n + c * 4;
      const float4_t a = *reinterpret_cast<const float4_t*>(x0 + o);
      const float4_t v = *reinterpret_cast<const float4_t*>(y + o);
      const float4_t bb = *reinterpret_cast<const float4_t*>(bias + c * 4);
      const float4_t xx = *reinterpret_cast<const float4_t*>(x + o);
      float4_t res;
#pragma unroll
      for (int k = 0; k < 4; ++k) res[k] = a[k] * (v[k] + bb[k]) + xx[k];
      *reinterpret_cast<float4_t*>(out + o) = res;
    } else {
      const int64_t o = r * n + c;
      out[o] = x0[o] * (y[o] + bias[c]) + x[o];
    }
  }
}

__global__ __launch_bounds__(kBlockThreads) void bias_relu_kernel(float* __restrict__ z, const float* __restrict__ bias,
                                                                  int64_t rows, int32_t n, int32_t vec) {
  const int64_t per_row = vec ? n / 4 : n;
  const int64_t total = rows * per_row;
  for (int64_t i = (int64_t)blockIdx.x * kBlockThreads + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kBlockThreads) {
    const int64_t r = i / per_row, c = i - r * per_row;
    if (vec) {
      float4_t* p = reinterpret_cast<float4_t*>(z + r * n) + c;
      float4_t v = *p;
      const float4_t bb = *reinterpret_cast<const float4_t*>(bias + c * 4);
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] = fmaxf(v[k] + bb[k], 0.f);
      *p = v;
    } else {
      float* p = z + r * n + c;
      *p = fmaxf(*p + bias[c], 0.f);
    }
  }
}

__global__ void mark_kernel(uint64_t* slot) {
  if (threadIdx.x == 0) *slot = (uint64_t)wall_clock64();
}

unsigned grid_for(int64_t work) {
  const int64_t blocks = (work + kBlockThreads - 1) / kBlockThreads;
  return (unsigned)std::min<int64_t>(std::max<int64_t>(blocks, 1), 4096);
}

}  // namespace

hipError_t launch_cross_fuse(const float* x0, const float* y, const float* bias, const float* x, float* out,
                             int64_t rows, int32_t n, hipStream_t s) {
  const int32_t vec = (n % 4 == 0) ? 1 : 0;
  hipLaunchKernelGGL(cross_fuse_kernel, dim3(grid_for(rows * (vec ? n / 4 : n))), dim3(kBlockThreads), 0, s, x0, y,
                     bias, x, out, rows, n, vec);
  return hipGetLastError();
}

hipError_t launch_bias_relu(float* z, const float* bias, int64_t rows, int32_t n, hipStream_t s) {
  const int32_t vec = (n % 4 == 0) ? 1 : 0;
  hipLaunchKernelGGL(bias_relu_kernel, dim3(grid_for(rows * (vec ? n / 4 : n))), dim3(kBlockThreads), 0, s, z, bias,
                     rows, n, vec);
  return hipGetLastError();
}

hipError_t launch_mark(uint64_t* slot, hipStream_t s) {
  hipLaunchKernelGGL(mark_kernel, dim3(1), dim3(kWaveSize), 0, s, slot);
  return hipGetLastError();
}

}  // namespace dpi
