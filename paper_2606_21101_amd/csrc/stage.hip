// Input consolidation (gfx950): one-hot and multi-hot batches.
//
// A CTR data loader hands over a batch's categorical features as one
// sample-major matrix x[B][row_stride] (column t = field t's id, often stored
// as float).  The paper's breakdown (§V) shows that moving every field to the
// GPU separately and converting each one to an integer type separately costs
// launches and copies; here the whole matrix travels in one copy and one
// kernel converts and transposes it into the field-major int32 ids of the
// lookup (the transpose of Algorithm 1's sample-major id matrix).
// 64 x 64 tiles through LDS: reads along a sample's fields and writes along a
// field's samples are both contiguous.
#include "gather.h"   // to_id: the conversion the one-launch lookup applies to a staged CSR too

namespace dpi {
namespace {

constexpr int kTile = 64;

template <typename TX>
__global__ __launch_bounds__(kTile * 4) void stage_onehot_kernel(const StageArgs args) {
  __shared__ int32_t tile[kTile][kTile + 1];
  const TX* __restrict__ x = reinterpret_cast<const TX*>(args.x);
  const int64_t b0 = (int64_t)blockIdx.x * kTile;
  const int64_t t0 = (int64_t)blockIdx.y * kTile;
  const int tx = threadIdx.x % kTile, ty = threadIdx.x / kTile;   // 64 x 4 threads
  // read: rows b0 + r, columns t0 + tx (contiguous along the fields)
  for (int r = ty; r < kTile; r += 4) {
    const int64_t b = b0 + r, t = t0 + tx;
    if (b < args.B && t < args.T) tile[r][tx] = to_id(x[b * args.row_stride + t]);
  }
  __syncthreads();
  // write: fields t0 + r, samples b0 + tx (contiguous along the samples)
  for (int r = ty; r < kTile; r += 4) {
    const int64_t t = t0 + r, b = b0 + tx;
    if (b < args.B && t < args.T) args.ids[t * args.B + b] = tile[tx][r];
  }
}

// Multi-hot batches: the device copy holds every field's offsets ([T][B+1])
// followed by the fields' ids; both are converted in one grid-stride pass.
template <typename TX>
__global__ __launch_bounds__(kBlockThreads) void stage_csr_kernel(const void* __restrict__ src, int64_t n_off,
                                                                  int64_t n_ids, int32_t* __restrict__ offsets,
                                                                  int32_t* __restrict__ ids) {
  const TX* __restrict__ x = reinterpret_cast<const TX*>(src);
  const int64_t n = n_off + n_ids;
  for (int64_t i = (int64_t)blockIdx.x * kBlockThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlockThreads) {
    const int32_t v = to_id(x[i]);
    if (i < n_off)
      offsets[i] = v;
    else
      ids[i - n_off] = v;
  }
}

}  // namespace

hipError_t launch_stage_csr(const void* src, int32_t x_dtype, int64_t n_off, int64_t n_ids, int32_t* offsets,
                            int32_t* ids, hipStream_t s) {
  const int64_t n = n_off + n_ids;
  if (n <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)std::min<int64_t>((n + kBlockThreads - 1) / kBlockThreads, 8192);
  switch (x_dtype) {
    case DPI_X_F32:
      hipLaunchKernelGGL(stage_csr_kernel<float>, dim3(blocks), dim3(kBlockThreads), 0, s, src, n_off, n_ids, offsets, ids);
      break;
    case DPI_X_I64:
      hipLaunchKernelGGL(stage_csr_kernel<int64_t>, dim3(blocks), dim3(kBlockThreads), 0, s, src, n_off, n_ids, offsets, ids);
      break;
    case DPI_X_I32:
      hipLaunchKernelGGL(stage_csr_kernel<int32_t>, dim3(blocks), dim3(kBlockThreads), 0, s, src, n_off, n_ids, offsets, ids);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_stage(const StageArgs& a, hipStream_t s) {
  if (a.B <= 0) return hipSuccess;
  const dim3 grid((unsigned)((a.B + kTile - 1) / kTile), (unsigned)((a.T + kTile - 1) / kTile));
  const dim3 block(kTile * 4);
  switch (a.x_dtype) {
    case DPI_X_F32: hipLaunchKernelGGL(stage_onehot_kernel<float>, grid, block, 0, s, a); break;
    case DPI_X_I64: hipLaunchKernelGGL(stage_onehot_kernel<int64_t>, grid, block, 0, s, a); break;
    case DPI_X_I32: hipLaunchKernelGGL(stage_onehot_kernel<int32_t>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace dpi
