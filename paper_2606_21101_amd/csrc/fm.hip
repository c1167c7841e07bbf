// Second-order factorization-machine term over the pooled field block, for
// gfx950 (MI355X).
//
// DeepFM's explicit interaction holds, besides GEMMs, element-wise squares,
// subtractions and reduce-sums; §IV-D fuses such neighbouring non-GEMM
// operators into one kernel whose threads fill the output element by element
// with contiguous reads.  For sample b of a [B, row_stride] block holding T
// fields of dim D:
//   out[b] = 1/2 * sum_c ((sum_t e[t][c])^2 - sum_t e[t][c]^2).
// One wave per sample.  Fast path (rows of D elements a multiple of 16 bytes,
// at most 1024): the wave is split into field slots of LPR lanes; lane k of a
// slot reads 16-byte piece k of every G-th field row, so a load instruction
// covers G consecutive field rows of the sample (contiguous in memory); the
// per-lane sums and sums of squares are then combined across slots by a fixed
// xor butterfly and reduced over the columns.  Otherwise lanes take columns.
// fp32 accumulation in a fixed order: deterministic.
#include "dpi_internal.h"

namespace dpi {
namespace {

typedef int raw16_t __attribute__((ext_vector_type(4)));
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kFmUnroll = 4;   // field rows in flight per lane

typedef const __attribute__((address_space(4))) FmArgs* FA;

template <typename T> struct Epl;
template <> struct Epl<float> { static constexpr int value = 4; };
template <> struct Epl<_Float16> { static constexpr int value = 8; };

__device__ __forceinline__ void unpack16(const raw16_t r, float* v, float) {
  const float4_t f = __builtin_bit_cast(float4_t, r);
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = f[i];
}
__device__ __forceinline__ void unpack16(const raw16_t r, float* v, _Float16) {
  const half8_t h = __builtin_bit_cast(half8_t, r);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (float)h[i];
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 1; m < kWaveSize; m <<= 1) v += __shfl_xor(v, m, kWaveSize);
  return v;
}

template <typename TIN, int LPR>
__device__ __forceinline__ float fm_fast(FA a, const char* row, int lane) {
  constexpr int EPL = Epl<TIN>::value;
  constexpr int G = kWaveSize / LPR;
  const int g = lane / LPR, k = lane % LPR;
  const int T = a->T;
  const int64_t field_bytes = (int64_t)a->dim * sizeof(TIN);
  const bool col = k * 16 < field_bytes;
  float s[EPL], q[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) s[i] = q[i] = 0.f;
  const char* p = row + (int64_t)g * field_bytes + k * 16;
  const int64_t step = (int64_t)G * field_bytes;
  int t = g;
  for (; t + (kFmUnroll - 1) * G < T; t += kFmUnroll * G) {
    raw16_t raw[kFmUnroll];
#pragma unroll
    for (int u = 0; u < kFmUnroll; ++u)
      raw[u] = col ? *reinterpret_cast<const raw16_t*>(p + u * step) : raw16_t{0, 0, 0, 0};
#pragma unroll
    for (int u = 0; u < kFmUnroll; ++u) {
      float v[EPL];
      unpack16(raw[u], v, TIN());
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        s[i] += v[i];
        q[i] += v[i] * v[i];
      }
    }
    p += kFmUnroll * step;
  }
  for (; t < T; t += G) {
    const raw16_t r = col ? *reinterpret_cast<const raw16_t*>(p) : raw16_t{0, 0, 0, 0};
    float v[EPL];
    unpack16(r, v, TIN());
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      s[i] += v[i];
      q[i] += v[i] * v[i];
    }
    p += step;
  }
  // sum over the slots (fields t = g mod G), then over this lane's columns
#pragma unroll
  for (int m = LPR; m < kWaveSize; m <<= 1) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      s[i] += __shfl_xor(s[i], m, kWaveSize);
      q[i] += __shfl_xor(q[i], m, kWaveSize);
    }
  }
  float y = 0.f;
  if (g == 0) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) y += s[i] * s[i] - q[i];
  }
  return wave_sum(y);
}

template <typename TIN>
__device__ __forceinline__ float fm_general(FA a, const TIN* row, int lane) {
  float y = 0.f;
  for (int c = lane; c < a->dim; c += kWaveSize) {
    float s = 0.f, q = 0.f;
    for (int t = 0; t < a->T; ++t) {
      const float v = (float)row[(int64_t)t * a->dim + c];
      s += v;
      q += v * v;
    }
    y += s * s - q;
  }
  return wave_sum(y);
}

template <typename TIN>
__global__ __launch_bounds__(kBlockThreads) void fm_kernel(const FmArgs args) {
  (void)args;
  const FA a = (FA)__builtin_amdgcn_kernarg_segment_ptr();
  const int lane = threadIdx.x & (kWaveSize - 1);
  const int64_t b = (int64_t)blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
  if (b >= a->B) return;
  const TIN* row = reinterpret_cast<const TIN*>(a->emb) + b * a->row_stride;
  float y;
  switch (a->lpr_log) {
#define DPI_FM_CASE(L, LPR) \
  case L:                   \
    y = fm_fast<TIN, LPR>(a, reinterpret_cast<const char*>(row), lane); \
    break;
    DPI_FM_CASE(0, 1) DPI_FM_CASE(1, 2) DPI_FM_CASE(2, 4) DPI_FM_CASE(3, 8) DPI_FM_CASE(4, 16)
    DPI_FM_CASE(5, 32) DPI_FM_CASE(6, 64)
#undef DPI_FM_CASE
    default:
      y = fm_general<TIN>(a, row, lane);
  }
  if (lane == 0) a->out[b] = 0.5f * y;
}

}  // namespace

hipError_t launch_fm(const FmArgs& a, hipStream_t s) {
  const int64_t blocks = (a.B + kWavesPerBlock - 1) / kWavesPerBlock;
  if (blocks <= 0) return hipSuccess;
  if (a.f16)
    hipLaunchKernelGGL(fm_kernel<_Float16>, dim3((unsigned)blocks), dim3(kBlockThreads), 0, s, a);
  else
    hipLaunchKernelGGL(fm_kernel<float>, dim3((unsigned)blocks), dim3(kBlockThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace dpi
