// Fused multi-table gather-pool kernel for gfx950 (MI355X).
//
// One launch covers every field and every sample of the batch (§IV-B: the k
// per-field lookups become a single operation writing the concatenated
// [B, sum dim] block).  Work is taken from the plan: wave w owns the item
// range [wave_item_begin[w], wave_item_begin[w+1]) of the field-major item
// list, i.e. a run of consecutive bags (whole bags in the interior, possibly a
// partial bag at either end).
//
// Mapping (the output-first allocation of §IV-C, restated for wave64): the
// lanes of a wavefront are split into row slots of LPR lanes; the LPR lanes of
// a slot read one table row as consecutive 16-byte pieces (coalesced along
// the row) and later write the pooled row as consecutive pieces of the
// output row.  Interior bags are dealt to slots (a slot pools a whole bag,
// fp32 accumulation, rows in bag order).  A bag split between waves is pooled
// cooperatively by all slots of each wave (rows dealt round-robin to slots, a
// fixed xor-butterfly across slots), its fp32 partial goes to the workspace,
// and the last wave to arrive (agent-scope ticket) adds the partials in wave
// order and writes the row -- deterministic, no floating-point atomics.
//
// Pooling: sum, or mean = fp32 sum / bag length (IEEE division); an empty bag
// gives zeros; one round-to-nearest-even conversion to the output dtype.
#include "dpi_internal.h"

namespace dpi {
namespace {

typedef int raw16_t __attribute__((ext_vector_type(4)));       // 16 raw bytes
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kUnroll = 4;      // rows in flight per slot

// Kernel arguments are read in place from the constant kernarg segment
// (scalar loads); a by-value copy would go to private memory because the
// table-pointer array is indexed at run time.
typedef const __attribute__((address_space(4))) LookupArgs* KA;

template <typename TIN> struct In;
template <> struct In<float> { static constexpr int EPL = 4; };       // elements per 16 B
template <> struct In<_Float16> { static constexpr int EPL = 8; };

__device__ __forceinline__ void unpack(const raw16_t r, float* v, float) {
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = __builtin_bit_cast(float, r[i]);
}
__device__ __forceinline__ void unpack(const raw16_t r, float* v, _Float16) {
  const half8_t h = __builtin_bit_cast(half8_t, r);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (float)h[i];
}

// Store EPL pooled values of one lane: one vector store when allowed.
template <typename TOUT, int EPL>
__device__ __forceinline__ void store_lane(TOUT* dst, const float* v, bool vec) {
  if (vec) {
    if constexpr (sizeof(TOUT) == 4) {
#pragma unroll
      for (int q = 0; q < EPL / 4; ++q) {
        float4_t x = {v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
        __builtin_nontemporal_store(x, reinterpret_cast<float4_t*>(dst) + q);
      }
    } else if constexpr (EPL == 8) {
      half8_t x;
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = (_Float16)v[i];
      __builtin_nontemporal_store(x, reinterpret_cast<half8_t*>(dst));
    } else {
      half4_t x;
#pragma unroll
      for (int i = 0; i < 4; ++i) x[i] = (_Float16)v[i];
      __builtin_nontemporal_store(x, reinterpret_cast<half4_t*>(dst));
    }
  } else {
#pragma unroll
    for (int i = 0; i < EPL; ++i) dst[i] = (TOUT)v[i];
  }
}

template <typename TOUT>
__device__ __forceinline__ TOUT* out_row(KA a, const TableInfo& ti, int64_t b) {
  return reinterpret_cast<TOUT*>(a->out) + b * a->total_d + ti.col_base;
}

__device__ __forceinline__ bool is_mean(KA a, int64_t t) {
  return (a->mean_bits[t >> 5] >> (t & 31)) & 1u;
}

// Positions [s, e) of bag b inside its field's id list, clamped to the list.
__device__ __forceinline__ void bag_span(KA a, const TableInfo& ti, int64_t t, int64_t b,
                                         int64_t& s, int64_t& e) {
  if (a->offsets) {
    const int32_t* o = a->offsets + t * (a->B + 1);
    s = o[b];
    e = o[b + 1];
    s = s < 0 ? 0 : (s > ti.nnz ? ti.nnz : s);
    e = e < s ? s : (e > ti.nnz ? ti.nnz : e);
  } else {
    s = b;
    e = b + 1;
  }
}

// ---------------------------------------------------------------------------
// Fast path: row bytes a multiple of 16 and at most 1024; LPR lanes per row.
// ---------------------------------------------------------------------------

// Whole bags [b_lo, b_hi) of field t, one bag per slot at a time.
template <typename TIN, typename TOUT, int LPR>
__device__ __attribute__((noinline)) int pool_bags_per_slot(KA a, int64_t t, int64_t b_lo, int64_t b_hi,
                                                            int lane) {
  constexpr int EPL = In<TIN>::EPL;
  const TableInfo ti = a->tinfo[t];
  int bad = 0;
  constexpr int G = kWaveSize / LPR;
  const int g = lane / LPR, k = lane % LPR;
  const TIN* __restrict__ table = reinterpret_cast<const TIN*>(a->tables[t]);
  const int32_t* __restrict__ ids = a->ids + ti.id_base;
  const int64_t dim = ti.dim, nrows = ti.num_rows;
  const bool col = k * EPL < dim;
  const bool mean = is_mean(a, t);
  const bool vec = (ti.flags & kTiOutVec) != 0;
  for (int64_t b = b_lo + g; b < b_hi; b += G) {
    int64_t s, e;
    bag_span(a, ti, t, b, s, e);
    float acc[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] = 0.f;
    for (int64_t p = s; p < e; p += kUnroll) {
      int32_t id[kUnroll];
      raw16_t raw[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) id[u] = (p + u < e) ? ids[p + u] : -1;
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        raw[u] = raw16_t{0, 0, 0, 0};
        const bool in_bag = p + u < e;
        const bool ok = in_bag && id[u] >= 0 && id[u] < nrows;
        bad |= (in_bag && !ok);
        if (ok && col)
          raw[u] = *reinterpret_cast<const raw16_t*>(table + (int64_t)id[u] * dim + k * EPL);
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        float v[EPL];
        unpack(raw[u], v, TIN());
#pragma unroll
        for (int i = 0; i < EPL; ++i) acc[i] += v[i];
      }
    }
    if (mean && e > s) {
      const float L = (float)(e - s);
#pragma unroll
      for (int i = 0; i < EPL; ++i) acc[i] = acc[i] / L;
    }
    if (col) store_lane<TOUT, EPL>(out_row<TOUT>(a, ti, b) + k * EPL, acc, vec);
  }
  return bad;
}

// Rows [r0, r1) (positions in the field's id list) pooled by all slots of the
// wave; on return every slot holds the total for its lane's columns.
template <typename TIN, int LPR>
__device__ __forceinline__ void pool_rows_coop(KA a, const TableInfo& ti, int64_t t, int64_t r0,
                                               int64_t r1, int lane, float* acc, int& bad) {
  constexpr int EPL = In<TIN>::EPL;
  constexpr int G = kWaveSize / LPR;
  const int g = lane / LPR, k = lane % LPR;
  const TIN* __restrict__ table = reinterpret_cast<const TIN*>(a->tables[t]);
  const int32_t* __restrict__ ids = a->ids + ti.id_base;
  const int64_t dim = ti.dim, nrows = ti.num_rows;
  const bool col = k * EPL < dim;
#pragma unroll
  for (int i = 0; i < EPL; ++i) acc[i] = 0.f;
  for (int64_t r = r0 + g; r < r1; r += (int64_t)G * kUnroll) {
    int32_t id[kUnroll];
    raw16_t raw[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) id[u] = (r + u * G < r1) ? ids[r + u * G] : -1;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      raw[u] = raw16_t{0, 0, 0, 0};
      const bool in_bag = r + u * G < r1;
      const bool ok = in_bag && id[u] >= 0 && id[u] < nrows;
      bad |= (in_bag && !ok);
      if (ok && col) raw[u] = *reinterpret_cast<const raw16_t*>(table + (int64_t)id[u] * dim + k * EPL);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      float v[EPL];
      unpack(raw[u], v, TIN());
#pragma unroll
      for (int i = 0; i < EPL; ++i) acc[i] += v[i];
    }
  }
#pragma unroll
  for (int m = LPR; m < kWaveSize; m <<= 1) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] += __shfl_xor(acc[i], m, kWaveSize);
  }
}

// Whole bags, all slots on one bag at a time (few long bags).
template <typename TIN, typename TOUT, int LPR>
__device__ __attribute__((noinline)) int pool_bags_coop(KA a, int64_t t, int64_t b_lo, int64_t b_hi, int lane) {
  constexpr int EPL = In<TIN>::EPL;
  const TableInfo ti = a->tinfo[t];
  int bad = 0;
  const int g = lane / LPR, k = lane % LPR;
  const bool col = k * EPL < ti.dim;
  const bool mean = is_mean(a, t);
  const bool vec = (ti.flags & kTiOutVec) != 0;
  for (int64_t b = b_lo; b < b_hi; ++b) {
    int64_t s, e;
    bag_span(a, ti, t, b, s, e);
    float acc[EPL];
    pool_rows_coop<TIN, LPR>(a, ti, t, s, e, lane, acc, bad);
    if (mean && e > s) {
      const float L = (float)(e - s);
#pragma unroll
      for (int i = 0; i < EPL; ++i) acc[i] = acc[i] / L;
    }
    if (g == 0 && col) store_lane<TOUT, EPL>(out_row<TOUT>(a, ti, b) + k * EPL, acc, vec);
  }
  return bad;
}

// Rows [row_lo, row_hi) of bag b (bag-relative), fp32 partial to `slot`.
template <typename TIN, int LPR>
__device__ __attribute__((noinline)) int partial_fast(KA a, int64_t t, int64_t b, int64_t row_lo, int64_t row_hi,
                                                      int64_t slot, int lane) {
  constexpr int EPL = In<TIN>::EPL;
  const TableInfo ti = a->tinfo[t];
  int bad = 0;
  const int g = lane / LPR, k = lane % LPR;
  int64_t s, e;
  bag_span(a, ti, t, b, s, e);
  const int64_t r0 = min(e, s + row_lo), r1 = min(e, s + row_hi);
  float acc[EPL];
  pool_rows_coop<TIN, LPR>(a, ti, t, r0, r1, lane, acc, bad);
  if (g == 0 && k * EPL < ti.dim) {
    float* dst = a->partial + slot * a->dmax + k * EPL;
#pragma unroll
    for (int i = 0; i < EPL; ++i) dst[i] = acc[i];
  }
  return bad;
}

// ---------------------------------------------------------------------------
// General path: any row of a multiple of 4 bytes.  Lanes cover 4-byte words.
// ---------------------------------------------------------------------------
template <typename TIN, typename TOUT>
__device__ __attribute__((noinline)) int pool_general(KA a, int64_t t, int64_t b, int64_t row_lo, int64_t row_hi,
                                                      bool complete, int64_t slot, int lane) {
  constexpr int EPW = 4 / sizeof(TIN);   // elements per 4-byte word
  const TableInfo ti = a->tinfo[t];
  int bad = 0;
  const int64_t words = ti.row_bytes / 4;
  int lpr = 1;
  while (lpr < words && lpr < kWaveSize) lpr <<= 1;
  const int G = kWaveSize / lpr;
  const int g = lane / lpr, k = lane % lpr;
  const TIN* __restrict__ table = reinterpret_cast<const TIN*>(a->tables[t]);
  const int32_t* __restrict__ ids = a->ids + ti.id_base;
  const int64_t dim = ti.dim, nrows = ti.num_rows;
  int64_t s, e;
  bag_span(a, ti, t, b, s, e);
  const int64_t r0 = min(e, s + row_lo), r1 = min(e, s + row_hi);
  const bool mean = is_mean(a, t);
  for (int64_t pass = 0; pass * kWaveSize < words; ++pass) {
    const int64_t w = pass * kWaveSize + k;
    float acc[EPW];
#pragma unroll
    for (int i = 0; i < EPW; ++i) acc[i] = 0.f;
    for (int64_t r = r0 + g; r < r1; r += G) {
      const int32_t id = ids[r];
      if (id < 0 || id >= nrows) {
        bad = 1;
        continue;
      }
      if (w < words) {
        const TIN* src = table + (int64_t)id * dim + w * EPW;
#pragma unroll
        for (int i = 0; i < EPW; ++i) acc[i] += (float)src[i];
      }
    }
    for (int m = lpr; m < kWaveSize; m <<= 1) {
#pragma unroll
      for (int i = 0; i < EPW; ++i) acc[i] += __shfl_xor(acc[i], m, kWaveSize);
    }
    if (g == 0 && w < words) {
      if (complete) {
        if (mean && r1 > r0) {
#pragma unroll
          for (int i = 0; i < EPW; ++i) acc[i] = acc[i] / (float)(r1 - r0);
        }
        TOUT* dst = out_row<TOUT>(a, ti, b) + w * EPW;
#pragma unroll
        for (int i = 0; i < EPW; ++i) dst[i] = (TOUT)acc[i];
      } else {
        float* dst = a->partial + slot * a->dmax + w * EPW;
#pragma unroll
        for (int i = 0; i < EPW; ++i) dst[i] = acc[i];
      }
    }
  }
  return bad;
}

// ---------------------------------------------------------------------------
// Split bags: publish this wave's partial; the last arrival combines.
// ---------------------------------------------------------------------------
template <typename TOUT>
__device__ __attribute__((noinline)) void finish_piece(KA a, int64_t w_first, int64_t bag, int lane) {
  if (w_first < 0 || w_first >= min(a->hdr[kHdrW], a->grid_waves)) return;   // malformed plan
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  int old = 0;
  if (lane == 0)
    old = __hip_atomic_fetch_add(a->tickets + w_first, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  old = __shfl(old, 0, kWaveSize);
  const int pieces = a->split_pieces[w_first];
  if (old != pieces - 1) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  const int64_t t = bag / a->B, b = bag - t * a->B;
  const TableInfo ti = a->tinfo[t];
  int64_t s, e;
  bag_span(a, ti, t, b, s, e);
  const bool mean = is_mean(a, t);
  const int64_t w_last = a->split_last[w_first];
  TOUT* dst = out_row<TOUT>(a, ti, b);
  for (int64_t c = lane; c < ti.dim; c += kWaveSize) {
    float sum = a->partial[(2 * w_first + 1) * a->dmax + c];
    for (int64_t v = w_first + 1; v <= w_last; ++v)
      if (a->wib[v] < a->wib[v + 1]) sum += a->partial[(2 * v) * a->dmax + c];
    if (mean && e > s) sum = sum / (float)(e - s);
    dst[c] = (TOUT)sum;
  }
  if (lane == 0) __hip_atomic_store(a->tickets + w_first, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// Dispatch on the field's row class (wave-uniform).
// ---------------------------------------------------------------------------
#define DPI_FOR_LPR(MACRO) \
  MACRO(0, 1) MACRO(1, 2) MACRO(2, 4) MACRO(3, 8) MACRO(4, 16) MACRO(5, 32) MACRO(6, 64)

template <typename TIN, typename TOUT>
__device__ int pool_segment_typed(KA a, int flags, int64_t t, int64_t b_lo, int64_t b_hi, int lane) {
  const int lg = (flags >> kTiLprShift) & 7;
  const int64_t slots = kWaveSize >> lg;
  const bool coop = (b_hi - b_lo) * 2 <= slots;
  switch (lg) {
#define DPI_CASE(L, LPR)                                                      \
  case L:                                                                     \
    return coop ? pool_bags_coop<TIN, TOUT, LPR>(a, t, b_lo, b_hi, lane)      \
                : pool_bags_per_slot<TIN, TOUT, LPR>(a, t, b_lo, b_hi, lane);
    DPI_FOR_LPR(DPI_CASE)
#undef DPI_CASE
    default:
      return 0;
  }
}

template <typename TOUT>
__device__ int pool_bag_range(KA a, int64_t lA, int64_t lB, int lane) {
  int bad = 0;
  while (lA < lB) {
    const int64_t t = __builtin_amdgcn_readfirstlane((int)(lA / a->B));
    const int64_t seg_end = min(lB, (t + 1) * a->B);
    const int flags = a->tinfo[t].flags;
    const int64_t b_lo = lA - t * a->B, b_hi = seg_end - t * a->B;
    if (flags & kTiFast) {
      if (flags & kTiF16)
        bad |= pool_segment_typed<_Float16, TOUT>(a, flags, t, b_lo, b_hi, lane);
      else
        bad |= pool_segment_typed<float, TOUT>(a, flags, t, b_lo, b_hi, lane);
    } else {
      for (int64_t b = b_lo; b < b_hi; ++b) {
        if (flags & kTiF16)
          bad |= pool_general<_Float16, TOUT>(a, t, b, 0, INT64_MAX / 2, true, 0, lane);
        else
          bad |= pool_general<float, TOUT>(a, t, b, 0, INT64_MAX / 2, true, 0, lane);
      }
    }
    lA = seg_end;
  }
  return bad;
}

template <typename TOUT>
__device__ int pool_partial(KA a, int64_t bag, int64_t row_lo, int64_t row_hi, int64_t slot, int64_t w_first,
                            int lane) {
  const int64_t t = __builtin_amdgcn_readfirstlane((int)(bag / a->B));
  const int64_t b = bag - t * a->B;
  const int flags = a->tinfo[t].flags;
  int bad = 0;
  if (flags & kTiFast) {
    const int lg = (flags >> kTiLprShift) & 7;
    const bool f16 = (flags & kTiF16) != 0;
    switch (lg) {
#define DPI_CASE(L, LPR)                                                              \
  case L:                                                                             \
    bad = f16 ? partial_fast<_Float16, LPR>(a, t, b, row_lo, row_hi, slot, lane)      \
              : partial_fast<float, LPR>(a, t, b, row_lo, row_hi, slot, lane);        \
    break;
      DPI_FOR_LPR(DPI_CASE)
#undef DPI_CASE
      default:
        break;
    }
  } else if (flags & kTiF16) {
    bad = pool_general<_Float16, TOUT>(a, t, b, row_lo, row_hi, false, slot, lane);
  } else {
    bad = pool_general<float, TOUT>(a, t, b, row_lo, row_hi, false, slot, lane);
  }
  finish_piece<TOUT>(a, w_first, bag, lane);
  return bad;
}

__device__ __forceinline__ int64_t xcd_affine_block(int64_t g, int64_t n) {
  // workgroups are dispatched round-robin over 8 XCDs; give XCD x the
  // contiguous logical range of its round-robin share
  const int64_t x = g & 7, i = g >> 3, q = n >> 3, r = n & 7;
  return x < r ? x * (q + 1) + i : r * (q + 1) + (x - r) * q + i;
}

template <typename TOUT>
__global__ __launch_bounds__(kBlockThreads) void lookup_kernel(const LookupArgs args) {
  (void)args;
  const KA a = (KA)__builtin_amdgcn_kernarg_segment_ptr();
  const int lane = threadIdx.x & (kWaveSize - 1);
  int64_t blk = blockIdx.x;
  if (a->xcd_affine) blk = xcd_affine_block(blk, gridDim.x);
  const int64_t w = blk * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
  const int64_t W = min(a->hdr[kHdrW], a->grid_waves);
  if (w >= W) return;
  if (*a->status & kStatusBadOffsets) return;   // the plan rejected the offsets
  const int64_t i0 = a->wib[w], i1 = a->wib[w + 1];
  if (i0 >= i1) return;
  const int64_t TB = a->B * a->T;
  const int64_t C = a->C;
  const int64_t la = a->wave_bag[w], lz = a->wave_bag[w + 1];
  const int64_t lb = (lz < TB && a->bib[lz] < i1) ? lz : lz - 1;
  const int64_t la_base = a->bib[la];
  const int64_t lb_base = a->bib[lb];
  const bool head = la_base < i0;
  const bool tail = a->bib[lb + 1] > i1;
  int bad = 0;
  if (la == lb && (head || tail)) {
    const int64_t slot = head ? 2 * w : 2 * w + 1;
    const int64_t w_first = head ? (int64_t)a->head_first[w] : w;
    bad |= pool_partial<TOUT>(a, la, (i0 - la_base) * C, (i1 - la_base) * C, slot, w_first, lane);
  } else {
    int64_t lA = la, lB = lb + 1;
    if (head) {
      bad |= pool_partial<TOUT>(a, la, (i0 - la_base) * C, INT64_MAX / 2, 2 * w, a->head_first[w], lane);
      lA = la + 1;
    }
    if (tail) lB = lb;
    bad |= pool_bag_range<TOUT>(a, lA, lB, lane);
    if (tail) bad |= pool_partial<TOUT>(a, lb, 0, (i1 - lb_base) * C, 2 * w + 1, w, lane);
  }
  if (__any(bad) && lane == 0)
    __hip_atomic_fetch_or(a->status, kStatusBadId, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace

hipError_t launch_lookup(const LookupArgs& a, hipStream_t s) {
  const int64_t blocks = (a.grid_waves + kWavesPerBlock - 1) / kWavesPerBlock;
  if (blocks <= 0) return hipSuccess;
  if (a.out_f16)
    hipLaunchKernelGGL(lookup_kernel<_Float16>, dim3((unsigned)blocks), dim3(kBlockThreads), 0, s, a);
  else
    hipLaunchKernelGGL(lookup_kernel<float>, dim3((unsigned)blocks), dim3(kBlockThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace dpi
