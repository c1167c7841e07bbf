// Device helpers shared by the plan-driven lookup kernels (lookup.hip) and the
// one-launch kernels of small batches (small.hip): the 16-byte row readers,
// fp32 accumulation, mean division, output stores, whole-wave pooling of a
// row range, bag-by-bag pooling and the one-hot row copy.  Functions that read
// kernel arguments take them as a pointer into the constant kernarg segment
// of either kernel family (template parameter KX); both argument structs name
// the fields these functions read (tables, ids, out, B, total_d, mean_bits)
// alike.
#pragma once

#include "dpi_internal.h"

namespace dpi {
namespace {

typedef int raw16_t __attribute__((ext_vector_type(4)));       // 16 raw bytes
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kUnroll = 8;        // rows in flight per slot
static_assert(kUnroll == kDirectGroupRows, "the host sizes direct bag groups by this");
constexpr uint32_t kBufferWord3 = 0x00020000;   // raw buffer descriptor, gfx9 family

// Values known to be equal across the wave; out-of-line functions receive
// them in vector registers, so they are re-read from the first lane to let
// the compiler keep them (and what derives from them) in scalar registers.
__device__ __forceinline__ int64_t uni(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}


__device__ __forceinline__ int32_t uni(int32_t x) { return __builtin_amdgcn_readfirstlane(x); }

// ids are valid in [0, min(num_rows, 2^31)): one unsigned 32-bit compare
__device__ __forceinline__ uint32_t id_limit(const TableInfo& ti) {
  return (uint32_t)(ti.num_rows < ((int64_t)1 << 31) ? ti.num_rows : ((int64_t)1 << 31));
}

template <typename TIN> struct In;
template <> struct In<float> { static constexpr int EPL = 4; };       // elements per 16 B
template <> struct In<_Float16> { static constexpr int EPL = 8; };

__device__ __forceinline__ void unpack(const raw16_t r, float* v, float) {
  // bit-cast the whole vector: a bit-cast of one vector element reads element 0
  const float4_t f = __builtin_bit_cast(float4_t, r);
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = f[i];
}
__device__ __forceinline__ void unpack(const raw16_t r, float* v, _Float16) {
  const half8_t h = __builtin_bit_cast(half8_t, r);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (float)h[i];
}

// acc[i] += element i of 16 raw bytes.  binary16 elements take one
// mixed-precision FMA each (the half, widened exactly, times 1.0 plus the fp32
// sum, rounded once: the same result as widening then adding, in one
// instruction instead of two); the compiler emits the widen-then-add pair
// for the plain expression.
template <typename TIN, int EPL>
__device__ __forceinline__ void accumulate(float* acc, const raw16_t r) {
  if constexpr (sizeof(TIN) == 2) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      asm("v_fma_mix_f32 %0, %1, 1.0, %0 op_sel_hi:[1,0,0]" : "+v"(acc[2 * q]) : "v"(r[q]));
      asm("v_fma_mix_f32 %0, %1, 1.0, %0 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "+v"(acc[2 * q + 1]) : "v"(r[q]));
    }
  } else {
    float v[EPL];
    unpack(r, v, TIN());
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] += v[i];
  }
}

// acc[i] / fl for the N sums of one lane, each rounded as IEEE binary32
// division.  One correctly rounded reciprocal y = 1/fl serves the whole bag;
// per element q = a*y, the remainder a - q*fl (exact, one fma) and the
// corrected quotient q + r*y (one fma).  With y correctly rounded and q within
// one ulp of a/fl, that is the correctly rounded a/fl (Markstein's correction
// theorem) while no step leaves the normal range, which holds for
// 2^-64 <= |a| <= FLT_MAX and fl < 2^31; a lane with an element outside that
// range (zero, tiny, infinite, NaN) divides instead.  The three
// instructions per element replace an eleven-instruction division.
template <int N>
__device__ __forceinline__ void mean_divide(float* acc, float fl) {
  // magnitudes as unsigned integers order like the floats, NaN above infinity
  uint32_t lo = 0xffffffffu, hi = 0;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const uint32_t m = __builtin_bit_cast(uint32_t, acc[i]) & 0x7fffffffu;
    lo = min(lo, m);
    hi = max(hi, m);
  }
  if (lo >= (63u << 23) && hi <= 0x7f7fffffu) {
    const float y = 1.0f / fl;
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const float q = acc[i] * y;
      acc[i] = __builtin_fmaf(__builtin_fmaf(-q, fl, acc[i]), y, q);
    }
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) acc[i] = acc[i] / fl;
  }
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

template <typename TOUT, typename KX>
__device__ __forceinline__ TOUT* out_row(KX a, const TableInfo& ti, int64_t b) {
  return reinterpret_cast<TOUT*>(a->out) + b * a->total_d + ti.col_base;
}

template <typename KX>
__device__ __forceinline__ bool is_mean(KX a, int64_t t) {
  return (a->mean_bits[t >> 5] >> (t & 31)) & 1u;
}

// 16-byte piece k of row `id` of a table.
template <bool BUF> struct RowReader;
template <> struct RowReader<true> {
  // raw buffer: the descriptor's record count and the per-lane offset are
  // unsigned 32-bit byte values, so tables up to 4 GiB - 1 bytes qualify.
  // (An indexed descriptor with the row bytes as stride, letting the load
  // form id * row_bytes itself, measured 5 % slower on the multi-hot batch.)
  __amdgpu_buffer_rsrc_t rsrc;
  uint32_t row_bytes, koff;
  __device__ RowReader(const void* table, const TableInfo& ti, int k)
      : rsrc(__builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(table), (short)0,
                                               (int)(uint32_t)(ti.num_rows * (int64_t)ti.row_bytes), kBufferWord3)),
        row_bytes((uint32_t)ti.row_bytes), koff((uint32_t)k * 16u) {}
  __device__ __forceinline__ raw16_t load(int32_t id) const {
    return __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)((uint32_t)id * row_bytes + koff), 0, 0);
  }
  // Row `id` when `take`, else zeros without a branch: the load goes to an
  // offset no table of this kind reaches (its byte size is a multiple of 16
  // below 2^32, so at most 2^32 - 16), and a raw buffer load outside the
  // descriptor's range returns zeros and touches no memory.
  __device__ __forceinline__ raw16_t load_if(int32_t id, bool take) const {
    const uint32_t o = take ? (uint32_t)id * row_bytes + koff : 0xfffffff0u;
    return __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)o, 0, 0);
  }
  // The row starting at byte `row_off` (a masked row: masked_row_offset).
  __device__ __forceinline__ raw16_t load_at(uint32_t row_off) const {
    return __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)(row_off + koff), 0, 0);
  }
};

// Start of a row no buffer-read table of rows of RB bytes (a power of two)
// reaches: such a table's byte size is a multiple of RB below 2^32, so at most
// 2^32 - RB, and every piece of the "row" from here lies past it.
template <int RB>
constexpr uint32_t masked_row_offset() { return (uint32_t)(0x100000000ull - RB); }

template <> struct RowReader<false> {
  const char* base;
  uint32_t row_bytes, koff;
  __device__ RowReader(const void* table, const TableInfo& ti, int k)
      : base(reinterpret_cast<const char*>(table)), row_bytes((uint32_t)ti.row_bytes), koff((uint32_t)k * 16u) {}
  __device__ __forceinline__ raw16_t load(int32_t id) const {
    return *reinterpret_cast<const raw16_t*>(base + (uint64_t)(uint32_t)id * row_bytes + koff);
  }
  __device__ __forceinline__ raw16_t load_if(int32_t id, bool take) const {
    raw16_t v = {0, 0, 0, 0};
    if (take) v = load(id);
    return v;
  }
};

// buffer descriptors hold an unsigned 32-bit byte range
__device__ __forceinline__ bool use_buffer(const TableInfo& ti) {
  return ti.num_rows * (int64_t)ti.row_bytes <= (int64_t)0xffffffffLL;
}

// Workgroups are dispatched round-robin over 8 XCDs.  group = 1: XCD x takes
// the contiguous logical range of its round-robin share.  group = 2: XCDs 2p
// and 2p + 1 share one contiguous range, alternating blocks (a bijection on
// [0, n) either way: the group's blocks in dispatch order, after the blocks
// of the XCDs before it).
__device__ __forceinline__ int64_t xcd_affine_block(int64_t g, int64_t n, int32_t group) {
  const int64_t x = g & 7, i = g >> 3, q = n >> 3, r = n & 7;
  const int64_t lo = group == 2 ? (x & ~(int64_t)1) : x;   // first XCD of x's group
  const int64_t m = x - lo;
  return lo * q + min(lo, r) + i * group + m;
}

#define DPI_FOR_LPR(MACRO) \
  MACRO(0, 1) MACRO(1, 2) MACRO(2, 4) MACRO(3, 8) MACRO(4, 16) MACRO(5, 32) MACRO(6, 64)

// ---------------------------------------------------------------------------
// Where a kernel reads the batch's offsets and ids.  NativeIds: the int32
// arrays dpi_plan and dpi_lookup take.  StagedIds<TX>: a staged copy of a
// data loader's packed CSR (every field's offsets, then the fields' ids, as
// float, int64 or int32), converted as it is read exactly as dpi_stage_csr
// converts it, and written out as the int32 arrays it would have produced
// (put_offset / put_id, called by the kernel once per element after its
// pooling: on gfx9 loads and stores share one counter, and a store still in
// flight makes every later wait for a load a wait for everything).
// ---------------------------------------------------------------------------
// a value that is not an integer in [0, 2^31) becomes -1
__device__ __forceinline__ int32_t to_id(float v) {
  return (v >= 0.f && v < 2147483648.f && v == truncf(v)) ? (int32_t)v : -1;
}
__device__ __forceinline__ int32_t to_id(int64_t v) { return (v >= 0 && v < ((int64_t)1 << 31)) ? (int32_t)v : -1; }
__device__ __forceinline__ int32_t to_id(int32_t v) { return v >= 0 ? v : -1; }

struct NativeIds {
  const int32_t* __restrict__ off;
  const int32_t* __restrict__ ids;
  __device__ __forceinline__ int32_t offset(int64_t i) const { return off[i]; }
  __device__ __forceinline__ int32_t id(int64_t i) const { return ids[i]; }
  __device__ __forceinline__ void put_offset(int64_t, int32_t) const {}
  __device__ __forceinline__ void put_id(int64_t, int32_t) const {}
  static constexpr bool kWrites = false;
};

template <typename TX>
struct StagedIds {
  const TX* __restrict__ off;     // [T][B+1]
  const TX* __restrict__ ids;     // [total_ids], right after the offsets
  int32_t* __restrict__ off_out;
  int32_t* __restrict__ ids_out;
  __device__ __forceinline__ int32_t offset(int64_t i) const { return to_id(off[i]); }
  __device__ __forceinline__ int32_t id(int64_t i) const { return to_id(ids[i]); }
  __device__ __forceinline__ void put_offset(int64_t i, int32_t v) const { off_out[i] = v; }
  __device__ __forceinline__ void put_id(int64_t i, int32_t v) const { ids_out[i] = v; }
  static constexpr bool kWrites = true;
};

// ---------------------------------------------------------------------------
// Fast path: row bytes a multiple of 16 and at most 1024; LPR lanes per row.
// ---------------------------------------------------------------------------

// Rows [r0, r1) of field t pooled by all slots of the wave, its ids read
// from `src`; on return every slot holds the total for its lane's columns.
template <typename TIN, int LPR, bool BUF, typename KX, typename S>
__device__ __forceinline__ void pool_rows_src(KX a, const S& src, const TableInfo& ti, int64_t t, int64_t r0,
                                              int64_t r1, int lane, float* acc, int& bad) {
  constexpr int EPL = In<TIN>::EPL;
  constexpr int G = kWaveSize / LPR;
  const int g = lane / LPR, k = lane % LPR;
  const RowReader<BUF> rows(a->tables[t], ti, k);
  const int64_t ib = ti.id_base;
  const uint32_t nrows = id_limit(ti);
  const bool col = k * EPL < ti.dim;
#pragma unroll
  for (int i = 0; i < EPL; ++i) acc[i] = 0.f;
  int32_t idn[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int64_t q = r0 + g + u * G;
    idn[u] = q < r1 ? src.id(ib + q) : -1;
  }
  for (int64_t r = r0 + g; r < r1; r += (int64_t)G * kUnroll) {
    raw16_t raw[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      raw[u] = raw16_t{0, 0, 0, 0};
      const bool in_bag = r + u * G < r1;
      const bool ok = in_bag && (uint32_t)idn[u] < nrows;
      bad |= (in_bag && !ok);
      if (ok && col) raw[u] = rows.load(idn[u]);
    }
    const int64_t rn = r + (int64_t)G * kUnroll;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t q = rn + u * G;
      idn[u] = q < r1 ? src.id(ib + q) : -1;
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) accumulate<TIN, EPL>(acc, raw[u]);
  }
#pragma unroll
  for (int m = LPR; m < kWaveSize; m <<= 1) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] += __shfl_xor(acc[i], m, kWaveSize);
  }
}

// The same with the ids of the kernel arguments.
template <typename TIN, int LPR, bool BUF, typename KX>
__device__ __forceinline__ void pool_rows_coop(KX a, const TableInfo& ti, int64_t t, int64_t r0, int64_t r1,
                                               int lane, float* acc, int& bad) {
  pool_rows_src<TIN, LPR, BUF>(a, NativeIds{a->offsets, a->ids}, ti, t, r0, r1, lane, acc, bad);
}

// ---------------------------------------------------------------------------
// Bag by bag.  Wave w takes J = 2^jlog consecutive bags of one field, read
// straight from the offsets: the G row slots of the wave form J groups of
// P = G/J slots, group j pools bag b0 + j with its P slots taking rows p,
// p + P, p + 2P, ... (8 in flight per slot, the next ids prefetched), and the
// P partial sums meet in a fixed xor butterfly.  A bag of more than
// long_rows ids is skipped (neither pooled nor written): the caller pools it
// in pieces.
// ---------------------------------------------------------------------------
// Lane j < J of the wave holds the offsets of bag b0 + j (loaded before the
// field's class is known); slots fetch theirs by a cross-lane read.
struct DirectOffsets {
  int32_t lo, hi;
};

template <typename TIN, typename TOUT, int LPR, bool BUF, typename KX, typename S>
__device__ __forceinline__ int direct_bags(KX a, const S& src, const TableInfo& ti, int64_t t, int64_t b0, int jlog,
                                           DirectOffsets o, int64_t long_rows, int lane) {
  constexpr int EPL = In<TIN>::EPL;
  constexpr int G = kWaveSize / LPR;
  constexpr int GLOG = __builtin_ctz(G);
  const int g = lane / LPR, k = lane % LPR;
  const int plog = GLOG - jlog;   // J <= G for every field (chosen on the host)
  const int P = 1 << plog;
  const int j = g >> plog, p = g & (P - 1);
  const int64_t b = b0 + j;
  const bool active = b < a->B;
  // clamped to the field's id list
  const int64_t nnz = ti.nnz;
  int64_t s = __shfl(o.lo, j, kWaveSize), e = __shfl(o.hi, j, kWaveSize);
  s = s < 0 ? 0 : (s > nnz ? nnz : s);
  e = e < 0 ? 0 : (e > nnz ? nnz : e);
  if (e < s || !active) e = s;
  const bool skip = e - s > long_rows;
  if (skip) e = s;
  const RowReader<BUF> rows(a->tables[t], ti, k);
  const int64_t ib = ti.id_base;
  const uint32_t nrows = id_limit(ti);
  const bool col = k * EPL < ti.dim;
  float acc[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) acc[i] = 0.f;
  int bad = 0;
  const int64_t stride = (int64_t)P * kUnroll;
  int32_t idn[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int64_t r = s + p + (int64_t)u * P;
    idn[u] = r < e ? src.id(ib + r) : -1;
  }
  for (int64_t r = s + p; r < e; r += stride) {
    raw16_t raw[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      raw[u] = raw16_t{0, 0, 0, 0};
      const bool in_bag = r + (int64_t)u * P < e;
      const bool ok = in_bag && (uint32_t)idn[u] < nrows;
      bad |= (in_bag && !ok);
      if (ok && col) raw[u] = rows.load(idn[u]);
    }
    const int64_t rn = r + stride;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t q = rn + (int64_t)u * P;
      idn[u] = q < e ? src.id(ib + q) : -1;
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) accumulate<TIN, EPL>(acc, raw[u]);
  }
  // the P slots of a bag are consecutive: combine them (every lane active)
  for (int m = LPR; m < LPR * P; m <<= 1) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] += __shfl_xor(acc[i], m, kWaveSize);
  }
  if (p == 0 && active && col && !skip) {
    if (is_mean(a, t) && e > s) {
      const float L = (float)(e - s);
#pragma unroll
      for (int i = 0; i < EPL; ++i) acc[i] = acc[i] / L;
    }
    store_lane<TOUT, EPL>(out_row<TOUT>(a, ti, b) + k * EPL, acc, (ti.flags & kTiOutVec) != 0);
  }
  return bad;
}

template <typename TOUT, typename KX, typename S>
__device__ __forceinline__ int direct_wave(KX a, const S& src, const TableInfo& ti, int64_t t, int64_t b0, int jlog,
                                           DirectOffsets o, int64_t long_rows, int lane) {
  const bool buf = use_buffer(ti), f16 = (ti.flags & kTiF16) != 0;
  switch ((ti.flags >> kTiLprShift) & 7) {
#define DPI_CASE(L, LPR)                                                                                   \
  case L:                                                                                                  \
    if (f16)                                                                                               \
      return buf ? direct_bags<_Float16, TOUT, LPR, true>(a, src, ti, t, b0, jlog, o, long_rows, lane)     \
                 : direct_bags<_Float16, TOUT, LPR, false>(a, src, ti, t, b0, jlog, o, long_rows, lane);   \
    return buf ? direct_bags<float, TOUT, LPR, true>(a, src, ti, t, b0, jlog, o, long_rows, lane)          \
               : direct_bags<float, TOUT, LPR, false>(a, src, ti, t, b0, jlog, o, long_rows, lane);
    DPI_FOR_LPR(DPI_CASE)
#undef DPI_CASE
    default:
      return 0;
  }
}

// ---------------------------------------------------------------------------
// One-hot rows (no offsets: every bag is one id, Algorithm 1's case) of one
// row class: the pooled row is the row itself.  A wave takes G * kOneHotRows
// consecutive samples of one field from sample wave_b0 on; each slot copies
// kOneHotRows rows with all their loads in flight, converting to the output
// dtype (a one-id mean divides by 1, which is exact).
// ---------------------------------------------------------------------------
constexpr int kOneHotRows = 8;    // rows in flight per slot

template <typename TIN, typename TOUT, int LPR, typename KX>
__device__ __forceinline__ int onehot_rows(KX a, const TableInfo& ti, int64_t t, int64_t wave_b0, int lane) {
  constexpr int EPL = In<TIN>::EPL;
  constexpr int IPL = (kOneHotRows + LPR - 1) / LPR;
  const int g = lane / LPR, k = lane % LPR;
  const RowReader<true> rows(a->tables[t], ti, k);
  const int32_t* __restrict__ ids = a->ids + ti.id_base;
  const uint32_t nrows = id_limit(ti);
  const bool col = k * EPL < ti.dim;
  const bool vec = (ti.flags & kTiOutVec) != 0;
  const int64_t b0 = wave_b0 + (int64_t)g * kOneHotRows;
  // ids: lane k of a slot loads ids k, k + LPR, ... and the slot exchanges them
  int32_t idm[IPL];
#pragma unroll
  for (int j = 0; j < IPL; ++j) {
    const int q = k + j * LPR;
    idm[j] = (q < kOneHotRows && b0 + q < a->B) ? ids[b0 + q] : -1;
  }
  int32_t idn[kOneHotRows];
#pragma unroll
  for (int u = 0; u < kOneHotRows; ++u)
    idn[u] = LPR == 1 ? idm[u] : __shfl(idm[u / LPR], g * LPR + u % LPR, kWaveSize);
  raw16_t raw[kOneHotRows];
  int bad = 0;
#pragma unroll
  for (int u = 0; u < kOneHotRows; ++u) {
    raw[u] = raw16_t{0, 0, 0, 0};
    const bool in_range = b0 + u < a->B;
    const bool ok = in_range && (uint32_t)idn[u] < nrows;
    bad |= (in_range && !ok);
    if (ok && col) raw[u] = rows.load(idn[u]);
  }
  TOUT* const out_lane = out_row<TOUT>(a, ti, 0) + k * EPL;
#pragma unroll
  for (int u = 0; u < kOneHotRows; ++u) {
    if (b0 + u < a->B && col) {
      float v[EPL];
      unpack(raw[u], v, TIN());
#pragma unroll
      for (int i = 0; i < EPL; ++i) v[i] = 0.f + v[i];   // a sum from +0, as for longer bags: -0 -> +0
      store_lane<TOUT, EPL>(out_lane + (b0 + u) * a->total_d, v, vec);
    }
  }
  return bad;
}

}  // namespace
}  // namespace dpi
