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
// the row) and write the pooled row as consecutive pieces of the output row.
//   * Interior bags: the wave stages the bags' offsets in LDS, gives each slot
//     a contiguous run of whole bags holding about the same number of rows,
//     and each slot walks its rows as one stream (ids prefetched one step
//     ahead and shared across the slot's lanes by permutes, kUnroll rows in
//     flight), closing a bag whenever the stream crosses the bag's end (fp32
//     accumulation, rows in bag order).
//   * Few, long bags: all slots of the wave pool one bag together (rows
//     dealt round-robin to slots, then a fixed xor-butterfly across slots).
//   * A bag split between waves is pooled cooperatively by each wave holding
//     a piece; its fp32 partial goes to the workspace and the last wave to
//     arrive (agent-scope ticket) adds the partials in wave order and writes
//     the row -- deterministic, no floating-point atomics.
// Kernels: one fully inlined kernel per row class when every field shares
// one (lookup_uniform_kernel), a per-field dispatching one otherwise
// (lookup_mixed_kernel), a plain row copy for one-hot batches of one row
// class (lookup_onehot_kernel), and the input-first allocation kept for
// comparison (lookup_input_first_kernel).  Workgroups are remapped so each
// of the 8 XCDs takes a contiguous range of waves (a few fields per L2).
// Rows are read with buffer loads (32-bit offsets, range-checked by the
// descriptor) when the table is below 4 GiB, with 64-bit global loads
// otherwise.
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

constexpr int kUnroll = 8;        // rows in flight per slot
static_assert(kUnroll == kDirectGroupRows, "the host sizes direct bag groups by this");
constexpr int kTileBags = 256;    // bags whose offsets a wave stages in LDS at once
constexpr uint32_t kBufferWord3 = 0x00020000;   // raw buffer descriptor, gfx9 family

// Kernel arguments are read in place from the constant kernarg segment
// (scalar loads); a by-value copy would go to private memory because the
// table-pointer array is indexed at run time.
typedef const __attribute__((address_space(4))) LookupArgs* KA;

// Values known to be equal across the wave; out-of-line functions receive
// them in vector registers, so they are re-read from the first lane to let
// the compiler keep them (and what derives from them) in scalar registers.
__device__ __forceinline__ int64_t uni(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ KA uni(KA p) {
  return (KA)(uint64_t)uni((int64_t)(uint64_t)p);
}

__device__ __forceinline__ int32_t uni(int32_t x) { return __builtin_amdgcn_readfirstlane(x); }

// A field's static info, held in scalar registers.
__device__ __forceinline__ TableInfo table_info(KA a, int64_t t) {
  const TableInfo x = a->tinfo[t];
  TableInfo u;
  u.num_rows = uni(x.num_rows);
  u.id_base = uni(x.id_base);
  u.nnz = uni(x.nnz);
  u.dim = uni(x.dim);
  u.col_base = uni(x.col_base);
  u.row_bytes = uni(x.row_bytes);
  u.out_bytes = uni(x.out_bytes);
  u.flags = uni(x.flags);
  u.pad = 0;
  return u;
}

// ids are valid in [0, min(num_rows, 2^31)): one unsigned 32-bit compare
__device__ __forceinline__ uint32_t id_limit(const TableInfo& ti) {
  return (uint32_t)(ti.num_rows < ((int64_t)1 << 31) ? ti.num_rows : ((int64_t)1 << 31));
}

// per-wave staging of bag offsets
__shared__ int32_t g_bag_off[kWavesPerBlock][kTileBags + 1];

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

template <typename TOUT>
__device__ __forceinline__ TOUT* out_row(KA a, const TableInfo& ti, int64_t b) {
  return reinterpret_cast<TOUT*>(a->out) + b * a->total_d + ti.col_base;
}

__device__ __forceinline__ bool is_mean(KA a, int64_t t) {
  return (a->mean_bits[t >> 5] >> (t & 31)) & 1u;
}

// Position of bag boundary b (0..B) in field t's id list, clamped to the list.
__device__ __forceinline__ int32_t bag_offset(KA a, const TableInfo& ti, int64_t t, int64_t b) {
  int64_t v = a->offsets ? (int64_t)a->offsets[t * (a->B + 1) + b] : b;
  v = v < 0 ? 0 : (v > ti.nnz ? ti.nnz : v);
  return (int32_t)v;
}

__device__ __forceinline__ void bag_span(KA a, const TableInfo& ti, int64_t t, int64_t b, int64_t& s, int64_t& e) {
  s = bag_offset(a, ti, t, b);
  e = bag_offset(a, ti, t, b + 1);
  if (e < s) e = s;
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

// ---------------------------------------------------------------------------
// Fast path: row bytes a multiple of 16 and at most 1024; LPR lanes per row.
// ---------------------------------------------------------------------------

// Rows [r0, r1) of field t pooled by all slots of the wave; on return every
// slot holds the total for its lane's columns.
template <typename TIN, int LPR, bool BUF>
__device__ __forceinline__ void pool_rows_coop(KA a, const TableInfo& ti, int64_t t, int64_t r0, int64_t r1,
                                               int lane, float* acc, int& bad) {
  constexpr int EPL = In<TIN>::EPL;
  constexpr int G = kWaveSize / LPR;
  const int g = lane / LPR, k = lane % LPR;
  const RowReader<BUF> rows(a->tables[t], ti, k);
  const int32_t* __restrict__ ids = a->ids + ti.id_base;
  const uint32_t nrows = id_limit(ti);
  const bool col = k * EPL < ti.dim;
#pragma unroll
  for (int i = 0; i < EPL; ++i) acc[i] = 0.f;
  int32_t idn[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) idn[u] = (r0 + g + u * G < r1) ? ids[r0 + g + u * G] : -1;
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
    for (int u = 0; u < kUnroll; ++u) idn[u] = (rn + u * G < r1) ? ids[rn + u * G] : -1;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) accumulate<TIN, EPL>(acc, raw[u]);
  }
#pragma unroll
  for (int m = LPR; m < kWaveSize; m <<= 1) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] += __shfl_xor(acc[i], m, kWaveSize);
  }
}

// Whole bags [b_lo, b_hi) of field t, the wave pooling one bag at a time.
template <typename TIN, typename TOUT, int LPR, bool BUF, bool LEAN>
__device__ __forceinline__ int pool_bags_coop(KA a, int64_t t, int64_t b_lo, int64_t b_hi, int lane) {
  constexpr int EPL = In<TIN>::EPL;
  a = uni(a);
  t = uni(t);
  b_lo = uni(b_lo);
  b_hi = uni(b_hi);
  const int g = lane / LPR, k = lane % LPR;
  const TableInfo ti = table_info(a, t);
  const bool col = k * EPL < ti.dim;
  const bool mean = is_mean(a, t);
  const bool vec = (ti.flags & kTiOutVec) != 0;
  int bad = 0;
  for (int64_t b = b_lo; b < b_hi; ++b) {
    int64_t s, e;
    bag_span(a, ti, t, b, s, e);
    float acc[EPL];
    pool_rows_coop<TIN, LPR, BUF>(a, ti, t, s, e, lane, acc, bad);
    if (mean && e > s) {
      const float L = (float)(e - s);
      if constexpr (LEAN) {
        mean_divide<EPL>(acc, L);
      } else {
#pragma unroll
        for (int q = 0; q < EPL; ++q) acc[q] = acc[q] / L;
      }
    }
    if (g == 0 && col) store_lane<TOUT, EPL>(out_row<TOUT>(a, ti, b) + k * EPL, acc, vec);
  }
  return bad;
}

// Whole bags [b_lo, b_hi) of field t.
// LEAN (the single-row-class kernel): rows not taken read zeros through the
// buffer range check instead of a branch per row, ids are checked once per
// group, and mean bags divide by reciprocal and correction; the other kernels
// keep the branch-per-row form, which holds their registers lower.
template <typename TIN, typename TOUT, int LPR, bool BUF, bool LEAN = false, int U = kUnroll>
__device__ __forceinline__ int pool_segment_fast(KA a, int64_t t, int64_t b_lo, int64_t b_hi, int lane) {
  constexpr int EPL = In<TIN>::EPL;
  constexpr int G = kWaveSize / LPR;
  a = uni(a);
  t = uni(t);
  b_lo = uni(b_lo);
  b_hi = uni(b_hi);
  const int g = lane / LPR, k = lane % LPR;
  const TableInfo ti = table_info(a, t);
  const RowReader<BUF> rows(a->tables[t], ti, k);
  const int32_t* __restrict__ ids = a->ids + ti.id_base;
  const uint32_t nrows = id_limit(ti);
  const bool col = k * EPL < ti.dim;
  const bool mean = is_mean(a, t);
  const bool vec = (ti.flags & kTiOutVec) != 0;
  TOUT* const out_lane = out_row<TOUT>(a, ti, 0) + k * EPL;
  const int64_t ostride = a->total_d;
  int32_t* const off = g_bag_off[threadIdx.x / kWaveSize];
  int bad = 0;

  for (int64_t tb0 = b_lo; tb0 < b_hi; tb0 += kTileBags) {
    const int nb = (int)min((int64_t)kTileBags, b_hi - tb0);
    if (nb * 2 <= G &&
        (int64_t)(bag_offset(a, ti, t, tb0 + nb) - bag_offset(a, ti, t, tb0)) >= (int64_t)nb * G) {
      // few bags, each at least G rows long on average: the whole wave pools
      // one bag at a time (short bags are faster one per slot, in parallel)
      bad |= pool_bags_coop<TIN, TOUT, LPR, BUF, LEAN>(a, t, tb0, tb0 + nb, lane);
      continue;
    }
    // stage the tile's bag boundaries (wave-private LDS; LDS operations of
    // one wave complete in order, so no barrier is needed)
    for (int i = lane; i <= nb; i += kWaveSize) off[i] = bag_offset(a, ti, t, tb0 + i);
    const int32_t P0 = off[0], R = off[nb] - P0;
    // slot g owns the bags whose first row lies at or after P0 + ceil(g*R/G)
    // and before the next slot's start
    auto first_bag_at = [&](int slot) -> int {
      if (slot <= 0) return 0;
      if (slot >= G) return nb;
      const int32_t target = P0 + (int32_t)(((int64_t)slot * R + G - 1) / G);
      int lo = 0, hi = nb;   // smallest i in [0, nb] with off[i] >= target
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (off[mid] < target) lo = mid + 1; else hi = mid;
      }
      return lo;
    };
    int cur = first_bag_at(g);
    const int endb = first_bag_at(g + 1);
    int32_t r = off[cur];
    const int32_t r_end = off[endb];
    int32_t bstart = r;
    int32_t bend = cur < endb ? off[cur + 1] : r;
    TOUT* optr = out_lane + (tb0 + cur) * ostride;   // output row of bag cur
    float acc[EPL];
#pragma unroll
    for (int q = 0; q < EPL; ++q) acc[q] = 0.f;

    // close the current bag (pool, store, reset) and every empty bag after it
    // until the stream position r lies inside a bag; the bound on cur only
    // matters for offsets other than the non-decreasing ones the plan checked
    auto close_bags = [&]() {
      while (cur < endb && r >= bend) {
        const int32_t L = bend - bstart;
        if (mean && L > 0) {
          if constexpr (LEAN) {
            mean_divide<EPL>(acc, (float)L);
          } else {
            const float fl = (float)L;
#pragma unroll
            for (int q = 0; q < EPL; ++q) acc[q] = acc[q] / fl;
          }
        }
        if (col) store_lane<TOUT, EPL>(LEAN ? optr : out_lane + (tb0 + cur) * ostride, acc, vec);
#pragma unroll
        for (int q = 0; q < EPL; ++q) acc[q] = 0.f;
        ++cur;
        if constexpr (LEAN) optr += ostride;
        bstart = bend;
        if (cur < endb) bend = off[cur + 1];
      }
    };

    close_bags();   // leading empty bags
    // ids of a group: lane k of a slot loads ids k, k + LPR, ... of the group
    // and the slot's lanes exchange them by cross-lane permutes, so a group
    // costs ceil(U / LPR) id loads per lane instead of U
    constexpr int IPL = (U + LPR - 1) / LPR;
    int32_t idm[IPL];
    bool idv[IPL];   // idm[j] holds an id of this slot's run
    auto fetch_ids = [&](int32_t p) {
#pragma unroll
      for (int j = 0; j < IPL; ++j) {
        const int q = k + j * LPR;
        idv[j] = q < U && (uint32_t)p + q < (uint32_t)r_end;
        idm[j] = idv[j] ? ids[p + q] : -1;
      }
    };
    fetch_ids(r);
    while (cur < endb) {
      // one group of up to U rows of the current bag; the lanes of a
      // slot are active together, so every permute reads an active lane
      // every id of the run passes through some lane's idm (a group reads
      // from its first row on), so checking the fetched ids once per group
      // finds every id outside the table
      // rows of this group; positions are below 2^31, so unsigned sums of a
      // position and at most U cannot overflow
      const int32_t n_in = (int32_t)(min((uint32_t)r + U, (uint32_t)bend) - (uint32_t)r);
      raw16_t raw[U];
      if constexpr (LEAN) {
        static_assert(BUF, "the single-row-class kernel reads tables through buffer descriptors");
        // A slot's lanes cover whole rows (LPR * 16 = row bytes, a power of
        // two): each lane turns the ids it fetched into row offsets, masking
        // the rows past the group's end and ids outside the table, and the
        // slot exchanges offsets, so a row costs one add per lane, not a
        // compare, a multiply and a select.
        constexpr uint32_t RB = LPR * 16;
        uint32_t roff[IPL];
#pragma unroll
        for (int j = 0; j < IPL; ++j) {
          const bool id_ok = (uint32_t)idm[j] < nrows;
          bad |= idv[j] && !id_ok;
          roff[j] = (k + j * LPR < n_in && id_ok) ? (uint32_t)idm[j] * RB : masked_row_offset<RB>();
        }
        uint32_t ro[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
          ro[u] = LPR == 1 ? roff[u] : (uint32_t)__shfl((int)roff[u / LPR], g * LPR + u % LPR, kWaveSize);
#pragma unroll
        for (int u = 0; u < U; ++u) raw[u] = rows.load_at(ro[u]);
        // all of the group's loads leave before the first add waits for one:
        // left to itself the scheduler moves adds between the loads, and each
        // add's wait then holds back the loads after it (multi-hot batch:
        // 81 -> 64 us)
        __builtin_amdgcn_sched_barrier(0);
      } else {
        int32_t idn[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
          idn[u] = LPR == 1 ? idm[u] : __shfl(idm[u / LPR], g * LPR + u % LPR, kWaveSize);
#pragma unroll
        for (int u = 0; u < U; ++u) {
          raw[u] = raw16_t{0, 0, 0, 0};
          const bool in_group = u < n_in;
          const bool ok = in_group && (uint32_t)idn[u] < nrows;
          bad |= (in_group && !ok);
          if (ok && col) raw[u] = rows.load(idn[u]);
        }
      }
      const int32_t ge = r + n_in;
      // the next group starts at ge: prefetch its ids
      if constexpr (LEAN && LPR <= U) {
        // inside the loop the run still holds a row (r < r_end), so the
        // clamped index is an id of the run and the load needs no branch;
        // with every load of the group issued unconditionally the adds wait
        // for the rows only, not for this prefetch (multi-hot batch of
        // 128-byte rows: -2 %; with 16 or more lanes per row, where lanes
        // past the group's ids load too, the large batch ran 4 % slower)
        static_assert(IPL * LPR == U, "every lane fetches one id of the group");
#pragma unroll
        for (int j = 0; j < IPL; ++j) {
          const int q = k + j * LPR;
          idv[j] = (uint32_t)ge + q < (uint32_t)r_end;
          idm[j] = ids[min((uint32_t)ge + q, (uint32_t)r_end - 1u)];
        }
      } else {
        fetch_ids(ge);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) accumulate<TIN, EPL>(acc, raw[u]);
      r = ge;
      close_bags();
    }
  }
  return bad;
}

// Rows [row_lo, row_hi) of bag b (bag-relative), fp32 partial to `slot`.
template <typename TIN, int LPR, bool BUF>
__device__ __forceinline__ int partial_fast(KA a, int64_t t, int64_t b, int64_t row_lo, int64_t row_hi,
                                           int64_t slot, int lane) {
  constexpr int EPL = In<TIN>::EPL;
  a = uni(a);
  t = uni(t);
  b = uni(b);
  row_lo = uni(row_lo);
  row_hi = uni(row_hi);
  slot = uni(slot);
  const int g = lane / LPR, k = lane % LPR;
  const TableInfo ti = table_info(a, t);
  int bad = 0;
  int64_t s, e;
  bag_span(a, ti, t, b, s, e);
  const int64_t r0 = min(e, s + row_lo), r1 = min(e, s + row_hi);
  float acc[EPL];
  pool_rows_coop<TIN, LPR, BUF>(a, ti, t, r0, r1, lane, acc, bad);
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
  a = uni(a);
  t = uni(t);
  b = uni(b);
  row_lo = uni(row_lo);
  row_hi = uni(row_hi);
  slot = uni(slot);
  const TableInfo ti = table_info(a, t);
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
__device__ __forceinline__ void finish_piece(KA a, int64_t w_first, int64_t bag, int lane) {
  a = uni(a);
  w_first = uni(w_first);
  bag = uni(bag);
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
  const TableInfo ti = table_info(a, t);
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
// Work of one wave, parameterised by how a field's rows are pooled.
//   Uniform<TIN, TOUT, LPR>: every field has the same row class and fits a
//     buffer descriptor; everything is inlined into one lean kernel.
//   Mixed<TOUT>: fields of different classes; a wave-uniform switch calls
//     out-of-line routines per class (including the general path).
// ---------------------------------------------------------------------------
#define DPI_FOR_LPR(MACRO) \
  MACRO(0, 1) MACRO(1, 2) MACRO(2, 4) MACRO(3, 8) MACRO(4, 16) MACRO(5, 32) MACRO(6, 64)

template <typename TIN, typename TOUT, int LPR, int U = kUnroll>
struct Uniform {
  static __device__ __forceinline__ int segment(KA a, int64_t t, int64_t b_lo, int64_t b_hi, int lane) {
    return pool_segment_fast<TIN, TOUT, LPR, true, true, U>(a, t, b_lo, b_hi, lane);
  }
  static __device__ __forceinline__ int partial(KA a, int64_t t, int64_t b, int64_t lo, int64_t hi, int64_t slot,
                                                int lane) {
    return partial_fast<TIN, LPR, true>(a, t, b, lo, hi, slot, lane);
  }
  static __device__ __forceinline__ void finish(KA a, int64_t w_first, int64_t bag, int lane) {
    finish_piece<TOUT>(a, w_first, bag, lane);
  }
};

template <typename TIN, typename TOUT, int LPR, bool BUF>
__device__ __attribute__((noinline)) int segment_call(KA a, int64_t t, int64_t b_lo, int64_t b_hi, int lane) {
  return pool_segment_fast<TIN, TOUT, LPR, BUF>(a, t, b_lo, b_hi, lane);
}
template <typename TIN, int LPR>
__device__ __attribute__((noinline)) int partial_call(KA a, int64_t t, int64_t b, int64_t lo, int64_t hi,
                                                      int64_t slot, int lane) {
  return partial_fast<TIN, LPR, false>(a, t, b, lo, hi, slot, lane);
}
template <typename TOUT>
__device__ __attribute__((noinline)) void finish_call(KA a, int64_t w_first, int64_t bag, int lane) {
  finish_piece<TOUT>(a, w_first, bag, lane);
}

// buffer descriptors hold an unsigned 32-bit byte range
__device__ __forceinline__ bool use_buffer(const TableInfo& ti) {
  return ti.num_rows * (int64_t)ti.row_bytes <= (int64_t)0xffffffffLL;
}

template <typename TOUT>
struct Mixed {
  static __device__ int segment(KA a, int64_t t, int64_t b_lo, int64_t b_hi, int lane) {
    const TableInfo ti = table_info(a, t);
    const int flags = ti.flags;
    if (!(flags & kTiFast)) {
      int bad = 0;
      for (int64_t b = b_lo; b < b_hi; ++b) {
        if (flags & kTiF16)
          bad |= pool_general<_Float16, TOUT>(a, t, b, 0, INT64_MAX / 2, true, 0, lane);
        else
          bad |= pool_general<float, TOUT>(a, t, b, 0, INT64_MAX / 2, true, 0, lane);
      }
      return bad;
    }
    const bool buf = use_buffer(ti), f16 = (flags & kTiF16) != 0;
    switch ((flags >> kTiLprShift) & 7) {
#define DPI_CASE(L, LPR)                                                                   \
  case L:                                                                                  \
    if (f16)                                                                               \
      return buf ? segment_call<_Float16, TOUT, LPR, true>(a, t, b_lo, b_hi, lane)         \
                 : segment_call<_Float16, TOUT, LPR, false>(a, t, b_lo, b_hi, lane);       \
    return buf ? segment_call<float, TOUT, LPR, true>(a, t, b_lo, b_hi, lane)              \
               : segment_call<float, TOUT, LPR, false>(a, t, b_lo, b_hi, lane);
      DPI_FOR_LPR(DPI_CASE)
#undef DPI_CASE
      default:
        return 0;
    }
  }
  static __device__ int partial(KA a, int64_t t, int64_t b, int64_t lo, int64_t hi, int64_t slot, int lane) {
    const int flags = table_info(a, t).flags;
    if (!(flags & kTiFast)) {
      return (flags & kTiF16) ? pool_general<_Float16, TOUT>(a, t, b, lo, hi, false, slot, lane)
                              : pool_general<float, TOUT>(a, t, b, lo, hi, false, slot, lane);
    }
    const bool f16 = (flags & kTiF16) != 0;
    switch ((flags >> kTiLprShift) & 7) {
#define DPI_CASE(L, LPR)                                                                          \
  case L:                                                                                         \
    return f16 ? partial_call<_Float16, LPR>(a, t, b, lo, hi, slot, lane)                         \
               : partial_call<float, LPR>(a, t, b, lo, hi, slot, lane);
      DPI_FOR_LPR(DPI_CASE)
#undef DPI_CASE
      default:
        return 0;
    }
  }
  static __device__ void finish(KA a, int64_t w_first, int64_t bag, int lane) {
    finish_call<TOUT>(a, w_first, bag, lane);
  }
};

// Bags [lA, lB) (global bag numbers, field-major), split at field ends.
template <typename P>
__device__ __forceinline__ int pool_bag_range(KA a, int64_t lA, int64_t lB, int lane) {
  int bad = 0;
  while (lA < lB) {
    const int64_t t = __builtin_amdgcn_readfirstlane((int)(lA / a->B));
    const int64_t seg_end = min(lB, (t + 1) * a->B);
    bad |= P::segment(a, t, lA - t * a->B, seg_end - t * a->B, lane);
    lA = seg_end;
  }
  return bad;
}

// Rows [row_lo, row_hi) of a bag shared with other waves: partial, then the
// arrival protocol.
template <typename P>
__device__ __forceinline__ int pool_partial(KA a, int64_t bag, int64_t row_lo, int64_t row_hi, int64_t slot,
                                            int64_t w_first, int lane) {
  const int64_t t = __builtin_amdgcn_readfirstlane((int)(bag / a->B));
  const int bad = P::partial(a, t, bag - t * a->B, row_lo, row_hi, slot, lane);
  P::finish(a, w_first, bag, lane);
  return bad;
}

__device__ __forceinline__ int64_t xcd_affine_block(int64_t g, int64_t n) {
  // workgroups are dispatched round-robin over 8 XCDs; give XCD x the
  // contiguous logical range of its round-robin share
  const int64_t x = g & 7, i = g >> 3, q = n >> 3, r = n & 7;
  return x < r ? x * (q + 1) + i : r * (q + 1) + (x - r) * q + i;
}

template <typename P>
__device__ __forceinline__ void wave_body(KA a) {
  const int lane = threadIdx.x & (kWaveSize - 1);
  int64_t blk = blockIdx.x;
  if (a->xcd_affine) blk = xcd_affine_block(blk, gridDim.x);
  const int64_t w = blk * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
  if (w >= a->grid_waves) return;
  // the plan's wave count and verdict and this wave's range, requested
  // together (the arrays hold grid_waves + 1 entries; values past the plan's
  // W are never used)
  const int64_t W = min(a->hdr[kHdrW], a->grid_waves);
  const int32_t st_err = *a->status;
  const int64_t i0 = a->wib[w], i1 = a->wib[w + 1];
  const int64_t la = a->wave_bag[w], lz = a->wave_bag[w + 1];
  const int64_t la_base = a->wbase[w], lz_base = a->wbase[w + 1];
  if (w >= W) return;
  if (st_err & kStatusBadOffsets) return;   // the plan rejected the offsets
  if (i0 >= i1) return;
  const int64_t TB = a->B * a->T;
  const int64_t C = a->C;
  // item i1 lies in bag lz: the wave ends inside lz (a tail piece, lz is the
  // last bag) exactly when lz starts before i1, else its last bag is lz - 1
  const bool tail = lz < TB && lz_base < i1;
  const int64_t lb = tail ? lz : lz - 1;
  const int64_t lb_base = lz_base;   // read only with tail
  const bool head = la_base < i0;
  int bad = 0;
  if (la == lb && (head || tail)) {
    const int64_t slot = head ? 2 * w : 2 * w + 1;
    const int64_t w_first = head ? (int64_t)a->head_first[w] : w;
    bad |= pool_partial<P>(a, la, (i0 - la_base) * C, (i1 - la_base) * C, slot, w_first, lane);
  } else {
    int64_t lA = la, lB = lb + 1;
    if (head) {
      bad |= pool_partial<P>(a, la, (i0 - la_base) * C, INT64_MAX / 2, 2 * w, a->head_first[w], lane);
      lA = la + 1;
    }
    if (tail) lB = lb;
    bad |= pool_bag_range<P>(a, lA, lB, lane);
    if (tail) bad |= pool_partial<P>(a, lb, 0, (i1 - lb_base) * C, 2 * w + 1, w, lane);
  }
  if (__any(bad) && lane == 0)
    __hip_atomic_fetch_or(a->status, kStatusBadId, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// five waves per SIMD: at most 96 VGPRs (512 per SIMD lane, granule 8)
template <typename TIN, typename TOUT, int LPR>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(5)))
void lookup_uniform_kernel(const LookupArgs args) {
  (void)args;
  wave_body<Uniform<TIN, TOUT, LPR>>((KA)__builtin_amdgcn_kernarg_segment_ptr());
}

// four waves per SIMD (at most 128 VGPRs): faster than the two an
// unconstrained allocation gives, despite some spilling
template <typename TOUT>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(4)))
void lookup_mixed_kernel(const LookupArgs args) {
  (void)args;
  wave_body<Mixed<TOUT>>((KA)__builtin_amdgcn_kernarg_segment_ptr());
}

// ---------------------------------------------------------------------------
// One-hot batches (no offsets: every bag is one id, Algorithm 1's case) of a
// uniform row class: the pooled row is the row itself, so the plan's
// partition is not needed.  A wave takes G * kOneHotRows consecutive samples
// of one field; each slot copies kOneHotRows rows with all their loads in
// flight, converting to the output dtype (a one-id mean divides by 1, which
// is exact).
// ---------------------------------------------------------------------------
constexpr int kOneHotRows = 8;    // rows in flight per slot

template <typename TIN, typename TOUT, int LPR>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(5)))
void lookup_onehot_kernel(const LookupArgs args) {
  (void)args;
  constexpr int EPL = In<TIN>::EPL;
  constexpr int G = kWaveSize / LPR;
  constexpr int64_t kRowsPerWave = (int64_t)G * kOneHotRows;
  constexpr int IPL = (kOneHotRows + LPR - 1) / LPR;
  const KA a = (KA)__builtin_amdgcn_kernarg_segment_ptr();
  const int lane = threadIdx.x & (kWaveSize - 1);
  const int g = lane / LPR, k = lane % LPR;
  const int64_t blk = a->xcd_affine ? xcd_affine_block(blockIdx.x, gridDim.x) : (int64_t)blockIdx.x;
  const int64_t per_field = (a->B + kRowsPerWave - 1) / kRowsPerWave;
  const int64_t gw = blk * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
  if (gw >= per_field * a->T) return;
  if (*a->status & kStatusBadOffsets) return;
  const int64_t t = uni(gw / per_field);
  const TableInfo ti = table_info(a, t);
  const RowReader<true> rows(a->tables[t], ti, k);
  const int32_t* __restrict__ ids = a->ids + ti.id_base;
  const uint32_t nrows = id_limit(ti);
  const bool col = k * EPL < ti.dim;
  const bool vec = (ti.flags & kTiOutVec) != 0;
  const int64_t b0 = (gw - t * per_field) * kRowsPerWave + (int64_t)g * kOneHotRows;
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
  if (__any(bad) && lane == 0)
    __hip_atomic_fetch_or(a->status, kStatusBadId, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// Small batches, bag by bag.  With few bags, none of them long, the plan's
// balanced partition buys nothing and costs a chain of dependent loads (wave
// range, bag bases, field info) before the first row is requested.  Here wave
// w takes J = 2^jlog consecutive bags of one field, read straight from the
// offsets: the G row slots of the wave form J groups of P = G/J slots, group
// j pools bag b0 + j with its P slots taking rows p, p + P, p + 2P, ... (8 in
// flight per slot, the next ids prefetched), and the P partial sums meet in a
// fixed xor butterfly.  J is the same for every field, so a field has
// ceil(B/J) waves and a wave finds its field by one division.  The plan still
// runs first: it validates the offsets and counts the bags longer than
// kDirectMaxItems chunks; with any such bag the launch falls back to the
// plan's partition (same kernel, wave_body), so one long bag never holds up
// a whole lookup.
// ---------------------------------------------------------------------------
// Lane j < J of the wave holds the offsets of bag b0 + j (loaded before the
// field's class is known); slots fetch theirs by a cross-lane read.
struct DirectOffsets {
  int32_t lo, hi;
};

template <typename TIN, typename TOUT, int LPR, bool BUF>
__device__ __forceinline__ int direct_bags(KA a, const TableInfo& ti, int64_t t, int64_t b0, int jlog,
                                           DirectOffsets o, int lane) {
  constexpr int EPL = In<TIN>::EPL;
  constexpr int G = kWaveSize / LPR;
  constexpr int GLOG = __builtin_ctz(G);
  const int g = lane / LPR, k = lane % LPR;
  const int plog = GLOG - jlog;   // J <= G for every field (chosen on the host)
  const int P = 1 << plog;
  const int j = g >> plog, p = g & (P - 1);
  const int64_t b = b0 + j;
  const bool active = b < a->B;
  // clamped to the field's id list as bag_span does
  const int64_t nnz = ti.nnz;
  int64_t s = __shfl(o.lo, j, kWaveSize), e = __shfl(o.hi, j, kWaveSize);
  s = s < 0 ? 0 : (s > nnz ? nnz : s);
  e = e < 0 ? 0 : (e > nnz ? nnz : e);
  if (e < s || !active) e = s;
  const RowReader<BUF> rows(a->tables[t], ti, k);
  const int32_t* __restrict__ ids = a->ids + ti.id_base;
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
    idn[u] = r < e ? ids[r] : -1;
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
      idn[u] = q < e ? ids[q] : -1;
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) accumulate<TIN, EPL>(acc, raw[u]);
  }
  // the P slots of a bag are consecutive: combine them (every lane active)
  for (int m = LPR; m < LPR * P; m <<= 1) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] += __shfl_xor(acc[i], m, kWaveSize);
  }
  if (p == 0 && active && col) {
    if (is_mean(a, t) && e > s) {
      const float L = (float)(e - s);
#pragma unroll
      for (int i = 0; i < EPL; ++i) acc[i] = acc[i] / L;
    }
    store_lane<TOUT, EPL>(out_row<TOUT>(a, ti, b) + k * EPL, acc, (ti.flags & kTiOutVec) != 0);
  }
  return bad;
}

template <typename TOUT>
__device__ __forceinline__ int direct_wave(KA a, const TableInfo& ti, int64_t t, int64_t b0, int jlog,
                                           DirectOffsets o, int lane) {
  const bool buf = use_buffer(ti), f16 = (ti.flags & kTiF16) != 0;
  switch ((ti.flags >> kTiLprShift) & 7) {
#define DPI_CASE(L, LPR)                                                                          \
  case L:                                                                                         \
    if (f16)                                                                                      \
      return buf ? direct_bags<_Float16, TOUT, LPR, true>(a, ti, t, b0, jlog, o, lane)            \
                 : direct_bags<_Float16, TOUT, LPR, false>(a, ti, t, b0, jlog, o, lane);          \
    return buf ? direct_bags<float, TOUT, LPR, true>(a, ti, t, b0, jlog, o, lane)                 \
               : direct_bags<float, TOUT, LPR, false>(a, ti, t, b0, jlog, o, lane);
    DPI_FOR_LPR(DPI_CASE)
#undef DPI_CASE
    default:
      return 0;
  }
}

// four waves per SIMD, as the mixed kernel it falls back to
template <typename TOUT>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(4)))
void lookup_direct_kernel(const LookupArgs args) {
  (void)args;
  const KA a = (KA)__builtin_amdgcn_kernarg_segment_ptr();
  const int lane = threadIdx.x & (kWaveSize - 1);
  const int64_t w = (int64_t)blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
  // the plan's verdicts, the field's info and the wave's bag offsets are all
  // requested before the first of them is needed (one round trip, not three)
  const int32_t st_err = a->status[0], st_long = a->status[1];
  const int64_t wpf = a->direct_wpf;
  const int64_t t = w < wpf * a->T ? uni(w / wpf) : 0;
  // this field's bags per wave (its slot count from the kernel arguments)
  const int jlog = min(6 - (int)a->lpr_log[t] - a->direct_plog, a->direct_jcap_log);
  const int64_t b0 = (w - t * wpf) << jlog;
  const bool mine = w < wpf * a->T && b0 < a->B;
  DirectOffsets o{0, 0};
  if (mine && lane < (1 << jlog)) {
    const int64_t bl = min(b0 + lane, a->B - 1);   // bags past the batch end are inactive
    if (a->offsets) {
      const int32_t* src = a->offsets + t * (a->B + 1) + bl;
      o.lo = src[0];
      o.hi = src[1];
    } else {
      o.lo = (int32_t)bl;
      o.hi = (int32_t)bl + 1;
    }
  }
  const TableInfo ti = table_info(a, t);
  if (st_err & kStatusBadOffsets) return;   // the plan rejected the offsets
  if (st_long != 0) {                       // a long bag: the plan's partition
    wave_body<Mixed<TOUT>>(a);
    return;
  }
  if (!mine) return;
  const int bad = direct_wave<TOUT>(a, ti, t, b0, jlog, o, lane);
  if (__any(bad) && lane == 0)
    __hip_atomic_fetch_or(a->status, kStatusBadId, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// Input-first allocation (the alternative of §IV-C, kept for the paper's
// allocation comparison): one lane per bag.  A wave takes 64 consecutive bags
// of one field; each lane walks its own bag's rows and, 16 bytes at a time,
// all of the row's columns, then writes its own output row.  Loads of a wave
// touch 64 different rows and its stores 64 different output rows; the work
// plan is used only for the field info and the offset check.
// ---------------------------------------------------------------------------
template <typename TIN, typename TOUT>
__device__ __forceinline__ int input_first_bag(KA a, const TableInfo& ti, int64_t t, int64_t b) {
  constexpr int EPL = In<TIN>::EPL;
  constexpr int EPW = 4 / sizeof(TIN);
  int64_t s, e;
  bag_span(a, ti, t, b, s, e);
  const int32_t* __restrict__ ids = a->ids + ti.id_base;
  const char* table = reinterpret_cast<const char*>(a->tables[t]);
  const uint32_t nrows = id_limit(ti);
  const bool mean = is_mean(a, t) && e > s;
  TOUT* dst = out_row<TOUT>(a, ti, b);
  const bool vec_in = (ti.row_bytes & 15) == 0;
  int bad = 0;
  const int64_t pieces = vec_in ? ti.row_bytes / 16 : ti.row_bytes / 4;
  for (int64_t q = 0; q < pieces; ++q) {
    if (vec_in) {
      float acc[EPL];
#pragma unroll
      for (int i = 0; i < EPL; ++i) acc[i] = 0.f;
      for (int64_t r = s; r < e; ++r) {
        const uint32_t id = (uint32_t)ids[r];
        if (id >= nrows) {
          bad = 1;
          continue;
        }
        accumulate<TIN, EPL>(acc, *reinterpret_cast<const raw16_t*>(table + (uint64_t)id * ti.row_bytes + q * 16));
      }
      if (mean) {
#pragma unroll
        for (int i = 0; i < EPL; ++i) acc[i] = acc[i] / (float)(e - s);
      }
      const int c0 = (int)q * EPL;
      const int cn = min(EPL, ti.dim - c0);
      if (cn == EPL && (ti.flags & kTiOutVec)) {
        store_lane<TOUT, EPL>(dst + c0, acc, true);
      } else {
        for (int i = 0; i < cn; ++i) dst[c0 + i] = (TOUT)acc[i];
      }
    } else {
      float acc[EPW];
#pragma unroll
      for (int i = 0; i < EPW; ++i) acc[i] = 0.f;
      for (int64_t r = s; r < e; ++r) {
        const uint32_t id = (uint32_t)ids[r];
        if (id >= nrows) {
          bad = 1;
          continue;
        }
        const TIN* src = reinterpret_cast<const TIN*>(table + (uint64_t)id * ti.row_bytes + q * 4);
#pragma unroll
        for (int i = 0; i < EPW; ++i) acc[i] += (float)src[i];
      }
      if (mean) {
#pragma unroll
        for (int i = 0; i < EPW; ++i) acc[i] = acc[i] / (float)(e - s);
      }
#pragma unroll
      for (int i = 0; i < EPW; ++i) dst[q * EPW + i] = (TOUT)acc[i];
    }
  }
  return bad;
}

template <typename TOUT>
__global__ __launch_bounds__(kBlockThreads) void lookup_input_first_kernel(const LookupArgs args) {
  (void)args;
  const KA a = (KA)__builtin_amdgcn_kernarg_segment_ptr();
  const int lane = threadIdx.x & (kWaveSize - 1);
  const int64_t per_field = (a->B + kWaveSize - 1) / kWaveSize;
  const int64_t gw = (int64_t)blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
  if (gw >= per_field * a->T) return;
  if (*a->status & kStatusBadOffsets) return;   // the plan rejected the offsets
  const int64_t t = gw / per_field;
  const int64_t b = (gw - t * per_field) * kWaveSize + lane;
  const TableInfo ti = table_info(a, t);
  int bad = 0;
  if (b < a->B) {
    bad = (ti.flags & kTiF16) ? input_first_bag<_Float16, TOUT>(a, ti, t, b)
                              : input_first_bag<float, TOUT>(a, ti, t, b);
  }
  if (__any(bad) && lane == 0)
    __hip_atomic_fetch_or(a->status, kStatusBadId, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace

hipError_t launch_lookup(const LookupArgs& a, hipStream_t s) {
  if (a.input_first) {
    const int64_t waves = (a.B + kWaveSize - 1) / kWaveSize * a.T;
    const int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    if (blocks <= 0) return hipSuccess;
    if (a.out_f16)
      hipLaunchKernelGGL(lookup_input_first_kernel<_Float16>, dim3((unsigned)blocks), dim3(kBlockThreads), 0, s, a);
    else
      hipLaunchKernelGGL(lookup_input_first_kernel<float>, dim3((unsigned)blocks), dim3(kBlockThreads), 0, s, a);
    return hipGetLastError();
  }
  if (a.onehot && a.uniform_class >= 0) {
    const int lpr = 1 << ((a.uniform_class >> kTiLprShift) & 7);
    const int64_t rows_per_wave = (int64_t)(kWaveSize / lpr) * kOneHotRows;
    const int64_t waves = (a.B + rows_per_wave - 1) / rows_per_wave * a.T;
    const int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    if (blocks <= 0) return hipSuccess;
    const dim3 grid((unsigned)blocks), block(kBlockThreads);
    const bool f16 = (a.uniform_class & kTiF16) != 0;
    switch ((a.uniform_class >> kTiLprShift) & 7) {
#define DPI_CASE(L, LPR)                                                                               \
  case L:                                                                                              \
    if (f16 && a.out_f16)                                                                              \
      hipLaunchKernelGGL((lookup_onehot_kernel<_Float16, _Float16, LPR>), grid, block, 0, s, a);       \
    else if (f16)                                                                                      \
      hipLaunchKernelGGL((lookup_onehot_kernel<_Float16, float, LPR>), grid, block, 0, s, a);          \
    else if (a.out_f16)                                                                                \
      hipLaunchKernelGGL((lookup_onehot_kernel<float, _Float16, LPR>), grid, block, 0, s, a);          \
    else                                                                                               \
      hipLaunchKernelGGL((lookup_onehot_kernel<float, float, LPR>), grid, block, 0, s, a);             \
    break;
      DPI_FOR_LPR(DPI_CASE)
#undef DPI_CASE
      default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  if (a.direct_plog >= 0) {
    // enough waves for either mode: bag groups, or the plan's waves
    const int64_t waves = std::max<int64_t>(a.direct_wpf * a.T, a.grid_waves);
    const int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    if (blocks <= 0) return hipSuccess;
    if (a.out_f16)
      hipLaunchKernelGGL(lookup_direct_kernel<_Float16>, dim3((unsigned)blocks), dim3(kBlockThreads), 0, s, a);
    else
      hipLaunchKernelGGL(lookup_direct_kernel<float>, dim3((unsigned)blocks), dim3(kBlockThreads), 0, s, a);
    return hipGetLastError();
  }
  const int64_t blocks = (a.grid_waves + kWavesPerBlock - 1) / kWavesPerBlock;
  if (blocks <= 0) return hipSuccess;
  const dim3 grid((unsigned)blocks), block(kBlockThreads);
  if (a.uniform_class < 0) {
    if (a.out_f16)
      hipLaunchKernelGGL(lookup_mixed_kernel<_Float16>, grid, block, 0, s, a);
    else
      hipLaunchKernelGGL(lookup_mixed_kernel<float>, grid, block, 0, s, a);
    return hipGetLastError();
  }
  const bool f16 = (a.uniform_class & kTiF16) != 0;
  switch ((a.uniform_class >> kTiLprShift) & 7) {
#define DPI_CASE(L, LPR)                                                                               \
  case L:                                                                                              \
    if (f16 && a.out_f16)                                                                              \
      hipLaunchKernelGGL((lookup_uniform_kernel<_Float16, _Float16, LPR>), grid, block, 0, s, a);      \
    else if (f16)                                                                                      \
      hipLaunchKernelGGL((lookup_uniform_kernel<_Float16, float, LPR>), grid, block, 0, s, a);         \
    else if (a.out_f16)                                                                                \
      hipLaunchKernelGGL((lookup_uniform_kernel<float, _Float16, LPR>), grid, block, 0, s, a);         \
    else                                                                                               \
      hipLaunchKernelGGL((lookup_uniform_kernel<float, float, LPR>), grid, block, 0, s, a);            \
    break;
    DPI_FOR_LPR(DPI_CASE)
#undef DPI_CASE
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace dpi
