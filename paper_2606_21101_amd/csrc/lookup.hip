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
#include "gather.h"

namespace dpi {
namespace {

constexpr int kTileBags = 256;    // bags whose offsets a wave stages in LDS at once

// Kernel arguments are read in place from the constant kernarg segment
// (scalar loads); a by-value copy would go to private memory because the
// table-pointer array is indexed at run time.
typedef const __attribute__((address_space(4))) LookupArgs* KA;

__device__ __forceinline__ KA uni(KA p) {
  return (KA)(uint64_t)uni((int64_t)(uint64_t)p);
}

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

// per-wave staging of bag offsets
__shared__ int32_t g_bag_off[kWavesPerBlock][kTileBags + 1];

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
//
// SPAN (LEAN only): a group runs on past the end of the current bag into the
// next one (never beyond it), so that a slot keeps up to U rows in flight
// across bag ends; each row is added to the accumulator of its bag (the
// current one, or the next one's, which becomes current when the bag closes).
// Used for 8-lane rows (bags of about ten rows, where groups cut at bag ends
// held five rows on average); it doubles the adds, which costs more than it
// gains where the adds already bound the kernel (16-lane rows).
template <typename TIN, typename TOUT, int LPR, bool BUF, bool LEAN = false, int U = kUnroll, bool SPAN = false>
__device__ __forceinline__ int pool_segment_fast(KA a, int64_t t, int64_t b_lo, int64_t b_hi, int lane) {
  static_assert(!SPAN || LEAN, "spanning groups need the single-row-class kernel's masked loads");
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
    // SPAN: the end of the bag after cur (bend when cur is the slot's last)
    int32_t bnext = SPAN ? (cur + 1 < endb ? off[cur + 2] : bend) : 0;
    TOUT* optr = out_lane + (tb0 + cur) * ostride;   // output row of bag cur
    float acc[EPL], acc2[SPAN ? EPL : 1];
#pragma unroll
    for (int q = 0; q < EPL; ++q) acc[q] = 0.f;
#pragma unroll
    for (int q = 0; q < (SPAN ? EPL : 1); ++q) acc2[q] = 0.f;

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
        if constexpr (SPAN) {
          // the next bag's rows summed so far become the current sum
#pragma unroll
          for (int q = 0; q < EPL; ++q) {
            acc[q] = acc2[q];
            acc2[q] = 0.f;
          }
        } else {
#pragma unroll
          for (int q = 0; q < EPL; ++q) acc[q] = 0.f;
        }
        ++cur;
        if constexpr (LEAN) optr += ostride;
        bstart = bend;
        if constexpr (SPAN) {
          bend = bnext;
          if (cur + 1 < endb) bnext = off[cur + 2];
        } else {
          if (cur < endb) bend = off[cur + 1];
        }
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
      // (SPAN: up to the end of the next bag; bnext >= bend > r)
      const int32_t n_in = (int32_t)(min((uint32_t)r + U, (uint32_t)(SPAN ? bnext : bend)) - (uint32_t)r);
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
      if constexpr (SPAN) {
        // rows [0, split) of the group belong to bag cur, the rest to the next
        const int32_t split = bend - r;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          // each row's bytes go to one accumulator, zeros to the other (a
          // select of the raw bits: a row's infinities or NaNs stay in its bag)
          const bool mine = u < split;
          raw16_t here, next;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            here[q] = mine ? raw[u][q] : 0;
            next[q] = mine ? 0 : raw[u][q];
          }
          accumulate<TIN, EPL>(acc, here);
          accumulate<TIN, EPL>(acc2, next);
        }
      } else {
#pragma unroll
        for (int u = 0; u < U; ++u) accumulate<TIN, EPL>(acc, raw[u]);
      }
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

template <typename TIN, typename TOUT, int LPR, int U = kUnroll>
struct Uniform {
  static __device__ __forceinline__ int segment(KA a, int64_t t, int64_t b_lo, int64_t b_hi, int lane) {
    return pool_segment_fast<TIN, TOUT, LPR, true, true, U, LPR == 8>(a, t, b_lo, b_hi, lane);
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

// Bags [lA, lB) (global bag numbers, field-major; lA in field t), split at
// field ends.
template <typename P>
__device__ __forceinline__ int pool_bag_range(KA a, int64_t t, int64_t lA, int64_t lB, int lane) {
  int bad = 0;
  while (lA < lB) {
    const int64_t seg_end = min(lB, (t + 1) * a->B);
    bad |= P::segment(a, t, lA - t * a->B, seg_end - t * a->B, lane);
    lA = seg_end;
    ++t;
  }
  return bad;
}

// Rows [row_lo, row_hi) of a bag (of field t) shared with other waves:
// partial, then the arrival protocol.
template <typename P>
__device__ __forceinline__ int pool_partial(KA a, int64_t t, int64_t bag, int64_t row_lo, int64_t row_hi,
                                            int64_t slot, int64_t w_first, int lane) {
  const int bad = P::partial(a, t, bag - t * a->B, row_lo, row_hi, slot, lane);
  P::finish(a, w_first, bag, lane);
  return bad;
}

template <typename P>
__device__ __forceinline__ void wave_body(KA a) {
  const int lane = threadIdx.x & (kWaveSize - 1);
  int64_t blk = blockIdx.x;
  if (a->xcd_affine) blk = xcd_affine_block(blk, gridDim.x, a->xcd_affine);
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
  // the fields of the wave's first and last bags, both divisions here (the
  // divisor's reciprocal is then dead before the pooling loops, where it
  // would cost a register or a spill)
  const int64_t ta = __builtin_amdgcn_readfirstlane((int)(la / a->B));
  const int64_t tb = __builtin_amdgcn_readfirstlane((int)(lb / a->B));
  int bad = 0;
  if (la == lb && (head || tail)) {
    const int64_t slot = head ? 2 * w : 2 * w + 1;
    const int64_t w_first = head ? (int64_t)a->head_first[w] : w;
    bad |= pool_partial<P>(a, ta, la, (i0 - la_base) * C, (i1 - la_base) * C, slot, w_first, lane);
  } else {
    int64_t lA = la, lB = lb + 1, tA = ta;
    if (head) {
      bad |= pool_partial<P>(a, ta, la, (i0 - la_base) * C, INT64_MAX / 2, 2 * w, a->head_first[w], lane);
      lA = la + 1;
      tA += lA == (ta + 1) * a->B ? 1 : 0;
    }
    if (tail) lB = lb;
    bad |= pool_bag_range<P>(a, tA, lA, lB, lane);
    if (tail) bad |= pool_partial<P>(a, tb, lb, 0, (i1 - lb_base) * C, 2 * w + 1, w, lane);
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

// One-hot batches of a uniform row class (the plan's partition is not
// needed: each pooled row is the row itself).
template <typename TIN, typename TOUT, int LPR>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(5)))
void lookup_onehot_kernel(const LookupArgs args) {
  (void)args;
  constexpr int64_t kRowsPerWave = (int64_t)(kWaveSize / LPR) * kOneHotRows;
  const KA a = (KA)__builtin_amdgcn_kernarg_segment_ptr();
  const int lane = threadIdx.x & (kWaveSize - 1);
  const int64_t blk = a->xcd_affine ? xcd_affine_block(blockIdx.x, gridDim.x, a->xcd_affine) : (int64_t)blockIdx.x;
  const int64_t per_field = (a->B + kRowsPerWave - 1) / kRowsPerWave;
  const int64_t gw = blk * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
  if (gw >= per_field * a->T) return;
  if (*a->status & kStatusBadOffsets) return;
  const int64_t t = uni(gw / per_field);
  const TableInfo ti = table_info(a, t);
  const int bad = onehot_rows<TIN, TOUT, LPR>(a, ti, t, (gw - t * per_field) * kRowsPerWave, lane);
  if (__any(bad) && lane == 0)
    __hip_atomic_fetch_or(a->status, kStatusBadId, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// Bag-by-bag batches planned by their own launch (larger than the one-launch
// kernels of small.hip take): the plan validated the offsets and counted the
// bags longer than kDirectMaxItems chunks; with any such bag the launch uses
// the plan's partition instead (same kernel, wave_body), so one long bag
// never holds up a whole lookup.
// ---------------------------------------------------------------------------
// four waves per SIMD, as the mixed kernel it falls back to
template <typename TOUT>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(4)))
void lookup_direct_kernel(const LookupArgs args) {
  (void)args;
  const KA a = (KA)__builtin_amdgcn_kernarg_segment_ptr();
  const int lane = threadIdx.x & (kWaveSize - 1);
  const int64_t w = (int64_t)blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
  // the plan's verdicts, the field's info and the wave's bag offsets are all
  // requested before the first of them is needed (one round trip, not three):
  // the slot count comes from a kernel-argument dword (a scalar load), and
  // every lane loads offsets from a clamped, valid index, keeping only its
  // own (a load under a branch is waited for before the branch joins)
  const int32_t st_err = a->status[0], st_long = a->status[kStatusLongWord];
  const int64_t wpf = a->direct_wpf;
  const int64_t t = w < wpf * a->T ? uni(w / wpf) : 0;
  const int lpr_log = (int)((a->lpr_log[t >> 2] >> (8 * (t & 3))) & 7);
  const int jlog = min(6 - lpr_log - a->direct_plog, a->direct_jcap_log);
  const int64_t b0 = (w - t * wpf) << jlog;
  const bool mine = w < wpf * a->T && b0 < a->B;
  const int64_t bl = min(b0 + lane, a->B - 1);   // bags past the batch end are inactive
  DirectOffsets o{(int32_t)bl, (int32_t)bl + 1};
  if (a->offsets) {
    const int32_t* src = a->offsets + t * (a->B + 1) + bl;
    o.lo = src[0];
    o.hi = src[1];
  }
  if (!(mine && lane < (1 << jlog))) o = DirectOffsets{0, 0};
  const TableInfo ti = table_info(a, t);
  if (st_err & kStatusBadOffsets) return;   // the plan rejected the offsets
  if (st_long != 0) {                       // a long bag: the plan's partition
    wave_body<Mixed<TOUT>>(a);
    return;
  }
  if (!mine) return;
  const int bad = direct_wave<TOUT>(a, NativeIds{a->offsets, a->ids}, ti, t, b0, jlog, o, INT64_MAX, lane);
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
