// One-launch lookups of small batches for gfx950.
//
// A small batch's lookup costs less than a launch (§I: for small inputs the
// launch overhead of a lookup operator exceeds its work), so for it the whole
// step -- the plan's checks and the fused gather-pool of every field (§IV-B)
// -- is one kernel, and dpi_plan enqueues nothing.  Two kernels:
//   * lookup_small_onehot_kernel: one-hot batches whose fields share one row
//     class; each pooled row is the row itself (field t's ids start at t*B).
//   * lookup_small_direct_kernel: bag-by-bag batches (every field on the
//     16-byte row path).  Every wave of field t reads all of the field's B+1
//     offsets (B <= kSmallMaxBatch) and every field's id count, so it derives
//     the field's first id (the exclusive prefix of the id counts, §IV-B's
//     flat id list) and checks the offsets itself: a first offset other than
//     zero, a decrease, a negative count or counts that do not add up to
//     total_ids latch DPI_ERR_BAD_OFFSETS and the wave writes nothing.  The
//     wave pools its own bags as the two-launch bag-by-bag kernel does, except
//     those of more than long_rows ids.  Those are cut along a grid of
//     long_rows-id windows of the batch's flat id list into pieces; every wave
//     of the field counts the same pieces in the same order and takes pieces
//     i, i + wpf, ... (i its rank in the field), pools each with all its slots
//     into an fp32 partial, and the last of a bag's pieces to arrive adds the
//     partials in piece order and writes the row (deterministic, as for bags
//     split between waves by the plan).
// Status word and long-bag tickets carry the plan's id in their high bits: a
// word holding another id counts as clear, so no launch resets them, and the
// last arrival of a bag clears its ticket for the next lookup of the plan.
#include "gather.h"
#include "wave_scan.h"

namespace dpi {
namespace {

typedef const __attribute__((address_space(4))) SmallArgs* KS;

constexpr int kScanMax = (int)(kSmallMaxBatch / kWaveSize);   // bags per lane in a field's scan

// Field t's static info from the kernel arguments; its first id and id count
// come from the caller.
__device__ __forceinline__ TableInfo small_info(KS a, int64_t t, int64_t id_base, int64_t nnz) {
  const uint32_t pk = a->packed[t];
  const int32_t dim = (int32_t)(pk & 0x1ffffu);
  const int32_t flags = (int32_t)(pk >> 17);
  TableInfo u;
  u.num_rows = a->nrows[t];
  u.id_base = uni(id_base);
  u.nnz = uni(nnz);
  u.dim = dim;
  u.col_base = a->col_base[t];
  u.row_bytes = dim * ((flags & kTiF16) ? 2 : 4);
  u.out_bytes = dim * (a->out_f16 ? 2 : 4);
  u.flags = flags;
  u.pad = 0;
  return u;
}

// OR error bits into the plan's status word (one lane).  A word tagged with
// another plan's id is replaced.  Each failed exchange means another lane's
// succeeded, so the loop ends.
__device__ void latch(KS a, uint32_t bits) {
  uint64_t* const w = a->status;
  const uint64_t tag = (uint64_t)a->tag;
  uint64_t old = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (;;) {
    const uint64_t base = (old >> kStatusTagShift) == tag ? old : (tag << kStatusTagShift);
    const uint64_t nv = base | bits;
    if (nv == old) return;
    if (__hip_atomic_compare_exchange_strong(w, &old, nv, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      return;
  }
}

// Count one arrival on a long bag's ticket (one lane); returns the arrivals
// so far, this one included.  A ticket tagged with another plan's id counts
// as zero.
__device__ int64_t ticket_arrive(uint64_t* tk, int64_t tag) {
  const uint64_t tg = (uint64_t)tag << kStatusTagShift;
  uint64_t old = __hip_atomic_load(tk, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (;;) {
    const uint64_t n = (old & ~kStatusBitsMask) == tg ? (old & kStatusBitsMask) : 0;
    if (__hip_atomic_compare_exchange_strong(tk, &old, tg | (n + 1), __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      return (int64_t)(n + 1);
  }
}

// Pieces of a long bag occupying flat ids [gs, ge): the windows of pr ids it
// meets.
__device__ __forceinline__ int64_t piece_count(int64_t gs, int64_t ge, int64_t pr) {
  return (ge - 1) / pr - gs / pr + 1;
}

// Rows [r0, r1) of field t (positions in the field's id list) pooled by the
// whole wave; the lanes of slot 0 write the fp32 sums of their columns to dst.
template <typename TIN, int LPR, bool BUF, typename S>
__device__ __forceinline__ int piece_fast(KS a, const S& src, const TableInfo& ti, int64_t t, int64_t r0, int64_t r1,
                                          float* dst, int lane) {
  constexpr int EPL = In<TIN>::EPL;
  float acc[EPL];
  int bad = 0;
  pool_rows_src<TIN, LPR, BUF>(a, src, ti, t, r0, r1, lane, acc, bad);
  const int g = lane / LPR, k = lane % LPR;
  if (g == 0 && k * EPL < ti.dim) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) dst[k * EPL + i] = acc[i];
  }
  return bad;
}

template <typename S>
__device__ __forceinline__ int piece_wave(KS a, const S& src, const TableInfo& ti, int64_t t, int64_t r0, int64_t r1,
                                          float* dst, int lane) {
  const bool buf = use_buffer(ti), f16 = (ti.flags & kTiF16) != 0;
  switch ((ti.flags >> kTiLprShift) & 7) {
#define DPI_CASE(L, LPR)                                                                     \
  case L:                                                                                    \
    if (f16)                                                                                 \
      return buf ? piece_fast<_Float16, LPR, true>(a, src, ti, t, r0, r1, dst, lane)         \
                 : piece_fast<_Float16, LPR, false>(a, src, ti, t, r0, r1, dst, lane);       \
    return buf ? piece_fast<float, LPR, true>(a, src, ti, t, r0, r1, dst, lane)              \
               : piece_fast<float, LPR, false>(a, src, ti, t, r0, r1, dst, lane);
    DPI_FOR_LPR(DPI_CASE)
#undef DPI_CASE
    default:
      return 0;
  }
}

// Piece q of field t's long bags.  Lane l's bags [first, first + nb) hold
// pieces [pre, pre + cnt) of the field (in bag order, each bag's pieces in
// window order).  Out of line: the rare path keeps its registers to itself.
template <typename TOUT, typename S>
__device__ __attribute__((noinline)) int long_piece(KS a, const S& src, const TableInfo& ti, int64_t t, int64_t q,
                                                    int64_t pre, int64_t cnt, int64_t first, int64_t nb, int lane) {
  const int64_t pr = a->long_rows;
  const uint64_t m = __ballot(cnt > 0 && pre <= q && q < pre + cnt);
  if (m == 0) return 0;   // q < the field's piece count, so some lane holds it
  const int owner = __builtin_ctzll(m);
  int64_t bag = 0, rank = 0, lo = 0, hi = 0;
  if (lane == owner) {
    // the owner's offsets again (one round trip), then a walk in registers
    const int64_t row = t * (a->B + 1) + first;
    int32_t u[kScanMax + 1];
#pragma unroll
    for (int j = 0; j <= kScanMax; ++j) u[j] = src.offset(row + min((int64_t)j, nb));
    int64_t r = q - pre;
    bool found = false;
#pragma unroll
    for (int j = 0; j < kScanMax; ++j) {
      const int64_t l0 = u[j], l1 = u[j + 1];
      if (!found && j < nb && l1 - l0 > pr) {
        const int64_t n = piece_count(ti.id_base + l0, ti.id_base + l1, pr);
        if (r < n) {
          found = true;
          bag = first + j;
          rank = r;
          lo = l0;
          hi = l1;
        } else {
          r -= n;
        }
      }
    }
  }
  bag = uni(__shfl(bag, owner, kWaveSize));
  rank = uni(__shfl(rank, owner, kWaveSize));
  lo = uni(__shfl(lo, owner, kWaveSize));
  hi = uni(__shfl(hi, owner, kWaveSize));
  if (hi - lo <= pr) return 0;   // offsets changed under the lookup
  const int64_t gs = ti.id_base + lo, ge = ti.id_base + hi;
  const int64_t wf = gs / pr;
  const int64_t n = (ge - 1) / pr - wf + 1;
  const int64_t win = wf + rank;
  // a window meets at most two long bags: the one covering its start (a piece
  // of rank > 0, slot 2 * win) and one starting inside it (rank 0, slot
  // 2 * win + 1), which reaches past the window's end
  const int64_t slot = 2 * win + (rank == 0 ? 1 : 0);
  const int64_t head = 2 * wf + 1;
  if (2 * (wf + n - 1) >= a->slots) return 0;   // not for offsets that passed the checks
  const int64_t r0 = (gs > win * pr ? gs : win * pr) - ti.id_base;
  const int64_t r1 = (ge < (win + 1) * pr ? ge : (win + 1) * pr) - ti.id_base;
  const int bad = piece_wave(a, src, ti, t, r0, r1, a->partial + slot * a->dmax, lane);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  int64_t arrived = 0;
  if (lane == 0) arrived = ticket_arrive(a->tickets + head, a->tag);
  arrived = __shfl(arrived, 0, kWaveSize);
  if (arrived != n) return bad;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  // the last piece to arrive: the pieces' sums in window order
  const bool mean = is_mean(a, t);
  const float fl = (float)(ge - gs);
  TOUT* const dst = out_row<TOUT>(a, ti, bag);
  for (int64_t c = lane; c < ti.dim; c += kWaveSize) {
    float sum = a->partial[head * a->dmax + c];
    for (int64_t k = 1; k < n; ++k) sum += a->partial[2 * (wf + k) * a->dmax + c];
    if (mean) sum = sum / fl;
    dst[c] = (TOUT)sum;
  }
  if (lane == 0)
    __hip_atomic_store(a->tickets + head, (uint64_t)a->tag << kStatusTagShift, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  return bad;
}

// Field t's converted offsets [row, row + B] (a staged input; B <=
// kSmallMaxBatch): every load first, then every store (one round trip).
template <typename S>
__device__ __forceinline__ void write_offsets(const S& src, int64_t row, int64_t B, int lane) {
  int32_t v[kScanMax + 1];
#pragma unroll
  for (int j = 0; j <= kScanMax; ++j) v[j] = src.offset(row + min((int64_t)lane + j * kWaveSize, B));
#pragma unroll
  for (int j = 0; j <= kScanMax; ++j)
    if (lane + j * kWaveSize <= B) src.put_offset(row + lane + j * kWaveSize, v[j]);
}

// Converted ids [r_lo, r_hi) of the flat id list, 8 per lane per round trip.
template <typename S>
__device__ __forceinline__ void write_ids(const S& src, int64_t r_lo, int64_t r_hi, int lane) {
  constexpr int kPer = 8;
  for (int64_t r0 = r_lo; r0 < r_hi; r0 += (int64_t)kPer * kWaveSize) {
    int32_t v[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) v[u] = src.id(min(r0 + lane + u * kWaveSize, r_hi - 1));
#pragma unroll
    for (int u = 0; u < kPer; ++u)
      if (r0 + lane + u * kWaveSize < r_hi) src.put_id(r0 + lane + u * kWaveSize, v[u]);
  }
}

// The bag-by-bag lookup, the offsets and ids read from `src`.
template <typename TOUT, typename S>
__device__ __forceinline__ void small_direct(KS a, const S& src, bool has_offsets) {
  const int lane = threadIdx.x & (kWaveSize - 1);
  const int64_t w = (int64_t)blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
  const int64_t wpf = a->direct_wpf;
  const int32_t T = a->T;
  if (w >= wpf * T) return;
  // grids hold fewer than 2^31 waves: a 32-bit division
  const int64_t t = uni((int32_t)((uint32_t)w / (uint32_t)wpf));
  const int64_t i = w - t * wpf;   // the wave's rank among the field's waves
  const int lpr_log = (int)((a->packed[t] >> (17 + kTiLprShift)) & 7);
  const int jlog = min(6 - lpr_log - a->direct_plog, a->direct_jcap_log);
  const int64_t B = a->B;
  const int64_t b0 = i << jlog;
  const bool mine = b0 < B;
  int bad = 0;
  DirectOffsets o{0, 0};
  if (!has_offsets) {
    if (mine && lane < (1 << jlog)) {
      const int64_t bl = min(b0 + lane, B - 1);   // bags past the batch end are inactive
      o.lo = (int32_t)bl;
      o.hi = (int32_t)bl + 1;
    }
    if (mine) {
      const TableInfo ti = small_info(a, t, t * B, B);
      bad = direct_wave<TOUT>(a, src, ti, t, b0, jlog, o, INT64_MAX, lane);
    }
  } else {
    // the wave's bag offsets, every field's id count and all of this field's
    // offsets (lane l: bags [l * bpl, l * bpl + bpl)), requested together:
    // every lane loads from a clamped, valid index and the values it does not
    // need are dropped afterwards (a load under a branch makes the compiler
    // wait for it before the branch joins, one round trip per branch)
    const int64_t row = t * (B + 1);
    const int64_t bl = min(b0 + lane, B - 1);
    const int32_t lo = src.offset(row + bl), hi = src.offset(row + bl + 1);
    const int32_t nz = src.offset((int64_t)min(lane, T - 1) * (B + 1) + B);
    const int64_t bpl = (B + kWaveSize - 1) / kWaveSize;
    const int64_t first = lane * bpl;
    int32_t v[kScanMax + 1];
#pragma unroll
    for (int j = 0; j <= kScanMax; ++j) {
      v[j] = 0;
      if (j <= bpl) v[j] = src.offset(row + min(first + j, B));   // bpl is the same for the whole wave
    }
    if (mine && lane < (1 << jlog)) {
      o.lo = lo;
      o.hi = hi;
    }
    const int64_t nnz_l = lane < T ? (int64_t)nz : 0;
    // the field's first id and id count (one DPP scan of the counts); the
    // counts must add up to total_ids.  The checks are branch-free up to the
    // first exit, so that no load above is moved below a branch.
    const int64_t incl = wave_incl_scan(nnz_l, lane);
    const int64_t total = lane_value(incl, kWaveSize - 1);
    const int64_t nnz = lane_value(nnz_l, (int)t);
    const int64_t id_base = lane_value(incl, (int)t) - nnz;
    const int64_t pr = a->long_rows;
    const int64_t nb = max((int64_t)0, min(bpl, B - first));   // the lane's bags
    int badf = (lane == 0 && v[0] != 0) | (o.hi < o.lo);
    int haslong = 0;
#pragma unroll
    for (int j = 0; j < kScanMax; ++j) {   // v[j], v[j + 1]: the lane's own offsets for j < nb
      const int in = j < nb;
      badf |= in & (v[j + 1] < v[j]);
      haslong |= in & ((int64_t)v[j + 1] - v[j] > pr);
    }
    // one exit for both verdicts (no short circuit): a bad count or total is
    // latched by the grid's first wave, a bad field by the field's first
    const int gbad = __any(nnz_l < 0) | (int)(total != a->total_ids);
    const int fbad = __any(badf);
    if (gbad | fbad) {
      if (S::kWrites && i == 0) write_offsets(src, row, B, lane);
      if ((gbad ? w : i) == 0 && lane == 0) latch(a, kStatusBadOffsets);
      return;
    }
    // pieces of the lane's long bags (rare: a 64-bit division each)
    int64_t cnt = 0;
    if (__any(haslong)) {
#pragma unroll
      for (int j = 0; j < kScanMax; ++j) {
        if (j < nb && (int64_t)v[j + 1] - v[j] > pr) cnt += piece_count(id_base + v[j], id_base + v[j + 1], pr);
      }
    }
    const int64_t pre = wave_incl_scan(cnt, lane) - cnt;
    const int64_t pieces = lane_value(pre + cnt, kWaveSize - 1);
    const TableInfo ti = small_info(a, t, id_base, nnz);
    if (mine) bad = direct_wave<TOUT>(a, src, ti, t, b0, jlog, o, pr, lane);
    for (int64_t q = i; q < pieces; q += wpf)
      bad |= long_piece<TOUT>(a, src, ti, t, q, pre, cnt, first, nb, lane);
    if (S::kWrites) {
      // the converted arrays, after the pooling: the field's offsets by its
      // first wave, the ids of the wave's own bags (long ones included) by
      // the wave
      if (i == 0) write_offsets(src, row, B, lane);
      if (mine) {
        const int64_t nbags = min((int64_t)1 << jlog, B - b0);
        const int64_t r_lo = min(max((int64_t)__shfl(o.lo, 0, kWaveSize), (int64_t)0), nnz);
        const int64_t r_hi = min(max((int64_t)__shfl(o.hi, (int)nbags - 1, kWaveSize), r_lo), nnz);
        write_ids(src, id_base + r_lo, id_base + r_hi, lane);
      }
    }
  }
  if (__any(bad) && lane == 0) latch(a, kStatusBadId);
}

// four waves per SIMD, as the two-launch bag-by-bag kernel
template <typename TOUT>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(4)))
void lookup_small_direct_kernel(const SmallArgs args) {
  (void)args;
  const KS a = (KS)__builtin_amdgcn_kernarg_segment_ptr();
  small_direct<TOUT>(a, NativeIds{a->offsets, a->ids}, a->offsets != nullptr);
}

// The same from a staged packed CSR of element type TX (dpi_lookup_csr): the
// input conversion of dpi_stage_csr happens as the lookup reads its input.
template <typename TOUT, typename TX>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(4)))
void lookup_small_staged_kernel(const SmallArgs args) {
  (void)args;
  const KS a = (KS)__builtin_amdgcn_kernarg_segment_ptr();
  const TX* raw = reinterpret_cast<const TX*>(a->staged);
  small_direct<TOUT>(a, StagedIds<TX>{raw, raw + (int64_t)a->T * (a->B + 1), a->offsets_out, a->ids_out}, true);
}

// one-hot batches of one row class
template <typename TIN, typename TOUT, int LPR>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(5)))
void lookup_small_onehot_kernel(const SmallArgs args) {
  (void)args;
  constexpr int64_t kRowsPerWave = (int64_t)(kWaveSize / LPR) * kOneHotRows;
  const KS a = (KS)__builtin_amdgcn_kernarg_segment_ptr();
  const int lane = threadIdx.x & (kWaveSize - 1);
  const int64_t blk = a->xcd_affine ? xcd_affine_block(blockIdx.x, gridDim.x, a->xcd_affine) : (int64_t)blockIdx.x;
  const int64_t per_field = (a->B + kRowsPerWave - 1) / kRowsPerWave;
  const int64_t gw = blk * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
  if (gw >= per_field * a->T) return;
  const int64_t t = uni(gw / per_field);
  const TableInfo ti = small_info(a, t, t * a->B, a->B);
  const int bad = onehot_rows<TIN, TOUT, LPR>(a, ti, t, (gw - t * per_field) * kRowsPerWave, lane);
  if (__any(bad) && lane == 0) latch(a, kStatusBadId);
}

__global__ void status_out_kernel(const uint64_t* word, int64_t tag, int32_t* dst) {
  if (threadIdx.x == 0) {
    const uint64_t v = *word;
    *dst = (v >> kStatusTagShift) == (uint64_t)tag ? (int32_t)(v & kStatusBitsMask) : 0;
  }
}

}  // namespace

hipError_t launch_lookup_small(const SmallArgs& a, hipStream_t s) {
  if (!a.offsets && a.uniform_class >= 0) {
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
      hipLaunchKernelGGL((lookup_small_onehot_kernel<_Float16, _Float16, LPR>), grid, block, 0, s, a); \
    else if (f16)                                                                                      \
      hipLaunchKernelGGL((lookup_small_onehot_kernel<_Float16, float, LPR>), grid, block, 0, s, a);    \
    else if (a.out_f16)                                                                                \
      hipLaunchKernelGGL((lookup_small_onehot_kernel<float, _Float16, LPR>), grid, block, 0, s, a);    \
    else                                                                                               \
      hipLaunchKernelGGL((lookup_small_onehot_kernel<float, float, LPR>), grid, block, 0, s, a);       \
    break;
      DPI_FOR_LPR(DPI_CASE)
#undef DPI_CASE
      default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  const int64_t waves = a.direct_wpf * a.T;
  const int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
  if (blocks <= 0) return hipSuccess;
  const dim3 grid((unsigned)blocks), block(kBlockThreads);
  if (a.staged) {
#define DPI_STAGED(TX)                                                                                 \
  if (a.out_f16)                                                                                       \
    hipLaunchKernelGGL((lookup_small_staged_kernel<_Float16, TX>), grid, block, 0, s, a);              \
  else                                                                                                 \
    hipLaunchKernelGGL((lookup_small_staged_kernel<float, TX>), grid, block, 0, s, a);
    switch (a.staged_dtype) {
      case DPI_X_F32: DPI_STAGED(float) break;
      case DPI_X_I64: DPI_STAGED(int64_t) break;
      case DPI_X_I32: DPI_STAGED(int32_t) break;
      default: return hipErrorInvalidValue;
    }
#undef DPI_STAGED
    return hipGetLastError();
  }
  if (a.out_f16)
    hipLaunchKernelGGL(lookup_small_direct_kernel<_Float16>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(lookup_small_direct_kernel<float>, grid, block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_status_out(const uint64_t* word, int64_t tag, int32_t* dst, hipStream_t s) {
  hipLaunchKernelGGL(status_out_kernel, dim3(1), dim3(kWaveSize), 0, s, word, tag, dst);
  return hipGetLastError();
}

}  // namespace dpi
