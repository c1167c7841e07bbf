// Work planner for the fused multi-table lookup (gfx950).
//
// The paper observes that the whole embedding workload of an inference batch
// is known before it runs (§III, opportunity 2) and fuses every field's
// lookup into one pass whose output size is fixed in advance (§IV-B), with
// the work spread over threads afterwards (§IV-C).  This file computes that
// plan on the device from the per-field offsets, in two launches (one, both
// steps in a single block, when the batch fits one tile):
//   plan_reduce    per tile of bags: sum of item counts and costs, offset
//                  validation; tile 0 also writes the per-field table info,
//                  column bases and id bases, and resets the per-wave arrays.
//   plan_scan      per tile: its exclusive prefix (sum of the preceding tile
//                  sums), the per-bag exclusive prefixes of items and cost,
//                  and every wave boundary that falls in a bag's cost interval.
//
// Definitions (the contract checked bit-for-bit against the CPU plan):
//   bag (t, b) is number t*B + b (field-major); it holds L ids, has
//   n = max(1, ceil(L/C)) items, item j costs rows_j*row_bytes_t
//   + (j == 0) * out_bytes_t + K.  W = min(requested, N).  Wave w starts at
//   the first item whose cost prefix reaches ceil(w*S/W); unless the exact
//   flag is set, a start strictly inside a bag moves to the bag's end when
//   the bag's cost beyond the target is at most floor(S/(2W)).
// All target arithmetic is exact: comparisons of 128-bit products, with
// floating point used only for first guesses that are then corrected.
#include "dpi_internal.h"

namespace dpi {
namespace {

typedef unsigned __int128 u128;
// Kernel arguments are read in place from the constant kernarg segment
// (scalar loads); the per-field arrays are indexed at run time.
typedef const __attribute__((address_space(4))) PlanArgs* PA;
typedef const __attribute__((address_space(4))) PlanParams& PPR;
typedef const __attribute__((address_space(4))) PlanDev& PDR;

__device__ __forceinline__ u128 mul128(int64_t a, int64_t b) { return (u128)(uint64_t)a * (uint64_t)b; }

// smallest q >= 0 with q * den >= num (den > 0; the result fits int64)
__device__ __forceinline__ int64_t ceil_div128(u128 num, int64_t den) {
  int64_t q = (int64_t)((double)num / (double)den);
  if (q < 0) q = 0;
  while (q > 0 && mul128(q - 1, den) >= num) --q;
  while (mul128(q, den) < num) ++q;
  return q;
}

// field of bag l: floor(l / B), exact
__device__ __forceinline__ int64_t field_of(int64_t l, int64_t B, double inv_b) {
  int64_t t = (int64_t)((double)l * inv_b);
  while (t > 0 && t * B > l) --t;
  while ((t + 1) * B <= l) ++t;
  return t;
}

__device__ __forceinline__ int32_t packed_dim(uint32_t pk) { return (int32_t)(pk & 0x1ffffu); }
__device__ __forceinline__ int32_t packed_flags(uint32_t pk) { return (int32_t)(pk >> 17); }

struct BagCost {
  int64_t items;
  int64_t cost;
};

__device__ __forceinline__ BagCost bag_cost(int64_t L, PPR p, uint32_t pk) {
  const int64_t dim = packed_dim(pk);
  const int64_t row_bytes = dim * ((packed_flags(pk) & kTiF16) ? 2 : 4);
  const int64_t out_bytes = dim * (p.out_dtype == DPI_F16 ? 2 : 4);
  const uint32_t C = (uint32_t)p.C;
  int64_t n = (int64_t)(((uint32_t)L + C - 1u) / C);   // L < 2^31, C < 2^31
  if (n < 1) n = 1;
  // every item pays K; rows sum to L; the first item also pays the output row
  return BagCost{n, L * row_bytes + out_bytes + n * (int64_t)p.K};
}

// Length of bag (t, b) and whether its offsets are well formed.
__device__ __forceinline__ int64_t bag_length(PPR p, int64_t t, int64_t b, bool& bad) {
  if (!p.offsets) return 1;
  const int32_t* o = p.offsets + t * (p.B + 1);
  const int64_t lo = o[b], hi = o[b + 1];
  if ((b == 0 && lo != 0) || hi < lo) {
    bad = true;
    return 0;
  }
  return hi - lo;
}

// Block-wide exclusive scan of a pair of int64 values (kScanThreads threads).
__device__ __forceinline__ void block_scan_pair(int64_t a, int64_t b, int64_t& ea, int64_t& eb, int64_t& ta,
                                                int64_t& tb) {
  __shared__ int64_t wsum[2][kScanThreads / kWaveSize];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int64_t ia = a, ib = b;
  for (int d = 1; d < 64; d <<= 1) {
    const int64_t xa = __shfl_up(ia, d, 64);
    const int64_t xb = __shfl_up(ib, d, 64);
    if (lane >= d) {
      ia += xa;
      ib += xb;
    }
  }
  if (lane == 63) {
    wsum[0][wv] = ia;
    wsum[1][wv] = ib;
  }
  __syncthreads();
  int64_t pa = 0, pb = 0;
  ta = 0;
  tb = 0;
  for (int v = 0; v < kScanThreads / kWaveSize; ++v) {
    if (v < wv) {
      pa += wsum[0][v];
      pb += wsum[1][v];
    }
    ta += wsum[0][v];
    tb += wsum[1][v];
  }
  ea = pa + ia - a;
  eb = pb + ib - b;
  __syncthreads();
}

__device__ __forceinline__ int64_t block_sum_i64(int64_t v) {
  int64_t e, d0, tot, d1;
  block_scan_pair(v, 0, e, d0, tot, d1);
  return tot;
}

// ---------------------------------------------------------------------------
// Launch 1: tile sums, validation, field info, wave-array reset.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void plan_reduce_block(PA pa, int64_t blk, int64_t nblocks) {
  PPR p = pa->p;
  PDR d = pa->d;
  const int tid = threadIdx.x;
  const double inv_b = p.B > 0 ? 1.0 / (double)p.B : 0.0;

  for (int64_t w = blk * kScanThreads + tid; w < p.waves_req; w += nblocks * kScanThreads) {
    d.head_first[w] = -1;
    d.split_pieces[w] = 0;
    d.split_last[w] = -1;
    d.tickets[w] = 0;
  }

  bool bad = false;
  int64_t items = 0, cost = 0;
  const int64_t tile0 = blk * (int64_t)kScanThreads * p.slabs;
#pragma unroll
  for (int k = 0; k < kScanPerThread; ++k) {
    if (k >= p.slabs) break;
    const int64_t l = tile0 + (int64_t)k * kScanThreads + tid;   // coalesced over threads
    if (l < p.TB) {
      const int64_t t = field_of(l, p.B, inv_b);
      const int64_t L = bag_length(p, t, l - t * p.B, bad);
      const BagCost bc = bag_cost(L, p, pa->packed[t]);
      items += bc.items;
      cost += bc.cost;
    }
  }

  if (blk == 0) {
    // per-field info: dims -> column bases, id counts -> id bases
    int64_t dim = 0, nnz = 0;
    if (tid < p.T) {
      dim = packed_dim(pa->packed[tid]);
      nnz = p.offsets ? (int64_t)p.offsets[(int64_t)tid * (p.B + 1) + p.B] : p.B;
      if (nnz < 0) {
        bad = true;
        nnz = 0;
      }
    }
    int64_t col, idb, tot_d, tot_ids;
    block_scan_pair(dim, nnz, col, idb, tot_d, tot_ids);
    if (tid < p.T) {
      TableInfo ti;
      ti.num_rows = pa->num_rows[tid];
      ti.id_base = idb;
      ti.nnz = nnz;
      ti.dim = (int32_t)dim;
      ti.col_base = (int32_t)col;
      ti.flags = packed_flags(pa->packed[tid]);
      ti.row_bytes = (int32_t)dim * ((ti.flags & kTiF16) ? 2 : 4);
      ti.out_bytes = (int32_t)dim * (p.out_dtype == DPI_F16 ? 2 : 4);
      ti.pad = 0;
      d.tinfo[tid] = ti;
      d.col_base[tid] = col;
      d.id_base[tid] = idb;
    }
    if (tid == 0) {
      d.col_base[p.T] = tot_d;
      d.id_base[p.T] = tot_ids;
      if (tot_ids != p.total_ids) bad = true;
    }
    if (tid < 16) d.hdr[tid] = 0;
  }

  int64_t ea, eb, ta, tb;
  block_scan_pair(items, cost, ea, eb, ta, tb);
  const int64_t any_bad = block_sum_i64(bad ? 1 : 0);
  if (tid == 0) {
    d.block_sum[3 * blk] = ta;
    d.block_sum[3 * blk + 1] = tb;
    d.block_sum[3 * blk + 2] = any_bad;
  }
}

// ---------------------------------------------------------------------------
// Launch 2: prefixes and partition.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void plan_scan_block(PA pa, int64_t blk) {
  PPR p = pa->p;
  PDR d = pa->d;
  const int tid = threadIdx.x;
  const int64_t nblk = p.nblk;

  // this tile's exclusive prefix and the totals, from the tile sums
  int64_t pre_i = 0, pre_c = 0, tot_i = 0, tot_c = 0, err = 0;
#pragma unroll 4
  for (int64_t i = tid; i < nblk; i += kScanThreads) {
    const int64_t si = d.block_sum[3 * i], sc = d.block_sum[3 * i + 1];
    if (i < blk) {
      pre_i += si;
      pre_c += sc;
    }
    tot_i += si;
    tot_c += sc;
    err |= d.block_sum[3 * i + 2];
  }
  int64_t e0, e1, s0, s1;
  block_scan_pair(pre_i, pre_c, e0, e1, s0, s1);
  pre_i = s0;
  pre_c = s1;
  block_scan_pair(tot_i, tot_c, e0, e1, s0, s1);
  const int64_t N = s0, S = s1;
  err = block_sum_i64(err);
  const int64_t W = p.waves_req < N ? p.waves_req : N;

  if (blk == 0 && tid == 0) {
    // the split counter was zeroed by plan_reduce; other blocks add to it
    int64_t* h = d.hdr;
    h[kHdrAbi] = DPI_ABI_VERSION;
    h[kHdrT] = p.T;
    h[kHdrB] = p.B;
    h[kHdrW] = W;
    h[kHdrC] = p.C;
    h[kHdrK] = p.K;
    h[kHdrOutDtype] = p.out_dtype;
    h[kHdrFlags] = p.flags;
    h[kHdrTotalD] = p.total_d;
    h[kHdrItems] = N;
    h[kHdrCost] = S;
    h[kHdrTotalIds] = p.total_ids;
    h[kHdrWaveReq] = p.waves_req;
    d.bib[p.TB] = N;
    d.bcb[p.TB] = S;
    d.wib[0] = 0;
    d.wave_bag[0] = 0;
    // the only writer of the status word during planning; lookups latch later
    *d.status = err ? kStatusBadOffsets : 0;
  }
  if (p.TB == 0) return;

  // the tile's bags as p.slabs coalesced slabs, one after the other:
  // thread tid holds bag tile0 + k*kScanThreads + tid of slab k; its
  // exclusive prefix is the running total of the earlier slabs plus a block
  // scan within the slab
  const double inv_b = p.B > 0 ? 1.0 / (double)p.B : 0.0;
  const int64_t tile0 = blk * (int64_t)kScanThreads * p.slabs;
  const bool exact = (p.flags & DPI_FLAG_EXACT_SPLIT) != 0;
  const int64_t slack = W > 0 ? S / (2 * W) : 0;
  const double w_per_cost = W > 0 ? (double)W / (double)S : 0.0;
  // all slabs' bag costs first (their offset loads overlap), kept in LDS
  __shared__ int32_t s_items[kScanPerThread][kScanThreads];
  __shared__ int64_t s_cost[kScanPerThread][kScanThreads];
#pragma unroll
  for (int k = 0; k < kScanPerThread; ++k) {
    if (k >= p.slabs) break;
    const int64_t bag = tile0 + (int64_t)k * kScanThreads + tid;
    int64_t n = 0, bag_c = 0;
    if (bag < p.TB) {
      const int64_t t = field_of(bag, p.B, inv_b);
      bool ignored = false;   // validation was done by plan_reduce
      const BagCost bc = bag_cost(bag_length(p, t, bag - t * p.B, ignored), p, pa->packed[t]);
      n = bc.items;
      bag_c = bc.cost;
    }
    s_items[k][tid] = (int32_t)n;   // n <= max(1, L) < 2^31
    s_cost[k][tid] = bag_c;
  }
  int64_t run_i = pre_i, run_c = pre_c;
#pragma unroll 1
  for (int k = 0; k < p.slabs; ++k) {
    const int64_t bag = tile0 + (int64_t)k * kScanThreads + tid;
    const int64_t n = s_items[k][tid], bag_c = s_cost[k][tid];   // this thread's own entries
    int64_t xi, xc, si, sc;
    block_scan_pair(n, bag_c, xi, xc, si, sc);   // every thread takes part
    const int64_t ibase = run_i + xi;
    const int64_t E_lo = run_c + xc, E_hi = E_lo + bag_c;
    run_i += si;
    run_c += sc;
    if (bag >= p.TB) continue;
    d.bib[bag] = ibase;
    d.bcb[bag] = E_lo;
    if (W == 0) continue;

    // wave boundaries whose targets fall in this bag's cost interval: first
    // w >= 1 with w*S > E_lo*W, i.e. ceil(w*S/W) > E_lo; the double product
    // is a first guess corrected by exact 128-bit comparisons
    const u128 lo_w = mul128(E_lo, W), hi_w = mul128(E_hi, W);
    int64_t w = (int64_t)((double)E_lo * w_per_cost);
    if (w < 0) w = 0;
    while (w > 0 && mul128(w, S) > lo_w) --w;
    while (mul128(w, S) <= lo_w) ++w;
    if (w > W || mul128(w, S) > hi_w) continue;   // no target in this bag (the common case)
    const int64_t t = field_of(bag, p.B, inv_b);
    const uint32_t pk = pa->packed[t];
    const int64_t dim = packed_dim(pk);
    const int64_t row_bytes = dim * ((packed_flags(pk) & kTiF16) ? 2 : 4);
    const int64_t out_bytes = dim * (p.out_dtype == DPI_F16 ? 2 : 4);
    const int64_t per_item = (int64_t)p.C * row_bytes + p.K;
    int64_t w_first = -1, begin_prev = -1, pieces = 1, w_last = -1;
    for (; w <= W && mul128(w, S) <= hi_w; ++w) {
      const int64_t c = ceil_div128(mul128(w, S), W);   // ceil(w*S/W), in (E_lo, E_hi]
      // smallest j in [1, n] whose cost prefix reaches c
      const int64_t num = c - E_lo - out_bytes;
      int64_t j = num <= 0 ? 1 : ceil_div128((u128)(uint64_t)num, per_item);
      if (j < 1) j = 1;
      if (j > n - 1) j = n;
      bool inside = j < n;
      int64_t begin = ibase + j;
      if (inside && !exact && E_hi - c <= slack) {
        inside = false;
        begin = ibase + n;
      }
      d.wib[w] = begin;
      d.wave_bag[w] = inside ? bag : bag + 1;
      if (inside && w < W) {
        if (w_first < 0) w_first = w - 1;   // the wave holding the bag's first item
        d.head_first[w] = (int32_t)w_first;
        if (begin_prev >= 0 && begin_prev < begin) ++pieces;   // previous inside wave was nonempty
        begin_prev = begin;
        w_last = w;
      }
    }
    if (w_first >= 0) {
      ++pieces;   // the last inside wave always holds the bag's remaining items
      d.split_pieces[w_first] = (int32_t)pieces;
      d.split_last[w_first] = (int32_t)w_last;
      atomicAdd((unsigned long long*)&d.hdr[kHdrSplit], 1ull);
    }
  }
}

__global__ __launch_bounds__(kScanThreads) void plan_reduce_kernel(const PlanArgs args) {
  (void)args;
  plan_reduce_block((PA)__builtin_amdgcn_kernarg_segment_ptr(), blockIdx.x, gridDim.x);
}

__global__ __launch_bounds__(kScanThreads) void plan_scan_kernel(const PlanArgs args) {
  (void)args;
  plan_scan_block((PA)__builtin_amdgcn_kernarg_segment_ptr(), blockIdx.x);
}

// A batch of one tile: both steps in one block, one launch (the barrier makes
// the first step's global writes visible to the whole block).
__global__ __launch_bounds__(kScanThreads) void plan_single_kernel(const PlanArgs args) {
  (void)args;
  const PA pa = (PA)__builtin_amdgcn_kernarg_segment_ptr();
  plan_reduce_block(pa, 0, 1);
  __syncthreads();
  plan_scan_block(pa, 0);
}

}  // namespace

hipError_t launch_plan(const PlanArgs& a, hipStream_t s) {
  const unsigned blocks = (unsigned)(a.p.nblk > 0 ? a.p.nblk : 1);
  if (blocks == 1) {
    hipLaunchKernelGGL(plan_single_kernel, dim3(1), dim3(kScanThreads), 0, s, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(plan_reduce_kernel, dim3(blocks), dim3(kScanThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(plan_scan_kernel, dim3(blocks), dim3(kScanThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace dpi
