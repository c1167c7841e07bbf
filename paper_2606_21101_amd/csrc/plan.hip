// Work planner for the fused multi-table lookup (gfx950).
//
// The paper observes that the whole embedding workload of an inference batch
// is known before it runs (§III, opportunity 2) and fuses every field's
// lookup into one pass whose output size is fixed in advance (§IV-B), with
// the work spread over threads afterwards (§IV-C).  This file computes that
// plan on the device from the per-field offsets:
//   1. field metadata (dims, row/output bytes, column bases)     plan_meta
//   2. per scan tile: sum of item counts and costs of its bags    plan_reduce
//   3. exclusive prefix of the tiles, per-field id bases, totals  plan_totals
//   4. per bag: exclusive prefixes of items and cost, and the
//      wave boundaries that fall in the bag's cost interval       plan_scan_partition
//
// Definitions (also the contract checked bit-for-bit against the CPU plan):
//   bag (t, b) is number t*B + b (field-major); it holds L ids, has
//   n = max(1, ceil(L/C)) items, item j costs rows_j*row_bytes_t
//   + (j == 0) * out_bytes_t + K.  W = min(requested, N).  Wave w starts at
//   the first item whose cost prefix reaches ceil(w*S/W); unless the exact
//   flag is set, a start strictly inside a bag moves to the bag's end when
//   the bag's cost beyond the target is at most floor(S/(2W)).
#include "dpi_internal.h"

namespace dpi {
namespace {

typedef unsigned __int128 u128;

__device__ __forceinline__ int64_t ceil_div_mul(int64_t w, int64_t S, int64_t W) {
  // ceil(w * S / W) with a 128-bit intermediate
  const u128 num = (u128)(uint64_t)w * (uint64_t)S;
  return (int64_t)((num + (uint64_t)W - 1) / (uint64_t)W);
}

__device__ __forceinline__ void latch_status(int32_t* status, int bits) {
  __hip_atomic_fetch_or(status, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Length of bag (t, b); validates the offsets it reads.
__device__ __forceinline__ int64_t bag_length(const int32_t* offsets, int64_t B, int64_t t, int64_t b,
                                              int32_t* status) {
  if (!offsets) return 1;
  const int32_t* o = offsets + t * (B + 1);
  const int64_t lo = o[b], hi = o[b + 1];
  if ((b == 0 && lo != 0) || hi < lo) {
    latch_status(status, kStatusBadOffsets);
    return 0;
  }
  return hi - lo;
}

struct BagCost {
  int64_t items;
  int64_t cost;
};

__device__ __forceinline__ BagCost bag_cost(int64_t L, int64_t C, int64_t K, int64_t row_bytes,
                                            int64_t out_bytes) {
  int64_t n = (L + C - 1) / C;
  if (n < 1) n = 1;
  // every item pays K; rows sum to L; the first item also pays the output row
  return BagCost{n, L * row_bytes + out_bytes + n * K};
}

// Block-wide exclusive scan of a pair of int64 values (256 threads = 4 waves).
__device__ __forceinline__ void block_scan_pair(int64_t a, int64_t b, int64_t& ea, int64_t& eb,
                                                int64_t& ta, int64_t& tb) {
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

__global__ void plan_meta_kernel(const MetaChunk chunk, int first, int count, PlanDev d,
                                 int clear_status, int osize) {
  const int i = threadIdx.x;
  if (clear_status && i == 0) *d.status = 0;
  if (i >= count) return;
  TableInfo ti;
  ti.num_rows = chunk.num_rows[i];
  ti.id_base = 0;
  ti.nnz = 0;
  ti.dim = chunk.dim[i];
  ti.col_base = chunk.col_base[i];
  ti.row_bytes = chunk.dim[i] * ((chunk.flags[i] & kTiF16) ? 2 : 4);
  ti.out_bytes = chunk.dim[i] * osize;
  ti.flags = chunk.flags[i];
  ti.pad = 0;
  d.tinfo[first + i] = ti;
  d.col_base[first + i] = chunk.col_base[i];
}

// Tile sums of (items, cost); also resets the per-wave arrays.
__global__ __launch_bounds__(kScanThreads) void plan_reduce_kernel(const PlanParams p, PlanDev d) {
  const int64_t tid = threadIdx.x;
  const int64_t blk = blockIdx.x;
  // per-wave arrays for the coming partition
  for (int64_t w = blk * kScanThreads + tid; w < p.waves_req; w += (int64_t)gridDim.x * kScanThreads) {
    d.head_first[w] = -1;
    d.split_pieces[w] = 0;
    d.split_last[w] = -1;
    d.tickets[w] = 0;
  }
  const int64_t first = blk * kScanTile + tid * kScanPerThread;
  int64_t items = 0, cost = 0;
  if (first < p.TB) {
    int64_t t = first / p.B, b = first - t * p.B;
    const int64_t last = min(first + kScanPerThread, p.TB);
    for (int64_t bag = first; bag < last; ++bag) {
      const TableInfo& ti = d.tinfo[t];
      const int64_t L = bag_length(p.offsets, p.B, t, b, d.status);
      const BagCost bc = bag_cost(L, p.C, p.K, ti.row_bytes, ti.out_bytes);
      items += bc.items;
      cost += bc.cost;
      if (++b == p.B) {
        b = 0;
        ++t;
      }
    }
  }
  int64_t ea, eb, ta, tb;
  block_scan_pair(items, cost, ea, eb, ta, tb);
  if (tid == 0) {
    d.block_sum[2 * blk] = ta;
    d.block_sum[2 * blk + 1] = tb;
  }
}

// One block: prefix of the tile sums, per-field id bases, header.
__global__ __launch_bounds__(kScanThreads) void plan_totals_kernel(const PlanParams p, PlanDev d) {
  const int tid = threadIdx.x;
  __shared__ int64_t carry[2];
  if (tid == 0) {
    carry[0] = 0;
    carry[1] = 0;
  }
  __syncthreads();
  for (int64_t base = 0; base < p.nblk; base += kScanThreads) {
    const int64_t i = base + tid;
    const int64_t a = i < p.nblk ? d.block_sum[2 * i] : 0;
    const int64_t b = i < p.nblk ? d.block_sum[2 * i + 1] : 0;
    int64_t ea, eb, ta, tb;
    block_scan_pair(a, b, ea, eb, ta, tb);
    if (i < p.nblk) {
      d.block_pre[2 * i] = carry[0] + ea;
      d.block_pre[2 * i + 1] = carry[1] + eb;
    }
    __syncthreads();
    if (tid == 0) {
      carry[0] += ta;
      carry[1] += tb;
    }
    __syncthreads();
  }
  const int64_t N = carry[0], S = carry[1];

  // per-field id bases (T <= DPI_MAX_TABLES = 256 = one value per thread)
  int64_t nnz = 0;
  if (tid < p.T) {
    nnz = p.offsets ? (int64_t)p.offsets[(int64_t)tid * (p.B + 1) + p.B] : p.B;
    if (nnz < 0) {
      latch_status(d.status, kStatusBadOffsets);
      nnz = 0;
    }
  }
  int64_t ebase, dummy, total, dummy2;
  block_scan_pair(nnz, 0, ebase, dummy, total, dummy2);
  if (tid < p.T) {
    d.id_base[tid] = ebase;
    d.tinfo[tid].id_base = ebase;
    d.tinfo[tid].nnz = nnz;
  }
  if (tid == 0) {
    d.id_base[p.T] = total;
    d.col_base[p.T] = p.total_d;
    if (total != p.total_ids) latch_status(d.status, kStatusBadOffsets);
    const int64_t W = p.waves_req < N ? p.waves_req : N;
    int64_t* h = d.hdr;
    for (int k = 0; k < 16; ++k) h[k] = 0;
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
    h[kHdrSplit] = 0;
    h[kHdrWaveReq] = p.waves_req;
    d.bib[p.TB] = N;
    d.bcb[p.TB] = S;
    d.wib[0] = 0;
    d.wave_bag[0] = 0;
  }
}

// Per bag: exclusive prefixes, then the wave starts whose targets fall in the
// bag's cost interval (E_lo, E_hi].
__global__ __launch_bounds__(kScanThreads) void plan_scan_partition_kernel(const PlanParams p, PlanDev d) {
  const int64_t tid = threadIdx.x;
  const int64_t blk = blockIdx.x;
  const int64_t first = blk * kScanTile + tid * kScanPerThread;
  const int64_t last = first < p.TB ? min(first + kScanPerThread, p.TB) : first;
  int64_t t0 = 0, b0 = 0;
  int64_t items = 0, cost = 0;
  if (first < p.TB) {
    t0 = first / p.B;
    b0 = first - t0 * p.B;
    int64_t t = t0, b = b0;
    for (int64_t bag = first; bag < last; ++bag) {
      const TableInfo& ti = d.tinfo[t];
      // validation already latched by plan_reduce; lengths recomputed quietly
      int64_t L = 1;
      if (p.offsets) {
        const int32_t* o = p.offsets + t * (p.B + 1);
        L = (int64_t)o[b + 1] - o[b];
        if (L < 0) L = 0;
      }
      const BagCost bc = bag_cost(L, p.C, p.K, ti.row_bytes, ti.out_bytes);
      items += bc.items;
      cost += bc.cost;
      if (++b == p.B) {
        b = 0;
        ++t;
      }
    }
  }
  int64_t ea, eb, ta, tb;
  block_scan_pair(items, cost, ea, eb, ta, tb);
  if (first >= p.TB) return;

  const int64_t W = d.hdr[kHdrW];
  const int64_t S = d.hdr[kHdrCost];
  const bool exact = (p.flags & DPI_FLAG_EXACT_SPLIT) != 0;
  const int64_t slack = W > 0 ? S / (2 * W) : 0;
  int64_t ib = d.block_pre[2 * blk] + ea;
  int64_t cb = d.block_pre[2 * blk + 1] + eb;
  int64_t t = t0, b = b0;
  for (int64_t bag = first; bag < last; ++bag) {
    const TableInfo& ti = d.tinfo[t];
    int64_t L = 1;
    if (p.offsets) {
      const int32_t* o = p.offsets + t * (p.B + 1);
      L = (int64_t)o[b + 1] - o[b];
      if (L < 0) L = 0;
    }
    const BagCost bc = bag_cost(L, p.C, p.K, ti.row_bytes, ti.out_bytes);
    d.bib[bag] = ib;
    d.bcb[bag] = cb;
    const int64_t E_lo = cb, E_hi = cb + bc.cost;
    if (W > 0) {
      // first w >= 1 with ceil(w*S/W) > E_lo
      int64_t w = (int64_t)(((u128)(uint64_t)E_lo * (uint64_t)W) / (uint64_t)S) + 1;
      const int64_t per_item = (int64_t)p.C * ti.row_bytes + p.K;
      int64_t w_first = -1, w_prev = -1, begin_prev = -1, pieces = 1, w_last = -1;
      for (; w <= W; ++w) {
        const int64_t c = ceil_div_mul(w, S, W);
        if (c > E_hi) break;
        // smallest j in [1, n] whose cost prefix reaches c
        const int64_t num = c - E_lo - ti.out_bytes;
        int64_t j = num <= 0 ? 1 : (num + per_item - 1) / per_item;
        if (j < 1) j = 1;
        if (j > bc.items - 1) j = bc.items;
        bool inside = j < bc.items;
        int64_t begin = ib + j;
        if (inside && !exact && E_hi - c <= slack) {
          inside = false;
          begin = ib + bc.items;
        }
        d.wib[w] = begin;
        d.wave_bag[w] = inside ? bag : bag + 1;
        if (inside && w < W) {
          if (w_first < 0) w_first = w - 1;   // the wave holding the bag's first item
          d.head_first[w] = (int32_t)w_first;
          if (w_prev >= 0 && begin_prev < begin) ++pieces;   // previous inside wave was nonempty
          w_prev = w;
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
    ib += bc.items;
    cb += bc.cost;
    if (++b == p.B) {
      b = 0;
      ++t;
    }
  }
}

}  // namespace

hipError_t launch_plan_meta(const MetaChunk& chunk, int first, int count, const PlanDev& d,
                            bool clear_status, int osize, hipStream_t s) {
  hipLaunchKernelGGL(plan_meta_kernel, dim3(1), dim3(kMetaChunk), 0, s, chunk, first, count, d,
                     clear_status ? 1 : 0, osize);
  return hipGetLastError();
}

hipError_t launch_plan_reduce(const PlanParams& p, const PlanDev& d, hipStream_t s) {
  hipLaunchKernelGGL(plan_reduce_kernel, dim3(p.nblk), dim3(kScanThreads), 0, s, p, d);
  return hipGetLastError();
}

hipError_t launch_plan_totals(const PlanParams& p, const PlanDev& d, hipStream_t s) {
  hipLaunchKernelGGL(plan_totals_kernel, dim3(1), dim3(kScanThreads), 0, s, p, d);
  return hipGetLastError();
}

hipError_t launch_plan_scan_partition(const PlanParams& p, const PlanDev& d, hipStream_t s) {
  hipLaunchKernelGGL(plan_scan_partition_kernel, dim3(p.nblk), dim3(kScanThreads), 0, s, p, d);
  return hipGetLastError();
}

}  // namespace dpi
