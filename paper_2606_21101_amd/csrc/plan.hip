// Work planner for the fused multi-table lookup (gfx950).
//
// The paper observes that the whole embedding workload of an inference batch
// is known before it runs (§III, opportunity 2) and fuses every field's
// lookup into one pass whose output size is fixed in advance (§IV-B), with
// the work spread over threads afterwards (§IV-C).  This file computes that
// plan on the device from the per-field offsets:
//   plan_reduce    per tile of bags: sums of item counts and costs, offset
//                  validation; tile 0 also writes the per-field table info,
//                  column bases and id bases.
//   plan_tiles     only when the batch has more than kPlanDirectTiles tiles:
//                  one block turns the tile sums into exclusive prefixes and
//                  totals, so the next launch reads one entry per tile.
//   plan_scan      per tile: its exclusive prefix, the per-bag exclusive
//                  prefixes of items and cost, and every wave boundary that
//                  falls in a bag's cost interval.
// A batch of one tile runs both steps in a single block (one launch); a batch
// of at most kPlanDirectTiles tiles runs both in one launch whose blocks
// exchange their tile sums (plan_fused: a block per tile when every tile's
// block fits on the device at once, else a resident grid whose blocks take
// several tiles each); a one-hot batch
// (no offsets) takes plan_onehot, which writes the closed forms of the same
// arrays in one fully parallel launch.
//
// A tile is V slabs of kScanThreads consecutive bags; thread i holds bag i of
// every slab, so the offset loads and prefix stores are coalesced.  The loads
// of a group of slabs carry no branches between them and are all in flight
// together.  Within a slab a bag's prefix is a DPP wave scan plus the totals
// of the slab's earlier waves, read from LDS after one barrier per group of
// slabs.
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
#include <atomic>

#include "dpi_internal.h"
#include "wave_scan.h"

namespace dpi {
namespace {

typedef unsigned __int128 u128;
// Kernel arguments are read in place from the constant kernarg segment
// (scalar loads); the per-field arrays are indexed at run time.
typedef const __attribute__((address_space(4))) PlanArgs* PA;
typedef const __attribute__((address_space(4))) PlanParams& PPR;
typedef const __attribute__((address_space(4))) PlanDev& PDR;

__device__ __forceinline__ u128 mul128(int64_t a, int64_t b) { return (u128)(uint64_t)a * (uint64_t)b; }

// A value every lane of the wave holds, moved to scalar registers.
__device__ __forceinline__ int64_t uniform64(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
  return (int64_t)((uint64_t)hi << 32 | lo);
}

// A double near a 128-bit value (two roundings; callers only use it as a
// first guess and then correct with exact comparisons).
__device__ __forceinline__ double approx_u128(u128 x) {
  return (double)(uint64_t)(x >> 64) * 0x1p64 + (double)(uint64_t)x;
}

// smallest q >= 0 with q * den >= num (den > 0; the result fits int64);
// inv_den approximates 1/den
__device__ __forceinline__ int64_t ceil_div128(u128 num, int64_t den, double inv_den) {
  int64_t q = (int64_t)(approx_u128(num) * inv_den);
  if (q < 0) q = 0;
  while (q > 0 && mul128(q - 1, den) >= num) --q;
  while (mul128(q, den) < num) ++q;
  return q;
}

// largest q >= 0 with q * den <= num, from a first guess g
__device__ __forceinline__ int64_t floor_div128(u128 num, int64_t den, double g) {
  int64_t q = (int64_t)g;
  if (q < 0) q = 0;
  while (q > 0 && mul128(q, den) > num) --q;
  while (mul128(q + 1, den) <= num) ++q;
  return q;
}

// The same quotients in 64-bit arithmetic, for callers whose products and
// corrected quotients times den stay below 2^63.
__device__ __forceinline__ uint64_t mul64(int64_t a, int64_t b) { return (uint64_t)a * (uint64_t)b; }

__device__ __forceinline__ int64_t ceil_div64(uint64_t num, int64_t den, double inv_den) {
  int64_t q = (int64_t)((double)num * inv_den);
  if (q < 0) q = 0;
  while (q > 0 && mul64(q - 1, den) >= num) --q;
  while (mul64(q, den) < num) ++q;
  return q;
}

__device__ __forceinline__ int64_t floor_div64(uint64_t num, int64_t den, double g) {
  int64_t q = (int64_t)g;
  if (q < 0) q = 0;
  while (q > 0 && mul64(q, den) > num) --q;
  while (mul64(q + 1, den) <= num) ++q;
  return q;
}

// Exact quotients for the wave-boundary arithmetic: 128-bit, or 64-bit when
// S*W < 2^62 (then every product below stays under 2^63: E <= S, w <= W, a
// corrected quotient exceeds the true one by less than one, and an item
// costs at most S).
template <bool F64> struct Quot;
template <> struct Quot<false> {
  static __device__ __forceinline__ int64_t floor_mul_div(int64_t a, int64_t b, int64_t den, double g) {
    return floor_div128(mul128(a, b), den, g);
  }
  static __device__ __forceinline__ int64_t ceil_mul_div(int64_t a, int64_t b, int64_t den, double inv) {
    return ceil_div128(mul128(a, b), den, inv);
  }
  static __device__ __forceinline__ int64_t ceil_div(int64_t num, int64_t den, double inv) {
    return ceil_div128((u128)(uint64_t)num, den, inv);
  }
  // a * b <= c (a, b, c >= 0)
  static __device__ __forceinline__ bool mul_le(int64_t a, int64_t b, int64_t c) {
    return mul128(a, b) <= (u128)(uint64_t)c;
  }
};
template <> struct Quot<true> {
  static __device__ __forceinline__ int64_t floor_mul_div(int64_t a, int64_t b, int64_t den, double g) {
    return floor_div64(mul64(a, b), den, g);
  }
  static __device__ __forceinline__ int64_t ceil_mul_div(int64_t a, int64_t b, int64_t den, double inv) {
    return ceil_div64(mul64(a, b), den, inv);
  }
  static __device__ __forceinline__ int64_t ceil_div(int64_t num, int64_t den, double inv) {
    return ceil_div64((uint64_t)num, den, inv);
  }
  static __device__ __forceinline__ bool mul_le(int64_t a, int64_t b, int64_t c) {
    return mul64(a, b) <= (uint64_t)c;
  }
};

// field of bag l: floor(l / B), exact (the quotient is below DPI_MAX_TABLES)
__device__ __forceinline__ int32_t field_of(int64_t l, int64_t B, double inv_b) {
  int32_t t = (int32_t)((double)l * inv_b);
  while (t > 0 && (int64_t)t * B > l) --t;
  while ((int64_t)(t + 1) * B <= l) ++t;
  return t;
}

__device__ __forceinline__ int32_t packed_dim(uint32_t pk) { return (int32_t)(pk & 0x1ffffu); }
__device__ __forceinline__ int32_t packed_flags(uint32_t pk) { return (int32_t)(pk >> 17); }

// Block-wide sums of M values (every thread of the block takes part; all
// threads receive the sums).  s holds one row per wave.
template <int M>
__device__ __forceinline__ void block_sums(int64_t (&v)[M], int64_t (&s)[kWavesPerBlock][M]) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
#pragma unroll
  for (int m = 0; m < M; ++m) {
    const int64_t x = wave_incl_scan(v[m], lane);
    if (lane == 63) s[wv][m] = x;
  }
  __syncthreads();
#pragma unroll
  for (int m = 0; m < M; ++m) {
    int64_t a = 0;
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; ++w) a += s[w][m];
    v[m] = a;
  }
}

// Block-wide exclusive scan of a pair (field info only: one block, once).
__device__ __forceinline__ void block_scan_pair(int64_t a, int64_t b, int64_t& ea, int64_t& eb, int64_t& ta,
                                                int64_t& tb) {
  __shared__ int64_t wsum[2][kWavesPerBlock];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t ia = wave_incl_scan(a, lane), ib = wave_incl_scan(b, lane);
  if (lane == 63) {
    wsum[0][wv] = ia;
    wsum[1][wv] = ib;
  }
  __syncthreads();
  int64_t pa = 0, pb = 0;
  ta = 0;
  tb = 0;
#pragma unroll
  for (int v = 0; v < kWavesPerBlock; ++v) {
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

// ---------------------------------------------------------------------------
// Bag lengths, item counts and costs of CH slabs, loads first.
// ---------------------------------------------------------------------------
// Per-field row and output-row bytes, staged in LDS by every block.
struct FieldBytes {
  int32_t row[DPI_MAX_TABLES];
  int32_t out[DPI_MAX_TABLES];
};

// (the caller's next barrier publishes them)
__device__ __forceinline__ void stage_fields(PA pa, FieldBytes& f) {
  PPR p = pa->p;
  for (int t = threadIdx.x; t < p.T; t += kScanThreads) {
    const uint32_t pk = pa->packed[t];
    const int32_t dim = packed_dim(pk);
    f.row[t] = dim * ((packed_flags(pk) & kTiF16) ? 2 : 4);
    f.out[t] = dim * (p.out_dtype == DPI_F16 ? 2 : 4);
  }
}

// Bag l of slab k is first + k*kScanThreads.  Lanes past the last bag read
// the last bag's offsets (always in bounds) and report items 0, cost 0.
// Loading (slab_load) and costing (slab_cost) are separate so that a group's
// loads can be issued before a barrier or before the previous group's work.
// Both require TB > 0.
template <int CH>
struct SlabRaw {
  int32_t t[CH];      // field
  int32_t lo[CH];     // offsets of the bag's first id and one past its last
  int32_t hi[CH];
  bool ok[CH];        // a bag of the batch
  bool first[CH];     // the first bag of its field
};

template <int CH>
struct SlabBags {
  int32_t t[CH];     // field
  int32_t n[CH];     // items (n <= max(1, L) < 2^31)
  int64_t c[CH];     // cost
  bool bad;          // some valid bag has malformed offsets
};

template <int CH>
__device__ __forceinline__ void slab_load(PA pa, int64_t first, SlabRaw<CH>& r, double inv_b) {
  PPR p = pa->p;
  const int64_t TB = p.TB, B = p.B;
  int64_t lc[CH];   // clamped bag number
#pragma unroll
  for (int k = 0; k < CH; ++k) {
    const int64_t l = first + (int64_t)k * kScanThreads;
    r.ok[k] = l < TB;
    lc[k] = r.ok[k] ? l : TB - 1;
  }
  if (B >= kScanThreads) {
    // consecutive slabs of a lane cross at most one field start
    int32_t t = field_of(lc[0], B, inv_b);
    int64_t start = (int64_t)t * B;
#pragma unroll
    for (int k = 0; k < CH; ++k) {
      const bool next = lc[k] >= start + B;
      t += next ? 1 : 0;
      start += next ? B : 0;
      r.t[k] = t;
      r.first[k] = lc[k] == start;
    }
  } else {
#pragma unroll
    for (int k = 0; k < CH; ++k) {
      r.t[k] = field_of(lc[k], B, inv_b);
      r.first[k] = lc[k] == (int64_t)r.t[k] * B;
    }
  }
  if (p.offsets) {
    // bag (t, b) = t*B + b has its offsets at t*(B+1) + b = l + t
#pragma unroll
    for (int k = 0; k < CH; ++k) {
      const int32_t* o = p.offsets + lc[k] + r.t[k];
      r.lo[k] = o[0];
      r.hi[k] = o[1];
    }
  } else {
#pragma unroll
    for (int k = 0; k < CH; ++k) {
      r.lo[k] = 0;
      r.hi[k] = 1;
    }
  }
}

template <int CH>
__device__ __forceinline__ void slab_cost(PA pa, const FieldBytes& f, const SlabRaw<CH>& r, SlabBags<CH>& s) {
  PPR p = pa->p;
  const uint32_t C = (uint32_t)p.C;
  const int32_t sh = p.c_shift;
  s.bad = false;
#pragma unroll
  for (int k = 0; k < CH; ++k) {
    const bool bad = (r.first[k] & (r.lo[k] != 0)) | (r.hi[k] < r.lo[k]);
    s.bad |= r.ok[k] & bad;
    const uint32_t L = bad ? 0u : (uint32_t)(r.hi[k] - r.lo[k]);
    const uint32_t up = L + C - 1u;   // L < 2^31, C < 2^31
    uint32_t n = sh >= 0 ? up >> sh : up / C;
    n = n < 1u ? 1u : n;
    const int t = r.t[k];
    const int64_t c = (int64_t)L * f.row[t] + f.out[t] + (int64_t)n * p.K;
    s.t[k] = t;
    // masked, not selected: a select would become a branch around the reads
    s.n[k] = (int32_t)n & -(int32_t)r.ok[k];
    s.c[k] = c & -(int64_t)r.ok[k];
  }
}

// The same for a tile whose cost sum fits 32 bits (so does every bag's cost,
// formed here modulo 2^32).
template <int CH>
struct SlabBags32 {
  int32_t t[CH];
  uint32_t n[CH];
  uint32_t c[CH];
};

template <int CH>
__device__ __forceinline__ void slab_cost32(PA pa, const FieldBytes& f, const SlabRaw<CH>& r, SlabBags32<CH>& s) {
  PPR p = pa->p;
  const uint32_t C = (uint32_t)p.C, K = (uint32_t)p.K;
  const int32_t sh = p.c_shift;
  uint32_t row[CH], out[CH], L[CH], n[CH];
#pragma unroll
  for (int k = 0; k < CH; ++k) {   // as slab_cost: reads together, no branch around them
    row[k] = (uint32_t)f.row[r.t[k]];
    out[k] = (uint32_t)f.out[r.t[k]];
  }
#pragma unroll
  for (int k = 0; k < CH; ++k) {
    const bool bad = (r.first[k] & (r.lo[k] != 0)) | (r.hi[k] < r.lo[k]);
    L[k] = bad ? 0u : (uint32_t)(r.hi[k] - r.lo[k]);
  }
  if (sh >= 0) {
#pragma unroll
    for (int k = 0; k < CH; ++k) n[k] = (L[k] + C - 1u) >> sh;
  } else {
#pragma unroll
    for (int k = 0; k < CH; ++k) n[k] = (L[k] + C - 1u) / C;
  }
#pragma unroll
  for (int k = 0; k < CH; ++k) {
    n[k] = n[k] < 1u ? 1u : n[k];
    const uint32_t m = 0u - (uint32_t)r.ok[k];
    s.t[k] = r.t[k];
    s.n[k] = n[k] & m;
    s.c[k] = (L[k] * row[k] + out[k] + n[k] * K) & m;
  }
}

// ---------------------------------------------------------------------------
// Launch 1: tile sums, validation, field info.
// ---------------------------------------------------------------------------
// Duties outside the bag sums, in block 0: the per-field info.  (Nothing here
// has to precede another block's work: the header and every per-wave entry
// are written once, by the block that resolves them.)  Returns whether the id
// counts are malformed.
__device__ __forceinline__ bool plan_setup_block(PA pa, int64_t blk) {
  PPR p = pa->p;
  PDR d = pa->d;
  const int tid = threadIdx.x;
  bool bad = false;
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
  }
  return bad;
}

// sums (optional): receives the tile's items, cost and malformed | long << 1
// on every thread.  UNROLL: groups of slabs unrolled (by default all of
// them up to four, so that the compiler can issue those groups' loads
// together; fewer keep the registers for a caller that scans afterwards in
// the same kernel).
//
// KEEP (tiles of one group of slabs): the field bytes and the tile's loaded
// offsets are the caller's s_f and raw, kept for its scan, which then loads
// nothing again.
template <int V, int UNROLL, bool KEEP>
__device__ __forceinline__ void plan_reduce_block_k(PA pa, int64_t blk, int64_t nblocks, int64_t* sums,
                                                    FieldBytes* keep_f,
                                                    SlabRaw<(V < kPlanChunk ? V : kPlanChunk)>* keep_raw) {
  PPR p = pa->p;
  PDR d = pa->d;
  const int tid = threadIdx.x;
  constexpr int CH = V < kPlanChunk ? V : kPlanChunk;
  static_assert(!KEEP || V <= kPlanChunk, "one group of slabs");
  bool bad = false;

  int64_t v[4] = {0, 0, 0, 0};   // items, cost, malformed offsets, long bags
  if (p.TB > 0) {
    __shared__ FieldBytes s_f_own;
    SlabRaw<CH> raw_own;
    FieldBytes& s_f = KEEP ? *keep_f : s_f_own;
    SlabRaw<CH>& raw = KEEP ? *keep_raw : raw_own;
    stage_fields(pa, s_f);
    const int64_t tile0 = blk * (int64_t)kScanThreads * V;
    const double inv_b = 1.0 / (double)p.B;   // (once: the loop below reuses it)
    slab_load<CH>(pa, tile0 + tid, raw, inv_b);   // in flight across the setup and the barrier
    bad = plan_setup_block(pa, blk);        // (tile 0: the field info, its loads behind the slabs')
    __syncthreads();
#pragma unroll UNROLL
    for (int c0 = 0; c0 < V; c0 += CH) {
      SlabBags<CH> s;
      slab_cost<CH>(pa, s_f, raw, s);
      if (c0 + CH < V) slab_load<CH>(pa, tile0 + (int64_t)(c0 + CH) * kScanThreads + tid, raw, inv_b);
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        v[0] += s.n[k];
        v[1] += s.c[k];
        v[3] += s.n[k] > kDirectMaxItems ? 1 : 0;
      }
      bad |= s.bad;
    }
  } else {
    bad = plan_setup_block(pa, blk);
  }
  v[2] = bad ? 1 : 0;
  __shared__ int64_t s_red[kWavesPerBlock][4];
  block_sums<4>(v, s_red);
  const int64_t flags = (v[2] != 0 ? 1 : 0) | (v[3] << 1);   // malformed flag, long bags above it
  if (sums) {
    sums[0] = v[0];
    sums[1] = v[1];
    sums[2] = flags;
  }
  if (tid == 0) {
    const int64_t nb = p.nblk;
    d.block_sum[blk] = v[0];
    d.block_sum[nb + blk] = v[1];
    d.block_sum[2 * nb + blk] = flags;
  }
}

template <int V, int UNROLL = (V < kPlanChunk ? 1 : (V / kPlanChunk < 4 ? V / kPlanChunk : 4))>
__device__ __forceinline__ void plan_reduce_block(PA pa, int64_t blk, int64_t nblocks, int64_t* sums = nullptr) {
  plan_reduce_block_k<V, UNROLL, false>(pa, blk, nblocks, sums, nullptr, nullptr);
}

// ---------------------------------------------------------------------------
// Launch 2 (large batches only): tile sums -> exclusive tile prefixes.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kScanThreads) void plan_tiles_kernel(const PlanArgs args) {
  (void)args;
  const PA pa = (PA)__builtin_amdgcn_kernarg_segment_ptr();
  PPR p = pa->p;
  PDR d = pa->d;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t nb = p.nblk;
  int64_t* bs = d.block_sum;
  __shared__ int64_t s_w[2][2][kWavesPerBlock];   // double-buffered per round
  int64_t run_i = 0, run_c = 0;
  int err = 0;
  int buf = 0;
  for (int64_t i0 = 0; i0 < nb; i0 += kScanThreads, buf ^= 1) {
    const int64_t i = i0 + tid;
    const bool in = i < nb;
    const int64_t ic = in ? i : nb - 1;
    const int64_t si = in ? bs[ic] : 0, sc = in ? bs[nb + ic] : 0;
    err |= (in && (bs[2 * nb + ic] & 1) != 0) ? 1 : 0;
    const int64_t xi = wave_incl_scan(si, lane), xc = wave_incl_scan(sc, lane);
    if (lane == 63) {
      s_w[buf][0][wv] = xi;
      s_w[buf][1][wv] = xc;
    }
    __syncthreads();
    int64_t bi = 0, bc = 0, ai = 0, ac = 0;
#pragma unroll
    for (int v = 0; v < kWavesPerBlock; ++v) {
      const int64_t a = s_w[buf][0][v], b = s_w[buf][1][v];
      ai += a;
      ac += b;
      if (v < wv) {
        bi += a;
        bc += b;
      }
    }
    if (in) {
      bs[i] = run_i + bi + xi - si;
      bs[nb + i] = run_c + bc + xc - sc;
    }
    run_i += ai;
    run_c += ac;
  }
  err = __syncthreads_or(err);
  if (tid == 0) {
    bs[3 * nb] = run_i;
    bs[3 * nb + 1] = run_c;
    bs[3 * nb + 2] = err ? 1 : 0;
  }
}

// ---------------------------------------------------------------------------
// Launch 3: prefixes and partition.
// ---------------------------------------------------------------------------
// Wave targets of a plan: c_w = ceil(w*S/W) for w = 1..W (shared by a block).
struct Targets {
  int64_t W, S;
  double scale;     // W / S
  double inv_w;     // 1 / W
  bool exact;       // no snapping of starts to bag ends
  bool fits64;      // S * W < 2^62: the boundary quotients in 64-bit arithmetic
};

// A bag whose cost interval may hold a wave target (after the filter in the
// scan loop); a wave collects these and resolves them together.
struct Cand {
  int64_t bag, ibase, E_lo, E_hi;
  int32_t t, n;
};

// Plan arrays the boundary writes go to, staged in LDS.
struct BoundaryOut {
  int64_t* wib;
  int64_t* wave_bag;
  int64_t* wbase;
  int32_t* head_first;
  int32_t* split_pieces;
  int32_t* split_last;
  int32_t* tickets;
  int64_t C, K;
  unsigned long long splits;   // bags of this tile cut between waves
};

// Wave boundaries whose targets fall in the cost interval (E_lo, E_hi] of a
// bag with n items whose first item is number ibase.  Target c_w lies in it
// exactly when floor(E_lo*W/S) < w <= floor(E_hi*W/S).  Every boundary w in
// [1, W] is resolved here by exactly one bag, which writes all of what a
// lookup reads of it: the wave start, its bag and the bag's first item, the
// head link of wave w, and the split entries of wave w - 1 (the wave ending
// at it), whose arrival counter it also clears.
// Returns whether the bag is split between waves.
template <bool F64>
__device__ __forceinline__ bool bag_boundaries(const BoundaryOut& o, const Targets& g, const FieldBytes& f,
                                               const Cand& cd) {
  typedef Quot<F64> Q;
  const int64_t W = g.W, S = g.S, E_lo = cd.E_lo, E_hi = cd.E_hi, n = cd.n;
  const int64_t f_lo = Q::floor_mul_div(E_lo, W, S, floor((double)E_lo * g.scale));
  int64_t f_hi = Q::floor_mul_div(E_hi, W, S, floor((double)E_hi * g.scale));
  if (f_hi > W) f_hi = W;
  const int64_t out_bytes = f.out[cd.t];
  const int64_t per_item = o.C * f.row[cd.t] + o.K;
  const double inv_item = 1.0 / (double)per_item;
  int64_t w_first = -1, begin_prev = -1, pieces = 1, w_last = -1;
  for (int64_t w = f_lo + 1; w <= f_hi; ++w) {
    const int64_t c = Q::ceil_mul_div(w, S, W, g.inv_w);   // ceil(w*S/W), in (E_lo, E_hi]
    // smallest j in [1, n] whose cost prefix reaches c
    const int64_t num = c - E_lo - out_bytes;
    int64_t j = num <= 0 ? 1 : Q::ceil_div(num, per_item, inv_item);
    if (j < 1) j = 1;
    if (j > n - 1) j = n;
    bool inside = j < n;
    int64_t begin = cd.ibase + j;
    // snapped to the bag's end when that lies within half a wave's cost:
    // E_hi - c <= floor(S / 2W), i.e. (E_hi - c) * 2W <= S (c <= E_hi, and
    // with 64-bit quotients (E_hi - c) * 2W <= 2SW < 2^63)
    if (inside && !g.exact && Q::mul_le(E_hi - c, 2 * W, S)) {
      inside = false;
      begin = cd.ibase + n;
    }
    o.wib[w] = begin;
    o.wave_bag[w] = inside ? cd.bag : cd.bag + 1;
    o.wbase[w] = inside ? cd.ibase : cd.ibase + n;   // first item of that bag
    o.tickets[w - 1] = 0;
    bool first_inside = false;
    if (inside && w < W) {
      first_inside = w_first < 0;
      if (first_inside) w_first = w - 1;   // the wave holding the bag's first item
      if (begin_prev >= 0 && begin_prev < begin) ++pieces;   // previous inside wave was nonempty
      begin_prev = begin;
      w_last = w;
    }
    if (w < W) o.head_first[w] = inside ? (int32_t)w_first : -1;
    if (!first_inside) {   // wave w - 1 is not the first wave of a split bag
      o.split_pieces[w - 1] = 0;
      o.split_last[w - 1] = -1;
    }
  }
  if (w_first >= 0) {
    ++pieces;   // the last inside wave always holds the bag's remaining items
    o.split_pieces[w_first] = (int32_t)pieces;
    o.split_last[w_first] = (int32_t)w_last;
    return true;
  }
  return false;
}

// Lanes [0, count) of the wave each resolve one collected candidate.
__device__ __forceinline__ void resolve_candidates(BoundaryOut& o, const Targets& g, const FieldBytes& f,
                                                   const Cand* list, int count, int lane) {
  // the list was written by other lanes of this wave: keep the reads after the writes
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  __builtin_amdgcn_wave_barrier();
  const bool split = lane < count && (g.fits64 ? bag_boundaries<true>(o, g, f, list[lane])
                                               : bag_boundaries<false>(o, g, f, list[lane]));
  const uint64_t m = __ballot(split);
  o.splits += (unsigned long long)__popcll(m);   // wave-uniform
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

template <int V>
constexpr int scan_chunk() { return V < kPlanChunk ? V : kPlanChunk; }

// Field bytes to LDS and the loads of the tile's first group of slabs; the
// caller issues them early so that they are in flight while the tile prefix
// (and, for a single block, the setup) is formed.
template <int V>
__device__ __forceinline__ void plan_scan_prologue(PA pa, int64_t blk, FieldBytes& s_f, SlabRaw<scan_chunk<V>()>& raw) {
  if (pa->p.TB > 0) {
    stage_fields(pa, s_f);
    slab_load<scan_chunk<V>()>(pa, blk * (int64_t)kScanThreads * V + threadIdx.x, raw, 1.0 / (double)pa->p.B);
  }
}

// A tile of at most kPlanChunk slabs whose sums fit 32 bits, already scanned
// inside the tile (local_scan): per slab, each thread's bag's local
// exclusive item and cost prefixes, items, cost and field.
template <int V>
struct LocalSlabs {
  uint32_t li[V], lc[V], n[V], c[V];
  int32_t t[V];
};

template <int V, bool LOCAL = false>
__device__ __forceinline__ void plan_scan_core(PA pa, int64_t blk, int64_t pre_i, int64_t pre_c, int64_t N,
                                               int64_t S, bool err, int64_t nlong, int64_t own_i, int64_t own_c,
                                               FieldBytes& s_f, SlabRaw<scan_chunk<V>()>& raw,
                                               const LocalSlabs<V>* loc = nullptr);

// SINGLE: the whole batch is this block's one group of slabs (V <= kPlanChunk);
// its sums come straight from the block instead of from plan_reduce, and
// setup_bad carries plan_setup_block's verdict.  s_f and raw come from
// plan_scan_prologue.
template <int V, bool SINGLE>
__device__ __forceinline__ void plan_scan_block(PA pa, int64_t blk, bool setup_bad, FieldBytes& s_f,
                                                SlabRaw<scan_chunk<V>()>& raw) {
  PPR p = pa->p;
  PDR d = pa->d;
  const int tid = threadIdx.x;
  const int64_t nb = p.nblk;
  const int64_t* bs = d.block_sum;
  constexpr int CH = scan_chunk<V>();

  // this tile's exclusive prefix, its own sums and the totals
  int64_t pre_i, pre_c, N, S, own_i, own_c;
  int64_t nlong = 1;   // bags of more than kDirectMaxItems items (not counted beyond kPlanDirectTiles tiles)
  bool err;
  if constexpr (SINGLE) {
    static_assert(V <= kPlanChunk, "one group of slabs");
    __syncthreads();   // field bytes
    int64_t v[4] = {0, 0, setup_bad ? 1 : 0, 0};
    if (p.TB > 0) {
      SlabBags<CH> s0;
      slab_cost<CH>(pa, s_f, raw, s0);
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        v[0] += s0.n[k];
        v[1] += s0.c[k];
        v[3] += s0.n[k] > kDirectMaxItems ? 1 : 0;
      }
      v[2] += s0.bad ? 1 : 0;
    }
    __shared__ int64_t s_tot[kWavesPerBlock][4];
    block_sums<4>(v, s_tot);
    pre_i = 0;
    pre_c = 0;
    N = v[0];
    S = v[1];
    err = v[2] != 0;
    nlong = v[3];
    own_i = N;
    own_c = S;
  } else if (nb <= kPlanDirectTiles) {
    // from the tile sums: every entry loaded at once, then block sums
    int64_t v[6] = {0, 0, 0, 0, 0, 0};   // prefix items, prefix cost, items, cost, malformed, long bags
#pragma unroll
    for (int j = 0; j < kPlanDirectTiles / kScanThreads; ++j) {
      const int64_t i = tid + (int64_t)j * kScanThreads;
      const int64_t ic = i < nb ? i : nb - 1;
      const int64_t si = bs[ic], sc = bs[nb + ic], se = bs[2 * nb + ic];
      const bool in = i < nb, before = i < blk;
      v[0] += before ? si : 0;
      v[1] += before ? sc : 0;
      v[2] += in ? si : 0;
      v[3] += in ? sc : 0;
      v[4] += (in && (se & 1) != 0) ? 1 : 0;
      v[5] += in ? se >> 1 : 0;
    }
    __shared__ int64_t s_red[kWavesPerBlock][6];
    block_sums<6>(v, s_red);
    pre_i = v[0];
    pre_c = v[1];
    N = v[2];
    S = v[3];
    err = v[4] != 0;
    nlong = v[5];
    own_i = bs[blk];
    own_c = bs[nb + blk];
  } else {
    // plan_tiles left exclusive prefixes in place and the totals after them
    __syncthreads();   // field bytes
    pre_i = bs[blk];
    pre_c = bs[nb + blk];
    N = bs[3 * nb];
    S = bs[3 * nb + 1];
    err = bs[3 * nb + 2] != 0;
    own_i = (blk + 1 < nb ? bs[blk + 1] : N) - pre_i;
    own_c = (blk + 1 < nb ? bs[nb + blk + 1] : S) - pre_c;
  }
  plan_scan_core<V>(pa, blk, pre_i, pre_c, N, S, err, nlong, own_i, own_c, s_f, raw);
}

// The scan and partition of tile blk, its exclusive prefix (pre_i items,
// pre_c cost) and the batch's totals (N items, S cost, malformed offsets,
// bags longer than kDirectMaxItems items) known.  Block 0 also writes the
// header and the status words.
template <int V, bool LOCAL>
__device__ __forceinline__ void plan_scan_core(PA pa, int64_t blk, int64_t pre_i, int64_t pre_c, int64_t N,
                                               int64_t S, bool err, int64_t nlong, int64_t own_i, int64_t own_c,
                                               FieldBytes& s_f, SlabRaw<scan_chunk<V>()>& raw,
                                               const LocalSlabs<V>* loc) {
  PPR p = pa->p;
  PDR d = pa->d;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t nb = p.nblk;
  constexpr int CH = scan_chunk<V>();
  const int64_t tile0 = blk * (int64_t)kScanThreads * V;
  const int64_t W = p.waves_req < N ? p.waves_req : N;
  // a batch the lookup pools bag by bag reads only the header, the status
  // words and the field info unless it has a long bag (then the lookup falls
  // back to the partition): no bag prefixes, no partition; the host plans
  // again in full when the plan is exported
  const bool partition = !(p.lazy_partition && nlong == 0);

  if (blk == 0 && tid == 0) {
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
    h[kHdrSplit] = 0;   // the split bags are counted per tile (an export adds them up)
    h[14] = 0;
    h[15] = 0;
    if (p.prefixes) {
      d.bib[p.TB] = N;
      d.bcb[p.TB] = S;
    }
    d.wib[0] = 0;
    d.wave_bag[0] = 0;
    d.wbase[0] = 0;
    if (W > 0 && partition) d.head_first[0] = -1;   // wave 0 starts at the first bag
    // the only writer of the status words during planning; lookups latch later
    *reinterpret_cast<uint64_t*>(d.status) = status_word(p.plan_id, err ? kStatusBadOffsets : 0);
    d.status[kStatusLongWord] = nlong < INT32_MAX ? (int32_t)nlong : INT32_MAX;
  }
  int64_t* const tile_splits = d.block_sum + 3 * nb + 3;
  if (p.TB == 0 || !partition) {   // block-uniform
    if (tid == 0) tile_splits[blk] = 0;
    return;
  }

  // The targets' quotients and the output pointers, per wave: no barrier
  // before the filter (every caller has published the field bytes with a
  // barrier of its own).  S and W are block-uniform; read once per wave.
  const int64_t Su = uniform64(S), Wu = uniform64(W);
  Targets g;
  g.W = Wu;
  g.S = Su;
  g.exact = (p.flags & DPI_FLAG_EXACT_SPLIT) != 0;
  {
    // two independent divisions, no branch between them (W > 0 implies
    // S > 0: every bag costs at least its output row)
    const bool any = Wu > 0;
    const double scale = (double)Wu / (double)(any ? Su : 1);   // 0 when W = 0
    const double inv_w = 1.0 / (double)(any ? Wu : 1);
    g.scale = scale;
    g.inv_w = any ? inv_w : 0.0;
  }
  g.fits64 = mul128(Su, Wu) < ((u128)1 << 62);
  BoundaryOut o;
  o.wib = d.wib;
  o.wave_bag = d.wave_bag;
  o.wbase = d.wbase;
  o.head_first = d.head_first;
  o.split_pieces = d.split_pieces;
  o.split_last = d.split_last;
  o.tickets = d.tickets;
  o.C = p.C;
  o.K = p.K;
  o.splits = 0;   // this wave's split bags
  const double scale = g.scale;
  __shared__ Cand s_cand[kWavesPerBlock][kWaveSize];
  int ncand = 0;   // collected candidates of this wave (wave-uniform)
  // Collects bag `bag` (items [ibase, ibase + n), cost interval (E_lo, E_hi])
  // when the filter passed for some lane; resolves a full list first.
  auto collect = [&](bool cand, int64_t bag, int64_t ibase, int64_t E_lo, int64_t E_hi, int32_t t, int32_t n) {
    const uint64_t m = __ballot(cand);
    if (m == 0) return;
    const int cnt = __popcll(m);
    if (ncand + cnt > kWaveSize) {
      resolve_candidates(o, g, s_f, s_cand[wv], ncand, lane);
      ncand = 0;
    }
    if (cand) {
      const int pos = ncand + __popcll(m & ((1ull << lane) - 1ull));
      Cand& e = s_cand[wv][pos];
      e.bag = bag;
      e.ibase = ibase;
      e.E_lo = E_lo;
      e.E_hi = E_hi;
      e.t = t;
      e.n = n;
    }
    ncand += cnt;
  };
  // filter in double: both products are within (x + 1) * 2^-50 of E*W/S,
  // so equal floors of the widened interval prove it holds no target
  auto may_hold_target = [](double x_lo, double x_hi) {
    const double margin = (x_hi + 1.0) * 0x1p-45;
    return floor(x_hi + margin) != floor(x_lo - margin);
  };
  if constexpr (LOCAL) {
    // scanned inside the tile before the tile sums were gathered: the tile
    // prefix added, then the filter
    (void)raw;
    (void)own_i;
    (void)own_c;
    const double base = (double)pre_c * scale;
    const int64_t TB = p.TB;
    if (p.prefixes) {   // block-uniform
#pragma unroll
      for (int k = 0; k < V; ++k) {
        const int64_t bag = tile0 + (int64_t)k * kScanThreads + tid;
        if (bag < TB) {
          d.bib[bag] = pre_i + loc->li[k];
          d.bcb[bag] = pre_c + loc->lc[k];
        }
      }
    }
    if (W > 0) {
      // every slab's filter first (straight-line), then the collection
      bool cand[V];
#pragma unroll
      for (int k = 0; k < V; ++k) {
        const double x_lo = fma((double)loc->lc[k], scale, base);
        const double x_hi = fma((double)(loc->lc[k] + loc->c[k]), scale, base);
        cand[k] = tile0 + (int64_t)k * kScanThreads + tid < TB && may_hold_target(x_lo, x_hi);
      }
#pragma unroll
      for (int k = 0; k < V; ++k)
        collect(cand[k], tile0 + (int64_t)k * kScanThreads + tid, pre_i + loc->li[k], pre_c + loc->lc[k],
                pre_c + loc->lc[k] + loc->c[k], loc->t[k], (int32_t)loc->n[k]);
    }
  } else if (own_i >= 0 && own_i <= (int64_t)UINT32_MAX && own_c >= 0 && own_c <= (int64_t)UINT32_MAX) {
    // Narrow tile (block-uniform): every sum inside the tile fits 32 bits, so
    // the costs, scans, wave totals and running sums are 32-bit and a bag's
    // 64-bit prefixes are the tile prefix plus its local ones.  The filter
    // forms E*W/S as fma(local, W/S, pre_c*W/S): three roundings of relative
    // size 2^-53, inside the same bound.
    __shared__ __align__(16) uint32_t s_w32[V][2][kWavesPerBlock];
    const double base = (double)pre_c * scale;
    const int64_t TB = p.TB;
    const bool prefixes = p.prefixes != 0;
    const double inv_b = 1.0 / (double)p.B;   // (once, not per group)
    uint32_t run_i = 0, run_c = 0;
#pragma unroll 1
    for (int c0 = 0; c0 < V; c0 += CH) {
      SlabBags32<CH> s;
      slab_cost32<CH>(pa, s_f, raw, s);
      if (c0 + CH < V) slab_load<CH>(pa, tile0 + (int64_t)(c0 + CH) * kScanThreads + tid, raw, inv_b);   // next group
      uint32_t xi[CH], xc[CH];
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        xi[k] = wave_incl_scan32(s.n[k], lane);
        xc[k] = wave_incl_scan32(s.c[k], lane);
        if (lane == 63) {
          s_w32[c0 + k][0][wv] = xi[k];
          s_w32[c0 + k][1][wv] = xc[k];
        }
      }
      __syncthreads();   // every slab of the group has its own LDS slots: one barrier per group
      // the group's prefixes and filters in straight-line code, then the
      // prefix stores and the collection
      uint32_t li[CH], lc[CH];
      bool cand[CH];
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        const uint4 wi = *reinterpret_cast<const uint4*>(s_w32[c0 + k][0]);
        const uint4 wc = *reinterpret_cast<const uint4*>(s_w32[c0 + k][1]);
        const uint32_t bi = (wv > 0 ? wi.x : 0u) + (wv > 1 ? wi.y : 0u) + (wv > 2 ? wi.z : 0u);
        const uint32_t bc = (wv > 0 ? wc.x : 0u) + (wv > 1 ? wc.y : 0u) + (wv > 2 ? wc.z : 0u);
        li[k] = run_i + bi + xi[k] - s.n[k];   // local exclusive prefixes
        lc[k] = run_c + bc + xc[k] - s.c[k];
        run_i += wi.x + wi.y + wi.z + wi.w;
        run_c += wc.x + wc.y + wc.z + wc.w;
        const double x_lo = fma((double)lc[k], scale, base), x_hi = fma((double)(lc[k] + s.c[k]), scale, base);
        cand[k] = tile0 + (int64_t)(c0 + k) * kScanThreads + tid < TB && may_hold_target(x_lo, x_hi);
      }
      if (prefixes) {   // block-uniform
#pragma unroll
        for (int k = 0; k < CH; ++k) {
          const int64_t bag = tile0 + (int64_t)(c0 + k) * kScanThreads + tid;
          if (bag < TB) {
            d.bib[bag] = pre_i + li[k];
            d.bcb[bag] = pre_c + lc[k];
          }
        }
      }
      if (W > 0) {
#pragma unroll
        for (int k = 0; k < CH; ++k)
          collect(cand[k], tile0 + (int64_t)(c0 + k) * kScanThreads + tid, pre_i + li[k], pre_c + lc[k],
                  pre_c + lc[k] + s.c[k], s.t[k], (int32_t)s.n[k]);
      }
    }
  } else {
    // Wide tile (a tile cost of 2^32 bytes or more: rows of hundreds of
    // kilobytes): 64-bit sums, one slab at a time with its own loads, two
    // barriers per slab -- slower, and light on registers, so that this rare
    // path does not cost the narrow one occupancy.
    __shared__ int64_t s_wt[2][kWavesPerBlock];
    int64_t run_i = pre_i, run_c = pre_c;
    const double inv_b = 1.0 / (double)p.B;
#pragma unroll 1
    for (int k = 0; k < V; ++k) {
      const int64_t bag = tile0 + (int64_t)k * kScanThreads + tid;
      SlabRaw<1> r1;
      slab_load<1>(pa, bag, r1, inv_b);
      SlabBags<1> s1;
      slab_cost<1>(pa, s_f, r1, s1);
      const int64_t xi = wave_incl_scan(s1.n[0], lane), xc = wave_incl_scan(s1.c[0], lane);
      __syncthreads();   // the previous slab's totals are read
      if (lane == 63) {
        s_wt[0][wv] = xi;
        s_wt[1][wv] = xc;
      }
      __syncthreads();
      int64_t bi = 0, bc = 0, ai = 0, ac = 0;
#pragma unroll
      for (int v = 0; v < kWavesPerBlock; ++v) {
        const int64_t a = s_wt[0][v], b = s_wt[1][v];
        ai += a;
        ac += b;
        bi += v < wv ? a : 0;
        bc += v < wv ? b : 0;
      }
      const int64_t ibase = run_i + bi + xi - s1.n[0];
      const int64_t E_lo = run_c + bc + xc - s1.c[0];
      const int64_t E_hi = E_lo + s1.c[0];
      run_i += ai;
      run_c += ac;
      const bool valid = bag < p.TB;
      if (valid && p.prefixes) {
        d.bib[bag] = ibase;
        d.bcb[bag] = E_lo;
      }
      if (W == 0) continue;
      const bool cand = valid && may_hold_target((double)E_lo * scale, (double)E_hi * scale);
      collect(cand, bag, ibase, E_lo, E_hi, s1.t[0], s1.n[0]);
    }
  }
  if (ncand > 0) resolve_candidates(o, g, s_f, s_cand[wv], ncand, lane);
  __shared__ unsigned long long s_splits[kWavesPerBlock];
  if (lane == 0) s_splits[wv] = o.splits;
  __syncthreads();
  if (tid == 0) {
    unsigned long long n = 0;
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; ++w) n += s_splits[w];
    tile_splits[blk] = (int64_t)n;
  }
}

template <int V>
__global__ __launch_bounds__(kScanThreads) void plan_reduce_kernel(const PlanArgs args) {
  (void)args;
  plan_reduce_block<V>((PA)__builtin_amdgcn_kernarg_segment_ptr(), blockIdx.x, gridDim.x);
}

template <int V>
__global__ __launch_bounds__(kScanThreads) __attribute__((amdgpu_waves_per_eu(2))) void plan_scan_kernel(const PlanArgs args) {
  (void)args;
  const PA pa = (PA)__builtin_amdgcn_kernarg_segment_ptr();
  __shared__ FieldBytes s_f;
  SlabRaw<scan_chunk<V>()> raw;
  plan_scan_prologue<V>(pa, blockIdx.x, s_f, raw);
  plan_scan_block<V, false>(pa, blockIdx.x, false, s_f, raw);
}

// A batch of one tile: one block, one launch; the bag sums never leave the
// block (the scan's barriers order the setup's header reset before the
// header writes and split counts).
template <int V>
__global__ __launch_bounds__(kScanThreads) void plan_single_kernel(const PlanArgs args) {
  (void)args;
  const PA pa = (PA)__builtin_amdgcn_kernarg_segment_ptr();
  __shared__ FieldBytes s_f;
  SlabRaw<scan_chunk<V>()> raw;
  plan_scan_prologue<V>(pa, 0, s_f, raw);   // the bags' offsets load during the setup
  const bool bad = plan_setup_block(pa, 0);
  plan_scan_block<V, true>(pa, 0, bad, s_f, raw);
}

// ---------------------------------------------------------------------------
// One-hot batches (no offsets): every bag holds one id and is one item, so
// the prefixes and the wave starts have closed forms and one fully parallel
// launch writes them.  Field t's bags each cost cost_t = row_bytes_t +
// out_bytes_t + K, its first bag starts at F_t = sum over t' < t of
// B*cost_t', and target c_w lies in bag (t, b) of field t with
// F_t < c_w <= F_{t+1} and b = ceil((c_w - F_t)/cost_t) - 1.  A one-item bag
// is never split: wave w starts after that bag.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kScanThreads) void plan_onehot_kernel(const PlanArgs args) {
  (void)args;
  const PA pa = (PA)__builtin_amdgcn_kernarg_segment_ptr();
  PPR p = pa->p;
  PDR d = pa->d;
  const int tid = threadIdx.x;
  const bool bad = __syncthreads_or(plan_setup_block(pa, blockIdx.x) ? 1 : 0) != 0;

  // per-field bag cost and the cost prefix over fields
  __shared__ int64_t s_cost[DPI_MAX_TABLES];
  __shared__ int64_t s_F[DPI_MAX_TABLES + 1];
  int64_t cost = 0;
  if (tid < p.T) {
    const uint32_t pk = pa->packed[tid];
    const int64_t dim = packed_dim(pk);
    cost = dim * ((packed_flags(pk) & kTiF16) ? 2 : 4) + dim * (p.out_dtype == DPI_F16 ? 2 : 4) + p.K;
  }
  int64_t F, unused0, S, unused1;
  block_scan_pair(p.B * cost, 0, F, unused0, S, unused1);
  if (tid < p.T) {
    s_cost[tid] = cost;
    s_F[tid] = F;
  }
  if (tid == 0) s_F[p.T] = S;
  __syncthreads();
  const int64_t TB = p.TB, N = TB;
  const int64_t W = p.waves_req < N ? p.waves_req : N;

  if (blockIdx.x == 0 && tid == 0) {
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
    h[kHdrSplit] = 0;
    h[14] = 0;
    h[15] = 0;
    *reinterpret_cast<uint64_t*>(d.status) = status_word(p.plan_id, bad ? kStatusBadOffsets : 0);
    d.status[kStatusLongWord] = 0;   // every bag is one item
  }
  const int64_t first = (int64_t)blockIdx.x * kScanThreads + tid, stride = (int64_t)gridDim.x * kScanThreads;
  for (int64_t j = first; j < p.nblk; j += stride) d.block_sum[3 * (int64_t)p.nblk + 3 + j] = 0;   // no split bags
  if (p.lazy_partition) return;   // the lookup reads neither the prefixes nor the partition
  const double inv_b = p.B > 0 ? 1.0 / (double)p.B : 0.0;
  for (int64_t l = first; p.prefixes && l <= TB; l += stride) {
    if (l == TB) {
      d.bib[l] = N;
      d.bcb[l] = S;
    } else {
      const int32_t t = field_of(l, p.B, inv_b);
      d.bib[l] = l;
      d.bcb[l] = s_F[t] + (l - (int64_t)t * p.B) * s_cost[t];
    }
  }
  const double inv_w = W > 0 ? 1.0 / (double)W : 0.0;
  for (int64_t w = first; w <= W; w += stride) {
    int64_t start = 0;
    if (w > 0) {
      const int64_t c = ceil_div128(mul128(w, S), W, inv_w);   // in (0, S]
      // the field with F_t < c <= F_{t+1}
      int lo = 0, hi = p.T - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s_F[mid] < c) lo = mid;
        else hi = mid - 1;
      }
      const int64_t ct = s_cost[lo], local = c - s_F[lo];   // in (0, B*ct]
      int64_t q = (int64_t)((double)local / (double)ct);     // then exact: q = ceil(local/ct)
      while (q > 0 && (q - 1) * ct >= local) --q;
      while (q * ct < local) ++q;
      start = (int64_t)lo * p.B + q;   // bag (lo, q - 1) ends where wave w starts
    }
    d.wib[w] = start;
    d.wave_bag[w] = start;
    d.wbase[w] = start;   // one item per bag
    if (w < W) {          // and never cut between waves
      d.head_first[w] = -1;
      d.split_pieces[w] = 0;
      d.split_last[w] = -1;
      d.tickets[w] = 0;
    }
  }
}

// ---------------------------------------------------------------------------
// One launch for batches of several tiles (at most kPlanDirectTiles; every
// block resident, a block per tile or several tiles per block): each block
// sums its tiles and publishes the sums, then
// gathers every tile's sums -- the partition needs the batch's total cost,
// so a block waits for the tiles after it as well as those before -- and
// scans and partitions its tiles.  A published sum travels as two 64-bit
// words, each holding the low 32 bits of the plan's id above 32 bits of the
// value, stored and loaded with device-scope atomics: a word is valid exactly
// when its id matches, so no fence (no write-back or invalidation of the
// L2s) is needed.  The wait is bounded: a tile whose words do not appear in
// time (its block not yet resident) is summed by the waiting thread itself
// from the offsets, so every block finishes whatever the residency.  No block
// relies on another block's writes other than the published sums: the header
// and each per-wave entry have a single writer.
// ---------------------------------------------------------------------------
constexpr int kPlanSpinLimit = 4096;   // polls of a tile's flag before summing the tile here

// Sums of tile j computed by one thread: items, cost, and the malformed and
// long-bag flags in the layout the blocks publish (malformed | long << 1).
template <int V>
__device__ int64_t tile_sums_serial(PA pa, const FieldBytes& f, int64_t j, int64_t& items, int64_t& cost) {
  PPR p = pa->p;
  const int64_t B = p.B, TB = p.TB;
  const uint32_t C = (uint32_t)p.C;
  const int64_t l0 = j * (int64_t)kScanThreads * V;
  const int64_t l1 = min(TB, l0 + (int64_t)kScanThreads * V);
  int64_t bad = 0, nlong = 0;
  items = 0;
  cost = 0;
  if (j == 0) {   // the id counts, as block 0's setup checks them
    int64_t tot = 0;
    for (int t = 0; t < p.T; ++t) {
      const int64_t nnz = p.offsets[(int64_t)t * (B + 1) + B];
      bad |= nnz < 0 ? 1 : 0;
      tot += nnz < 0 ? 0 : nnz;
    }
    bad |= tot != p.total_ids ? 1 : 0;
  }
  int64_t t = l0 / B;
  for (int64_t l = l0; l < l1; ++l) {
    while ((t + 1) * B <= l) ++t;
    const int32_t lo = p.offsets[l + t], hi = p.offsets[l + t + 1];
    const bool malformed = (l == t * B && lo != 0) || hi < lo;
    bad |= malformed ? 1 : 0;
    const uint32_t L = malformed ? 0u : (uint32_t)(hi - lo);
    uint32_t n = (L + C - 1u) / C;
    n = n < 1u ? 1u : n;
    items += n;
    cost += (int64_t)L * f.row[t] + f.out[t] + (int64_t)n * p.K;
    nlong += n > (uint32_t)kDirectMaxItems ? 1 : 0;
  }
  return bad | (nlong << 1);
}

// Publishes tile blk's sums (items, cost, malformed | long << 1) as tagged
// words (one thread).  Short form, the usual case: one pair of words,
// items and cost, when the items fit 32 bits, the cost 31 bits and the
// flags are clear.  Otherwise the long form: six words (each sum's two
// halves), after every tile's pair, and a pair whose cost word has bit 31
// set.  A reader of the pair reads the long form only when it sees that bit.
constexpr int kTileWords = 6;             // long form
constexpr uint32_t kLongForm = 0x80000000u;

__device__ __forceinline__ void publish_tile_sums(int64_t* flags, int64_t nb, int64_t blk, uint64_t tag,
                                                  const int64_t (&mine)[3]) {
  uint64_t* const pair = reinterpret_cast<uint64_t*>(flags) + 2 * blk;
  const bool shrt = (uint64_t)mine[0] <= 0xffffffffu && (uint64_t)mine[1] < kLongForm && mine[2] == 0;
  if (!shrt) {
    uint64_t* const w = reinterpret_cast<uint64_t*>(flags) + 2 * nb + blk * kTileWords;
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      __hip_atomic_store(w + 2 * q, tag | ((uint64_t)mine[q] & 0xffffffffu), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(w + 2 * q + 1, tag | ((uint64_t)mine[q] >> 32), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __hip_atomic_store(pair, tag | (shrt ? (uint64_t)mine[0] : 0u), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(pair + 1, tag | (shrt ? (uint64_t)mine[1] : (uint64_t)kLongForm), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

// Every tile's published sums, gathered for tile blk (thread i takes tiles i,
// i + 256, ...): v = prefix items, prefix cost, items, cost, malformed tiles,
// long bags, block-reduced on every thread; own = tile blk's items and cost.
// A thread requests all of its tiles' pairs at once, one 16-byte load per
// tile at agent scope (sc1: served past the XCD's L2, as an agent-scope
// atomic load is; every 8-byte word carries its own tag, so the pair need not
// be read atomically), so the usual case -- every tile published in the short
// form -- costs one round trip, and each further polling round one more for
// all of the thread's tiles still missing.  A long form is polled by its
// thread alone.
template <int V>
__device__ __forceinline__ void gather_tile_sums(PA pa, int64_t blk, uint64_t tag, const int64_t* flags,
                                                 const FieldBytes& s_f, int64_t (&v)[6], int64_t (&own)[2]) {
  typedef int i32x4 __attribute__((ext_vector_type(4)));
  constexpr int kSc1 = 1 << 4;   // buffer cache policy: agent scope
  const int tid = threadIdx.x;
  const int64_t nb = pa->p.nblk;
  constexpr int kPer = kPlanDirectTiles / kScanThreads;
  const uint32_t tag_hi = (uint32_t)(tag >> 32);
  __shared__ int64_t s_own[2];
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int64_t*>(flags), (short)0, (int)(nb * (2 + kTileWords) * 8), 0x00020000);
  i32x4 pr[kPer];
  bool ready[kPer];
  auto load_pair = [&](int m) {
    const int64_t j = min(tid + (int64_t)m * kScanThreads, nb - 1);
    pr[m] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)(j * 16), 0, kSc1);
  };
  auto tagged = [&](int m) { return (uint32_t)pr[m].y == tag_hi && (uint32_t)pr[m].w == tag_hi; };
#pragma unroll
  for (int m = 0; m < kPer; ++m)
    if ((int64_t)m * kScanThreads < nb) load_pair(m);   // block-uniform
#pragma unroll
  for (int m = 0; m < kPer; ++m) ready[m] = tid + (int64_t)m * kScanThreads >= nb || tagged(m);
  // tiles not yet published: every missing tile of the thread polled again
  // per round, one round trip each round
  for (int spin = 0; spin < kPlanSpinLimit; ++spin) {
    bool all = true;
#pragma unroll
    for (int m = 0; m < kPer; ++m) all &= ready[m];
    if (all) break;
    __builtin_amdgcn_s_sleep(1);
#pragma unroll
    for (int m = 0; m < kPer; ++m)
      if (!ready[m]) load_pair(m);
#pragma unroll
    for (int m = 0; m < kPer; ++m) ready[m] = ready[m] || tagged(m);
  }
#pragma unroll
  for (int q = 0; q < 6; ++q) v[q] = 0;
#pragma unroll
  for (int m = 0; m < kPer; ++m) {
    if ((int64_t)m * kScanThreads >= nb) break;
    const int64_t j = tid + (int64_t)m * kScanThreads;
    if (j >= nb) continue;
    int64_t si = (uint32_t)pr[m].x, sc = (uint32_t)pr[m].z, se = 0;
    bool have = ready[m] && ((uint32_t)pr[m].z & kLongForm) == 0;
    if (ready[m] && !have) {
      // the long form (bounded poll; its words may land after the pair)
      const int base = (int)((2 * nb + j * kTileWords) * 8);
      for (int spin = 0; spin < kPlanSpinLimit && !have; ++spin) {
        const i32x4 r0 = __builtin_amdgcn_raw_buffer_load_b128(rsrc, base, 0, kSc1);
        const i32x4 r1 = __builtin_amdgcn_raw_buffer_load_b128(rsrc, base + 16, 0, kSc1);
        const i32x4 r2 = __builtin_amdgcn_raw_buffer_load_b128(rsrc, base + 32, 0, kSc1);
        have = (uint32_t)r0.y == tag_hi && (uint32_t)r0.w == tag_hi && (uint32_t)r1.y == tag_hi &&
               (uint32_t)r1.w == tag_hi && (uint32_t)r2.y == tag_hi && (uint32_t)r2.w == tag_hi;
        if (have) {
          si = (int64_t)((uint64_t)(uint32_t)r0.x | (uint64_t)(uint32_t)r0.z << 32);
          sc = (int64_t)((uint64_t)(uint32_t)r1.x | (uint64_t)(uint32_t)r1.z << 32);
          se = (int64_t)((uint64_t)(uint32_t)r2.x | (uint64_t)(uint32_t)r2.z << 32);
        } else {
          __builtin_amdgcn_s_sleep(1);
        }
      }
    }
    if (!have) se = tile_sums_serial<V>(pa, s_f, j, si, sc);   // not published in time: summed here
    v[0] += j < blk ? si : 0;
    v[1] += j < blk ? sc : 0;
    v[2] += si;
    v[3] += sc;
    v[4] += (se & 1) != 0 ? 1 : 0;
    v[5] += se >> 1;
    if (j == blk) {
      s_own[0] = si;
      s_own[1] = sc;
    }
  }
  __shared__ int64_t s_red[kWavesPerBlock][6];
  block_sums<6>(v, s_red);   // its barrier also publishes s_own
  own[0] = s_own[0];
  own[1] = s_own[1];
}

// The scan inside a tile of one group of slabs whose sums fit 32 bits, from
// its loaded offsets: what the narrow scan does before it adds the tile
// prefix.  Run while the other blocks publish their sums, so that a block
// polls for them later and its polling loads do not hold up their stores.
template <int V>
__device__ __forceinline__ void local_scan(PA pa, const FieldBytes& s_f, const SlabRaw<V>& raw, LocalSlabs<V>& loc) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  __shared__ __align__(16) uint32_t s_w[V][2][kWavesPerBlock];
  SlabBags32<V> s;
  slab_cost32<V>(pa, s_f, raw, s);
  uint32_t xi[V], xc[V];
#pragma unroll
  for (int k = 0; k < V; ++k) {
    loc.n[k] = s.n[k];
    loc.c[k] = s.c[k];
    loc.t[k] = s.t[k];
    xi[k] = wave_incl_scan32(s.n[k], lane);
    xc[k] = wave_incl_scan32(s.c[k], lane);
    if (lane == 63) {
      s_w[k][0][wv] = xi[k];
      s_w[k][1][wv] = xc[k];
    }
  }
  __syncthreads();
  uint32_t run_i = 0, run_c = 0;
#pragma unroll
  for (int k = 0; k < V; ++k) {
    const uint4 wi = *reinterpret_cast<const uint4*>(s_w[k][0]);
    const uint4 wc = *reinterpret_cast<const uint4*>(s_w[k][1]);
    const uint32_t bi = (wv > 0 ? wi.x : 0u) + (wv > 1 ? wi.y : 0u) + (wv > 2 ? wi.z : 0u);
    const uint32_t bc = (wv > 0 ? wc.x : 0u) + (wv > 1 ? wc.y : 0u) + (wv > 2 ? wc.z : 0u);
    loc.li[k] = run_i + bi + xi[k] - s.n[k];
    loc.lc[k] = run_c + bc + xc[k] - s.c[k];
    run_i += wi.x + wi.y + wi.z + wi.w;
    run_c += wc.x + wc.y + wc.z + wc.w;
  }
}

// A block per tile.  SPREAD = false: every block resident at once, each
// sums its own tile.  SPREAD = true: more tiles than resident blocks; blocks
// b < p.reduce_blocks (the first to start, all resident together) sum tiles
// b, b + reduce_blocks, ... and publish all of them before any block waits,
// and the later blocks, which start as the first ones finish, only gather
// and scan.  At least two waves per SIMD, so that every tile count the
// planner picks (at most 512 tiles) stays resident.
template <int V, bool SPREAD>
__global__ __launch_bounds__(kScanThreads) __attribute__((amdgpu_waves_per_eu(2))) void plan_fused_kernel(const PlanArgs args) {
  (void)args;
  const PA pa = (PA)__builtin_amdgcn_kernarg_segment_ptr();
  PPR p = pa->p;
  PDR d = pa->d;
  const int tid = threadIdx.x;
  const int64_t blk = blockIdx.x, nb = p.nblk;
  int64_t* const flags = d.block_sum + 4 * nb + 3;
  const uint64_t tag = (uint64_t)p.plan_id << 32;

  __shared__ FieldBytes s_f;
  SlabRaw<scan_chunk<V>()> raw;
  // tile sums (tile 0: also the field info), published
  int64_t mine_i = 0, mine_c = 0;
  if constexpr (!SPREAD) {
    int64_t mine[3];
    if constexpr (V <= kPlanChunk) {
      // one group of slabs: the sums' loads and field bytes serve the scan too
      plan_reduce_block_k<V, 1, true>(pa, blk, nb, mine, &s_f, &raw);
    } else {
      plan_reduce_block<V>(pa, blk, nb, mine);
    }
    if (tid == 0) publish_tile_sums(flags, nb, blk, tag, mine);
    mine_i = mine[0];
    mine_c = mine[1];
  } else {
    const int64_t G = p.reduce_blocks;
#pragma unroll 1
    for (int64_t j = blk; blk < G && j < nb; j += G) {
      int64_t mine[3];
      plan_reduce_block<V, 1>(pa, j, nb, mine);
      if (tid == 0) publish_tile_sums(flags, nb, j, tag, mine);
      __syncthreads();   // the next tile's sums reuse the block's LDS
    }
  }

  if constexpr (!SPREAD && V <= kPlanChunk) {
    // the tile's own sums are known (block-uniform): a tile whose sums fit
    // 32 bits scans now, the rest after the gather as usual
    const bool narrow = mine_i <= (int64_t)UINT32_MAX && mine_c <= (int64_t)UINT32_MAX;
    int64_t v[6], own[2];
    if (narrow) {
      LocalSlabs<V> loc;
      local_scan<V>(pa, s_f, raw, loc);
      gather_tile_sums<V>(pa, blk, tag, flags, s_f, v, own);
      plan_scan_core<V, true>(pa, blk, v[0], v[1], v[2], v[3], v[4] != 0, v[5], own[0], own[1], s_f, raw, &loc);
    } else {
      gather_tile_sums<V>(pa, blk, tag, flags, s_f, v, own);
      plan_scan_core<V>(pa, blk, v[0], v[1], v[2], v[3], v[4] != 0, v[5], own[0], own[1], s_f, raw);
    }
  } else {
    plan_scan_prologue<V>(pa, blk, s_f, raw);   // field bytes, and the first loads of the scan in flight
    __syncthreads();
    int64_t v[6], own[2];
    gather_tile_sums<V>(pa, blk, tag, flags, s_f, v, own);
    plan_scan_core<V>(pa, blk, v[0], v[1], v[2], v[3], v[4] != 0, v[5], own[0], own[1], s_f, raw);
  }
}

// Blocks of plan_fused_kernel<V, SPREAD> resident at once on the current
// device (0 if the runtime cannot say), asked once per device.
constexpr int kCapacityDevices = 64;
template <int V, bool SPREAD>
int64_t plan_fused_capacity() {
  static std::atomic<int64_t> cap[kCapacityDevices];   // 0: not asked yet; else capacity + 1
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  std::atomic<int64_t>* slot = dev >= 0 && dev < kCapacityDevices ? &cap[dev] : nullptr;
  const int64_t known = slot ? slot->load(std::memory_order_relaxed) : 0;
  if (known > 0) return known - 1;
  int n = 0, cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, plan_fused_kernel<V, SPREAD>, kScanThreads, 0) != hipSuccess)
    return 0;   // asked again next time
  const int64_t c = (int64_t)n * cus;
  if (slot) slot->store(c + 1, std::memory_order_relaxed);
  return c;
}

template <int V>
hipError_t launch_plan_v(const PlanArgs& a, hipStream_t s) {
  const unsigned blocks = (unsigned)a.p.nblk;
  if constexpr (V <= kPlanChunk) {
    if (blocks == 1) {
      hipLaunchKernelGGL(plan_single_kernel<V>, dim3(1), dim3(kScanThreads), 0, s, a);
      return hipGetLastError();
    }
  }
  if (blocks <= (unsigned)kPlanDirectTiles) {
    // one launch: every tile's block resident, or the first resident blocks
    // summing the tiles of those that start later
    if ((int64_t)blocks <= plan_fused_capacity<V, false>()) {
      hipLaunchKernelGGL((plan_fused_kernel<V, false>), dim3(blocks), dim3(kScanThreads), 0, s, a);
      return hipGetLastError();
    }
    const int64_t cap = plan_fused_capacity<V, true>();
    if (cap > 0) {
      PlanArgs b = a;
      b.p.reduce_blocks = (int32_t)cap;
      hipLaunchKernelGGL((plan_fused_kernel<V, true>), dim3(blocks), dim3(kScanThreads), 0, s, b);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL(plan_reduce_kernel<V>, dim3(blocks), dim3(kScanThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (blocks > (unsigned)kPlanDirectTiles) {
    hipLaunchKernelGGL(plan_tiles_kernel, dim3(1), dim3(kScanThreads), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(plan_scan_kernel<V>, dim3(blocks), dim3(kScanThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_plan(const PlanArgs& a, hipStream_t s) {
  if (a.p.nblk < 1) return hipErrorInvalidValue;
  if (!a.p.offsets) {
    // enough threads for the larger of the bag and wave arrays, grid-strided beyond
    const int64_t span = std::max<int64_t>(a.p.TB, a.p.waves_req) + 1;
    const int64_t blocks = std::min<int64_t>((span + kScanThreads - 1) / kScanThreads, 16384);
    hipLaunchKernelGGL(plan_onehot_kernel, dim3((unsigned)blocks), dim3(kScanThreads), 0, s, a);
    return hipGetLastError();
  }
  switch (a.p.slabs) {
    case 1: return launch_plan_v<1>(a, s);
    case 2: return launch_plan_v<2>(a, s);
    case 4: return launch_plan_v<4>(a, s);
    case 8: return launch_plan_v<8>(a, s);
    case 16: return launch_plan_v<16>(a, s);
    case 32: return launch_plan_v<32>(a, s);
    case 64: return launch_plan_v<64>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace dpi
