// Internal definitions shared by the host API and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <stdint.h>

#include "dpi.h"

namespace dpi {

constexpr int kWaveSize = 64;
constexpr int kBlockThreads = 256;          // 4 independent waves per workgroup
constexpr int kWavesPerBlock = kBlockThreads / kWaveSize;
constexpr int kScanThreads = 256;           // plan: threads per block (one bag per thread per slab)
constexpr int kPlanMaxSlabs = 32;           // most slabs per tile
constexpr int kPlanChunk = 8;               // slabs whose offset loads are in flight together
constexpr int kPlanTargetTiles = 512;       // a tile grows until the batch has at most this many
constexpr int kPlanDirectTiles = 1024;      // most tiles whose sums every scan block reads itself
constexpr int kDefaultChunkRows = 32;
constexpr int kDefaultItemCost = 64;
constexpr int kDefaultRowsPerWave = 2048;
constexpr int kDefaultWavesPerCU = 16;
// Small batches are looked up bag by bag, without the plan's partition, when
// no bag holds more than kDirectMaxItems chunks of C ids (the plan counts the
// longer ones) and the batch has at most kDirectMaxBags bags (measured
// crossover against the partition: bag by bag is 8-12 % faster per step at
// 106 K and 160 K bags, 7 % slower at 213 K and 240 K).
constexpr int kDirectMaxItems = 4;
constexpr int kDirectGroupRows = 8;   // rows in flight per slot
constexpr int64_t kDirectMaxBags = 180000;

// status word bits (device-latched errors)
constexpr int kStatusBadOffsets = 1;
constexpr int kStatusBadId = 2;

// header16 slots
enum : int {
  kHdrAbi = 0, kHdrT, kHdrB, kHdrW, kHdrC, kHdrK, kHdrOutDtype, kHdrFlags, kHdrTotalD,
  kHdrItems, kHdrCost, kHdrTotalIds, kHdrSplit, kHdrWaveReq
};

// TableInfo.flags
constexpr int kTiF16 = 1 << 0;              // table dtype is binary16
constexpr int kTiFast = 1 << 1;             // row bytes multiple of 16 and <= 1024
constexpr int kTiLprShift = 2;              // log2(lanes per row), 3 bits
constexpr int kTiOutVec = 1 << 5;           // output rows allow vector stores

// Static description of a field, written to the workspace by the plan.
struct alignas(16) TableInfo {
  int64_t num_rows;
  int64_t id_base;     // first position of the field's ids
  int64_t nnz;         // number of ids of the field
  int32_t dim;
  int32_t col_base;
  int32_t row_bytes;
  int32_t out_bytes;
  int32_t flags;
  int32_t pad;
};

// Device pointers of a plan inside the caller's workspace.
struct PlanDev {
  int64_t* hdr;          // [16]
  int32_t* status;       // [4]: error bits; bags of more than kDirectMaxItems items; then the int64
                         // id of the plan that last planned into this workspace
  TableInfo* tinfo;      // [T]
  int64_t* col_base;     // [T+1]
  int64_t* id_base;      // [T+1]
  int64_t* block_sum;    // [10 * nblk + 3]: per tile items, then costs, then malformed-offset flags; three
                         // totals (when the tiles are scanned by their own launch); per tile split bags;
                         // per tile six words of published sums (one-launch planning)
  int64_t* bib;          // bag_item_base [TB+1]
  int64_t* bcb;          // bag_cost_base [TB+1]
  int64_t* wib;          // wave_item_begin [Wreq+1]
  int64_t* wave_bag;     // bag holding wib[w], [Wreq+1]
  int64_t* wbase;        // first item of bag wave_bag[w], [Wreq+1] (what a lookup needs of bib)
  int32_t* head_first;   // [Wreq] first wave of the bag this wave starts inside, or -1
  int32_t* split_pieces; // [Wreq] for the first wave of a split bag: nonempty waves covering it
  int32_t* split_last;   // [Wreq] ... and the last of them
  int32_t* tickets;      // [Wreq] arrival counters of split bags (zero between lookups)
  float* partial;        // [2 * Wreq][dmax] fp32 partial sums of split bags
};

struct PlanParams {
  int32_t T;
  int32_t C;
  int32_t K;
  int32_t out_dtype;
  uint32_t flags;
  int32_t nblk;       // tiles of slabs * kScanThreads bags (at least 1)
  int32_t slabs;      // bags per thread: 1, 2, 4, ..., kPlanMaxSlabs
  int32_t c_shift;    // log2(C) when C is a power of two, else -1
  int32_t lazy_partition;  // skip the bag prefixes and the wave partition when no bag is longer than
                           // kDirectMaxItems items (the lookup kernel does not read them)
  int32_t prefixes;        // write the per-bag prefixes bib / bcb (read only by an export)
  int64_t B;
  int64_t TB;
  int64_t total_ids;
  int64_t waves_req;
  int64_t total_d;
  int64_t plan_id;         // written next to the status words: tells a plan whether its workspace
                           // still holds it
  const int32_t* offsets;  // device [T][B+1] or nullptr
};

// Kernel arguments of both planning launches.  packed[t] = dim | flags << 17
// (flags as in TableInfo).
struct PlanArgs {
  PlanParams p;
  PlanDev d;
  uint32_t packed[DPI_MAX_TABLES];
  int64_t num_rows[DPI_MAX_TABLES];
};

struct LookupArgs {
  const void* tables[DPI_MAX_TABLES];
  uint32_t mean_bits[DPI_MAX_TABLES / 32];
  const int32_t* ids;
  const int32_t* offsets;
  void* out;
  const int64_t* hdr;
  int32_t* status;
  const TableInfo* tinfo;
  const int64_t* wbase;
  const int64_t* wib;
  const int64_t* wave_bag;
  const int32_t* head_first;
  const int32_t* split_pieces;
  const int32_t* split_last;
  int32_t* tickets;
  float* partial;
  int64_t B;
  int64_t total_d;
  int32_t T;
  int32_t C;
  int32_t dmax;
  int32_t out_f16;
  int32_t xcd_affine;
  int32_t uniform_class;   // TableInfo class bits shared by every field, or -1
  int32_t input_first;     // one lane per bag instead of the plan's waves
  int32_t onehot;          // no offsets: every bag holds one id
  int64_t grid_waves;
  // bag by bag (direct_plog >= 0; -1: the plan's partition): field t's waves
  // take J_t = min(G_t >> direct_plog, 2^direct_jcap_log) bags each, G_t = 64
  // >> lpr_log[t] slots per wave; every field has direct_wpf waves (enough for
  // the field with the fewest slots; the others leave their last ones idle)
  int32_t direct_plog;
  int32_t direct_jcap_log;
  int64_t direct_wpf;
  uint8_t lpr_log[DPI_MAX_TABLES];
};

// Second-order FM term over a [B, row_stride] block of T fields of dim D.
struct FmArgs {
  const void* emb;
  float* out;
  int64_t B;
  int64_t row_stride;   // elements
  int32_t T;
  int32_t dim;
  int32_t f16;
  int32_t lpr_log;      // log2 of lanes per field row on the 16-byte path, -1: column path
};

// One-hot input consolidation: sample-major device matrix -> field-major ids.
struct StageArgs {
  const void* x;        // device copy of the host matrix
  int32_t* ids;         // [T * B]
  int64_t B;
  int64_t row_stride;   // elements
  int32_t T;
  int32_t x_dtype;      // dpi_x_dtype
};

// Slabs per plan tile (bags per plan thread), a power of two.  A batch of at
// most kPlanChunk slabs is one tile, planned by a single block in one launch;
// a larger one takes the fewest slabs (at most kPlanMaxSlabs) that keep the
// tile count at most kPlanTargetTiles.
inline int32_t plan_slabs(int64_t TB) {
  int32_t s = 1;
  if (TB <= (int64_t)kScanThreads * kPlanChunk) {
    while ((int64_t)kScanThreads * s < TB) s <<= 1;
    return s;
  }
  while (s < kPlanMaxSlabs && (TB + (int64_t)kScanThreads * s - 1) / ((int64_t)kScanThreads * s) > kPlanTargetTiles)
    s <<= 1;
  return s;
}

// Plan tiles of a batch of TB bags (at least one, so an empty batch still
// runs the block that writes the header).
inline int64_t plan_tiles(int64_t TB) {
  const int64_t tile = (int64_t)kScanThreads * plan_slabs(TB);
  const int64_t n = (TB + tile - 1) / tile;
  return n > 1 ? n : 1;
}

// kernel launchers (plan.hip / lookup.hip); return the launch's hipError_t
hipError_t launch_plan(const PlanArgs& a, hipStream_t s);
hipError_t launch_lookup(const LookupArgs& a, hipStream_t s);
hipError_t launch_fm(const FmArgs& a, hipStream_t s);
hipError_t launch_stage(const StageArgs& a, hipStream_t s);
hipError_t launch_stage_csr(const void* src, int32_t x_dtype, int64_t n_off, int64_t n_ids, int32_t* offsets,
                            int32_t* ids, hipStream_t s);
// interaction modules' fused element-wise operators (16-byte alignment of all
// pointers is required when n is a multiple of 4)
hipError_t launch_cross_fuse(const float* x0, const float* y, const float* bias, const float* x, float* out,
                             int64_t rows, int32_t n, hipStream_t s);
hipError_t launch_bias_relu(float* z, const float* bias, int64_t rows, int32_t n, hipStream_t s);
hipError_t launch_mark(uint64_t* slot, hipStream_t s);

}  // namespace dpi
