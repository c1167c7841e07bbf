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
constexpr int kPlanMaxSlabs = 64;           // most slabs per tile
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

// Status words in the workspace.  Word 0 (64 bits): device-latched error
// bits in the low kStatusTagShift bits, the id of the plan they belong to
// above them; a word holding another plan's id holds no error of this plan,
// so a plan needs no launch to clear it.  Word kStatusLongWord (32 bits): the
// bags of more than kDirectMaxItems items the planning launch counted.
constexpr int kStatusBadOffsets = 1;
constexpr int kStatusBadId = 2;
constexpr int kStatusTagShift = 24;
constexpr uint64_t kStatusBitsMask = (1ull << kStatusTagShift) - 1;
constexpr int64_t kPlanIdMask = ((int64_t)1 << (64 - kStatusTagShift)) - 1;
constexpr int kStatusLongWord = 2;

__host__ __device__ inline uint64_t status_word(int64_t plan_id, uint32_t bits) {
  return ((uint64_t)(plan_id & kPlanIdMask) << kStatusTagShift) | bits;
}

// One-launch batches: at most kSmallMaxFields fields (their static info
// travels in the kernel arguments) and, with offsets, at most kSmallMaxBatch
// bags per field (every wave of a field reads all of the field's offsets).
constexpr int kSmallMaxFields = 64;
constexpr int64_t kSmallMaxBatch = 1024;

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
  int32_t* status;       // [4]: the status words (kStatus*)
  TableInfo* tinfo;      // [T]
  int64_t* col_base;     // [T+1]
  int64_t* id_base;      // [T+1]
  int64_t* block_sum;    // [12 * nblk + 3]: per tile items, then costs, then malformed-offset flags; three
                         // totals (when the tiles are scanned by their own launch); per tile split bags;
                         // published sums (one-launch planning): per tile a pair of words, then per
                         // tile six words of the long form
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
  int32_t reduce_blocks;   // one-launch planner: blocks that sum tiles (0: every block its own tile)
  int64_t B;
  int64_t TB;
  int64_t total_ids;
  int64_t waves_req;
  int64_t total_d;
  int64_t plan_id;         // tags the status word
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
  int32_t xcd_affine;      // XCDs per contiguous range of blocks (1 or 2), 0: linear order
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
  uint32_t lpr_log[DPI_MAX_TABLES / 4];   // byte t & 3 of word t >> 2 (a dword: one scalar load)
};

// Kernel arguments of the one-launch lookups (small.hip): one-hot batches of
// one row class, and bag-by-bag batches whose fields all take the 16-byte row
// path.  Nothing of the batch is planned beforehand: the kernel derives each
// field's first id from the offsets, checks the offsets, and pools bags of
// more than long_rows ids in pieces of at most long_rows ids spread over the
// field's waves (fp32 partials combined by the last piece to arrive).
struct SmallArgs {
  const void* tables[kSmallMaxFields];
  uint32_t packed[kSmallMaxFields];     // dim | TableInfo flags << 17
  uint32_t nrows[kSmallMaxFields];      // min(num_rows, 2^31)
  int32_t col_base[kSmallMaxFields];
  uint32_t mean_bits[kSmallMaxFields / 32];
  const int32_t* ids;
  const int32_t* offsets;               // device [T][B+1], or nullptr (one id per bag)
  void* out;
  // a staged packed CSR read instead of offsets / ids (nullptr: none): its
  // dpi_x_dtype, and where the converted int32 offsets and ids go
  const void* staged;
  int32_t staged_dtype;
  int32_t* offsets_out;
  int32_t* ids_out;
  uint64_t* status;                     // status word 0
  uint64_t* tickets;                    // [slots] arrival counters of long bags (tagged like the status)
  float* partial;                       // [slots][dmax] fp32 sums of long-bag pieces
  int64_t slots;                        // 2 * ceil(total_ids / long_rows) + 2
  int64_t B;
  int64_t total_d;
  int64_t total_ids;
  int64_t tag;                          // the plan's id (masked by kPlanIdMask)
  int64_t long_rows;                    // kDirectMaxItems * C
  int32_t T;
  int32_t dmax;
  int32_t out_f16;
  int32_t xcd_affine;
  int32_t uniform_class;                // one-hot: the class shared by every field
  // bag by bag (as in LookupArgs)
  int32_t direct_plog;
  int32_t direct_jcap_log;
  int64_t direct_wpf;
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
hipError_t launch_lookup_small(const SmallArgs& a, hipStream_t s);
// *dst = the error bits of status word *word when it belongs to plan `tag`, else 0
hipError_t launch_status_out(const uint64_t* word, int64_t tag, int32_t* dst, hipStream_t s);
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
