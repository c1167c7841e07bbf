// Host side of the C ABI declared in include/dpi.h: argument validation,
// workspace layout, kernel launches on the caller's stream, plan export.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <unordered_map>
#include <vector>

#include "dpi_internal.h"

using namespace dpi;

namespace {

thread_local char g_last_error[512] = "";

dpi_status fail(dpi_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

dpi_status hip_fail(hipError_t e, const char* what) {
  return fail(DPI_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

constexpr int64_t kSmallBagsPerWave = 8;   // default-wave rule for small batches

struct Layout {
  size_t hdr, status, tinfo, col_base, id_base, block_sum, bib, bcb, wib, wave_bag, wbase, head_first, split_pieces,
      split_last, tickets, partial, small_tickets, small_partial, total;
  int64_t small_slots;   // long-bag piece slots of a one-launch lookup (0: no one-launch bag-by-bag lookup)
};

// Piece slots a one-launch bag-by-bag lookup of this batch needs (two per
// window of long_rows ids), or 0 when such a batch is planned by its own
// launch: more than kSmallMaxFields fields or kSmallMaxBatch bags per field,
// an explicit wave count, the input-first allocation, or so many windows that
// a bag's piece count could overflow its ticket.
int64_t small_slots(int64_t T, int64_t B, int64_t total_ids, const dpi_plan_opts& o, bool waves_given) {
  if (T > kSmallMaxFields || B < 1 || B > kSmallMaxBatch || waves_given || (o.flags & DPI_FLAG_INPUT_FIRST))
    return 0;
  const int64_t pr = (int64_t)kDirectMaxItems * o.chunk_rows;
  const int64_t windows = (total_ids + pr - 1) / pr;
  if (windows >= ((int64_t)1 << 22)) return 0;
  return 2 * windows + 2;
}

// o: resolved options.  prefixes: room for the per-bag prefixes, which only an
// export writes (the no-allocation entry point never exports, and leaves them
// out).
Layout make_layout(int64_t T, int64_t B, int64_t total_ids, const dpi_plan_opts& o, bool waves_given, int64_t dmax,
                   bool prefixes = true) {
  Layout L{};
  const int64_t waves_req = o.num_waves;
  const int64_t TB = T * B;
  const int64_t nblk = plan_tiles(TB);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align256(off + bytes);
    return at;
  };
  L.hdr = take(16 * sizeof(int64_t));
  L.status = take(2 * sizeof(int32_t) + sizeof(int64_t));
  L.tinfo = take(T * sizeof(TableInfo));
  L.col_base = take((T + 1) * sizeof(int64_t));
  L.id_base = take((T + 1) * sizeof(int64_t));
  L.block_sum = take((12 * nblk + 3) * sizeof(int64_t));
  L.bib = take(prefixes ? (TB + 1) * sizeof(int64_t) : 0);
  L.bcb = take(prefixes ? (TB + 1) * sizeof(int64_t) : 0);
  L.wib = take((waves_req + 1) * sizeof(int64_t));
  L.wave_bag = take((waves_req + 1) * sizeof(int64_t));
  L.wbase = take((waves_req + 1) * sizeof(int64_t));
  L.head_first = take(waves_req * sizeof(int32_t));
  L.split_pieces = take(waves_req * sizeof(int32_t));
  L.split_last = take(waves_req * sizeof(int32_t));
  L.tickets = take(waves_req * sizeof(int32_t));
  L.partial = take(2 * waves_req * dmax * sizeof(float));
  L.small_slots = small_slots(T, B, total_ids, o, waves_given);
  L.small_tickets = take(L.small_slots * sizeof(uint64_t));
  L.small_partial = take(L.small_slots * dmax * sizeof(float));
  L.total = off;
  return L;
}

int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return 256;
  return cus;
}

int ilog2(int x) {
  int l = 0;
  while ((1 << l) < x) ++l;
  return l;
}

// The plan that last planned into each workspace (by address): a plan whose
// workspace holds a later one is refused by dpi_lookup, the status query and
// the export.
std::mutex g_holder_mu;
std::unordered_map<uintptr_t, int64_t> g_holder;

void set_holder(const void* ws, int64_t plan_id) {
  std::lock_guard<std::mutex> lock(g_holder_mu);
  g_holder[reinterpret_cast<uintptr_t>(ws)] = plan_id;
}

bool is_holder(const void* ws, int64_t plan_id) {
  std::lock_guard<std::mutex> lock(g_holder_mu);
  const auto it = g_holder.find(reinterpret_cast<uintptr_t>(ws));
  return it != g_holder.end() && it->second == plan_id;
}

dpi_status superseded() {
  return fail(DPI_ERR_INVALID_ARG, "the plan's workspace holds a later plan: a plan is used up when another plan "
                                   "is built into its workspace");
}

void drop_holder(const void* ws, int64_t plan_id) {
  std::lock_guard<std::mutex> lock(g_holder_mu);
  const auto it = g_holder.find(reinterpret_cast<uintptr_t>(ws));
  if (it != g_holder.end() && it->second == plan_id) g_holder.erase(it);
}

}  // namespace

// error helpers for the other host files (not part of the C ABI)
__attribute__((visibility("hidden"))) dpi_status dpi_fail_status(dpi_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

__attribute__((visibility("hidden"))) dpi_status dpi_hip_status(hipError_t e, const char* what) {
  return hip_fail(e, what);
}

struct dpi_plan_s {
  int32_t T;
  int64_t B;
  int64_t total_ids;
  int64_t waves_req;
  int32_t C, K, out_dtype;
  uint32_t flags;
  int32_t dmax;
  int64_t total_d;
  bool onehot;
  int32_t uniform_class;   // shared row class of every field, or -1
  int32_t direct_jlog;     // small batches looked up bag by bag: log2 of bags per wave, or -1
  int32_t direct_jcap_log; // ... log2 of the most bags a wave of any field takes
  int64_t plan_id;         // unique in the process; tags the workspace's status word
  int32_t sticky_status;   // status bits latched by lookups before a re-plan
  bool partitioned;        // the plan has been planned again in full (first export)
  // one launch per lookup: dpi_plan enqueued nothing, each lookup checks the
  // offsets itself (small_args holds everything of a lookup but the batch's
  // pointers)
  bool one_launch;
  bool looked_up;          // a lookup has been enqueued
  bool validated;          // the status query ran the planning launch (no lookup before it)
  SmallArgs small_args;
  const int32_t* offsets_arg;   // the offsets pointer given to dpi_plan
  // the partition as the planning launch wrote it (what lookups read), copied
  // before the first export plans again; empty when that launch wrote none
  bool snap_valid;
  std::vector<int64_t> snap_wib, snap_wave_bag, snap_wbase;
  std::vector<int32_t> snap_head_first, snap_split_pieces, snap_split_last;
  PlanArgs args;           // the planning launch (re-run in full on export)
  hipStream_t stream;
  char* ws;
  Layout layout;
  int32_t row_class[DPI_MAX_TABLES];
};

// Small batches (at most kDirectMaxBags bags, every field on the 16-byte row
// path) are looked up bag by bag when the caller left the wave count to the
// library: a wave takes J = 2^jlog bags of one field, each pooled by G/J row
// slots, where G = 64 / (row bytes / 16) is the field's slot count.  J (at
// most the smallest G) is chosen so that an average bag needs about one group
// of 8 rows per slot, then doubled while the grid holds more than
// kDefaultWavesPerCU waves per compute unit, and no larger than the batch.
// Every field gets the waves this J needs; when that grid is several times
// what the GPU holds, fields with more slots take more bags per wave at the
// same slots per bag (dpi_plan sets the cap) and leave their last waves idle.
// Returns jlog, or -1 for the plan's partition (also the choice for one-hot
// batches of one row class, which have their own kernel, and for the
// input-first allocation).
int32_t direct_jlog(int32_t T, int64_t B, int64_t total_ids, const int32_t* row_class, bool onehot,
                    int32_t uniform_class, uint32_t flags, bool waves_given) {
  if (waves_given || (flags & DPI_FLAG_INPUT_FIRST) || (onehot && uniform_class >= 0)) return -1;
  if (B < 1 || (int64_t)T * B > kDirectMaxBags) return -1;
  int gmin = kWaveSize;
  for (int t = 0; t < T; ++t) {
    if (!(row_class[t] & kTiFast)) return -1;
    gmin = std::min(gmin, kWaveSize >> ((row_class[t] >> kTiLprShift) & 7));
  }
  const int64_t bags = (int64_t)T * B;
  const int64_t avg = (total_ids + bags - 1) / bags;          // ids per bag, rounded up
  int64_t slots = 1;                                          // slots an average bag fills with groups of 8
  while (slots * kDirectGroupRows < avg && slots < gmin) slots <<= 1;
  int64_t J = std::max<int64_t>(1, gmin / slots);
  // larger batches: more bags per wave (up to one per slot) until the grid
  // is no larger than the partition's default for mid-size batches
  while (J < gmin && (int64_t)T * ((B + J - 1) / J) > (int64_t)kDefaultWavesPerCU * device_cus()) J <<= 1;
  while (J > 1 && J > B) J >>= 1;
  return ilog2((int)J);
}

extern "C" {

int dpi_abi_version(void) { return DPI_ABI_VERSION; }

const char* dpi_last_error(void) { return g_last_error; }

const char* dpi_status_str(dpi_status s) {
  switch (s) {
    case DPI_OK: return "ok";
    case DPI_ERR_INVALID_ARG: return "invalid argument";
    case DPI_ERR_UNSUPPORTED: return "unsupported table shape";
    case DPI_ERR_MISALIGNED: return "misaligned pointer";
    case DPI_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case DPI_ERR_BAD_OFFSETS: return "malformed offsets";
    case DPI_ERR_BAD_ID: return "id out of range";
    case DPI_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

int64_t dpi_default_waves(int32_t num_tables, int64_t batch, int64_t total_ids) {
  const int64_t units = total_ids + (int64_t)num_tables * batch;
  // large batches: about kDefaultRowsPerWave rows and bags per wave.  Small
  // ones: enough waves for the GPU, but at least ~8 bags per wave (fewer,
  // shorter waves cut bags between waves, and a cut bag costs a cross-wave
  // combine) and few fields per wave when batches are tiny (a wave walks its
  // fields one after the other).
  const int64_t by_work = (units + kDefaultRowsPerWave - 1) / kDefaultRowsPerWave;
  const int64_t bags = (int64_t)num_tables * batch;
  const int64_t items_bound = (total_ids + kDefaultChunkRows - 1) / kDefaultChunkRows + bags;
  const int64_t by_bags = std::max<int64_t>((bags + kSmallBagsPerWave - 1) / kSmallBagsPerWave,
                                            std::min<int64_t>(items_bound, kSmallBagsPerWave * num_tables));
  const int64_t fill = std::min<int64_t>((int64_t)kDefaultWavesPerCU * device_cus(), by_bags);
  return std::max<int64_t>(std::max<int64_t>(fill, by_work), 1);
}

static dpi_status resolve_opts(const dpi_plan_opts* opts, int32_t T, int64_t B, int64_t total_ids,
                               dpi_plan_opts& o) {
  o = dpi_plan_opts{};
  if (opts) o = *opts;
  if (o.chunk_rows < 0 || o.item_cost_k < 0 || o.num_waves < 0)
    return fail(DPI_ERR_INVALID_ARG, "negative plan option");
  if (o.out_dtype != DPI_F32 && o.out_dtype != DPI_F16) return fail(DPI_ERR_INVALID_ARG, "bad out_dtype");
  if (o.flags & ~(uint32_t)(DPI_FLAG_EXACT_SPLIT | DPI_FLAG_LINEAR_BLOCKS | DPI_FLAG_INPUT_FIRST))
    return fail(DPI_ERR_INVALID_ARG, "unknown flag bits 0x%x", o.flags);
  if (o.chunk_rows == 0) o.chunk_rows = kDefaultChunkRows;
  if (o.item_cost_k == 0) o.item_cost_k = kDefaultItemCost;
  if (o.num_waves == 0) o.num_waves = dpi_default_waves(T, B, total_ids);
  if (o.num_waves > ((int64_t)1 << 31) - 2) return fail(DPI_ERR_UNSUPPORTED, "too many waves");
  return DPI_OK;
}

size_t dpi_plan_workspace_bytes(int32_t num_tables, int64_t batch, int64_t total_ids, int32_t max_dim,
                                const dpi_plan_opts* opts) {
  if (num_tables < 1 || num_tables > DPI_MAX_TABLES || batch < 0 || total_ids < 0 || max_dim < 1 ||
      max_dim > DPI_MAX_DIM)
    return 0;
  dpi_plan_opts o;
  if (resolve_opts(opts, num_tables, batch, total_ids, o) != DPI_OK) return 0;
  return make_layout(num_tables, batch, total_ids, o, opts && opts->num_waves != 0, max_dim).total;
}

}  // extern "C"

// Validate a batch, fill *plan (caller-owned storage) and, unless its lookups
// take one launch each, enqueue the planning launch into `workspace`;
// allocates nothing.  prefixes: the workspace has room for the per-bag
// prefixes (plans that may be exported).
static dpi_status plan_init(dpi_plan_s* plan, const dpi_table_meta* table_meta, int32_t num_tables,
                            const int32_t* offsets, int64_t batch, int64_t total_ids, const dpi_plan_opts* opts,
                            void* workspace, size_t workspace_bytes, void* stream, bool prefixes) {
  if (!table_meta) return fail(DPI_ERR_INVALID_ARG, "table_meta is NULL");
  if (num_tables < 1 || num_tables > DPI_MAX_TABLES)
    return fail(DPI_ERR_INVALID_ARG, "num_tables %d outside [1, %d]", num_tables, DPI_MAX_TABLES);
  if (batch < 0) return fail(DPI_ERR_INVALID_ARG, "negative batch");
  if (batch > ((int64_t)1 << 31) - 2) return fail(DPI_ERR_UNSUPPORTED, "batch too large");
  if (total_ids < 0) return fail(DPI_ERR_INVALID_ARG, "negative total_ids");
  if (!offsets && total_ids != (int64_t)num_tables * batch)
    return fail(DPI_ERR_INVALID_ARG, "one-hot batch needs total_ids == T*B");
  if (offsets && (reinterpret_cast<uintptr_t>(offsets) & 3))
    return fail(DPI_ERR_MISALIGNED, "offsets not 4-byte aligned");
  dpi_plan_opts o;
  dpi_status st = resolve_opts(opts, num_tables, batch, total_ids, o);
  if (st != DPI_OK) return st;
  const int osize = o.out_dtype == DPI_F16 ? 2 : 4;

  int64_t col = 0;
  int32_t dmax = 1;
  int64_t col_base[DPI_MAX_TABLES];
  int32_t row_class[DPI_MAX_TABLES];
  for (int t = 0; t < num_tables; ++t) {
    const dpi_table_meta& m = table_meta[t];
    if (m.dtype != DPI_F32 && m.dtype != DPI_F16) return fail(DPI_ERR_INVALID_ARG, "table %d: bad dtype", t);
    if (m.dim < 1) return fail(DPI_ERR_INVALID_ARG, "table %d: dim < 1", t);
    if (m.dim > DPI_MAX_DIM) return fail(DPI_ERR_UNSUPPORTED, "table %d: dim > %d", t, DPI_MAX_DIM);
    if (m.num_rows < 0) return fail(DPI_ERR_INVALID_ARG, "table %d: negative num_rows", t);
    const int esize = m.dtype == DPI_F16 ? 2 : 4;
    const int64_t row_bytes = (int64_t)m.dim * esize;
    if (row_bytes % 4) return fail(DPI_ERR_UNSUPPORTED, "table %d: row of %lld bytes is not a multiple of 4", t,
                                   (long long)row_bytes);
    int flags = m.dtype == DPI_F16 ? kTiF16 : 0;
    if (row_bytes % 16 == 0 && row_bytes <= 1024) {
      flags |= kTiFast;
      flags |= ilog2((int)(row_bytes / 16)) << kTiLprShift;
    }
    row_class[t] = flags;
    col_base[t] = col;
    col += m.dim;
    if (col > ((int64_t)1 << 31) - 1) return fail(DPI_ERR_UNSUPPORTED, "sum of dims too large");
    dmax = std::max(dmax, m.dim);
  }
  const int64_t total_d = col;
  // vector stores need every output row piece aligned to min(16, bytes per lane)
  for (int t = 0; t < num_tables; ++t) {
    int flags = row_class[t];
    if (flags & kTiFast) {
      const int epl = (flags & kTiF16) ? 8 : 4;
      const int64_t a = std::min(16, epl * osize);
      if ((total_d * osize) % a == 0 && (col_base[t] * osize) % a == 0) flags |= kTiOutVec;
    }
    row_class[t] = flags;
  }

  // one specialised kernel serves batches whose fields share a row class and
  // fit a buffer descriptor (at most 4 GiB - 1 bytes each)
  const int class_mask = kTiF16 | kTiFast | (7 << kTiLprShift);
  int32_t uniform_class = row_class[0] & class_mask;
  for (int t = 0; t < num_tables; ++t) {
    const int64_t bytes = table_meta[t].num_rows * (int64_t)table_meta[t].dim * (table_meta[t].dtype == DPI_F16 ? 2 : 4);
    if (!(row_class[t] & kTiFast) || (row_class[t] & class_mask) != uniform_class || bytes > (int64_t)0xffffffffLL)
      uniform_class = -1;
  }

  const bool waves_given = opts && opts->num_waves != 0;
  const Layout L = make_layout(num_tables, batch, total_ids, o, waves_given, dmax, prefixes);
  if (!workspace) return fail(DPI_ERR_INVALID_ARG, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) & 15) return fail(DPI_ERR_MISALIGNED, "workspace not 16-byte aligned");
  if (workspace_bytes < L.total)
    return fail(DPI_ERR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", workspace_bytes, L.total);

  plan->T = num_tables;
  plan->B = batch;
  plan->total_ids = total_ids;
  plan->waves_req = o.num_waves;
  plan->C = o.chunk_rows;
  plan->K = o.item_cost_k;
  plan->out_dtype = o.out_dtype;
  plan->flags = o.flags;
  plan->dmax = dmax;
  plan->total_d = total_d;
  plan->onehot = offsets == nullptr;
  plan->offsets_arg = offsets;
  plan->uniform_class = uniform_class;
  plan->direct_jlog = direct_jlog(num_tables, batch, total_ids, row_class, offsets == nullptr, uniform_class,
                                  o.flags, waves_given);
  plan->direct_jcap_log = plan->direct_jlog;
  if (plan->direct_jlog >= 0) {
    // a grid of several times the waves the GPU holds: fields with more slots
    // than the smallest take more bags per wave (up to the batch size), so
    // fewer, fuller waves amortise their prologues; below that, spreading the
    // bags over more waves is faster
    const int64_t wpf = (batch + (1 << plan->direct_jlog) - 1) >> plan->direct_jlog;
    if ((int64_t)num_tables * wpf > 4 * (int64_t)kDefaultWavesPerCU * device_cus()) {
      int jcap_log = 0;
      while (jcap_log < 6 && ((int64_t)2 << jcap_log) <= batch) ++jcap_log;
      plan->direct_jcap_log = std::max(jcap_log, plan->direct_jlog);
    }
  }
  plan->stream = reinterpret_cast<hipStream_t>(stream);
  plan->ws = reinterpret_cast<char*>(workspace);
  plan->layout = L;
  std::memcpy(plan->row_class, row_class, sizeof(int32_t) * num_tables);

  char* ws = plan->ws;
  PlanDev d;
  d.hdr = reinterpret_cast<int64_t*>(ws + L.hdr);
  d.status = reinterpret_cast<int32_t*>(ws + L.status);
  d.tinfo = reinterpret_cast<TableInfo*>(ws + L.tinfo);
  d.col_base = reinterpret_cast<int64_t*>(ws + L.col_base);
  d.id_base = reinterpret_cast<int64_t*>(ws + L.id_base);
  d.block_sum = reinterpret_cast<int64_t*>(ws + L.block_sum);
  d.bib = reinterpret_cast<int64_t*>(ws + L.bib);
  d.bcb = reinterpret_cast<int64_t*>(ws + L.bcb);
  d.wib = reinterpret_cast<int64_t*>(ws + L.wib);
  d.wave_bag = reinterpret_cast<int64_t*>(ws + L.wave_bag);
  d.wbase = reinterpret_cast<int64_t*>(ws + L.wbase);
  d.head_first = reinterpret_cast<int32_t*>(ws + L.head_first);
  d.split_pieces = reinterpret_cast<int32_t*>(ws + L.split_pieces);
  d.split_last = reinterpret_cast<int32_t*>(ws + L.split_last);
  d.tickets = reinterpret_cast<int32_t*>(ws + L.tickets);
  d.partial = reinterpret_cast<float*>(ws + L.partial);

  PlanArgs pa;
  std::memset(&pa, 0, sizeof(pa));
  PlanParams& p = pa.p;
  p.T = num_tables;
  p.C = o.chunk_rows;
  p.K = o.item_cost_k;
  p.c_shift = (o.chunk_rows & (o.chunk_rows - 1)) == 0 ? ilog2(o.chunk_rows) : -1;
  p.out_dtype = o.out_dtype;
  p.flags = o.flags;
  p.B = batch;
  p.TB = (int64_t)num_tables * batch;
  p.slabs = plan_slabs(p.TB);
  p.nblk = (int32_t)plan_tiles(p.TB);
  p.total_ids = total_ids;
  p.waves_req = o.num_waves;
  p.total_d = total_d;
  static std::atomic<int64_t> next_plan_id{1};
  plan->plan_id = next_plan_id.fetch_add(1, std::memory_order_relaxed);
  p.plan_id = plan->plan_id;
  p.offsets = offsets;
  // lookups that never read the partition: bag by bag, the one-hot kernel,
  // the input-first allocation (the latter two never split a bag either)
  const bool onehot_kernel = offsets == nullptr && uniform_class >= 0 && !(o.flags & DPI_FLAG_INPUT_FIRST);
  const bool input_first = (o.flags & DPI_FLAG_INPUT_FIRST) != 0;
  p.lazy_partition = (plan->direct_jlog >= 0 || onehot_kernel || input_first) ? 1 : 0;
  p.prefixes = 0;   // lookups read only the bases of the waves' first bags
  pa.d = d;
  for (int t = 0; t < num_tables; ++t) {
    pa.packed[t] = (uint32_t)table_meta[t].dim | ((uint32_t)row_class[t] << 17);
    pa.num_rows[t] = table_meta[t].num_rows;
  }
  plan->args = pa;
  // One launch per lookup (no planning launch) for one-hot batches of one row
  // class and for bag-by-bag batches, when the fields' info fits the kernel
  // arguments and, with offsets, the batch fits the lookup's own offset scan.
  const bool small_fields = num_tables <= kSmallMaxFields;
  plan->one_launch = small_fields && batch > 0 &&
                     (onehot_kernel || (plan->direct_jlog >= 0 && (offsets == nullptr || L.small_slots > 0)));
  plan->looked_up = false;
  plan->validated = false;
  if (plan->one_launch) {
    SmallArgs& sa = plan->small_args;
    std::memset(&sa, 0, sizeof(sa));
    for (int t = 0; t < num_tables; ++t) {
      sa.packed[t] = pa.packed[t];
      sa.nrows[t] = (uint32_t)std::min<int64_t>(table_meta[t].num_rows, (int64_t)1 << 31);
      sa.col_base[t] = (int32_t)col_base[t];
    }
    sa.status = reinterpret_cast<uint64_t*>(ws + L.status);
    sa.tickets = reinterpret_cast<uint64_t*>(ws + L.small_tickets);
    sa.partial = reinterpret_cast<float*>(ws + L.small_partial);
    sa.slots = L.small_slots;
    sa.B = batch;
    sa.total_d = total_d;
    sa.total_ids = total_ids;
    sa.tag = plan->plan_id & kPlanIdMask;
    sa.long_rows = (int64_t)kDirectMaxItems * o.chunk_rows;
    sa.T = num_tables;
    sa.dmax = dmax;
    sa.out_f16 = o.out_dtype == DPI_F16;
    sa.xcd_affine = (o.flags & DPI_FLAG_LINEAR_BLOCKS) ? 0 : 1;
    sa.uniform_class = onehot_kernel ? uniform_class : -1;
    sa.direct_plog = -1;
    if (plan->direct_jlog >= 0) {
      int glog_min = 6;
      for (int t = 0; t < num_tables; ++t) glog_min = std::min(glog_min, 6 - ((row_class[t] >> kTiLprShift) & 7));
      sa.direct_plog = glog_min - plan->direct_jlog;
      sa.direct_jcap_log = plan->direct_jcap_log;
      sa.direct_wpf = (batch + (1 << plan->direct_jlog) - 1) >> plan->direct_jlog;
    }
    return DPI_OK;
  }
  const hipError_t e = launch_plan(pa, plan->stream);
  if (e != hipSuccess) return hip_fail(e, "plan launch");
  return DPI_OK;
}

// A staged packed CSR a one-launch lookup reads instead of int32 offsets and
// ids (dpi_lookup_csr).
struct StagedInput {
  const void* data;
  int32_t x_dtype;
};

// Enqueue the fused lookup of a plan; allocates nothing.  staged: read the
// batch from a staged packed CSR and write the converted int32 arrays to
// offsets / ids (one-launch plans only).
static dpi_status lookup_enqueue(dpi_plan_s* plan, const void* const* tables, const int32_t* ids,
                                 const int32_t* offsets, const int32_t* pooling, void* out, void* stream,
                                 const StagedInput* staged = nullptr) {
  if (!tables) return fail(DPI_ERR_INVALID_ARG, "tables is NULL");
  if ((offsets == nullptr) != plan->onehot)
    return fail(DPI_ERR_INVALID_ARG, "offsets must be NULL exactly when the plan was built without offsets");
  if (plan->total_ids > 0 && !ids) return fail(DPI_ERR_INVALID_ARG, "ids is NULL");
  if (ids && (reinterpret_cast<uintptr_t>(ids) & 3)) return fail(DPI_ERR_MISALIGNED, "ids not 4-byte aligned");
  if (plan->B > 0 && !out) return fail(DPI_ERR_INVALID_ARG, "out is NULL");
  LookupArgs a{};
  for (int t = 0; t < plan->T; ++t) {
    if (!tables[t]) return fail(DPI_ERR_INVALID_ARG, "tables[%d] is NULL", t);
    if (reinterpret_cast<uintptr_t>(tables[t]) & 15) return fail(DPI_ERR_MISALIGNED, "tables[%d] not 16-byte aligned", t);
    a.tables[t] = tables[t];
    const int32_t pm = pooling ? pooling[t] : DPI_POOL_SUM;
    if (pm != DPI_POOL_SUM && pm != DPI_POOL_MEAN) return fail(DPI_ERR_INVALID_ARG, "pooling[%d] invalid", t);
    if (pm == DPI_POOL_MEAN) a.mean_bits[t >> 5] |= 1u << (t & 31);
  }
  if (out && (reinterpret_cast<uintptr_t>(out) & 15)) return fail(DPI_ERR_MISALIGNED, "out not 16-byte aligned");
  if (plan->B == 0 || plan->waves_req == 0) return DPI_OK;
  if (plan->one_launch) {
    SmallArgs sa = plan->small_args;
    for (int t = 0; t < plan->T; ++t) sa.tables[t] = tables[t];
    for (int q = 0; q < kSmallMaxFields / 32; ++q) sa.mean_bits[q] = a.mean_bits[q];
    sa.ids = ids;
    sa.offsets = offsets;
    sa.out = out;
    if (staged) {
      sa.staged = staged->data;
      sa.staged_dtype = staged->x_dtype;
      sa.offsets_out = const_cast<int32_t*>(offsets);
      sa.ids_out = const_cast<int32_t*>(ids);
    }
    const hipError_t e = launch_lookup_small(sa, reinterpret_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "lookup launch");
    plan->looked_up = true;
    return DPI_OK;
  }
  const Layout& L = plan->layout;
  char* ws = plan->ws;
  a.ids = ids;
  a.offsets = offsets;
  a.out = out;
  a.hdr = reinterpret_cast<const int64_t*>(ws + L.hdr);
  a.status = reinterpret_cast<int32_t*>(ws + L.status);
  a.tinfo = reinterpret_cast<const TableInfo*>(ws + L.tinfo);
  a.wib = reinterpret_cast<const int64_t*>(ws + L.wib);
  a.wave_bag = reinterpret_cast<const int64_t*>(ws + L.wave_bag);
  a.wbase = reinterpret_cast<const int64_t*>(ws + L.wbase);
  a.head_first = reinterpret_cast<const int32_t*>(ws + L.head_first);
  a.split_pieces = reinterpret_cast<const int32_t*>(ws + L.split_pieces);
  a.split_last = reinterpret_cast<const int32_t*>(ws + L.split_last);
  a.tickets = reinterpret_cast<int32_t*>(ws + L.tickets);
  a.partial = reinterpret_cast<float*>(ws + L.partial);
  a.B = plan->B;
  a.total_d = plan->total_d;
  a.T = plan->T;
  a.C = plan->C;
  a.dmax = plan->dmax;
  a.out_f16 = plan->out_dtype == DPI_F16;
  // XCD-grouped block order: one XCD per range, or a pair of XCDs per range
  // for rows of at most 128 bytes in one row class (the multi-hot workload's
  // lookup 60.0 -> 57.5 us; the large workload's 256-byte rows, one-hot and
  // bag-by-bag batches gain nothing from pairs)
  const bool small_rows = plan->uniform_class >= 0 && ((plan->uniform_class >> kTiLprShift) & 7) <= 3;
  a.xcd_affine = (plan->flags & DPI_FLAG_LINEAR_BLOCKS) ? 0 : (small_rows ? 2 : 1);
  a.input_first = (plan->flags & DPI_FLAG_INPUT_FIRST) ? 1 : 0;
  a.onehot = plan->onehot ? 1 : 0;
  a.uniform_class = plan->uniform_class;
  // the plan has W = min(requested, N) waves, and N = sum over bags of
  // max(1, ceil(L / C)) <= ceil(total_ids / C) + T * B: launch no more
  a.grid_waves = std::min<int64_t>(plan->waves_req,
                                   (plan->total_ids + plan->C - 1) / plan->C + (int64_t)plan->T * plan->B);
  a.direct_plog = -1;
  if (plan->direct_jlog >= 0) {
    // J = 2^direct_jlog bags per wave in the field with the fewest slots
    // (gmin), i.e. P = gmin / J slots per bag; a field with more slots takes
    // more bags per wave at the same P, up to the batch size
    int glog_min = 6;
    for (int t = 0; t < plan->T; ++t) glog_min = std::min(glog_min, 6 - ((plan->row_class[t] >> kTiLprShift) & 7));
    a.direct_plog = glog_min - plan->direct_jlog;
    a.direct_jcap_log = plan->direct_jcap_log;
    a.direct_wpf = (plan->B + (1 << plan->direct_jlog) - 1) >> plan->direct_jlog;
    for (int t = 0; t < plan->T; ++t)
      a.lpr_log[t >> 2] |= (uint32_t)((plan->row_class[t] >> kTiLprShift) & 7) << (8 * (t & 3));
  }
  const hipError_t e = launch_lookup(a, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "lookup launch");
  return DPI_OK;
}

// The no-allocation entry point's work (csrc/noalloc.hip supplies the device
// scratch): plan into the scratch without room for per-bag prefixes, then
// look up, then copy the status word out.  Not part of the C ABI.
__attribute__((visibility("hidden"))) dpi_status dpi_plan_lookup_into(
    const dpi_table_meta* table_meta, int32_t num_tables, const void* const* tables, const int32_t* ids,
    const int32_t* offsets, int64_t batch, int64_t total_ids, const int32_t* pooling, const dpi_plan_opts* opts,
    void* out, int32_t* device_status, void* scratch, size_t scratch_bytes, void* stream) {
  if (!table_meta) return fail(DPI_ERR_INVALID_ARG, "table_meta is NULL");
  if (num_tables < 1 || num_tables > DPI_MAX_TABLES)
    return fail(DPI_ERR_INVALID_ARG, "num_tables %d outside [1, %d]", num_tables, DPI_MAX_TABLES);
  if (device_status && (reinterpret_cast<uintptr_t>(device_status) & 3))
    return fail(DPI_ERR_MISALIGNED, "device_status not 4-byte aligned");
  int32_t dmax = 1;
  for (int t = 0; t < num_tables; ++t) dmax = std::max(dmax, std::min(table_meta[t].dim, (int32_t)DPI_MAX_DIM));
  dpi_plan_opts o;
  if (batch >= 0 && total_ids >= 0 && resolve_opts(opts, num_tables, batch, total_ids, o) == DPI_OK) {
    const size_t need =
        make_layout(num_tables, batch, total_ids, o, opts && opts->num_waves != 0, dmax, false).total;
    if (need > scratch_bytes)
      return fail(DPI_ERR_WORKSPACE_TOO_SMALL,
                  "this batch needs %zu bytes of scratch (%lld waves), the no-allocation entry point holds %zu",
                  need, (long long)o.num_waves, scratch_bytes);
  }
  dpi_plan_s plan{};
  dpi_status st = plan_init(&plan, table_meta, num_tables, offsets, batch, total_ids, opts, scratch, scratch_bytes,
                            stream, false);
  if (st != DPI_OK) return st;
  st = lookup_enqueue(&plan, tables, ids, offsets, pooling, out, stream);
  if (st != DPI_OK) return st;
  if (device_status) {
    const hipError_t e = launch_status_out(reinterpret_cast<const uint64_t*>(plan.ws + plan.layout.status),
                                           plan.plan_id & kPlanIdMask, device_status, plan.stream);
    if (e != hipSuccess) return hip_fail(e, "status launch");
  }
  return DPI_OK;
}

// The plan's error bits from its workspace's status word (zero when the word
// belongs to another plan) and the planning launch's long-bag count.
static dpi_status read_status(const dpi_plan_s* plan, int32_t* bits, int32_t* nlong) {
  uint64_t words[2] = {0, 0};
  const hipError_t e = hipMemcpy(words, plan->ws + plan->layout.status, sizeof(words), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpy status");
  const bool mine = (words[0] >> kStatusTagShift) == (uint64_t)(plan->plan_id & kPlanIdMask);
  *bits = mine ? (int32_t)(words[0] & kStatusBitsMask) : 0;
  if (nlong) *nlong = (int32_t)(words[1] & 0xffffffffu);
  return DPI_OK;
}

extern "C" {

dpi_status dpi_plan(const dpi_table_meta* table_meta, int32_t num_tables, const int32_t* offsets, int64_t batch,
                    int64_t total_ids, const dpi_plan_opts* opts, void* workspace, size_t workspace_bytes,
                    void* stream, dpi_plan_t* plan_out) {
  if (!plan_out) return fail(DPI_ERR_INVALID_ARG, "plan_out is NULL");
  *plan_out = nullptr;
  dpi_plan_s* plan = new (std::nothrow) dpi_plan_s{};
  if (!plan) return fail(DPI_ERR_INVALID_ARG, "out of host memory");
  const dpi_status st = plan_init(plan, table_meta, num_tables, offsets, batch, total_ids, opts, workspace,
                                  workspace_bytes, stream, true);
  if (st != DPI_OK) {
    delete plan;
    return st;
  }
  set_holder(plan->ws, plan->plan_id);
  *plan_out = plan;
  return DPI_OK;
}

dpi_status dpi_lookup(dpi_plan_t plan, const void* const* tables, const int32_t* ids, const int32_t* offsets,
                      const int32_t* pooling, void* out, void* stream) {
  if (!plan) return fail(DPI_ERR_INVALID_ARG, "plan is NULL");
  if (!is_holder(plan->ws, plan->plan_id)) return superseded();
  return lookup_enqueue(plan, tables, ids, offsets, pooling, out, stream);
}

dpi_status dpi_lookup_csr(dpi_plan_t plan, const void* packed, int32_t x_dtype, void* staging, size_t staging_bytes,
                          const void* const* tables, const int32_t* pooling, int32_t* offsets, int32_t* ids, void* out,
                          void* stream) {
  if (!plan) return fail(DPI_ERR_INVALID_ARG, "plan is NULL");
  if (!is_holder(plan->ws, plan->plan_id)) return superseded();
  if (!plan->one_launch || plan->onehot)
    return fail(DPI_ERR_UNSUPPORTED, "dpi_lookup_csr needs a plan whose lookups take one launch (bag by bag, at "
                                     "most 64 fields and 1024 bags per field): stage with dpi_stage_csr, then "
                                     "call dpi_lookup");
  if (!offsets || offsets != plan->offsets_arg)
    return fail(DPI_ERR_INVALID_ARG, "offsets must be the pointer the plan was built with");
  int esize = 0;
  switch (x_dtype) {
    case DPI_X_F32: esize = 4; break;
    case DPI_X_I64: esize = 8; break;
    case DPI_X_I32: esize = 4; break;
    default: return fail(DPI_ERR_INVALID_ARG, "bad x_dtype");
  }
  const int64_t n = (int64_t)plan->T * (plan->B + 1) + plan->total_ids;
  const size_t bytes = (size_t)n * (size_t)esize;
  if (!packed || !staging) return fail(DPI_ERR_INVALID_ARG, "packed or staging is NULL");
  if (staging_bytes < bytes) return fail(DPI_ERR_INVALID_ARG, "staging %zu bytes, need %zu", staging_bytes, bytes);
  if (reinterpret_cast<uintptr_t>(staging) & 15) return fail(DPI_ERR_MISALIGNED, "staging not 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(packed) % esize) return fail(DPI_ERR_MISALIGNED, "packed not element-aligned");
  if ((reinterpret_cast<uintptr_t>(offsets) | reinterpret_cast<uintptr_t>(ids)) & 3)
    return fail(DPI_ERR_MISALIGNED, "offsets or ids not 4-byte aligned");
  const hipError_t e = hipMemcpyAsync(staging, packed, bytes, hipMemcpyHostToDevice,
                                      reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
  const StagedInput st{staging, x_dtype};
  return lookup_enqueue(plan, tables, ids, offsets, pooling, out, stream, &st);
}

dpi_status dpi_fm_second_order(const void* emb, int32_t emb_dtype, int64_t batch, int32_t num_fields,
                               int32_t dim, int64_t row_stride, float* out, void* stream) {
  if (batch < 0) return fail(DPI_ERR_INVALID_ARG, "negative batch");
  if (num_fields < 1 || dim < 1) return fail(DPI_ERR_INVALID_ARG, "num_fields and dim must be >= 1");
  if (emb_dtype != DPI_F32 && emb_dtype != DPI_F16) return fail(DPI_ERR_INVALID_ARG, "bad emb_dtype");
  if (dim > DPI_MAX_DIM || num_fields > 65536) return fail(DPI_ERR_UNSUPPORTED, "dim or num_fields too large");
  if (row_stride < (int64_t)num_fields * dim) return fail(DPI_ERR_INVALID_ARG, "row_stride < num_fields * dim");
  if (batch == 0) return DPI_OK;
  if (!emb || !out) return fail(DPI_ERR_INVALID_ARG, "emb or out is NULL");
  const int esize = emb_dtype == DPI_F16 ? 2 : 4;
  if (reinterpret_cast<uintptr_t>(emb) % esize) return fail(DPI_ERR_MISALIGNED, "emb not element-aligned");
  if (reinterpret_cast<uintptr_t>(out) & 3) return fail(DPI_ERR_MISALIGNED, "out not 4-byte aligned");
  FmArgs a{};
  a.emb = emb;
  a.out = out;
  a.B = batch;
  a.row_stride = row_stride;
  a.T = num_fields;
  a.dim = dim;
  a.f16 = emb_dtype == DPI_F16;
  const int64_t field_bytes = (int64_t)dim * esize;
  a.lpr_log = -1;
  if (field_bytes % 16 == 0 && field_bytes <= 1024 && (row_stride * esize) % 16 == 0 &&
      (reinterpret_cast<uintptr_t>(emb) & 15) == 0)
    a.lpr_log = ilog2((int)(field_bytes / 16));
  const hipError_t e = launch_fm(a, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "fm launch");
  return DPI_OK;
}

dpi_status dpi_stage_onehot(const void* x, int32_t x_dtype, int64_t batch, int32_t num_fields,
                            int64_t row_stride, void* staging, size_t staging_bytes, int32_t* ids,
                            void* stream) {
  if (batch < 0) return fail(DPI_ERR_INVALID_ARG, "negative batch");
  if (num_fields < 1 || row_stride < num_fields)
    return fail(DPI_ERR_INVALID_ARG, "num_fields must be >= 1 and <= row_stride");
  int esize = 0;
  switch (x_dtype) {
    case DPI_X_F32: esize = 4; break;
    case DPI_X_I64: esize = 8; break;
    case DPI_X_I32: esize = 4; break;
    default: return fail(DPI_ERR_INVALID_ARG, "bad x_dtype");
  }
  if (batch == 0) return DPI_OK;
  if (!x || !staging || !ids) return fail(DPI_ERR_INVALID_ARG, "x, staging or ids is NULL");
  const size_t bytes = (size_t)batch * (size_t)row_stride * (size_t)esize;
  if (staging_bytes < bytes) return fail(DPI_ERR_INVALID_ARG, "staging %zu bytes, need %zu", staging_bytes, bytes);
  if (reinterpret_cast<uintptr_t>(staging) & 15) return fail(DPI_ERR_MISALIGNED, "staging not 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(x) % esize) return fail(DPI_ERR_MISALIGNED, "x not element-aligned");
  if (reinterpret_cast<uintptr_t>(ids) & 3) return fail(DPI_ERR_MISALIGNED, "ids not 4-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(staging, x, bytes, hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
  StageArgs a{};
  a.x = staging;
  a.ids = ids;
  a.B = batch;
  a.row_stride = row_stride;
  a.T = num_fields;
  a.x_dtype = x_dtype;
  e = launch_stage(a, s);
  if (e != hipSuccess) return hip_fail(e, "stage launch");
  return DPI_OK;
}

dpi_status dpi_stage_csr(const void* packed, int32_t x_dtype, int32_t num_fields, int64_t batch,
                         int64_t total_ids, void* staging, size_t staging_bytes, int32_t* offsets, int32_t* ids,
                         void* stream) {
  if (batch < 0 || total_ids < 0 || num_fields < 1)
    return fail(DPI_ERR_INVALID_ARG, "batch and total_ids must be >= 0, num_fields >= 1");
  int esize = 0;
  switch (x_dtype) {
    case DPI_X_F32: esize = 4; break;
    case DPI_X_I64: esize = 8; break;
    case DPI_X_I32: esize = 4; break;
    default: return fail(DPI_ERR_INVALID_ARG, "bad x_dtype");
  }
  const int64_t n_off = (int64_t)num_fields * (batch + 1);
  const size_t bytes = (size_t)(n_off + total_ids) * (size_t)esize;
  if (!packed || !staging || !offsets || (total_ids > 0 && !ids))
    return fail(DPI_ERR_INVALID_ARG, "packed, staging, offsets or ids is NULL");
  if (staging_bytes < bytes) return fail(DPI_ERR_INVALID_ARG, "staging %zu bytes, need %zu", staging_bytes, bytes);
  if (reinterpret_cast<uintptr_t>(staging) & 15) return fail(DPI_ERR_MISALIGNED, "staging not 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(packed) % esize) return fail(DPI_ERR_MISALIGNED, "packed not element-aligned");
  if ((reinterpret_cast<uintptr_t>(offsets) | reinterpret_cast<uintptr_t>(ids)) & 3)
    return fail(DPI_ERR_MISALIGNED, "offsets or ids not 4-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(staging, packed, bytes, hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
  e = launch_stage_csr(staging, x_dtype, n_off, total_ids, offsets, ids, s);
  if (e != hipSuccess) return hip_fail(e, "stage launch");
  return DPI_OK;
}

dpi_status dpi_plan_sync_status(dpi_plan_t plan) {
  if (!plan) return fail(DPI_ERR_INVALID_ARG, "plan is NULL");
  if (!is_holder(plan->ws, plan->plan_id)) return superseded();
  hipError_t e;
  if (plan->one_launch && !plan->looked_up && !plan->validated) {
    // nothing has checked the offsets yet: the planning launch does
    e = launch_plan(plan->args, plan->stream);
    if (e != hipSuccess) return hip_fail(e, "plan launch");
    plan->validated = true;
  }
  e = hipStreamSynchronize(plan->stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  int32_t status = 0;
  dpi_status st = read_status(plan, &status, nullptr);
  if (st != DPI_OK) return st;
  status |= plan->sticky_status;
  if (status & kStatusBadOffsets) return fail(DPI_ERR_BAD_OFFSETS, "device rejected the offsets");
  if (status & kStatusBadId) return fail(DPI_ERR_BAD_ID, "a lookup met an id outside its table");
  return DPI_OK;
}

}  // extern "C"

namespace {

template <typename V>
hipError_t copy_out(std::vector<V>& v, const char* src, int64_t count) {
  v.resize((size_t)std::max<int64_t>(count, 0));
  if (count <= 0) return hipSuccess;
  return hipMemcpy(v.data(), src, (size_t)count * sizeof(V), hipMemcpyDeviceToHost);
}

// First export of a plan: keep the partition the planning launch wrote (the
// arrays lookups read), then plan again in full -- the planning launch wrote no
// per-bag prefixes, and for a lookup that reads no partition no partition
// either unless a bag was long -- from the offsets given to dpi_plan, keeping
// the status bits earlier lookups latched.
dpi_status replan_for_export(dpi_plan_t plan) {
  if (!is_holder(plan->ws, plan->plan_id)) return superseded();
  hipError_t e = hipStreamSynchronize(plan->stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  const Layout& L = plan->layout;
  if (plan->partitioned) return DPI_OK;
  int32_t bits = 0, nlong = 0;
  const dpi_status st = read_status(plan, &bits, &nlong);
  if (st != DPI_OK) return st;
  plan->sticky_status |= bits & kStatusBadId;
  // what lookups read: the planning launch's partition, if it ran and wrote one
  const bool written = !plan->one_launch && !(plan->args.p.lazy_partition && nlong == 0);
  plan->snap_valid = false;
  if (written && plan->B > 0) {
    int64_t hdr[16];
    e = hipMemcpy(hdr, plan->ws + L.hdr, sizeof(hdr), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy header");
    const int64_t W = hdr[kHdrW];
    if (W < 0 || W > plan->waves_req) return fail(DPI_ERR_HIP, "plan header holds %lld waves", (long long)W);
    if ((e = copy_out(plan->snap_wib, plan->ws + L.wib, W + 1)) != hipSuccess ||
        (e = copy_out(plan->snap_wave_bag, plan->ws + L.wave_bag, W + 1)) != hipSuccess ||
        (e = copy_out(plan->snap_wbase, plan->ws + L.wbase, W + 1)) != hipSuccess ||
        (e = copy_out(plan->snap_head_first, plan->ws + L.head_first, W)) != hipSuccess ||
        (e = copy_out(plan->snap_split_pieces, plan->ws + L.split_pieces, W)) != hipSuccess ||
        (e = copy_out(plan->snap_split_last, plan->ws + L.split_last, W)) != hipSuccess)
      return hip_fail(e, "hipMemcpy partition");
    plan->snap_valid = true;
  }
  PlanArgs full = plan->args;
  full.p.lazy_partition = 0;
  full.p.prefixes = 1;
  e = launch_plan(full, plan->stream);
  if (e != hipSuccess) return hip_fail(e, "plan launch");
  e = hipStreamSynchronize(plan->stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  plan->partitioned = true;
  return DPI_OK;
}

}  // namespace

extern "C" {

dpi_status dpi_plan_export(dpi_plan_t plan, int64_t* header16, int64_t* col_base, int64_t* id_base,
                           int64_t* bag_item_base, int64_t* bag_cost_base, int64_t* wave_item_begin) {
  if (!plan) return fail(DPI_ERR_INVALID_ARG, "plan is NULL");
  dpi_status st = replan_for_export(plan);
  if (st != DPI_OK) return st;
  const Layout& L = plan->layout;
  int64_t hdr[16];
  hipError_t e = hipMemcpy(hdr, plan->ws + L.hdr, sizeof(hdr), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpy header");
  {
    // split bags are counted per tile of bags
    const int64_t nb = plan->args.p.nblk;
    std::vector<int64_t> splits((size_t)nb);
    e = hipMemcpy(splits.data(), plan->ws + L.block_sum + (3 * nb + 3) * sizeof(int64_t), nb * sizeof(int64_t),
                  hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy split counts");
    hdr[kHdrSplit] = 0;
    for (int64_t v : splits) hdr[kHdrSplit] += v;
  }
  const int64_t T = plan->T, TB = (int64_t)plan->T * plan->B, W = hdr[kHdrW];
  struct Part {
    int64_t* dst;
    size_t off;
    int64_t count;
  } parts[] = {{col_base, L.col_base, T + 1},       {id_base, L.id_base, T + 1},
               {bag_item_base, L.bib, TB + 1},      {bag_cost_base, L.bcb, TB + 1},
               {wave_item_begin, L.wib, W + 1}};
  for (const Part& p : parts) {
    if (!p.dst) continue;
    if (p.dst == wave_item_begin && plan->snap_valid) {
      if ((int64_t)plan->snap_wib.size() != W + 1) return fail(DPI_ERR_HIP, "partition changed on re-plan");
      std::memcpy(p.dst, plan->snap_wib.data(), (W + 1) * sizeof(int64_t));
      continue;
    }
    e = hipMemcpy(p.dst, plan->ws + p.off, p.count * sizeof(int64_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy plan array");
  }
  if (header16) std::memcpy(header16, hdr, sizeof(hdr));
  return DPI_OK;
}

dpi_status dpi_plan_export_waves(dpi_plan_t plan, int64_t* wave_bag, int64_t* wave_bag_base, int32_t* head_first,
                                 int32_t* split_pieces, int32_t* split_last, int32_t* source) {
  if (!plan) return fail(DPI_ERR_INVALID_ARG, "plan is NULL");
  dpi_status st = replan_for_export(plan);
  if (st != DPI_OK) return st;
  const Layout& L = plan->layout;
  int64_t hdr[16];
  hipError_t e = hipMemcpy(hdr, plan->ws + L.hdr, sizeof(hdr), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpy header");
  const int64_t W = hdr[kHdrW];
  if (source) *source = plan->snap_valid ? 1 : 0;
  if (plan->snap_valid) {
    if ((int64_t)plan->snap_wave_bag.size() != W + 1) return fail(DPI_ERR_HIP, "partition changed on re-plan");
    if (wave_bag) std::memcpy(wave_bag, plan->snap_wave_bag.data(), (W + 1) * sizeof(int64_t));
    if (wave_bag_base) std::memcpy(wave_bag_base, plan->snap_wbase.data(), (W + 1) * sizeof(int64_t));
    if (W > 0) {
      if (head_first) std::memcpy(head_first, plan->snap_head_first.data(), W * sizeof(int32_t));
      if (split_pieces) std::memcpy(split_pieces, plan->snap_split_pieces.data(), W * sizeof(int32_t));
      if (split_last) std::memcpy(split_last, plan->snap_split_last.data(), W * sizeof(int32_t));
    }
    return DPI_OK;
  }
  struct Part {
    void* dst;
    size_t off, bytes;
  } parts[] = {{wave_bag, L.wave_bag, (size_t)(W + 1) * sizeof(int64_t)},
               {wave_bag_base, L.wbase, (size_t)(W + 1) * sizeof(int64_t)},
               {head_first, L.head_first, (size_t)W * sizeof(int32_t)},
               {split_pieces, L.split_pieces, (size_t)W * sizeof(int32_t)},
               {split_last, L.split_last, (size_t)W * sizeof(int32_t)}};
  for (const Part& p : parts) {
    if (!p.dst || p.bytes == 0) continue;
    e = hipMemcpy(p.dst, plan->ws + p.off, p.bytes, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy plan array");
  }
  return DPI_OK;
}

void dpi_plan_destroy(dpi_plan_t plan) {
  if (!plan) return;
  drop_holder(plan->ws, plan->plan_id);
  delete plan;
}

}  // extern "C"
