/*
 * dpi.h -- C ABI of the fused multi-table embedding lookup for MI355X (gfx950).
 *
 * What it computes (DPIFrame, §IV-B and §IV-C): every sparse field t has its
 * own embedding table E_t (num_rows x dim, row-major).  For a batch of B
 * samples, field t of sample b holds a bag of row ids; the bag's rows are
 * gathered and pooled (sum, or mean over the bag length), and the pooled rows
 * of all fields are written side by side, in field order, into one
 * [B, sum_t dim_t] block -- the input of the interaction layers.  All fields
 * and samples are processed by one launch driven by a work plan computed in
 * advance from the bags' lengths (§III opportunity 2: the whole embedding
 * workload is known before execution).  One-hot fields are bags of one id;
 * multi-hot fields are delimited by offsets (last paragraph of §IV-B).
 * Pooling, empty bags and accumulation precision are not defined by the
 * paper; this library's reading: per-field sum or mean, an empty bag yields
 * zeros, accumulation in fp32 for fp32 and fp16 tables, a mean equal to the
 * correctly rounded fp32 quotient of that sum and the bag length, one
 * round-to-nearest-even conversion to the output dtype.
 *
 * Memory and streams
 *   - The caller owns every device buffer (tables, ids, offsets, out,
 *     workspace).  The library allocates only the small host objects behind
 *     dpi_plan_t and dpi_dcn_t (the latter also holds a rocBLAS handle, which
 *     manages device memory of its own).  A plan borrows its workspace: the
 *     workspace must outlive the plan and every lookup issued with it.
 *     Planning into a workspace again supersedes the plan before it:
 *     dpi_lookup, dpi_plan_sync_status and dpi_plan_export refuse a
 *     superseded plan (DPI_ERR_INVALID_ARG).
 *   - dpi_plan and dpi_lookup validate host-visible arguments synchronously,
 *     enqueue kernels on `stream` (a hipStream_t; NULL = default stream) and
 *     return without synchronizing.  Device-detected errors (malformed
 *     offsets, out-of-range ids) are latched into a status word in the
 *     workspace and reported by dpi_plan_sync_status.
 *   - One lookup in flight per plan: bags cut between two waves combine
 *     their partial sums through workspace memory.  Distinct plans (distinct
 *     workspaces) may run concurrently on distinct streams.
 *   - Nothing aborts, exits or prints.  Identical inputs give bitwise
 *     identical plans and outputs (no floating-point atomics; partial sums
 *     are combined in a fixed order).
 *
 * Layouts
 *   offsets: int32 [T][B+1]; row t is local to field t: offsets[t][0] == 0,
 *            non-decreasing, offsets[t][B] = number of ids of field t
 *            (< 2^31).  NULL means every bag holds exactly one id.
 *   ids:     int32, the fields' id lists concatenated in field order; bag
 *            (t, b) is ids[id_base[t] + offsets[t][b] .. id_base[t] +
 *            offsets[t][b+1]) with id_base the exclusive prefix of the fields'
 *            id counts.  With offsets == NULL bag (t, b) is {ids[t*B + b]}:
 *            the transpose of the sample-major id matrix of Algorithm 1.
 *            Ids outside [0, num_rows) contribute nothing and latch
 *            DPI_ERR_BAD_ID.
 *   tables:  host array [T] of device pointers, 16-byte aligned.
 *   out:     device [B][sum_t dim_t] of the plan's out dtype; field t
 *            occupies columns [col_base[t], col_base[t+1]), col_base the
 *            exclusive prefix of the dims.  Every element is written.
 */
#ifndef DPI_H
#define DPI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DPI_ABI_VERSION 1
#define DPI_MAX_TABLES 256      /* fields per plan */
#define DPI_MAX_DIM 65536       /* elements per row */

typedef enum {
  DPI_OK = 0,
  DPI_ERR_INVALID_ARG = 1,         /* null pointer, negative size, bad enum, table count */
  DPI_ERR_UNSUPPORTED = 2,         /* dim * element size not a multiple of 4 bytes, dim too large */
  DPI_ERR_MISALIGNED = 3,          /* table, out or workspace not 16-byte aligned */
  DPI_ERR_WORKSPACE_TOO_SMALL = 4,
  DPI_ERR_BAD_OFFSETS = 5,         /* offsets[t][0] != 0, decreasing, or ids != total_ids */
  DPI_ERR_BAD_ID = 6,              /* an id outside [0, num_rows) was met by a lookup */
  DPI_ERR_HIP = 7                  /* HIP runtime error; text in dpi_last_error() */
} dpi_status;

typedef enum { DPI_F32 = 0, DPI_F16 = 1 } dpi_dtype;
typedef enum { DPI_POOL_SUM = 0, DPI_POOL_MEAN = 1 } dpi_pooling;
typedef enum { DPI_X_F32 = 0, DPI_X_I64 = 1, DPI_X_I32 = 2 } dpi_x_dtype;   /* host feature matrix */

/* plan flags */
enum {
  DPI_FLAG_EXACT_SPLIT = 1u << 1,  /* never move a wave boundary to a bag's end (many split bags) */
  DPI_FLAG_LINEAR_BLOCKS = 1u << 2, /* workgroup i takes waves 4i..4i+3 (default: each XCD of the
                                       chip, or each pair of XCDs when every row is at most 128
                                       bytes, takes a contiguous range of waves, so one field's
                                       rows meet in few L2s) */
  DPI_FLAG_INPUT_FIRST = 1u << 3    /* dpi_lookup allocates one lane per bag (the input-first
                                       alternative of §IV-C) instead of the plan's waves; same
                                       results, kept for comparison */
};

typedef struct {
  int64_t num_rows;  /* rows of the table (ids must lie in [0, num_rows)) */
  int32_t dim;       /* elements per row, 1..DPI_MAX_DIM */
  int32_t dtype;     /* dpi_dtype of the table */
} dpi_table_meta;

typedef struct {
  int32_t chunk_rows;   /* C: rows per work item; 0 -> 32 */
  int32_t item_cost_k;  /* K: fixed cost per work item; 0 -> 64 */
  int64_t num_waves;    /* requested waves; 0 -> dpi_default_waves(...) */
  int32_t out_dtype;    /* dpi_dtype of the output */
  uint32_t flags;       /* DPI_FLAG_* */
} dpi_plan_opts;

typedef struct dpi_plan_s* dpi_plan_t;

/*
 * Default wave count for a batch: max(min(16 * compute units of the current
 * device, max(ceil(T*B / 8), min(ceil(total_ids / 32) + T*B, 8 * T))),
 * ceil((total_ids + T*B) / 2048), 1).  Large batches get about 2048 rows and
 * bags per wave; small ones enough waves for the device but about 8 bags per
 * wave (fewer bags cut between waves), and tiny ones about one work item per
 * wave (a wave walks its fields one after the other).  The plan uses
 * W = min(requested, number of work items).
 */
int64_t dpi_default_waves(int32_t num_tables, int64_t batch, int64_t total_ids);

/*
 * Bytes of device workspace dpi_plan needs for these sizes (0 on invalid
 * arguments).  max_dim is the largest dim over the fields.  Batches that may
 * take one launch per lookup also get room for the pieces of long bags:
 * (16 + 8 * max_dim) / (4 * C) bytes per id.
 */
size_t dpi_plan_workspace_bytes(int32_t num_tables, int64_t batch, int64_t total_ids,
                                int32_t max_dim, const dpi_plan_opts* opts);

/*
 * Build the work plan of one batch (§III opportunity 2, §IV-B, §IV-C):
 * the bags' item counts and costs, their exclusive prefix sums over all
 * fields (field-major), and a partition of the items into W waves of nearly
 * equal cost.  The plan's arrays are defined step by step in the oracle's
 * documentation and exported by dpi_plan_export (which notes when the
 * partition is computed).
 *   table_meta: host [num_tables]; offsets: device [T][B+1] or NULL;
 *   total_ids:  number of ids (sum of offsets[t][B], or T*B);
 *   opts:       NULL for defaults;
 *   workspace:  device, 16-byte aligned, >= dpi_plan_workspace_bytes(...);
 *   stream:     hipStream_t or NULL;  plan_out: receives the plan handle.
 * Errors: INVALID_ARG, UNSUPPORTED, MISALIGNED, WORKSPACE_TOO_SMALL, HIP
 * synchronously; BAD_OFFSETS later through dpi_plan_sync_status.
 * One launch per lookup: for a one-hot batch whose fields share one row
 * class, and for a batch pooled bag by bag (see dpi_lookup) of at most 64
 * fields and, with offsets, at most 1024 bags per field, dpi_plan enqueues
 * nothing; each lookup derives the fields' first ids from the offsets and
 * checks them itself (§I: for small batches a launch costs more than the
 * lookup's work), and dpi_plan_sync_status before any lookup runs the check.
 */
dpi_status dpi_plan(const dpi_table_meta* table_meta, int32_t num_tables, const int32_t* offsets,
                    int64_t batch, int64_t total_ids, const dpi_plan_opts* opts, void* workspace,
                    size_t workspace_bytes, void* stream, dpi_plan_t* plan_out);

/*
 * Fused gather-pool of every field's bags into `out` (Algorithm 1 of §IV-B
 * generalised to bags, heterogeneous dims and pooling; lanes of a wavefront
 * cover the contiguous columns of one row, the output-first allocation of
 * §IV-C).
 *   tables:  host [T] of device pointers (16-byte aligned);
 *   ids, offsets: the batch the plan was built from (same contents);
 *   pooling: host [T] of dpi_pooling, NULL = all sum;
 *   out:     device [B][sum dim] of the plan's out dtype.
 * With malformed offsets (DPI_ERR_BAD_OFFSETS) the lookup writes no row of
 * a field whose offsets are malformed; whether it writes the other fields is
 * unspecified.
 * Small and mid-size batches (at most 180000 bags, every row a multiple of
 * 16 bytes and at most 1024 bytes, wave count left at 0) are pooled bag by
 * bag, without the plan's partition: a wave takes a few bags of one field,
 * each bag several row slots.  A bag of more than 4 work items (4*C ids) is
 * pooled in pieces of at most 4*C ids spread over the field's waves when the
 * lookup is the batch's only launch (see dpi_plan); otherwise, if the plan
 * counted such a bag, the lookup uses the partition instead.  An explicit
 * wave count always uses the partition.  Either way the results are within
 * the same tolerance and deterministic.
 */
dpi_status dpi_lookup(dpi_plan_t plan, const void* const* tables, const int32_t* ids,
                      const int32_t* offsets, const int32_t* pooling, void* out, void* stream);

/*
 * Second-order factorization-machine term of DeepFM's explicit interaction
 * over a block of T fields of one dim D -- typically dpi_lookup's output.
 * §IV-D fuses the interaction's neighbouring non-GEMM operators (element-wise
 * square, subtraction, reduce-sum) into one kernel; this is that kernel:
 *   out[b] = 1/2 * sum_c ((sum_t e[b][t][c])^2 - sum_t e[b][t][c]^2),
 *   e[b][t][c] = emb[b * row_stride + t * dim + c]  (row_stride in elements),
 * i.e. the sum over field pairs t < u of <e[b][t], e[b][u]>.
 *   emb:  device, dpi_dtype emb_dtype, element-aligned, read only;
 *   out:  device fp32 [batch], fully written;  stream: hipStream_t or NULL.
 * fp32 accumulation in a fixed order (deterministic).  Rows of dim elements
 * that are a multiple of 16 bytes (at most 1024) with a 16-byte aligned block
 * and row stride take the vector path; any other shape the column path.
 * Errors: INVALID_ARG (NULL pointer with batch > 0, batch < 0, num_fields < 1,
 * dim < 1, row_stride < num_fields * dim, bad dtype), UNSUPPORTED (dim >
 * DPI_MAX_DIM or num_fields > 65536), MISALIGNED (emb not element-aligned,
 * out not 4-byte aligned), HIP.
 */
dpi_status dpi_fm_second_order(const void* emb, int32_t emb_dtype, int64_t batch, int32_t num_fields,
                               int32_t dim, int64_t row_stride, float* out, void* stream);

/*
 * Input consolidation for one-hot fields (the paper's breakdown, §V: moving
 * each field to the GPU and converting each to an integer type separately is
 * replaced by one transfer and one conversion).  The batch's categorical
 * features arrive as one sample-major host matrix x[batch][row_stride] whose
 * columns [0, num_fields) hold the fields' ids (float, int64 or int32, as a
 * data loader produces them).  One asynchronous host-to-device copy moves the
 * matrix into `staging`, then one kernel converts and transposes it into the
 * field-major int32 ids that dpi_plan / dpi_lookup take with offsets == NULL:
 *   ids[t * batch + b] = x[b][t].
 * A value that is not an integer in [0, 2^31) becomes -1, which a lookup
 * reports as DPI_ERR_BAD_ID.
 *   x:       host, batch * row_stride elements; pinned memory (hipHostMalloc)
 *            makes the copy asynchronous; it must stay valid until the copy
 *            has run (synchronize the stream before reusing it);
 *   staging: device, 16-byte aligned, >= batch * row_stride * element size;
 *   ids:     device int32 [num_fields * batch], 4-byte aligned.
 * Errors: INVALID_ARG (NULL pointer with batch > 0, batch < 0, num_fields < 1,
 * row_stride < num_fields, bad x_dtype, staging too small), MISALIGNED, HIP.
 */
dpi_status dpi_stage_onehot(const void* x, int32_t x_dtype, int64_t batch, int32_t num_fields,
                            int64_t row_stride, void* staging, size_t staging_bytes, int32_t* ids,
                            void* stream);

/*
 * Input consolidation for multi-hot fields: one host array `packed` of
 * x_dtype elements holds every field's offsets ([num_fields][batch + 1], local
 * per field as dpi_plan takes them) followed by the fields' concatenated ids
 * (total_ids), as a data loader can lay them out; one asynchronous copy moves
 * it into `staging` and one kernel converts both parts to the int32 `offsets`
 * and `ids` of dpi_plan / dpi_lookup.  Values that are not integers in
 * [0, 2^31) become -1 (dpi_plan then reports malformed offsets, a lookup a
 * bad id).
 *   packed:  host, (num_fields * (batch + 1) + total_ids) elements, ideally
 *            pinned, valid until the copy has run;
 *   staging: device, 16-byte aligned, at least that many elements;
 *   offsets: device int32 [num_fields][batch + 1];  ids: device int32 [total_ids].
 * Errors: INVALID_ARG, MISALIGNED, HIP.
 */
dpi_status dpi_stage_csr(const void* packed, int32_t x_dtype, int32_t num_fields, int64_t batch,
                         int64_t total_ids, void* staging, size_t staging_bytes, int32_t* offsets, int32_t* ids,
                         void* stream);

/*
 * Input consolidation folded into the lookup (§V breakdown): for a plan whose
 * lookups take one launch (bag by bag, see dpi_plan and dpi_lookup), one
 * asynchronous copy moves the packed host CSR that dpi_stage_csr takes
 * (every field's offsets [T][B+1], then the fields' ids, as x_dtype) into
 * `staging`, and the lookup kernel reads it there: each offset and id is
 * converted as dpi_stage_csr converts it (not an integer in [0, 2^31): -1)
 * when the kernel reads it, written to `offsets` / `ids` (the int32 arrays
 * dpi_stage_csr would have produced), and pooled into `out` -- one copy and
 * one kernel for the whole step, the same `out` bits as dpi_stage_csr then
 * dpi_lookup.
 *   plan:    built by dpi_plan with `offsets` as its offsets pointer (dpi_plan
 *            reads nothing of them for such a plan, so they may still be
 *            unwritten); batch sizes from the plan;
 *   packed:  host, (T*(B+1) + total_ids) elements, ideally pinned, valid until
 *            the copy has run;  staging: device, 16-byte aligned, that many
 *            elements;  offsets, ids: device int32 outputs;
 *   tables, pooling, out: as for dpi_lookup.
 * With malformed offsets the converted arrays and `out` are unspecified (the
 * status reports DPI_ERR_BAD_OFFSETS).  Query the status after the lookup.
 * Errors: UNSUPPORTED (a plan that is not one launch per lookup: stage with
 * dpi_stage_csr, then dpi_lookup), INVALID_ARG, MISALIGNED, HIP.
 */
dpi_status dpi_lookup_csr(dpi_plan_t plan, const void* packed, int32_t x_dtype, void* staging, size_t staging_bytes,
                          const void* const* tables, const int32_t* pooling, int32_t* offsets, int32_t* ids, void* out,
                          void* stream);

/*
 * Breadth-first two-stream scheduling of the interaction modules (§IV-E,
 * Algorithm 2).  A model's explicit interaction module (e.g. a cross network)
 * and implicit one (an MLP) are independent, so each gets a stream; the host
 * enqueues their operators interleaved one by one, starting with the module
 * that has more operators (the explicit one on a tie) and ending with the
 * longer module's remaining operators, so both modules start at once.
 * An operator is a host callback that enqueues its work on the stream given.
 */
enum { DPI_SCHED_BREADTH_FIRST = 0,   /* Algorithm 2's queue, two streams */
       DPI_SCHED_DEPTH_FIRST = 1,     /* all explicit operators, then all implicit ones, two streams */
       DPI_SCHED_ONE_STREAM = 2 };    /* depth-first on stream_explicit only (no overlap) */

typedef struct {
  dpi_status (*launch)(void* ctx, void* stream);   /* enqueue on `stream` (a hipStream_t) */
  void* ctx;
} dpi_op;

/* Algorithm 2's queue for n_explicit and n_implicit operators: order[k] = i
 * for explicit operator i, -(j + 1) for implicit operator j; order holds
 * n_explicit + n_implicit entries.  Host only. */
dpi_status dpi_breadth_first_order(int32_t n_explicit, int32_t n_implicit, int32_t* order);

/* Enqueue both modules' operators in `mode`'s order on their streams.  Both
 * streams first wait for the work already enqueued on `after` (e.g. the
 * lookup); `after` then waits for both.  Streams are caller-owned, default
 * priority.  An operator's error stops the enqueueing and is returned. */
dpi_status dpi_launch_two_streams(const dpi_op* explicit_ops, int32_t n_explicit, const dpi_op* implicit_ops,
                                  int32_t n_implicit, int32_t mode, void* stream_explicit, void* stream_implicit,
                                  void* after);

/* Tick rate in kHz of the device wall clock that dpi_dcn_forward's marks read. */
int64_t dpi_wall_clock_khz(void);

/*
 * Interaction head of the paper's DCN-style models over the pooled block
 * x0 [batch][dim] (fp32, row-major), to drive the scheduler with real work:
 *   explicit: a DCNv2 cross network, x_{l+1} = x0 * (x_l W_l^T + b_l) + x_l,
 *             W_l [dim][dim], b_l [dim], l < n_cross;  out_cross = x_{n_cross};
 *   implicit: an MLP, h_{l+1} = max(0, h_l V_l^T + c_l), h_0 = x0,
 *             V_l [mlp_dims[l]][previous dim], c_l [mlp_dims[l]];  out_mlp = h_{n_mlp}.
 * Each GEMM is a rocBLAS fp32 GEMM; the element-wise run after it is one fused
 * kernel (the non-GEMM fusion of §IV-D).  All pointers are device memory owned
 * by the caller; biases and activations 16-byte aligned when their row length
 * is a multiple of 4.  The head borrows the weights and a workspace of
 * dpi_dcn_workspace_bytes (256-byte aligned) and owns a rocBLAS handle (which
 * manages its own device workspace).  One forward in flight per head.
 */
typedef struct {
  int64_t batch;
  int32_t dim;
  int32_t n_cross;
  int32_t n_mlp;
  const int32_t* mlp_dims;          /* host [n_mlp] */
  const float* const* cross_w;      /* host [n_cross] of device pointers */
  const float* const* cross_b;
  const float* const* mlp_w;        /* host [n_mlp] of device pointers */
  const float* const* mlp_b;
} dpi_dcn_desc;

typedef struct dpi_dcn_s* dpi_dcn_t;

size_t dpi_dcn_workspace_bytes(const dpi_dcn_desc* desc);   /* 0 on invalid arguments */
dpi_status dpi_dcn_create(const dpi_dcn_desc* desc, void* workspace, size_t workspace_bytes, dpi_dcn_t* out);
/* marks: NULL, or device uint64 [2] receiving the device wall clock when each
 * module's first operator starts (explicit, implicit). */
dpi_status dpi_dcn_forward(dpi_dcn_t head, const float* x0, float* out_cross, float* out_mlp, int32_t mode,
                           void* stream_explicit, void* stream_implicit, void* after, uint64_t* marks);
void dpi_dcn_destroy(dpi_dcn_t head);

/*
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation: dpi_plan
 * followed by dpi_lookup in one call, with the plan's workspace taken from a
 * fixed device array of this library (DPI_NOALLOC_SCRATCH_BYTES per GPU,
 * held by each GPU the library runs on until the process ends) instead of a
 * caller's buffer.  Calls no allocating routine, host or device.
 *   Arguments as for dpi_plan (with opts) and dpi_lookup; `out` receives the
 *   same values, bit for bit, as that pair with a caller workspace.
 *   device_status: NULL, or device int32 receiving (asynchronously, by a
 *   one-thread kernel after the lookup) the call's device-detected errors:
 *   DPI_DEVSTAT_BAD_OFFSETS, DPI_DEVSTAT_BAD_ID, 0 when none.
 *   stream: a stream of the current device.
 * Every call on a GPU shares that GPU's array, which keeps the last call's
 * contents (each call resets what it reads): calls that overlap on one GPU --
 * on different streams, or from different host threads -- race, and must be
 * serialized by the caller.  A batch whose plan needs more than the array
 * holds (per-wave state and split-bag partials, about 12 + 8 * max dim bytes
 * per wave, plus 48 bytes per field and 24 bytes per tile of bags, plus the
 * long-bag pieces of dpi_plan_workspace_bytes) returns
 * DPI_ERR_WORKSPACE_TOO_SMALL and enqueues nothing; other errors as for
 * dpi_plan and dpi_lookup.
 */
#define DPI_NOALLOC_SCRATCH_BYTES (64u << 20)
#define DPI_DEVSTAT_BAD_OFFSETS 1
#define DPI_DEVSTAT_BAD_ID 2
dpi_status dpi_lookup_noalloc(const dpi_table_meta* table_meta, int32_t num_tables, const void* const* tables,
                              const int32_t* ids, const int32_t* offsets, int64_t batch, int64_t total_ids,
                              const int32_t* pooling, const dpi_plan_opts* opts, void* out, int32_t* device_status,
                              void* stream);

/* Synchronize the plan's stream and report device-detected errors
 * (BAD_OFFSETS before BAD_ID).  Lookups on other streams must be
 * synchronized by the caller first. */
dpi_status dpi_plan_sync_status(dpi_plan_t plan);

/*
 * Copy the plan to host arrays (synchronizes the plan's stream).  Any
 * pointer may be NULL.  Sizes: header16[16], col_base[T+1], id_base[T+1],
 * bag_item_base[T*B+1], bag_cost_base[T*B+1], wave_item_begin[W+1] with W =
 * header16[3].  header16 = [abi, T, B, W, C, K, out_dtype, flags, total_dim,
 * items N, total cost S, total_ids, split bags, requested waves, 0, 0].
 * The planning launch writes what lookups read: the per-bag prefixes
 * (bag_item_base, bag_cost_base) are left out -- a lookup needs only the
 * first item of each wave's first bag -- and so is the wave partition when
 * dpi_lookup will not read it (a batch pooled bag by bag, a one-hot batch of
 * one row class, the input-first allocation) unless some bag is longer than
 * 4 items; a plan of one launch per lookup has no planning launch at all.
 * The first export of a plan therefore plans the batch again in full, on the
 * plan's stream, from the offsets given to dpi_plan -- they must still hold
 * the batch, and no lookup of this plan may be in flight on another stream.
 */
dpi_status dpi_plan_export(dpi_plan_t plan, int64_t* header16, int64_t* col_base, int64_t* id_base,
                           int64_t* bag_item_base, int64_t* bag_cost_base, int64_t* wave_item_begin);

/*
 * Copy what a lookup reads of the plan besides the wave starts (synchronizes
 * the plan's stream; plans again in full on the first export, as
 * dpi_plan_export does).  With W = header16[3] of dpi_plan_export:
 *   wave_bag[W+1]      bag (t*B + b) holding wave w's first item (T*B at the end);
 *   wave_bag_base[W+1] that bag's first item;
 *   head_first[W]      for a wave that starts strictly inside a bag, the wave
 *                      holding the bag's first item, else -1;
 *   split_pieces[W]    for that first wave, the number of nonempty waves holding
 *                      items of the bag, else 0;
 *   split_last[W]      ... and the last of them, else -1.
 * These follow from wave_item_begin and bag_item_base (§IV-C: the work is
 * spread over threads after the whole workload is known).  *source receives 1
 * when the arrays (and dpi_plan_export's wave_item_begin) are the ones the
 * planning launch wrote, copied before the first re-plan -- the arrays a
 * lookup of this plan reads -- and 0 when no planning launch wrote a
 * partition (the plan's lookup reads none: a batch pooled bag by bag without a
 * long bag or in one launch, a one-hot batch of one row class, the
 * input-first allocation) and the export's re-plan computed them.  Any
 * pointer may be NULL.
 */
dpi_status dpi_plan_export_waves(dpi_plan_t plan, int64_t* wave_bag, int64_t* wave_bag_base, int32_t* head_first,
                                 int32_t* split_pieces, int32_t* split_last, int32_t* source);

/* Free the host object (not the workspace).  NULL is ignored. */
void dpi_plan_destroy(dpi_plan_t plan);

const char* dpi_status_str(dpi_status s);
const char* dpi_last_error(void);   /* thread-local detail of the last error */
int dpi_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* DPI_H */
