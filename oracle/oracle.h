/*
 * CPU oracle for the fused multi-table embedding lookup -- TEST INFRASTRUCTURE.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * load this library.  It is a plain, slow, sequential definition of what the
 * GPU path computes; it shares no code, header or constant with the GPU path.
 *
 * Parity status: oracle_lookup is pinned by hand-typed bags, by the flat
 * index map of the paper's multi-table lookup algorithm (§IV-B, Algorithm 1)
 * for one-hot fields, by per-field embedding_bag + concatenation, and by
 * invariants.  oracle_plan is pinned by brute-force enumeration of the work
 * items, hand-computed plans and invariants; oracle_plan_waves by hand-computed
 * plans and by a brute-force assignment of every item to its wave.
 * oracle_fm_second_order (value and magnitude) is pinned by the pairwise forms
 * of the term and of its magnitude, closed forms and a hand-typed example.  The
 * plan's format is this library's own design (the paper prints none), so no
 * paper value pins it.
 */
#ifndef DPI_ORACLE_H
#define DPI_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  ORACLE_OK = 0,
  ORACLE_BAD_ARG = 1,
  ORACLE_BAD_OFFSETS = 5,
  ORACLE_BAD_ID = 6
};

/* dtypes: 0 = IEEE binary32, 1 = IEEE binary16.  pooling: 0 = sum, 1 = mean. */

/*
 * Pooled lookup (§IV-B; multi-hot bags through offsets, last paragraph of
 * §IV-B).  For every field t and sample b:
 *   out[b][col_base[t] + c] = sum over the bag's ids, in order, of
 *                             decode(E_t[id][c]), in fp64;
 *   mean pooling divides by the bag length; an empty bag gives 0.
 * mag (optional) receives the same with |decode(...)|, the scale of the
 * componentwise error bound.
 * tables[t] points to n_t * dims[t] elements, row-major.
 * ids: table-major concatenation; offsets: [T][B+1] per-table local prefix
 * (offsets[t][0] == 0), or NULL for one id per bag (ids[t*B + b]).
 * nthreads <= 0 uses the OpenMP default.
 */
int oracle_lookup(int32_t num_tables, int64_t batch, const int64_t* num_rows,
                  const int32_t* dims, const int32_t* dtypes, const void* const* tables,
                  const int32_t* ids, const int32_t* offsets, const int32_t* pooling,
                  double* out, double* mag, int32_t nthreads);

/*
 * Work plan: items are (field, bag, row-chunk) triples in field-major order;
 * each costs its rows' bytes plus, for the bag's first chunk, the bag's
 * output bytes, plus a constant; waves receive contiguous item ranges split
 * at equal fractions of the total cost.  See oracle.c for the step-by-step
 * definition.
 *   header16: [abi, T, B, W, C, K, out_dtype, flags, total_D, N, S,
 *              total_ids, num_split_bags, W_requested, 0, 0]
 *   col_base[T+1], id_base[T+1], bag_item_base[T*B+1], bag_cost_base[T*B+1],
 *   wave_item_begin[W_requested+1] (only the first W+1 are written).
 */
int oracle_plan(int32_t num_tables, int64_t batch, const int32_t* dims, const int32_t* dtypes,
                int32_t out_dtype, const int32_t* offsets, int64_t total_ids,
                int32_t chunk_rows, int32_t item_cost_k, int64_t waves_requested,
                uint32_t flags, int64_t* header16, int64_t* col_base, int64_t* id_base,
                int64_t* bag_item_base, int64_t* bag_cost_base, int64_t* wave_item_begin);

/*
 * The per-wave arrays a lookup reads of a plan, as closed forms of wave_item_begin
 * and bag_item_base (both from oracle_plan): for w in [0, W] the bag holding the
 * wave's first item and that bag's first item; for w in [0, W) the split-bag
 * bookkeeping (head_first: for a boundary strictly inside a bag, the wave holding the
 * bag's first item; for that wave, split_last: the last wave holding items of the
 * bag, split_pieces: the number of nonempty waves from it to split_last).  See
 * oracle.c for the step-by-step definition.
 *   wave_bag[W+1], wave_bag_base[W+1], head_first[W], split_pieces[W], split_last[W].
 */
int oracle_plan_waves(int64_t num_bags, const int64_t* bag_item_base, int64_t num_waves,
                      const int64_t* wave_item_begin, int64_t* wave_bag, int64_t* wave_bag_base,
                      int32_t* head_first, int32_t* split_pieces, int32_t* split_last);

/* bit of `flags`: boundaries are never moved to a bag end */
#define ORACLE_FLAG_EXACT_SPLIT (1u << 1)

/*
 * Second-order factorization-machine term of DeepFM's explicit interaction
 * module (§IV-D names it among the non-GEMM operators fused into one), over
 * the pooled block of T fields of one dim D: for every sample b, with
 * e[t][c] = decode(emb[b * row_stride + t * D + c]),
 *   out[b] = 1/2 * sum over c of ((sum over t of e[t][c])^2 - sum over t of e[t][c]^2),
 * i.e. the sum over field pairs t < u of the dot products <e[t], e[u]>.
 * mag (optional) receives 1/2 * sum over c of ((sum_t |e|)^2 + sum_t e^2), the
 * scale of the error bound.  dtype: 0 binary32, 1 binary16.  fp64 throughout.
 */
int oracle_fm_second_order(int64_t batch, int32_t num_fields, int32_t dim, int64_t row_stride,
                           int32_t dtype, const void* emb, double* out, double* mag);

#ifdef __cplusplus
}
#endif
#endif
