/*
 * CPU oracle for the fused multi-table embedding lookup -- TEST INFRASTRUCTURE.
 *
 * Loaded only by the test suite, the smoke check and the benchmark's CPU
 * baseline.  Plain C, fp64 accumulation, sequential per bag; OpenMP only
 * spreads independent bags over threads (each bag's sum order is fixed, so
 * the result does not depend on the thread count).
 *
 * Parity status: see oracle.h.  No function here is "parity unpinned".
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_ABI 1

/* IEEE 754 binary16 -> double, from the format's definition:
 *   exponent field 0:  (-1)^s * m * 2^-24              (subnormal / zero)
 *   exponent field 31: infinity (m == 0) or NaN
 *   otherwise:         (-1)^s * (1024 + m) * 2^(e - 25)  = (1 + m/1024) * 2^(e-15) */
static double decode_binary16(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1f;
  int m = h & 0x3ff;
  double v;
  if (e == 0) {
    v = ldexp((double)m, -24);
  } else if (e == 31) {
    v = m ? NAN : INFINITY;
  } else {
    v = ldexp((double)(1024 + m), e - 25);
  }
  return sign ? -v : v;
}

static double table_value(const void* table, int32_t dtype, int64_t index) {
  if (dtype == 1) return decode_binary16(((const uint16_t*)table)[index]);
  return (double)((const float*)table)[index];
}

/* ---------------------------------------------------------------------------------- */
/* Pooled lookup.  §IV-B: one table per field, the fields' results concatenated in  */
/* field order into a [b, sum of dims] block; multi-hot fields are delimited by     */
/* offsets.  Pooling (sum / mean, empty bag -> 0) is this library's reading; the    */
/* paper does not define it.                                                        */
/* ---------------------------------------------------------------------------------- */
int oracle_lookup(int32_t num_tables, int64_t batch, const int64_t* num_rows,
                  const int32_t* dims, const int32_t* dtypes, const void* const* tables,
                  const int32_t* ids, const int32_t* offsets, const int32_t* pooling,
                  double* out, double* mag, int32_t nthreads) {
  if (num_tables < 1 || batch < 0 || !dims || !dtypes || !tables || !num_rows || !out)
    return ORACLE_BAD_ARG;
  const int64_t T = num_tables, B = batch;

  int64_t* col_base = (int64_t*)calloc((size_t)T + 1, sizeof(int64_t));
  int64_t* id_base = (int64_t*)calloc((size_t)T + 1, sizeof(int64_t));
  if (!col_base || !id_base) { free(col_base); free(id_base); return ORACLE_BAD_ARG; }
  for (int64_t t = 0; t < T; ++t) {
    col_base[t + 1] = col_base[t] + dims[t];
    int64_t nnz = offsets ? offsets[t * (B + 1) + B] : B;
    id_base[t + 1] = id_base[t] + nnz;
  }
  const int64_t total_d = col_base[T];
  int status = ORACLE_OK;

#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(static) reduction(max : status)
#endif
  for (int64_t bag = 0; bag < T * B; ++bag) {
    const int64_t t = bag / B, b = bag % B;
    const int64_t D = dims[t];
    int64_t start, end;
    if (offsets) {
      start = offsets[t * (B + 1) + b];
      end = offsets[t * (B + 1) + b + 1];
    } else {
      start = b;
      end = b + 1;
    }
    double* o = out + b * total_d + col_base[t];
    double* g = mag ? mag + b * total_d + col_base[t] : NULL;
    for (int64_t c = 0; c < D; ++c) {
      o[c] = 0.0;
      if (g) g[c] = 0.0;
    }
    for (int64_t j = start; j < end; ++j) {
      const int64_t id = ids[id_base[t] + j];
      if (id < 0 || id >= num_rows[t]) {
        status = ORACLE_BAD_ID;
        continue;
      }
      for (int64_t c = 0; c < D; ++c) {
        const double v = table_value(tables[t], dtypes[t], id * D + c);
        o[c] += v;
        if (g) g[c] += fabs(v);
      }
    }
    const int64_t len = end - start;
    if (pooling && pooling[t] == 1 && len > 0) {
      for (int64_t c = 0; c < D; ++c) {
        o[c] /= (double)len;
        if (g) g[c] /= (double)len;
      }
    }
  }
  free(col_base);
  free(id_base);
  return status;
}

/* ---------------------------------------------------------------------------------- */
/* Work plan.  The paper's premise (§III, opportunity 2; §IV-B) is that the whole   */
/* embedding workload is known before execution, so it can be computed in advance   */
/* and spread over threads (§IV-C).  This plan is the library's concrete form of    */
/* that idea; its definition, step by step:                                         */
/*  1. esize_t = 4 (fp32) or 2 (fp16); row_bytes_t = dims[t]*esize_t;               */
/*     out_bytes_t = dims[t]*osize.                                                 */
/*  2. col_base = exclusive prefix of dims; id_base = exclusive prefix of the       */
/*     tables' id counts (offsets[t][B], or B for one-hot).                          */
/*  3. Bags are visited field-major (bag = t*B + b).  A bag of L ids has            */
/*     n = max(1, ceil(L/C)) items; item j covers rows [j*C, min(L, (j+1)*C)) and   */
/*     costs rows*row_bytes_t + (j == 0 ? out_bytes_t : 0) + K.                     */
/*  4. bag_item_base / bag_cost_base: exclusive prefixes of the bags' item counts   */
/*     and costs; their last entries are N and S.                                   */
/*  5. W = min(W_requested, N).  E_i = exclusive prefix of item costs.  For         */
/*     w = 0..W: c_w = ceil(w*S/W), i_w = min{ i : E_i >= c_w }.                    */
/*  6. Unless the exact-split flag is set, a boundary i_w that falls strictly       */
/*     inside a bag moves to that bag's end when the bag's cost beyond c_w is at    */
/*     most floor(S / (2W)).                                                        */
/*  7. num_split_bags counts bags that some inner boundary (0 < w < W) cuts.        */
/* ---------------------------------------------------------------------------------- */
/* number of ids in bag (t, b); one-hot fields (no offsets) hold exactly one */
static int64_t bag_length(const int32_t* offsets, int64_t t, int64_t b, int64_t B) {
  if (!offsets) return 1;
  return (int64_t)offsets[t * (B + 1) + b + 1] - offsets[t * (B + 1) + b];
}

/* number of items of a bag of L ids: max(1, ceil(L / C)) */
static int64_t bag_items(int64_t L, int64_t C) {
  int64_t n = (L + C - 1) / C;
  return n < 1 ? 1 : n;
}

/* cost of item j of a bag of L ids */
static int64_t item_cost(int64_t L, int64_t j, int64_t C, int64_t row_bytes, int64_t out_bytes,
                         int64_t K) {
  int64_t lo = j * C, hi = (j + 1) * C;
  if (hi > L) hi = L;
  const int64_t rows = hi > lo ? hi - lo : 0;
  return rows * row_bytes + (j == 0 ? out_bytes : 0) + K;
}

int oracle_plan(int32_t num_tables, int64_t batch, const int32_t* dims, const int32_t* dtypes,
                int32_t out_dtype, const int32_t* offsets, int64_t total_ids,
                int32_t chunk_rows, int32_t item_cost_k, int64_t waves_requested,
                uint32_t flags, int64_t* header16, int64_t* col_base, int64_t* id_base,
                int64_t* bag_item_base, int64_t* bag_cost_base, int64_t* wave_item_begin) {
  if (num_tables < 1 || batch < 0 || !dims || !dtypes || chunk_rows < 1 || item_cost_k < 1 ||
      waves_requested < 1 || (out_dtype != 0 && out_dtype != 1))
    return ORACLE_BAD_ARG;
  const int64_t T = num_tables, B = batch, C = chunk_rows, K = item_cost_k;
  const int64_t osize = out_dtype == 1 ? 2 : 4;

  /* step 1-2 */
  col_base[0] = 0;
  id_base[0] = 0;
  for (int64_t t = 0; t < T; ++t) {
    if (dims[t] < 1 || (dtypes[t] != 0 && dtypes[t] != 1)) return ORACLE_BAD_ARG;
    const int64_t esize = dtypes[t] == 1 ? 2 : 4;
    if ((dims[t] * esize) % 4 != 0) return ORACLE_BAD_ARG;
    col_base[t + 1] = col_base[t] + dims[t];
    int64_t nnz = B;
    if (offsets) {
      const int32_t* o = offsets + t * (B + 1);
      if (o[0] != 0) return ORACLE_BAD_OFFSETS;
      for (int64_t b = 0; b < B; ++b)
        if (o[b + 1] < o[b]) return ORACLE_BAD_OFFSETS;
      nnz = o[B];
    }
    id_base[t + 1] = id_base[t] + nnz;
  }
  if (id_base[T] != total_ids) return ORACLE_BAD_OFFSETS;

  /* step 3-4 */
  bag_item_base[0] = 0;
  bag_cost_base[0] = 0;
  for (int64_t t = 0; t < T; ++t) {
    const int64_t row_bytes = (int64_t)dims[t] * (dtypes[t] == 1 ? 2 : 4);
    const int64_t out_bytes = (int64_t)dims[t] * osize;
    for (int64_t b = 0; b < B; ++b) {
      const int64_t bag = t * B + b;
      const int64_t L = bag_length(offsets, t, b, B);
      const int64_t n = bag_items(L, C);
      int64_t cost = 0;
      for (int64_t j = 0; j < n; ++j) cost += item_cost(L, j, C, row_bytes, out_bytes, K);
      bag_item_base[bag + 1] = bag_item_base[bag] + n;
      bag_cost_base[bag + 1] = bag_cost_base[bag] + cost;
    }
  }
  const int64_t N = bag_item_base[T * B];
  const int64_t S = bag_cost_base[T * B];
  const int64_t W = waves_requested < N ? waves_requested : N;

  /* step 5: explicit item list (cost prefix E and owning bag) */
  int64_t* E = (int64_t*)malloc(sizeof(int64_t) * (size_t)(N + 1));
  int64_t* item_bag = (int64_t*)malloc(sizeof(int64_t) * (size_t)(N > 0 ? N : 1));
  if (!E || !item_bag) { free(E); free(item_bag); return ORACLE_BAD_ARG; }
  {
    int64_t i = 0;
    E[0] = 0;
    for (int64_t t = 0; t < T; ++t) {
      const int64_t row_bytes = (int64_t)dims[t] * (dtypes[t] == 1 ? 2 : 4);
      const int64_t out_bytes = (int64_t)dims[t] * osize;
      for (int64_t b = 0; b < B; ++b) {
        const int64_t bag = t * B + b;
        const int64_t L = bag_length(offsets, t, b, B);
        const int64_t n = bag_item_base[bag + 1] - bag_item_base[bag];
        for (int64_t j = 0; j < n; ++j) {
          E[i + 1] = E[i] + item_cost(L, j, C, row_bytes, out_bytes, K);
          item_bag[i] = bag;
          ++i;
        }
      }
    }
  }
  int64_t split = 0;
  if (W > 0) {
    const int64_t slack = (flags & ORACLE_FLAG_EXACT_SPLIT) ? -1 : S / (2 * W);
    int64_t i = 0;
    for (int64_t w = 0; w <= W; ++w) {
      const unsigned __int128 num = (unsigned __int128)(uint64_t)w * (uint64_t)S;
      const int64_t target = (int64_t)((num + (uint64_t)W - 1) / (uint64_t)W);
      while (E[i] < target) ++i; /* E is strictly increasing and E[N] = S >= target */
      int64_t begin = i;
      if (i < N) {
        const int64_t bag = item_bag[i];
        if (i > bag_item_base[bag] && slack >= 0 && bag_cost_base[bag + 1] - target <= slack)
          begin = bag_item_base[bag + 1];
      }
      wave_item_begin[w] = begin;
    }
    /* step 7 */
    int64_t last_split = -1;
    for (int64_t w = 1; w < W; ++w) {
      const int64_t b0 = wave_item_begin[w];
      if (b0 >= N) continue;
      const int64_t bag = item_bag[b0];
      if (b0 > bag_item_base[bag] && bag != last_split) {
        ++split;
        last_split = bag;
      }
    }
  } else {
    wave_item_begin[0] = 0;
  }
  free(E);
  free(item_bag);

  if (header16) {
    memset(header16, 0, 16 * sizeof(int64_t));
    header16[0] = ORACLE_ABI;
    header16[1] = T;
    header16[2] = B;
    header16[3] = W;
    header16[4] = C;
    header16[5] = K;
    header16[6] = out_dtype;
    header16[7] = flags;
    header16[8] = col_base[T];
    header16[9] = N;
    header16[10] = S;
    header16[11] = total_ids;
    header16[12] = split;
    header16[13] = waves_requested;
  }
  return ORACLE_OK;
}

/* ---------------------------------------------------------------------------------- */
/* What a wave of the lookup reads of the plan besides its item range.  Closed forms   */
/* of wave_item_begin (i_w) and bag_item_base (first item of each bag), following the  */
/* partition's definition above:                                                      */
/*  - wave_bag[w]: the bag that holds item i_w (T*B when i_w = N); wave_bag_base[w]:   */
/*    that bag's first item (N for T*B).                                              */
/*  - An inner boundary w (0 < w < W, i_w < N) lies strictly inside its bag when      */
/*    i_w > wave_bag_base[w].  The bag is then cut between waves; the wave holding its */
/*    first item is v = the largest v < w with i_v <= wave_bag_base[w], and           */
/*    head_first[w] = v.                                                              */
/*  - For such a v: split_last[v] = the largest inner boundary inside that bag (the   */
/*    wave holding the bag's last items), split_pieces[v] = the number of waves u in  */
/*    [v, split_last[v]] whose item range [i_u, i_{u+1}) is not empty.                */
/*  - Every other entry: head_first = -1, split_pieces = 0, split_last = -1.          */
/* ---------------------------------------------------------------------------------- */
int oracle_plan_waves(int64_t num_bags, const int64_t* bag_item_base, int64_t num_waves,
                      const int64_t* wave_item_begin, int64_t* wave_bag, int64_t* wave_bag_base,
                      int32_t* head_first, int32_t* split_pieces, int32_t* split_last) {
  if (num_bags < 0 || num_waves < 0 || !bag_item_base || !wave_item_begin || !wave_bag || !wave_bag_base)
    return ORACLE_BAD_ARG;
  if (num_waves > 0 && (!head_first || !split_pieces || !split_last)) return ORACLE_BAD_ARG;
  const int64_t TB = num_bags, W = num_waves, N = bag_item_base[TB];
  /* the bag of each boundary: bags are visited in order, boundaries are non-decreasing */
  int64_t bag = 0;
  for (int64_t w = 0; w <= W; ++w) {
    const int64_t i = wave_item_begin[w];
    if (i >= N) {
      wave_bag[w] = TB;
    } else {
      while (bag_item_base[bag + 1] <= i) ++bag;
      while (bag > 0 && bag_item_base[bag] > i) --bag;
      wave_bag[w] = bag;
    }
    wave_bag_base[w] = bag_item_base[wave_bag[w]];
  }
  for (int64_t w = 0; w < W; ++w) {
    head_first[w] = -1;
    split_pieces[w] = 0;
    split_last[w] = -1;
  }
  for (int64_t w = 1; w < W; ++w) {
    const int64_t i = wave_item_begin[w];
    if (i >= N || i <= wave_bag_base[w]) continue;
    int64_t v = w - 1;
    while (wave_item_begin[v] > wave_bag_base[w]) --v;   /* i_0 = 0 ends the search */
    head_first[w] = (int32_t)v;
    split_last[v] = (int32_t)w;
  }
  for (int64_t v = 0; v < W; ++v) {
    if (split_last[v] < 0) continue;
    int32_t pieces = 0;
    for (int64_t u = v; u <= split_last[v]; ++u)
      if (wave_item_begin[u] < wave_item_begin[u + 1]) ++pieces;
    split_pieces[v] = pieces;
  }
  return ORACLE_OK;
}

/* ---------------------------------------------------------------------------------- */
/* Second-order FM term (§IV-D: the explicit interaction of DeepFM holds the element- */
/* wise square and reduce-sum operators fused there).  Written from the term's       */
/* square-of-sum form; the tests check it against the pairwise dot-product form.     */
/* ---------------------------------------------------------------------------------- */
int oracle_fm_second_order(int64_t batch, int32_t num_fields, int32_t dim, int64_t row_stride,
                           int32_t dtype, const void* emb, double* out, double* mag) {
  if (batch < 0 || num_fields < 1 || dim < 1 || row_stride < (int64_t)num_fields * dim ||
      (dtype != 0 && dtype != 1) || (batch > 0 && (!emb || !out)))
    return ORACLE_BAD_ARG;
  for (int64_t b = 0; b < batch; ++b) {
    double y = 0.0, m = 0.0;
    for (int32_t c = 0; c < dim; ++c) {
      double s = 0.0, sa = 0.0, q = 0.0;
      for (int32_t t = 0; t < num_fields; ++t) {
        const double e = table_value(emb, dtype, b * row_stride + (int64_t)t * dim + c);
        s += e;
        sa += fabs(e);
        q += e * e;
      }
      y += s * s - q;
      m += sa * sa + q;
    }
    out[b] = 0.5 * y;
    if (mag) mag[b] = 0.5 * m;
  }
  return ORACLE_OK;
}
