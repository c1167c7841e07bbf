// Breadth-first two-stream scheduling of the interaction modules (§IV-E,
// Algorithm 2) and an interaction head to drive it: a DCNv2 cross network
// (explicit module) and an MLP (implicit module) over the pooled block.
//
// The two modules are independent, so they can run on two streams; what
// decides how early the second module starts is the order in which the host
// enqueues operators.  Algorithm 2 interleaves the modules' operators one by
// one (starting with the module that has more operators), so the second
// module's first operator is enqueued right after the first module's first
// one instead of after all of them.  GEMMs run in rocBLAS; the element-wise
// runs between them are one fused kernel each (interact.hip).
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

#include <cstring>
#include <new>
#include <vector>

#include "dpi_internal.h"

using namespace dpi;

__attribute__((visibility("hidden"))) dpi_status dpi_fail_status(dpi_status s, const char* fmt, ...);   // api.cpp
__attribute__((visibility("hidden"))) dpi_status dpi_hip_status(hipError_t e, const char* what);        // api.cpp

namespace {

struct Queued {
  int module;   // 0 explicit, 1 implicit
  int index;
};

// Algorithm 2's queue: interleave, longer module first (explicit on a tie),
// then the longer module's remaining operators.
std::vector<Queued> breadth_first(int32_t ne, int32_t ni) {
  std::vector<Queued> q;
  q.reserve((size_t)ne + (size_t)ni);
  const int first = ni > ne ? 1 : 0;
  const int32_t n_first = first ? ni : ne, n_second = first ? ne : ni;
  for (int32_t i = 0; i < n_second; ++i) {
    q.push_back({first, i});
    q.push_back({1 - first, i});
  }
  for (int32_t j = n_second; j < n_first; ++j) q.push_back({first, j});
  return q;
}

}  // namespace

extern "C" {

dpi_status dpi_breadth_first_order(int32_t n_explicit, int32_t n_implicit, int32_t* order) {
  if (n_explicit < 0 || n_implicit < 0) return dpi_fail_status(DPI_ERR_INVALID_ARG, "negative operator count");
  if (n_explicit + n_implicit > 0 && !order) return dpi_fail_status(DPI_ERR_INVALID_ARG, "order is NULL");
  const std::vector<Queued> q = breadth_first(n_explicit, n_implicit);
  for (size_t k = 0; k < q.size(); ++k) order[k] = q[k].module == 0 ? q[k].index : -(q[k].index + 1);
  return DPI_OK;
}

dpi_status dpi_launch_two_streams(const dpi_op* explicit_ops, int32_t n_explicit, const dpi_op* implicit_ops,
                                  int32_t n_implicit, int32_t mode, void* stream_explicit, void* stream_implicit,
                                  void* after) {
  if (n_explicit < 0 || n_implicit < 0) return dpi_fail_status(DPI_ERR_INVALID_ARG, "negative operator count");
  if ((n_explicit > 0 && !explicit_ops) || (n_implicit > 0 && !implicit_ops))
    return dpi_fail_status(DPI_ERR_INVALID_ARG, "operator list is NULL");
  if (mode != DPI_SCHED_BREADTH_FIRST && mode != DPI_SCHED_DEPTH_FIRST && mode != DPI_SCHED_ONE_STREAM)
    return dpi_fail_status(DPI_ERR_INVALID_ARG, "bad scheduling mode %d", mode);
  for (int32_t i = 0; i < n_explicit; ++i)
    if (!explicit_ops[i].launch) return dpi_fail_status(DPI_ERR_INVALID_ARG, "explicit op %d has no launch", i);
  for (int32_t i = 0; i < n_implicit; ++i)
    if (!implicit_ops[i].launch) return dpi_fail_status(DPI_ERR_INVALID_ARG, "implicit op %d has no launch", i);
  hipStream_t se = reinterpret_cast<hipStream_t>(stream_explicit);
  hipStream_t si = mode == DPI_SCHED_ONE_STREAM ? se : reinterpret_cast<hipStream_t>(stream_implicit);
  hipStream_t sa = reinterpret_cast<hipStream_t>(after);

  std::vector<Queued> q;
  if (mode == DPI_SCHED_BREADTH_FIRST) {
    q = breadth_first(n_explicit, n_implicit);
  } else {
    for (int32_t i = 0; i < n_explicit; ++i) q.push_back({0, i});
    for (int32_t j = 0; j < n_implicit; ++j) q.push_back({1, j});
  }
  // both module streams start after the work already on `after`
  hipEvent_t ev[3];
  for (int k = 0; k < 3; ++k) {
    hipError_t e = hipEventCreateWithFlags(&ev[k], hipEventDisableTiming);
    if (e != hipSuccess) {
      for (int j = 0; j < k; ++j) (void)hipEventDestroy(ev[j]);
      return dpi_hip_status(e, "hipEventCreateWithFlags");
    }
  }
  struct Guard {
    hipEvent_t* ev;
    ~Guard() {
      for (int k = 0; k < 3; ++k) (void)hipEventDestroy(ev[k]);
    }
  } guard{ev};
  hipError_t e = hipEventRecord(ev[0], sa);
  if (e == hipSuccess) e = hipStreamWaitEvent(se, ev[0], 0);
  if (e == hipSuccess && si != se) e = hipStreamWaitEvent(si, ev[0], 0);
  if (e != hipSuccess) return dpi_hip_status(e, "stream ordering");
  for (const Queued& x : q) {
    const dpi_op& op = x.module == 0 ? explicit_ops[x.index] : implicit_ops[x.index];
    const dpi_status st = op.launch(op.ctx, x.module == 0 ? (void*)se : (void*)si);
    if (st != DPI_OK) return st;
  }
  // `after` continues once both modules are done
  e = hipEventRecord(ev[1], se);
  if (e == hipSuccess) e = hipStreamWaitEvent(sa, ev[1], 0);
  if (e == hipSuccess && si != se) e = hipEventRecord(ev[2], si);
  if (e == hipSuccess && si != se) e = hipStreamWaitEvent(sa, ev[2], 0);
  if (e != hipSuccess) return dpi_hip_status(e, "stream join");
  return DPI_OK;
}

int64_t dpi_wall_clock_khz(void) {
  int dev = 0, khz = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess) return 0;
  return khz;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Interaction head: cross network + MLP over x0 [B, d].
// ---------------------------------------------------------------------------
struct dpi_dcn_s {
  int64_t B = 0;
  int32_t d = 0;
  std::vector<int32_t> mlp_dims;
  std::vector<const float*> cw, cb, mw, mb;
  float* y = nullptr;         // [B][d] cross GEMM output
  float* xa = nullptr;        // [B][d] cross ping
  float* xb = nullptr;        // [B][d] cross pong
  float* ha = nullptr;        // [B][hmax] MLP ping
  float* hb = nullptr;        // [B][hmax] MLP pong
  rocblas_handle blas = nullptr;
};

namespace {

struct Layout2 {
  size_t y, xa, xb, ha, hb, total;
};

Layout2 dcn_layout(int64_t B, int32_t d, int32_t hmax) {
  auto al = [](size_t x) { return (x + 255) & ~size_t(255); };
  Layout2 L{};
  size_t off = 0;
  const size_t xd = (size_t)B * d * sizeof(float), xh = (size_t)B * hmax * sizeof(float);
  L.y = off;
  off = al(off + xd);
  L.xa = off;
  off = al(off + xd);
  L.xb = off;
  off = al(off + xd);
  L.ha = off;
  off = al(off + xh);
  L.hb = off;
  off = al(off + xh);
  L.total = off;
  return L;
}

dpi_status check_desc(const dpi_dcn_desc* desc, int32_t& hmax) {
  if (!desc) return dpi_fail_status(DPI_ERR_INVALID_ARG, "desc is NULL");
  if (desc->batch < 1 || desc->dim < 1 || desc->n_cross < 1 || desc->n_mlp < 1)
    return dpi_fail_status(DPI_ERR_INVALID_ARG, "batch, dim, n_cross and n_mlp must be >= 1");
  if (desc->batch > INT32_MAX || desc->dim > 65536 || desc->n_cross > 64 || desc->n_mlp > 64)
    return dpi_fail_status(DPI_ERR_UNSUPPORTED, "interaction head too large");
  if (!desc->mlp_dims || !desc->cross_w || !desc->cross_b || !desc->mlp_w || !desc->mlp_b)
    return dpi_fail_status(DPI_ERR_INVALID_ARG, "NULL weight list");
  hmax = 0;
  for (int32_t l = 0; l < desc->n_mlp; ++l) {
    if (desc->mlp_dims[l] < 1 || desc->mlp_dims[l] > 65536) return dpi_fail_status(DPI_ERR_INVALID_ARG, "bad MLP dim");
    hmax = std::max(hmax, desc->mlp_dims[l]);
  }
  for (int32_t l = 0; l < desc->n_cross; ++l)
    if (!desc->cross_w[l] || !desc->cross_b[l]) return dpi_fail_status(DPI_ERR_INVALID_ARG, "NULL cross weight");
  for (int32_t l = 0; l < desc->n_mlp; ++l)
    if (!desc->mlp_w[l] || !desc->mlp_b[l]) return dpi_fail_status(DPI_ERR_INVALID_ARG, "NULL MLP weight");
  return DPI_OK;
}

// Y[rows][dout] = X[rows][din] * W^T, W row-major [dout][din] (fp32)
dpi_status gemm(rocblas_handle h, hipStream_t s, const float* X, const float* W, float* Y, int64_t rows, int32_t din,
                int32_t dout) {
  if (rocblas_set_stream(h, s) != rocblas_status_success)
    return dpi_fail_status(DPI_ERR_HIP, "rocblas_set_stream failed");
  const float one = 1.f, zero = 0.f;
  // column-major view: Y^T (dout x rows) = W (dout x din) * X^T (din x rows)
  const rocblas_status st = rocblas_sgemm(h, rocblas_operation_transpose, rocblas_operation_none, dout, (int)rows, din,
                                          &one, W, din, X, din, &zero, Y, dout);
  if (st != rocblas_status_success) return dpi_fail_status(DPI_ERR_HIP, "rocblas_sgemm failed (%d)", (int)st);
  return DPI_OK;
}

struct OpCtx {
  dpi_dcn_s* head;
  int kind;   // 0 cross gemm, 1 cross fuse, 2 mlp gemm, 3 mlp bias+relu, 4 mark
  const float* x0;
  const float* in;
  const float* w;
  const float* bias;
  const float* prev;
  float* out;
  int32_t din, dout;
  uint64_t* mark;
};

dpi_status run_op(void* ctx, void* stream) {
  const OpCtx& c = *static_cast<const OpCtx*>(ctx);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = hipSuccess;
  switch (c.kind) {
    case 0:
    case 2:
      return gemm(c.head->blas, s, c.in, c.w, c.out, c.head->B, c.din, c.dout);
    case 1:
      e = launch_cross_fuse(c.x0, c.in, c.bias, c.prev, c.out, c.head->B, c.dout, s);
      break;
    case 3:
      e = launch_bias_relu(c.out, c.bias, c.head->B, c.dout, s);
      break;
    case 4:
      e = launch_mark(c.mark, s);
      break;
    default:
      return dpi_fail_status(DPI_ERR_INVALID_ARG, "bad op");
  }
  return e == hipSuccess ? DPI_OK : dpi_hip_status(e, "interaction kernel launch");
}

}  // namespace

extern "C" {

size_t dpi_dcn_workspace_bytes(const dpi_dcn_desc* desc) {
  int32_t hmax = 0;
  if (check_desc(desc, hmax) != DPI_OK) return 0;
  return dcn_layout(desc->batch, desc->dim, hmax).total;
}

dpi_status dpi_dcn_create(const dpi_dcn_desc* desc, void* workspace, size_t workspace_bytes, dpi_dcn_t* out) {
  if (!out) return dpi_fail_status(DPI_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  int32_t hmax = 0;
  const dpi_status st = check_desc(desc, hmax);
  if (st != DPI_OK) return st;
  const Layout2 L = dcn_layout(desc->batch, desc->dim, hmax);
  if (!workspace) return dpi_fail_status(DPI_ERR_INVALID_ARG, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) & 255) return dpi_fail_status(DPI_ERR_MISALIGNED, "workspace not 256-byte aligned");
  if (workspace_bytes < L.total)
    return dpi_fail_status(DPI_ERR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", workspace_bytes, L.total);
  for (int32_t l = 0; l < desc->n_cross; ++l)
    if ((reinterpret_cast<uintptr_t>(desc->cross_b[l]) & 15) && desc->dim % 4 == 0)
      return dpi_fail_status(DPI_ERR_MISALIGNED, "cross bias %d not 16-byte aligned", l);
  for (int32_t l = 0; l < desc->n_mlp; ++l)
    if ((reinterpret_cast<uintptr_t>(desc->mlp_b[l]) & 15) && desc->mlp_dims[l] % 4 == 0)
      return dpi_fail_status(DPI_ERR_MISALIGNED, "MLP bias %d not 16-byte aligned", l);
  dpi_dcn_s* h = new (std::nothrow) dpi_dcn_s();
  if (!h) return dpi_fail_status(DPI_ERR_INVALID_ARG, "out of host memory");
  h->B = desc->batch;
  h->d = desc->dim;
  h->mlp_dims.assign(desc->mlp_dims, desc->mlp_dims + desc->n_mlp);
  h->cw.assign(desc->cross_w, desc->cross_w + desc->n_cross);
  h->cb.assign(desc->cross_b, desc->cross_b + desc->n_cross);
  h->mw.assign(desc->mlp_w, desc->mlp_w + desc->n_mlp);
  h->mb.assign(desc->mlp_b, desc->mlp_b + desc->n_mlp);
  char* ws = static_cast<char*>(workspace);
  h->y = reinterpret_cast<float*>(ws + L.y);
  h->xa = reinterpret_cast<float*>(ws + L.xa);
  h->xb = reinterpret_cast<float*>(ws + L.xb);
  h->ha = reinterpret_cast<float*>(ws + L.ha);
  h->hb = reinterpret_cast<float*>(ws + L.hb);
  if (rocblas_create_handle(&h->blas) != rocblas_status_success) {
    delete h;
    return dpi_fail_status(DPI_ERR_HIP, "rocblas_create_handle failed");
  }
  *out = h;
  return DPI_OK;
}

dpi_status dpi_dcn_forward(dpi_dcn_t head, const float* x0, float* out_cross, float* out_mlp, int32_t mode,
                           void* stream_explicit, void* stream_implicit, void* after, uint64_t* marks) {
  if (!head) return dpi_fail_status(DPI_ERR_INVALID_ARG, "head is NULL");
  if (!x0 || !out_cross || !out_mlp) return dpi_fail_status(DPI_ERR_INVALID_ARG, "NULL activation pointer");
  const bool vec_d = head->d % 4 == 0;
  if (vec_d && ((reinterpret_cast<uintptr_t>(x0) | reinterpret_cast<uintptr_t>(out_cross)) & 15))
    return dpi_fail_status(DPI_ERR_MISALIGNED, "x0 and out_cross must be 16-byte aligned");
  if (head->mlp_dims.back() % 4 == 0 && (reinterpret_cast<uintptr_t>(out_mlp) & 15))
    return dpi_fail_status(DPI_ERR_MISALIGNED, "out_mlp must be 16-byte aligned");
  const int32_t nc = (int32_t)head->cw.size(), nm = (int32_t)head->mw.size();
  std::vector<OpCtx> ex, im;
  ex.reserve(2 * nc + 1);
  im.reserve(2 * nm + 1);
  if (marks) {
    ex.push_back(OpCtx{head, 4, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, 0, marks});
    im.push_back(OpCtx{head, 4, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, 0, marks + 1});
  }
  // cross network: x_{l+1} = x0 * (x_l W_l^T + b_l) + x_l; the last layer writes out_cross
  const float* x = x0;
  for (int32_t l = 0; l < nc; ++l) {
    float* nxt = l == nc - 1 ? out_cross : (l % 2 == 0 ? head->xa : head->xb);
    ex.push_back(OpCtx{head, 0, x0, x, head->cw[l], nullptr, nullptr, head->y, head->d, head->d, nullptr});
    ex.push_back(OpCtx{head, 1, x0, head->y, nullptr, head->cb[l], x, nxt, head->d, head->d, nullptr});
    x = nxt;
  }
  // MLP: h_{l+1} = max(0, h_l V_l^T + c_l); the last layer writes out_mlp
  const float* hcur = x0;
  int32_t din = head->d;
  for (int32_t l = 0; l < nm; ++l) {
    const int32_t dout = head->mlp_dims[l];
    float* nxt = l == nm - 1 ? out_mlp : (l % 2 == 0 ? head->ha : head->hb);
    im.push_back(OpCtx{head, 2, nullptr, hcur, head->mw[l], nullptr, nullptr, nxt, din, dout, nullptr});
    im.push_back(OpCtx{head, 3, nullptr, nullptr, nullptr, head->mb[l], nullptr, nxt, din, dout, nullptr});
    hcur = nxt;
    din = dout;
  }
  std::vector<dpi_op> exo(ex.size()), imo(im.size());
  for (size_t i = 0; i < ex.size(); ++i) exo[i] = dpi_op{run_op, &ex[i]};
  for (size_t i = 0; i < im.size(); ++i) imo[i] = dpi_op{run_op, &im[i]};
  return dpi_launch_two_streams(exo.data(), (int32_t)exo.size(), imo.data(), (int32_t)imo.size(), mode,
                                stream_explicit, stream_implicit, after);
}

void dpi_dcn_destroy(dpi_dcn_t head) {
  if (!head) return;
  if (head->blas) (void)rocblas_destroy_handle(head->blas);
  delete head;
}

}  // extern "C"
