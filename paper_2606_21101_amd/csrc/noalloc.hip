// Plan-and-lookup entry point that allocates nothing, for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid it).  Its workspace is a fixed device array of this
// library; each GPU the library runs on holds its own copy of it until the
// process ends.
#include <mutex>

#include "dpi_internal.h"

// the shared internals of dpi_plan and dpi_lookup (api.cpp)
dpi_status dpi_plan_lookup_into(const dpi_table_meta* table_meta, int32_t num_tables, const void* const* tables,
                                const int32_t* ids, const int32_t* offsets, int64_t batch, int64_t total_ids,
                                const int32_t* pooling, const dpi_plan_opts* opts, void* out,
                                int32_t* device_status, void* scratch, size_t scratch_bytes, void* stream);
dpi_status dpi_fail_status(dpi_status s, const char* fmt, ...);
dpi_status dpi_hip_status(hipError_t e, const char* what);

namespace {

// The workspace of every dpi_lookup_noalloc call on a device.  In host code
// this name is only a stand-in for the device array: its device address comes
// from hipGetSymbolAddress, once per device, and only that address is passed
// to kernels.
__device__ __align__(256) unsigned char scratch[DPI_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
void* g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of the current device's scratch array (looked up on the
// device's first call, with that device current).
dpi_status scratch_of_current_device(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return dpi_hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return dpi_fail_status(DPI_ERR_UNSUPPORTED, "device %d", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return dpi_hip_status(e, "hipGetSymbolAddress(scratch)");
    if (!p || (reinterpret_cast<uintptr_t>(p) & 255))
      return dpi_fail_status(DPI_ERR_HIP, "scratch array at an unusable address");
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return DPI_OK;
}

}  // namespace

extern "C" dpi_status dpi_lookup_noalloc(const dpi_table_meta* table_meta, int32_t num_tables,
                                         const void* const* tables, const int32_t* ids, const int32_t* offsets,
                                         int64_t batch, int64_t total_ids, const int32_t* pooling,
                                         const dpi_plan_opts* opts, void* out, int32_t* device_status,
                                         void* stream) {
  void* ws = nullptr;
  const dpi_status st = scratch_of_current_device(&ws);
  if (st != DPI_OK) return st;
  return dpi_plan_lookup_into(table_meta, num_tables, tables, ids, offsets, batch, total_ids, pooling, opts, out,
                              device_status, ws, DPI_NOALLOC_SCRATCH_BYTES, stream);
}
