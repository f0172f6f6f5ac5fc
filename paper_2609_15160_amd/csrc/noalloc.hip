// tlf_gs_plan_noalloc: the multi-workgroup active-set planner of the
// training gather-scatter (tlf_gs_plan_ws) for callers that cannot allocate
// device memory (code under HIP graph capture, tight loops, harnesses that
// forbid hipMalloc).  Its per-chunk counts live in a fixed array of the
// library's own device memory instead of a caller workspace.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "kernels.h"
#include "tlf.h"

// One int32 count per chunk of TLF_GS_PLAN_CHUNK_ROWS rows, up to
// TLF_GS_PLAN_NOALLOC_MAX_ROWS rows (16 KiB).  Every GPU that runs the library
// holds its own copy until the process ends.  In host code this name is only
// a stand-in: the kernels receive the address hipGetSymbolAddress reports for
// the current device.
static __device__ __align__(256) int32_t scratch[TLF_GS_PLAN_NOALLOC_MAX_ROWS / TLF_GS_PLAN_CHUNK_ROWS];

namespace {

constexpr int kMaxDevices = 64;
int32_t* g_scratch[kMaxDevices];  // device address of `scratch` on each device, once looked up
std::mutex g_scratch_mu;

// Address of this device's copy of `scratch`, looked up once per device with
// that device current.
int scratch_on_current_device(int32_t** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return TLF_E_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) return TLF_E_INVALID_ARG;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return TLF_E_HIP;
    }
    g_scratch[dev] = static_cast<int32_t*>(p);
  }
  *out = g_scratch[dev];
  return TLF_OK;
}

}  // namespace

extern "C" int tlf_gs_plan_noalloc(const int32_t* d_depth, int32_t batch, int32_t seq_len, int32_t loop,
                                   int32_t* d_index, int32_t* d_slot, int32_t* d_offsets, int32_t* d_count,
                                   void* stream) {
  int64_t rows = 0;
  int st = tlf::gs_plan_chunked_args(d_depth, batch, seq_len, d_index, d_count, TLF_GS_PLAN_NOALLOC_MAX_ROWS, &rows);
  if (st != TLF_OK) return st;
  int32_t* counts = nullptr;
  st = scratch_on_current_device(&counts);
  if (st != TLF_OK) return st;
  // every count the second launch reads is written by the first: nothing to clear
  return tlf::launch_gs_plan_chunked(d_depth, batch, seq_len, loop, d_index, d_slot, d_offsets, d_count, counts,
                                     rows, (hipStream_t)stream);
}
