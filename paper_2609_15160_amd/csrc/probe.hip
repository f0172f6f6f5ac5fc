// Measurement probe: the read bandwidth a streaming kernel can reach on this
// device with the load the decode attention uses for the KV cache (16-byte
// non-temporal vector loads), as the practical ceiling its achieved
// bandwidth is compared with.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tlf.h"

namespace {

constexpr int kThreads = 256;
constexpr int kPer = 8;  // 16-byte loads in flight per thread
static_assert(kThreads * kPer * 16 == TLF_PROBE_READ_GRAIN, "grain in tlf.h");

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Each workgroup reads one grain of kThreads x kPer x 16 bytes: load k of
// thread t is vector blockIdx.x * kThreads * kPer + k * kThreads + t, so every
// load instruction of a wave covers 1 KB contiguous.  The loaded words are
// folded into one value that is stored only if it equals a value no real
// buffer produces by chance, which keeps every load without writing memory.
__global__ __launch_bounds__(kThreads) void k_probe_read(const u32x4* __restrict__ buf, unsigned int magic,
                                                         unsigned int* __restrict__ sink) {
  const int64_t base = (int64_t)blockIdx.x * kThreads * kPer + threadIdx.x;
  u32x4 v[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) v[k] = __builtin_nontemporal_load(buf + base + k * kThreads);
  unsigned int acc = 0;
#pragma unroll
  for (int k = 0; k < kPer; ++k) acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
  if (acc == magic) sink[0] = acc;
}

}  // namespace

extern "C" int tlf_probe_read(const void* d_buf, size_t bytes, unsigned int* d_sink, void* stream) {
  if (!d_buf || !d_sink || bytes == 0 || bytes % TLF_PROBE_READ_GRAIN != 0 || ((uintptr_t)d_buf & 15u) != 0)
    return TLF_E_INVALID_ARG;
  const size_t blocks = bytes / TLF_PROBE_READ_GRAIN;
  if (blocks > 0x7FFFFFFFu) return TLF_E_INVALID_ARG;
  hipLaunchKernelGGL(k_probe_read, dim3((unsigned)blocks), dim3(kThreads), 0, (hipStream_t)stream,
                     reinterpret_cast<const u32x4*>(d_buf), 0x9E3779B9u, d_sink);
  return hipGetLastError() == hipSuccess ? TLF_OK : TLF_E_HIP;
}
